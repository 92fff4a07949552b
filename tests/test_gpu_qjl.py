"""GPU parity of the qjl rotation (Sec. 4.2: encode applies a caller-supplied
orthogonal S after the normalization, decode S^T after the undither), against
the oracle: KV streams (dither, fp16 norms, appended in chunks) with codes
and words bit-exact on every lattice and the decode within 1e-5 of the
lattice unit (its S^T y runs on the matrix cores), the fused attention over
qjl streams, and the entry points that take no qjl plan.  S is a Haar draw made on the host (QR of a seeded
Gaussian matrix with the sign fix)."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from tests import parity as PT
from tests.test_gpu_attention import check, paged
from tests.test_gpu_parity import check_roundtrip, gauss

pytestmark = pytest.mark.gpu

LAT_NAMES = {O.E8: "E8", O.D4: "D4", O.A2: "A2", O.Z: "Z"}
SNR = {O.E8: PT.op_snr("E8", 2.0), O.D4: 12.0, O.A2: PT.op_snr("A2", 1.7), O.Z: PT.op_snr("Z", 1.7)}
N = 128


@pytest.fixture(scope="module")
def hq():
    from paper_2606_23406_amd import hq as H
    H.lib()
    assert torch.cuda.is_available()
    return H


def haar(seed):
    g = np.random.default_rng(seed).standard_normal((N, N))
    q, r = np.linalg.qr(g)
    return (q * np.sign(np.diag(r))).astype(np.float32)


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.A2, O.Z])
def test_qjl_kv_roundtrip(hq, lat):
    # 48 rows x 1024 appended 16 at a time: codes, words and the fp32 decode
    # against the oracle at the bar of the other KV tests
    P = PT.oracle_params(lat, SNR[lat], rht_seed=3, rotation=2, dither=True, dither_seed=1234 + lat,
                         norm_fp16=True, qjl=haar(20 + lat))
    x = gauss(48, 1024, 50 + lat, 1.0, torch.bfloat16)
    x[:, 5::128] *= 10
    check_roundtrip(hq, P, SNR[lat], x, f"qjl kv {LAT_NAMES[lat]}", append_chunks=16)


@pytest.mark.parametrize("lat", [O.E8, O.Z])
def test_qjl_without_dither(hq, lat):
    P = PT.oracle_params(lat, SNR[lat], rht_seed=4, rotation=2, qjl=haar(30 + lat))
    x = gauss(40, 512, 60 + lat, 1.0, torch.bfloat16)
    check_roundtrip(hq, P, SNR[lat], x, f"qjl no dither {LAT_NAMES[lat]}")


def coded(hq, P, x, chunk=16):
    rows, cols = x.shape
    plan = PT.gpu_plan(hq, P, SNR[P.lattice], cols)
    s = hq.EncodedStream(plan, rows)
    xd = x.cuda()
    for r0 in range(0, rows, chunk):
        hq.hq_encode(plan, xd[r0:r0 + chunk], s, append=r0 > 0)
    torch.cuda.synchronize()
    res = PT.compare_streams(P, x.float().numpy(), PT.gpu_stream_arrays(s, rows))
    codes = res["codes"] if res["gpu_codes"] is None else res["gpu_codes"]
    return plan, s, codes, res["norms"]


@pytest.mark.parametrize("lat", [O.E8, O.A2])
def test_qjl_attention(hq, lat):
    # keys and values with their own Haar rotations; 8 KV heads, 4 query heads each
    rng = np.random.default_rng(70 + lat)
    g = torch.Generator().manual_seed(71 + lat)
    k = torch.randn((40 * 16, 8 * N), generator=g)
    k[:, 3::N] *= 10
    v = torch.randn((40 * 16, 8 * N), generator=g)
    k, v = k.to(torch.bfloat16), v.to(torch.bfloat16)
    pk = PT.oracle_params(lat, SNR[lat], rht_seed=41, rotation=2, dither=True, dither_seed=43,
                          norm_fp16=True, qjl=haar(44))
    pv = PT.oracle_params(lat, SNR[lat], rht_seed=51, rotation=2, dither=True, dither_seed=53,
                          norm_fp16=True, qjl=haar(54))
    K, V = (pk,) + coded(hq, pk, k), (pv,) + coded(hq, pv, v)
    lens = [300, 17, 0, 190]
    table = paged(rng, lens, 16, 40)
    q = torch.from_numpy(rng.standard_normal((4, 32, N)).astype(np.float32))
    check(hq, K, V, q, table, lens, 16, f"qjl attention {LAT_NAMES[lat]}")


def test_qjl_plan_rules(hq):
    S = haar(5)
    with pytest.raises(hq.HQError):  # qjl without a matrix
        hq.hq_plan(128, hq.HQ_E8, 0.0, 1, -1, 512, rotation=hq.HQ_ROT_QJL, snr_db=12.0)
    plan = hq.hq_plan(128, hq.HQ_E8, 0.0, 1, -1, 512, rotation=hq.HQ_ROT_QJL, snr_db=12.0, qjl=S)
    s = hq.EncodedStream(plan, 4)
    x = torch.randn((4, 512), device="cuda")
    with pytest.raises(hq.HQError):  # group launches take no qjl plan
        hq.hq_encode_group([plan], [x], [s])
    hq.hq_encode(plan, x, s)
    with pytest.raises(hq.HQError):  # nor the int8 codes path (rotated codes)
        hq.hq_decode_int8(plan, s)
    torch.cuda.synchronize()


@pytest.mark.parametrize("row0,rows", [(0, 7), (5, 33), (37, 13), (49, 1)])
def test_qjl_partial_decodes_match_the_whole(hq, row0, rows):
    # the matrix-core decode takes 16 sub-streams per pass; a tile's result
    # does not depend on which tiles share its pass, so a row range decoded
    # alone (ragged passes, row0 past the first pass) equals those rows of
    # the whole decode bit for bit, in fp32 and in bf16
    P = PT.oracle_params(O.E8, SNR[O.E8], rht_seed=6, rotation=2, dither=True, dither_seed=7,
                         norm_fp16=True, qjl=haar(8))
    x = gauss(50, 1024, 9, 1.0, torch.bfloat16)
    plan = PT.gpu_plan(hq, P, SNR[O.E8], 1024)
    s = hq.EncodedStream(plan, 50)
    hq.hq_encode(plan, x.cuda(), s)
    print(f"[qjl] partial decode rows {row0}..{row0 + rows - 1} of 50", flush=True)
    for dt in (torch.float32, torch.bfloat16):
        whole = hq.hq_decode(plan, s, out_dtype=dt)
        part = hq.hq_decode(plan, s, row0=row0, rows=rows, out_dtype=dt)
        torch.cuda.synchronize()
        assert torch.equal(part.cpu(), whole[row0:row0 + rows].cpu()), dt
    assert s.read_stats()["status"] == 0
