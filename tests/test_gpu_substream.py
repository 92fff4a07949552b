"""GPU parity of sub-streams of S = 1024 and 2048 symbols (Sec. 5.3: S trades
metadata against parallel occupancy; 512 is the default) for weight plans,
through the C ABI, against the oracle: every sub-stream's words, word
offsets and k bytes bit-exact (the same exemption rule as the 512-symbol
tests), the fp32 reconstruction bit-exact and bf16 its RNE rounding, at tile
128 and at long tiles (a tile holding several sub-streams, and a sub-stream
holding several tiles), on ragged row counts.  The paths built for S = 512
only (KV plans, the int8 / fp8 / MXFP4 casts, the fused GEMV, group calls)
return HQ_ERR_UNSUPPORTED."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from tests import parity as PT
from tests.test_gpu_tiles import gauss

pytestmark = pytest.mark.gpu

NAMES = {O.E8: "E8", O.D4: "D4", O.A2: "A2", O.Z: "Z"}


@pytest.fixture(scope="module")
def hq():
    from paper_2606_23406_amd import hq as H
    H.lib()
    assert torch.cuda.is_available()
    return H


def roundtrip(hq, P, snr, x, label):
    rows, cols = x.shape
    n, S = P.tile, P.substream
    print(f"[substream] {label} S={S} tile={n} shape={tuple(x.shape)} dtype={x.dtype}", flush=True)
    plan = PT.gpu_plan(hq, P, snr, cols)
    assert plan.info.subs_per_row == cols // S
    s = hq.EncodedStream(plan, rows)
    hq.hq_encode(plan, x.cuda(), s)
    torch.cuda.synchronize()
    st = s.read_stats()
    assert st["status"] == 0, st
    res = PT.compare_streams(P, x.float().numpy(), PT.gpu_stream_arrays(s, rows))
    assert res["exempt_blocks"] <= max(2, res["substreams"] // 1000), res["exempt_blocks"]
    assert st["payload_bits"] == res["payload_bits"] or res["exempt_substreams"] > 0
    y32 = hq.hq_decode(plan, s, out_dtype=torch.float32).cpu().numpy()
    y16 = hq.hq_decode(plan, s, out_dtype=torch.bfloat16).cpu().float().numpy()
    torch.cuda.synchronize()
    assert s.read_stats()["corrupt_substreams"] == 0
    ref = O.backend(P, res["codes"], res["norms"])
    skip = PT.tiles_with_code_diffs(res["codes"], res["gpu_codes"], tile=n).reshape(rows, -1)
    exact = np.mean(y32.reshape(rows, -1, n)[~skip] == ref.reshape(rows, -1, n)[~skip])
    ref16 = torch.from_numpy(ref).to(torch.bfloat16).float().numpy()
    assert np.all((y16 == ref16).reshape(rows, -1, n)[~skip])
    print(f"[substream] {label} S={S} tile={n}: {res['substreams']} sub-streams, exempt blocks "
          f"{res['exempt_blocks']}, fp32 bit-exact fraction {exact:.6f}, "
          f"{res['payload_bits'] / x.numel():.4f} b/s", flush=True)
    # a row range decodes to the same values as the whole stream's rows
    r0, nr = rows // 3, rows - rows // 3 - 1
    part = hq.hq_decode(plan, s, row0=r0, rows=nr, out_dtype=torch.float32).cpu().numpy()
    assert np.array_equal(part, y32[r0:r0 + nr])
    return exact


@pytest.mark.parametrize("S", [1024, 2048])
def test_e8_substreams_bf16(hq, S):
    # 37 rows x 4096: the last workgroup partial
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=31 + S, substream=S)
    x = gauss(37, 4096, 500 + S)
    x[:, 91] *= 20  # an outlier column
    x[5] = 0.0  # an all-zero row
    assert roundtrip(hq, P, snr, x, "E8@4 bf16") == 1.0


@pytest.mark.parametrize("S", [1024, 2048])
@pytest.mark.parametrize("lat", [O.D4, O.A2, O.Z])
def test_other_lattices_substreams(hq, lat, S):
    snr = {O.D4: PT.op_snr("D4", 3.0), O.A2: PT.op_snr("A2", 4.0), O.Z: PT.op_snr("Z", 4.0)}[lat]
    P = PT.oracle_params(lat, snr, rht_seed=9 + lat, substream=S)
    x = gauss(21, 2048, 600 + lat + S)
    assert roundtrip(hq, P, snr, x, f"{NAMES[lat]} bf16") == 1.0


@pytest.mark.parametrize("tile,S", [(2048, 1024), (512, 2048), (1024, 2048)])
def test_long_tiles_with_substreams(hq, tile, S):
    # a tile over several sub-streams (2048 over 1024) and sub-streams over
    # several tiles (2048 over 512 and 1024); fp32 input
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=41 + tile, tile=tile, substream=S)
    x = gauss(13, 4096, 700 + tile + S, dtype=torch.float32)
    assert roundtrip(hq, P, snr, x, "E8@4 fp32") == 1.0


@pytest.mark.parametrize("S", [1024, 2048])
def test_fixed_k_substreams(hq, S):
    snr = PT.op_snr("E8", 3.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=43, rice_k=2, substream=S)
    x = gauss(9, 2048, 800 + S)
    assert roundtrip(hq, P, snr, x, "E8@3 k=2 bf16") == 1.0


def test_substreams_reject_the_512_paths(hq):
    snr = PT.op_snr("E8", 4.0)
    plan = hq.hq_plan(128, hq.HQ_E8, 0.0, 1, -1, 2048, snr_db=snr, substream=1024)
    s = hq.EncodedStream(plan, 4)
    x = gauss(4, 2048, 7).cuda()
    hq.hq_encode(plan, x, s)
    for fn in (lambda: hq.hq_decode_int8(plan, s), lambda: hq.hq_decode_fp8(plan, s),
               lambda: hq.hq_decode_mxfp4(plan, s),
               lambda: hq.hq_decode_gemv(plan, s, x[0].contiguous()),
               lambda: hq.hq_encode_group([plan], [x], [hq.EncodedStream(plan, 4)])):
        with pytest.raises(hq.HQError) as e:
            fn()
        assert e.value.status == -2
    # KV plans (rotation, dither, fp16 norms) and other lengths keep S = 512
    for kw in (dict(rotation=1, rot_seed=3), dict(dither=True, dither_seed=4), dict(norm_fp16=True)):
        with pytest.raises(hq.HQError) as e:
            hq.hq_plan(128, hq.HQ_E8, 0.0, 1, -1, 2048, snr_db=snr, substream=1024, **kw)
        assert e.value.status == -2
    for S in (256, 4096):
        with pytest.raises(hq.HQError) as e:
            hq.hq_plan(128, hq.HQ_E8, 0.0, 1, -1, 8192, snr_db=snr, substream=S)
        assert e.value.status == -2


@pytest.mark.parametrize("S", [1024, 2048])
def test_c2_whole_stream_per_substream_length(hq, S):
    """C2 (4096 x 4096 bf16, Student-t with outlier columns) at E8 @ 4 bps with
    sub-streams of S symbols, in the launch configuration the bench times:
    every sub-stream bit-exact, every row's fp32 decode equal to the oracle's
    reconstruction."""
    from paper_2606_23406_amd import workloads
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=2, substream=S)
    x = workloads.heavy_tailed_weight()
    assert roundtrip(hq, P, snr, x, "C2 E8@4") == 1.0
