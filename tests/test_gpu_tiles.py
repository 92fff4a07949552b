"""GPU parity of the codec at RHT tiles of 256 .. 2048 (Sec. 7.2 sweeps the
tile over 128 .. 2048 for the weight path), through the C ABI, against the
oracle: streams bit-exact per sub-stream (the same exemption rule as the
128-tile tests), fp32 reconstruction bit-exact and bf16 = RNE of it, on
ragged row counts (a partial last workgroup) and at the C2 size."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from tests import parity as PT

pytestmark = pytest.mark.gpu

TILES = [256, 512, 1024, 2048]
NAMES = {O.E8: "E8", O.D4: "D4", O.A2: "A2", O.Z: "Z"}


@pytest.fixture(scope="module")
def hq():
    from paper_2606_23406_amd import hq as H
    H.lib()
    assert torch.cuda.is_available()
    return H


def roundtrip(hq, P, snr, x, label):
    rows, cols = x.shape
    n = P.tile
    print(f"[tiles] {label} tile={n} shape={tuple(x.shape)} dtype={x.dtype}", flush=True)
    plan = PT.gpu_plan(hq, P, snr, cols)
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
    unit = PT.lattice_unit(P, res["norms"]).reshape(rows, -1)
    err = np.abs(y32.astype(np.float64) - ref).reshape(rows, -1, n).max(axis=2)
    assert np.all(err[~skip] <= 1e-5 * unit[~skip]), err.max()
    exact = np.mean(y32.reshape(rows, -1, n)[~skip] == ref.reshape(rows, -1, n)[~skip])
    ref16 = torch.from_numpy(ref).to(torch.bfloat16).float().numpy()
    assert np.all((y16 == ref16).reshape(rows, -1, n)[~skip])
    print(f"[tiles] {label} tile={n}: {res['substreams']} sub-streams, exempt blocks "
          f"{res['exempt_blocks']}, fp32 bit-exact fraction {exact:.6f}, "
          f"{res['payload_bits'] / x.numel():.4f} b/s", flush=True)
    return exact


def gauss(rows, cols, seed, scale=0.02, dtype=torch.bfloat16):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn((rows, cols), generator=g) * scale).to(dtype)


@pytest.mark.parametrize("tile", TILES)
def test_e8_tiles_bf16(hq, tile):
    # 37 rows x 4096: 296 sub-streams, the last workgroup partial
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=17 + tile, tile=tile)
    x = gauss(37, 4096, 300 + tile)
    x[:, 77] *= 20  # an outlier column
    assert roundtrip(hq, P, snr, x, "E8@4 bf16") == 1.0


@pytest.mark.parametrize("tile", [256, 2048])
@pytest.mark.parametrize("lat", [O.D4, O.A2, O.Z])
def test_other_lattices_tiles(hq, lat, tile):
    snr = {O.D4: PT.op_snr("D4", 3.0), O.A2: PT.op_snr("A2", 4.0), O.Z: PT.op_snr("Z", 4.0)}[lat]
    P = PT.oracle_params(lat, snr, rht_seed=5 + lat, tile=tile)
    x = gauss(21, 2048, 400 + lat + tile)
    assert roundtrip(hq, P, snr, x, f"{NAMES[lat]} bf16") == 1.0


@pytest.mark.parametrize("tile", [512, 1024])
def test_fp32_input_and_fixed_k(hq, tile):
    snr = 17.0
    P = PT.oracle_params(O.E8, snr, rht_seed=9, rice_k=2, tile=tile)
    x = gauss(19, 4096, 500 + tile, 1.0, torch.float32)
    roundtrip(hq, P, snr, x, "E8 fp32 k=2")


@pytest.mark.parametrize("tile", [256, 1024])
def test_zero_and_nonfinite_tiles(hq, tile):
    # a zero tile and a non-finite tile at a long tile: zero codes, the
    # overflow reported once per bad tile, every other tile bit-exact
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=31, tile=tile)
    x = gauss(8, 4096, 600 + tile)
    x[2, :tile] = 0.0
    x[5, tile + 3] = float("inf")
    xn = x.float().numpy()
    codes, norms, _, rc = O.frontend(P, xn)
    assert rc == O.ERR_OVERFLOW
    o_pay, o_off, o_kp, _ = O.pack(P, codes)
    plan = PT.gpu_plan(hq, P, snr, 4096)
    s = hq.EncodedStream(plan, 8)
    hq.hq_encode(plan, x.cuda(), s)
    torch.cuda.synchronize()
    st = s.read_stats()
    assert st["status"] == (-4 & 0xFFFFFFFF) and st["overflow_tiles"] == 1, st
    g_pay, g_off, g_kp, g_norm = PT.gpu_stream_arrays(s, 8)
    assert np.array_equal(g_off, o_off) and np.array_equal(g_kp, o_kp)
    assert np.array_equal(g_pay, o_pay[:o_off[-1]])
    bad = ~np.isfinite(norms)
    assert np.array_equal(g_norm[~bad].view(np.uint32), norms[~bad].view(np.uint32))
    y = hq.hq_decode(plan, s, out_dtype=torch.float32).cpu()
    assert torch.all(y[2, :tile] == 0)


def test_long_tiles_reject_the_128_paths(hq):
    # the int8 / fp8 / MXFP4 casts, the GEMM, the fused GEMV and group launches are
    # built for 128-tiles: a long-tile plan gets HQ_ERR_UNSUPPORTED
    snr = PT.op_snr("E8", 4.0)
    plan = hq.hq_plan(512, hq.HQ_E8, 0.0, 1, -1, 2048, snr_db=snr)
    s = hq.EncodedStream(plan, 4)
    x = gauss(4, 2048, 7).cuda()
    hq.hq_encode(plan, x, s)
    for fn in (lambda: hq.hq_decode_int8(plan, s), lambda: hq.hq_decode_fp8(plan, s),
               lambda: hq.hq_decode_gemv(plan, s, x[0].contiguous()),
               lambda: hq.hq_encode_group([plan], [x], [hq.EncodedStream(plan, 4)]),
               lambda: hq.hq_act_prep(plan, x), lambda: hq.hq_decode_mxfp4(plan, s),
               lambda: hq.hq_act_prep_mxfp4(plan, x)):
        with pytest.raises(hq.HQError) as e:
            fn()
        assert e.value.status == -2


@pytest.mark.parametrize("tile", TILES)
def test_c2_whole_stream_per_tile(hq, tile):
    """C2 (4096 x 4096 bf16, Student-t with outlier columns) at E8 @ 4 bps for
    each long tile: every sub-stream bit-exact, every row's fp32 decode equal
    to the oracle's reconstruction."""
    from paper_2606_23406_amd import workloads
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=2, tile=tile)
    x = workloads.heavy_tailed_weight()
    assert roundtrip(hq, P, snr, x, "C2 E8@4") == 1.0
