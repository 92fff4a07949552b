"""GPU parity of the HIP codec (through the C ABI) against the oracle.

Bar: lattice indices and Rice bitstreams bit-exact per sub-stream, except
blocks whose oracle Voronoi margin is below 1e-6 (counted, and their
sub-stream must be exactly the oracle's Rice code of the GPU's symbols);
reconstruction within 1e-5 of the tile's lattice unit in fp32 (bit-exact in
practice); GEMM within 1e-3 relative to max(|ref|, rms(ref)).
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from tests import parity as PT

pytestmark = pytest.mark.gpu

LAT_NAMES = {O.E8: "E8", O.D4: "D4", O.A2: "A2", O.Z: "Z"}


@pytest.fixture(scope="module")
def hq():
    from paper_2606_23406_amd import hq as H
    H.lib()
    assert torch.cuda.is_available()
    return H


def encode_gpu(hq, P, snr, x, rows_capacity=None, append_chunks=None):
    rows, cols = x.shape
    plan = PT.gpu_plan(hq, P, snr, cols)
    s = hq.EncodedStream(plan, rows_capacity or rows)
    xd = x.cuda()
    if append_chunks:
        for r0 in range(0, rows, append_chunks):
            hq.hq_encode(plan, xd[r0:r0 + append_chunks], s, append=r0 > 0)
    else:
        hq.hq_encode(plan, xd, s)
    torch.cuda.synchronize()
    return plan, s


def check_roundtrip(hq, P, snr, x, label, append_chunks=None):
    print(f"[parity] {label} shape={tuple(x.shape)} dtype={x.dtype}", flush=True)
    plan, s = encode_gpu(hq, P, snr, x, append_chunks=append_chunks)
    rows = x.shape[0]
    st = s.read_stats()
    assert st["status"] == 0, st
    gpu = PT.gpu_stream_arrays(s, rows)
    x_np = x.float().numpy()
    res = PT.compare_streams(P, x_np, gpu)
    assert res["exempt_blocks"] <= max(2, res["substreams"] // 1000), res["exempt_blocks"]
    assert st["payload_bits"] == res["payload_bits"] or res["exempt_substreams"] > 0
    # decode: fp32 against the oracle's fp32 reconstruction, bf16 = bf16(that)
    y32 = hq.hq_decode(plan, s, out_dtype=torch.float32)
    y16 = hq.hq_decode(plan, s, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    st2 = s.read_stats()
    assert st2["corrupt_substreams"] == 0
    ref = O.backend(P, res["codes"], res["norms"], row0=0)
    g = y32.cpu().numpy()
    skip = PT.tiles_with_code_diffs(res["codes"], res["gpu_codes"]).reshape(rows, -1)
    unit = PT.lattice_unit(P, res["norms"]).reshape(rows, -1)
    err = np.abs(g.astype(np.float64) - ref).reshape(rows, -1, 128).max(axis=2)
    assert np.all(err[~skip] <= 1e-5 * unit[~skip]), err.max()
    exact = np.mean(g.reshape(rows, -1, 128)[~skip] == ref.reshape(rows, -1, 128)[~skip])
    # bf16 output = RNE(fp32 reconstruction); compared by value (+0 == -0).
    # The qjl decode sums S^T y on the matrix cores, equal to the oracle's
    # left-to-right fp32 sums only to rounding (the tolerance above), so its
    # bf16 output is held to RNE of its own fp32 output.
    ref16 = torch.from_numpy(g if P.rotation == 2 else ref).to(torch.bfloat16).float()
    b16 = (y16.cpu().float() == ref16).numpy().reshape(rows, -1, 128)
    assert b16[~skip].all()
    print(f"[parity] {label}: {res['substreams']} sub-streams, exempt blocks "
          f"{res['exempt_blocks']}, fp32 bit-exact fraction {exact:.6f}", flush=True)
    return plan, s, res


def gauss(rows, cols, seed, scale=1.0, dtype=torch.float32):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn((rows, cols), generator=g) * scale).to(dtype)


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.A2, O.Z])
def test_weights_roundtrip_bf16(hq, lat):
    # 63 rows x 1024: 126 sub-streams, so the last workgroup is ragged
    snr = {O.E8: PT.op_snr("E8", 4.0), O.D4: PT.op_snr("D4", 3.0), O.A2: PT.op_snr("A2", 4.0),
           O.Z: PT.op_snr("Z", 4.0)}[lat]
    P = PT.oracle_params(lat, snr, rht_seed=11)
    x = gauss(63, 1024, 100 + lat, 0.02, torch.bfloat16)
    check_roundtrip(hq, P, snr, x, f"weights {LAT_NAMES[lat]}")


def test_single_matrix_fp32_e8(hq):
    from paper_2606_23406_amd import workloads
    x = torch.from_numpy(workloads.single_matrix_fp32())
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=0)
    check_roundtrip(hq, P, snr, x, "512x512 fp32 E8@4")


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.A2, O.Z])
@pytest.mark.parametrize("rice_k", [0, 2, 5])
def test_fixed_rice_k(hq, lat, rice_k):
    snr = 15.0
    P = PT.oracle_params(lat, snr, rht_seed=5, rice_k=rice_k)
    x = gauss(16, 2048, 7 + lat, 1.0)
    check_roundtrip(hq, P, snr, x, f"fixed k={rice_k} {LAT_NAMES[lat]}")


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.A2, O.Z])
def test_kv_rotation_dither_fp16_append(hq, lat):
    # KV path: signs rotation + subtractive dither + fp16 norms, appended in
    # chunks of 16 rows; the oracle encodes all rows at once.
    snr = {O.E8: PT.op_snr("E8", 2.0), O.D4: 12.0, O.A2: PT.op_snr("A2", 1.7),
           O.Z: PT.op_snr("Z", 1.7)}[lat]
    P = PT.oracle_params(lat, snr, rht_seed=3, rotation=1, rot_seed=99, dither=True,
                         dither_seed=1234 + lat, norm_fp16=True)
    x = gauss(48, 1024, 50 + lat, 1.0, torch.bfloat16)
    x[:, 5::128] *= 10  # outlier channels
    check_roundtrip(hq, P, snr, x, f"kv {LAT_NAMES[lat]}", append_chunks=16)


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.A2, O.Z])
def test_exact_zeros_after_the_rht(hq, lat):
    """Tiles whose RHT output is exactly a sparse integer vector v (x = D H v /
    128, exact in bf16): most coordinates of z are exact zeros, which the
    GPU's sign-twisted transform and signed scale turn into -0 on half of the
    lanes.  Codes and streams must still be the oracle's (regression test for
    an E8 parity read from the sign bit of a -0 rounding error)."""
    rng = np.random.default_rng(500 + lat)
    rows, cols, n = 48, 1024, 128
    v = np.zeros((rows, cols))
    for r in range(rows):
        for t in range(cols // n):
            k = rng.integers(1, 4)
            idx = rng.choice(n, k, replace=False)
            v[r, t * n + idx] = rng.integers(-3, 4, k)
    x = O.fwht(v.reshape(-1, n)).reshape(rows, cols) / n * O.signs(19, cols)
    xt = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16)
    assert np.array_equal(xt.float().numpy(), x.astype(np.float32))  # exact in bf16
    snr = 20.0
    P = PT.oracle_params(lat, snr, rht_seed=19)
    check_roundtrip(hq, P, snr, xt, f"exact zeros after the RHT {LAT_NAMES[lat]}")


def test_zero_tiles_and_tiny_norms(hq):
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=2)
    x = gauss(8, 1024, 3, 0.02)
    x[1] = 0.0
    x[2, 128:256] = 0.0
    x[3, :128] = 1e-30
    plan, s, res = check_roundtrip(hq, P, snr, x, "zero tiles")
    y = hq.hq_decode(plan, s, out_dtype=torch.float32).cpu()
    assert torch.all(y[1] == 0) and torch.all(y[2, 128:256] == 0)


def test_fp16_norm_overflow_is_reported(hq):
    P = PT.oracle_params(O.E8, 20.0, norm_fp16=True)
    x = gauss(4, 512, 1, 1e5)
    plan = PT.gpu_plan(hq, P, 20.0, 512)
    s = hq.EncodedStream(plan, 4)
    hq.hq_encode(plan, x.cuda(), s)
    torch.cuda.synchronize()
    st = s.read_stats()
    assert st["status"] == (-4 & 0xFFFFFFFF) and st["overflow_tiles"] == 16


def test_empty_and_capacity_errors(hq):
    P = PT.oracle_params(O.E8, 20.0)
    plan = PT.gpu_plan(hq, P, 20.0, 1024)
    s = hq.EncodedStream(plan, 4)
    hq.hq_encode(plan, torch.zeros((0, 1024), device="cuda"), s)
    assert s.rows == 0
    with pytest.raises(hq.HQError):
        hq.hq_encode(plan, torch.zeros((5, 1024), device="cuda"), s)


def test_deterministic_bitstream(hq):
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=8)
    x = gauss(256, 4096, 9, 0.02, torch.bfloat16).cuda()
    plan = PT.gpu_plan(hq, P, snr, 4096)
    a = hq.EncodedStream(plan, 256)
    b = hq.EncodedStream(plan, 256)
    hq.hq_encode(plan, x, a)
    hq.hq_encode(plan, x, b)
    hq.hq_encode(plan, x, b)  # re-encode over the same buffers (new scan epoch)
    torch.cuda.synchronize()
    n = a.end_words()
    assert n == b.end_words()
    assert torch.equal(a.payload[:n], b.payload[:n]) and torch.equal(a.offsets, b.offsets)


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.Z])
def test_decode_int8_codes_and_factors(hq, lat):
    snr = PT.op_snr("E8", 4.0) if lat == O.E8 else 16.0
    P = PT.oracle_params(lat, snr, rht_seed=21)
    x = gauss(40, 1024, 31, 0.02, torch.bfloat16)
    print(f"[parity] decode_int8 {LAT_NAMES[lat]}", flush=True)
    plan, s = encode_gpu(hq, P, snr, x)
    codes, g = hq.hq_decode_int8(plan, s)
    torch.cuda.synchronize()
    oc, norms, _, _ = O.frontend(P, x.float().numpy())
    og = O.weight_factors(P, norms, 40, 1024)
    assert np.array_equal(codes.cpu().numpy().astype(np.int32), np.clip(oc, -127, 127))
    assert np.array_equal(g.cpu().numpy(), og)


def test_act_prep(hq):
    from paper_2606_23406_amd import workloads
    a = workloads.activations(tokens=64, features=1024)
    P = PT.oracle_params(O.E8, 20.0, rht_seed=41)
    plan = PT.gpu_plan(hq, P, 20.0, 1024)
    print("[parity] act_prep 64x1024", flush=True)
    xq, sx = hq.hq_act_prep(plan, a.cuda())
    torch.cuda.synchronize()
    oxq, osx = O.act_prep(a.float().numpy(), 128, 41)
    assert np.array_equal(sx.cpu().numpy(), osx)
    assert np.array_equal(xq.cpu().numpy(), oxq)


@pytest.mark.parametrize("M,N,K", [(128, 256, 1024), (200, 384, 1024), (64, 96, 1024),
                                   (300, 200, 512), (40, 136, 2560), (70, 100, 512)])
def test_gemm_int8_blockscaled(hq, M, N, K):
    # K = 512: four stages (the shortest K a plan takes); 2560: twenty, the LDS ring wrapping;
    # N = 100: bf16 output rows of 200 bytes, every other one off 16-byte alignment (element stores)
    from paper_2606_23406_amd import workloads
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=51)
    w = gauss(N, K, 61, 0.02, torch.bfloat16)
    a = workloads.activations(tokens=M, features=K)
    print(f"[parity] gemm M={M} N={N} K={K}", flush=True)
    plan, s = encode_gpu(hq, P, snr, w)
    out32 = hq.hq_dequant_gemm_int8(plan, s, a.cuda(), out_dtype=torch.float32)
    out16 = hq.hq_dequant_gemm_int8(plan, s, a.cuda(), out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    codes, norms, _, _ = O.frontend(P, w.float().numpy())
    g = O.weight_factors(P, norms, N, K)
    xq, sx = O.act_prep(a.float().numpy(), 128, 51)
    ref = O.gemm_blockscaled(codes, g, xq, sx, 128)
    got = out32.cpu().numpy().astype(np.float64)
    denom = np.maximum(np.abs(ref), np.sqrt((ref ** 2).mean()))
    assert np.max(np.abs(got - ref) / denom) <= 1e-3
    ref16 = torch.from_numpy(ref.astype(np.float32)).to(torch.bfloat16).float().numpy()
    got16 = out16.cpu().float().numpy()
    # one bf16 ulp of the reference, or fp32 accumulation noise near zero
    tol = np.maximum(np.abs(ref16) * 2.0 ** -7, 1e-5 * np.sqrt((ref ** 2).mean()))
    assert np.all(np.abs(got16 - ref16) <= tol)


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.Z])
def test_group_calls_match_single_calls(hq, lat):
    """hq_encode_group / hq_decode_group give the single-matrix calls' bits:
    eighteen matrices of mixed shapes and seeds (more than one launch's worth
    of members), ragged row counts, bf16 and fp32 outputs."""
    shapes = [(64, 4096), (16, 1024), (40, 512), (1, 1536), (7, 2048), (33, 512), (128, 1024),
              (5, 4096), (2, 512), (19, 1536), (3, 1024), (11, 512), (6, 2048), (1, 512), (9, 1024),
              (4, 1536), (17, 512), (2, 4096)]
    print(f"[parity] group {LAT_NAMES[lat]} x{len(shapes)}", flush=True)
    snr = 20.0
    plans, xs, grp, one = [], [], [], []
    for i, (r, c) in enumerate(shapes):
        plan = hq.hq_plan(128, lat, 0.0, 300 + i, -1, c, snr_db=snr)
        plans.append(plan)
        xs.append(gauss(r, c, 400 + i, 0.02, torch.bfloat16).cuda())
        grp.append(hq.EncodedStream(plan, r))
        one.append(hq.EncodedStream(plan, r))
    hq.hq_encode_group(plans, xs, grp)
    for plan, x, s in zip(plans, xs, one):
        hq.hq_encode(plan, x, s)
    torch.cuda.synchronize()
    for a, b in zip(grp, one):
        assert a.rows == b.rows
        n = b.end_words()
        assert a.end_words() == n
        assert torch.equal(a.payload[:n], b.payload[:n])
        assert torch.equal(a.offsets, b.offsets) and torch.equal(a.kparam, b.kparam)
        assert torch.equal(a.norms, b.norms)
        assert a.read_stats() == b.read_stats()
    for dt in (torch.bfloat16, torch.float32):
        ys = [torch.empty(x.shape, dtype=dt, device="cuda") for x in xs]
        hq.hq_decode_group(plans, grp, ys)
        for plan, s, y in zip(plans, one, ys):
            assert torch.equal(y, hq.hq_decode(plan, s, out_dtype=dt))


@pytest.mark.parametrize("rows", [2048, 2049])
def test_launch_shapes_agree_at_the_small_launch_bound(hq, rows):
    """A single encode of at most 16384 sub-streams runs one sub-stream per
    wave (sixteen waves per workgroup), a larger one and every group launch
    four per wave: the same matrix through both shapes gives the same bits.
    2048 x 4096 is exactly 16384 sub-streams; one more row crosses over."""
    print(f"[parity] launch shapes rows={rows}", flush=True)
    plan = hq.hq_plan(128, O.E8, 0.0, 77, -1, 4096, snr_db=20.0)
    x = gauss(rows, 4096, 78, 0.02, torch.bfloat16).cuda()
    a, b = hq.EncodedStream(plan, rows), hq.EncodedStream(plan, rows)
    hq.hq_encode(plan, x, a)
    hq.hq_encode_group([plan], [x], [b])
    torch.cuda.synchronize()
    n = a.end_words()
    assert b.end_words() == n
    assert torch.equal(a.payload[:n], b.payload[:n])
    assert torch.equal(a.offsets, b.offsets) and torch.equal(a.kparam, b.kparam)
    assert torch.equal(a.norms, b.norms)
    assert a.read_stats() == b.read_stats()



@pytest.mark.parametrize("kv", [False, True])
def test_decode_launch_shapes_agree(hq, kv):
    """A single decode of fewer than 16384 sub-streams runs one sub-stream per
    wave, a larger one and every group launch four per wave: 2049 x 4096
    (16392 sub-streams) decoded whole, in two row ranges below the bound and
    as a group member gives the same values, fp32 and bf16."""
    print(f"[parity] decode launch shapes kv={kv}", flush=True)
    opts = dict(rotation=1, rot_seed=5, dither=True, dither_seed=6, norm_fp16=True) if kv else {}
    plan = hq.hq_plan(128, O.E8, 0.0, 79, -1, 4096, snr_db=20.0, **opts)
    rows = 2049
    x = gauss(rows, 4096, 80, 0.02, torch.bfloat16).cuda()
    s = hq.EncodedStream(plan, rows)
    hq.hq_encode(plan, x, s)
    for dt in (torch.float32, torch.bfloat16):
        whole = hq.hq_decode(plan, s, out_dtype=dt)
        lo = hq.hq_decode(plan, s, row0=0, rows=1024, out_dtype=dt)
        hi = hq.hq_decode(plan, s, row0=1024, rows=rows - 1024, out_dtype=dt)
        torch.cuda.synchronize()
        assert torch.equal(torch.cat([lo, hi]).cpu(), whole.cpu()), dt
        if not kv:  # the group launch checked on the weight plan
            g = torch.empty_like(whole)
            hq.hq_decode_group([plan], [s], [g])
            torch.cuda.synchronize()
            assert torch.equal(g.cpu(), whole.cpu()), dt
    assert s.read_stats()["status"] == 0

@pytest.mark.parametrize("lat", [O.E8, O.D4, O.A2, O.Z])
def test_decode_gemv_matches_oracle(hq, lat):
    """hq_decode_gemv (the decode fused with a matrix-vector product) against
    the oracle's decoded rows times x in fp64: row windows with ragged
    counts, bf16 and fp32 x, fp32 and bf16 y.  Tolerance 1e-6 of
    sum_k |W^[r, k] x[k]| (fp32 sums, some 60x the largest error seen; one
    wrong element moves y by about 1/1536 of it); the bf16 result is the
    fp32 one rounded to nearest even."""
    snr = 20.0
    rows, cols = 37, 1536
    P = PT.oracle_params(lat, snr, rht_seed=71)
    w = gauss(rows, cols, 72, 0.02, torch.bfloat16)
    plan, s = encode_gpu(hq, P, snr, w)
    res = PT.compare_streams(P, w.float().numpy(), PT.gpu_stream_arrays(s, rows))
    gc = res["codes"] if res["gpu_codes"] is None else res["gpu_codes"]  # the stream's codes
    wd = O.backend(P, gc, res["norms"]).astype(np.float64)
    worst = 0.0
    for xdt in (torch.float32, torch.bfloat16):
        x = gauss(1, cols, 73, 1.0, xdt)[0]
        xs = x.float().numpy().astype(np.float64)
        for row0, n in ((0, rows), (5, 17), (36, 1)):
            print(f"[parity] decode_gemv {LAT_NAMES[lat]} x={xdt} rows {row0}+{n}", flush=True)
            ref = O.decode_gemv(P, gc[row0:row0 + n], res["norms"][row0:row0 + n], xs, row0=row0)
            scale = np.abs(wd[row0:row0 + n]) @ np.abs(xs)
            y = hq.hq_decode_gemv(plan, s, x.cuda(), row0=row0, rows=n).cpu().numpy()
            err = np.abs(y.astype(np.float64) - ref) / scale
            worst = max(worst, float(err.max()))
            assert np.all(err <= 1e-6), (row0, n, err.max())
            yb = hq.hq_decode_gemv(plan, s, x.cuda(), row0=row0, rows=n, out_dtype=torch.bfloat16)
            assert torch.equal(yb.cpu(), torch.from_numpy(y).to(torch.bfloat16))
    print(f"[parity] decode_gemv {LAT_NAMES[lat]}: worst error {worst:.2e} of sum |w x|", flush=True)
    assert s.read_stats()["corrupt_substreams"] == 0


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.A2, O.Z])
def test_decode_gemv_wave_per_row(hq, lat):
    """From 8192 rows a call runs one wave per row: 8195 rows (a ragged last
    workgroup) and windows at and just below the switch, each against the
    oracle at the same bar as the workgroup-per-row shape."""
    snr = 20.0
    rows, cols = 8195, 512
    P = PT.oracle_params(lat, snr, rht_seed=77)
    w = gauss(rows, cols, 78, 0.02, torch.bfloat16)
    plan, s = encode_gpu(hq, P, snr, w)
    res = PT.compare_streams(P, w.float().numpy(), PT.gpu_stream_arrays(s, rows))
    gc = res["codes"] if res["gpu_codes"] is None else res["gpu_codes"]
    wd = O.backend(P, gc, res["norms"]).astype(np.float64)
    x = gauss(1, cols, 79, 1.0, torch.bfloat16)[0]
    xs = x.float().numpy().astype(np.float64)
    worst = 0.0
    for row0, n in ((0, rows), (3, 8192), (2, 8191)):
        print(f"[parity] decode_gemv one wave per row {LAT_NAMES[lat]} rows {row0}+{n}", flush=True)
        ref = O.decode_gemv(P, gc[row0:row0 + n], res["norms"][row0:row0 + n], xs, row0=row0)
        scale = np.abs(wd[row0:row0 + n]) @ np.abs(xs)
        y = hq.hq_decode_gemv(plan, s, x.cuda(), row0=row0, rows=n).cpu().numpy()
        err = np.abs(y.astype(np.float64) - ref) / scale
        worst = max(worst, float(err.max()))
        assert np.all(err <= 1e-6), (row0, n, err.max())
    print(f"[parity] decode_gemv one wave per row {LAT_NAMES[lat]}: worst error {worst:.2e}", flush=True)
    assert s.read_stats()["corrupt_substreams"] == 0


def test_decode_gemv_argument_errors(hq):
    P = PT.oracle_params(O.E8, 20.0)
    plan = PT.gpu_plan(hq, P, 20.0, 512)
    s = hq.EncodedStream(plan, 4)
    hq.hq_encode(plan, torch.zeros((4, 512), device="cuda"), s)
    x = torch.zeros(512, device="cuda")
    with pytest.raises(hq.HQError):  # workspace too small
        hq.hq_decode_gemv(plan, s, x, workspace=torch.empty(16, dtype=torch.uint8, device="cuda"))
    with pytest.raises(hq.HQError):  # rows past the stream
        hq.hq_decode_gemv(plan, s, x, row0=3, rows=2)
    kv = hq.hq_plan(128, hq.HQ_E8, 0.0, 5, -1, 512, snr_db=20.0, rotation=1, dither=True)
    skv = hq.EncodedStream(kv, 4)
    hq.hq_encode(kv, torch.zeros((4, 512), device="cuda"), skv)
    with pytest.raises(hq.HQError):  # dithered / rotated streams are not supported
        hq.hq_decode_gemv(kv, skv, x)
    torch.cuda.synchronize()


def spike_matrix(rows, cols, rht_seed, seed, frac=0.5):
    """bf16-exact rows where a fraction of the tiles are D times a row of the
    Hadamard matrix (times +-1/16): the RHT maps such a tile to one spike of
    height n, so its normalized coordinate is alpha sqrt(n), the largest code
    the scale allows.  The other tiles are Gaussian."""
    from scipy.linalg import hadamard
    n = 128
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((rows, cols)) * 0.02).astype(np.float32)
    d = O.signs(rht_seed, cols).astype(np.float32)
    H = hadamard(n).astype(np.float32)
    for r in range(rows):
        for t in range(cols // n):
            if rng.random() < frac:
                k = int(rng.integers(n))
                x[r, t * n:(t + 1) * n] = H[k] * d[t * n:(t + 1) * n] * np.float32(rng.choice([-1, 1]) / 16)
    return torch.from_numpy(x).to(torch.bfloat16)


@pytest.mark.parametrize("snr,limit", [(PT.op_snr("E8", 5.0), 127), (38.0, 448)])
def test_decode_clamps_and_saturation(hq, snr, limit):
    """int8 codes clamp at +-127 (E8 at 5 bps: a spike tile's code is about
    alpha sqrt(128) = 166) and E4M3 codes saturate at 448 (38 dB: about 481),
    each counted; the codes are the oracle's, clipped or cast."""
    P = PT.oracle_params(O.E8, snr, rht_seed=23)
    x = spike_matrix(24, 1024, 23, 7 + limit)
    plan, s, res = check_roundtrip(hq, P, snr, x, f"spikes at {snr:.2f} dB")
    oc = res["codes"]
    assert np.abs(oc).max() > limit
    s.reset_stats()
    codes, g = hq.hq_decode_int8(plan, s)
    torch.cuda.synchronize()
    assert np.array_equal(codes.cpu().numpy().astype(np.int32), np.clip(oc, -127, 127))
    assert s.read_stats()["clamps"] == int((np.abs(oc) > 127).sum())
    assert np.array_equal(g.cpu().numpy(), O.weight_factors(P, res["norms"], 24, 1024))
    s.reset_stats()
    c8, g8 = hq.hq_decode_fp8(plan, s)
    torch.cuda.synchronize()
    assert np.array_equal(c8.cpu().numpy(), O.weight_codes_fp8(oc))
    assert s.read_stats()["clamps"] == int((np.abs(oc) > 448).sum())


def test_payload_capacity_overflow_is_reported(hq):
    """A payload buffer declared smaller than the stream: HQ_ERR_CAPACITY in
    the stats, no word written at or past the declared capacity, the offset
    table complete, and every sub-stream that fits written in full."""
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=27)
    x = gauss(32, 1024, 28, 0.02, torch.bfloat16)
    codes, norms, _, _ = O.frontend(P, x.float().numpy())
    o_pay, o_off, o_kp, _ = O.pack(P, codes)
    need = int(o_off[-1])
    for label, group in (("one launch", False), ("group launch", True)):
        print(f"[parity] capacity {label}", flush=True)
        plan = PT.gpu_plan(hq, P, snr, 1024)
        s = hq.EncodedStream(plan, 32)
        cap = need // 2
        s.payload.fill_(0x5A5A5A5A)
        s.c.capacity_words = cap
        if group:
            hq.hq_encode_group([plan], [x.cuda()], [s])
        else:
            hq.hq_encode(plan, x.cuda(), s)
        torch.cuda.synchronize()
        st = s.read_stats()
        assert st["status"] == (-3 & 0xFFFFFFFF), st
        pay = s.payload.cpu().numpy().view(np.uint32)
        assert np.all(pay[cap:] == 0x5A5A5A5A)
        off = s.offsets[:o_off.size].cpu().numpy().view(np.uint32)
        assert np.array_equal(off, o_off)
        fits = np.nonzero(o_off[1:] <= cap)[0]
        assert fits.size > 0
        for sub in fits:
            assert np.array_equal(pay[o_off[sub]:o_off[sub + 1]], o_pay[o_off[sub]:o_off[sub + 1]])


def test_nonfinite_tiles_are_zero_coded_and_reported(hq):
    """Tiles with an infinite or NaN value: HQ_ERR_OVERFLOW, one count per bad
    tile, the bad tiles coded as zeros and every other tile bit-exact with
    the oracle (which codes a non-finite tile as zeros), in both launch
    shapes."""
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=29)
    x = gauss(16, 1024, 30, 0.02, torch.bfloat16)
    x[2, 130] = float("inf")
    x[9, 700] = float("nan")
    x[9, 701] = float("-inf")
    x[11, 1000] = float("-inf")
    xn = x.float().numpy()
    codes, norms, _, rc = O.frontend(P, xn)
    assert rc == O.ERR_OVERFLOW
    o_pay, o_off, o_kp, _ = O.pack(P, codes)
    bad = ~np.isfinite(norms)
    assert bad.sum() == 3
    for label, group in (("one launch", False), ("group launch", True)):
        print(f"[parity] non-finite tiles, {label}", flush=True)
        plan = PT.gpu_plan(hq, P, snr, 1024)
        s = hq.EncodedStream(plan, 16)
        if group:
            hq.hq_encode_group([plan], [x.cuda()], [s])
        else:
            hq.hq_encode(plan, x.cuda(), s)
        torch.cuda.synchronize()
        st = s.read_stats()
        assert st["status"] == (-4 & 0xFFFFFFFF) and st["overflow_tiles"] == 3, st
        g_pay, g_off, g_kp, g_norm = PT.gpu_stream_arrays(s, 16)
        assert np.array_equal(g_off, o_off) and np.array_equal(g_kp, o_kp)
        assert np.array_equal(g_pay, o_pay[:o_off[-1]])
        assert np.array_equal(g_norm[~bad].view(np.uint32), norms[~bad].view(np.uint32))
        assert not np.any(np.isfinite(g_norm[bad]))
