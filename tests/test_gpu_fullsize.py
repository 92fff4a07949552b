"""GPU parity at the full workload sizes, in the launch shapes the bench uses.

The HIP path encodes and decodes each whole configuration; the oracle then
recomputes a seeded sample of rows.  Sub-streams never cross a row and, apart
from the KV dither (which takes the global row index), a row's words, k and
norm depend only on that row, so a sampled row must match the oracle's
encoding of that row alone, bit for bit.  Properties that hold at any size are
checked over everything: the stream parses, the stats add up, and the
reconstruction SNR sits at the operating point.  Same bar as the small-size
parity tests.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from tests import parity as PT

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hq():
    from paper_2606_23406_amd import hq as H
    H.lib()
    assert torch.cuda.is_available()
    return H


def row_stream(gpu, r, spr):
    """The sub-streams of row r of a GPU stream, as a one-row stream tuple."""
    pay, off, kp, norms = gpu
    o = off[r * spr:(r + 1) * spr + 1]
    return pay[o[0]:o[-1]], o, kp[r * spr:(r + 1) * spr], norms[r:r + 1]


def check_sampled_rows(hq, plan, s, P, x, rows_idx, label, dither=False):
    """Bit-exact words, k and norms of the sampled rows, and their decode."""
    spr = plan.info.subs_per_row
    gpu = PT.gpu_stream_arrays(s, s.rows)
    exempt = 0
    for r in rows_idx:
        xr = x[r:r + 1].float().numpy()
        res = PT.compare_streams(P, xr, row_stream(gpu, int(r), spr), row0=int(r) if dither else 0)
        exempt += res["exempt_blocks"]
        y32 = hq.hq_decode(plan, s, row0=int(r), rows=1, out_dtype=torch.float32)
        y16 = hq.hq_decode(plan, s, row0=int(r), rows=1, out_dtype=torch.bfloat16)
        ref = O.backend(P, res["codes"], res["norms"], row0=int(r) if dither else 0)
        skip = PT.tiles_with_code_diffs(res["codes"], res["gpu_codes"])
        unit = PT.lattice_unit(P, res["norms"])
        got = y32.cpu().numpy().astype(np.float64).reshape(-1, 128)
        err = np.abs(got - ref.reshape(-1, 128)).max(axis=1)
        assert np.all(err[~skip] <= 1e-5 * unit[~skip]), (label, r, err.max())
        ref16 = torch.from_numpy(ref.astype(np.float32)).to(torch.bfloat16).float().numpy()
        eq16 = (y16.cpu().float().numpy() == ref16).reshape(-1, 128)
        assert eq16[~skip].all(), (label, r)
    print(f"[fullsize] {label}: {len(rows_idx)} sampled rows bit-exact "
          f"(exempt blocks {exempt})", flush=True)
    assert exempt <= max(2, len(rows_idx) * spr // 100)


def snr_db(x, y):
    x = x.float()
    e = (y.float() - x)
    return 10.0 * torch.log10((x * x).sum() / (e * e).sum()).item()


@pytest.mark.parametrize("bps", [4.0, 3.0])
def test_c2_heavy_tailed_4096(hq, bps):
    from paper_2606_23406_amd import workloads as W
    print(f"[fullsize] C2 4096x4096 bf16 Student-t + outlier columns, E8@{bps}", flush=True)
    x = W.heavy_tailed_weight()
    snr = PT.op_snr("E8", bps)
    P = PT.oracle_params(O.E8, snr, rht_seed=17)
    plan = PT.gpu_plan(hq, P, snr, 4096)
    s = hq.EncodedStream(plan, 4096)
    xd = x.cuda()
    hq.hq_encode(plan, xd, s)
    y = hq.hq_decode(plan, s, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    st = s.read_stats()
    assert st["status"] == 0 and st["corrupt_substreams"] == 0, st
    rate = st["payload_bits"] / x.numel()
    q = snr_db(xd, y)
    print(f"[fullsize] C2 E8@{bps}: {rate:.4f} bits/scalar, SNR {q:.3f} dB "
          f"(operating point {snr:.3f} dB)", flush=True)
    assert abs(q - snr) < 0.5
    assert abs(rate - bps) < 0.25
    rng = np.random.default_rng(int(bps * 10))
    rows = np.sort(rng.choice(4096, 24, replace=False))
    check_sampled_rows(hq, plan, s, P, x, rows, f"C2 E8@{bps}")


WHOLE = {
    "C2_E8@4": ("c2", O.E8, 4.0), "C2_E8@3": ("c2", O.E8, 3.0),
    "C3_l0_gate_E8@4": ("gate", O.E8, 4.0), "C3_l0_down_D4@3": ("down", O.D4, 3.0),
    "C4_keys_E8@2": ("keys", O.E8, 2.0), "C4_keys_A2@1.7": ("keys", O.A2, 1.7),
    "C4_keys_Z@1.7": ("keys", O.Z, 1.7),
    "C4_keys_E8@2_qjl": ("keys_qjl", O.E8, 2.0),
}


def haar128(seed):
    g = np.random.default_rng(seed).standard_normal((128, 128))
    q, r = np.linalg.qr(g)
    return (q * np.sign(np.diag(r))).astype(np.float32)


@pytest.mark.parametrize("case", list(WHOLE))
def test_whole_stream_bit_exact(hq, kv_keys, case):
    """Every sub-stream of a full-size encode (C2 whole, C3 layer 0's gate and
    down, C4 keys appended in 128-token blocks with signs + dither + fp16
    norms; one case with the qjl rotation instead of the signs) against the
    oracle's encode of the same input: words, k and norms
    bit for bit, codes different only in blocks within 1e-6 of a Voronoi
    boundary (counted; at most 1 in 10^5); then every decoded tile against
    the oracle's reconstruction."""
    from paper_2606_23406_amd import workloads as W
    what, lat, bps = WHOLE[case]
    lname = {O.E8: "E8", O.D4: "D4", O.A2: "A2", O.Z: "Z"}[lat]
    snr = PT.op_snr(lname, bps)
    kv = what.startswith("keys")
    if what == "c2":
        x, seed = W.heavy_tailed_weight(), 17
    elif kv:
        x, seed = kv_keys, 71
    else:
        idx = 4 if what == "gate" else 6
        x, seed = W.llama_linear(0, idx, device="cuda").cpu(), W.llama_linear_seed(0, idx)
    rows, cols = x.shape
    print(f"[fullsize] whole stream {case}: {rows}x{cols}", flush=True)
    opts = dict(rotation=1, rot_seed=72, dither=True, dither_seed=73 + lat, norm_fp16=True) if kv else {}
    if what == "keys_qjl":
        opts.update(rotation=2, qjl=haar128(74))
    P = PT.oracle_params(lat, snr, rht_seed=seed, **opts)
    plan = PT.gpu_plan(hq, P, snr, cols)
    s = hq.EncodedStream(plan, rows)
    xd = x.cuda()
    step = 128 if kv else rows
    for r0 in range(0, rows, step):
        hq.hq_encode(plan, xd[r0:r0 + step], s, append=r0 > 0)
    torch.cuda.synchronize()
    del xd
    st = s.read_stats()
    assert st["status"] == 0, st
    res = PT.compare_streams(P, x.float().numpy(), PT.gpu_stream_arrays(s, rows))
    blocks = x.numel() // O.DIM[lat]
    print(f"[fullsize] whole stream {case}: {res['substreams']} sub-streams, {blocks} blocks, "
          f"exempt blocks {res['exempt_blocks']} (sub-streams {res['exempt_substreams']})", flush=True)
    assert res["exempt_blocks"] <= max(2, blocks // 100000)
    assert st["payload_bits"] == res["payload_bits"] or res["exempt_substreams"] > 0
    # and the whole decode: every tile within 1e-5 of its lattice unit of the
    # oracle's fp32 reconstruction from the stream's own codes
    codes = res["codes"] if res["gpu_codes"] is None else res["gpu_codes"]
    y = hq.hq_decode(plan, s, out_dtype=torch.float32).cpu().numpy()
    ref = O.backend(P, codes, res["norms"])
    unit = PT.lattice_unit(P, res["norms"]).reshape(-1)
    err = np.abs(y.astype(np.float64) - ref).reshape(-1, 128).max(axis=1)
    exact = float(np.mean(y == ref))
    print(f"[fullsize] whole stream {case}: decode max error {float((err / unit).max()):.2e} of the "
          f"lattice unit, bit-exact fraction {exact:.6f}", flush=True)
    assert np.all(err <= 1e-5 * unit)


@pytest.mark.parametrize("layer", [0, 15, 31])
@pytest.mark.parametrize("lat,bps", [(O.E8, 4.0), (O.D4, 3.0)])
def test_c3_llama_linears(hq, layer, lat, bps):
    """All seven linears of one layer (generated on the device, as the bench
    does): the whole matrix through the HIP path, stats and SNR over all of
    it, 8 sampled rows each bit for bit against the oracle."""
    from paper_2606_23406_amd import workloads as W
    lname = "E8" if lat == O.E8 else "D4"
    snr = PT.op_snr(lname, bps)
    for idx, (name, out_f, in_f) in enumerate(W.LLAMA_LINEARS):
        print(f"[fullsize] C3 layer {layer} {name} {out_f}x{in_f} {lname}@{bps}", flush=True)
        xd = W.llama_linear(layer, idx, device="cuda")
        P = PT.oracle_params(lat, snr, rht_seed=W.llama_linear_seed(layer, idx))
        plan = PT.gpu_plan(hq, P, snr, in_f)
        s = hq.EncodedStream(plan, out_f)
        hq.hq_encode(plan, xd, s)
        y = hq.hq_decode(plan, s, out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
        st = s.read_stats()
        assert st["status"] == 0 and st["corrupt_substreams"] == 0, st
        q = snr_db(xd, y)
        rate = st["payload_bits"] / xd.numel()
        print(f"[fullsize] C3 {name} {lname}@{bps}: {rate:.4f} bits/scalar, SNR {q:.3f} dB", flush=True)
        assert abs(q - snr) < 0.5 and abs(rate - bps) < 0.25
        rng = np.random.default_rng(1000 * layer + 10 * idx + lat)
        rows = np.sort(rng.choice(out_f, 8, replace=False))
        x = torch.zeros((out_f, in_f), dtype=torch.bfloat16)
        x[rows] = xd[torch.from_numpy(rows).cuda()].cpu()
        check_sampled_rows(hq, plan, s, P, x, rows, f"C3 layer {layer} {name} {lname}@{bps}")
        del xd, y, s


def test_c3_first_launch_group_as_benched(hq):
    """The bench's first launch of the E8@4 stack: sixteen matrices (layers 0
    and 1, then layer 2's q and k) through one hq_encode_group and one
    hq_decode_group launch.  Every stream and output equals the
    single-matrix calls word for word, and sampled rows of one member of each
    shape match the oracle bit for bit."""
    from paper_2606_23406_amd import workloads as W
    snr = PT.op_snr("E8", 4.0)
    members = [(layer, idx) for layer in range(3) for idx in range(len(W.LLAMA_LINEARS))][:16]
    plans, Ps, xs, grp = [], [], [], []
    for layer, idx in members:
        _, out_f, in_f = W.LLAMA_LINEARS[idx]
        P = PT.oracle_params(O.E8, snr, rht_seed=W.llama_linear_seed(layer, idx))
        plan = PT.gpu_plan(hq, P, snr, in_f)
        plans.append(plan)
        Ps.append(P)
        xs.append(W.llama_linear(layer, idx, device="cuda"))
        grp.append(hq.EncodedStream(plan, out_f))
    print("[fullsize] C3 first launch group: 16 matrices, E8@4", flush=True)
    hq.hq_encode_group(plans, xs, grp)
    ys = [torch.empty_like(x) for x in xs]
    hq.hq_decode_group(plans, grp, ys)
    torch.cuda.synchronize()
    shapes = set()
    for (layer, idx), plan, P, x, s, y in zip(members, plans, Ps, xs, grp, ys):
        name, out_f, in_f = W.LLAMA_LINEARS[idx]
        assert s.read_stats()["status"] == 0
        one = hq.EncodedStream(plan, out_f)
        hq.hq_encode(plan, x, one)
        y1 = hq.hq_decode(plan, one, out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
        n = one.end_words()
        assert s.end_words() == n and torch.equal(s.payload[:n], one.payload[:n]), (layer, name)
        assert torch.equal(s.offsets, one.offsets) and torch.equal(s.kparam, one.kparam)
        assert torch.equal(s.norms, one.norms) and torch.equal(y, y1), (layer, name)
        if (out_f, in_f) not in shapes:
            shapes.add((out_f, in_f))
            rng = np.random.default_rng(7000 + 10 * layer + idx)
            rows = np.sort(rng.choice(out_f, 4, replace=False))
            xc = torch.zeros((out_f, in_f), dtype=torch.bfloat16)
            xc[rows] = x[torch.from_numpy(rows).cuda()].cpu()
            check_sampled_rows(hq, plan, s, P, xc, rows, f"C3 group launch, layer {layer} {name}")
        del one, y1
    assert len(shapes) == 4


def test_c3_decode_gemv_gate(hq):
    """The fused decode-GEMV on layer 0's gate matrix (14336 x 4096, E8@4) with
    one bf16 token: sampled rows against the oracle's decoded row times x in
    fp64, to 1e-6 of sum_k |W^[r, k] x[k]|."""
    from paper_2606_23406_amd import workloads as W
    snr = PT.op_snr("E8", 4.0)
    idx = [n for n, _, _ in W.LLAMA_LINEARS].index("gate")
    _, out_f, in_f = W.LLAMA_LINEARS[idx]
    P = PT.oracle_params(O.E8, snr, rht_seed=W.llama_linear_seed(0, idx))
    plan = PT.gpu_plan(hq, P, snr, in_f)
    xd = W.llama_linear(0, idx, device="cuda")
    s = hq.EncodedStream(plan, out_f)
    hq.hq_encode(plan, xd, s)
    x = W.activations(tokens=1, features=in_f)[0].cuda()
    print(f"[fullsize] decode_gemv gate {out_f}x{in_f}", flush=True)
    y = hq.hq_decode_gemv(plan, s, x).cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    assert s.read_stats()["status"] == 0
    xs = x.float().cpu().numpy().astype(np.float64)
    spr = plan.info.subs_per_row
    gpu = PT.gpu_stream_arrays(s, s.rows)
    rng = np.random.default_rng(77)
    worst = 0.0
    for r in np.sort(rng.choice(out_f, 8, replace=False)):
        xr = xd[int(r):int(r) + 1].float().cpu().numpy()
        res = PT.compare_streams(P, xr, row_stream(gpu, int(r), spr))
        gc = res["codes"] if res["gpu_codes"] is None else res["gpu_codes"]  # the stream's codes
        ref = O.decode_gemv(P, gc, res["norms"], xs)[0]
        scale = np.abs(O.backend(P, gc, res["norms"]).astype(np.float64)[0]) @ np.abs(xs)
        err = abs(y[r] - ref) / scale
        worst = max(worst, err)
        assert err <= 1e-6, (r, err)
    print(f"[fullsize] decode_gemv gate: 8 sampled rows, worst error {worst:.2e} of sum |w x|",
          flush=True)


@pytest.fixture(scope="module")
def kv_keys():
    from paper_2606_23406_amd import workloads as W
    k = W.kv_cache(role="k")  # [16, 8192, 8, 128]
    return k.reshape(16 * 8192, 8 * 128)


@pytest.mark.parametrize("lat,bps", [(O.E8, 2.0), (O.A2, 1.7), (O.Z, 1.7)])
def test_c4_kv_cache_keys(hq, kv_keys, lat, bps):
    """Keys [16, 8192, 8, 128] quantized on append in 128-token blocks with the
    bias correction (sign rotation + subtractive dither, fp16 norms); one
    stream row = one token's 8 head vectors (8 tiles)."""
    from paper_2606_23406_amd import workloads as W
    lname = {O.E8: "E8", O.A2: "A2", O.Z: "Z"}[lat]
    x = kv_keys
    rows, cols = x.shape
    print(f"[fullsize] C4 keys {rows}x{cols} {lname}@{bps}, 128-token appends", flush=True)
    snr = PT.op_snr(lname, bps)
    P = PT.oracle_params(lat, snr, rht_seed=71, rotation=1, rot_seed=72, dither=True,
                         dither_seed=73 + lat, norm_fp16=True)
    plan = PT.gpu_plan(hq, P, snr, cols)
    s = hq.EncodedStream(plan, rows)
    xd = x.cuda()
    for r0 in range(0, rows, 128):
        hq.hq_encode(plan, xd[r0:r0 + 128], s, append=r0 > 0)
    y = hq.hq_decode(plan, s, out_dtype=torch.float32)
    torch.cuda.synchronize()
    st = s.read_stats()
    assert s.rows == rows
    assert st["status"] == 0 and st["corrupt_substreams"] == 0, st
    q = snr_db(xd, y)
    rate = st["payload_bits"] / x.numel()
    print(f"[fullsize] C4 {lname}@{bps}: {rate:.4f} bits/scalar, SNR {q:.3f} dB", flush=True)
    assert abs(rate - bps) < 0.3
    rng = np.random.default_rng(200 + lat)
    sample = np.sort(rng.choice(rows, 16, replace=False))
    check_sampled_rows(hq, plan, s, P, x, sample, f"C4 keys {lname}@{bps}", dither=True)
    # unbiased inner products: for each of 1024 fixed queries, the mean of
    # q . (k_hat - k) over every key of head 0 is zero within its standard error
    qs = W.queries(device="cpu").cuda()
    k = xd[:, :128].float()
    d = y[:, :128] - k
    e = d @ qs.t()  # [keys, queries]
    n = e.shape[0]
    z = e.mean(0) / (e.std(0) / np.sqrt(n))
    print(f"[fullsize] C4 {lname}: max |mean error| / standard error over 1024 queries "
          f"{z.abs().max().item():.2f}", flush=True)
    assert z.abs().max().item() < 5.0


@pytest.mark.parametrize("lat,bps", [(O.E8, 2.0), (O.A2, 1.7), (O.Z, 1.7)])
def test_c4_per_pair_unbiased(hq, kv_keys, lat, bps):
    """Per (query, key) pair, over R = 64 dither seeds: the mean of
    <q, k_hat> - <q, k> is zero (|t| > 4 no more often than a t distribution
    with 63 degrees of freedom and some slack allow), and its variance is the
    closed form of the subtractive-dither theorem (Sec. 3.4, Prop. on the
    composed codec): sigma_Vor^2 |q|^2 (r_s / (alpha sqrt(n)))^2.  Control:
    with the dither off the error is the same on every run (a fixed bias per
    pair, not centred).  256 sampled keys (head 0 of each sampled row),
    1024 queries."""
    from paper_2606_23406_amd import workloads as W
    lname = {O.E8: "E8", O.A2: "A2", O.Z: "Z"}[lat]
    R, nk = 64, 256
    rng = np.random.default_rng(300 + lat)
    rows = np.sort(rng.choice(kv_keys.shape[0], nk, replace=False))
    kfull = kv_keys[torch.from_numpy(rows)].contiguous().cuda()  # one row = 8 head vectors
    k = kfull[:, :128]
    qs = W.queries(device="cpu").cuda()  # [1024, 128]
    snr = PT.op_snr(lname, bps)
    print(f"[fullsize] C4 per-pair bias {lname}@{bps}: {nk} keys x {qs.shape[0]} queries, "
          f"R = {R} dither seeds", flush=True)
    exact = k.float() @ qs.t()

    def run(seed, dither):
        plan = hq.hq_plan(128, lat, 0.0, 71, -1, 1024, rotation=1, dither=dither, rot_seed=72,
                          dither_seed=seed, norm_fp16=True, snr_db=snr)
        s = hq.EncodedStream(plan, nk)
        hq.hq_encode(plan, kfull, s)
        y = hq.hq_decode(plan, s, out_dtype=torch.float32)[:, :128]
        rs = s.norms[:nk * 8].float().reshape(nk, 8)[:, 0]
        return y, rs, plan.info.alpha

    acc = torch.zeros_like(exact, dtype=torch.float64)
    acc2 = torch.zeros_like(acc)
    for r in range(R):
        y, rs, alpha = run(1000 + r, True)
        e = (y @ qs.t() - exact).double()
        acc += e
        acc2 += e * e
    torch.cuda.synchronize()
    mean = acc / R
    var = (acc2 - R * mean * mean) / (R - 1)
    t = mean / torch.sqrt(var / R)
    frac = (t.abs() > 4.0).double().mean().item()
    qn2 = (qs.double() ** 2).sum(1)
    pred = O.sigma2_vor(lat) * qn2[None, :] * (rs.double()[:, None] / (alpha * np.sqrt(128.0))) ** 2
    ratio = (var / pred).mean().item()
    print(f"[fullsize] C4 {lname}: fraction |t| > 4 = {frac:.2e}, mean var / closed form = {ratio:.4f}",
          flush=True)
    assert frac < 1e-3
    assert abs(ratio - 1.0) < 0.05
    # control: no dither -> the same error on every run, a fixed per-pair bias
    y0, _, _ = run(5, False)
    y1, _, _ = run(6, False)
    assert torch.equal(y0, y1)
    b = (y0 @ qs.t() - exact).double()
    big = (b.abs() > 0.1 * torch.sqrt(pred)).double().mean().item()
    print(f"[fullsize] C4 {lname} no dither: fraction of pairs with |bias| > 0.1 sd = {big:.3f}",
          flush=True)
    assert big > 0.8


def test_c4_kv_cache_values_e8(hq):
    from paper_2606_23406_amd import workloads as W
    x = W.kv_cache(role="v").reshape(16 * 8192, 1024)
    rows, cols = x.shape
    print(f"[fullsize] C4 values {rows}x{cols} E8@2, 128-token appends", flush=True)
    snr = PT.op_snr("E8", 2.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=81, rotation=1, rot_seed=82, dither=True,
                         dither_seed=83, norm_fp16=True)
    plan = PT.gpu_plan(hq, P, snr, cols)
    s = hq.EncodedStream(plan, rows)
    xd = x.cuda()
    for r0 in range(0, rows, 128):
        hq.hq_encode(plan, xd[r0:r0 + 128], s, append=r0 > 0)
    torch.cuda.synchronize()
    st = s.read_stats()
    assert st["status"] == 0, st
    rng = np.random.default_rng(300)
    check_sampled_rows(hq, plan, s, P, x, np.sort(rng.choice(rows, 12, replace=False)),
                       "C4 values E8@2", dither=True)


def test_c4_decode_attention_as_benched(hq):
    """hq_decode_attention at the KV workload's full size, in the layout and
    launch shape the bench times: keys and values [16, 8192, 8, 128] E8 at 2
    bps (signs rotation, dither, fp16 norms) appended in 128-token blocks, a
    stream row being (block, sequence, token); 32 query heads (4 per KV
    head), one sequence cut to 5000 tokens; without and with a 32-token exact
    window (the ring holding the last 32 tokens of the unquantized cache).
    Three sampled sequences against the oracle over those sequences' rows,
    within 2e-5 of max |v^|."""
    from paper_2606_23406_amd import workloads as W
    B, T, Hkv, Hq, bt = 16, 8192, 8, 32, 128
    snr = PT.op_snr("E8", 2.0)
    streams, rings = [], []
    for role, seed in (("k", 91), ("v", 95)):
        x = W.kv_cache(role=role)
        lens_ring = np.full(B, T)
        lens_ring[5] = 5000
        # ring slot t % 32 holds token t of the last 32 of each sequence
        ring = torch.stack([x[b, n - 32:n].reshape(32, Hkv * 128).roll(n % 32, 0)
                            for b, n in enumerate(lens_ring)]).contiguous()
        rings.append(ring)
        x = x.permute(1, 0, 2, 3).reshape(T // bt, bt, B, Hkv * 128)
        x = x.permute(0, 2, 1, 3).reshape(-1, Hkv * 128).contiguous()
        P = PT.oracle_params(O.E8, snr, rht_seed=seed, rotation=1, rot_seed=seed + 1, dither=True,
                             dither_seed=seed + 2, norm_fp16=True)
        plan = PT.gpu_plan(hq, P, snr, Hkv * 128)
        s = hq.EncodedStream(plan, x.shape[0])
        xd = x.cuda()
        for r0 in range(0, x.shape[0], B * bt):
            hq.hq_encode(plan, xd[r0:r0 + B * bt], s, append=r0 > 0)
        del xd
        streams.append((P, plan, s))
    (pk, plk, sk), (pv, plv, sv) = streams
    table = (np.arange(T // bt)[None, :] * B + np.arange(B)[:, None]).astype(np.int32)
    lens = np.full(B, T, dtype=np.int32)
    lens[5] = 5000
    q = W.queries(n=B * Hq).reshape(B, Hq, 128).to(torch.bfloat16)
    print(f"[fullsize] C4 decode attention: batch {B}, {T} tokens, {Hkv} KV heads, {Hq} query "
          f"heads, E8@2 keys and values", flush=True)
    out = hq.hq_decode_attention(plk, sk, plv, sv, q.cuda(), torch.from_numpy(table).cuda(),
                                 torch.from_numpy(lens).cuda(), bt)
    outw = hq.hq_decode_attention(plk, sk, plv, sv, q.cuda(), torch.from_numpy(table).cuda(),
                                  torch.from_numpy(lens).cuda(), bt, window_k=rings[0].cuda(),
                                  window_v=rings[1].cuda())
    torch.cuda.synchronize()
    for st in (sk.read_stats(), sv.read_stats()):
        assert st["status"] == 0 and st["corrupt_substreams"] == 0, st
    got = out.cpu().numpy().astype(np.float64)
    arrays = [PT.gpu_stream_arrays(s, s.rows) for s in (sk, sv)]
    worst = 0.0
    for b in (0, 5, 15):
        rows = np.concatenate([table[b, k] * bt + np.arange(bt) for k in range(-(-lens[b] // bt))])
        codes, norms = [], []
        for P, (pay, off, kp, nrm) in zip((pk, pv), arrays):
            parts = []
            for k in range(0, rows.size, bt):  # one 128-row block at a time
                r0 = int(rows[k])
                o = off[r0 * 2:(r0 + bt) * 2 + 1]
                c, rc = O.unpack(P, pay[o[0] - off[0]:o[-1] - off[0]], o - o[0],
                                 kp[r0 * 2:(r0 + bt) * 2], bt, Hkv * 128, 0)
                assert rc == O.OK
                parts.append(c)
            codes.append(np.concatenate(parts))
            norms.append(nrm[rows])
        ref = O.decode_attention(pk, codes[0], norms[0], pv, codes[1], norms[1],
                                 q[b:b + 1].float().numpy(), table[b:b + 1], lens[b:b + 1], bt,
                                 128 ** -0.5, rows=rows)[0]
        refw = O.decode_attention(pk, codes[0], norms[0], pv, codes[1], norms[1],
                                  q[b:b + 1].float().numpy(), table[b:b + 1], lens[b:b + 1], bt,
                                  128 ** -0.5, rows=rows, window=32,
                                  window_k=rings[0][b:b + 1].float().numpy(),
                                  window_v=rings[1][b:b + 1].float().numpy())[0]
        gotw = outw.cpu().numpy().astype(np.float64)
        vd = np.concatenate([O.backend(pv, codes[1][k:k + bt], norms[1][k:k + bt], row0=int(rows[k]))
                             for k in range(0, rows.size, bt)])
        for h in range(Hq):
            cs = slice((h // 4) * 128, (h // 4 + 1) * 128)
            err = np.abs(got[b, h] - ref[h]).max() / np.abs(vd[:lens[b], cs]).max()
            unit_w = max(np.abs(vd[:lens[b] - 32, cs]).max(),
                         float(rings[1][b, :, cs].float().abs().max()))
            errw = np.abs(gotw[b, h] - refw[h]).max() / unit_w
            worst = max(worst, err, errw)
            assert err <= 2e-5 and errw <= 2e-5, (b, h, err, errw)
    print(f"[fullsize] C4 decode attention (plain and 32-token window): 3 sequences x {Hq} heads, "
          f"worst error {worst:.2e} of max |v|", flush=True)


def test_c5_gemm_fullsize(hq):
    from paper_2606_23406_amd import workloads as W
    print("[fullsize] C5 gemm W 14336x4096 E8@4, A 4096x4096", flush=True)
    w = W.llama_linear(0, 4)
    a = W.activations()
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=W.llama_linear_seed(0, 4))
    plan = PT.gpu_plan(hq, P, snr, 4096)
    s = hq.EncodedStream(plan, 14336)
    hq.hq_encode(plan, w.cuda(), s)
    out = hq.hq_dequant_gemm_int8(plan, s, a.cuda(), out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert s.read_stats()["status"] == 0
    rng = np.random.default_rng(400)
    mi = np.sort(rng.choice(4096, 48, replace=False))
    ni = np.sort(rng.choice(14336, 48, replace=False))
    codes, norms, _, _ = O.frontend(P, w[ni].float().numpy())
    g = O.weight_factors(P, norms, len(ni), 4096)
    xq, sx = O.act_prep(a[mi].float().numpy(), 128, P.rht_seed)
    ref = O.gemm_blockscaled(codes, g, xq, sx, 128)
    got = out.cpu().numpy()[mi][:, ni].astype(np.float64)
    denom = np.maximum(np.abs(ref), np.sqrt((ref ** 2).mean()))
    rel = np.max(np.abs(got - ref) / denom)
    print(f"[fullsize] C5 sampled 48x48 outputs: max relative error {rel:.2e}", flush=True)
    assert rel <= 1e-3
    # the fp8 E4M3 cast path on the same operands, same samples
    x8, sx8 = hq.hq_act_prep_fp8(plan, a.cuda())
    c8, g8 = hq.hq_decode_fp8(plan, s)
    out8 = hq.hq_gemm_fp8_blockscaled(plan, x8, sx8, c8, g8, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ox8, osx8 = O.act_prep_fp8(a[mi].float().numpy(), 128, P.rht_seed)
    assert np.array_equal(x8.cpu().numpy()[mi], ox8) and np.array_equal(sx8.cpu().numpy()[mi], osx8)
    assert np.array_equal(c8.cpu().numpy()[ni], O.weight_codes_fp8(codes))
    ref8 = O.gemm_fp8_blockscaled(O.weight_codes_fp8(codes), g, ox8, osx8, 128)
    got8 = out8.cpu().numpy()[mi][:, ni].astype(np.float64)
    rel8 = np.max(np.abs(got8 - ref8) / np.maximum(np.abs(ref8), np.sqrt((ref8 ** 2).mean())))
    print(f"[fullsize] C5 fp8 sampled 48x48 outputs: max relative error {rel8:.2e}", flush=True)
    assert rel8 <= 1e-4
    # and the MXFP4 cast path (E2M1 values with E8M0 scales per 32 along K)
    del x8, c8, out8
    x4, xs4 = hq.hq_act_prep_mxfp4(plan, a.cuda())
    c4, ws4 = hq.hq_decode_mxfp4(plan, s)
    out4 = hq.hq_gemm_mxfp4_blockscaled(plan, x4, xs4, c4, ws4, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ox4, oxs4 = O.act_prep_mxfp4(a[mi].float().numpy(), 128, P.rht_seed)
    ow4, ows4 = O.weight_codes_mxfp4(codes, g, 128)

    def nib(c):
        c = np.asarray(c, dtype=np.uint8)
        return (c[:, 0::2] | (c[:, 1::2] << 4)).astype(np.uint8)

    assert np.array_equal(x4.cpu().numpy()[mi], nib(ox4)) and np.array_equal(xs4.cpu().numpy()[mi], oxs4)
    assert np.array_equal(c4.cpu().numpy()[ni], nib(ow4)) and np.array_equal(ws4.cpu().numpy()[ni], ows4)
    ref4 = O.gemm_mxfp4(ow4, ows4, ox4, oxs4)
    got4 = out4.cpu().numpy()[mi][:, ni].astype(np.float64)
    rel4 = np.max(np.abs(got4 - ref4) / np.maximum(np.abs(ref4), np.sqrt((ref4 ** 2).mean())))
    print(f"[fullsize] C5 MXFP4 sampled 48x48 outputs: max relative error {rel4:.2e}", flush=True)
    assert rel4 <= 1e-4


def test_corrupt_streams_are_reported(hq):
    """Damaged tables and payloads decode without faults: each damaged
    sub-stream is counted once and decodes as zeros over its whole 512-column
    span (every lane, not just the lanes whose codes failed to parse), the
    fused GEMV takes zero from it, and every other sub-stream decodes
    unchanged."""
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=91)
    g = torch.Generator().manual_seed(92)
    x = (torch.randn((16, 1024), generator=g) * 0.02).to(torch.bfloat16)
    plan = PT.gpu_plan(hq, P, snr, 1024)
    s = hq.EncodedStream(plan, 16)
    hq.hq_encode(plan, x.cuda(), s)
    good = hq.hq_decode(plan, s, out_dtype=torch.float32).cpu()
    torch.cuda.synchronize()
    spr = plan.info.subs_per_row
    assert spr == 2
    # Each damage is one the decoder must detect:
    #   row 3:  k = 15 needs more remainder bits than the sub-stream has;
    #   row 7:  sub-stream 0 ends before it starts, so sub-stream 1 spans
    #           more words than any sub-stream may hold;
    #   row 11: sub-stream 0's words zeroed, so its codes have no terminators;
    #   row 13: an end offset past the capacity (sub-streams 0 and 1).
    kp = s.kparam.clone()
    kp[3 * spr] = 15
    s.kparam.copy_(kp)
    off = s.offsets.clone()
    off[7 * spr + 1] = off[7 * spr] - 1
    s.offsets.copy_(off)
    o11 = int(s.offsets[11 * spr].item()) & 0xFFFFFFFF
    o12 = int(s.offsets[11 * spr + 1].item()) & 0xFFFFFFFF
    s.payload[o11:o12] = 0
    off = s.offsets.clone()
    off[13 * spr + 1] = s.c.capacity_words + 5
    s.offsets.copy_(off)
    assert (int(s.offsets[7 * spr + 2]) - int(s.offsets[7 * spr + 1])) > plan.info.max_words_per_substream
    s.reset_stats()
    bad = hq.hq_decode(plan, s, out_dtype=torch.float32).cpu()
    torch.cuda.synchronize()
    st = s.read_stats()
    assert st["status"] == (-6 & 0xFFFFFFFF), st  # HQ_ERR_CORRUPT
    damaged = {(3, 0), (7, 0), (7, 1), (11, 0), (13, 0), (13, 1)}
    assert st["corrupt_substreams"] == len(damaged), st
    for r in range(16):
        for j in range(spr):
            span = slice(512 * j, 512 * (j + 1))
            if (r, j) in damaged:
                assert torch.all(bad[r, span] == 0), (r, j)
            else:
                assert torch.equal(bad[r, span], good[r, span]), (r, j)
    # the fused GEMV: damaged sub-streams contribute zero, the rest as decoded
    xv = torch.randn(1024, generator=g).cuda()
    s.reset_stats()
    yv = hq.hq_decode_gemv(plan, s, xv, out_dtype=torch.float32).cpu().double()
    torch.cuda.synchronize()
    assert s.read_stats()["corrupt_substreams"] == len(damaged)
    ref = bad.double() @ xv.cpu().double()
    scale = bad.double().abs() @ xv.cpu().double().abs()
    assert torch.all((yv - ref).abs() <= 1e-5 * scale + 1e-30)
