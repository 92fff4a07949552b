#!/usr/bin/env python3
"""Headline benchmark of the HyperQuant codec on one MI355X.

Metric: encode + decode GB/s of bf16 input (E8 lattice, 4 bits per scalar)
and its fraction of HBM peak.  Workload: the whole Llama-3.1-8B-shaped linear
stack (32 layers x {q, k, v, o, gate, up, down}, 6.98e9 bf16 weights,
N(0, 0.02^2) with log-uniform per-output-channel scales, seeded synthetic
data).  One step = encode all 224 matrices (RHT, normalize, E8, strip, Rice,
offset scan) and then decode all of them back to bf16 (Rice decode, unstrip,
inverse RHT, denormalize), every input resident in HBM.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Prints one JSON line.  The CPU oracle is timed on a bounded sample of the
same workload beside it (cpu_baseline).
"""
import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, vendor figure
INT8_PEAK_TOPS = 5000.0    # MI355X dense int8 MFMA, vendor figure
FP8_PEAK_TFLOPS = 5000.0   # MI355X dense fp8 MFMA, vendor figure
FP4_PEAK_TFLOPS = 10100.0  # MI355X dense fp4 MFMA, vendor figure


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--bps", type=float, default=4.0)
    ap.add_argument("--snr", type=float, default=None,
                    help="plan at this SNR instead of the library's bps calibration")
    ap.add_argument("--layers", type=int, default=32)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gemm", action="store_true")
    ap.add_argument("--no-attention", action="store_true")
    ap.add_argument("--no-other", action="store_true", help="skip the C1, C2, C3-D4 and C4 measurements")
    ap.add_argument("--group", type=int, default=16,
                    help="matrices per encode/decode launch (hq_encode_group); 1 = one launch each")
    return ap.parse_args()


def build_workload(H, W, layers, bps, dev, snr=None):
    """Plans, resident bf16 inputs, encoded-stream buffers and decode outputs."""
    mats = []
    for layer in range(layers):
        for idx, (name, out_f, in_f) in enumerate(W.LLAMA_LINEARS):
            seed = W.llama_linear_seed(layer, idx)
            plan = H.hq_plan(128, H.HQ_E8, bps, seed, -1, in_f, snr_db=snr)
            x = W.llama_linear(layer, idx, device=dev)
            s = H.EncodedStream(plan, out_f, device=dev)
            y = torch.empty_like(x)
            mats.append({"name": name, "layer": layer, "seed": seed, "plan": plan, "x": x, "s": s, "y": y})
    return mats


def groups_of(mats, size):
    """The stack in launch groups of `size` consecutive matrices."""
    return [mats[i:i + size] for i in range(0, len(mats), size)]


def encode_all(H, mats, group=16):
    if group <= 1:
        for m in mats:
            H.hq_encode(m["plan"], m["x"], m["s"])
        return
    for g in groups_of(mats, group):
        H.hq_encode_group([m["plan"] for m in g], [m["x"] for m in g], [m["s"] for m in g])


def decode_all(H, mats, group=16):
    if group <= 1:
        for m in mats:
            H.hq_decode(m["plan"], m["s"], out=m["y"])
        return
    for g in groups_of(mats, group):
        H.hq_decode_group([m["plan"] for m in g], [m["s"] for m in g], [m["y"] for m in g])


def cpu_baseline(mats, seconds):
    """The oracle as it stands on row slices of layer 0's seven matrices: one
    thread, then one thread per host core the process may run on (at most 16),
    each encoding and decoding its own slices (the oracle's C calls release
    the GIL), for about `seconds` of wall time each.  Its alpha is the
    oracle's own E8 at 4 bps operating point."""
    from concurrent.futures import ThreadPoolExecutor
    from oracle import oracle as O
    from paper_2606_23406_amd import workloads as W
    pts = json.load(open(os.path.join(ROOT, "tests", "golden", "operating_points.json")))["points"]
    snr = [p["snr_db"] for p in pts if p["lattice"] == "E8" and p["bps"] == 4.0][0]
    names = [n for n, _, _ in W.LLAMA_LINEARS]
    rows_per = {"q": 256, "k": 128, "v": 128, "o": 256, "gate": 512, "up": 512, "down": 256}
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    sample = []
    for m in mats[:7]:
        x = m["x"][:rows_per[m["name"]] * threads].float().cpu().numpy()
        seed = W.llama_linear_seed(m["layer"], names.index(m["name"]))
        P = O.Params(tile=128, lattice=O.E8, alpha=O.alpha(O.E8, snr), rht_seed=seed)
        sample.append((P, x, rows_per[m["name"]]))

    def work(tid, nthreads, budget):
        n = 0
        t_enc = t_dec = 0.0
        t_start = time.perf_counter()
        while time.perf_counter() - t_start < budget:
            for P, x, rows in sample:
                xs = x[(tid % nthreads) * rows:(tid % nthreads + 1) * rows]
                t0 = time.perf_counter()
                st = O.encode(P, xs)
                t1 = time.perf_counter()
                O.decode(P, st)
                t2 = time.perf_counter()
                t_enc += t1 - t0
                t_dec += t2 - t1
                n += xs.size
        return n, t_enc, t_dec

    n1, e1, d1 = work(0, 1, seconds / 2)
    gbs1 = 2.0 * n1 / (e1 + d1) / 1e9
    t0 = time.perf_counter()
    with ThreadPoolExecutor(threads) as ex:
        res = list(ex.map(lambda t: work(t, threads, seconds / 2), range(threads)))
    wall = time.perf_counter() - t0
    nT = sum(r[0] for r in res)
    gbsT = 2.0 * nT / wall / 1e9
    desc = (f"oracle encode+decode on row slices of layer 0 (per thread: q 256, k 128, v 128, o 256, "
            f"gate 512, up 512, down 256 rows), {threads} threads over their own slices: "
            f"{nT / 1e6:.1f}M scalars in {wall:.1f}s wall; 1 thread: {n1 / 1e6:.1f}M scalars "
            f"in {e1 + d1:.1f}s")
    cpu_model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(gbsT, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": desc, "cpu_model": cpu_model,
            "host_cpus_allowed": len(os.sched_getaffinity(0)), "value_1thread": round(gbs1, 4),
            "encode_GBs_1thread": round(2.0 * n1 / e1 / 1e9, 4),
            "decode_GBs_1thread": round(2.0 * n1 / d1 / 1e9, 4)}


def copy_bandwidth(dev, nbytes=1 << 30, reps=5):
    """Device-to-device copy of `nbytes` (hipMemcpyAsync's copy kernel): the
    practical HBM ceiling, and the known-size kernel that scales the HBM byte
    counters."""
    src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) * 1e-3 / reps
    del src, dst
    return round(2.0 * nbytes / t / 1e9, 1)


def measured_traffic(kernel_key):
    """HBM bytes per launch of a codec kernel on this workload, from the
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary in profiles/, if it was taken on
    the current kernel source (else None)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "codec_e8_4bps_llama8b_stack_hbm_traffic.txt")
    src = os.path.join(ROOT, "paper_2606_23406_amd", "csrc", "hq_kernels.hip")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != hashlib.sha256(open(src, "rb").read()).hexdigest():
        return None
    try:
        return float(kv[kernel_key + "_hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _median_ms(fn, reps, flush=None):
    """Median over `reps` runs of fn() on the current stream, each preceded by
    an untimed 1 GiB scratch write when `flush` is given (so inputs smaller
    than the 256 MB last-level cache are read cold)."""
    times = []
    for _ in range(reps):
        if flush is not None:
            flush.fill_(0.0)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        b.synchronize()
        times.append(a.elapsed_time(b))
    times.sort()
    return times[len(times) // 2]


def other_workloads(H, W, dev, reps=20):
    """The other synthetic configurations at 1 GPU: C1 (512x512 fp32), C2
    (4096x4096 bf16 Student-t + outlier columns, E8 at 4 and 3 bps) and C4 (KV
    keys [16, 8192, 8, 128] bf16 with signs rotation, dither and fp16 norms,
    and once at E8@2 with the qjl rotation instead of the signs: 64 appends of
    [16, 128] tokens, then one full dequant), cold (1 GiB
    scratch write between runs).  GB/s are of input bytes (bf16, or fp32 for
    C1); pct_hbm is algorithmic bytes over time against 8 TB/s."""
    import numpy as np
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    out = {}

    def codec(name, x, lattice, bps, kv=False, rows_per_append=None, qjl=None, tile=128, substream=0):
        print(f"[bench] {name}", file=sys.stderr, flush=True)
        rows, cols = x.shape
        opts = dict(rotation=1, dither=True, rot_seed=72, dither_seed=73, norm_fp16=True) if kv else {}
        if qjl is not None:
            opts.update(rotation=H.HQ_ROT_QJL, qjl=qjl)
        plan = H.hq_plan(tile, lattice, bps, 17, -1, cols, substream=substream, **opts)
        s = H.EncodedStream(plan, rows)
        y = torch.empty((rows, cols), dtype=torch.bfloat16, device=dev)
        esz = x.element_size()

        def enc():
            if rows_per_append:
                for r0 in range(0, rows, rows_per_append):
                    H.hq_encode(plan, x[r0:r0 + rows_per_append], s, append=r0 > 0)
            else:
                H.hq_encode(plan, x, s)

        enc()
        H.hq_decode(plan, s, out=y)
        torch.cuda.synchronize()
        s.reset_stats()
        enc()
        torch.cuda.synchronize()
        bits = s.read_stats()["payload_bits"]
        n = x.numel()
        te = _median_ms(enc, reps, flush) * 1e-3
        td = _median_ms(lambda: H.hq_decode(plan, s, out=y), reps, flush) * 1e-3
        side = n / tile * (2 if kv else 4) + n / (substream or 512) * 5
        alg_e = n * esz + bits / 8 + side
        alg_d = bits / 8 + side + n * 2
        e = (y.float() - x.float())
        snr_db = float(10 * torch.log10((x.float() ** 2).sum() / (e * e).sum()))
        out[name] = {"scalars": n, "bits_per_scalar": round(bits / n, 4), "snr_db": round(snr_db, 3),
                     "encode_us": round(te * 1e6, 1), "decode_us": round(td * 1e6, 1),
                     "encode_GBs_in": round(n * esz / te / 1e9, 1),
                     "decode_GBs_out": round(n * 2 / td / 1e9, 1),
                     "encode_pct_hbm": round(100 * alg_e / te / 1e9 / HBM_PEAK_GBS, 2),
                     "decode_pct_hbm": round(100 * alg_d / td / 1e9 / HBM_PEAK_GBS, 2)}
        del s, y

    x1 = torch.from_numpy(W.single_matrix_fp32()).to(dev)
    codec("C1_512x512_fp32_E8@4", x1, H.HQ_E8, 4.0)
    x2 = W.heavy_tailed_weight().to(dev)
    codec("C2_4096x4096_bf16_E8@4", x2, H.HQ_E8, 4.0)
    codec("C2_4096x4096_bf16_E8@3", x2, H.HQ_E8, 3.0)
    # the RHT tile sweep of Sec. 7.2 on the same matrix (weights, E8 at 4 bps)
    for t in (256, 512, 1024, 2048):
        codec(f"C2_4096x4096_bf16_E8@4_tile{t}", x2, H.HQ_E8, 4.0, tile=t)
    # the sub-stream length S of Sec. 5.3 (metadata against parallel occupancy)
    for sl in (1024, 2048):
        codec(f"C2_4096x4096_bf16_E8@4_S{sl}", x2, H.HQ_E8, 4.0, substream=sl)
    del x2
    k = W.kv_cache(device="cpu", role="k")  # [16, 8192, 8, 128], appended 128 tokens at a time
    xk = k.permute(1, 0, 2, 3).reshape(64, 128, 16, 1024).permute(0, 2, 1, 3).reshape(-1, 1024)
    xk = xk.contiguous().to(dev)  # rows (token block, batch, token), one row = 8 head vectors
    del k
    for name, lat, bps in (("E8@2", H.HQ_E8, 2.0), ("A2@1.7", H.HQ_A2, 1.7), ("Z@1.7", H.HQ_Z, 1.7)):
        codec(f"C4_kv_keys_16x8192x8x128_{name}", xk, lat, bps, kv=True, rows_per_append=16 * 128)
    # the qjl rotation (a Haar S drawn here: QR of a seeded Gaussian, sign-fixed)
    g = np.random.default_rng(74).standard_normal((128, 128))
    q, r = np.linalg.qr(g)
    codec("C4_kv_keys_16x8192x8x128_E8@2_qjl", xk, H.HQ_E8, 2.0, kv=True, rows_per_append=16 * 128,
          qjl=(q * np.sign(np.diag(r))).astype(np.float32))
    del xk, flush
    torch.cuda.empty_cache()
    return out


def stack_d4(H, mats, reps=3):
    """The same linear stack with the D4 lattice at 3 bps (whole-model encode
    then decode), on the inputs already resident; median of `reps` steps."""
    print("[bench] C3_llama8b_stack_D4@3", file=sys.stderr, flush=True)
    d4 = []
    for m in mats:
        plan = H.hq_plan(128, H.HQ_D4, 3.0, m["seed"], -1, m["x"].shape[1])
        d4.append({"plan": plan, "x": m["x"], "s": H.EncodedStream(plan, m["x"].shape[0]), "y": m["y"]})
    encode_all(H, d4)
    decode_all(H, d4)
    torch.cuda.synchronize()
    te, td = [], []
    for _ in range(reps):
        a, b, c = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        for m in d4:
            m["s"].reset_stats()
        a.record()
        encode_all(H, d4)
        b.record()
        decode_all(H, d4)
        c.record()
        c.synchronize()
        te.append(a.elapsed_time(b) * 1e-3)
        td.append(b.elapsed_time(c) * 1e-3)
    te, td = sorted(te)[reps // 2], sorted(td)[reps // 2]
    n = sum(m["x"].numel() for m in d4)
    bits = sum(m["s"].read_stats()["payload_bits"] for m in d4)
    ok = all(m["s"].read_stats()["status"] == 0 for m in d4)
    stream_bytes = bits / 8 + 4 * n / 128 + 5 * n / 512
    out = {"scalars": n, "bits_per_scalar": round(bits / n, 4), "encode_ms": round(te * 1e3, 3),
           "decode_ms": round(td * 1e3, 3), "GBs_bf16_in": round(2 * n / (te + td) / 1e9, 1),
           "encode_pct_hbm": round(100 * (2 * n + stream_bytes) / te / 1e9 / HBM_PEAK_GBS, 2),
           "decode_pct_hbm": round(100 * (2 * n + stream_bytes) / td / 1e9 / HBM_PEAK_GBS, 2),
           "device_status_ok": ok}
    del d4
    torch.cuda.empty_cache()
    return out


def gemm_extra(H, W, mats, dev):
    """Dequant-fused int8 GEMM: gate-shaped E8@4 weights x 4096 bf16 tokens."""
    gate = [m for m in mats if m["name"] == "gate"][0]
    plan, s = gate["plan"], gate["s"]
    a = W.activations(device=dev)
    M, N, K = a.shape[0], s.rows, plan.cols
    ws = torch.empty(H.hq_gemm_workspace_bytes(plan, M, N), dtype=torch.uint8, device=dev)
    out = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    xq, sx = H.hq_act_prep(plan, a)
    codes, g = H.hq_decode_int8(plan, s)
    for _ in range(3):
        H.hq_dequant_gemm_int8(plan, s, a, workspace=ws, out=out)
        H.hq_gemm_int8_blockscaled(plan, xq, sx, codes, g, out=out)
    torch.cuda.synchronize()
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    reps = 10
    e0.record()
    for _ in range(reps):
        H.hq_gemm_int8_blockscaled(plan, xq, sx, codes, g, out=out)
    e1.record()
    for _ in range(reps):
        H.hq_dequant_gemm_int8(plan, s, a, workspace=ws, out=out)
    e2.record()
    torch.cuda.synchronize()
    t_gemm = e0.elapsed_time(e1) / reps * 1e-3
    t_e2e = e1.elapsed_time(e2) / reps * 1e-3
    # the fp8 E4M3 cast path on the same operands: GEMM alone, and act prep +
    # decode to E4M3 + GEMM
    x8, sx8 = H.hq_act_prep_fp8(plan, a)
    c8, g8 = H.hq_decode_fp8(plan, s)

    def fp8_e2e():
        xa, sa = H.hq_act_prep_fp8(plan, a)
        cw, gw = H.hq_decode_fp8(plan, s)
        H.hq_gemm_fp8_blockscaled(plan, xa, sa, cw, gw, out=out)

    for _ in range(3):
        H.hq_gemm_fp8_blockscaled(plan, x8, sx8, c8, g8, out=out)
        fp8_e2e()
    torch.cuda.synchronize()
    f0, f1, f2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    f0.record()
    for _ in range(reps):
        H.hq_gemm_fp8_blockscaled(plan, x8, sx8, c8, g8, out=out)
    f1.record()
    for _ in range(reps):
        fp8_e2e()
    f2.record()
    torch.cuda.synchronize()
    t_gemm8 = f0.elapsed_time(f1) / reps * 1e-3
    t_e2e8 = f1.elapsed_time(f2) / reps * 1e-3
    # the MXFP4 cast path: GEMM alone, and act prep + decode to MXFP4 + GEMM
    x4, xs4 = H.hq_act_prep_mxfp4(plan, a)
    c4, ws4 = H.hq_decode_mxfp4(plan, s)

    def mx_e2e():
        xa, xsa = H.hq_act_prep_mxfp4(plan, a)
        cw, wsw = H.hq_decode_mxfp4(plan, s)
        H.hq_gemm_mxfp4_blockscaled(plan, xa, xsa, cw, wsw, out=out)

    for _ in range(3):
        H.hq_gemm_mxfp4_blockscaled(plan, x4, xs4, c4, ws4, out=out)
        mx_e2e()
    torch.cuda.synchronize()
    f0.record()
    for _ in range(reps):
        H.hq_gemm_mxfp4_blockscaled(plan, x4, xs4, c4, ws4, out=out)
    f1.record()
    for _ in range(reps):
        mx_e2e()
    f2.record()
    torch.cuda.synchronize()
    t_gemm4 = f0.elapsed_time(f1) / reps * 1e-3
    t_e2e4 = f1.elapsed_time(f2) / reps * 1e-3
    ops = 2.0 * M * N * K
    # the same product at long RHT tiles (Sec. 7.2): the weight factors span
    # the tile, so the int8 / fp8 rescale runs tile / 128 times less often
    # (MXFP4's block scales carry the factors at any tile)
    sweep = {}
    for tile in (512, 2048):
        tp = H.hq_plan(tile, H.HQ_E8, 4.0, gate["seed"], -1, K)
        ts = H.EncodedStream(tp, N)
        H.hq_encode(tp, gate["x"], ts)
        ci, gi = H.hq_decode_int8(tp, ts)
        xi, sxi = H.hq_act_prep(tp, a)
        cf, gf = H.hq_decode_fp8(tp, ts)
        xf, sxf = H.hq_act_prep_fp8(tp, a)
        cm, wm = H.hq_decode_mxfp4(tp, ts)
        xm, xsm = H.hq_act_prep_mxfp4(tp, a)
        row = {}
        for name, fn, peak in (
                ("int8", lambda: H.hq_gemm_int8_blockscaled(tp, xi, sxi, ci, gi, out=out), INT8_PEAK_TOPS),
                ("fp8", lambda: H.hq_gemm_fp8_blockscaled(tp, xf, sxf, cf, gf, out=out), FP8_PEAK_TFLOPS),
                ("mxfp4", lambda: H.hq_gemm_mxfp4_blockscaled(tp, xm, xsm, cm, wm, out=out),
                 FP4_PEAK_TFLOPS)):
            for _ in range(3):
                fn()
            torch.cuda.synchronize()
            f0.record()
            for _ in range(reps):
                fn()
            f1.record()
            torch.cuda.synchronize()
            tt = f0.elapsed_time(f1) / reps * 1e-3
            row[f"{name}_ms"] = round(tt * 1e3, 4)
            row[f"{name}_frac_peak"] = round(ops / tt / 1e12 / peak, 4)
        sweep[f"tile{tile}"] = row
        del ts, ci, gi, xi, cf, gf, xf, cm, wm, xm
    return {"workload": f"W {N}x{K} E8@4 Rice stream, A {M}x{K} bf16 (1% outlier channels x30)",
            "gemm_ms": round(t_gemm * 1e3, 4), "gemm_TOPS": round(ops / t_gemm / 1e12, 2),
            "gemm_frac_int8_peak": round(ops / t_gemm / 1e12 / INT8_PEAK_TOPS, 4),
            "end_to_end_ms": round(t_e2e * 1e3, 4),
            "end_to_end_TOPS": round(ops / t_e2e / 1e12, 2),
            "fp8_gemm_ms": round(t_gemm8 * 1e3, 4), "fp8_gemm_TOPS": round(ops / t_gemm8 / 1e12, 2),
            "fp8_gemm_frac_fp8_peak": round(ops / t_gemm8 / 1e12 / FP8_PEAK_TFLOPS, 4),
            "fp8_end_to_end_ms": round(t_e2e8 * 1e3, 4),
            "mxfp4_gemm_ms": round(t_gemm4 * 1e3, 4), "mxfp4_gemm_TOPS": round(ops / t_gemm4 / 1e12, 2),
            "mxfp4_gemm_frac_fp4_peak": round(ops / t_gemm4 / 1e12 / FP4_PEAK_TFLOPS, 4),
            "mxfp4_end_to_end_ms": round(t_e2e4 * 1e3, 4),
            "long_tiles": sweep}


def gemv_extra(H, W, mats, dev, reps=10):
    """Fused decode-GEMV (hq_decode_gemv) for one bf16 token through layer 0's
    seven E8@4 matrices, against a bf16 GEMV (torch.mv) on the same weights
    decoded to bf16; both cold (1 GiB scratch write before each run)."""
    layer = [m for m in mats if m["layer"] == 0]
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    xs = [W.activations(device=dev, tokens=1, features=m["plan"].cols)[0].contiguous() for m in layer]
    ws = [torch.empty(H.hq_gemv_workspace_bytes(m["plan"]), dtype=torch.uint8, device=dev)
          for m in layer]
    ys = [torch.empty((m["s"].rows,), dtype=torch.float32, device=dev) for m in layer]
    wb = [H.hq_decode(m["plan"], m["s"], out_dtype=torch.bfloat16) for m in layer]
    yb = [torch.empty((m["s"].rows,), dtype=torch.bfloat16, device=dev) for m in layer]

    def fused():
        for m, x, w, y in zip(layer, xs, ws, ys):
            H.hq_decode_gemv(m["plan"], m["s"], x, workspace=w, out=y)

    def dense():
        for w, x, y in zip(wb, xs, yb):
            torch.mv(w, x, out=y)

    def decode_then_gemv():
        # the unfused baseline: decode each matrix to bf16 in HBM, then GEMV
        for m, w, x, y in zip(layer, wb, xs, yb):
            H.hq_decode(m["plan"], m["s"], out=w)
            torch.mv(w, x, out=y)

    fused()
    dense()
    decode_then_gemv()
    torch.cuda.synchronize()
    tf = _median_ms(fused, reps, flush) * 1e-3
    td = _median_ms(dense, reps, flush) * 1e-3
    tdd = _median_ms(decode_then_gemv, reps, flush) * 1e-3
    n = sum(m["x"].numel() for m in layer)
    stream_bytes = sum(int(m["s"].end_words()) * 4 for m in layer) + n / 128 * 4 + n / 512 * 5
    del flush, wb
    torch.cuda.empty_cache()
    return {"workload": "layer 0 of the stack (7 matrices, 218M E8@4 weights), one bf16 token",
            "fused_ms": round(tf * 1e3, 4), "bf16_gemv_ms": round(td * 1e3, 4),
            "decode_then_gemv_ms": round(tdd * 1e3, 4),
            "speedup_vs_decode_then_gemv": round(tdd / tf, 3),
            "fused_weights_per_s_e9": round(n / tf / 1e9, 1),
            "fused_stream_GBs": round(stream_bytes / tf / 1e9, 1),
            "bf16_gemv_GBs": round(2 * n / td / 1e9, 1),
            "speedup_vs_bf16": round(td / tf, 3)}


def attention_extra(H, W, dev, reps=10):
    """Fused decode-attention (hq_decode_attention): one bf16 query token per
    sequence over the KV workload's cache (batch 16, 8192 tokens, 8 KV heads
    of 128; keys and values E8 at 2 bps with signs rotation, dither and fp16
    norms, appended in 128-token blocks, a stream row being (block,
    sequence, token)), 32 query heads (4 per KV head).  Beside it: decoding
    both streams to bf16 (hq_decode) and attention over a bf16 cache of the
    same shape held contiguous per head (two batched matmuls with contiguous
    right operands and an fp32 softmax); all cold."""
    B, T, Hkv, Hq, D, bt = 16, 8192, 8, 32, 128, 128
    G = Hq // Hkv
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    streams, dense = [], []
    for role, seed in (("k", 91), ("v", 95)):
        x = W.kv_cache(role=role)  # [B, T, Hkv, D]
        dense.append(x.permute(0, 2, 1, 3).contiguous().to(dev))  # [B, Hkv, T, D]
        xr = x.permute(1, 0, 2, 3).reshape(T // bt, bt, B, Hkv * D).permute(0, 2, 1, 3)
        xr = xr.reshape(-1, Hkv * D).contiguous().to(dev)
        del x
        plan = H.hq_plan(128, H.HQ_E8, 2.0, seed, -1, Hkv * D, rotation=1, dither=True,
                         rot_seed=seed + 1, dither_seed=seed + 2, norm_fp16=True)
        s = H.EncodedStream(plan, xr.shape[0])
        for r0 in range(0, xr.shape[0], B * bt):
            H.hq_encode(plan, xr[r0:r0 + B * bt], s, append=r0 > 0)
        del xr
        streams.append((plan, s))
    (pk, sk), (pv, sv) = streams
    table = (torch.arange(T // bt)[None, :] * B + torch.arange(B)[:, None]).to(torch.int32).to(dev)
    lens = torch.full((B,), T, dtype=torch.int32, device=dev)
    q = W.queries(n=B * Hq).reshape(B, Hq, D).to(torch.bfloat16).to(dev)
    ws = torch.empty(H.hq_attention_workspace_bytes(pk, B, Hq, T), dtype=torch.uint8, device=dev)
    out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=dev)
    ybuf = [torch.empty((B * T, Hkv * D), dtype=torch.bfloat16, device=dev) for _ in range(2)]
    qT = q.reshape(B, Hkv, G, D).transpose(-1, -2).contiguous()  # [B, Hkv, D, G]

    def fused():
        H.hq_decode_attention(pk, sk, pv, sv, q, table, lens, bt, workspace=ws, out=out)

    # the 32 most recent tokens kept exact (ring slot t % 32; T is a multiple of 32)
    wk, wv = (d[:, :, T - 32:, :].permute(0, 2, 1, 3).reshape(B, 32, Hkv * D).contiguous()
              for d in dense)

    def fused_window():
        H.hq_decode_attention(pk, sk, pv, sv, q, table, lens, bt, workspace=ws, out=out,
                              window_k=wk, window_v=wv)

    def decode_both():
        H.hq_decode(pk, sk, out=ybuf[0])
        H.hq_decode(pv, sv, out=ybuf[1])

    def attend_bf16():
        sc = torch.matmul(dense[0], qT).float() * D ** -0.5  # [B, Hkv, T, G]
        p = torch.softmax(sc, dim=2).to(torch.bfloat16).transpose(-1, -2).contiguous()
        return torch.matmul(p, dense[1])  # [B, Hkv, G, D]

    fused()
    decode_both()
    ref = attend_bf16()
    torch.cuda.synchronize()
    st = [s.read_stats()["status"] for s in (sk, sv)]
    err = (out.float() - ref.reshape(B, Hq, D).float()).abs().max().item()
    tf = _median_ms(fused, reps, flush) * 1e-3
    tw = _median_ms(fused_window, reps, flush) * 1e-3
    td = _median_ms(decode_both, reps, flush) * 1e-3
    ta = _median_ms(attend_bf16, reps, flush) * 1e-3
    n = 2 * B * T * Hkv * D
    stream_bytes = sum(int(s.end_words()) * 4 for s in (sk, sv)) + n / 128 * 2 + n / 512 * 5
    del flush, ybuf, dense, streams, sk, sv, ws, wk, wv
    torch.cuda.empty_cache()
    return {"workload": "KV cache 16 x 8192 tokens x 8 KV heads x 128, keys and values E8@2, "
                        "32 query heads, one bf16 query token per sequence",
            "fused_ms": round(tf * 1e3, 4), "fused_window32_ms": round(tw * 1e3, 4),
            "decode_then_attend_ms": round((td + ta) * 1e3, 4),
            "decode_both_ms": round(td * 1e3, 4), "bf16_resident_attend_ms": round(ta * 1e3, 4),
            "fused_scalars_per_s_e9": round(n / tf / 1e9, 1),
            "fused_stream_GBs": round(stream_bytes / tf / 1e9, 1),
            "bf16_attend_GBs": round(2 * n / ta / 1e9, 1),
            "speedup_vs_decode_then_attend": round((td + ta) / tf, 3),
            "speedup_vs_bf16_resident": round(ta / tf, 3),
            "cache_bytes_coded": int(stream_bytes), "cache_bytes_bf16": 2 * n,
            "max_abs_diff_vs_unquantized_bf16_attend": round(err, 4), "status": st}


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the codec needs no collective and this build runs on a "
              f"single MI355X (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    from paper_2606_23406_amd import hq as H
    from paper_2606_23406_amd import workloads as W
    H.lib()
    dev = "cuda"
    torch.cuda.set_device(0)

    mats = build_workload(H, W, args.layers, args.bps, dev, args.snr)
    n_scalars = sum(m["x"].numel() for m in mats)
    n_tiles = n_scalars // 128
    n_subs = n_scalars // 512
    torch.cuda.synchronize()

    for _ in range(args.warmup):
        encode_all(H, mats, args.group)
        decode_all(H, mats, args.group)
    for m in mats:
        m["s"].reset_stats()
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        a, b, c = ev[k]
        a.record(stream)
        encode_all(H, mats, args.group)
        b.record(stream)
        decode_all(H, mats, args.group)
        c.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    t_enc = sum(a.elapsed_time(b) for a, b, _ in ev) * 1e-3 / args.steps
    t_dec = sum(b.elapsed_time(c) for _, b, c in ev) * 1e-3 / args.steps
    t_step = t_enc + t_dec

    # realized rate: stats accumulated over the timed steps
    payload_bits = sum(m["s"].read_stats()["payload_bits"] for m in mats) / args.steps
    status = [m["s"].read_stats()["status"] for m in mats]
    bps = payload_bits / n_scalars
    stream_bytes = payload_bits / 8 + 4 * n_tiles + 5 * n_subs  # payload + fp32 norms + offset/k
    enc_bytes = 2 * n_scalars + stream_bytes
    dec_bytes = stream_bytes + 2 * n_scalars
    value = 2.0 * n_scalars / t_step / 1e9
    enc_gbs = enc_bytes / t_enc / 1e9
    dec_gbs = dec_bytes / t_dec / 1e9

    copy_gbs = copy_bandwidth(dev)
    launches = len(groups_of(mats, args.group)) if args.group > 1 else len(mats)
    alg_enc_launch = enc_bytes / launches
    alg_dec_launch = dec_bytes / launches
    tr_enc = measured_traffic("encode")
    tr_dec = measured_traffic("decode")
    out = {
        "metric": "encode+decode GB/s of bf16 input (E8, 4 bps) and % of HBM peak, 1 GPU",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_step * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "Llama-3.1-8B-shaped linear stack, 32 layers x {q,k,v,o,gate,up,down}, "
                               "6.98e9 bf16 weights, E8 lattice at 4 bps, RHT tile 128, encode then "
                               "decode per step",
                   "scalars": n_scalars, "matrices": len(mats), "bps_target": args.bps,
                   "bps_realized": round(bps, 4)},
        "pct_hbm_peak": round(100.0 * (enc_bytes + dec_bytes) / t_step / 1e9 / HBM_PEAK_GBS, 2),
        "roofline": {"bound": "hbm", "kernel": "hq_encode_group_kernel (E8, bf16 in)",
                     "achieved": round(enc_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(enc_gbs / HBM_PEAK_GBS, 4),
                     "traffic": None if tr_enc is None else round(tr_enc),
                     "algorithmic_bytes_per_launch": round(alg_enc_launch),
                     "algorithmic_bytes_per_scalar": round(enc_bytes / n_scalars, 4),
                     "launches_per_step": launches},
        "decode_roofline": {"bound": "hbm", "kernel": "hq_decode_group_kernel (E8, bf16 out)",
                            "achieved": round(dec_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                            "frac": round(dec_gbs / HBM_PEAK_GBS, 4),
                            "traffic": None if tr_dec is None else round(tr_dec),
                            "algorithmic_bytes_per_launch": round(alg_dec_launch),
                            "launches_per_step": launches,
                            "algorithmic_bytes_per_scalar": round(dec_bytes / n_scalars, 4)},
        "copy_GBs_device": copy_gbs,
        "encode_ms": round(t_enc * 1e3, 4),
        "decode_ms": round(t_dec * 1e3, 4),
        "encode_GBs_bf16_in": round(2.0 * n_scalars / t_enc / 1e9, 1),
        "decode_GBs_bf16_out": round(2.0 * n_scalars / t_dec / 1e9, 1),
        "wall_s_timed": round(wall, 3),
        "device_status_ok": all(s == 0 for s in status),
    }
    if not args.no_gemm:
        out["gemm_int8"] = gemm_extra(H, W, mats, dev)
        out["decode_gemv"] = gemv_extra(H, W, mats, dev)
    if not args.no_attention:
        out["decode_attention"] = attention_extra(H, W, dev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(mats, args.cpu_seconds)
    if not args.no_other:
        other = {"C3_llama8b_stack_D4@3": stack_d4(H, mats)}
        other.update(other_workloads(H, W, dev))
        out["other_workloads"] = other
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
