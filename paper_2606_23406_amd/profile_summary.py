"""Turn rocprofv3 counter CSVs of a bench.py run into the short text
summaries kept under profiles/.

    python -m paper_2606_23406_amd.profile_summary traffic FETCH.csv WRITE.csv BENCH.log OUT.txt CMD...
    python -m paper_2606_23406_amd.profile_summary counters OUT.txt SCALARS CSV... -- CMD...
    python -m paper_2606_23406_amd.profile_summary stats KERNEL_STATS.csv BENCH.log OUT.md CMD

`traffic`: HBM bytes per launch of the E8 bf16 encode and decode kernels.
FETCH_SIZE and WRITE_SIZE (KiB per dispatch) come from two separate runs;
each is scaled by what the same counter reads for the 1 GiB device-to-device
copy that bench.py performs (a kernel of known traffic: 1 GiB read, 1 GiB
written).  The summary carries the SHA-256 of the kernel source it was taken
on, so bench.py reports the figure only while the kernels are unchanged.

`stats`: rocprofv3 --stats kernel times of a default bench.py run next to the
bench line's own HIP-event figures.

`counters`: instruction and cycle counters of the codec kernels, the three
GEMMs and the fused one-token kernels, summed over every dispatch of each
kernel; the codec columns also per scalar, SCALARS being the scalars each
codec direction processed in the run.  Derived lines, for the kernels whose
counters include SQ_BUSY_CYCLES: SQ_BUSY_CYCLES counts each of the 32 shader
engines (it reads four times GRBM_GUI_ACTIVE, which counts each of the 8
XCDs), so a dispatch's SIMD-cycles are SQ_BUSY_CYCLES / 32 x 1024 SIMDs, and
  VALU (SALU) instructions per SIMD-cycle = SQ_INSTS_VALU (SALU) / (32 SQ_BUSY_CYCLES),
  MFMA busy                                = SQ_VALU_MFMA_BUSY_CYCLES / (32 SQ_BUSY_CYCLES).
A SIMD issues at most one wave64 VALU instruction per ~2.5 cycles of the fast
forms and ~4.3 of the slow ones (0.4 and 0.23 per cycle).
"""
import csv
import hashlib
import json
import os
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2606_23406_amd", "csrc", "hq_kernels.hip")
KERNELS = {
    "encode": "hq_encode_group_kernel<0, 0, false>",
    "decode": "hq_decode_group_kernel<0, 1, false>",
    "gemm": "hq_gemm_i8_kernel",
    "gemm_fp8": "hq_gemm_f8_kernel",
    "gemm_mxfp4": "hq_gemm_mx4_kernel",
    "decode_gemv": "hq_decode_gemv_kernel",
    "decode_gemv_rows": "hq_decode_gemv_rows_kernel",
    "attention_keys": "hq_attn_kernel<0, 4, false>",
    "attention_values": "hq_attn_kernel<0, 4, true>",
    "copy": "__amd_rocclr_copyBuffer",
}
CODEC = ("encode", "decode")
SIMDS, SHADER_ENGINES = 1024, 32


def read_counter(path, counter):
    """{kernel key: [value per dispatch]} for one counter."""
    out = defaultdict(list)
    per_dispatch = defaultdict(float)
    names = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        d = r.get("Dispatch_Id") or r.get("Correlation_Id") or str(len(per_dispatch))
        per_dispatch[d] += float(r["Counter_Value"])
        names[d] = r["Kernel_Name"]
    for d, v in per_dispatch.items():
        for key, pat in KERNELS.items():
            if pat in names[d]:
                out[key].append(v)
    return out


def bench_json(log):
    for line in open(log):
        line = line.strip()
        if line.startswith("{") and '"metric"' in line:
            return json.loads(line)
    raise ValueError(f"no bench JSON line in {log}")


def traffic(fetch_csv, write_csv, log, out, cmd):
    fetch = read_counter(fetch_csv, "FETCH_SIZE")
    write = read_counter(write_csv, "WRITE_SIZE")
    gib_kib = float(1 << 20)
    # the 1 GiB copies are the copy dispatches that read at least half a GiB
    cf = [v for v in fetch["copy"] if v >= gib_kib / 2]
    cw = [v for v in write["copy"] if v >= gib_kib / 2]
    sf, sw = gib_kib / (sum(cf) / len(cf)), gib_kib / (sum(cw) / len(cw))
    b = bench_json(log)
    lines = [
        "# HBM traffic per launch: E8 at 4 bps, bf16, Llama-3.1-8B-shaped linear stack (224 matrices)",
        "# FETCH_SIZE and WRITE_SIZE (KiB per dispatch, two rocprofv3 runs), each scaled by",
        "# 1 GiB / (the same counter on bench.py's 1 GiB device copy). Commands (repository root):",
    ] + [f"#   {c}" for c in cmd] + [
        f"source_sha256 = {hashlib.sha256(open(SRC, 'rb').read()).hexdigest()}",
        f"copy_dispatches = {len(cf)}",
        f"copy_fetch_kib = {sum(cf) / len(cf):.1f}",
        f"copy_write_kib = {sum(cw) / len(cw):.1f}",
        f"scale_fetch = {sf:.5f}",
        f"scale_write = {sw:.5f}",
    ]
    for key, roof in (("encode", "roofline"), ("decode", "decode_roofline")):
        f, w = fetch[key], write[key]
        fk, wk = sum(f) / len(f), sum(w) / len(w)
        hbm = fk * 1024 * sf + wk * 1024 * sw
        alg = b[roof]["algorithmic_bytes_per_launch"]
        lines += [
            f"{key}_dispatches = {len(f)}",
            f"{key}_fetch_kib_per_launch = {fk:.1f}",
            f"{key}_write_kib_per_launch = {wk:.1f}",
            f"{key}_hbm_bytes_per_launch = {hbm:.0f}",
            f"{key}_algorithmic_bytes_per_launch = {alg}",
            f"{key}_traffic_over_algorithmic = {hbm / alg:.4f}",
        ]
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def counters(out, scalars, csvs, cmd):
    vals = defaultdict(lambda: defaultdict(float))
    disp = defaultdict(set)
    for path in csvs:
        for r in csv.DictReader(open(path)):
            for key, pat in KERNELS.items():
                if pat in r["Kernel_Name"]:
                    vals[key][r["Counter_Name"]] += float(r["Counter_Value"])
                    disp[(key, r["Counter_Name"])].add(r.get("Dispatch_Id", ""))
    lines = ["# Instruction and cycle counters, summed over every dispatch of each kernel.",
             "# Commands (repository root):"] + [f"#   {c}" for c in cmd]
    lines.append(f"# per scalar = total / {scalars:.0f} scalars (codec kernels)")
    for key in KERNELS:
        if key not in vals or key == "copy":
            continue
        lines.append(f"[{key}: {KERNELS[key]}]")
        for c in sorted(vals[key]):
            n = len(disp[(key, c)])
            per = f"  per scalar {vals[key][c] / scalars:.4f}" if key in CODEC else ""
            lines.append(f"{c:28s} total {vals[key][c]:.4g}  dispatches {n}{per}")
        v = vals[key]
        busy = v.get("SQ_BUSY_CYCLES", 0.0)
        if busy > 0:
            simd_cycles = busy / SHADER_ENGINES * SIMDS
            for c, label in (("SQ_INSTS_VALU", "VALU instructions per SIMD-cycle"),
                             ("SQ_INSTS_SALU", "SALU instructions per SIMD-cycle"),
                             ("SQ_VALU_MFMA_BUSY_CYCLES", "MFMA busy")):
                if c in v:
                    lines.append(f"= {label:36s} {v[c] / simd_cycles:.4f}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def stats(stats_csv, log, out, cmd):
    b = bench_json(log)
    steps = b["steps"] + b["warmup"]
    n = b["config"]["scalars"]
    rows = list(csv.DictReader(open(stats_csv)))
    lines = ["# Kernel time: E8 at 4 bps codec over the Llama-3.1-8B-shaped linear stack", "",
             "Command (repository root, one MI355X):", "", f"    {cmd}", "",
             f"One step = encode then decode of the 224 matrices ({n} bf16 weights) in "
             f"{b['roofline']['launches_per_step']} launches each way (hq_encode_group / "
             f"hq_decode_group, up to 16 matrices per launch); {steps} steps ran "
             f"({b['warmup']} warmup + {b['steps']} timed). The other rows come from the rest "
             "of the run (the GEMM, the fused decode-GEMV and decode-attention legs, the D4 "
             "stack, the C1/C2/C4 configurations).", "",
             "| kernel | calls | total ms | avg us | min us | max us |", "|---|---|---|---|---|---|"]
    per = {}
    for r in rows:
        name = r["Name"]
        if "hq_" not in name and "copyBuffer" not in name:
            continue
        short = name.replace("void ", "").replace("(anonymous namespace)::", "").split("(")[0]
        lines.append(f"| `{short}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
                     f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                     f"{float(r['MaxNs']) / 1e3:.2f} |")
        for key in ("encode", "decode"):
            if KERNELS[key] in name:
                per[key] = float(r["TotalDurationNs"]) / steps * 1e-9
    te, td = per["encode"], per["decode"]
    lines += ["", f"Kernel time per step: encode {te * 1e3:.2f} ms, decode {td * 1e3:.2f} ms; "
              f"bf16 input rate encode {2 * n / te / 1e9:.0f} GB/s, decode {2 * n / td / 1e9:.0f} GB/s, "
              f"encode + decode {2 * n / (te + td) / 1e9:.0f} GB/s.",
              f"The bench line of the same run (HIP events on the launch stream): value {b['value']} GB/s, "
              f"encode {b['encode_ms']} ms, decode {b['decode_ms']} ms per step; "
              f"encode roofline {b['roofline']['achieved']} GB/s of algorithmic bytes "
              f"({b['roofline']['frac']:.4f} of 8 TB/s); device copy {b.get('copy_GBs_device')} GB/s."]
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    mode = sys.argv[1]
    if mode == "traffic":
        traffic(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5], sys.argv[6:])
    elif mode == "stats":
        stats(sys.argv[2], sys.argv[3], sys.argv[4], " ".join(sys.argv[5:]))
    elif mode == "counters":
        args = sys.argv[2:]
        cut = args.index("--")
        counters(args[0], float(args[1]), args[2:cut], args[cut + 1:])
    else:
        raise SystemExit(__doc__)
