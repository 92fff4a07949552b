"""Measure this library's SNR -> bits-per-scalar curves and write
csrc/calib_table.inc (App. B: the target rate is mapped to an SNR by
inverting the realized Rice rate measured on iid-Gaussian tiles).

For every lattice and Rice setting (automatic k and fixed k = 0..6) the
library's own encoder runs on 2^15 seeded N(0, 1) tiles of 128 scalars at an
SNR grid of -10 .. 40 dB in 0.1 dB steps; the realized rate is the unpadded
payload bits per scalar reported by the encoder.  Needs a GPU.

    python -m paper_2606_23406_amd.calibrate [--out PATH]
"""
import argparse
import os
import time

import numpy as np
import torch

from . import hq as H
from . import workloads

SNR0, SNR1, STEP = -10.0, 40.0, 0.1
N_TILES = 1 << 15
RICE = [-1, 0, 1, 2, 3, 4, 5, 6]


def measure_curve(x, lattice, rice_k, snrs):
    out = np.zeros(len(snrs), dtype=np.float64)
    s = None
    for i, snr in enumerate(snrs):
        plan = H.hq_plan(128, lattice, 0.0, 42, rice_k, x.shape[1], snr_db=float(snr))
        if s is None or s.plan.info.max_words_per_row < plan.info.max_words_per_row:
            s = H.EncodedStream(plan, x.shape[0])
        else:
            s.plan = plan
        s.reset_stats()
        H.hq_encode(plan, x, s)
        st = s.read_stats()
        if st["status"] != 0:
            raise RuntimeError(f"encode status {st['status']} at {lattice} k={rice_k} snr={snr}")
        out[i] = st["payload_bits"] / x.numel()
    return out


def write_inc(path, curves):
    lines = [
        "// SNR -> realized payload bits-per-scalar curves (App. B), one per lattice and",
        "// Rice setting, measured by paper_2606_23406_amd/calibrate.py with this",
        "// library's own encoder on 2^15 seeded iid N(0, 1) tiles of 128 scalars",
        "// (running maximum over the grid, so the curve is monotone).  Generated file.",
        "struct hq_calib_curve {",
        "  int lattice;",
        "  int rice_k;",
        "  double snr0;",
        "  double step;",
        "  int n;",
        "  const float* bps;",
        "};",
    ]
    names = []
    for (lat, k), v in curves.items():
        name = f"kCurve_{lat}_{'auto' if k < 0 else k}"
        names.append((lat, k, name, len(v)))
        vals = ", ".join(f"{x:.6f}f" for x in v)
        lines.append(f"static const float {name}[{len(v)}] = {{{vals}}};")
    lines.append("static const hq_calib_curve kCalib[] = {")
    for lat, k, name, n in names:
        lines.append(f"    {{{lat}, {k}, {SNR0:.1f}, {STEP:.1f}, {n}, {name}}},")
    lines.append("};")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=os.path.join(os.path.dirname(__file__), "csrc",
                                                  "calib_table.inc"))
    args = ap.parse_args()
    snrs = np.round(np.arange(SNR0, SNR1 + 1e-9, STEP), 4)
    x = workloads.gaussian_tiles(N_TILES, 128, seed=42, device="cuda").reshape(-1, 512).contiguous()
    curves = {}
    t0 = time.time()
    for lat in (H.HQ_E8, H.HQ_D4, H.HQ_A2, H.HQ_Z):
        for k in RICE:
            v = np.maximum.accumulate(measure_curve(x, lat, k, snrs))
            curves[(lat, k)] = v
            print(f"lattice {lat} k {k}: bps {v[0]:.3f} .. {v[-1]:.3f}  ({time.time() - t0:.1f}s)",
                  flush=True)
    write_inc(args.out, curves)
    print("wrote", args.out)


if __name__ == "__main__":
    main()
