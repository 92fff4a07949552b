"""Write tests/golden/operating_points.json with the oracle only.

App. B: the target rate b is turned into an SNR by inverting the realized
Rice rate measured on iid-Gaussian tiles (~1e5 tiles, seed 42 in the paper).
Here each operating point is found by bisection on the SNR, with the oracle
encoding 2^12 seeded N(0, 1) tiles of 128 scalars per evaluation (the rate
is the unpadded payload bits per scalar).  Test infrastructure only.

Usage: python -m oracle.make_operating_points
"""
import json
import os

import numpy as np

from . import oracle as O

POINTS = [("E8", 2.0), ("E8", 3.0), ("E8", 4.0), ("E8", 5.0), ("D4", 3.0), ("D4", 4.0), ("D4", 5.0),
          ("A2", 1.7), ("A2", 4.0), ("A2", 5.0), ("Z", 1.7), ("Z", 4.0), ("Z", 5.0)]
N_TILES = 4096
TILE = 128
SEED = 42


def gaussian_rows(seed=SEED, n_tiles=N_TILES, tile=TILE, substream=512):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n_tiles, tile)).astype(np.float32)
    return x.reshape(-1, substream)


def realized_bps(lat, snr_db, x, rice_k=-1):
    P = O.Params(tile=TILE, lattice=lat, alpha=O.alpha(lat, snr_db), rice_k=rice_k)
    st = O.encode(P, x)
    return st.payload_bits / x.size


def snr_for_bps(lat, bps, x, lo=-10.0, hi=50.0, iters=40):
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        if realized_bps(lat, mid, x) < bps:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def main():
    x = gaussian_rows()
    out = {"source": "oracle bisection on 2^12 iid N(0,1) tiles of 128, numpy PCG64 seed 42",
           "points": []}
    for name, bps in POINTS:
        lat = O.LATTICES[name]
        snr = snr_for_bps(lat, bps, x)
        out["points"].append({"lattice": name, "bps": bps, "snr_db": round(snr, 4),
                              "realized_bps": round(realized_bps(lat, round(snr, 4), x), 5),
                              "alpha": float(O.alpha(lat, round(snr, 4)))})
        print(out["points"][-1], flush=True)
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "tests",
                        "golden", "operating_points.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
