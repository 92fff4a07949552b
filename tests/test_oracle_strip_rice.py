"""Pins of the oracle's strip, zig-zag and Rice stages (CPU only)."""
import math

import numpy as np
import pytest

from oracle import oracle as O
from tests.test_oracle_lattice import enumerate_box, member

LATS = [O.E8, O.D4, O.A2, O.Z]
GOLDEN = __import__("os").path.join(__import__("os").path.dirname(__file__), "golden")


def test_zigzag_values_and_bijection():
    # Sec. 4.6: zigzag(n) = 2n for n >= 0, -2n - 1 for n < 0.
    assert [O.zigzag(v) for v in (0, -1, 1, -2, 2, -3, 3)] == [0, 1, 2, 3, 4, 5, 6]
    vals = list(range(-3000, 3000))
    zz = [O.zigzag(v) for v in vals]
    assert sorted(zz) == list(range(6000))
    assert [O.unzigzag(m) for m in zz] == vals


@pytest.mark.parametrize("lat,box", [(O.D4, 6), (O.A2, 9), (O.Z, 60)])
def test_strip_bijection_exhaustive(lat, box):
    # P6: on every lattice code of a box, unstrip(strip(c)) = c ...
    m = O.DIM[lat]
    c = enumerate_box(lat, [-box] * m, [box] * m)
    s = O.strip(lat, c)
    assert np.array_equal(O.unstrip(lat, s), c)
    # ... and strip is onto Z^m: every symbol tuple comes from a member.
    sy = enumerate_box(O.Z, [0] * m, [7] * m) if m > 1 else np.arange(8)[:, None]
    sy = np.array(np.meshgrid(*[np.arange(8)] * m, indexing="ij")).reshape(m, -1).T
    cc = O.unstrip(lat, sy.astype(np.uint32))
    assert np.all(member(lat, cc))
    assert np.array_equal(O.strip(lat, cc), sy.astype(np.uint32))


def test_strip_bijection_e8_random():
    rng = np.random.default_rng(11)
    sy = rng.integers(0, 200, size=(200000, 8)).astype(np.uint32)
    c = O.unstrip(O.E8, sy)
    assert np.all(member(O.E8, c))
    assert np.array_equal(O.strip(O.E8, c), sy)
    c2 = O.unstrip(O.E8, O.strip(O.E8, c))
    assert np.array_equal(c2, c)


@pytest.mark.parametrize("lat,saving", [(O.E8, 1.0), (O.D4, 0.25), (O.A2, 0.5), (O.Z, 0.0)])
def test_strip_saving_is_the_lattice_index(lat, saving):
    # Tab. lattices-int: bits stripped per scalar = log2([Z^m : lattice]) / m.
    # Count members in a box that is a union of 4Z^m cells: exact density.
    m = O.DIM[lat]
    B = 2 if lat == O.E8 else 8  # 2B divisible by 4
    c = enumerate_box(lat, [-B] * m, [B - 1] * m)
    dens = c.shape[0] / (2 * B) ** m
    assert math.isclose(-math.log2(dens) / m, saving, abs_tol=1e-12)


def test_rice_golden_split_layout():
    g = {}
    for line in open(f"{GOLDEN}/rice_split_layout.txt"):
        if line.strip() and not line.startswith("#"):
            key, *vals = line.split()
            g[key] = [int(v) for v in vals]
    P = O.Params(lattice=O.Z)
    words, nbits = O.rice_put(P, np.array(g["symbols"], dtype=np.uint32), g["k"][0])
    assert nbits == g["bits"][0]
    assert list(words) == g["words"]


@pytest.mark.parametrize("lat", LATS)
@pytest.mark.parametrize("k", [0, 1, 3, 7])
def test_rice_round_trip_and_length(lat, k):
    # P8: lossless round trip; length = sum(floor(m/2^k) + 1 + k) exactly.
    rng = np.random.default_rng(17 + k + 10 * lat)
    S = 512
    sym = rng.geometric(0.15, size=S).astype(np.uint32) - 1
    sym[::37] += 300  # long unary codes too
    P = O.Params(lattice=lat)
    k1 = max(k - 1, 0) if lat == O.D4 else (k + 2 if lat == O.A2 else k)
    words, nbits = O.rice_put(P, sym, k, k1)
    m = O.DIM[lat]
    kk = np.array([(k1 if ((lat == O.D4 and i % m == 3) or (lat == O.A2 and i % m == 1)) else k)
                   for i in range(S)])
    assert nbits == int(((sym.astype(np.int64) >> kk) + 1 + kk).sum())
    back, used = O.rice_get(P, words, S, k, k1)
    assert used == nbits
    assert np.array_equal(back, sym)
    # truncated stream is detected, not over-read
    _, used_t = O.rice_get(P, words[: max(len(words) - 3, 0)], S, k, k1)
    assert used_t == -1


def test_rice_kstar_formula_vs_brute_force():
    # Sec. 3.3 prints k* = floor(log2(ceil(-ln(2-p)/ln(1-p)))): the floor of
    # log2 of the optimal Golomb parameter of a geometric source
    # P(m) = p (1-p)^m.  Brute force over the exact expected Rice length
    # k + 1 + E[floor(m / 2^k)] = k + 1 + a / (1 - a), a = (1-p)^(2^k), shows
    # that the optimal Rice parameter is always k* or k* + 1 (the printed
    # formula alone is short by one step for part of the range).  This is
    # what the codec's per-sub-stream k implements: the better of k* and k*+1.
    ps = np.concatenate([np.linspace(1e-4, 0.999, 20000), np.exp(np.linspace(np.log(3e-5), np.log(0.5), 3000))])
    formula_short = 0
    for p in ps:
        a = (1 - p) ** (2.0 ** np.arange(24))
        costs = np.arange(24) + 1 + a / (1 - a)
        best = costs.min()
        kst = O.rice_kstar(p)
        assert min(costs[kst], costs[kst + 1]) - best < 1e-9, p
        formula_short += costs[kst] - best > 1e-9
    assert formula_short > 0


def test_rice_k_auto_is_monotone():
    # the geometric parameter estimate p = n / (n + sum) falls as the sum
    # grows, so k never decreases
    for n in (256, 384, 512):
        ks = [O.rice_k_auto(n, s) for s in range(0, 60000, 7)]
        assert all(b >= a for a, b in zip(ks, ks[1:]))
        assert ks[0] == 0
