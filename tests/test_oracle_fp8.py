"""Pins of the oracle's fp8 cast path (Sec. 4.8 / 6.3: E4M3 at the MMA
boundary), CPU only.  The cast is pinned to the OCP E4M3 format: every finite
code round-trips, printed values (1, 448, the smallest subnormal 2^-9), ties
to the even code, saturation at 448; the activation prep against the int8
one's transform; the GEMM against a dense product of the cast values."""
import numpy as np
import pytest

from oracle import oracle as O


def test_every_finite_code_round_trips():
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)
    v = O.e4m3_value(codes)
    back = O.e4m3_bits(v)
    assert np.array_equal(back, codes)  # -0 included (0x80)


def test_printed_values_and_ties():
    assert O.e4m3_value(np.array([0x38], np.uint8))[0] == 1.0
    assert O.e4m3_value(np.array([0x7E], np.uint8))[0] == 448.0
    assert O.e4m3_value(np.array([0x01], np.uint8))[0] == 2.0 ** -9
    assert O.e4m3_value(np.array([0x08], np.uint8))[0] == 2.0 ** -6   # smallest normal
    vals = O.e4m3_value(O.e4m3_bits([17.0, 19.0, 21.0, 2.0 ** -10, 3 * 2.0 ** -10, -17.0, 500.0, -1e9]))
    # 17 ties 16 / 18 -> 16 (even); 19 ties 18 / 20 -> 20; 21 -> 20; 2^-10 ties 0 / 2^-9 -> 0;
    # 3 * 2^-10 ties 2^-9 / 2^-8 -> 2^-8 (code 2, even); saturation at 448
    assert list(vals) == [16.0, 20.0, 20.0, 0.0, 2.0 ** -8, -16.0, 448.0, -448.0]
    # integers are exact to 16, then spaced by 2, 4, 8 ...
    ints = np.arange(-16, 17)
    assert np.array_equal(O.e4m3_value(O.e4m3_bits(ints)), ints)


def test_nearest_value_by_brute_force():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(4000) * 10, rng.standard_normal(1000) * 1e-2])
    allv = O.e4m3_value(np.arange(0x7F, dtype=np.uint8))
    got = np.abs(O.e4m3_value(O.e4m3_bits(x)))
    best = allv[np.argmin(np.abs(np.abs(x)[:, None] - allv[None, :]), axis=1)]
    assert np.array_equal(got, best)  # no exact ties in random data


def test_act_prep_fp8_transform_and_scale():
    rng = np.random.default_rng(2)
    a = rng.standard_normal((6, 512)).astype(np.float32)
    x8, sx = O.act_prep_fp8(a, 128, 9)
    y = O.fwht((a * O.signs(9, 512)).reshape(6, 4, 128).astype(np.float64)).reshape(6, 512)
    assert np.allclose(sx * 448.0, np.abs(y).max(axis=1), rtol=1e-6)
    rec = O.e4m3_value(x8) * sx[:, None]
    # E4M3 keeps 3 fraction bits: relative error at most 2^-4 above the subnormals
    big = np.abs(y) > 2.0 ** -6 * sx[:, None] * 2
    assert np.all(np.abs(rec - y)[big] <= np.abs(y)[big] * 2.0 ** -4 + 1e-7)
    assert np.all(np.abs(O.e4m3_value(x8)) <= 448.0)
    assert np.any(np.abs(O.e4m3_value(x8)) == 448.0)


def test_gemm_fp8_matches_dense_product():
    rng = np.random.default_rng(3)
    w8 = O.weight_codes_fp8(rng.integers(-40, 41, (24, 256)))
    x8 = O.e4m3_bits(rng.standard_normal((5, 256)) * 50)
    g = rng.random((24, 2)).astype(np.float32)
    sx = rng.random(5).astype(np.float32)
    out = O.gemm_fp8_blockscaled(w8, g, x8, sx, 128)
    W = O.e4m3_value(w8) * np.repeat(g.astype(np.float64), 128, axis=1)
    ref = (O.e4m3_value(x8) @ W.T) * sx[:, None].astype(np.float64)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-9)
