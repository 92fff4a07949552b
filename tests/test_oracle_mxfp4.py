"""Pins of the oracle's MXFP4 cast path (Sec. 4.8 Cast and Sec. 6.4: the
lattice output fed to MXFP4, 32-element blocks with power-of-two scales),
CPU only.  The cast is pinned to the OCP Microscaling format it names: the
E2M1 element values and codes, ties to the even code, saturation at 6, the
E8M0 scale rule X = floor(log2 amax) - 2 at block boundaries, brute-force
nearest values, the activation side's transform, the weight side's cast of
the reconstruction (the tile factor inside the cast: a worked example, a
power-of-two property, the MX error bound) and the GEMM against a
brute-force sum of the cast values."""
import numpy as np
import pytest

from oracle import oracle as O


def test_every_code_round_trips_and_values():
    codes = np.arange(16, dtype=np.uint8)
    v = O.e2m1_value(codes)
    assert list(v[:8]) == [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
    assert np.array_equal(v[8:], -v[:8])
    assert np.array_equal(O.e2m1_bits(v), codes)  # -0 is code 8


def test_ties_to_even_and_saturation():
    x = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 7.0, 100.0, -0.25, -5.0, 0.2, -0.1]
    got = list(O.e2m1_value(O.e2m1_bits(x)))
    # each tie goes to the neighbour with an even code (0, 2, 4, 6 -> 0, 1, 2, 4)
    assert got == [0.0, 1.0, 1.0, 2.0, 2.0, 4.0, 4.0, 6.0, 6.0, 0.0, -4.0, 0.0, 0.0]
    assert O.e2m1_bits([-0.1])[0] == 8  # sign kept


def test_nearest_value_by_brute_force():
    rng = np.random.default_rng(4)
    x = rng.standard_normal(5000) * 3
    got = np.abs(O.e2m1_value(O.e2m1_bits(x)))
    best = O._E2M1[np.argmin(np.abs(np.minimum(np.abs(x), 6.0)[:, None] - O._E2M1[None, :]), axis=1)]
    assert np.array_equal(got, best)  # no exact ties in random data


def test_scale_rule_at_block_boundaries():
    # X = floor(log2 amax) - 2: amax 6 -> 2^0 (6 exact), 8 -> 2^1 (8 -> 4),
    # 7 -> 2^0 (7 saturates to 6), 0.75 -> 2^-3 (6 exactly), 1e-3 ->
    # 2^-12; an all-zero block -> 2^-127 (code 0)
    for amax, X, top in [(6.0, 0, 6.0), (8.0, 1, 4.0), (7.0, 0, 6.0), (0.75, -3, 6.0),
                         (1e-3, -12, None), (0.0, -127, 0.0)]:
        v = np.zeros((1, 32))
        v[0, 5] = amax
        codes, scales = O.mxfp4_cast(v)
        assert int(scales[0, 0]) - 127 == X, (amax, scales)
        if top is not None:
            assert O.e2m1_value(codes)[0, 5] == top
    # 2^X times a code never exceeds amax by more than the top saturation
    rng = np.random.default_rng(5)
    v = rng.standard_normal((64, 256)) * np.exp(rng.uniform(-8, 8, (64, 1)))
    codes, scales = O.mxfp4_cast(v)
    rec = O.mxfp4_value(codes, scales)
    amax = np.abs(v).reshape(64, 8, 32).max(axis=2)
    step = np.ldexp(1.0, scales.astype(np.int32) - 127)
    assert np.all(amax / step >= 4) and np.all(amax / step < 8)
    err = np.abs(rec - v).reshape(64, 8, 32)
    # half the largest spacing (2 at the top binade) plus the saturation of [6, 8)
    assert np.all(err <= (2.0 * step)[:, :, None] + 1e-12)


def test_act_prep_mxfp4_transform():
    rng = np.random.default_rng(6)
    a = rng.standard_normal((5, 512)).astype(np.float32)
    a[:, 3] *= 30
    codes, scales = O.act_prep_mxfp4(a, 128, 8)
    y = O.fwht((a * O.signs(8, 512)).reshape(5, 4, 128).astype(np.float64)).reshape(5, 512)
    rec = O.mxfp4_value(codes, scales)
    amax = np.abs(y).reshape(5, 16, 32).max(axis=2)
    assert np.array_equal(scales.astype(np.int32) - 127, O.mx_scale_exponent(amax))
    assert np.all(np.abs(rec - y).reshape(5, 16, 32) <= (amax / 4)[:, :, None] + 1e-5)


def test_weight_cast_carries_the_tile_factor():
    # worked example: codes 8 and 3 in one block, tile factor 0.75 -> the
    # reconstruction 6.0 and 2.25; amax 6 -> X = 0; 6.0 is code 7 and 2.25
    # rounds to 2 (code 4).  Casting the bare codes instead would give X = 1
    # and 8 -> 4.0, 3 -> 1.5, i.e. 6.0 and 2.25 after the factor: the two
    # readings differ exactly there.
    c = np.zeros((1, 128), dtype=np.int32)
    c[0, 0], c[0, 1] = 8, 3
    codes, scales = O.weight_codes_mxfp4(c, np.array([[0.75]], np.float32), 128)
    assert int(scales[0, 0]) == 127
    assert list(codes[0, :2]) == [7, 4]
    assert list(O.mxfp4_value(codes, scales)[0, :2]) == [6.0, 2.0]
    assert (codes[0, 2:] == 0).all() and (scales[0, 1:] == 0).all()  # all-zero blocks: X = -127


def test_power_of_two_factor_only_moves_the_scales():
    # g = 2^-3 is exact in every product: the element codes are the bare
    # codes' and each block scale is 3 binades lower
    rng = np.random.default_rng(9)
    c = rng.integers(-60, 61, (6, 256))
    g = np.full((6, 2), 0.125, np.float32)
    k1, s1 = O.weight_codes_mxfp4(c, g, 128)
    k0, s0 = O.mxfp4_cast(c.astype(np.float64))
    assert np.array_equal(k1, k0)
    nz = s0 > 0
    assert np.array_equal(s1.astype(np.int32)[nz], s0.astype(np.int32)[nz] - 3)


def test_weight_cast_within_the_mx_bound_of_the_reconstruction():
    rng = np.random.default_rng(10)
    c = rng.integers(-90, 91, (8, 512))
    g = (rng.random((8, 4)) * 0.03 + 1e-3).astype(np.float32)
    codes, scales = O.weight_codes_mxfp4(c, g, 128)
    v = c * np.repeat(g.astype(np.float64), 128, axis=1)
    rec = O.mxfp4_value(codes, scales)
    step = np.ldexp(1.0, scales.astype(np.int32) - 127)
    # half the largest spacing of E2M1 (2 at the top binade) plus the saturation of [6, 8)
    assert np.all(np.abs(rec - v).reshape(8, 16, 32) <= (2.0 * step)[:, :, None] + 1e-9)


def test_gemm_mxfp4_matches_brute_force():
    rng = np.random.default_rng(7)
    w4, ws = O.weight_codes_mxfp4(rng.integers(-40, 41, (6, 256)),
                                  rng.random((6, 2)).astype(np.float32), 128)
    x4, xs = O.mxfp4_cast(rng.standard_normal((3, 256)) * 50)
    out = O.gemm_mxfp4(w4, ws, x4, xs)
    ref = np.zeros((3, 6))
    for m in range(3):
        for n in range(6):
            for k in range(256):
                ref[m, n] += (float(O.e2m1_value(x4[m, k])) * 2.0 ** (int(xs[m, k // 32]) - 127) *
                              float(O.e2m1_value(w4[n, k])) * 2.0 ** (int(ws[n, k // 32]) - 127))
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-9)
