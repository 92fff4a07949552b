"""Pins of the oracle's RHT, generators and fp16 storage (CPU only).

Each check fixes the oracle against something other than itself: a library
construction of the Hadamard matrix, the algebraic identities of eq. rht,
published known-answer vectors of the two counter-based generators, and
numpy's IEEE binary16 conversion.
"""
import numpy as np
import pytest
import scipy.linalg

from oracle import oracle as O


@pytest.mark.parametrize("n", [2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048])
def test_fwht_is_sylvester_hadamard(n):
    # FWHT of the unit vectors = the columns of H_n (eq. rht); compare with
    # scipy's Sylvester construction H_2n = [[H, H], [H, -H]] and H H^T = n I.
    H = O.fwht(np.eye(n, dtype=np.int64)).T
    assert np.array_equal(H, scipy.linalg.hadamard(n).astype(np.int64))
    Hf = H.astype(np.float64)  # exact: integer entries, |sums| <= n
    assert np.array_equal(Hf @ Hf.T, n * np.eye(n))


@pytest.mark.parametrize("n", [8, 128, 1024])
def test_fwht_exact_on_integers_and_involution(n):
    rng = np.random.default_rng(n)
    v = rng.integers(-1000, 1000, size=(16, n)).astype(np.int64)
    H = scipy.linalg.hadamard(n).astype(np.int64)
    w = O.fwht(v)
    assert np.array_equal(w, (v.astype(np.float64) @ H.T.astype(np.float64)).astype(np.int64))
    assert np.array_equal(O.fwht(w), n * v)
    # fp32 on small integers is exact too: the same values
    vf = v.astype(np.float32)
    assert np.array_equal(O.fwht(vf).astype(np.int64), w)


@pytest.mark.parametrize("n", [128, 1024])
def test_rht_inverse_and_norm(n):
    # RHT(x) = H D x; RHT^-1(y) = D H y / n (H symmetric, H^2 = n I, D^2 = I).
    rng = np.random.default_rng(7)
    x = rng.standard_normal((32, n))
    d = O.signs(123, n).astype(np.float64)
    y = O.fwht(x * d)
    assert np.allclose(np.linalg.norm(y, axis=1), np.sqrt(n) * np.linalg.norm(x, axis=1), rtol=1e-13)
    back = O.fwht(y) * d / n
    err = np.linalg.norm(back - x, axis=1) / np.linalg.norm(x, axis=1)
    assert err.max() < 1e-12
    x32 = x.astype(np.float32)
    y32 = O.fwht(x32 * d.astype(np.float32))
    back32 = O.fwht(y32) * d.astype(np.float32) / np.float32(n)
    err32 = np.linalg.norm(back32 - x32, axis=1) / np.linalg.norm(x32, axis=1)
    assert err32.max() < 1e-6


def test_splitmix64_known_answers():
    # Reference SplitMix64 sequence for seed 0 (Steele et al.; the values
    # every published implementation reproduces).
    assert O.splitmix64(0, 0) == 0xE220A8397B1DCDAF
    assert O.splitmix64(0, 1) == 0x6E789E6AA1B965F4
    assert O.splitmix64(0, 2) == 0x06C45D188009454F


def test_philox4x32_10_known_answers():
    # Known-answer vectors published with Random123 for philox4x32-10.
    assert list(O.philox([0, 0, 0, 0], [0, 0])) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]
    assert list(O.philox([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2)) == [0x408F276D, 0x41C83B0E,
                                                                 0xA20BC7C6, 0x6D5451FD]
    assert list(O.philox([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344],
                         [0xA4093822, 0x299F31D0])) == [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]


def test_rht_signs_are_balanced_and_uncorrelated():
    # eq. rht asks for iid uniform +-1; check the seeded diagonal looks so.
    s = O.signs(2024, 200000).astype(np.float64)
    assert abs(s.mean()) < 4.5 / np.sqrt(s.size)
    assert abs(np.mean(s[1:] * s[:-1])) < 4.5 / np.sqrt(s.size)
    assert not np.array_equal(O.signs(1, 64), O.signs(2, 64))


def test_f16_rounding_matches_ieee():
    rng = np.random.default_rng(3)
    vals = np.concatenate([
        rng.uniform(0, 70000, 3000),
        np.exp(rng.uniform(np.log(1e-8), np.log(6e4), 3000)),
        # exact binary16 midpoints (ties to even) and the overflow edge
        (np.arange(1, 2000) + 0.5) * 2.0**-10,
        (np.arange(1, 200) + 0.5) * 2.0**-24,
        np.array([65504.0, 65519.0, 65520.0, 65536.0, 0.0, 2.0**-25, 2.0**-24]),
    ]).astype(np.float32)
    ours = O.f32_to_f16_bits(vals)
    with np.errstate(over="ignore"):
        ref = vals.astype(np.float16).view(np.uint16)
    assert np.array_equal(ours, ref)
    back = O.f16_bits_to_f32(ref)
    assert np.array_equal(back, ref.view(np.float16).astype(np.float32))
