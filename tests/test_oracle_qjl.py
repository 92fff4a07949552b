"""Pins of the oracle's qjl rotation (Sec. 4.2: encode applies a Haar
orthogonal S, decode its transpose), CPU only.  S is an input, the Haar draw
made by the caller (here: QR of a seeded Gaussian matrix with the sign fix
that makes the distribution Haar).  Pins: S = I reproduces the plain codec
and S = diag(signs) the signs rotation, bit for bit; a Haar S keeps the
realized SNR at the operating point (a transposed S on decode would not) and
stays lossless through pack and unpack."""
import numpy as np
import pytest

from oracle import oracle as O

LATS = [O.E8, O.D4, O.A2, O.Z]
N = 128


def haar(seed, n=N):
    g = np.random.default_rng(seed).standard_normal((n, n))
    q, r = np.linalg.qr(g)
    return (q * np.sign(np.diag(r))).astype(np.float32)


def kv(lat, rotation, qjl=None, dither=True):
    return O.Params(lattice=lat, alpha=O.alpha(lat, 12.0), rht_seed=5, rotation=rotation, rot_seed=6,
                    dither=dither, dither_seed=7, norm_fp16=True, qjl=qjl)


def data(seed=3):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((32, 512)).astype(np.float32)
    x[:, 3::N] *= 10
    return x


@pytest.mark.parametrize("lat", LATS)
@pytest.mark.parametrize("dither", [True, False])
def test_identity_is_the_plain_codec(lat, dither):
    x = data()
    a = O.frontend(kv(lat, 0, dither=dither), x)
    b = O.frontend(kv(lat, 2, np.eye(N, dtype=np.float32), dither=dither), x)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    ya = O.backend(kv(lat, 0, dither=dither), a[0], a[1])
    yb = O.backend(kv(lat, 2, np.eye(N, dtype=np.float32), dither=dither), b[0], b[1])
    assert np.array_equal(ya, yb)


@pytest.mark.parametrize("lat", LATS)
def test_sign_diagonal_is_the_signs_rotation(lat):
    x = data(4)
    S = np.diag(O.signs(6, N).astype(np.float32))
    a = O.frontend(kv(lat, 1), x)
    b = O.frontend(kv(lat, 2, S), x)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert np.array_equal(O.backend(kv(lat, 1), a[0], a[1]), O.backend(kv(lat, 2, S), b[0], b[1]))


@pytest.mark.parametrize("lat", LATS)
def test_haar_rotation_round_trip(lat):
    x = data(5)
    S = haar(11)
    assert np.abs(S.astype(np.float64) @ S.T.astype(np.float64) - np.eye(N)).max() < 1e-5
    P = kv(lat, 2, S)
    st, codes, _ = O.encode(P, x, want_codes=True)
    y = O.decode(P, st)
    snr = 10 * np.log10((x.astype(np.float64) ** 2).sum() / ((y - x).astype(np.float64) ** 2).sum())
    assert abs(snr - 12.0) < 1.0, snr
    # the transpose matters: decoding with S in place of S^T is far off
    Pw = kv(lat, 2, S.T.copy())
    yw = O.backend(Pw, codes, st.norms)
    snrw = 10 * np.log10((x.astype(np.float64) ** 2).sum() / ((yw - x).astype(np.float64) ** 2).sum())
    assert snrw < 3.0, snrw
    # and the codes survive pack / unpack
    back, rc = O.unpack(P, st.payload, st.offsets, st.kparam, st.rows, st.cols)
    assert rc == O.OK and np.array_equal(back, codes)
