"""Pins of the oracle's one-token attention over a coded KV cache (CPU only).

decode_attention gathers decoded key and value rows through a block table
and applies a softmax per query head.  Each pin is a case whose answer is
fixed without that formula: one token (the value row itself), a zero query
(the plain mean of hand-listed rows), two tokens (the logistic closed form),
a huge scale (the arg-max row), an empty sequence (zeros), and grouped
heads (same query, same answer; other KV heads' columns untouched).  The
last test pins the identity the fused GPU kernel evaluates: a key's score is
g (S H D q) . (code - U), with the value sum taken in the same rotated
coordinates and transformed back once per head."""
import numpy as np
import pytest

from oracle import oracle as O

LATS = [O.E8, O.D4, O.A2, O.Z]
N = 128


def kv_params(lat, rht_seed, dither_seed):
    # the KV variant: signs rotation, subtractive dither, fp16 norms
    return O.Params(lattice=lat, alpha=O.alpha(lat, 12.0), rht_seed=rht_seed, rotation=1,
                    rot_seed=rht_seed + 1, dither=True, dither_seed=dither_seed, norm_fp16=True)


def coded_cache(lat, rows, hkv, seed):
    rng = np.random.default_rng(seed)
    pk, pv = kv_params(lat, 31, 1001), kv_params(lat, 37, 2002)
    k = rng.standard_normal((rows, hkv * N)).astype(np.float32)
    k[:, 3::N] *= 10  # outlier channels
    v = rng.standard_normal((rows, hkv * N)).astype(np.float32)
    kc, kn, _, _ = O.frontend(pk, k)
    vc, vn, _, _ = O.frontend(pv, v)
    return pk, kc, kn, pv, vc, vn


# 6 blocks of 16 rows; sequence 0 holds 37 tokens in blocks 4, 1, 5,
# sequence 1 one token in block 2, sequence 2 nothing
BT = 16
TABLE = np.array([[4, 1, 5], [2, 0, 0], [3, 3, 3]], dtype=np.int32)
ROWS0 = list(range(64, 80)) + list(range(16, 32)) + list(range(80, 85))
ROWS1 = [32]


@pytest.fixture(scope="module", params=LATS, ids=lambda l: {0: "E8", 1: "D4", 2: "A2", 3: "Z"}[l])
def cache(request):
    lat = request.param
    pk, kc, kn, pv, vc, vn = coded_cache(lat, 96, 4, 500 + lat)
    kd = O.backend(pk, kc, kn).astype(np.float64)
    vd = O.backend(pv, vc, vn).astype(np.float64)
    return dict(pk=pk, kc=kc, kn=kn, pv=pv, vc=vc, vn=vn, kd=kd, vd=vd)


def attend(c, q, lens, scale=1.0):
    return O.decode_attention(c["pk"], c["kc"], c["kn"], c["pv"], c["vc"], c["vn"], q, TABLE,
                              np.asarray(lens), BT, scale)


def test_zero_query_is_the_mean_of_the_listed_rows(cache):
    q = np.zeros((3, 8, N))
    out = attend(cache, q, [37, 1, 0])
    vd = cache["vd"]
    for h in range(8):
        cs = slice((h // 2) * N, (h // 2 + 1) * N)
        np.testing.assert_allclose(out[0, h], vd[ROWS0, cs].mean(axis=0), rtol=0, atol=1e-12)
        assert np.array_equal(out[1, h], vd[ROWS1[0], cs])  # one token: p = 1
    assert np.array_equal(out[2], np.zeros((8, N)))  # empty sequence


def test_two_tokens_logistic(cache):
    rng = np.random.default_rng(3)
    q = rng.standard_normal((3, 8, N))
    out = attend(cache, q, [2, 1, 0], scale=0.05)
    kd, vd = cache["kd"], cache["vd"]
    r0, r1 = ROWS0[0], ROWS0[1]
    for h in range(8):
        cs = slice((h // 2) * N, (h // 2 + 1) * N)
        s0, s1 = 0.05 * (kd[r0, cs] @ q[0, h]), 0.05 * (kd[r1, cs] @ q[0, h])
        w = 1.0 / (1.0 + np.exp(s0 - s1))
        np.testing.assert_allclose(out[0, h], vd[r0, cs] + w * (vd[r1, cs] - vd[r0, cs]),
                                   rtol=0, atol=1e-12)


def test_huge_scale_picks_the_best_key(cache):
    rng = np.random.default_rng(4)
    q = rng.standard_normal((3, 8, N))
    out = attend(cache, q, [37, 1, 0], scale=1e6)
    kd, vd = cache["kd"], cache["vd"]
    for h in range(8):
        cs = slice((h // 2) * N, (h // 2 + 1) * N)
        best = ROWS0[int(np.argmax(kd[ROWS0, cs] @ q[0, h]))]
        np.testing.assert_allclose(out[0, h], vd[best, cs], rtol=0, atol=1e-9)


def test_grouped_heads_share_their_kv_head(cache):
    rng = np.random.default_rng(5)
    q = rng.standard_normal((3, 8, N))
    q[:, 5] = q[:, 4]  # heads 4 and 5 both read KV head 2
    out = attend(cache, q, [37, 1, 0])
    assert np.array_equal(out[:, 4], out[:, 5])
    # changing KV head 3's columns changes heads 6, 7 only
    c2 = dict(cache)
    vc = cache["vc"].copy()
    vc[:, 3 * N:] = 0
    c2["vc"] = vc
    out2 = attend(c2, q, [37, 1, 0])
    assert np.array_equal(out2[:, :6], out[:, :6])
    assert not np.allclose(out2[0, 6:], out[0, 6:])


@pytest.mark.parametrize("lat", LATS)
def test_rotated_domain_identity(lat):
    # a decoded key tile is k^ = g D H S (code - U) (Sec. 4.1, 4.2, 4.4, with H
    # symmetric), so q . k^ = g (S H D q) . (code - U); likewise sum_t p_t v^_t
    # = D H S sum_t p_t g_t (code_t - U_t)
    pk, kc, kn, pv, vc, vn = coded_cache(lat, 8, 4, 900 + lat)
    kd = O.backend(pk, kc, kn).astype(np.float64)
    rng = np.random.default_rng(6)
    q = rng.standard_normal(N)
    m = O.DIM[lat]
    S = O.signs(pk.rot_seed, N).astype(np.float64)
    gk = O.weight_factors(pk, kn, 8, 4 * N).astype(np.float64)
    pts = O.lattice_points(lat, kc)
    for r in range(8):
        for t in range(4):
            D = O.signs(pk.rht_seed, N, start=t * N).astype(np.float64)
            qt = S * O.fwht(D * q)
            u = np.concatenate([O.dither_block(lat, pk.dither_seed, r, t * N + b) for b in range(0, N, m)])
            y = pts[r, t * N:(t + 1) * N] - u
            score = gk[r, t] * (qt @ y)
            ref = kd[r, t * N:(t + 1) * N] @ q
            assert abs(score - ref) <= 1e-5 * (np.abs(kd[r, t * N:(t + 1) * N]) @ np.abs(q))
    # the value side: the transform-back of a weighted sum of rotated tiles
    vd = O.backend(pv, vc, vn).astype(np.float64)
    gv = O.weight_factors(pv, vn, 8, 4 * N).astype(np.float64)
    ptsv = O.lattice_points(lat, vc)
    p = rng.random(8)
    Sv = O.signs(pv.rot_seed, N).astype(np.float64)
    Dv = O.signs(pv.rht_seed, N, start=N).astype(np.float64)
    acc = np.zeros(N)
    for r in range(8):
        u = np.concatenate([O.dither_block(lat, pv.dither_seed, r, N + b) for b in range(0, N, m)])
        acc += p[r] * gv[r, 1] * (ptsv[r, N:2 * N] - u)
    back = Dv * O.fwht(Sv * acc)
    np.testing.assert_allclose(back, p @ vd[:, N:2 * N], rtol=0, atol=1e-5 * np.abs(vd).max())


def test_subset_of_rows_at_their_indices(cache):
    # passing only the rows a sequence reaches, at their stored indices, gives
    # the same answer as passing every row
    rng = np.random.default_rng(8)
    q = rng.standard_normal((3, 8, N))
    full = attend(cache, q, [37, 1, 0])
    keep = np.array(sorted(ROWS0 + ROWS1))
    c = cache
    sub = O.decode_attention(c["pk"], c["kc"][keep], c["kn"][keep], c["pv"], c["vc"][keep],
                             c["vn"][keep], q, TABLE, np.array([37, 1, 0]), BT, 1.0, rows=keep)
    assert np.array_equal(sub, full)


def test_residual_window(cache):
    # the last min(W, len) tokens come exact from the ring slots t % W
    rng = np.random.default_rng(9)
    W = 8
    wk = rng.standard_normal((3, W, 4 * N))
    wv = rng.standard_normal((3, W, 4 * N))
    c = cache

    def att(q, lens, scale=1.0):
        return O.decode_attention(c["pk"], c["kc"], c["kn"], c["pv"], c["vc"], c["vn"], q, TABLE,
                                  np.asarray(lens), BT, scale, window=W, window_k=wk, window_v=wv)

    q = np.zeros((3, 8, N))
    out = att(q, [37, 1, 0])
    vd = c["vd"]
    for h in range(8):
        cs = slice((h // 2) * N, (h // 2 + 1) * N)
        # tokens 0..28 coded (rows listed by hand), 29..36 exact in slots 5, 6, 7, 0, 1, 2, 3, 4
        rows = ROWS0[:29]
        allv = np.concatenate([vd[rows, cs], wv[0, [5, 6, 7, 0, 1, 2, 3, 4], cs]])
        np.testing.assert_allclose(out[0, h], allv.mean(axis=0), rtol=0, atol=1e-12)
        # one token, exact: slot 0 of sequence 1
        assert np.array_equal(out[1, h], wv[1, 0, cs])
    assert np.array_equal(out[2], np.zeros((8, N)))
    # a huge scale picks the best key, coded or exact
    q = rng.standard_normal((3, 8, N))
    out = att(q, [37, 1, 0], scale=1e6)
    kd = c["kd"]
    for h in range(8):
        cs = slice((h // 2) * N, (h // 2 + 1) * N)
        keys = np.concatenate([kd[ROWS0[:29], cs], wk[0, [5, 6, 7, 0, 1, 2, 3, 4], cs]])
        vals = np.concatenate([vd[ROWS0[:29], cs], wv[0, [5, 6, 7, 0, 1, 2, 3, 4], cs]])
        np.testing.assert_allclose(out[0, h], vals[int(np.argmax(keys @ q[0, h]))], rtol=0, atol=1e-9)
    # W = 0 is the plain coded cache
    q = rng.standard_normal((3, 8, N))
    plain = attend(c, q, [37, 1, 0])
    zero = O.decode_attention(c["pk"], c["kc"], c["kn"], c["pv"], c["vc"], c["vn"], q, TABLE,
                              np.array([37, 1, 0]), BT, 1.0, window=0)
    assert np.array_equal(plain, zero)
