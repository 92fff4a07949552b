"""numpy front door to the CPU oracle (test infrastructure only).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import this module.  It loads oracle/libhqoracle.so (built from hq_oracle.c by
oracle/build.py) and never touches the HIP library.  Every function mirrors
one step of the paper's pipeline; see hq_oracle.c for the passages.
"""
import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

from . import build as _build

E8, D4, A2, Z = 0, 1, 2, 3
LATTICES = {"E8": E8, "D4": D4, "A2": A2, "Z": Z}
DIM = {E8: 8, D4: 4, A2: 2, Z: 1}

OK, ERR_ARG, ERR_CAPACITY, ERR_OVERFLOW, ERR_CORRUPT = 0, -1, -3, -4, -6

_lib = None


class _Params(C.Structure):
    _fields_ = [
        ("tile", C.c_int32),
        ("lattice", C.c_int32),
        ("substream", C.c_int32),
        ("rice_k", C.c_int32),
        ("alpha", C.c_float),
        ("norm_fp16", C.c_int32),
        ("rht_seed", C.c_uint64),
        ("rotation", C.c_int32),
        ("dither", C.c_int32),
        ("rot_seed", C.c_uint64),
        ("dither_seed", C.c_uint64),
        ("qjl", C.c_void_p),
    ]


def lib():
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
            _build.build(force=True)
        L = C.CDLL(path)
        p = C.c_void_p
        i64 = C.c_int64
        L.hqo_alpha.restype = C.c_float
        L.hqo_alpha.argtypes = [C.c_int, C.c_double]
        L.hqo_alpha64.restype = C.c_double
        L.hqo_alpha64.argtypes = [C.c_int, C.c_double]
        L.hqo_nsm.restype = C.c_double
        L.hqo_nsm.argtypes = [C.c_int]
        L.hqo_covolume.restype = C.c_double
        L.hqo_covolume.argtypes = [C.c_int]
        L.hqo_splitmix64.restype = C.c_uint64
        L.hqo_splitmix64.argtypes = [C.c_uint64, C.c_uint64]
        L.hqo_sign.restype = C.c_int
        L.hqo_sign.argtypes = [C.c_uint64, i64]
        L.hqo_philox4x32_10.argtypes = [p, p, p]
        L.hqo_fwht_f32.argtypes = [p, C.c_int]
        L.hqo_fwht_f64.argtypes = [p, C.c_int]
        L.hqo_fwht_i64.argtypes = [p, C.c_int]
        L.hqo_f32_to_f16.restype = C.c_uint16
        L.hqo_f32_to_f16.argtypes = [C.c_float]
        L.hqo_f16_to_f32.restype = C.c_float
        L.hqo_f16_to_f32.argtypes = [C.c_uint16]
        L.hqo_quantize.argtypes = [C.c_int, p, i64, p]
        L.hqo_margins.argtypes = [C.c_int, p, p, i64, p]
        L.hqo_strip.argtypes = [C.c_int, p, i64, p]
        L.hqo_unstrip.argtypes = [C.c_int, p, i64, p]
        L.hqo_zigzag.restype = C.c_uint32
        L.hqo_zigzag.argtypes = [C.c_int32]
        L.hqo_unzigzag.restype = C.c_int32
        L.hqo_unzigzag.argtypes = [C.c_uint32]
        L.hqo_rice_kstar.restype = C.c_int
        L.hqo_rice_kstar.argtypes = [C.c_double]
        L.hqo_rice_k_auto.restype = C.c_int
        L.hqo_rice_k_auto.argtypes = [i64, i64]
        L.hqo_rice_length.restype = i64
        L.hqo_rice_length.argtypes = [C.c_uint32, C.c_int]
        L.hqo_rice_put_substream.restype = i64
        L.hqo_rice_put_substream.argtypes = [p, p, C.c_int, p, p]
        L.hqo_rice_get_substream.restype = i64
        L.hqo_rice_get_substream.argtypes = [p, p, i64, C.c_int, p, p]
        L.hqo_dither_block.argtypes = [C.c_int, C.c_uint64, i64, i64, p]
        L.hqo_frontend.restype = C.c_int
        L.hqo_frontend.argtypes = [p, p, i64, i64, i64, i64, p, p, p]
        L.hqo_pack.restype = C.c_int
        L.hqo_pack.argtypes = [p, p, i64, i64, i64, p, i64, i64, p, p, p]
        L.hqo_unpack.restype = C.c_int
        L.hqo_unpack.argtypes = [p, p, p, p, i64, i64, i64, p]
        L.hqo_backend.restype = C.c_int
        L.hqo_backend.argtypes = [p, p, p, i64, i64, i64, p]
        L.hqo_encode.restype = C.c_int
        L.hqo_encode.argtypes = [p, p, i64, i64, i64, i64, p, i64, i64, p, p, p, p]
        L.hqo_decode.restype = C.c_int
        L.hqo_decode.argtypes = [p, p, p, p, p, i64, i64, i64, p]
        L.hqo_weight_factors.argtypes = [p, p, i64, i64, p]
        L.hqo_act_prep.argtypes = [p, i64, i64, C.c_int, C.c_uint64, p, p]
        L.hqo_gemm_blockscaled.argtypes = [p, p, p, p, i64, i64, i64, C.c_int, p]
        _lib = L
    return _lib


def _ptr(a):
    return a.ctypes.data_as(C.c_void_p) if a is not None else None


@dataclass
class Params:
    """Codec parameters, the knobs of the paper's parameter table (Sec. 4.9)."""
    tile: int = 128
    lattice: int = E8
    alpha: float = 1.0
    substream: int = 512
    rice_k: int = -1
    norm_fp16: bool = False
    rht_seed: int = 0
    rotation: int = 0
    dither: bool = False
    rot_seed: int = 0
    dither_seed: int = 0
    qjl: object = None  # rotation 2: the tile x tile orthogonal S (Sec. 4.2), float32

    def c(self):
        if self.qjl is not None:
            self._qjl32 = np.ascontiguousarray(self.qjl, dtype=np.float32)  # kept alive with self
            assert self._qjl32.shape == (self.tile, self.tile)
        q = self._qjl32.ctypes.data_as(C.c_void_p) if self.qjl is not None else None
        return _Params(self.tile, self.lattice, self.substream, self.rice_k, np.float32(self.alpha),
                       int(self.norm_fp16), self.rht_seed & (2**64 - 1), self.rotation,
                       int(self.dither), self.rot_seed & (2**64 - 1), self.dither_seed & (2**64 - 1), q)


# ---------------------------------------------------------------- constants

def nsm(lat):
    return lib().hqo_nsm(lat)


def covolume(lat):
    return lib().hqo_covolume(lat)


def alpha(lat, snr_db):
    """fp32 alpha of App. B eq. alpha-calib."""
    return np.float32(lib().hqo_alpha(lat, float(snr_db)))


def alpha64(lat, snr_db):
    return lib().hqo_alpha64(lat, float(snr_db))


def sigma2_vor(lat):
    """Per-coordinate Voronoi second moment G * V^(2/m) of the realization."""
    return nsm(lat) * covolume(lat) ** (2.0 / DIM[lat])


# ---------------------------------------------------------------- generators

def splitmix64(seed, j):
    return lib().hqo_splitmix64(seed & (2**64 - 1), j)


def signs(seed, n, start=0):
    L = lib()
    return np.array([L.hqo_sign(seed & (2**64 - 1), start + j) for j in range(n)], dtype=np.int8)


def philox(ctr, key):
    c = np.asarray(ctr, dtype=np.uint32)
    k = np.asarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().hqo_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def dither_block(lat, seed, row, col0):
    u = np.zeros(8, dtype=np.float32)
    lib().hqo_dither_block(lat, seed & (2**64 - 1), row, col0, _ptr(u))
    return u[:DIM[lat]].copy()


# ---------------------------------------------------------------- transforms

def fwht(v):
    """Unnormalized Sylvester FWHT of the last axis (stages h = 1 .. n/2)."""
    v = np.array(v, copy=True)
    n = v.shape[-1]
    flat = v.reshape(-1, n)
    fn = {np.dtype(np.float32): lib().hqo_fwht_f32, np.dtype(np.float64): lib().hqo_fwht_f64,
          np.dtype(np.int64): lib().hqo_fwht_i64}[flat.dtype]
    flat = np.ascontiguousarray(flat)
    for r in range(flat.shape[0]):
        row = flat[r]
        fn(row.ctypes.data_as(C.c_void_p), n)
    return flat.reshape(v.shape)


def f32_to_f16_bits(x):
    L = lib()
    return np.array([L.hqo_f32_to_f16(float(v)) for v in np.ravel(x)], dtype=np.uint16)


def f16_bits_to_f32(h):
    L = lib()
    return np.array([L.hqo_f16_to_f32(int(v)) for v in np.ravel(h)], dtype=np.float32)


# ---------------------------------------------------------------- lattices

def quantize(lat, z):
    z = np.ascontiguousarray(z, dtype=np.float32)
    m = DIM[lat]
    assert z.size % m == 0
    c = np.zeros(z.shape, dtype=np.int32)
    lib().hqo_quantize(lat, _ptr(z), z.size // m, _ptr(c))
    return c


def margins(lat, z, c):
    z = np.ascontiguousarray(z, dtype=np.float32)
    c = np.ascontiguousarray(c, dtype=np.int32)
    m = DIM[lat]
    out = np.zeros(z.size // m, dtype=np.float64)
    lib().hqo_margins(lat, _ptr(z), _ptr(c), z.size // m, _ptr(out))
    return out


def lattice_points(lat, c):
    """Integer codes -> points of R^m (fp64)."""
    p = np.asarray(c, dtype=np.float64).copy()
    if lat == A2:
        p[..., 0::2] *= np.sqrt(3.0)
    return p


def strip(lat, c):
    c = np.ascontiguousarray(c, dtype=np.int32)
    s = np.zeros(c.shape, dtype=np.uint32)
    lib().hqo_strip(lat, _ptr(c), c.size // DIM[lat], _ptr(s))
    return s


def unstrip(lat, s):
    s = np.ascontiguousarray(s, dtype=np.uint32)
    c = np.zeros(s.shape, dtype=np.int32)
    lib().hqo_unstrip(lat, _ptr(s), s.size // DIM[lat], _ptr(c))
    return c


def zigzag(v):
    return lib().hqo_zigzag(int(v))


def unzigzag(m):
    return lib().hqo_unzigzag(int(m))


# ---------------------------------------------------------------- Rice

def rice_kstar(p):
    return lib().hqo_rice_kstar(float(p))


def rice_k_auto(count, total):
    return lib().hqo_rice_k_auto(int(count), int(total))


def rice_length(m, k):
    return lib().hqo_rice_length(int(m), int(k))


def rice_put(params: Params, sym, k0, k1=None):
    sym = np.ascontiguousarray(sym, dtype=np.uint32)
    k = np.array([k0, k0 if k1 is None else k1], dtype=np.int32)
    words = np.zeros(int(sym.size * (2 + 32)) + 64, dtype=np.uint32)
    P = params.c()
    nbits = lib().hqo_rice_put_substream(C.byref(P), _ptr(sym), sym.size, _ptr(k), _ptr(words))
    return words[: (nbits + 31) // 32].copy(), nbits


def rice_get(params: Params, words, S, k0, k1=None):
    words = np.ascontiguousarray(words, dtype=np.uint32)
    k = np.array([k0, k0 if k1 is None else k1], dtype=np.int32)
    sym = np.zeros(S, dtype=np.uint32)
    P = params.c()
    used = lib().hqo_rice_get_substream(C.byref(P), _ptr(words), words.size, S, _ptr(k), _ptr(sym))
    return sym, used


# ---------------------------------------------------------------- codec

@dataclass
class Stream:
    """A whole encoded tensor: payload words, sub-stream word offsets, k bytes, norms."""
    payload: np.ndarray
    offsets: np.ndarray
    kparam: np.ndarray
    norms: np.ndarray
    rows: int
    cols: int
    payload_bits: int

    @property
    def end(self):
        return int(self.offsets[-1])


def capacity_words(params: Params, rows, cols):
    """A generous capacity for the oracle (it grows nothing on the fly)."""
    return int(rows * cols * 2 + 64)


def frontend(params: Params, x, row0=0, want_z=False):
    x = np.ascontiguousarray(x, dtype=np.float32)
    rows, cols = x.shape
    codes = np.zeros((rows, cols), dtype=np.int32)
    tpr = cols // params.tile
    norms = np.zeros((rows, tpr), dtype=np.uint16 if params.norm_fp16 else np.float32)
    zin = np.zeros((rows, cols), dtype=np.float32) if want_z else None
    P = params.c()
    rc = lib().hqo_frontend(C.byref(P), _ptr(x), rows, cols, cols, row0, _ptr(codes), _ptr(norms),
                            _ptr(zin))
    if rc not in (OK, ERR_OVERFLOW):
        raise ValueError(f"hqo_frontend failed: {rc}")
    return codes, norms, zin, rc


def pack(params: Params, codes, row0=0, word0=0, payload=None, offsets=None, kparam=None,
         total_rows=None):
    codes = np.ascontiguousarray(codes, dtype=np.int32)
    rows, cols = codes.shape
    total_rows = total_rows or (row0 + rows)
    spr = cols // params.substream
    if payload is None:
        payload = np.zeros(capacity_words(params, total_rows, cols), dtype=np.uint32)
    if offsets is None:
        offsets = np.zeros(total_rows * spr + 1, dtype=np.uint32)
    if kparam is None:
        kparam = np.zeros(total_rows * spr, dtype=np.uint8)
    bits = C.c_int64(0)
    P = params.c()
    rc = lib().hqo_pack(C.byref(P), _ptr(codes), rows, cols, row0, _ptr(payload), payload.size,
                        word0, _ptr(offsets), _ptr(kparam), C.byref(bits))
    if rc != OK:
        raise ValueError(f"hqo_pack failed: {rc}")
    return payload, offsets, kparam, bits.value


def unpack(params: Params, payload, offsets, kparam, rows, cols, row0=0):
    codes = np.zeros((rows, cols), dtype=np.int32)
    P = params.c()
    rc = lib().hqo_unpack(C.byref(P), _ptr(np.ascontiguousarray(payload, dtype=np.uint32)),
                          _ptr(np.ascontiguousarray(offsets, dtype=np.uint32)),
                          _ptr(np.ascontiguousarray(kparam, dtype=np.uint8)), rows, cols, row0,
                          _ptr(codes))
    return codes, rc


def backend(params: Params, codes, norms, row0=0):
    codes = np.ascontiguousarray(codes, dtype=np.int32)
    rows, cols = codes.shape
    y = np.zeros((rows, cols), dtype=np.float32)
    norms = np.ascontiguousarray(norms)
    P = params.c()
    rc = lib().hqo_backend(C.byref(P), _ptr(codes), _ptr(norms), rows, cols, row0, _ptr(y))
    if rc != OK:
        raise ValueError(f"hqo_backend failed: {rc}")
    return y


def encode(params: Params, x, row0=0, want_codes=False, want_z=False):
    """Front end + pack of a whole rows x cols matrix into a fresh stream."""
    codes, norms, zin, rc = frontend(params, x, row0=row0, want_z=want_z)
    payload, offsets, kparam, bits = pack(params, codes, row0=row0)
    end = int(offsets[-1])
    st = Stream(payload[:end].copy(), offsets, kparam, norms, x.shape[0], x.shape[1], bits)
    if want_codes or want_z:
        return st, codes, zin
    return st


def decode(params: Params, st: Stream):
    codes, rc = unpack(params, st.payload, st.offsets, st.kparam, st.rows, st.cols)
    if rc != OK:
        raise ValueError(f"hqo_unpack failed: {rc}")
    return backend(params, codes, st.norms)


def decode_gemv(params: Params, codes, norms, x, row0=0):
    """The decode fused with a matrix-vector product (the fused decode-GEMV of
    Sec. 6.6): y = W^ x for one token, W^ the decoded rows exactly as the
    decode defines them (backend), the products summed in fp64."""
    w = backend(params, codes, norms, row0=row0).astype(np.float64)
    return w @ np.asarray(x, dtype=np.float64)


def decode_attention(pk: Params, k_codes, k_norms, pv: Params, v_codes, v_norms, q,
                     block_table, seq_lens, block_tokens, scale, rows=None, window=0,
                     window_k=None, window_v=None):
    """One-token attention over a coded KV cache (the KV path of Sec. 5.2 and
    the decode of Sec. 5.3 feeding attention, as the end-to-end runs of Sec.
    6.6 use it): the cached keys and values are the decoded rows exactly as
    the decode defines them (backend), gathered per sequence through a block
    table, and each query head attends with a softmax in fp64.
      k_codes, v_codes  all stored rows' lattice codes, [rows, H_kv * tile].
      q                 [batch, H_q, tile]; query head h reads KV head
                        h // (H_q / H_kv).
      block_table       [batch, max_blocks]: token t of sequence b is stored
                        row block_table[b, t // block_tokens] * block_tokens
                        + t % block_tokens.
      seq_lens          [batch] token counts; an empty sequence gives zeros.
      rows              optional stored-row index of each given code row
                        (default 0, 1, ...): lets a caller pass only the rows
                        the table reaches; each is decoded at its own index
                        (the dither depends on it).
      window            residual window W (the most recent tokens kept exact,
                        as in the KV comparison of Sec. 6.7.2, where W = 32
                        costs about 0.1 bps): the last min(W, seq_len)
                        tokens of a sequence are read from window_k /
                        window_v [batch, W, H_kv * tile] at slot t % W, the
                        rest from the coded rows.
    Returns [batch, H_q, tile] fp64."""
    if rows is None:
        kd = backend(pk, k_codes, k_norms).astype(np.float64)
        vd = backend(pv, v_codes, v_norms).astype(np.float64)
        local = None
    else:
        rows = np.asarray(rows, dtype=np.int64)
        kd = np.zeros(k_codes.shape)
        vd = np.zeros(v_codes.shape)
        cut = np.flatnonzero(np.diff(rows) != 1) + 1  # runs of consecutive stored rows
        for a, b in zip(np.r_[0, cut], np.r_[cut, rows.size]):
            kd[a:b] = backend(pk, k_codes[a:b], k_norms[a:b], row0=int(rows[a]))
            vd[a:b] = backend(pv, v_codes[a:b], v_norms[a:b], row0=int(rows[a]))
        order = np.argsort(rows)
        local = (rows[order], order)
    q = np.asarray(q, dtype=np.float64)
    B, Hq, n = q.shape
    G = Hq // (kd.shape[1] // n)
    out = np.zeros((B, Hq, n))
    for b in range(B):
        T = int(seq_lens[b])
        if T == 0:
            continue
        w = min(window, T)
        tw = np.arange(T - w, T)  # exact tokens, ring slots tw % window
        T -= w
        t = np.arange(T)
        r = np.asarray(block_table[b])[t // block_tokens].astype(np.int64) * block_tokens + t % block_tokens
        if local is not None:
            i = np.searchsorted(local[0], r)
            assert np.array_equal(local[0][i], r), "a row the table reaches was not given"
            r = local[1][i]
        for h in range(Hq):
            cs = slice((h // G) * n, (h // G + 1) * n)
            keys, vals = kd[r, cs], vd[r, cs]
            if w:
                keys = np.concatenate([keys, np.asarray(window_k, np.float64)[b, tw % window, cs]])
                vals = np.concatenate([vals, np.asarray(window_v, np.float64)[b, tw % window, cs]])
            s = (keys @ q[b, h]) * scale
            p = np.exp(s - s.max())
            out[b, h] = (p / p.sum()) @ vals
    return out


def weight_factors(params: Params, norms, rows, cols):
    g = np.zeros((rows, cols // params.tile), dtype=np.float32)
    P = params.c()
    lib().hqo_weight_factors(C.byref(P), _ptr(np.ascontiguousarray(norms)), rows, cols, _ptr(g))
    return g


def act_prep(a, tile, rht_seed):
    a = np.ascontiguousarray(a, dtype=np.float32)
    M, K = a.shape
    xq = np.zeros((M, K), dtype=np.int8)
    sx = np.zeros(M, dtype=np.float32)
    lib().hqo_act_prep(_ptr(a), M, K, tile, rht_seed & (2**64 - 1), _ptr(xq), _ptr(sx))
    return xq, sx


def gemm_blockscaled(codes, g, xq, sx, tile):
    codes = np.ascontiguousarray(codes, dtype=np.int32)
    N, K = codes.shape
    M = xq.shape[0]
    out = np.zeros((M, N), dtype=np.float64)
    lib().hqo_gemm_blockscaled(_ptr(codes), _ptr(np.ascontiguousarray(g, dtype=np.float32)),
                               _ptr(np.ascontiguousarray(xq, dtype=np.int8)),
                               _ptr(np.ascontiguousarray(sx, dtype=np.float32)), M, N, K, tile,
                               _ptr(out))
    return out


# ---------------------------------------------------------------- fp8 cast (Sec. 4.8)
# OCP FP8 E4M3: sign, 4 exponent bits (bias 7), 3 fraction bits; exponent 0
# is subnormal (m / 8) 2^-6; code 0x7F / 0xFF is NaN and there is no infinity,
# so the largest finite magnitude is (1 + 6/8) 2^8 = 448.

def _e4m3_magnitudes():
    """The 127 finite non-negative E4M3 values, in code order 0x00 .. 0x7E."""
    v = []
    for code in range(0x7F):
        e, m = code >> 3, code & 7
        v.append((m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7))
    return np.array(v)


def e4m3_bits(x):
    """Round each value to the nearest E4M3 value, ties to the even code (even
    fraction), magnitudes above 448 saturating to 448, the sign kept (a
    negative value that rounds to zero gives -0, 0x80); returns the bytes."""
    x = np.asarray(x, dtype=np.float64)
    mag = _e4m3_magnitudes()
    a = np.minimum(np.abs(x), mag[-1])
    hi = np.clip(np.searchsorted(mag, a), 0, mag.size - 1)  # first value >= a
    lo = np.maximum(hi - 1, 0)
    dlo, dhi = a - mag[lo], mag[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo).astype(np.uint8)
    return (code | np.where(np.signbit(x), 0x80, 0).astype(np.uint8)).astype(np.uint8)


def e4m3_value(bits):
    bits = np.asarray(bits, dtype=np.uint8)
    v = _e4m3_magnitudes()[np.minimum(bits & 0x7F, 0x7E)]
    return np.where(bits & 0x80, -v, v)


def weight_codes_fp8(codes):
    """The fp8 cast of the weight side: E4M3 of each lattice code."""
    return e4m3_bits(np.asarray(codes, dtype=np.float64))


def act_prep_fp8(a, tile, rht_seed):
    """Activation side in fp8: per K-tile y = H D a (fp32, the weights' signs),
    then per token x = E4M3(y * (448 / amax)) and s_x = amax / 448, all in
    fp32 as written."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    M, K = a.shape
    y = (a * signs(rht_seed, K).astype(np.float32)).reshape(M, K // tile, tile)
    y = fwht(y.astype(np.float32)).reshape(M, K)
    amax = np.abs(y).max(axis=1).astype(np.float32)
    inv = np.where(amax == 0, np.float32(0), np.float32(448.0) / np.where(amax == 0, 1, amax))
    xq = e4m3_bits((y * inv[:, None].astype(np.float32)).astype(np.float32))
    return xq, (amax / np.float32(448.0)).astype(np.float32)


def gemm_fp8_blockscaled(w8, g, x8, sx, tile):
    """out[m, n] = s_x[m] sum_t g[n, t] sum_{k in t} x[m, k] w[n, k] over the
    E4M3 values, in fp64."""
    w = e4m3_value(w8)
    x = e4m3_value(x8)
    N, K = w.shape
    T = K // tile
    out = np.zeros((x.shape[0], N))
    for t in range(T):
        ks = slice(t * tile, (t + 1) * tile)
        out += (x[:, ks] @ w[:, ks].T) * np.asarray(g, np.float64)[:, t][None, :]
    return out * np.asarray(sx, np.float64)[:, None]


# ---------------------------------------------------------------- MXFP4 cast (Sec. 4.8, 6.4)
# OCP Microscaling MXFP4: blocks of 32 consecutive values (along K) share one
# E8M0 scale 2^X, stored as the byte X + 127; each element is FP4 E2M1 --
# sign, 2 exponent bits (bias 1), 1 fraction bit -- with magnitudes 0, 0.5,
# 1, 1.5, 2, 3, 4, 6 (codes 0 .. 7; exponent 0 is the subnormal 0.5).  The
# MX conversion takes X = floor(log2(amax)) - 2 (2: E2M1's largest exponent)
# and each element E2M1(v / 2^X), nearest value with ties to the even code,
# magnitudes above 6 saturating to 6.  An all-zero block takes X = -127.

MX_BLOCK = 32
_E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def e2m1_bits(x):
    """Nearest E2M1 value of each x (ties to the even code, saturation at 6,
    sign kept: a negative value that rounds to zero gives -0, code 8)."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), 6.0)
    hi = np.clip(np.searchsorted(_E2M1, a), 0, 7)
    lo = np.maximum(hi - 1, 0)
    dlo, dhi = a - _E2M1[lo], _E2M1[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo).astype(np.uint8)
    return (code | np.where(np.signbit(x), 8, 0).astype(np.uint8)).astype(np.uint8)


def e2m1_value(bits):
    bits = np.asarray(bits, dtype=np.uint8)
    v = _E2M1[bits & 7]
    return np.where(bits & 8, -v, v)


def mx_scale_exponent(amax):
    """X = floor(log2(amax)) - 2 per block (exact, from the binary exponent),
    clamped to E8M0's range [-127, 127]; -127 for an all-zero block."""
    amax = np.asarray(amax, dtype=np.float64)
    _, e = np.frexp(amax)  # amax = m 2^e, m in [0.5, 1)
    x = np.where(amax > 0, e - 1 - 2, -127)
    return np.clip(x, -127, 127).astype(np.int32)


def mxfp4_cast(v):
    """MXFP4 of a [rows, K] array along K: E2M1 codes (one per byte, low
    nibble) and the blocks' E8M0 scale bytes [rows, K / 32]."""
    v = np.asarray(v, dtype=np.float64)
    rows, K = v.shape
    b = v.reshape(rows, K // MX_BLOCK, MX_BLOCK)
    X = mx_scale_exponent(np.abs(b).max(axis=2))
    codes = e2m1_bits(b / np.ldexp(1.0, X)[:, :, None]).reshape(rows, K)
    return codes, (X + 127).astype(np.uint8)


def mxfp4_value(codes, scales):
    """The values an MXFP4 array stands for: E2M1 value times 2^X per block."""
    c = e2m1_value(codes)
    rows, K = c.shape
    X = np.asarray(scales, dtype=np.int32) - 127
    return (c.reshape(rows, K // MX_BLOCK, MX_BLOCK) * np.ldexp(1.0, X)[:, :, None]).reshape(rows, K)


def weight_codes_mxfp4(codes, g, tile):
    """The MXFP4 cast of the weight side (Sec. 4.8 Cast: the reconstruction
    is what is cast at the matmul boundary).  In the rotated coordinates the
    reconstruction of coordinate k of row n is g[n, t] c[n, k], t the tile of
    k: one fp32 product per coordinate, then the MX cast 32 along K per
    block.  A block lies inside one tile, so its E8M0 scale carries the tile
    factor's binade and its elements the rest."""
    c = np.asarray(codes).astype(np.float32)
    gk = np.repeat(np.asarray(g, dtype=np.float32), tile, axis=1)
    return mxfp4_cast((c * gk).astype(np.float64))


def act_prep_mxfp4(a, tile, rht_seed):
    """Activation side in MXFP4: per K-tile y = H D a (fp32, the weights'
    signs), then the MX cast of y per 32 values; the block scales carry the
    magnitude, so there is no per-token factor."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    M, K = a.shape
    y = (a * signs(rht_seed, K).astype(np.float32)).reshape(M, K // tile, tile)
    y = fwht(y.astype(np.float32)).reshape(M, K)
    return mxfp4_cast(y)


def gemm_mxfp4(w4, ws, x4, xs):
    """out[m, n] = sum_k X[m, k] W[n, k] over the MXFP4 values (element times
    block scale), in fp64: the block scales carry every factor."""
    return mxfp4_value(x4, xs) @ mxfp4_value(w4, ws).T


