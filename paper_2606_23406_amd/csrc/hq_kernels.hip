// HyperQuant codec kernels for gfx950 (MI355X).
//
// Lane layout (encode and decode): one wave64 owns one sub-stream of 512
// scalars = four 128-scalar tiles.  Lane l holds tile l / 16, coordinates
// 8 (l % 16) .. 8 (l % 16) + 7 (one 16-byte bf16 load), i.e. one E8 block,
// two D4 blocks, four A2 blocks or eight Z scalars; the symbol index of its
// j-th value inside the sub-stream is 8 l + j.  The Walsh-Hadamard stages
// h = 1, 2, 4 run in registers, h = 8, 16, 32, 64 across lanes l ^ 1, 2, 4, 8,
// in that order, so every fp32 value equals the reference stage order.
//
// Floating-point contraction is off for this file: each a * b + c that the
// method writes as two roundings stays two roundings; the few fused
// multiply-adds used below are exact (a multiplier of +-2 or an integer sum).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hq_internal.h"

#pragma clang fp contract(off)

namespace {

constexpr float kSqrt3 = 1.7320508075688772f;       // fp32 nearest sqrt(3)
constexpr float kInv2Sqrt3 = 0.28867513459481287f;  // fp32 nearest 1/(2 sqrt(3))
constexpr int kE8 = HQ_E8, kD4 = HQ_D4, kA2 = HQ_A2, kZ = HQ_Z;

// ------------------------------------------------------------------ helpers

__device__ __forceinline__ uint32_t readfirst(uint32_t v) {
  return __builtin_amdgcn_readfirstlane(v);
}

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// Inclusive prefix sum over the 64 lanes.
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t o = __shfl_up(v, d, 64);
    if (lane >= d) v += o;
  }
  return v;
}

__device__ __forceinline__ uint32_t zigzag(int32_t v) {
  return (uint32_t)((v << 1) ^ (v >> 31));
}

__device__ __forceinline__ int32_t unzigzag(uint32_t m) {
  return (int32_t)(m >> 1) ^ -(int32_t)(m & 1u);
}

// Position (0..31) of the r-th set bit (r from 0) of w.
__device__ __forceinline__ uint32_t select32(uint32_t w, uint32_t r) {
  uint32_t pos = 0, c;
  c = __popc(w & 0xFFFFu);
  if (r >= c) { r -= c; w >>= 16; pos += 16; }
  c = __popc(w & 0xFFu);
  if (r >= c) { r -= c; w >>= 8; pos += 8; }
  c = __popc(w & 0xFu);
  if (r >= c) { r -= c; w >>= 4; pos += 4; }
  c = __popc(w & 0x3u);
  if (r >= c) { r -= c; w >>= 2; pos += 2; }
  c = w & 1u;
  if (r >= c) { pos += 1; }
  return pos;
}

__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// IEEE round-to-nearest-even fp32 -> bf16 bits.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// ------------------------------------------------------------- Philox4x32-10
// Salmon, Moraes, Dror, Shaw (SC'11): ten rounds of two 32x32->64 products
// with the Weyl key schedule.
__device__ __forceinline__ void philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                              uint32_t k0, uint32_t k1, uint32_t out[4]) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
    const uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

// ------------------------------------------------------ nearest-point decoders
// Conway & Sloane's closest-point algorithms on the integer realizations:
// 2E8 (two D8 cosets), D4 (round + parity fix), A2 (two rectangular cosets),
// Z (round).  rint is round-half-even; argmax ties take the lowest index.

template <int N>
__device__ __forceinline__ int argmax_abs(const float* e) {
  float best = __builtin_fabsf(e[0]);
  int j = 0;
#pragma unroll
  for (int i = 1; i < N; ++i) {
    const float a = __builtin_fabsf(e[i]);
    const bool gt = a > best;
    best = gt ? a : best;
    j = gt ? i : j;
  }
  return j;
}

__device__ __forceinline__ float tree8(const float* s) {
  return ((s[0] + s[1]) + (s[2] + s[3])) + ((s[4] + s[5]) + (s[6] + s[7]));
}

__device__ __forceinline__ void quant_e8(const float* z, int32_t* c) {
  float ka[8], fb[8], ea[8], eb[8];
  int32_t sa = 0, sb = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float h = z[i] * 0.5f;
    ka[i] = __builtin_rintf(h);
    fb[i] = __builtin_floorf(h);
    ea[i] = __builtin_fmaf(-2.0f, ka[i], z[i]);        // z - 2k, one rounding
    eb[i] = z[i] - __builtin_fmaf(2.0f, fb[i], 1.0f);  // z - (2f + 1)
    sa += (int32_t)ka[i];
    sb += (int32_t)fb[i];
  }
  if (sa & 1) {
    const int j = argmax_abs<8>(ea);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (i == j) {
        ka[i] += (ea[i] >= 0.0f) ? 1.0f : -1.0f;
        ea[i] = __builtin_fmaf(-2.0f, ka[i], z[i]);
      }
  }
  if (sb & 1) {
    const int j = argmax_abs<8>(eb);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (i == j) {
        fb[i] += (eb[i] >= 0.0f) ? 1.0f : -1.0f;
        eb[i] = z[i] - __builtin_fmaf(2.0f, fb[i], 1.0f);
      }
  }
  float sqa[8], sqb[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    sqa[i] = ea[i] * ea[i];
    sqb[i] = eb[i] * eb[i];
  }
  const bool even = tree8(sqa) <= tree8(sqb);
#pragma unroll
  for (int i = 0; i < 8; ++i) c[i] = even ? 2 * (int32_t)ka[i] : 2 * (int32_t)fb[i] + 1;
}

__device__ __forceinline__ void quant_d4(const float* z, int32_t* c) {
  float k[4], e[4];
  int32_t s = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    k[i] = __builtin_rintf(z[i]);
    e[i] = z[i] - k[i];
    c[i] = (int32_t)k[i];
    s += c[i];
  }
  if (s & 1) {
    const int j = argmax_abs<4>(e);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (i == j) c[i] += (e[i] >= 0.0f) ? 1 : -1;
  }
}

__device__ __forceinline__ void quant_a2(const float* z, int32_t* c) {
  const float y = z[0], x = z[1];
  const float a0 = __builtin_rintf(y * kInv2Sqrt3);
  const float b0 = __builtin_rintf(x * 0.5f);
  const float a1 = __builtin_rintf((y - kSqrt3) * kInv2Sqrt3);
  const float b1 = __builtin_rintf((x - 1.0f) * 0.5f);
  const int32_t ny0 = 2 * (int32_t)a0, nx0 = 2 * (int32_t)b0;
  const int32_t ny1 = 2 * (int32_t)a1 + 1, nx1 = 2 * (int32_t)b1 + 1;
  const float ey0 = y - kSqrt3 * (float)ny0, ex0 = x - (float)nx0;
  const float ey1 = y - kSqrt3 * (float)ny1, ex1 = x - (float)nx1;
  const float d0 = ey0 * ey0 + ex0 * ex0;
  const float d1 = ey1 * ey1 + ex1 * ex1;
  const bool first = d0 <= d1;
  c[0] = first ? ny0 : ny1;
  c[1] = first ? nx0 : nx1;
}

template <int LAT>
__device__ __forceinline__ void quantize8(const float* z, int32_t* c) {
  if constexpr (LAT == kE8) {
    quant_e8(z, c);
  } else if constexpr (LAT == kD4) {
    quant_d4(z, c);
    quant_d4(z + 4, c + 4);
  } else if constexpr (LAT == kA2) {
#pragma unroll
    for (int b = 0; b < 4; ++b) quant_a2(z + 2 * b, c + 2 * b);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = (int32_t)__builtin_rintf(z[i]);
  }
}

// Lattice code -> coordinate in R (the A2 y axis carries sqrt(3)).
template <int LAT>
__device__ __forceinline__ float code_coord(int32_t c, int j) {
  if constexpr (LAT == kA2) {
    return (j & 1) ? (float)c : kSqrt3 * (float)c;
  } else {
    return (float)c;
  }
}

// Dither U = b - Q(b) for the lane's 8 coordinates (columns col0 .. col0+7 of
// global row `row`, col0 a multiple of 8): b is a uniform point of a box that
// is a fundamental domain of a sublattice ([-2, 2)^m for 2E8, D4, Z;
// [-sqrt3, sqrt3) x [-1, 1) for A2), drawn from 24 bits of Philox word
// (col mod 4) at counter (col / 4, row_lo, row_hi, 0).
template <int LAT>
__device__ __forceinline__ void dither8(uint64_t seed, int64_t row, int64_t col0, float* u) {
  uint32_t r[8];
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  const uint32_t rl = (uint32_t)(uint64_t)row, rh = (uint32_t)((uint64_t)row >> 32);
  philox4x32_10((uint32_t)((uint64_t)col0 >> 2), rl, rh, 0u, k0, k1, r);
  philox4x32_10((uint32_t)((uint64_t)col0 >> 2) + 1u, rl, rh, 0u, k0, k1, r + 4);
  float b[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float centered = (float)((int32_t)(r[i] >> 8) - 8388608);
    if constexpr (LAT == kA2) {
      b[i] = (i & 1) ? centered * 0x1p-23f : (centered * 0x1p-23f) * kSqrt3;
    } else {
      b[i] = centered * 0x1p-22f;
    }
  }
  int32_t c[8];
  quantize8<LAT>(b, c);
#pragma unroll
  for (int i = 0; i < 8; ++i) u[i] = b[i] - code_coord<LAT>(c[i], i);
}

// --------------------------------------------------------------- strip / unstrip

template <int LAT>
__device__ __forceinline__ void strip8(const int32_t* c, uint32_t* s) {
  if constexpr (LAT == kE8) {
    const int32_t cb = c[0] & 1;
    int32_t h[8], p = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = (c[i] - cb) >> 1;
#pragma unroll
    for (int i = 0; i < 7; ++i) p += h[i];
    p &= 1;
    const int32_t t = (h[7] - p) >> 1;
#pragma unroll
    for (int i = 0; i < 7; ++i) s[i] = zigzag(h[i]);
    s[7] = 2u * zigzag(t) + (uint32_t)cb;
  } else if constexpr (LAT == kD4) {
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int32_t* cc = c + 4 * b;
      const int32_t p = (cc[0] + cc[1] + cc[2]) & 1;
      s[4 * b + 0] = zigzag(cc[0]);
      s[4 * b + 1] = zigzag(cc[1]);
      s[4 * b + 2] = zigzag(cc[2]);
      s[4 * b + 3] = zigzag((cc[3] - p) >> 1);
    }
  } else if constexpr (LAT == kA2) {
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int32_t p = c[2 * b + 1] & 1;
      s[2 * b] = zigzag((c[2 * b] - p) >> 1);
      s[2 * b + 1] = zigzag(c[2 * b + 1]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) s[i] = zigzag(c[i]);
  }
}

template <int LAT>
__device__ __forceinline__ void unstrip8(const uint32_t* s, int32_t* c) {
  if constexpr (LAT == kE8) {
    const int32_t cb = (int32_t)(s[7] & 1u);
    const int32_t t = unzigzag(s[7] >> 1);
    int32_t h[8], p = 0;
#pragma unroll
    for (int i = 0; i < 7; ++i) {
      h[i] = unzigzag(s[i]);
      p += h[i];
    }
    h[7] = 2 * t + (p & 1);
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = 2 * h[i] + cb;
  } else if constexpr (LAT == kD4) {
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      int32_t* cc = c + 4 * b;
      cc[0] = unzigzag(s[4 * b + 0]);
      cc[1] = unzigzag(s[4 * b + 1]);
      cc[2] = unzigzag(s[4 * b + 2]);
      cc[3] = 2 * unzigzag(s[4 * b + 3]) + ((cc[0] + cc[1] + cc[2]) & 1);
    }
  } else if constexpr (LAT == kA2) {
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      c[2 * b + 1] = unzigzag(s[2 * b + 1]);
      c[2 * b] = 2 * unzigzag(s[2 * b]) + (c[2 * b + 1] & 1);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = unzigzag(s[i]);
  }
}

// Rice class of the lane's j-th symbol: D4 codes its halved symbol and A2
// its n_x with a second parameter.
template <int LAT>
__device__ __forceinline__ constexpr int sym_class(int j) {
  return LAT == kD4 ? ((j & 3) == 3) : (LAT == kA2 ? (j & 1) : 0);
}

// Remainder bits of one lane (8 symbols) for parameters k0 (class 0), k1.
template <int LAT>
__device__ __forceinline__ uint32_t lane_rem_bits(uint32_t k0, uint32_t k1) {
  if constexpr (LAT == kD4) return 6 * k0 + 2 * k1;
  if constexpr (LAT == kA2) return 4 * k0 + 4 * k1;
  return 8 * k0;
}

// ----------------------------------------------------------- Walsh-Hadamard

__device__ __forceinline__ void fwht8_inlane(float* v) {
#pragma unroll
  for (int h = 1; h < 8; h <<= 1)
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if ((i & h) == 0) {
        const float a = v[i], b = v[i + h];
        v[i] = a + b;
        v[i + h] = a - b;
      }
}

__device__ __forceinline__ void fwht8_inlane_i(int32_t* v) {
#pragma unroll
  for (int h = 1; h < 8; h <<= 1)
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if ((i & h) == 0) {
        const int32_t a = v[i], b = v[i + h];
        v[i] = a + b;
        v[i + h] = a - b;
      }
}

// Butterfly with lane l ^ M: the lower lane keeps a + b, the upper a - b,
// with a the lower lane's value.
template <int M>
__device__ __forceinline__ void fwht_xlane(float* v, int lane) {
  const bool upper = (lane & M) != 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float p = __shfl_xor(v[j], M, 64);
    v[j] = upper ? (p - v[j]) : (v[j] + p);
  }
}

template <int M>
__device__ __forceinline__ void fwht_xlane_i(int32_t* v, int lane) {
  const bool upper = (lane & M) != 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int32_t p = __shfl_xor(v[j], M, 64);
    v[j] = upper ? (p - v[j]) : (v[j] + p);
  }
}

__device__ __forceinline__ void fwht128(float* v, int lane) {
  fwht8_inlane(v);
  fwht_xlane<1>(v, lane);
  fwht_xlane<2>(v, lane);
  fwht_xlane<4>(v, lane);
  fwht_xlane<8>(v, lane);
}

__device__ __forceinline__ void fwht128_i(int32_t* v, int lane) {
  fwht8_inlane_i(v);
  fwht_xlane_i<1>(v, lane);
  fwht_xlane_i<2>(v, lane);
  fwht_xlane_i<4>(v, lane);
  fwht_xlane_i<8>(v, lane);
}

// The 8 sign bits of columns col0 .. col0 + 7 (col0 a multiple of 8).
__device__ __forceinline__ uint32_t sign_bits8(const uint32_t* mask, int64_t col0) {
  return (mask[col0 >> 5] >> (uint32_t)(col0 & 31)) & 0xFFu;
}

__device__ __forceinline__ float flip(float v, uint32_t bits, int j) {
  return __uint_as_float(__float_as_uint(v) ^ (((bits >> j) & 1u) << 31));
}

// ------------------------------------------------------------ look-back scan
// Decoupled look-back (Merrill & Garland, 2016) over workgroups in ticket
// order.  The scan scratch starts with one 64-bit counter holding
// (epoch << 32 | next ticket); the workgroup that draws the last ticket of a
// launch resets the ticket and advances the epoch, so every launch -- also a
// replayed graph -- gets a fresh epoch without host help.  A status word packs
// the value (32 bits: words since the start of this launch), a flag (2 bits:
// 1 = aggregate, 2 = inclusive prefix) and the epoch (30 bits), so the array
// never needs clearing.  Waits are bounded: a status that never arrives (only
// possible after a corrupted scratch) ends the wait with an error status.

constexpr uint32_t kEpochMask = 0x3FFFFFFFu;
constexpr uint32_t kSpinLimit = 1u << 24;

__device__ __forceinline__ unsigned long long pack_status(uint32_t epoch, uint32_t flag,
                                                          uint32_t value) {
  return ((unsigned long long)(epoch & kEpochMask) << 34) | ((unsigned long long)flag << 32) |
         (unsigned long long)value;
}

__device__ __forceinline__ void store_status(unsigned long long* p, unsigned long long v) {
  __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ unsigned long long load_status(unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------ bit assembly

// OR `nbits` (<= 32) bits of v into the LDS bit array at bit position pos.
__device__ __forceinline__ void or_bits(uint32_t* buf, uint32_t pos, uint32_t v) {
  if (v == 0) return;
  const uint32_t w = pos >> 5, sh = pos & 31;
  atomicOr(&buf[w], v << sh);
  if (sh) {
    const uint32_t hi = v >> (32 - sh);
    if (hi) atomicOr(&buf[w + 1], hi);
  }
}

// ------------------------------------------------------------ encode kernel

template <int LAT, int XT>
__global__ __launch_bounds__(256) void hq_encode_kernel(hq_encode_args A) {
  extern __shared__ uint32_t smem[];
  __shared__ uint32_t s_ticket, s_epoch;
  __shared__ uint32_t s_words[HQ_WAVES_PER_WG];
  __shared__ unsigned long long s_base;
  __shared__ unsigned long long s_bits[2];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (tid == 0) {
    const unsigned long long tk = atomicAdd(A.ticket, 1ull);
    const uint32_t t = (uint32_t)tk, ep = (uint32_t)(tk >> 32);
    // the last ticket of this launch: restart the tickets, advance the epoch
    if (t == A.nwg - 1) atomicExch(A.ticket, (unsigned long long)(ep + 1u) << 32);
    s_ticket = t;
    s_epoch = ep & kEpochMask;
    s_bits[0] = 0;
    s_bits[1] = 0;
  }
  __syncthreads();
  const uint32_t wg = s_ticket, epoch = s_epoch;
  if (wg >= A.nwg) {  // only a corrupted scan scratch hands out such a ticket
    if (tid == 0 && A.stats) atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_INVALID_ARG);
    return;
  }
  const int64_t sub = (int64_t)wg * HQ_WAVES_PER_WG + wave;  // sub-stream within this call
  const bool active = sub < A.nsub;

  const int64_t lrow = active ? sub / A.spr : 0;              // row within x
  const int64_t col0 = (active ? sub % A.spr : 0) * HQ_SUB;   // first column of the sub-stream
  const int tile_in_sub = lane >> 4, q = lane & 15;
  const int64_t col = col0 + tile_in_sub * HQ_TILE + q * 8;   // lane's first column
  const int64_t grow = A.first_row + lrow;

  // ---- load 8 scalars
  float x[8];
  if (active) {
    if constexpr (XT == HQ_BF16) {
      const uint4 raw = *(const uint4*)((const uint16_t*)A.x + lrow * A.ld + col);
      const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[2 * i] = bf16_to_f32(w4[i] & 0xFFFFu);
        x[2 * i + 1] = bf16_to_f32(w4[i] >> 16);
      }
    } else {
      const float4* p = (const float4*)((const float*)A.x + lrow * A.ld + col);
      const float4 a = p[0], b = p[1];
      x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
      x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = 0.0f;
  }

  // ---- Normalize: tile norm as a pairwise tree in index order
  float sq[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) sq[i] = x[i] * x[i];
  float ss = tree8(sq);
  ss = ss + __shfl_xor(ss, 1, 64);
  ss = ss + __shfl_xor(ss, 2, 64);
  ss = ss + __shfl_xor(ss, 4, 64);
  ss = ss + __shfl_xor(ss, 8, 64);
  const float r = __builtin_sqrtf(ss);
  float rs = r;
  bool bad_tile = !(r <= 3.0e38f);  // non-finite input
  if (A.norm_fp16) {
    const _Float16 h = (_Float16)r;
    rs = (float)h;
    bad_tile = bad_tile || !(rs <= 65504.0f);
  }
  const float scale = (rs == 0.0f || bad_tile) ? 0.0f : A.alpha / rs;
  if (active && q == 0) {
    const int64_t t = grow * A.tpr + col / HQ_TILE;
    if (A.norm_fp16) {
      const _Float16 h = (_Float16)r;
      ((_Float16*)A.norms)[t] = h;
    } else {
      ((float*)A.norms)[t] = r;
    }
    if (bad_tile && A.stats) {
      atomicAdd(&A.stats->overflow_tiles, 1u);
      atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_OVERFLOW);
    }
  }

  // ---- RHT: v = H D x
  const uint32_t dbits = sign_bits8(A.dmask, col);
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = flip(x[i], dbits, i);
  fwht128(x, lane);

  // ---- scale, rotate, dither
  const uint32_t sbits = A.rotation ? sign_bits8(A.smask, q * 8) : 0u;
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = flip(x[i] * scale, sbits, i);
  if (A.dither) {
    float u[8];
    dither8<LAT>(A.dither_seed, grow, col, u);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = x[i] + u[i];
  }

  // ---- quantize + strip
  int32_t c[8];
  quantize8<LAT>(x, c);
  bool huge = false;
#pragma unroll
  for (int i = 0; i < 8; ++i) huge = huge || (c[i] > 65536 || c[i] < -65536);
  if (huge || !active) {
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = 0;
  }
  uint32_t sym[8];
  strip8<LAT>(c, sym);

  // ---- Rice parameters (uniform per wave)
  uint32_t sum0 = 0, sum1 = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    if (sym_class<LAT>(j)) sum1 += sym[j]; else sum0 += sym[j];
  }
  uint32_t k0, k1;
  if (A.rice_k >= 0) {
    k0 = (uint32_t)A.rice_k;
    k1 = (LAT == kD4) ? (k0 > 0 ? k0 - 1 : 0) : k0;
  } else {
    sum0 = readfirst(wave_sum_u32(sum0));
    if (LAT == kA2) sum1 = readfirst(wave_sum_u32(sum1));
    uint32_t a0 = 0, a1 = 0;
#pragma unroll
    for (int t = 1; t <= HQ_KMAX; ++t) {
      a0 += sum0 >= A.thr0[t];
      a1 += sum1 >= A.thr1[t];
    }
    // the better of k* and k* + 1 on this sub-stream's symbols
    const uint32_t b0 = a0 < HQ_KMAX ? a0 + 1 : a0;
    const uint32_t b1 = a1 < HQ_KMAX ? a1 + 1 : a1;
    uint32_t la = 0, lb = 0, ma = 0, mb = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (LAT == kD4) {
        const uint32_t ka = sym_class<LAT>(j) ? (a0 > 0 ? a0 - 1 : 0) : a0;
        const uint32_t kb = sym_class<LAT>(j) ? (b0 > 0 ? b0 - 1 : 0) : b0;
        la += (sym[j] >> ka) + ka;
        lb += (sym[j] >> kb) + kb;
      } else if (LAT == kA2 && sym_class<LAT>(j)) {
        ma += (sym[j] >> a1) + a1;
        mb += (sym[j] >> b1) + b1;
      } else {
        la += (sym[j] >> a0) + a0;
        lb += (sym[j] >> b0) + b0;
      }
    }
    la = readfirst(wave_sum_u32(la));
    lb = readfirst(wave_sum_u32(lb));
    k0 = lb < la ? b0 : a0;
    if (LAT == kA2) {
      ma = readfirst(wave_sum_u32(ma));
      mb = readfirst(wave_sum_u32(mb));
      k1 = mb < ma ? b1 : a1;
    } else {
      k1 = (LAT == kD4) ? (k0 > 0 ? k0 - 1 : 0) : k0;
    }
  }

  // ---- code lengths: remainder region then unary region
  uint32_t qv[8], rv[8], ulen = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t kk = sym_class<LAT>(j) ? k1 : k0;
    qv[j] = sym[j] >> kk;
    rv[j] = sym[j] & ((1u << kk) - 1u);
    ulen += qv[j] + 1;
  }
  const uint32_t lrem = lane_rem_bits<LAT>(k0, k1);
  const uint32_t R = 64 * lrem;
  const uint32_t uincl = wave_incl_scan_u32(ulen, lane);
  const uint32_t U = readfirst(__shfl(uincl, 63, 64));
  const uint32_t uoff = uincl - ulen;
  uint32_t W = (R + U + 31) >> 5;
  const bool overflow = active && W > A.lds_words;
  if (!active) W = 0;

  // A sub-stream that does not fit the plan's bound (only non-finite or
  // out-of-range input can do that) is written as all-zero symbols with
  // k = 0: 512 unary terminators, 16 words.
  if (overflow) W = HQ_SUB / 32;
  if (lane == 0) s_words[wave] = W;
  __syncthreads();

  // ---- publish this workgroup's aggregate at once, so successors can pass it
  uint32_t agg = 0;
  for (int w = 0; w < HQ_WAVES_PER_WG; ++w) agg += s_words[w];
  if (tid == 0 && wg > 0) store_status(&A.status[wg], pack_status(epoch, 1u, agg));

  // ---- assemble the sub-stream in LDS (needs no global offset)
  uint32_t* buf = smem + wave * A.lds_words;
  for (uint32_t w = lane; w < W; w += 64) buf[w] = 0u;
  __syncthreads();
  if (active && !overflow) {
    uint32_t pos = lane * lrem;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t kk = sym_class<LAT>(j) ? k1 : k0;
      or_bits(buf, pos, rv[j]);
      pos += kk;
    }
    pos = R + uoff;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      pos += qv[j];
      or_bits(buf, pos, 1u);
      pos += 1;
    }
  } else if (active && overflow) {
    for (uint32_t w = lane; w < W; w += 64) buf[w] = 0xFFFFFFFFu;
  }

  // ---- look-back by wave 0: 64 predecessors per round trip
  if (wave == 0) {
    uint32_t prefix = 0;
    bool timed_out = false;
    int64_t hi = (int64_t)wg - 1;
    while (hi >= 0) {
      const int64_t idx = hi - lane;
      unsigned long long st = 0;
      bool ready = idx < 0;
      uint32_t spins = 0;
      // wait until every predecessor in this window has published something
      for (;;) {
        if (!ready) {
          st = load_status(&A.status[idx]);
          ready = (uint32_t)(st >> 34) == epoch && ((st >> 32) & 3u) != 0u;
        }
        if (__all(ready)) break;
        if (++spins > kSpinLimit) {
          timed_out = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      if (timed_out) break;
      const bool incl = idx >= 0 && ((st >> 32) & 3u) == 2u;
      const unsigned long long pmask = __ballot(incl);
      const int stop = pmask ? __builtin_ctzll(pmask) : 64;  // nearest inclusive prefix
      uint32_t v = (idx >= 0 && lane <= stop) ? (uint32_t)st : 0u;
      v = wave_sum_u32(v);
      prefix += v;
      if (pmask) break;
      hi -= 64;
    }
    if (lane == 0) {
      store_status(&A.status[wg], pack_status(epoch, 2u, prefix + agg));
      if (timed_out && A.stats) atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_HIP);
      const unsigned long long base = A.append ? (unsigned long long)A.offsets[A.first_sub] : 0ull;
      s_base = base + prefix;
    }
  }
  __syncthreads();

  uint32_t before = 0;
  for (int w = 0; w < wave; ++w) before += s_words[w];
  const unsigned long long start = s_base + before;

  // ---- write payload, offsets, k
  if (active) {
    const bool fits = start + W <= (unsigned long long)A.cap_words;
    if (fits) {
      for (uint32_t w = lane; w < W; w += 64) A.payload[start + w] = buf[w];
    }
    if (lane == 0) {
      const int64_t gsub = A.first_sub + sub;
      if (sub == 0 && !A.append) A.offsets[A.first_sub] = 0u;
      A.offsets[gsub + 1] = (uint32_t)(start + W);
      const uint32_t kb = overflow ? 0u : (LAT == kA2 ? (k0 | (k1 << 4)) : k0);
      A.kparam[gsub] = (uint8_t)kb;
      if (A.stats) {
        if (!fits) atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_CAPACITY);
        if (overflow) {
          atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_OVERFLOW);
        }
        const uint32_t bits = overflow ? (uint32_t)HQ_SUB : R + U;
        atomicAdd(&s_bits[0], (unsigned long long)bits);
        atomicAdd(&s_bits[1], (unsigned long long)(W * 32u - bits));
      }
    }
  }
  if (A.stats) {
    __syncthreads();
    if (tid == 0) {
      atomicAdd(&A.stats->payload_bits, s_bits[0]);
      atomicAdd(&A.stats->pad_bits, s_bits[1]);
    }
  }
}

// ------------------------------------------------------------ decode kernel
// Rice decode of one sub-stream per wave: the remainder fields are at fixed
// positions; the unary terminators are located by per-word popcounts, a
// wave prefix sum and a select inside the word that holds terminator 8 l - 1,
// after which lane l walks its own 8 codes.  MODE 0: fp32 out, 1: bf16 out,
// 2: int8 lattice codes and per-tile g (no inverse RHT).

template <int LAT>
__device__ __forceinline__ bool decode_symbols(const hq_decode_args& A, int64_t gsub, int lane,
                                               uint32_t* buf, uint32_t* starts, bool active,
                                               uint32_t* sym) {
  uint32_t start = 0, end = 0, kb = 0;
  if (active) {
    start = A.offsets[gsub];
    end = A.offsets[gsub + 1];
    kb = A.kparam[gsub];
  }
  const uint32_t k0 = (LAT == kA2) ? (kb & 15u) : kb;
  const uint32_t k1 = (LAT == kA2) ? (kb >> 4) : (LAT == kD4 ? (k0 > 0 ? k0 - 1 : 0) : k0);
  const uint32_t W = end - start;
  const uint32_t lrem = lane_rem_bits<LAT>(k0, k1);
  const uint32_t R = 64 * lrem;
  bool ok = active && end >= start && (int64_t)end <= A.cap_words && W <= A.lds_words &&
            k0 <= HQ_KMAX && R <= 32u * W;
  const uint32_t Wl = ok ? W : 0u;
  for (uint32_t w = lane; w < Wl; w += 64) buf[w] = A.payload[start + w];
  starts[lane] = (lane == 0) ? R : 0xFFFFFFFFu;
  __syncthreads();

  // unary terminators: popcount prefix, then the start of each lane's codes
  const uint32_t uw0 = R >> 5;
  const uint32_t nuw = ok ? Wl - uw0 : 0u;
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nuw; base += 64) {
    const uint32_t wi = base + lane;
    const uint32_t v = (wi < nuw) ? buf[uw0 + wi] : 0u;
    const uint32_t cnt = __popc(v);
    const uint32_t incl = wave_incl_scan_u32(cnt, lane);
    const uint32_t P = carry + incl - cnt;
    for (uint32_t t = (P & ~7u) + 7u; t < P + cnt; t += 8u) {
      const uint32_t j = (t + 1u) >> 3;
      if (j < 64u) starts[j] = (uw0 + wi) * 32u + select32(v, t - P) + 1u;
    }
    carry += __shfl(incl, 63, 64);
  }
  __syncthreads();

  // lane's 8 quotients
  uint32_t pos = starts[lane];
  uint32_t qv[8];
  const uint32_t nbits = 32u * Wl;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    uint32_t q = 0;
    if (ok && pos < nbits) {
      uint32_t wi = pos >> 5, b = pos & 31u;
      uint32_t v = buf[wi] >> b;
      while (v == 0u) {
        q += 32u - b;
        b = 0;
        ++wi;
        if (wi >= Wl) break;
        v = buf[wi];
      }
      if (v == 0u) {
        ok = false;
      } else {
        const uint32_t tz = __builtin_ctz(v);
        q += tz;
        pos = wi * 32u + b + tz + 1u;
      }
    } else {
      ok = false;
    }
    qv[j] = q;
  }
  // lane's 8 remainders
  uint32_t rp = lane * lrem;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t kk = sym_class<LAT>(j) ? k1 : k0;
    uint32_t r = 0;
    if (ok && kk) {
      const uint32_t wi = rp >> 5, sh = rp & 31u;
      const unsigned long long lo = buf[wi];
      const unsigned long long hi = (wi + 1 < Wl) ? buf[wi + 1] : 0ull;
      r = (uint32_t)(((hi << 32) | lo) >> sh) & ((1u << kk) - 1u);
    }
    rp += kk;
    sym[j] = (qv[j] << kk) | r;
  }
  if (!ok) {
#pragma unroll
    for (int j = 0; j < 8; ++j) sym[j] = 0;
  }
  return ok;
}

template <int LAT, int MODE>
__global__ __launch_bounds__(256) void hq_decode_kernel(hq_decode_args A) {
  extern __shared__ uint32_t smem[];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t sub = (int64_t)blockIdx.x * HQ_WAVES_PER_WG + wave;
  const bool active = sub < A.nsub;
  const int64_t gsub = A.first_sub + sub;
  uint32_t* buf = smem + wave * (A.lds_words + 64);
  uint32_t* starts = buf + A.lds_words;

  uint32_t sym[8];
  const bool ok = decode_symbols<LAT>(A, gsub, lane, buf, starts, active, sym);
  if (active && !ok && lane == 0 && A.stats) {
    atomicAdd(&A.stats->corrupt_substreams, 1u);
    atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_CORRUPT);
  }
  int32_t c[8];
  unstrip8<LAT>(sym, c);

  const int64_t lrow = active ? sub / A.spr : 0;
  const int64_t col0 = (active ? sub % A.spr : 0) * HQ_SUB;
  const int tile_in_sub = lane >> 4, q = lane & 15;
  const int64_t col = col0 + tile_in_sub * HQ_TILE + q * 8;
  const int64_t grow = A.first_row + lrow;
  const int64_t tix = grow * A.tpr + col / HQ_TILE;
  float rs = 0.0f;
  if (active) rs = A.norm_fp16 ? (float)((const _Float16*)A.norms)[tix] : ((const float*)A.norms)[tix];
  const float g = rs / A.alpha_n;

  if constexpr (MODE == 2) {
    if (!active) return;
    uint32_t packed[2] = {0u, 0u};
    uint32_t clamps = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      int32_t v = c[j];
      if (v > 127) { v = 127; ++clamps; }
      if (v < -127) { v = -127; ++clamps; }
      packed[j >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (j & 3));
    }
    int8_t* out = (int8_t*)A.y + lrow * A.ld + col;
    *(uint2*)out = make_uint2(packed[0], packed[1]);
    if (q == 0) A.g[lrow * A.tpr + col / HQ_TILE] = g;
    if (clamps && A.stats) atomicAdd(&A.stats->clamps, clamps);
    return;
  } else {
    float y[8];
    const bool exact = !A.dither && LAT != kA2;
    const uint32_t sbits = A.rotation ? sign_bits8(A.smask, q * 8) : 0u;
    const uint32_t dbits = sign_bits8(A.dmask, col);
    if (exact) {
      int32_t v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = ((sbits >> j) & 1u) ? -c[j] : c[j];
      fwht128_i(v, lane);
#pragma unroll
      for (int j = 0; j < 8; ++j) y[j] = (float)(((dbits >> j) & 1u) ? -v[j] : v[j]) * g;
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) y[j] = code_coord<LAT>(c[j], j);
      if (A.dither) {
        float u[8];
        dither8<LAT>(A.dither_seed, grow, col, u);
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = y[j] - u[j];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) y[j] = flip(y[j], sbits, j);
      fwht128(y, lane);
#pragma unroll
      for (int j = 0; j < 8; ++j) y[j] = flip(y[j], dbits, j) * g;
    }
    if (!active) return;
    if constexpr (MODE == 0) {
      float4* out = (float4*)((float*)A.y + lrow * A.ld + col);
      out[0] = make_float4(y[0], y[1], y[2], y[3]);
      out[1] = make_float4(y[4], y[5], y[6], y[7]);
    } else {
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = f32_to_bf16(y[2 * i]) | (f32_to_bf16(y[2 * i + 1]) << 16);
      *(uint4*)((uint16_t*)A.y + lrow * A.ld + col) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

// ------------------------------------------------------------ activation prep
// One workgroup per token row: per 128-column tile y = H D a (canonical stage
// order, the weights' signs), amax over the row, then int8.

__global__ __launch_bounds__(256) void hq_act_prep_kernel(hq_actprep_args A) {
  extern __shared__ float ybuf[];
  __shared__ float s_max[4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t row = blockIdx.x;
  const uint16_t* arow = (const uint16_t*)A.a + row * A.lda;
  float amax = 0.0f;
  for (int64_t base = (int64_t)wave * HQ_SUB; base < A.K; base += 4 * HQ_SUB) {
    const int64_t col = base + (lane >> 4) * HQ_TILE + (lane & 15) * 8;
    float v[8];
    const uint4 raw = *(const uint4*)(arow + col);
    const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = bf16_to_f32(w4[i] & 0xFFFFu);
      v[2 * i + 1] = bf16_to_f32(w4[i] >> 16);
    }
    const uint32_t dbits = sign_bits8(A.dmask, col);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = flip(v[i], dbits, i);
    fwht128(v, lane);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      amax = __builtin_fmaxf(amax, __builtin_fabsf(v[i]));
      ybuf[col + i] = v[i];
    }
  }
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) amax = __builtin_fmaxf(amax, __shfl_xor(amax, m, 64));
  if (lane == 0) s_max[wave] = amax;
  __syncthreads();
  amax = __builtin_fmaxf(__builtin_fmaxf(s_max[0], s_max[1]), __builtin_fmaxf(s_max[2], s_max[3]));
  const float inv = (amax == 0.0f) ? 0.0f : 127.0f / amax;
  int8_t* xrow = A.xq + row * A.K;
  for (int64_t col = (int64_t)tid * 4; col < A.K; col += 1024) {
    uint32_t packed = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float qv = __builtin_rintf(ybuf[col + i] * inv);
      qv = __builtin_fminf(__builtin_fmaxf(qv, -127.0f), 127.0f);
      packed |= ((uint32_t)(int32_t)qv & 0xFFu) << (8 * i);
    }
    *(uint32_t*)(xrow + col) = packed;
  }
  if (tid == 0) A.sx[row] = amax / 127.0f;
}


// ------------------------------------------------------------ block-scaled int8 GEMM
// out[m, n] = s_x[m] * sum_t g[n, t] * P_t[m, n], P_t the exact int32 sum of
// one 128-deep K tile on the int8 matrix cores (v_mfma_i32_32x32x32_i8).
// Workgroup tile 128 (tokens) x 128 (weight rows), four waves in 2 x 2, each
// 64 x 64 = 2 x 2 MFMA blocks.  A and B stage through LDS one K tile at a
// time.  Both operands are K-contiguous rows and every lane loads the same
// 16 contiguous k for A and B, so the contraction pairs identical k whatever
// order the instruction assigns inside its 32-deep step.  Output lane l of a
// 32 x 32 block holds column l % 32 and rows 8 (r / 4) + 4 (l / 32) + r % 4.

typedef int v4i_t __attribute__((ext_vector_type(4)));
typedef int v16i_t __attribute__((ext_vector_type(16)));

constexpr int kGemmTile = 128;
constexpr int kGemmLd = 144;  // padded LDS row (bytes)

__global__ __launch_bounds__(256) void hq_gemm_i8_kernel(hq_gemm_args A) {
  __shared__ __attribute__((aligned(16))) int8_t sa[kGemmTile * kGemmLd];
  __shared__ __attribute__((aligned(16))) int8_t sb[kGemmTile * kGemmLd];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t m0 = (int64_t)blockIdx.y * kGemmTile, n0 = (int64_t)blockIdx.x * kGemmTile;
  const int64_t T = A.K / HQ_TILE;

  float accf[2][2][16];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) accf[a][b][r] = 0.0f;

  for (int64_t t = 0; t < T; ++t) {
    // stage the K tile: 128 rows x 128 bytes each for A and B
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i;
      const int row = c >> 3, kc = (c & 7) * 16;
      const int64_t ma = m0 + row, nb = n0 + row;
      uint4 va = make_uint4(0, 0, 0, 0), vb = make_uint4(0, 0, 0, 0);
      if (ma < A.M) va = *(const uint4*)(A.xq + ma * A.K + t * HQ_TILE + kc);
      if (nb < A.N) vb = *(const uint4*)(A.w + nb * A.K + t * HQ_TILE + kc);
      *(uint4*)(sa + row * kGemmLd + kc) = va;
      *(uint4*)(sb + row * kGemmLd + kc) = vb;
    }
    __syncthreads();
    v16i_t acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) acc[a][b] = (v16i_t){};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int koff = ks * 32 + (lane >> 5) * 16;
      v4i_t fa[2], fb[2];
#pragma unroll
      for (int a = 0; a < 2; ++a)
        fa[a] = *(const v4i_t*)(sa + (wm * 64 + a * 32 + (lane & 31)) * kGemmLd + koff);
#pragma unroll
      for (int b = 0; b < 2; ++b)
        fb[b] = *(const v4i_t*)(sb + (wn * 64 + b * 32 + (lane & 31)) * kGemmLd + koff);
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[a], fb[b], acc[a][b], 0, 0, 0);
    }
    // rescale the exact tile sums by the weight factor of column n
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int64_t n = n0 + wn * 64 + b * 32 + (lane & 31);
      const float gv = (n < A.N) ? A.g[n * T + t] : 0.0f;
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int r = 0; r < 16; ++r) accf[a][b][r] = accf[a][b][r] + (float)acc[a][b][r] * gv;
    }
    __syncthreads();
  }

#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t m = m0 + wm * 64 + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (m >= A.M) continue;
      const float sxm = A.sx[m];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int64_t n = n0 + wn * 64 + b * 32 + (lane & 31);
        if (n >= A.N) continue;
        const float v = sxm * accf[a][b][r];
        if (A.out_bf16)
          ((uint16_t*)A.out)[m * A.N + n] = (uint16_t)f32_to_bf16(v);
        else
          ((float*)A.out)[m * A.N + n] = v;
      }
    }
}

// ------------------------------------------------------------ utilities

__global__ void hq_zero_kernel(uint32_t* p, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

template <int LAT>
int launch_encode_lat(const hq_encode_args& a, int xt, hipStream_t st) {
  const size_t lds = (size_t)a.lds_words * HQ_WAVES_PER_WG * sizeof(uint32_t);
  if (xt == HQ_BF16)
    hipLaunchKernelGGL((hq_encode_kernel<LAT, HQ_BF16>), dim3(a.nwg), dim3(256), lds, st, a);
  else
    hipLaunchKernelGGL((hq_encode_kernel<LAT, HQ_FP32>), dim3(a.nwg), dim3(256), lds, st, a);
  return (int)hipGetLastError();
}

template <int LAT>
int launch_decode_lat(const hq_decode_args& a, int mode, hipStream_t st) {
  const uint32_t nwg = (uint32_t)((a.nsub + HQ_WAVES_PER_WG - 1) / HQ_WAVES_PER_WG);
  const size_t lds = (size_t)(a.lds_words + 64) * HQ_WAVES_PER_WG * sizeof(uint32_t);
  if (mode == 0)
    hipLaunchKernelGGL((hq_decode_kernel<LAT, 0>), dim3(nwg), dim3(256), lds, st, a);
  else if (mode == 1)
    hipLaunchKernelGGL((hq_decode_kernel<LAT, 1>), dim3(nwg), dim3(256), lds, st, a);
  else
    hipLaunchKernelGGL((hq_decode_kernel<LAT, 2>), dim3(nwg), dim3(256), lds, st, a);
  return (int)hipGetLastError();
}

}  // namespace

int hq_launch_encode(const hq_plan_s* p, const hq_encode_args& a, int xt, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  switch (p->lattice) {
    case HQ_E8: return launch_encode_lat<kE8>(a, xt, st);
    case HQ_D4: return launch_encode_lat<kD4>(a, xt, st);
    case HQ_A2: return launch_encode_lat<kA2>(a, xt, st);
    default: return launch_encode_lat<kZ>(a, xt, st);
  }
}

int hq_launch_decode(const hq_plan_s* p, const hq_decode_args& a, int yt, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const int mode = (yt == HQ_FP32) ? 0 : 1;
  switch (p->lattice) {
    case HQ_E8: return launch_decode_lat<kE8>(a, mode, st);
    case HQ_D4: return launch_decode_lat<kD4>(a, mode, st);
    case HQ_A2: return launch_decode_lat<kA2>(a, mode, st);
    default: return launch_decode_lat<kZ>(a, mode, st);
  }
}

int hq_launch_decode_int8(const hq_plan_s* p, const hq_decode_args& a, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  switch (p->lattice) {
    case HQ_E8: return launch_decode_lat<kE8>(a, 2, st);
    case HQ_D4: return launch_decode_lat<kD4>(a, 2, st);
    default: return launch_decode_lat<kZ>(a, 2, st);
  }
}

int hq_launch_act_prep(const hq_actprep_args& a, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const size_t lds = (size_t)a.K * sizeof(float);
  hipLaunchKernelGGL(hq_act_prep_kernel, dim3((uint32_t)a.M), dim3(256), lds, st, a);
  return (int)hipGetLastError();
}

int hq_launch_gemm(const hq_gemm_args& a, void* stream) {
  if (a.K % HQ_TILE != 0) return -1;
  const dim3 grid((uint32_t)((a.N + kGemmTile - 1) / kGemmTile), (uint32_t)((a.M + kGemmTile - 1) / kGemmTile));
  hipLaunchKernelGGL(hq_gemm_i8_kernel, grid, dim3(256), 0, (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

int hq_launch_zero(void* ptr, size_t bytes, void* stream) {
  const size_t n = bytes / 4;
  if (n == 0) return 0;
  hipLaunchKernelGGL(hq_zero_kernel, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0,
                     (hipStream_t)stream, (uint32_t*)ptr, n);
  return (int)hipGetLastError();
}
