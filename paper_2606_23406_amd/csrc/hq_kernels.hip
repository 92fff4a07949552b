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
// method writes as two roundings stays two roundings.  The fused
// multiply-adds used below either have a multiplier of +-1 or +-2 (one
// rounding of a sum or difference, the same as the add or subtract they
// replace) or work on integer values (exact); the one exception is the int8
// GEMM's per-tile rescale, a floating-point accumulation whose results are
// held to a tolerance rather than bit for bit.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

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

// DPP lane moves (data-parallel primitives of the gfx9 VALU): dst lane l reads
// src lane f(l) inside its 16-lane row; lanes whose row/bank is masked off
// keep `old`, lanes with no source read 0 when BC is set.
template <int CTRL, int RM = 0xF, int BM = 0xF, bool BC = false>
__device__ __forceinline__ uint32_t dpp(uint32_t old, uint32_t src) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)src, CTRL, RM, BM, BC);
}

constexpr int kDppQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]
constexpr int kDppRowShl4 = 0x104;  // lane l reads l + 4
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppRowRor8 = 0x128;  // lane l reads (l + 8) mod 16 = l ^ 8
constexpr int kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143;

// Value of lane l ^ M (M in 1, 2, 4, 8: inside the 16-lane row).
template <int M>
__device__ __forceinline__ uint32_t xor_lane(uint32_t v) {
  if constexpr (M == 1) {
    return dpp<kDppQuadXor1>(v, v);
  } else if constexpr (M == 2) {
    return dpp<kDppQuadXor2>(v, v);
  } else if constexpr (M == 4) {
    const uint32_t t = dpp<kDppRowShl4, 0xF, 0x5>(v, v);  // banks 0, 2 read l + 4
    return dpp<kDppRowShr4, 0xF, 0xA>(t, v);              // banks 1, 3 read l - 4
  } else {
    return dpp<kDppRowRor8>(v, v);
  }
}

template <int M>
__device__ __forceinline__ float xor_lane_f(float v) {
  return __uint_as_float(xor_lane<M>(__float_as_uint(v)));
}

// Inclusive prefix sum over the 64 lanes (row shifts, then row broadcasts).
__device__ __forceinline__ uint32_t wave_scan_incl(uint32_t x) {
  x += dpp<kDppRowShr1, 0xF, 0xF, true>(0u, x);
  x += dpp<kDppRowShr2, 0xF, 0xF, true>(0u, x);
  x += dpp<kDppRowShr4, 0xF, 0xF, true>(0u, x);
  x += dpp<kDppRowShr8, 0xF, 0xF, true>(0u, x);
  x += dpp<kDppRowBcast15, 0xA, 0xF>(0u, x);
  x += dpp<kDppRowBcast31, 0xC, 0xF>(0u, x);
  return x;
}

// Two inclusive prefix sums over the 64 lanes at once (interleaved, so the
// two chains' latencies overlap).
__device__ __forceinline__ void wave_scan_incl2(uint32_t& a, uint32_t& b) {
  a += dpp<kDppRowShr1, 0xF, 0xF, true>(0u, a);
  b += dpp<kDppRowShr1, 0xF, 0xF, true>(0u, b);
  a += dpp<kDppRowShr2, 0xF, 0xF, true>(0u, a);
  b += dpp<kDppRowShr2, 0xF, 0xF, true>(0u, b);
  a += dpp<kDppRowShr4, 0xF, 0xF, true>(0u, a);
  b += dpp<kDppRowShr4, 0xF, 0xF, true>(0u, b);
  a += dpp<kDppRowShr8, 0xF, 0xF, true>(0u, a);
  b += dpp<kDppRowShr8, 0xF, 0xF, true>(0u, b);
  a += dpp<kDppRowBcast15, 0xA, 0xF>(0u, a);
  b += dpp<kDppRowBcast15, 0xA, 0xF>(0u, b);
  a += dpp<kDppRowBcast31, 0xC, 0xF>(0u, a);
  b += dpp<kDppRowBcast31, 0xC, 0xF>(0u, b);
}

// Sum over the 64 lanes, as a wave-uniform value.
__device__ __forceinline__ uint32_t wave_total(uint32_t x) {
  return __builtin_amdgcn_readlane(wave_scan_incl(x), 63);
}

// a ^ b ^ c in one instruction (gfx950 three-input bitwise op, truth table
// 0x96 over S0 = 0xF0, S1 = 0xCC, S2 = 0xAA).
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t r;
  asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// (a << sh) | c and (1 << sh) | c in one instruction each.
__device__ __forceinline__ uint32_t lshl_or(uint32_t a, uint32_t sh, uint32_t c) {
  uint32_t r;
  asm("v_lshl_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(sh), "v"(c));
  return r;
}
// (a << sh) | c with a wave-uniform shift held in a scalar register
__device__ __forceinline__ uint32_t lshl_or_s(uint32_t a, uint32_t sh, uint32_t c) {
  uint32_t r;
  asm("v_lshl_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "s"(sh), "v"(c));
  return r;
}
__device__ __forceinline__ uint32_t bit_or(uint32_t sh, uint32_t c) {
  uint32_t r;
  asm("v_lshl_or_b32 %0, 1, %1, %2" : "=v"(r) : "v"(sh), "v"(c));
  return r;
}

// 2 v ^ (v >> 31); the doubling as an add, which gfx950 issues at the fast
// VALU rate (a left shift takes the slow one).
__device__ __forceinline__ uint32_t zigzag(int32_t v) {
  uint32_t d;
  asm("v_add_u32 %0, %1, %1" : "=v"(d) : "v"(v));
  return d ^ (uint32_t)(v >> 31);
}

__device__ __forceinline__ int32_t unzigzag(uint32_t m) {
  return (int32_t)(m >> 1) ^ -(int32_t)(m & 1u);
}

// In-byte select table: entry v packs, 4 bits per rank k = 0..7, the position
// of the k-th set bit of the byte value v (entries for ranks past popc(v)
// are unused).
__device__ __forceinline__ uint32_t byte_select_entry(uint32_t v) {
  uint32_t e = 0, k = 0;
#pragma unroll
  for (uint32_t b = 0; b < 8; ++b) {
    if ((v >> b) & 1u) {
      e |= b << (4 * k);
      ++k;
    }
  }
  return e;
}

// The whole table, built at compile time; kernels copy it into LDS.
struct ByteSelectTable {
  uint32_t e[256];
  constexpr ByteSelectTable() : e() {
    for (uint32_t v = 0; v < 256; ++v) {
      uint32_t x = 0, k = 0;
      for (uint32_t b = 0; b < 8; ++b)
        if ((v >> b) & 1u) {
          x |= b << (4 * k);
          ++k;
        }
      e[v] = x;
    }
  }
};
__constant__ ByteSelectTable kByteSelect = ByteSelectTable();

// Position (0..31) of the r-th set bit (r from 0, r < popc(w)) of w: the
// byte from cumulative byte popcounts, the bit from the table.
__device__ __forceinline__ uint32_t select32_lut(uint32_t w, uint32_t r, const uint32_t* tbl) {
  const uint32_t c1 = __popc(w & 0xFFu), c2 = __popc(w & 0xFFFFu), c3 = __popc(w & 0xFFFFFFu);
  const uint32_t b = (uint32_t)(r >= c1) + (uint32_t)(r >= c2) + (uint32_t)(r >= c3);
  const uint32_t below = b == 0 ? 0u : (b == 1 ? c1 : (b == 2 ? c2 : c3));
  const uint32_t byte = __builtin_amdgcn_ubfe(w, 8 * b, 8);
  return 8 * b + __builtin_amdgcn_ubfe(tbl[byte], 4 * (r - below), 3);
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

// Two fp32 -> bf16 (round to nearest even) in one word: lo in bits 0-15.
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  uint32_t r;
  asm("v_cvt_pk_bf16_f32 %0, %1, %2" : "=v"(r) : "v"(lo), "v"(hi));
  return r;
}

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
    // each 64-bit product is one v_mad_u64_u32 (both halves in one issue)
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
    const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
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

// E8's U = b - Q(b) for a box point b in [-2, 2)^8 whose coordinates are
// multiples of 2^-22: the point quant_e8 picks, without its roundings and
// branches.  Every coset error is exact here: the even coset's is
// b - 2 rint(b / 2) (rint by the 1.5 * 2^23 shift, whose low bit is k's
// parity), the odd coset's b - sign(b) (floor(b / 2) is 0 or -1), and
// neither is ever -0.  A coset whose parity is odd moves its first
// coordinate of largest error to the next point on the other side, which
// turns that error e into e - 2 sign(e); the squared errors are summed in
// the same fp32 tree as quant_e8's, and U is the nearer coset's error vector
// (the even one on a tie).
__device__ __forceinline__ void dither_e8(const float* b, float* u) {
  constexpr float kShift = 12582912.0f;  // 1.5 * 2^23
  float ea[8], eb[8];
  uint32_t pa = 0, pb = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float t = b[i] * 0.5f + kShift;
    ea[i] = __builtin_fmaf(-2.0f, t - kShift, b[i]);
    pa ^= __float_as_uint(t);
    const uint32_t sb = __float_as_uint(b[i]) & 0x80000000u;
    eb[i] = b[i] - __uint_as_float(sb | 0x3F800000u);
    pb ^= sb;
  }
  auto fix = [](float* e, bool odd) {
    float m = __builtin_fabsf(e[0]);
#pragma unroll
    for (int i = 1; i < 8; ++i) m = __builtin_fmaxf(m, __builtin_fabsf(e[i]));
    bool done = !odd;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const bool hit = !done && __builtin_fabsf(e[i]) == m;
      const float two = __uint_as_float((__float_as_uint(e[i]) & 0x80000000u) | 0x40000000u);
      e[i] = hit ? e[i] - two : e[i];
      done = done || hit;
    }
  };
  fix(ea, pa & 1u);
  fix(eb, pb >> 31);
  float sa[8], sq[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    sa[i] = ea[i] * ea[i];
    sq[i] = eb[i] * eb[i];
  }
  const bool even = tree8(sa) <= tree8(sq);
#pragma unroll
  for (int i = 0; i < 8; ++i) u[i] = even ? ea[i] : eb[i];
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
  if constexpr (LAT == kE8) {
    dither_e8(b, u);
  } else {
    int32_t c[8];
    quantize8<LAT>(b, c);
#pragma unroll
    for (int i = 0; i < 8; ++i) u[i] = b[i] - code_coord<LAT>(c[i], i);
  }
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

// E8 unstrip (Sec. 4.6) in closed form: 2 unzz(s) = s ^ -(s & 1), so
// c_i = 2 h_i + cb = (s_i ^ -(s_i & 1)) + cb for i < 7; h_i = unzz(s_i) has the
// parity of bit 1 ^ bit 0 of s_i, so p = bit 1 ^ bit 0 of the XOR of s_0..s_6;
// s_7 = 2 zz(t) + cb gives 2 t = z ^ -(z & 1) with z = s_7 >> 1, and
// c_7 = 2 (2 t + p) + cb.
__device__ __forceinline__ void e8_unstrip(const uint32_t* s, int32_t* c) {
  const uint32_t cb = s[7] & 1u;
#pragma unroll
  for (int i = 0; i < 7; ++i)
    c[i] = (int32_t)((s[i] ^ (uint32_t)__builtin_amdgcn_sbfe((int32_t)s[i], 0, 1)) + cb);
  const uint32_t X = xor3(xor3(s[0], s[1], s[2]), s[3], s[4]) ^ s[5] ^ s[6];
  const uint32_t p = ((X >> 1) ^ X) & 1u;
  const uint32_t t2 = (s[7] >> 1) ^ (uint32_t)__builtin_amdgcn_sbfe((int32_t)s[7], 1, 1);
  c[7] = (int32_t)((t2 << 1) + ((p << 1) | cb));
}

template <int LAT>
__device__ __forceinline__ void unstrip8(const uint32_t* s, int32_t* c) {
  if constexpr (LAT == kE8) {
    e8_unstrip(s, c);
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

// Butterfly with lane l ^ M: the lower lane keeps a + b, the upper a - b,
// with a the lower lane's value.  s = +1 (lower) or -1 (upper) makes it one
// exact-multiplier fma: fma(v, s, p) = round(p + s v).
template <int M>
__device__ __forceinline__ void fwht_xlane(float* v, float s) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float p = xor_lane_f<M>(v[j]);
    v[j] = __builtin_fmaf(v[j], s, p);
  }
}

// Per-lane butterfly signs for the cross-lane stages (h = 8, 16, 32, 64).
struct XSigns {
  float f[4];
  __device__ __forceinline__ explicit XSigns(int lane) {
#pragma unroll
    for (int b = 0; b < 4; ++b) f[b] = ((lane >> b) & 1) ? -1.0f : 1.0f;
  }
};

__device__ __forceinline__ void fwht128(float* v, const XSigns& sg) {
  fwht8_inlane(v);
  fwht_xlane<1>(v, sg.f[0]);
  fwht_xlane<2>(v, sg.f[1]);
  fwht_xlane<4>(v, sg.f[2]);
  fwht_xlane<8>(v, sg.f[3]);
}


// The 8 sign bits of columns col0 .. col0 + 7 (col0 a multiple of 8).
__device__ __forceinline__ uint32_t sign_bits8(const uint32_t* mask, int64_t col0) {
  return (mask[col0 >> 5] >> (uint32_t)(col0 & 31)) & 0xFFu;
}

__device__ __forceinline__ float flip(float v, uint32_t bits, int j) {
  return __uint_as_float(__float_as_uint(v) ^ (((bits >> j) & 1u) << 31));
}

// Four fp32 values as OCP E4M3 bytes (v_cvt_pk_fp8_f32: round to nearest
// even), the first in the low byte; the caller keeps them within +-448.
__device__ __forceinline__ uint32_t e4m3x4(float a, float b, float c, float d) {
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c, d, lo, true);
}

// OCP FP4 E2M1 code of v (magnitudes 0, .5, 1, 1.5, 2, 3, 4, 6 as codes 0 .. 7):
// the nearest value, ties to the even code, saturating at 6, the sign bit
// (bit 3) kept also when v rounds to zero.  The comparisons place each tie
// on its even side.
__device__ __forceinline__ uint32_t e2m1_code(float v) {
  const float a = __builtin_fabsf(v);
  const uint32_t c = (uint32_t)(a > 0.25f) + (uint32_t)(a >= 0.75f) + (uint32_t)(a > 1.25f) +
                     (uint32_t)(a >= 1.75f) + (uint32_t)(a > 2.5f) + (uint32_t)(a >= 3.5f) +
                     (uint32_t)(a > 5.0f);
  return c | ((__float_as_uint(v) >> 28) & 8u);
}

// The MX block exponent X = floor(log2 amax) - 2 of a block whose largest
// magnitude is amax (E8M0's range; -127 for an all-zero block).
__device__ __forceinline__ int32_t mx_exponent(float amax) {
  if (!(amax > 0.0f)) return -127;
  const int32_t e = __builtin_amdgcn_frexp_expf(amax);  // amax = m 2^e, m in [0.5, 1)
  return max(-127, min(127, e - 3));
}

// Lanes of one wave exchange values through LDS: every lane's earlier LDS
// writes are visible to the others' later reads.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// v <- M v for the tile of the lane's group of 16 (its coordinates
// 8 (lane % 16) + j): the qjl rotation of Sec. 4.2 with M = S (encode) or S^T
// (decode).  Mt is M^T row-major, so row k holds column k of M and a lane's 8
// outputs read 32 contiguous bytes of it per k.  Each output is the
// left-to-right fp32 sum of the rounded products from k = 0, the order the
// oracle defines; v passes through the group's 128 floats of `stage` (LDS).
__device__ __forceinline__ void qjl_tile(const float* __restrict__ Mt, float* stage, int lane,
                                         float* v) {
  float* t = stage + (lane >> 4) * HQ_TILE;
  const int c0 = (lane & 15) * 8;
  *(float4*)(t + c0) = make_float4(v[0], v[1], v[2], v[3]);
  *(float4*)(t + c0 + 4) = make_float4(v[4], v[5], v[6], v[7]);
  wave_lds_sync();
  float acc[8];
  {
    const float z = t[0];
    const float4 a = *(const float4*)(Mt + c0), b = *(const float4*)(Mt + c0 + 4);
    acc[0] = a.x * z; acc[1] = a.y * z; acc[2] = a.z * z; acc[3] = a.w * z;
    acc[4] = b.x * z; acc[5] = b.y * z; acc[6] = b.z * z; acc[7] = b.w * z;
  }
#pragma unroll 4
  for (int k = 1; k < HQ_TILE; ++k) {
    const float z = t[k];
    const float4 a = *(const float4*)(Mt + k * HQ_TILE + c0);
    const float4 b = *(const float4*)(Mt + k * HQ_TILE + c0 + 4);
    acc[0] = acc[0] + a.x * z; acc[1] = acc[1] + a.y * z;
    acc[2] = acc[2] + a.z * z; acc[3] = acc[3] + a.w * z;
    acc[4] = acc[4] + b.x * z; acc[5] = acc[5] + b.y * z;
    acc[6] = acc[6] + b.z * z; acc[7] = acc[7] + b.w * z;
  }
  wave_lds_sync();  // every lane has read the stage before it is written again
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = acc[i];
}

// ------------------------------------------------------------ look-back scan
// Decoupled look-back (Merrill & Garland, 2016) over workgroups in index
// order.  Workgroups are dispatched in increasing index order, and a group
// only ever waits for lower indices, so every wait ends; each wait is also
// bounded, and a status that never arrives ends the wait with an error
// status instead of a hang.  The scan scratch starts with a 64-bit epoch word
// that the last workgroup of a launch advances after it has published its
// inclusive prefix (by then every group has read the epoch, since that prefix
// sums every group's published aggregate), so every launch -- also a
// replayed graph -- gets a fresh epoch without host help.  A status word
// packs the value (32 bits: words since the start of this launch), a flag
// (2 bits: 1 = aggregate, 2 = inclusive prefix) and the epoch (30 bits), so
// the array never needs clearing.

constexpr uint32_t kEpochMask = 0x3FFFFFFFu;
constexpr uint32_t kSpinLimit = 1u << 24;

__device__ __forceinline__ unsigned long long pack_status(uint32_t epoch, uint32_t flag,
                                                          uint32_t value) {
  return ((unsigned long long)(epoch & kEpochMask) << 34) | ((unsigned long long)flag << 32) |
         (unsigned long long)value;
}

// Relaxed is enough: a status word carries its own value, and no other data
// published by the workgroup is read through it.
__device__ __forceinline__ void store_status(unsigned long long* p, unsigned long long v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ unsigned long long load_status(unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------ bit assembly

// OR the 64 bits of v into the LDS bit array at bit position pos.
__device__ __forceinline__ void or_bits64(uint32_t* buf, uint32_t pos, uint64_t v) {
  if (v == 0) return;
  const uint32_t w = pos >> 5, sh = pos & 31u;
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  const uint32_t o0 = lo << sh;
  const uint32_t o1 = sh ? ((hi << sh) | (lo >> (32u - sh))) : hi;
  const uint32_t o2 = sh ? (hi >> (32u - sh)) : 0u;
  if (o0) atomicOr(&buf[w], o0);
  if (o1) atomicOr(&buf[w + 1], o1);
  if (o2) atomicOr(&buf[w + 2], o2);
}

// 64 bits of the LDS bit array starting at bit pos (words past nw read 0).
__device__ __forceinline__ uint64_t load_bits64(const uint32_t* buf, uint32_t pos, uint32_t nw) {
  const uint32_t w = pos >> 5, sh = pos & 31u;
  const uint32_t a = w < nw ? buf[w] : 0u;
  const uint32_t b = w + 1 < nw ? buf[w + 1] : 0u;
  const uint32_t c = w + 2 < nw ? buf[w + 2] : 0u;
  const uint32_t lo = sh ? ((a >> sh) | (b << (32u - sh))) : a;
  const uint32_t hi = sh ? ((b >> sh) | (c << (32u - sh))) : b;
  return ((uint64_t)hi << 32) | lo;
}

// Bit offset of field j inside a lane's remainder region.
template <int LAT>
__device__ __forceinline__ uint32_t rem_offset(int j, uint32_t k0, uint32_t k1) {
  if constexpr (LAT == kD4) {
    return (uint32_t)(j >> 2) * (3u * k0 + k1) + (uint32_t)(j & 3) * k0;
  } else if constexpr (LAT == kA2) {
    return (uint32_t)(j >> 1) * (k0 + k1) + (uint32_t)(j & 1) * k0;
  } else {
    return (uint32_t)j * k0;
  }
}

// ------------------------------------------------------------ twisted FWHT
// A cross-lane butterfly written as one multiply-add per value,
//   u <- u + s * u[l ^ M]      (s = +1 on the lower lane, -1 on the upper),
// leaves the lower lane a + b and the upper lane b - a = -(a - b): the
// butterfly output times s, rounded identically (round-to-nearest-even
// commutes with negation).  The partner lane of a stage shares the signs of
// every earlier stage, so earlier factors pull out of the butterfly and four
// chained stages leave each lane its outputs times sigma, the product of its
// four stage signs.  Callers fold sigma into the per-tile factor that
// follows.  The h = 8, 16, 64 stages are one DPP-fused v_fmac each
// (quad_perm and row_ror lane moves); the h = 32 stage (lane l ^ 4) reads
// its partner through ds_swizzle.

#define HQ_DPP_FULL "row_mask:0xf bank_mask:0xf bound_ctrl:1"
// v[j] += s * v[partner lane][j] for the 8 values of a lane; the s_nop pairs
// cover the two wait states between a VALU write and a DPP read of a VGPR.
#define HQ_FMAC_DPP8(CTRL, v, s)                                                            \
  asm("s_nop 1\n\t"                                                                         \
      "v_fmac_f32_dpp %0, %0, %8 " CTRL " " HQ_DPP_FULL "\n\t"                              \
      "v_fmac_f32_dpp %1, %1, %8 " CTRL " " HQ_DPP_FULL "\n\t"                              \
      "v_fmac_f32_dpp %2, %2, %8 " CTRL " " HQ_DPP_FULL "\n\t"                              \
      "v_fmac_f32_dpp %3, %3, %8 " CTRL " " HQ_DPP_FULL "\n\t"                              \
      "v_fmac_f32_dpp %4, %4, %8 " CTRL " " HQ_DPP_FULL "\n\t"                              \
      "v_fmac_f32_dpp %5, %5, %8 " CTRL " " HQ_DPP_FULL "\n\t"                              \
      "v_fmac_f32_dpp %6, %6, %8 " CTRL " " HQ_DPP_FULL "\n\t"                              \
      "v_fmac_f32_dpp %7, %7, %8 " CTRL " " HQ_DPP_FULL "\n\t"                              \
      "s_nop 1"                                                                             \
      : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]), \
        "+v"(v[7])                                                                          \
      : "v"(s))

// Value of lane l ^ 4 (ds_swizzle bit-mask mode: and 0x1F, or 0, xor 4).
__device__ __forceinline__ float swz_xor4(float v) {
  return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x101F));
}

// Value of lane l ^ 16 (the same mode with xor 16) and of lane l ^ 32.
__device__ __forceinline__ float swz_xor16(float v) {
  return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x401F));
}
__device__ __forceinline__ float lane_xor32(float v) {
  return __int_as_float(__shfl_xor(__float_as_int(v), 32, 64));
}



// Value of lane l ^ M for M = 1, 2, 8 (bound_ctrl DPP moves, which fold into
// the consuming VOP2 instruction).
template <int M>
__device__ __forceinline__ float dpp_xor(float v) {
  constexpr int ctrl = M == 1 ? kDppQuadXor1 : (M == 2 ? kDppQuadXor2 : kDppRowRor8);
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), ctrl, 0xF, 0xF, true));
}

// Stage signs of a lane (h = 8, 16, 32, 64 <-> lane bits 0..3) and sigma's
// sign bit.
struct TwSigns {
  float f[4];
  uint32_t sigma;  // 0 or 0x80000000
  __device__ __forceinline__ explicit TwSigns(int lane) {
#pragma unroll
    for (int b = 0; b < 4; ++b) f[b] = ((lane >> b) & 1) ? -1.0f : 1.0f;
    sigma = (uint32_t)(__popc((uint32_t)lane & 15u) & 1) << 31;
    // kept in registers for the whole kernel rather than recomputed from
    // the lane index before every transform
#pragma unroll
    for (int b = 0; b < 4; ++b) asm volatile("" : "+v"(f[b]));
    asm volatile("" : "+v"(sigma));
  }
};

// v = sigma * (H v) over the tile (in-lane stages h = 1, 2, 4 first).
__device__ __forceinline__ void fwht128_tw(float* v, const TwSigns& sg) {
  fwht8_inlane(v);
  HQ_FMAC_DPP8("quad_perm:[1,0,3,2]", v, sg.f[0]);
  HQ_FMAC_DPP8("quad_perm:[2,3,0,1]", v, sg.f[1]);
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = __builtin_fmaf(swz_xor4(v[j]), sg.f[2], v[j]);
  HQ_FMAC_DPP8("row_ror:8", v, sg.f[3]);
}

// Tiles longer than 128 (Sec. 7.2 sweeps 128 .. 2048).  A wave holds four
// consecutive sub-streams of 512 scalars, lane l coordinates 8 l .. 8 l + 7
// of each, so a tile of n <= 512 spans n / 8 lanes of one sub-stream and a
// longer one spans n / 512 whole sub-streams of the wave.  The transform's
// stages h = 128 and 256 pair lanes l ^ 16 and l ^ 32 (twisted as the
// h = 8 .. 64 stages, which multiplies sigma by the two lane signs); the
// stages h = 512 and 1024 pair sub-streams i ^ 1 and i ^ 2 of the same lane,
// plain butterflies (both operands carry the lane's sigma).  Returns the
// sign bit of the lane's sigma.
__device__ __forceinline__ uint32_t fwht_tiled(float (*x)[8], int lane, uint32_t tile,
                                               const TwSigns& sg) {
  uint32_t sigma = sg.sigma;
#pragma unroll
  for (int i = 0; i < 4; ++i) fwht128_tw(x[i], sg);
  if (tile >= 256u) {
    const float s4 = (lane & 16) ? -1.0f : 1.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) x[i][j] = __builtin_fmaf(swz_xor16(x[i][j]), s4, x[i][j]);
    sigma ^= (uint32_t)(lane & 16) << 27;
  }
  if (tile >= 512u) {
    const float s5 = (lane & 32) ? -1.0f : 1.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) x[i][j] = __builtin_fmaf(lane_xor32(x[i][j]), s5, x[i][j]);
    sigma ^= (uint32_t)(lane & 32) << 26;
  }
  if (tile >= 1024u) {
#pragma unroll
    for (int i = 0; i < 4; i += 2)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float a = x[i][j], b = x[i + 1][j];
        x[i][j] = a + b;
        x[i + 1][j] = a - b;
      }
  }
  if (tile >= 2048u) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float a = x[i][j], b = x[i + 2][j];
        x[i][j] = a + b;
        x[i + 2][j] = a - b;
      }
  }
  return sigma;
}

__device__ __forceinline__ float xor_sign(float v, uint32_t bit) {
  return __uint_as_float(__float_as_uint(v) ^ bit);
}

// --------------------------------------------------- E8 decision in closed form
// The decision works on w = z / 2 (the encoder's scale carries the factor
// 1/2, which is exact), where the two classes of the 2E8 realization are the
// integer points with even sum (D8 / 2) and that set shifted by 1/2.  With
// k_i = rint(w_i), ea_i = w_i - k_i (exact, |ea_i| <= 1/2), the nearest
// point of the shifted class takes floor(w_i) + 1/2 per coordinate, at
// distance 1/2 - |ea_i|.  Before the parity fixes
// sum(ea^2) - sum(eb^2) = sum(|ea_i| - 1/4); a fix moves one coordinate by 1,
// adding 1 - 2 max|ea| (first class) or 2 min|ea| (second) to its distance.
// In quarters of the full-scale difference:
//   D = sum|ea_i| - 2 + [odd_a] (1 - 2 max|ea|) - [odd_b] 2 min|ea|,
// odd_a the parity of sum k_i and odd_b that of sum floor(w_i), which differs
// from odd_a by the number of negative ea_i (the parity of the XOR of their
// sign bits).  Rounding moves the fp32 sums by far less than kE8Tie / 4, so
// a lane outside the band takes the same class as the two-sum comparison; a
// wave with any lane inside it runs quant_e8 step by step on z = 2 w.
//
// The chosen point, as h = (c - cb) / 2 (the stripped coordinates), is
// k_i for the first class and floor(w_i) = k_i - [ea_i < 0] for the second,
// plus the parity fix: +-1 on the first coordinate of largest error.  That
// error is |ea_i| in the first class and fl(1/2 - |ea_i|) in the second
// (fp32 w - (floor(w) + 1/2) has that magnitude with the reference's
// rounding), and the fix moves towards w: +1 when ea_j >= 0 (first class),
// +1 when ea_j < 0 (second; a coordinate with ea_j = +1/2 would move +1 too,
// so min|ea| = 1/2 also takes the step-by-step path).  Every +-1 is a lane
// mask folded into an add or subtract with carry.

constexpr float kE8Tie = 1.0e-3f;  // band on the full-scale distance difference

// x + carry-in / x - borrow-in, the carry a lane mask (bit l for lane l).
__device__ __forceinline__ int32_t add_lanemask(int32_t x, uint64_t m) {
  int32_t r;
  uint64_t co;
  asm("v_addc_co_u32_e64 %0, %1, %2, 0, %3" : "=v"(r), "=s"(co) : "v"(x), "s"(m));
  return r;
}
__device__ __forceinline__ int32_t sub_lanemask(int32_t x, uint64_t m) {
  int32_t r;
  uint64_t co;
  asm("v_subb_co_u32_e64 %0, %1, %2, 0, %3" : "=v"(r), "=s"(co) : "v"(x), "s"(m));
  return r;
}


// The class decision of a block inside the tie band, exactly as the
// step-by-step procedure takes it: the two classes' squared distances in
// fp32 (z units, z = 2 w), each error rebuilt exactly from ea = w - rint(w).
// The first class's error on coordinate i is 2 ea_i, and its parity fix
// (the first coordinate of largest |ea|) leaves 2 (1 - |ea_j|) in magnitude;
// the second class's is 2 (1/2 - |ea_i|), and its fix (the first coordinate
// of largest 1/2 - |ea|) leaves 2 (|ea_j| + 1/2).  Every doubling is exact,
// so each value is the procedure's own rounding; the squares are summed in
// its tree order, and the first class wins ties.
__device__ __forceinline__ bool e8_even_exact(const float* ea, float mx, float mn, bool odd_a,
                                              bool odd_b) {
  const float topb = 0.5f - mn;
  bool fixa = odd_a, fixb = odd_b;
  float sa[8], sb[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float a = __builtin_fabsf(ea[i]);
    float ua = a, ub = 0.5f - a;
    if (fixa && a == mx) {
      ua = 1.0f - a;
      fixa = false;
    }
    if (fixb && ub == topb) {
      ub = a + 0.5f;
      fixb = false;
    }
    ua = ua + ua;
    ub = ub + ub;
    sa[i] = ua * ua;
    sb[i] = ub * ub;
  }
  return tree8(sa) <= tree8(sb);
}

__device__ __forceinline__ void e8_nearest(const float* w, int32_t* h, int32_t& cb) {
  float ea[8];
  int32_t K[8];
  uint32_t eb[8];
  // rint(w) by the shift 1.5 * 2^23: for |w| < 2^22 (the scale bounds |w| by
  // alpha sqrt(128) / 2) the sum lies in [2^23, 2^24), where the fp32
  // spacing is 1, so it rounds w to the nearest integer, ties to even (the
  // shift is even); the integer is the sum's bit pattern less the shift's.
  // Four fast-rate adds instead of a rounding and a conversion.
  // ea = w + (shift - t) = w - rint(w), exact; written as a sum so that it is
  // never -0 (w = -0, which the signed scale makes of an exact zero, gives
  // -0 + +0 = +0, where w - rint(w) would give -0): the parity below reads
  // the sign bits of ea, the rounding the sign of its value, and the two
  // must agree.
  constexpr float kShift = 12582912.0f;  // 1.5 * 2^23, bits 0x4B400000
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float t = w[i] + kShift;
    const float nk = kShift - t;
    ea[i] = w[i] + nk;
    K[i] = (int32_t)(__float_as_uint(t) - 0x4B400000u);
    eb[i] = __float_as_uint(ea[i]);
  }
  float Sabs = __builtin_fabsf(ea[0]) + __builtin_fabsf(ea[1]);
#pragma unroll
  for (int i = 2; i < 8; ++i) Sabs += __builtin_fabsf(ea[i]);
  float mx = __builtin_fabsf(ea[0]), mn = mx;
#pragma unroll
  for (int i = 1; i < 8; ++i) {
    mx = __builtin_fmaxf(mx, __builtin_fabsf(ea[i]));
    mn = __builtin_fminf(mn, __builtin_fabsf(ea[i]));
  }
  // parities: sum k_i (low bits of the XOR) and the count of negative ea_i
  const uint32_t kp = xor3(xor3(xor3((uint32_t)K[0], (uint32_t)K[1], (uint32_t)K[2]), (uint32_t)K[3],
                                (uint32_t)K[4]),
                           (uint32_t)K[5], (uint32_t)K[6]) ^ (uint32_t)K[7];
  const uint32_t sx = xor3(xor3(xor3(eb[0], eb[1], eb[2]), eb[3], eb[4]), eb[5], eb[6]) ^ eb[7];
  const bool odd_a = kp & 1u;
  const bool odd_b = ((kp << 31) ^ sx) >> 31;
  const float D0 = Sabs - 2.0f;
  const float D1 = odd_a ? __builtin_fmaf(-2.0f, mx, Sabs - 1.0f) : D0;
  const float D = odd_b ? __builtin_fmaf(-2.0f, mn, D1) : D1;
  bool even = D < 0.0f;
  // Inside the tie band (or with every |ea_i| = 1/2, where the second
  // class's fix moves up from ea_j = +1/2 too) the lane takes the exact
  // decision; a wave with no such lane skips it.
  const bool tie = __builtin_fabsf(D) <= 0.25f * kE8Tie || mn >= 0.5f;
  const bool any_tie = __ballot(tie) != 0ull;
  if (any_tie && tie) even = e8_even_exact(ea, mx, mn, odd_a, odd_b);
  // lane masks: the class, whether its parity needs the fix, and per
  // coordinate the largest-error hits and the sign of ea.  The error of
  // coordinate i in the lane's class is key_i = fma(|ea_i|, +-1, 0 or 1/2):
  // |ea_i| (exact) in the first class, fl(1/2 - |ea_i|) (one rounding, as
  // the subtraction) in the second; its largest value is mx or fl(1/2 - mn).
  const uint64_t E = __ballot(even);
  const uint64_t need = (E & __ballot(odd_a)) | (~E & __ballot(odd_b));
  const float ks = even ? 1.0f : -1.0f, kc = even ? 0.0f : 0.5f;
  const float top = even ? mx : 0.5f - mn;
  uint64_t done = ~need;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint64_t hit = __ballot(__builtin_fmaf(__builtin_fabsf(ea[i]), ks, kc) == top);
    const uint64_t fix = hit & ~done;
    done |= hit;
    const uint64_t neg = __ballot(ea[i] < 0.0f);
    // up by the fix where the class and the sign agree to move up; down by
    // the fix otherwise, or by the odd class's floor (never both)
    const uint64_t t = E ^ neg;
    const uint64_t up = fix & t;
    const uint64_t down = (fix & ~t) | (neg & ~E);
    h[i] = sub_lanemask(add_lanemask(K[i], up), down);
  }
  // every |ea_i| = 1/2: the second class wins and its fix (coordinate 0)
  // moves up also from ea_0 = +1/2, where the masks above moved it down
  if (any_tie && mn >= 0.5f && !even && odd_b && ea[0] > 0.0f) h[0] += 2;
  cb = even ? 0 : 1;
}

// E8 strip (Sec. 4.6) from h = (c - cb) / 2: s_i = zz(h_i) for i < 7,
// s_7 = 2 zz(t) + cb with t = (h_7 - p) / 2 and p the parity of
// h_0 + .. + h_6.
__device__ __forceinline__ void e8_strip(const int32_t* h, int32_t cb, uint32_t* s) {
#pragma unroll
  for (int i = 0; i < 7; ++i) s[i] = zigzag(h[i]);
  const uint32_t p = xor3(xor3((uint32_t)h[0], (uint32_t)h[1], (uint32_t)h[2]), (uint32_t)h[3],
                          (uint32_t)h[4]) ^ (uint32_t)h[5] ^ (uint32_t)h[6];
  const int32_t t = (h[7] - (int32_t)(p & 1u)) >> 1;
  s[7] = 2u * zigzag(t) + (uint32_t)cb;
}

// ------------------------------------------------------------ encode kernel
// One workgroup encodes HQ_ENC_SUBS_PER_WG consecutive sub-streams (four
// waves with four each, one at a time, or sixteen waves with one each) and
// keeps their bits in LDS; then its first wave alone publishes the group's
// word count, looks back for the group's absolute word offset and writes
// payload and offsets.  KV = false is the weight path (no rotation, no
// dither, fp32 norms) compiled without those branches; KV = true reads the
// three options at run time.

// Number of k in 1..KMAX with sum >= thr[k] (thresholds clamped below 2^30
// on the host, sums below 2^26), on scalar registers.
__device__ __forceinline__ uint32_t kstar_count(uint32_t sum, const uint32_t* thr) {
  // thr[1..15] is nondecreasing, so the count is the largest t with
  // sum >= thr[t]: a binary search, each level's threshold picked by selects
  uint32_t a = sum >= thr[8] ? 8u : 0u;
  const uint32_t t4 = a ? thr[12] : thr[4];
  a += sum >= t4 ? 4u : 0u;
  const uint32_t t2 = a < 8u ? (a ? thr[6] : thr[2]) : (a == 8u ? thr[10] : thr[14]);
  a += sum >= t2 ? 2u : 0u;
  const uint32_t t1 = a < 8u ? (a < 4u ? (a ? thr[3] : thr[1]) : (a == 4u ? thr[5] : thr[7]))
                             : (a < 12u ? (a == 8u ? thr[9] : thr[11]) : (a == 12u ? thr[13] : thr[15]));
  a += sum >= t1 ? 1u : 0u;
  return a;
}

// One look-back round over the NR * 64 workgroups hi, hi - 1, ... (lane l
// takes distances r * 64 + l below hi + 1, r < NR): waits until each has
// published, then adds their values down to the nearest inclusive prefix
// into `prefix`.  Returns true when that prefix was among them (or the wait
// timed out: then `timed_out` is set).
template <int NR>
__device__ __forceinline__ bool lookback_round(unsigned long long* status, int64_t hi,
                                               uint32_t epoch, int lane, uint32_t& prefix,
                                               bool& timed_out) {
  unsigned long long st[NR];
  bool ready[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    st[r] = 0ull;
    ready[r] = hi - (r * 64 + lane) < 0;
  }
  uint32_t spins = 0;
  for (;;) {
    bool all = true;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      if (!ready[r]) {
        st[r] = load_status(&status[hi - (r * 64 + lane)]);
        ready[r] = (uint32_t)(st[r] >> 34) == epoch && ((st[r] >> 32) & 3u) != 0u;
      }
      all = all && ready[r];
    }
    if (__ballot(!all) == 0ull) break;
    if (++spins > kSpinLimit) {
      timed_out = true;
      return true;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  // nearest inclusive prefix: the first r with one, then its lowest lane
  uint32_t stop = 64u * NR;
#pragma unroll
  for (int r = NR - 1; r >= 0; --r) {
    const bool incl = hi - (r * 64 + lane) >= 0 && ((st[r] >> 32) & 3u) == 2u;
    const unsigned long long m = __ballot(incl);
    if (m) stop = (uint32_t)(r * 64) + (uint32_t)__builtin_ctzll(m);
  }
  uint32_t v = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r)
    if (hi - (r * 64 + lane) >= 0 && (uint32_t)(r * 64 + lane) <= stop) v += (uint32_t)st[r];
  prefix += wave_total(v);
  return stop < 64u * NR;
}

// Position of one wave's sub-stream: wave-uniform row and first column.
struct SubPos {
  bool active;
  uint32_t lrow, col0;
};

// The 16 (bf16) or 32 (fp32) input bytes of one lane and its RHT signs:
// bf16 XOR words (bit 15 / bit 31 of each column pair) or fp32 sign bits.
struct LaneInput {
  uint4 a, b, sw;
};

// An inactive sub-stream (past the last row; its results are discarded) has
// lrow = col0 = 0 and reads the first row, so no lane is zero-filled.
template <int XT>
__device__ __forceinline__ LaneInput load_lane_input(const hq_encode_args& A, const SubPos& P,
                                                     int lane) {
  // uniform row base plus a 32-bit per-lane byte offset (columns < 2^28)
  LaneInput in;
  const uint32_t col = P.col0 + 8u * (uint32_t)lane;
  if constexpr (XT == HQ_BF16) {
    const char* row = (const char*)((const uint16_t*)A.x + (int64_t)P.lrow * A.ld);
    in.a = *(const uint4*)(row + (col << 1));
    in.b = make_uint4(0u, 0u, 0u, 0u);
    in.sw = *(const uint4*)((const char*)A.dsign16 + (col << 1));
  } else {
    const char* row = (const char*)((const float*)A.x + (int64_t)P.lrow * A.ld);
    const uint4* p = (const uint4*)(row + (col << 2));
    in.a = p[0];
    in.b = p[1];
    in.sw = make_uint4(sign_bits8(A.dmask, col), 0u, 0u, 0u);
  }
  return in;
}

// OR the low 32 + sh bits of v << sh into buf at bit pos (two words).
__device__ __forceinline__ void or_word(uint32_t* buf, uint32_t pos, uint32_t v) {
  const uint64_t t = (uint64_t)v << (pos & 31u);
  atomicOr(&buf[pos >> 5], (uint32_t)t);
  atomicOr(&buf[(pos >> 5) + 1], (uint32_t)(t >> 32));
}

// The lane's 8 input values with the RHT signs D applied, kept in their
// loaded form until the transform needs them: four bf16 pairs or eight fp32
// words.  A wave holding several sub-streams keeps the pending ones at half
// the registers of their fp32 values (bf16), which is what lets the encoder
// run eight waves per SIMD.
template <int XT>
struct Packed {
  uint32_t w[XT == HQ_BF16 ? 4 : 8];
};

template <int XT>
__device__ __forceinline__ Packed<XT> pack_signed(const LaneInput& in) {
  Packed<XT> p;
  if constexpr (XT == HQ_BF16) {
    p.w[0] = in.a.x ^ in.sw.x;
    p.w[1] = in.a.y ^ in.sw.y;
    p.w[2] = in.a.z ^ in.sw.z;
    p.w[3] = in.a.w ^ in.sw.w;
  } else {
    const uint32_t w8[8] = {in.a.x, in.a.y, in.a.z, in.a.w, in.b.x, in.b.y, in.b.z, in.b.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) p.w[i] = w8[i] ^ (((in.sw.x >> i) & 1u) << 31);
  }
  return p;
}

template <int XT>
__device__ __forceinline__ void unpack(const Packed<XT>& p, float* x) {
  if constexpr (XT == HQ_BF16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(p.w[i] << 16);
      x[2 * i + 1] = __uint_as_float(p.w[i] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = __uint_as_float(p.w[i]);
  }
}

// The tile's sum of squares: a pairwise tree in index order (the lane
// butterflies 1, 2, 4, 8 add the same pairs in the same order).
template <int XT>
__device__ __forceinline__ float tile_sumsq(const Packed<XT>& p) {
  float x[8], sq[8];
  unpack<XT>(p, x);
#pragma unroll
  for (int i = 0; i < 8; ++i) sq[i] = x[i] * x[i];
  float ss = tree8(sq);
  ss = ss + dpp_xor<1>(ss);
  ss = ss + dpp_xor<2>(ss);
  ss = ss + swz_xor4(ss);
  ss = ss + dpp_xor<8>(ss);
  return ss;
}

// Value of lane (l & ~3) | I for every lane l (a quad broadcast).
template <int I>
__device__ __forceinline__ float quad_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), I * 0x55, 0xF, 0xF, true));
}

// The lane's 8 remainder fields (k0 / k1 bits by class, packed in symbol
// order), ORed into the buffer at bit rpos.
template <int LAT>
__device__ __forceinline__ void put_remainders(uint32_t* buf, uint32_t rpos, const uint32_t (&sym)[8],
                                               uint32_t k0, uint32_t k1, uint32_t lrem) {
  if (lrem <= 32) {
    uint32_t acc = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t kk = sym_class<LAT>(j) ? k1 : k0;
      acc = lshl_or_s(sym[j] & ((1u << kk) - 1u), readfirst(rem_offset<LAT>(j, k0, k1)), acc);
    }
    or_word(buf, rpos, acc);
  } else if (lrem <= 64) {
    uint64_t acc = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t kk = sym_class<LAT>(j) ? k1 : k0;
      acc |= (uint64_t)(sym[j] & ((1u << kk) - 1u)) << rem_offset<LAT>(j, k0, k1);
    }
    or_bits64(buf, rpos, acc);
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t kk = sym_class<LAT>(j) ? k1 : k0;
      or_bits64(buf, rpos + rem_offset<LAT>(j, k0, k1), sym[j] & ((1u << kk) - 1u));
    }
  }
}

// The lane's 8 unary codes (q zeros and a one each, ulen bits in all),
// ORed into the buffer from bit upos.
__device__ __forceinline__ void put_unary(uint32_t* buf, uint32_t upos, const uint32_t (&qv)[8],
                                          uint32_t ulen) {
  if (ulen <= 32) {
    uint32_t m = 0, t = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      t += qv[j];
      m = bit_or(t, m);
      t += 1;
    }
    or_word(buf, upos, m);
  } else if (ulen <= 64) {
    uint64_t m = 0;
    uint32_t t = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      t += qv[j];
      m |= 1ull << t;
      t += 1;
    }
    or_bits64(buf, upos, m);
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      upos += qv[j];
      or_bits64(buf, upos, 1ull);
      upos += 1;
    }
  }
}

template <int LAT, int XT, bool KV>
__device__ __forceinline__ void encode_substream(const hq_encode_args& A, const hq_rice_thr& T,
                                                 const SubPos& P, int lane, float* x, float scale_tw,
                                                 uint32_t* buf, float* stage, uint32_t& W_out,
                                                 uint32_t& kb_out, uint32_t& bits_out,
                                                 bool& overflow_out) {
  const bool active = P.active;  // wave-uniform
  const uint32_t col = P.col0 + 8u * (uint32_t)lane;  // tile lane/16, coordinates 8 (lane % 16) + j
  const int64_t grow = A.first_row + P.lrow;
  const bool use_rot = KV && A.rotation == HQ_ROT_SIGNS;
  const bool use_dither = KV && A.dither;

  // ---- z = (sigma H D x) * (sigma alpha / r): the scale carries the sign sigma
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = x[i] * scale_tw;
  if (use_rot) {
    const uint32_t sbits = sign_bits8(A.smask, (lane & 15) * 8);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = flip(x[i], sbits, i);
  }
  // z <- S z, S^T read from global memory (a workgroup copy in LDS measured
  // 3x slower on the one-sub-stream-per-wave appends)
  if (KV && A.rotation == HQ_ROT_QJL) qjl_tile(A.qjlt, stage, lane, x);
  if (use_dither) {
    float u[8];
    dither8<LAT>(A.dither_seed, grow, col, u);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = x[i] + (LAT == kE8 ? 0.5f * u[i] : u[i]);
  }

  // ---- quantize + strip
  uint32_t sym[8];
  bool huge = false;
  if constexpr (LAT == kE8) {
    int32_t h[8], cb;  // c = 2 h + cb
    e8_nearest(x, h, cb);  // an inactive sub-stream's symbols are never written
    e8_strip(h, cb, sym);
  } else {
    int32_t c[8];
    quantize8<LAT>(x, c);
#pragma unroll
    for (int i = 0; i < 8; ++i) huge = huge || (c[i] > 65536 || c[i] < -65536);
    if (huge || !active) {
#pragma unroll
      for (int i = 0; i < 8; ++i) c[i] = 0;
    }
    strip8<LAT>(c, sym);
  }

  // ---- Rice parameters (wave-uniform), quotients and the unary-length scan
  uint32_t k0, k1, qv[8], ulen, uincl = 0;  // uincl: set by the k* scan or below
  bool scanned = false;
  if constexpr (LAT == kE8 || LAT == kZ) {
    uint32_t s0 = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) s0 += sym[j];
    if (A.rice_k >= 0) {
      k0 = (uint32_t)A.rice_k;
      ulen = 8;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        qv[j] = sym[j] >> k0;
        ulen += qv[j];
      }
    } else {
      const uint32_t a0 = kstar_count(wave_total(s0), T.thr0);
      // the better of k* and k* + 1: k* + 1 saves sum((m >> k) - (m >> (k+1)))
      // unary bits and costs one remainder bit per symbol.  Both candidates'
      // unary-length scans run in one pass; their totals give that saving,
      // and the chosen one's scan places the codes.
      uint32_t ga = 0, gb = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        qv[j] = sym[j] >> a0;
        ga += qv[j];
        gb += qv[j] >> 1;
      }
      uint32_t ia = 8 + ga, ib = 8 + gb;
      wave_scan_incl2(ia, ib);
      const uint32_t Ua = __builtin_amdgcn_readlane(ia, 63), Ub = __builtin_amdgcn_readlane(ib, 63);
      const uint32_t d = (a0 < HQ_KMAX && Ua - Ub > (uint32_t)HQ_SUB) ? 1u : 0u;
      k0 = a0 + d;
#pragma unroll
      for (int j = 0; j < 8; ++j) qv[j] >>= d;
      ulen = 8 + (d ? gb : ga);
      uincl = d ? ib : ia;
      scanned = true;
    }
    k1 = k0;
  } else {
    if (A.rice_k >= 0) {
      k0 = (uint32_t)A.rice_k;
      k1 = (LAT == kD4) ? (k0 > 0 ? k0 - 1 : 0) : k0;
    } else {
      uint32_t s0 = 0, s1 = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (sym_class<LAT>(j)) s1 += sym[j]; else s0 += sym[j];
      }
      const uint32_t a0 = kstar_count(wave_total(s0), T.thr0);
      const uint32_t a1 = (LAT == kA2) ? kstar_count(wave_total(s1), T.thr1) : 0u;
      const uint32_t b0 = a0 < HQ_KMAX ? a0 + 1 : a0;
      const uint32_t b1 = a1 < HQ_KMAX ? a1 + 1 : a1;
      uint32_t g0 = 0, g1 = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (LAT == kD4) {
          const uint32_t ka = sym_class<LAT>(j) ? (a0 > 0 ? a0 - 1 : 0) : a0;
          const uint32_t kb = sym_class<LAT>(j) ? (b0 > 0 ? b0 - 1 : 0) : b0;
          g0 += (sym[j] >> ka) - (sym[j] >> kb);
        } else if (sym_class<LAT>(j)) {
          g1 += (sym[j] >> a1) - (sym[j] >> b1);
        } else {
          g0 += (sym[j] >> a0) - (sym[j] >> b0);
        }
      }
      const uint32_t gain0 = wave_total(g0);
      uint32_t cost0;
      if (LAT == kD4) {
        cost0 = (b0 - a0) * (3u * HQ_SUB / 4u) +
                ((b0 > 0 ? b0 - 1 : 0) - (a0 > 0 ? a0 - 1 : 0)) * (HQ_SUB / 4u);
      } else {
        cost0 = (b0 - a0) * (HQ_SUB / 2u);
      }
      k0 = gain0 > cost0 ? b0 : a0;
      if (LAT == kA2) {
        const uint32_t gain1 = wave_total(g1);
        k1 = gain1 > (b1 - a1) * (HQ_SUB / 2u) ? b1 : a1;
      } else {
        k1 = k0 > 0 ? k0 - 1 : 0;
      }
    }
    ulen = 8;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      qv[j] = sym[j] >> (sym_class<LAT>(j) ? k1 : k0);
      ulen += qv[j];
    }
  }

  // ---- code lengths: remainder region then unary region
  const uint32_t lrem = lane_rem_bits<LAT>(k0, k1);
  const uint32_t R = 64 * lrem;
  if (!scanned) uincl = wave_scan_incl(ulen);
  const uint32_t U = __builtin_amdgcn_readlane(uincl, 63);
  const uint32_t uoff = uincl - ulen;
  uint32_t W = (R + U + 31) >> 5;
  // A sub-stream that does not fit the plan's bound (only non-finite or
  // out-of-range input can do that) is written as all-zero symbols with
  // k = 0: 512 unary terminators, 16 words.
  const bool overflow = active && W > A.lds_words;
  if (!active) W = 0;
  if (overflow) W = HQ_SUB / 32;

  // ---- assemble in this sub-stream's LDS buffer (two spare words past W
  //      take the zero high halves of the ORs)
  for (uint32_t w = lane; w < W; w += 64) buf[w] = overflow ? 0xFFFFFFFFu : 0u;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  if (active && !overflow) {
    // remainder fields, packed per lane
    put_remainders<LAT>(buf, __umul24((uint32_t)lane, lrem), sym, k0, k1, lrem);  // lrem < 2^24
    // unary codes
    put_unary(buf, R + uoff, qv, ulen);
  }
  W_out = W;
  kb_out = overflow ? 0u : (LAT == kA2 ? (k0 | (k1 << 4)) : k0);
  bits_out = overflow ? (uint32_t)HQ_SUB : R + U;
  overflow_out = overflow;
}

// One sub-stream of B consecutive 512-symbol blocks (S = 512 B, weight
// plans): x[b] holds block b's transformed values and scl[b] its tile scale.
// Every block is quantized and stripped first; the Rice parameters then
// follow from the whole sub-stream's symbols (the sums and the k* / k* + 1
// decision taken over all S symbols), and the split layout places the S
// remainder fields (block b's at bit b 64 lrem) before the S unary codes
// (block b's after the unary bits of blocks 0 .. b - 1).
template <int LAT, int B>
__device__ __forceinline__ void encode_multiblock(const hq_encode_args& A, const hq_rice_thr& T,
                                                  bool active, int lane, float (*x)[8],
                                                  const float* scl, uint32_t tsig, uint32_t* buf,
                                                  uint32_t& W_out, uint32_t& kb_out,
                                                  uint32_t& bits_out, bool& overflow_out) {
  constexpr uint32_t S = (uint32_t)HQ_SUB * B;
  uint32_t sym[B][8];
#pragma unroll
  for (int b = 0; b < B; ++b) {
    float z[8];
    const float sc = xor_sign(scl[b], tsig);
#pragma unroll
    for (int i = 0; i < 8; ++i) z[i] = x[b][i] * sc;
    if constexpr (LAT == kE8) {
      int32_t h[8], cb;
      e8_nearest(z, h, cb);
      e8_strip(h, cb, sym[b]);
    } else {
      int32_t c[8];
      quantize8<LAT>(z, c);
      bool huge = false;
#pragma unroll
      for (int i = 0; i < 8; ++i) huge = huge || (c[i] > 65536 || c[i] < -65536);
      if (huge || !active) {
#pragma unroll
        for (int i = 0; i < 8; ++i) c[i] = 0;
      }
      strip8<LAT>(c, sym[b]);
    }
  }
  // ---- Rice parameters over the whole sub-stream (wave-uniform)
  uint32_t k0, k1;
  if (A.rice_k >= 0) {
    k0 = (uint32_t)A.rice_k;
    k1 = (LAT == kD4) ? (k0 > 0 ? k0 - 1 : 0) : k0;
  } else if constexpr (LAT == kE8 || LAT == kZ) {
    uint32_t s0 = 0;
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
      for (int j = 0; j < 8; ++j) s0 += sym[b][j];
    const uint32_t a0 = kstar_count(wave_total(s0), T.thr0);
    // k* + 1 saves sum((m >> k*) - (m >> (k* + 1))) unary bits for S remainder bits
    uint32_t g = 0;
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t q = sym[b][j] >> a0;
        g += q - (q >> 1);
      }
    k0 = (a0 < HQ_KMAX && wave_total(g) > S) ? a0 + 1 : a0;
    k1 = k0;
  } else {
    uint32_t s0 = 0, s1 = 0;
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (sym_class<LAT>(j)) s1 += sym[b][j]; else s0 += sym[b][j];
      }
    const uint32_t a0 = kstar_count(wave_total(s0), T.thr0);
    const uint32_t a1 = (LAT == kA2) ? kstar_count(wave_total(s1), T.thr1) : 0u;
    const uint32_t b0 = a0 < HQ_KMAX ? a0 + 1 : a0;
    const uint32_t b1 = a1 < HQ_KMAX ? a1 + 1 : a1;
    uint32_t g0 = 0, g1 = 0;
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t m = sym[b][j];
        if (LAT == kD4) {
          const uint32_t ka = sym_class<LAT>(j) ? (a0 > 0 ? a0 - 1 : 0) : a0;
          const uint32_t kb = sym_class<LAT>(j) ? (b0 > 0 ? b0 - 1 : 0) : b0;
          g0 += (m >> ka) - (m >> kb);
        } else if (sym_class<LAT>(j)) {
          g1 += (m >> a1) - (m >> b1);
        } else {
          g0 += (m >> a0) - (m >> b0);
        }
      }
    const uint32_t gain0 = wave_total(g0);
    // one more remainder bit on each symbol of the class (D4: 3 S / 4 of
    // class 0, S / 4 of class 1; A2: S / 2 each)
    const uint32_t cost0 = (LAT == kD4)
                               ? (b0 - a0) * (3u * S / 4u) +
                                     ((b0 > 0 ? b0 - 1 : 0) - (a0 > 0 ? a0 - 1 : 0)) * (S / 4u)
                               : (b0 - a0) * (S / 2u);
    k0 = gain0 > cost0 ? b0 : a0;
    if (LAT == kA2) {
      const uint32_t gain1 = wave_total(g1);
      k1 = gain1 > (b1 - a1) * (S / 2u) ? b1 : a1;
    } else {
      k1 = k0 > 0 ? k0 - 1 : 0;
    }
  }
  // ---- code lengths: the B remainder regions, then the B unary regions
  const uint32_t lrem = lane_rem_bits<LAT>(k0, k1);
  const uint32_t Rb = 64 * lrem, Rt = (uint32_t)B * Rb;
  uint32_t ulen[B], uincl[B], U = 0;
#pragma unroll
  for (int b = 0; b < B; ++b) {
    ulen[b] = 8;
#pragma unroll
    for (int j = 0; j < 8; ++j) ulen[b] += sym[b][j] >> (sym_class<LAT>(j) ? k1 : k0);
    uincl[b] = wave_scan_incl(ulen[b]);
    U += __builtin_amdgcn_readlane(uincl[b], 63);
  }
  uint32_t W = (Rt + U + 31) >> 5;
  // a sub-stream past the plan's bound is written as S zero symbols with k = 0
  const bool overflow = active && W > A.lds_words;
  if (!active) W = 0;
  if (overflow) W = S / 32;
  for (uint32_t w = lane; w < W; w += 64) buf[w] = overflow ? 0xFFFFFFFFu : 0u;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  if (active && !overflow) {
    uint32_t ubase = Rt;  // where block b's unary codes begin
#pragma unroll
    for (int b = 0; b < B; ++b) {
      uint32_t qv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) qv[j] = sym[b][j] >> (sym_class<LAT>(j) ? k1 : k0);
      put_remainders<LAT>(buf, (uint32_t)b * Rb + __umul24((uint32_t)lane, lrem), sym[b], k0, k1, lrem);
      put_unary(buf, ubase + uincl[b] - ulen[b], qv, ulen[b]);
      ubase += __builtin_amdgcn_readlane(uincl[b], 63);
    }
  }
  W_out = W;
  kb_out = overflow ? 0u : (LAT == kA2 ? (k0 | (k1 << 4)) : k0);
  bits_out = overflow ? S : Rt + U;
  overflow_out = overflow;
}

// TILED: a plan whose tile is not 128 (weights only: no rotation or
// dither); the wave takes four consecutive sub-streams, so that every tile
// of up to 2048 scalars lies inside one wave.
template <int LAT, int XT, bool KV, int SPW, bool TILED = false, int MB = 1>
__device__ __forceinline__ void encode_wg(const hq_encode_args& A, const hq_rice_thr& T,
                                          const uint32_t wg) {
  static_assert(SPW == 1 || SPW == 4, "one or four sub-streams per wave");
  static_assert(!TILED || (SPW == 4 && !KV), "long tiles: four sub-streams per wave, weights");
  static_assert(MB == 1 || (TILED && (MB == 2 || MB == 4)), "multi-block sub-streams: long-tile front end");
  constexpr int NSUB = HQ_ENC_SUBS_PER_WG;  // sub-streams per workgroup
  constexpr int WAVES = NSUB / SPW;         // wave64s per workgroup
  extern __shared__ uint32_t smem[];
  __shared__ uint32_t s_epoch;
  __shared__ uint32_t s_words[NSUB];
  __shared__ uint32_t s_pad[WAVES];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = (int)readfirst((uint32_t)(tid >> 6));
  const uint32_t stride = A.lds_words + 2;  // words per sub-stream buffer
  if (tid == 0)
    s_epoch = (uint32_t)__hip_atomic_load(A.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) &
              kEpochMask;
  const TwSigns sg(lane);
  // sub-streams of MB > 1 consecutive 512-symbol blocks (the long-tile
  // front end, any tile): positions below count blocks
  constexpr uint32_t mb = (uint32_t)MB;
  const uint32_t nblk = (uint32_t)A.nsub * mb;

  // ---- this wave's sub-streams: wg * NSUB + i * WAVES + wave, i < SPW (row and
  //      column advanced on scalar registers)
  SubPos pos[SPW];
  {
    const uint32_t spr = (uint32_t)A.spr * mb;
    const uint32_t step = TILED ? 1u : (uint32_t)WAVES;
    const uint32_t sub0 = wg * NSUB + (uint32_t)wave * (TILED ? (uint32_t)SPW : 1u);
    uint32_t row = sub0 / spr, c = sub0 - row * spr;
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      pos[i].active = sub0 + (uint32_t)i * step < nblk;
      pos[i].lrow = pos[i].active ? row : 0u;
      pos[i].col0 = pos[i].active ? c * HQ_SUB : 0u;
      c += step;
      while (c >= spr) {
        c -= spr;
        ++row;
      }
    }
  }
  Packed<XT> pk[SPW];
  float ss[SPW];
  bool nonfinite = false;
  float xt[TILED ? SPW : 1][8];  // long tiles: the transformed values of the wave
  uint32_t tsig = 0;             // long tiles: the sign bit of the lane's sigma
  if constexpr (TILED) {
    // ---- long tiles: every load first, then each 128-block's sum of squares
    //      (tree8 and the lane butterflies 1, 2, 4, 8), widened to the tile
    //      by lanes l ^ 16, l ^ 32 and then across sub-streams, in the
    //      pairwise tree's order
    const uint32_t n = (uint32_t)A.tile;
#pragma unroll
    for (int i = 0; i < SPW; ++i) unpack<XT>(pack_signed<XT>(load_lane_input<XT>(A, pos[i], lane)), xt[i]);
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      float sq[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) sq[j] = xt[i][j] * xt[i][j];
      float v = tree8(sq);
      v = v + dpp_xor<1>(v);
      v = v + dpp_xor<2>(v);
      v = v + swz_xor4(v);
      v = v + dpp_xor<8>(v);
      if (n >= 256u) v = v + swz_xor16(v);
      if (n >= 512u) v = v + lane_xor32(v);
      ss[i] = v;
    }
    if (n >= 1024u) {
      const float a = ss[0] + ss[1], b = ss[2] + ss[3];
      ss[0] = a; ss[1] = a; ss[2] = b; ss[3] = b;
    }
    if (n >= 2048u) {
      const float a = ss[0] + ss[2];
      ss[0] = a; ss[1] = a; ss[2] = a; ss[3] = a;
    }
    // ---- norms and scales: every lane its own tile's; the lane holding a
    //      tile's first coordinate stores the norm
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const float r = __builtin_sqrtf(ss[i]);
      const bool bad = !(r <= 3.0e38f);  // an infinite or NaN input
      nonfinite = nonfinite || bad;
      ss[i] = (r == 0.0f || bad) ? 0.0f : (LAT == kE8 ? A.alpha_half : A.alpha) / r;
      const uint32_t sub = wg * NSUB + (uint32_t)(wave * SPW + i);
      const uint64_t flat = (uint64_t)sub * HQ_SUB + 8u * (uint32_t)lane;
      if (pos[i].active && (flat & (n - 1u)) == 0u) {
        ((float*)A.norms)[A.first_row * A.tpr + (int64_t)(flat / n)] = r;
        if (bad && A.stats) {
          atomicAdd(&A.stats->overflow_tiles, 1u);
          atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_OVERFLOW);
        }
      }
    }
    if (__ballot(nonfinite) != 0ull) {
#pragma unroll
      for (int i = 0; i < SPW; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) xt[i][j] = ss[i] == 0.0f ? 0.0f : xt[i][j];
    }
    tsig = fwht_tiled(xt, lane, n, sg);
  } else {
  // ---- every input load of the wave's sub-streams is issued first; each is
  //      kept packed with its signs applied, and its tile sums of squares
  //      taken (the transforms wait until each sub-stream is coded)
#pragma unroll
  for (int i = 0; i < SPW; ++i) pk[i] = pack_signed<XT>(load_lane_input<XT>(A, pos[i], lane));
#pragma unroll
  for (int i = 0; i < SPW; ++i) ss[i] = tile_sumsq<XT>(pk[i]);

  // ---- tile norms and scales, once for the wave's tiles: with four
  //      sub-streams lane l takes sub-stream i = l & 3, tile t = l >> 4 (each
  //      tile's 16 lanes hold its sum of squares, so the merged value repeats
  //      in every quad); with one, every lane takes its own tile l >> 4
  {
    const int qi = SPW == 4 ? (lane & 3) : 0;
    float ssm = ss[0];
    if constexpr (SPW == 4) ssm = qi == 0 ? ss[0] : (qi == 1 ? ss[1] : (qi == 2 ? ss[2] : ss[3]));
    const bool fp16_norm = KV && A.norm_fp16;
    const float r = __builtin_sqrtf(ssm);
    float rs = r;
    nonfinite = !(r <= 3.0e38f);  // an infinite or NaN input (r is at most 2^64 otherwise)
    bool bad_tile = nonfinite;
    if (fp16_norm) {
      rs = (float)(_Float16)r;
      bad_tile = bad_tile || !(rs <= 65504.0f);
    }
    // E8 decides on z / 2: its scale is (alpha / 2) / r_s, exactly half of alpha / r_s
    const float scale =
        (rs == 0.0f || bad_tile) ? 0.0f : (LAT == kE8 ? A.alpha_half : A.alpha) / rs;
    const uint32_t sub_l = wg * NSUB + (uint32_t)(qi * WAVES + wave);
    const bool writer = SPW == 4 ? ((lane >> 2) & 3) == 0 : (lane & 15) == 0;
    if (writer && sub_l < (uint32_t)A.nsub) {
      // tile (lane >> 4) of sub-stream sub_l: 4 tiles per sub-stream, rows contiguous
      const int64_t t = A.first_row * A.tpr + 4 * (int64_t)sub_l + (lane >> 4);
      if (fp16_norm) {
        ((_Float16*)A.norms)[t] = (_Float16)r;
      } else {
        ((float*)A.norms)[t] = r;
      }
      if (bad_tile && A.stats) {
        atomicAdd(&A.stats->overflow_tiles, 1u);
        atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_OVERFLOW);
      }
    }
    if constexpr (SPW == 4) {
      ss[0] = quad_bcast<0>(scale);
      ss[1] = quad_bcast<1>(scale);
      ss[2] = quad_bcast<2>(scale);
      ss[3] = quad_bcast<3>(scale);
    } else {
      ss[0] = scale;
    }
  }
  // A non-finite tile has scale 0 and is coded as if its transform were
  // zero (its values would turn the product into NaN); zero tiles, the other
  // tiles with scale 0, hold zeros already.
  if (__ballot(nonfinite) != 0ull) {
#pragma unroll
    for (int i = 0; i < SPW; ++i)
#pragma unroll
      for (int j = 0; j < (XT == HQ_BF16 ? 4 : 8); ++j) pk[i].w[j] = ss[i] == 0.0f ? 0u : pk[i].w[j];
  }
  }  // 128-tiles

  // ---- quantize and Rice-code each sub-stream into its LDS buffer
  uint32_t padsum = 0;
  if constexpr (MB > 1) {
    // sub-streams of MB blocks: the wave's four blocks are 4 / MB of them,
    // sub-stream ls of the group in buffer ls (s_words past the group's
    // 16 / MB sub-streams stay 0)
    constexpr uint32_t ns = (uint32_t)NSUB / MB;
    if (lane == 0 && wave == 0)
      for (uint32_t q = ns; q < (uint32_t)NSUB; ++q) s_words[q] = 0;
#pragma unroll
    for (int j = 0; j < SPW / MB; ++j) {
      const uint32_t ls = (uint32_t)wave * (uint32_t)(SPW / MB) + (uint32_t)j;
      const uint32_t gs = wg * ns + ls;
      const bool act = pos[j * MB].active;
      uint32_t W, kb, bits;
      bool ovf;
      encode_multiblock<LAT, MB>(A, T, act, lane, xt + j * MB, ss + j * MB, tsig, smem + ls * stride,
                                 W, kb, bits, ovf);
      if (act) {
        if (lane == 0) {
          A.kparam[A.first_sub + gs] = (uint8_t)kb;
          s_words[ls] = W;
          if (ovf && A.stats) atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_OVERFLOW);
        }
        padsum += W * 32u - bits;
      } else if (lane == 0) {
        s_words[ls] = 0;
      }
    }
  } else
#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    // 128-tiles: neighbouring waves take neighbouring sub-streams
    const int li = TILED ? wave * SPW + i : i * WAVES + wave;
    const uint32_t sub = wg * NSUB + (uint32_t)li;
    uint32_t W, kb, bits;
    bool ovf;
    float x[8];  // x <- sigma H D x
    if constexpr (TILED) {
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = xt[i][j];
    } else {
      unpack<XT>(pk[i], x);
      fwht128_tw(x, sg);
    }
    encode_substream<LAT, XT, KV>(A, T, pos[i], lane, x, xor_sign(ss[i], TILED ? tsig : sg.sigma),
                                  smem + li * stride,
                                  (float*)(smem + NSUB * stride) + wave * HQ_QJL_STAGE, W, kb,
                                  bits, ovf);
    if (pos[i].active) {
      if (lane == 0) {
        A.kparam[A.first_sub + sub] = (uint8_t)kb;
        s_words[li] = W;
        if (ovf && A.stats) atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_OVERFLOW);
      }
      padsum += W * 32u - bits;
    } else if (lane == 0) {
      s_words[li] = 0;
    }
  }
  if (lane == 0) {
    s_pad[wave] = padsum;
  }
  __syncthreads();
  // The other waves are done: their slots go to the next workgroups while wave 0
  // alone waits for the group's offset and writes every sub-stream out.
  // (No workgroup barrier follows.)
  if (wave != 0) return;

  const uint32_t epoch = readfirst(s_epoch);
  // ---- publish this group's word count at once, so successors can pass it;
  //      the group's pad bits go to its stats word first (packed as
  //      words << 11 | pad: at most 2^19 words and 64 * 31 pad bits)
  static_assert(NSUB <= 64, "one sub-stream word count per lane");
  const uint32_t agg = wave_total(lane < NSUB ? s_words[lane] : 0u);
  if (lane == 0) {
    if (A.stats) {
      uint32_t gp = 0;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) gp += s_pad[w];
      store_status(&A.wgstat[wg], pack_status(epoch, 1u, (agg << 11) | gp));
    }
    if (wg > 0) store_status(&A.status[wg], pack_status(epoch, 1u, agg));
  }

  // ---- look-back: 256 predecessors per round trip, until the nearest
  //      published inclusive prefix
  uint32_t prefix = 0;
  bool timed_out = false;
  for (int64_t hi = (int64_t)wg - 1; hi >= 0; hi -= 256)
    if (lookback_round<4>(A.status, hi, epoch, lane, prefix, timed_out)) break;
  // an append to an empty stream starts at word 0, like a fresh encode
  const unsigned long long base =
      (A.first_sub > 0 ? (unsigned long long)readfirst(A.offsets[A.first_sub]) : 0ull) + prefix;
  if (lane == 0) {
    store_status(&A.status[wg], pack_status(epoch, 2u, prefix + agg));
    // the last group: every group has read this launch's epoch; advance it
    if (wg == A.nwg - 1)
      __hip_atomic_store(A.epoch, (unsigned long long)((epoch + 1u) & kEpochMask), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    if (timed_out && A.stats) atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_HIP);
  }

  // ---- write payload and offsets of all of the group's sub-streams: lane
  //      l < NSUB takes sub-stream l's word count (0 when inactive) and its
  //      prefix inside the group; then 16 lanes per sub-stream copy four
  //      sub-streams at a time, every load of a lane issued before its stores
  static_assert(NSUB <= 16, "one row of lanes holds the group's word counts");
  {
    const uint32_t wl = lane < NSUB ? s_words[lane] : 0u;
    uint32_t il = wl;  // inclusive prefix inside the first row of 16 lanes
    il += dpp<kDppRowShr1, 0xF, 0xF, true>(0u, il);
    il += dpp<kDppRowShr2, 0xF, 0xF, true>(0u, il);
    il += dpp<kDppRowShr4, 0xF, 0xF, true>(0u, il);
    il += dpp<kDppRowShr8, 0xF, 0xF, true>(0u, il);
    const uint32_t xl = il - wl;
    const uint32_t ns = (uint32_t)NSUB / mb;  // sub-streams per group
    const uint32_t sub_l = wg * ns + (uint32_t)lane;
    if ((uint32_t)lane < ns && sub_l < (uint32_t)A.nsub) {
      const unsigned long long end = base + il;
      if (sub_l == 0 && A.first_sub == 0) A.offsets[0] = 0u;
      A.offsets[A.first_sub + sub_l + 1] = (uint32_t)end;
      if (end > (unsigned long long)A.cap_words && A.stats)
        atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_CAPACITY);
    }
#pragma unroll
    for (int r = 0; r < NSUB / 4; ++r) {
      const int li = 4 * r + (lane >> 4);
      const uint32_t W = (uint32_t)__shfl((int)wl, li);
      const unsigned long long st = base + (uint32_t)__shfl((int)xl, li);
      if (st + W > (unsigned long long)A.cap_words) continue;  // reported above
      const uint32_t* buf = smem + li * stride;
      for (uint32_t j = (uint32_t)(lane & 15); j < W; j += 64) {
        uint32_t v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = j + 16u * u < W ? buf[j + 16u * u] : 0u;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (j + 16u * u < W) A.payload[st + j + 16u * u] = v[u];
      }
    }
  }
  // ---- bit counts: the last group of every 256 adds up their stats words
  //      (all of them were stored before their owners' aggregates, which this
  //      group's look-back has passed), so the stats block takes one atomic
  //      per 256 groups instead of one per group
  if (A.stats && ((wg & 255u) == 255u || wg == A.nwg - 1)) {
    uint32_t gw = 0, gp = 0;  // words, pad bits
    bool late = false;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint32_t idx = (wg & ~255u) + (uint32_t)(r * 64 + lane);
      if (idx > wg) continue;
      uint32_t spins = 0;
      for (;;) {
        const unsigned long long st = load_status(&A.wgstat[idx]);
        if ((uint32_t)(st >> 34) == epoch && ((st >> 32) & 3u) != 0u) {
          gw += (uint32_t)st >> 11;
          gp += (uint32_t)st & 2047u;
          break;
        }
        if (++spins > kSpinLimit) {
          late = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    const uint32_t tw = wave_total(gw), tp = wave_total(gp);  // < 2^27 words, < 2^19 pad bits
    if (late) atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_HIP);
    if (lane == 0) {
      atomicAdd(&A.stats->payload_bits, 32ull * tw - tp);
      atomicAdd(&A.stats->pad_bits, (unsigned long long)tp);
    }
  }
}

template <int LAT, int XT, bool KV, int SPW>
__global__ __launch_bounds__(64 * HQ_ENC_SUBS_PER_WG / SPW) void hq_encode_kernel(hq_encode_args A,
                                                                                hq_rice_thr T) {
  encode_wg<LAT, XT, KV, SPW>(A, T, blockIdx.x);
}

// MB: 512-symbol blocks per sub-stream (1, or 2 / 4 for S = 1024 / 2048)
template <int LAT, int XT, int MB>
__global__ __launch_bounds__(64 * HQ_ENC_WAVES) void hq_encode_tiled_kernel(hq_encode_args A,
                                                                           hq_rice_thr T) {
  encode_wg<LAT, XT, false, HQ_ENC_SUBS_PER_WAVE, true, MB>(A, T, blockIdx.x);
}

// Several matrices in one launch: workgroups wg_begin[i] .. wg_begin[i+1]-1
// encode member i (its own stream, scan scratch and epoch), so small
// matrices share the machine instead of each filling only part of it.
template <int LAT, int XT, bool KV>
__global__ __launch_bounds__(64 * HQ_ENC_WAVES) void hq_encode_group_kernel(hq_encode_group_args G) {
  int mi = 0;
  for (int i = 1; i < G.count; ++i) mi = blockIdx.x >= G.wg_begin[i] ? i : mi;
  encode_wg<LAT, XT, KV, HQ_ENC_SUBS_PER_WAVE>(G.m[mi], G.thr, blockIdx.x - G.wg_begin[mi]);
}

// ------------------------------------------------------------ decode kernel
// Rice decode of one sub-stream per wave: the remainder fields are at fixed
// positions; the unary terminators are located by per-word popcounts, a
// wave prefix sum and a select inside the word that holds terminator 8 l - 1.
// Lane l then reads its 8 codes from a 32-bit window at that position (the
// common case: its codes span at most 32 bits), clearing one terminator per
// code; a lane whose codes run past the window walks a 64-bit window that
// slides along the bit array.  Each wave only touches its own LDS region.
// MODE 0: fp32 out, 1: bf16 out, 2: int8 lattice codes and per-tile g (no
// inverse RHT).

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Bits [pos, pos + 32) of the LDS bit array (the word after the last one
// read must exist).
__device__ __forceinline__ uint32_t bits32_at(const uint32_t* buf, uint32_t pos) {
  const uint32_t w = pos >> 5;
  return __builtin_amdgcn_alignbit(buf[w + 1], buf[w], pos & 31u);
}

// One sub-stream's table entry, checked against the buffers, and its first
// 128 payload words (two per lane): loaded one sub-stream ahead of its decode.
struct DecHead {
  uint32_t start, kb, W, R;  // wave-uniform
  bool ok;                   // entry within bounds (wave-uniform)
  uint32_t w0, w1;           // payload words lane and lane + 64
};

template <int LAT>
__device__ __forceinline__ DecHead dec_head(const hq_decode_args& A, bool active, uint32_t start,
                                            uint32_t end, uint32_t kb, int lane) {
  DecHead h;
  const uint32_t k0 = (LAT == kA2) ? (kb & 15u) : kb;
  const uint32_t k1 = (LAT == kA2) ? (kb >> 4) : (LAT == kD4 ? (k0 > 0 ? k0 - 1 : 0) : k0);
  h.start = start;
  h.kb = kb;
  h.W = end - start;
  h.R = 64 * lane_rem_bits<LAT>(k0, k1);
  h.ok = active && end >= start && (int64_t)end <= A.cap_words && h.W <= A.lds_words &&
         k0 <= HQ_KMAX && h.R <= 32u * h.W;
  const uint32_t Wl = h.ok ? h.W : 0u;
  h.w0 = (uint32_t)lane < Wl ? A.payload[(uint64_t)start + lane] : 0u;
  h.w1 = (uint32_t)lane + 64u < Wl ? A.payload[(uint64_t)start + 64u + lane] : 0u;
  return h;
}

template <int LAT>
__device__ __forceinline__ bool decode_symbols(const hq_decode_args& A, const DecHead& h, int lane,
                                               uint32_t* buf, uint32_t* starts,
                                               const uint32_t* seltbl, uint32_t* sym) {
  const uint32_t kb = h.kb;
  const uint32_t k0 = (LAT == kA2) ? (kb & 15u) : kb;
  const uint32_t k1 = (LAT == kA2) ? (kb >> 4) : (LAT == kD4 ? (k0 > 0 ? k0 - 1 : 0) : k0);
  const uint32_t lrem = lane_rem_bits<LAT>(k0, k1);
  const uint32_t R = h.R;
  bool ok = h.ok;
  const uint32_t Wl = ok ? h.W : 0u;
  if ((uint32_t)lane < Wl) buf[lane] = h.w0;
  if ((uint32_t)lane + 64u < Wl) buf[lane + 64] = h.w1;
  for (uint32_t w = 128u + lane; w < Wl; w += 64) buf[w] = A.payload[(uint64_t)h.start + w];
  if (lane < 2) buf[Wl + lane] = 0u;  // two zero words past the end
  starts[lane] = (lane == 0) ? R : 0xFFFFFFFFu;
  wave_sync_lds();

  // unary terminators: popcount prefix over the unary words, then the start
  // of each lane's codes (just past terminator 8 l - 1)
  const uint32_t uw0 = R >> 5;
  const uint32_t nuw = ok ? Wl - uw0 : 0u;
  uint32_t pos;
  if (nuw <= 64u) {
    // one word per lane: word w holds terminators excl_w .. incl_w - 1, and
    // lane l >= 1 starts just past terminator 8 l - 1, so word w is the
    // start word of lanes l in [(excl_w + 8) / 8, incl_w / 8] (at most four,
    // a word holding at most 32 terminators).  Each word's lane writes its
    // index and excl_w into those lanes' slots; each lane then reads its own
    // and selects inside that word.  A lane past the last terminator (8 l >
    // the total) gets no slot and reports a corrupt sub-stream.
    const uint32_t v = ((uint32_t)lane < nuw) ? buf[uw0 + lane] : 0u;
    const uint32_t cnt = __popc(v);
    const uint32_t incl = wave_scan_incl(cnt);
    const uint32_t total = __builtin_amdgcn_readlane(incl, 63);
    const uint32_t excl = incl - cnt;
    const uint32_t llo = (excl + 8u) >> 3, lhi = incl >> 3;
    const uint32_t entry = (uint32_t)lane | (excl << 8);
#pragma unroll
    for (uint32_t i = 0; i < 4; ++i)
      if (llo + i <= lhi && llo + i < 64u) starts[llo + i] = entry;
    wave_sync_lds();
    const uint32_t target = 8u * (uint32_t)lane;  // terminators before this lane's codes
    if (lane == 0) {
      pos = R;
    } else {
      ok = ok && target <= total;
      const uint32_t e = ok ? starts[lane] : 0u;
      const uint32_t w = e & 0xFFu;
      const uint32_t word = ok ? buf[uw0 + w] : 0u;
      pos = ok ? (uw0 + w) * 32u + select32_lut(word, target - 1u - (e >> 8), seltbl) + 1u : 0u;
    }
  } else {
    uint32_t carry = 0;
    for (uint32_t base = 0; base < nuw; base += 64) {
      const uint32_t wi = base + lane;
      const uint32_t v = (wi < nuw) ? buf[uw0 + wi] : 0u;
      const uint32_t cnt = __popc(v);
      const uint32_t incl = wave_scan_incl(cnt);
      const uint32_t P = carry + incl - cnt;
      for (uint32_t t = (P & ~7u) + 7u; t < P + cnt; t += 8u) {
        const uint32_t j = (t + 1u) >> 3;
        if (j < 64u) starts[j] = (uw0 + wi) * 32u + select32(v, t - P) + 1u;
      }
      carry += __builtin_amdgcn_readlane(incl, 63);
    }
    wave_sync_lds();
    pos = starts[lane];
  }

  // lane's 8 quotients
  const uint32_t nbits = 32u * Wl;
  ok = ok && pos < nbits;
  uint32_t qv[8];
  bool fast = false;
  if (ok) {
    // q_j = the zeros before the next terminator: shift the window past
    // each code (all 8 terminators lie inside it on this path, so every
    // shift is below 32; otherwise the values are discarded below)
    const uint32_t win = bits32_at(buf, pos);
    fast = __popc(win) >= 8;
    uint32_t sh = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      qv[j] = (uint32_t)__builtin_ctz(win >> sh);
      sh += qv[j] + 1u;
    }
  }
  if (ok && !fast) {
    // the codes run past 32 bits: a 64-bit window sliding along the array
    uint64_t win = load_bits64(buf, pos, Wl);
    uint32_t valid = 64;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      uint32_t q = 0;
      while (ok && win == 0ull) {
        q += valid;
        pos += valid;
        if (pos >= nbits) {
          ok = false;
          break;
        }
        win = load_bits64(buf, pos, Wl);
        valid = 64;
      }
      const uint32_t lo = (uint32_t)win, hi = (uint32_t)(win >> 32);
      const uint32_t tz =
          lo ? (uint32_t)__builtin_ctz(lo) : 32u + (uint32_t)__builtin_ctz(hi | (hi == 0u));
      q += tz;
      pos += tz + 1;
      valid -= tz + 1;
      win = (tz >= 63u) ? 0ull : (win >> (tz + 1));
      qv[j] = q;
    }
  }
  // lane's 8 remainders (fields at fixed positions)
  const uint32_t rpos = __umul24((uint32_t)lane, lrem);  // lrem < 2^24
  if (lrem <= 32) {
    const uint32_t acc = (ok && lrem) ? bits32_at(buf, rpos) : 0u;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t kk = sym_class<LAT>(j) ? k1 : k0;
      sym[j] = (qv[j] << kk) | __builtin_amdgcn_ubfe(acc, rem_offset<LAT>(j, k0, k1), kk);
    }
  } else if (lrem <= 64) {
    const uint64_t acc = ok ? ((uint64_t)bits32_at(buf, rpos + 32) << 32) | bits32_at(buf, rpos) : 0ull;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t kk = sym_class<LAT>(j) ? k1 : k0;
      const uint32_t r = (uint32_t)(acc >> rem_offset<LAT>(j, k0, k1)) & ((1u << kk) - 1u);
      sym[j] = (qv[j] << kk) | r;
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t kk = sym_class<LAT>(j) ? k1 : k0;
      const uint32_t r = ok ? (uint32_t)load_bits64(buf, rpos + rem_offset<LAT>(j, k0, k1), Wl) : 0u;
      sym[j] = (qv[j] << kk) | (r & ((1u << kk) - 1u));
    }
  }
  // a corrupt sub-stream (any lane's parse failed) decodes as all-zero
  // symbols in every lane; callers drop its factor too
  if (__ballot(!ok) != 0ull) {
#pragma unroll
    for (int j = 0; j < 8; ++j) sym[j] = 0u;
  }
  return ok;
}

// SPW consecutive sub-streams per wave: 4, or 1 for launches too small to
// fill the chip with four per wave.
template <int LAT, int MODE, bool KV, int SPW = HQ_DEC_SUBS_PER_WAVE>
__device__ __forceinline__ void decode_wg(const hq_decode_args& A, const uint32_t wgi) {
  extern __shared__ uint32_t smem[];
  __shared__ uint32_t s_sel[256];
  const int tid = threadIdx.x, lane = tid & 63;
  const uint32_t wave = readfirst((uint32_t)(tid >> 6));
  uint32_t* buf = smem + wave * (A.lds_words + 66);
  uint32_t* starts = buf + A.lds_words + 2;
  const bool use_rot = KV && A.rotation == HQ_ROT_SIGNS;
  const bool use_qjl = KV && A.rotation == HQ_ROT_QJL;
  const bool use_dither = KV && A.dither;
  const bool fp16_norm = KV && A.norm_fp16;
  // qjl: this wave's stage after the four buffers, then the workgroup's copy of S
  float* const qstage = (float*)(smem + HQ_WAVES_PER_WG * (A.lds_words + 66)) + wave * HQ_QJL_STAGE;
  float* const qmat = (float*)(smem + HQ_WAVES_PER_WG * (A.lds_words + 66)) +
                      HQ_WAVES_PER_WG * HQ_QJL_STAGE;
  if (use_qjl)
    for (int i = tid; i < HQ_TILE * HQ_TILE / 4; i += 256)
      ((float4*)qmat)[i] = ((const float4*)A.qjl)[i];
  s_sel[tid] = byte_select_entry((uint32_t)tid);  // 256 threads, one entry each
  __syncthreads();

  // this wave's sub-streams: SPW consecutive ones; their table entries are
  // read at once, each one's payload one sub-stream ahead
  const uint32_t sub0 = (wgi * HQ_WAVES_PER_WG + wave) * SPW;
  const uint32_t nsub = (uint32_t)A.nsub;
  uint32_t off[SPW + 1], kbs[SPW];
#pragma unroll
  for (int i = 0; i <= SPW; ++i) {
    const uint32_t sub = sub0 + (uint32_t)i;
    off[i] = sub <= nsub ? readfirst(A.offsets[(uint32_t)A.first_sub + sub]) : 0u;
    if (i < SPW)
      kbs[i] = sub < nsub ? readfirst(A.kparam[(uint32_t)A.first_sub + sub]) : 0u;
  }
  DecHead head = dec_head<LAT>(A, sub0 < nsub, off[0], off[1], kbs[0], lane);
  const uint32_t spr = (uint32_t)A.spr;
  const TwSigns sg(lane);
  const uint32_t sbits = use_rot ? sign_bits8(A.smask, (lane & 15) * 8) : 0u;
  // tile factors g = r_s / (alpha n), once for the wave's tiles: lane l
  // takes sub-stream l & 3 (SPW = 4) or the one sub-stream, and tile l >> 4
  // (rows are contiguous, 4 tiles per sub-stream); with four, sub-stream i
  // reads them back by a quad broadcast
  static_assert(SPW == 4 || SPW == 1, "one sub-stream per lane of a quad, or one per wave");
  float gm = 0.0f;
  {
    const uint32_t subq = sub0 + (SPW == 4 ? (uint32_t)(lane & 3) : 0u);
    if (subq < nsub) {
      // the casts (MODE >= 2) also serve long-tile weight plans: tile of the
      // 128 columns at flat position subq * 512 + 128 (lane >> 4)
      const int64_t t =
          MODE >= 2 ? A.first_row * A.tpr + (int64_t)((((uint64_t)subq << 9) + (uint64_t)((lane >> 4) << 7)) >>
                                                       __builtin_ctz((uint32_t)A.tile))
                    : A.first_row * A.tpr + 4 * (int64_t)subq + (lane >> 4);
      const float rs = fp16_norm ? (float)((const _Float16*)A.norms)[t] : ((const float*)A.norms)[t];
      gm = rs / A.alpha_n;
    }
  }

#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    const uint32_t sub = sub0 + (uint32_t)i;
    if (sub >= nsub) break;
    DecHead next;
    if (i + 1 < SPW)
      next = dec_head<LAT>(A, sub + 1 < nsub, off[i + 1], off[i + 2], kbs[i + 1], lane);
    const uint32_t lrow = sub / spr;
    const uint32_t col = (sub - lrow * spr) * HQ_SUB + 8u * (uint32_t)lane;
    const int64_t grow = A.first_row + lrow;
    // output signs, loaded before the bit walk
    uint4 sw = make_uint4(0u, 0u, 0u, 0u);
    if (MODE == 1) sw = *(const uint4*)(A.dsign16 + (col >> 1));

    uint32_t sym[8];
    const bool ok = decode_symbols<LAT>(A, head, lane, buf, starts, s_sel, sym);
    const unsigned long long bad = __ballot(!ok);  // wave-uniform
    if (bad && A.stats) {
      // count the sub-stream once (its first failing lane reports)
      if ((unsigned)lane == (unsigned)__builtin_ctzll(bad)) {
        atomicAdd(&A.stats->corrupt_substreams, 1u);
        atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_CORRUPT);
      }
    }
    int32_t c[8];
    unstrip8<LAT>(sym, c);
    float g = SPW == 1 ? gm
                       : (i == 0 ? quad_bcast<0>(gm)
                                 : (i == 1 ? quad_bcast<1>(gm) : (i == 2 ? quad_bcast<2>(gm) : quad_bcast<3>(gm))));
    if (bad) g = 0.0f;  // a corrupt sub-stream decodes as zeros, dither included

    if constexpr (MODE == 2) {
      uint32_t packed[2] = {0u, 0u};
      uint32_t clamps = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        int32_t v = c[j];
        if (v > 127) { v = 127; ++clamps; }
        if (v < -127) { v = -127; ++clamps; }
        packed[j >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (j & 3));
      }
      int8_t* out = (int8_t*)A.y + (int64_t)lrow * A.ld + col;
      *(uint2*)out = make_uint2(packed[0], packed[1]);
      if ((col & (uint32_t)(A.tile - 1)) == 0)
        A.g[(int64_t)lrow * A.tpr + (col >> __builtin_ctz((uint32_t)A.tile))] = g;
      if (clamps && A.stats) atomicAdd(&A.stats->clamps, clamps);
    } else if constexpr (MODE == 4) {
      // the MXFP4 cast of the reconstruction (Sec. 4.8, Sec. 6.4): v = g c in
      // the rotated coordinates (one fp32 product); blocks of 32 values (four
      // lanes, inside one tile) share X = floor(log2 amax) - 2, and each value
      // becomes E2M1(v / 2^X), two per byte (the even k in the low nibble),
      // the scale byte X + 127
      float v[8], am = 0.0f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        v[j] = (float)c[j] * g;
        am = __builtin_fmaxf(am, __builtin_fabsf(v[j]));
      }
      am = __builtin_fmaxf(am, dpp_xor<1>(am));
      am = __builtin_fmaxf(am, dpp_xor<2>(am));
      const int32_t X = mx_exponent(am);
      const float inv = __builtin_ldexpf(1.0f, -X);  // exact: v / 2^X is exact
      uint32_t packed = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) packed |= e2m1_code(v[j] * inv) << (4 * j);
      uint8_t* out = (uint8_t*)A.y + (int64_t)lrow * A.ld + (col >> 1);
      *(uint32_t*)out = packed;
      if ((lane & 3) == 0) A.mxs[(int64_t)lrow * (A.spr * (HQ_SUB / 32)) + (col >> 5)] = (uint8_t)(X + 127);
    } else if constexpr (MODE == 3) {
      // the fp8 cast (Sec. 4.8): E4M3 of each code, round to nearest even,
      // magnitudes beyond 448 saturated and counted
      float v[8];
      uint32_t clamps = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        v[j] = (float)c[j];
        if (v[j] > 448.0f) { v[j] = 448.0f; ++clamps; }
        if (v[j] < -448.0f) { v[j] = -448.0f; ++clamps; }
      }
      const uint32_t w0 = e4m3x4(v[0], v[1], v[2], v[3]), w1 = e4m3x4(v[4], v[5], v[6], v[7]);
      uint8_t* out = (uint8_t*)A.y + (int64_t)lrow * A.ld + col;
      *(uint2*)out = make_uint2(w0, w1);
      if ((col & (uint32_t)(A.tile - 1)) == 0)
        A.g[(int64_t)lrow * A.tpr + (col >> __builtin_ctz((uint32_t)A.tile))] = g;
      if (clamps && A.stats) atomicAdd(&A.stats->clamps, clamps);
    } else {
      // y = D H^T (S) (code - U) * r / (alpha n); the integer codes make the
      // transform exact in fp32 (|sum| <= 128 * 65536 < 2^24) whenever there
      // is no dither
      float y[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) y[j] = code_coord<LAT>(c[j], j);
      if (use_dither) {
        float u[8];
        dither8<LAT>(A.dither_seed, grow, col, u);
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = y[j] - u[j];
      }
      if (use_rot) {
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = flip(y[j], sbits, j);
      }
      if (use_qjl) qjl_tile(qmat, qstage, lane, y);  // y <- S^T y
      fwht128_tw(y, sg);
      const float g_tw = xor_sign(g, sg.sigma);
#pragma unroll
      for (int j = 0; j < 8; ++j) y[j] = y[j] * g_tw;
      if constexpr (MODE == 0) {
        const uint32_t dbits = sign_bits8(A.dmask, col);
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = flip(y[j], dbits, j);
        float4* out = (float4*)((float*)A.y + (int64_t)lrow * A.ld + col);
        out[0] = make_float4(y[0], y[1], y[2], y[3]);
        out[1] = make_float4(y[4], y[5], y[6], y[7]);
      } else {
        uint4 o;
        o.x = cvt_pk_bf16(y[0], y[1]) ^ sw.x;
        o.y = cvt_pk_bf16(y[2], y[3]) ^ sw.y;
        o.z = cvt_pk_bf16(y[4], y[5]) ^ sw.z;
        o.w = cvt_pk_bf16(y[6], y[7]) ^ sw.w;
        *(uint4*)((uint16_t*)A.y + (int64_t)lrow * A.ld + col) = o;
      }
    }
    if (i + 1 < SPW) head = next;
  }
}

// Block b of a sub-stream of B 512-symbol blocks (already in `buf`, Wl
// words): its remainder fields sit at bit b 64 lrem, its unary codes begin
// at bit ustart (anywhere in a word: the bits below it belong to block
// b - 1).  Lane l's codes start just past this block's terminator 8 l - 1,
// found by a popcount scan from ustart that stops once all 64 starts are
// known.  Returns false (in every lane) for a parse that runs out of words;
// `uend` becomes the bit past the block's last code.
template <int LAT>
__device__ __forceinline__ bool decode_block_mb(const uint32_t* buf, uint32_t Wl, uint32_t* starts,
                                                uint32_t ustart, uint32_t rem_base, uint32_t k0,
                                                uint32_t k1, int lane, bool ok, uint32_t* sym,
                                                uint32_t& uend) {
  const uint32_t lrem = lane_rem_bits<LAT>(k0, k1);
  const uint32_t nbits = 32u * Wl;
  starts[lane] = (lane == 0) ? ustart : 0xFFFFFFFFu;
  wave_sync_lds();
  const uint32_t uw0 = ustart >> 5;
  const uint32_t nuw = (ok && Wl > uw0) ? Wl - uw0 : 0u;
  const uint32_t lowmask = ~((1u << (ustart & 31u)) - 1u);
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nuw && carry < 504u; base += 64) {
    const uint32_t wi = base + lane;
    uint32_t v = (wi < nuw) ? buf[uw0 + wi] : 0u;
    if (wi == 0u) v &= lowmask;
    const uint32_t cnt = __popc(v);
    const uint32_t incl = wave_scan_incl(cnt);
    const uint32_t P = carry + incl - cnt;
    for (uint32_t t = (P & ~7u) + 7u; t < P + cnt; t += 8u) {
      const uint32_t j = (t + 1u) >> 3;
      if (j < 64u) starts[j] = (uw0 + wi) * 32u + select32(v, t - P) + 1u;
    }
    carry += __builtin_amdgcn_readlane(incl, 63);
  }
  wave_sync_lds();
  uint32_t pos = starts[lane];
  ok = ok && pos < nbits;
  uint32_t qv[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) qv[j] = 0;
  if (ok) {
    // the q_j: zeros before each of the lane's 8 terminators, a 64-bit
    // window sliding along the buffer
    uint64_t win = load_bits64(buf, pos, Wl);
    uint32_t valid = 64;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      uint32_t q = 0;
      while (ok && win == 0ull) {
        q += valid;
        pos += valid;
        if (pos >= nbits) {
          ok = false;
          break;
        }
        win = load_bits64(buf, pos, Wl);
        valid = 64;
      }
      const uint32_t lo = (uint32_t)win, hi = (uint32_t)(win >> 32);
      const uint32_t tz =
          lo ? (uint32_t)__builtin_ctz(lo) : 32u + (uint32_t)__builtin_ctz(hi | (hi == 0u));
      q += tz;
      pos += tz + 1;
      valid -= tz + 1;
      win = (tz >= 63u) ? 0ull : (win >> (tz + 1));
      qv[j] = q;
    }
  }
  uend = __builtin_amdgcn_readlane(pos, 63);
  // the lane's 8 remainders
  const uint32_t rpos = rem_base + __umul24((uint32_t)lane, lrem);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t kk = sym_class<LAT>(j) ? k1 : k0;
    const uint32_t r = (ok && kk) ? (uint32_t)load_bits64(buf, rpos + rem_offset<LAT>(j, k0, k1), Wl) : 0u;
    sym[j] = (qv[j] << kk) | (r & ((1u << kk) - 1u));
  }
  return __ballot(!ok) == 0ull;
}

// Long tiles (weights, bf16 or fp32 out): the wave's four consecutive
// sub-streams are decoded first and kept as lattice coordinates, then the
// tiles they form are transformed together (fwht_tiled) and denormalized.
// A corrupt sub-stream's codes count as zeros in its tile.
template <int LAT, int MODE>
__device__ __forceinline__ void decode_wg_tiled(const hq_decode_args& A, const uint32_t wgi) {
  extern __shared__ uint32_t smem[];
  __shared__ uint32_t s_sel[256];
  const int tid = threadIdx.x, lane = tid & 63;
  const uint32_t wave = readfirst((uint32_t)(tid >> 6));
  uint32_t* buf = smem + wave * (A.lds_words + 66);
  uint32_t* starts = buf + A.lds_words + 2;
  s_sel[tid] = byte_select_entry((uint32_t)tid);  // 256 threads, one entry each
  __syncthreads();

  const uint32_t n = (uint32_t)A.tile;
  const uint32_t mb = (uint32_t)A.mb;
  float y[HQ_DEC_SUBS_PER_WAVE][8];
  // the wave's four consecutive 512-symbol blocks (sub-streams when mb = 1)
  const uint32_t sub0 = (wgi * HQ_WAVES_PER_WG + wave) * HQ_DEC_SUBS_PER_WAVE;
  const uint32_t nsub = (uint32_t)A.nsub * mb;  // blocks
  const uint32_t spr = (uint32_t)A.spr * mb;
  const TwSigns sg(lane);
  if (mb > 1u) {
    // sub-streams of mb blocks: the whole sub-stream goes to the wave's
    // buffer, then its blocks are parsed in order (each block's unary codes
    // start where the previous block's end); a corrupt sub-stream decodes
    // as zeros in all of its blocks
    for (uint32_t j = 0; j < HQ_DEC_SUBS_PER_WAVE / mb; ++j) {
      const uint32_t s = sub0 / mb + j;  // sub-stream
      const bool act = s < (uint32_t)A.nsub;
      uint32_t start = 0, end = 0, kb = 0;
      if (act) {
        start = readfirst(A.offsets[(uint32_t)A.first_sub + s]);
        end = readfirst(A.offsets[(uint32_t)A.first_sub + s + 1]);
        kb = readfirst(A.kparam[(uint32_t)A.first_sub + s]);
      }
      const uint32_t k0 = (LAT == kA2) ? (kb & 15u) : kb;
      const uint32_t k1 = (LAT == kA2) ? (kb >> 4) : (LAT == kD4 ? (k0 > 0 ? k0 - 1 : 0) : k0);
      const uint32_t Rb = 64u * lane_rem_bits<LAT>(k0, k1);
      const uint32_t W = end - start;
      bool ok = act && end >= start && (int64_t)end <= A.cap_words && W <= A.lds_words &&
                k0 <= HQ_KMAX && mb * Rb <= 32u * W;
      const uint32_t Wl = ok ? W : 0u;
      for (uint32_t w = lane; w < Wl; w += 64) buf[w] = A.payload[(uint64_t)start + w];
      if (lane < 2) buf[Wl + lane] = 0u;  // two zero words past the end
      wave_sync_lds();
      uint32_t ustart = mb * Rb;
      for (uint32_t b = 0; b < mb; ++b) {
        uint32_t sym[8], uend;
        ok = decode_block_mb<LAT>(buf, Wl, starts, ustart, b * Rb, k0, k1, lane, ok, sym, uend);
        ustart = uend;
        int32_t c[8];
        unstrip8<LAT>(sym, c);
        const uint32_t i = j * mb + b;
#pragma unroll
        for (int q = 0; q < HQ_DEC_SUBS_PER_WAVE; ++q)
          if ((uint32_t)q == i)
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) y[q][jj] = act ? code_coord<LAT>(c[jj], jj) : 0.0f;
      }
      if (act && !ok) {
#pragma unroll
        for (int q = 0; q < HQ_DEC_SUBS_PER_WAVE; ++q)
          if ((uint32_t)q / mb == j)
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) y[q][jj] = 0.0f;
        if (A.stats && lane == 0) {
          atomicAdd(&A.stats->corrupt_substreams, 1u);
          atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_CORRUPT);
        }
      }
    }
  } else {
  uint32_t off[HQ_DEC_SUBS_PER_WAVE + 1], kbs[HQ_DEC_SUBS_PER_WAVE];
#pragma unroll
  for (int i = 0; i <= HQ_DEC_SUBS_PER_WAVE; ++i) {
    const uint32_t sub = sub0 + (uint32_t)i;
    off[i] = sub <= nsub ? readfirst(A.offsets[(uint32_t)A.first_sub + sub]) : 0u;
    if (i < HQ_DEC_SUBS_PER_WAVE)
      kbs[i] = sub < nsub ? readfirst(A.kparam[(uint32_t)A.first_sub + sub]) : 0u;
  }
  DecHead head = dec_head<LAT>(A, sub0 < nsub, off[0], off[1], kbs[0], lane);
#pragma unroll
  for (int i = 0; i < HQ_DEC_SUBS_PER_WAVE; ++i) {
    const uint32_t sub = sub0 + (uint32_t)i;
    DecHead next;
    if (i + 1 < HQ_DEC_SUBS_PER_WAVE)
      next = dec_head<LAT>(A, sub + 1 < nsub, off[i + 1], off[i + 2], kbs[i + 1], lane);
    if (sub < nsub) {
      uint32_t sym[8];
      const bool ok = decode_symbols<LAT>(A, head, lane, buf, starts, s_sel, sym);
      const unsigned long long bad = __ballot(!ok);
      if (bad && A.stats && (unsigned)lane == (unsigned)__builtin_ctzll(bad)) {
        atomicAdd(&A.stats->corrupt_substreams, 1u);
        atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_CORRUPT);
      }
      int32_t c[8];
      unstrip8<LAT>(sym, c);
#pragma unroll
      for (int j = 0; j < 8; ++j) y[i][j] = code_coord<LAT>(c[j], j);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) y[i][j] = 0.0f;
    }
    if (i + 1 < HQ_DEC_SUBS_PER_WAVE) head = next;
  }
  }  // one block per sub-stream
  // y = D H^T code * r / (alpha n): the tiles' transforms, then each lane
  // its own tile's factor
  const uint32_t sigma = fwht_tiled(y, lane, n, sg);
#pragma unroll
  for (int i = 0; i < HQ_DEC_SUBS_PER_WAVE; ++i) {
    const uint32_t sub = sub0 + (uint32_t)i;
    if (sub >= nsub) break;
    const uint32_t lrow = sub / spr;
    const uint32_t col = (sub - lrow * spr) * HQ_SUB + 8u * (uint32_t)lane;
    const uint64_t flat = (uint64_t)sub * HQ_SUB + 8u * (uint32_t)lane;
    const float rs = ((const float*)A.norms)[A.first_row * A.tpr + (int64_t)(flat / n)];
    const float g_tw = xor_sign(rs / A.alpha_n, sigma);
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = y[i][j] * g_tw;
    if constexpr (MODE == 0) {
      const uint32_t dbits = sign_bits8(A.dmask, col);
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = flip(v[j], dbits, j);
      float4* out = (float4*)((float*)A.y + (int64_t)lrow * A.ld + col);
      out[0] = make_float4(v[0], v[1], v[2], v[3]);
      out[1] = make_float4(v[4], v[5], v[6], v[7]);
    } else {
      const uint4 sw = *(const uint4*)(A.dsign16 + (col >> 1));
      uint4 o;
      o.x = cvt_pk_bf16(v[0], v[1]) ^ sw.x;
      o.y = cvt_pk_bf16(v[2], v[3]) ^ sw.y;
      o.z = cvt_pk_bf16(v[4], v[5]) ^ sw.z;
      o.w = cvt_pk_bf16(v[6], v[7]) ^ sw.w;
      *(uint4*)((uint16_t*)A.y + (int64_t)lrow * A.ld + col) = o;
    }
  }
}

template <int LAT, int MODE>
__global__ __launch_bounds__(256) void hq_decode_tiled_kernel(hq_decode_args A) {
  decode_wg_tiled<LAT, MODE>(A, blockIdx.x);
}

// ------------------------------------------------------------ qjl decode on the matrix cores
// KV streams with the qjl rotation, decoded to fp32 or bf16.  S^T y is a
// dense 128 x 128 contraction per tile, so it runs on the fp32 matrix cores
// (v_mfma_f32_16x16x4_f32) instead of the VALU with S streamed from LDS.
// A workgroup takes 16 consecutive sub-streams (64 tiles) per pass:
//  1. each wave decodes its four sub-streams, undithers them and writes
//     y = code - U into the workgroup's tile array Y in LDS (tile rows of
//     kQjlRow floats: the 16 rows one operand load reads fall in distinct
//     banks);
//  2. wave w forms columns 32 w .. 32 w + 31 of Z = Y S for all 64 tiles
//     (row z of Z is (S^T y)^T) with its 32 columns of S held in registers,
//     then, once every wave has read Y, writes them over it;
//  3. each wave finishes its own tiles from Z: inverse RHT, scale, signs,
//     store.
// The contraction sums in the matrix cores' order, so the output equals
// the oracle's left-to-right fp32 sums to rounding, not bit for bit.
typedef float v4f_t __attribute__((ext_vector_type(4)));
constexpr int kQjlRow = 130;            // floats per tile row of Y
constexpr int kQjlTiles = 64;           // tiles per workgroup pass (16 sub-streams)

template <int LAT, int MODE>
__global__ __launch_bounds__(256) void hq_decode_qjl_kernel(hq_decode_args A) {
  extern __shared__ uint32_t smem[];
  __shared__ uint32_t s_sel[256];
  const int tid = threadIdx.x, lane = tid & 63;
  const uint32_t wave = readfirst((uint32_t)(tid >> 6));
  uint32_t* buf = smem + wave * (A.lds_words + 66);
  uint32_t* starts = buf + A.lds_words + 2;
  float* const Y = (float*)(smem + HQ_WAVES_PER_WG * (A.lds_words + 66));
  s_sel[tid] = byte_select_entry((uint32_t)tid);
  // B operands: step s covers k = 4 s .. 4 s + 3 (lane / 16 picks k), block
  // cb the columns n = 32 wave + 16 cb + lane % 16
  float sb[32][2];
#pragma unroll
  for (int s = 0; s < 32; ++s) {
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
      sb[s][cb] = A.qjl[(4 * s + (lane >> 4)) * HQ_TILE + 32 * (int)wave + 16 * cb + (lane & 15)];
  }
  __syncthreads();
  const TwSigns sg(lane);
  const uint32_t nsub = (uint32_t)A.nsub, spr = (uint32_t)A.spr;
  const uint32_t ngroups = (nsub + 15u) / 16u;
  for (uint32_t grp = blockIdx.x; grp < ngroups; grp += gridDim.x) {
    const uint32_t sub0 = grp * 16u + wave * 4u;
    // ---- 1. decode into Y rows wave * 16 + 4 i + lane / 16
    float gi[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t sub = sub0 + (uint32_t)i;
      gi[i] = 0.0f;
      if (sub >= nsub) continue;  // wave-uniform; the row's Z is never stored
      const uint32_t o0 = readfirst(A.offsets[(uint32_t)A.first_sub + sub]);
      const uint32_t o1 = readfirst(A.offsets[(uint32_t)A.first_sub + sub + 1]);
      const uint32_t kb = readfirst(A.kparam[(uint32_t)A.first_sub + sub]);
      const DecHead head = dec_head<LAT>(A, true, o0, o1, kb, lane);
      const int64_t t = A.first_row * A.tpr + 4 * (int64_t)sub + (lane >> 4);
      const float rs = A.norm_fp16 ? (float)((const _Float16*)A.norms)[t] : ((const float*)A.norms)[t];
      const uint32_t lrow = sub / spr;
      const uint32_t col = (sub - lrow * spr) * HQ_SUB + 8u * (uint32_t)lane;
      uint32_t sym[8];
      const bool ok = decode_symbols<LAT>(A, head, lane, buf, starts, s_sel, sym);
      const unsigned long long bad = __ballot(!ok);
      if (bad && A.stats && (unsigned)lane == (unsigned)__builtin_ctzll(bad)) {
        atomicAdd(&A.stats->corrupt_substreams, 1u);
        atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_CORRUPT);
      }
      gi[i] = bad ? 0.0f : rs / A.alpha_n;  // a corrupt sub-stream decodes as zeros
      int32_t c[8];
      unstrip8<LAT>(sym, c);
      float y[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) y[j] = code_coord<LAT>(c[j], j);
      if (A.dither) {
        float u[8];
        dither8<LAT>(A.dither_seed, A.first_row + lrow, col, u);
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = y[j] - u[j];
      }
      float* row = Y + (wave * 16u + 4u * (uint32_t)i + (uint32_t)(lane >> 4)) * kQjlRow + (lane & 15) * 8;
#pragma unroll
      for (int j = 0; j < 8; j += 2) *(float2*)(row + j) = make_float2(y[j], y[j + 1]);
    }
    __syncthreads();
    // ---- 2. Z[:, 32 wave .. +31] = Y S
    v4f_t acc[4][2];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) acc[rb][cb] = v4f_t{0.0f, 0.0f, 0.0f, 0.0f};
    }
#pragma unroll  // sb is indexed by s: only a full unroll keeps it in registers
    for (int s = 0; s < 32; ++s) {
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        const float a = Y[(rb * 16 + (lane & 15)) * kQjlRow + 4 * s + (lane >> 4)];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, sb[s][cb], acc[rb][cb], 0, 0, 0);
      }
    }
    __syncthreads();  // every wave has read Y
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          Y[(rb * 16 + 4 * (lane >> 4) + r) * kQjlRow + 32 * (int)wave + 16 * cb + (lane & 15)] = acc[rb][cb][r];
      }
    }
    __syncthreads();
    // ---- 3. this wave's tiles: inverse RHT, scale, signs, store
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t sub = sub0 + (uint32_t)i;
      if (sub >= nsub) break;
      const uint32_t lrow = sub / spr;
      const uint32_t col = (sub - lrow * spr) * HQ_SUB + 8u * (uint32_t)lane;
      const float* row = Y + (wave * 16u + 4u * (uint32_t)i + (uint32_t)(lane >> 4)) * kQjlRow + (lane & 15) * 8;
      float y[8];
#pragma unroll
      for (int j = 0; j < 8; j += 2) {
        const float2 v = *(const float2*)(row + j);
        y[j] = v.x;
        y[j + 1] = v.y;
      }
      fwht128_tw(y, sg);
      const float g_tw = xor_sign(gi[i], sg.sigma);
#pragma unroll
      for (int j = 0; j < 8; ++j) y[j] = y[j] * g_tw;
      if constexpr (MODE == 0) {
        const uint32_t dbits = sign_bits8(A.dmask, col);
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = flip(y[j], dbits, j);
        float4* out = (float4*)((float*)A.y + (int64_t)lrow * A.ld + col);
        out[0] = make_float4(y[0], y[1], y[2], y[3]);
        out[1] = make_float4(y[4], y[5], y[6], y[7]);
      } else {
        const uint4 sw = *(const uint4*)(A.dsign16 + (col >> 1));
        uint4 o;
        o.x = cvt_pk_bf16(y[0], y[1]) ^ sw.x;
        o.y = cvt_pk_bf16(y[2], y[3]) ^ sw.y;
        o.z = cvt_pk_bf16(y[4], y[5]) ^ sw.z;
        o.w = cvt_pk_bf16(y[6], y[7]) ^ sw.w;
        *(uint4*)((uint16_t*)A.y + (int64_t)lrow * A.ld + col) = o;
      }
    }
  }
}

template <int LAT, int MODE, bool KV>
__global__ __launch_bounds__(256) void hq_decode_kernel(hq_decode_args A) {
  decode_wg<LAT, MODE, KV>(A, blockIdx.x);
}

// Single matrices of fewer than HQ_DEC_SMALL sub-streams: one per wave.
template <int LAT, int MODE, bool KV>
__global__ __launch_bounds__(256) void hq_decode_small_kernel(hq_decode_args A) {
  decode_wg<LAT, MODE, KV, 1>(A, blockIdx.x);
}

template <int LAT, int MODE, bool KV>
__global__ __launch_bounds__(256) void hq_decode_group_kernel(hq_decode_group_args G) {
  int mi = 0;
  for (int i = 1; i < G.count; ++i) mi = blockIdx.x >= G.wg_begin[i] ? i : mi;
  decode_wg<LAT, MODE, KV>(G.m[mi], blockIdx.x - G.wg_begin[mi]);
}

// ------------------------------------------------------------ fused decode + GEMV
// y[r] = sum_k W^[r, k] x[k] for one token: the decode fused with a
// matrix-vector product (the fused decode-GEMV kernel of Sec. 6.6).  On a
// weight plan, tile t of decoded row r is
// g_t D_t H coord(c_t) with H the symmetric unnormalized Walsh-Hadamard
// matrix (the RHT absorbed into the product, Sec. 4.1), so its product with
// x_t is g_t coord(c_t) . (H D_t x_t): the transform moves from every row
// onto x, once per call (hq_gemv_prep_kernel), and a row costs its Rice
// decode, the unstrip and one dot product per lattice block.  One workgroup
// per row: each wave walks a fixed share of the row's sub-streams with a
// per-lane partial sum, a fixed butterfly over the wave and a fixed order
// over the four waves follow, so the result does not depend on scheduling.

// xt = H D x per 128-column tile, fp32; one wave per 512 columns.
__global__ __launch_bounds__(256) void hq_gemv_prep_kernel(const void* x, int x_bf16, int64_t K,
                                                           const uint32_t* dmask, float* xt) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t base = ((int64_t)blockIdx.x * 4 + (tid >> 6)) * HQ_SUB;
  if (base >= K) return;  // K is a multiple of 512
  const int64_t col = base + (lane >> 4) * HQ_TILE + (lane & 15) * 8;
  float v[8];
  if (x_bf16) {
    const uint4 raw = *(const uint4*)((const uint16_t*)x + col);
    const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = bf16_to_f32(w4[i] & 0xFFFFu);
      v[2 * i + 1] = bf16_to_f32(w4[i] >> 16);
    }
  } else {
    const float4 a = *(const float4*)((const float*)x + col);
    const float4 b = *(const float4*)((const float*)x + col + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
  const uint32_t dbits = sign_bits8(dmask, col);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = flip(v[i], dbits, i);
  const XSigns sg(lane);
  fwht128(v, sg);
  *(float4*)(xt + col) = make_float4(v[0], v[1], v[2], v[3]);
  *(float4*)(xt + col + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

template <int LAT>
__global__ __launch_bounds__(256) void hq_decode_gemv_kernel(hq_decode_args A, const float* xt,
                                                             void* y, int y_bf16) {
  extern __shared__ uint32_t smem[];
  __shared__ uint32_t s_sel[256];
  __shared__ float s_part[HQ_WAVES_PER_WG];
  const int tid = threadIdx.x, lane = tid & 63;
  const uint32_t wave = readfirst((uint32_t)(tid >> 6));
  uint32_t* buf = smem + wave * (A.lds_words + 66);
  uint32_t* starts = buf + A.lds_words + 2;
  s_sel[tid] = kByteSelect.e[tid];  // 256 threads, one entry each
  __syncthreads();
  // one row per workgroup: wave w takes the row's sub-streams w, w + 4, ...,
  // each one's table entry and first payload words loaded a step ahead
  const uint32_t spr = (uint32_t)A.spr;
  const int64_t row = blockIdx.x;  // within the call's rows
  const uint32_t sub0 = (uint32_t)A.first_sub + (uint32_t)row * spr;
  const bool fp16_norm = A.norm_fp16;
  auto head_of = [&](uint32_t j) {
    const uint32_t start = readfirst(A.offsets[sub0 + j]), end = readfirst(A.offsets[sub0 + j + 1]);
    return dec_head<LAT>(A, true, start, end, readfirst(A.kparam[sub0 + j]), lane);
  };
  float acc = 0.0f;
  DecHead head;
  if (wave < spr) head = head_of(wave);
  for (uint32_t j = wave; j < spr; j += HQ_WAVES_PER_WG) {
    DecHead next;
    if (j + HQ_WAVES_PER_WG < spr) next = head_of(j + HQ_WAVES_PER_WG);
    uint32_t sym[8];
    const bool ok = decode_symbols<LAT>(A, head, lane, buf, starts, s_sel, sym);
    if (!ok && A.stats) {
      const unsigned long long bad = __ballot(!ok);
      if ((unsigned)lane == (unsigned)__builtin_ctzll(bad)) {
        atomicAdd(&A.stats->corrupt_substreams, 1u);
        atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_CORRUPT);
      }
    }
    int32_t c[8];
    unstrip8<LAT>(sym, c);
    const int64_t col = (int64_t)j * HQ_SUB + 8 * lane;
    const float4 xa = *(const float4*)(xt + col);
    const float4 xb = *(const float4*)(xt + col + 4);
    const float xv[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
    float d = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) d = __builtin_fmaf(code_coord<LAT>(c[i], i), xv[i], d);
    const int64_t t = (A.first_row + row) * A.tpr + 4 * (int64_t)j + (lane >> 4);
    const float rs = fp16_norm ? (float)((const _Float16*)A.norms)[t] : ((const float*)A.norms)[t];
    acc = __builtin_fmaf(rs, d, acc);  // the common 1 / (alpha n) once per row
    head = next;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if (lane == 0) s_part[wave] = acc;
  __syncthreads();
  if (tid == 0) {
    const float v = (((s_part[0] + s_part[1]) + s_part[2]) + s_part[3]) / A.alpha_n;
    if (y_bf16)
      ((uint16_t*)y)[row] = (uint16_t)f32_to_bf16(v);
    else
      ((float*)y)[row] = v;
  }
}

// The same product with one wave per row (rows >= HQ_GEMV_WAVE_ROWS): the
// wave walks all of its row's sub-streams, each one's table entry and first
// payload words a step ahead, and a butterfly over the wave ends the sum; no
// barrier after the table copy.
template <int LAT>
__global__ __launch_bounds__(256) void hq_decode_gemv_rows_kernel(hq_decode_args A, const float* xt,
                                                                  void* y, int y_bf16, int64_t rows) {
  extern __shared__ uint32_t smem[];
  __shared__ uint32_t s_sel[256];
  const int tid = threadIdx.x, lane = tid & 63;
  const uint32_t wave = readfirst((uint32_t)(tid >> 6));
  s_sel[tid] = kByteSelect.e[tid];  // 256 threads, one entry each
  __syncthreads();
  const int64_t row = (int64_t)blockIdx.x * HQ_WAVES_PER_WG + wave;  // within the call's rows
  if (row >= rows) return;  // whole waves; no barrier follows
  uint32_t* buf = smem + wave * (A.lds_words + 66);
  uint32_t* starts = buf + A.lds_words + 2;
  const uint32_t spr = (uint32_t)A.spr;
  const uint32_t sub0 = (uint32_t)A.first_sub + (uint32_t)row * spr;
  const bool fp16_norm = A.norm_fp16;
  auto head_of = [&](uint32_t j) {
    const uint32_t start = readfirst(A.offsets[sub0 + j]), end = readfirst(A.offsets[sub0 + j + 1]);
    return dec_head<LAT>(A, true, start, end, readfirst(A.kparam[sub0 + j]), lane);
  };
  const int64_t t0 = (A.first_row + row) * A.tpr + (lane >> 4);
  float acc = 0.0f;
  DecHead head = head_of(0);
  float rs = fp16_norm ? (float)((const _Float16*)A.norms)[t0] : ((const float*)A.norms)[t0];
  bool bad = false;
  for (uint32_t j = 0; j < spr; ++j) {
    DecHead next;
    float rs_next = 0.0f;
    if (j + 1 < spr) {
      next = head_of(j + 1);
      const int64_t t = t0 + 4 * (int64_t)(j + 1);
      rs_next = fp16_norm ? (float)((const _Float16*)A.norms)[t] : ((const float*)A.norms)[t];
    }
    uint32_t sym[8];
    bad |= !decode_symbols<LAT>(A, head, lane, buf, starts, s_sel, sym);
    int32_t c[8];
    unstrip8<LAT>(sym, c);
    const int64_t col = (int64_t)j * HQ_SUB + 8 * lane;
    const float4 xa = *(const float4*)(xt + col);
    const float4 xb = *(const float4*)(xt + col + 4);
    const float xv[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
    float d = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) d = __builtin_fmaf(code_coord<LAT>(c[i], i), xv[i], d);
    acc = __builtin_fmaf(rs, d, acc);  // the common 1 / (alpha n) once per row
    head = next;
    rs = rs_next;
  }
  if (bad && A.stats) {
    const unsigned long long anyb = __ballot(bad);
    if ((unsigned)lane == (unsigned)__builtin_ctzll(anyb)) {
      atomicAdd(&A.stats->corrupt_substreams, 1u);
      atomicCAS(&A.stats->status, 0u, (uint32_t)HQ_ERR_CORRUPT);
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if (lane == 0) {
    const float v = acc / A.alpha_n;
    if (y_bf16)
      ((uint16_t*)y)[row] = (uint16_t)f32_to_bf16(v);
    else
      ((float*)y)[row] = v;
  }
}

// ------------------------------------------------------------ fused decode + attention
// One query token per sequence attending over its coded KV cache (the KV
// path of Sec. 5.2, read back as in Sec. 5.3, for the one-token decoding of
// Sec. 6.6).  A decoded key tile is k^ = g D H S (code - U), H the symmetric
// unnormalized Walsh-Hadamard matrix (Sec. 4.1, 4.2, 4.4), so
// q . k^ = g (S H D q) . (code - U): the query moves into the coded
// coordinates once per call (hq_attn_prep_kernel) and a key then costs its
// Rice decode, the unstrip, its dither and one dot product.  The values are
// summed in the same coordinates, sum_t p_t v^_t = D H S sum_t p_t g_t
// (code_t - U_t), and transformed back once per head (hq_attn_combine_kernel).
// The softmax runs online in base 2 (the query carries scale * log2 e).
// Work: one workgroup per (sequence, sub-stream column j, split of 4 * chunk
// tokens); wave w walks its chunk of tokens, its lane group of 16 holding one
// KV head's tile and the G query heads that read it.  Every sum has a fixed
// order, so results depend on the call's shape only, not on scheduling.

// Sum over the 16 lanes of a row; every lane gets the same bits.
__device__ __forceinline__ float row16_sum(float v) {
  v += xor_lane_f<8>(v);
  v += xor_lane_f<4>(v);
  v += xor_lane_f<2>(v);
  v += xor_lane_f<1>(v);
  return v;
}

// One step of a transposed row sum over lane bit M: of the N values a lane
// holds, the lanes with that bit set keep the upper half and the others the
// lower half, each adding its partner's copy of the half it keeps (N = 1:
// a plain butterfly step).
template <int M, int N>
__device__ __forceinline__ void tsum_step(float* d, int lane) {
  if constexpr (N > 1) {
    const bool up = (lane & M) != 0;
#pragma unroll
    for (int h = 0; h < N / 2; ++h) {
      const float keep = up ? d[h + N / 2] : d[h];
      const float send = up ? d[h] : d[h + N / 2];
      d[h] = keep + xor_lane_f<M>(send);
    }
  } else {
    d[0] += xor_lane_f<M>(d[0]);
  }
}

// Sums over the 16 lanes of a row of G per-lane values at once: lane l
// returns the sum of value (l mod 16) / (16 / G), every lane of a run of
// 16 / G the same bits.
template <int G>
__device__ __forceinline__ float row16_sums(float* d, int lane) {
  tsum_step<8, G>(d, lane);
  tsum_step<4, (G > 1 ? G / 2 : 1)>(d, lane);
  tsum_step<2, (G > 3 ? G / 4 : 1)>(d, lane);
  tsum_step<1, (G > 7 ? G / 8 : 1)>(d, lane);
  return d[0];
}

// Value of lane N of the lane's 16-lane row (DPP row_newbcast).
template <int N>
__device__ __forceinline__ float row_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x150 + N, 0xF, 0xF, false));
}

// v of each of the row's G head runs (lane g (16 / G) for head g).
template <int G>
__device__ __forceinline__ void bcast_heads(float v, float* out) {
  out[0] = row_bcast<0>(v);
  if constexpr (G > 1) out[1] = row_bcast<16 / G>(v);
  if constexpr (G > 2) {
    out[2] = row_bcast<2 * (16 / G)>(v);
    out[3] = row_bcast<3 * (16 / G)>(v);
  }
  if constexpr (G > 4) {
    out[4] = row_bcast<8>(v);
    out[5] = row_bcast<10>(v);
    out[6] = row_bcast<12>(v);
    out[7] = row_bcast<14>(v);
  }
}

// Token count of sequence b, clamped to what its table row can hold; a bad
// value is reported in the key stream's counters.
__device__ __forceinline__ int64_t attn_seq_len(const hq_attn_args& A, int64_t b, bool report) {
  const int64_t cap = (int64_t)A.max_blocks * A.block_tokens;
  int64_t len = A.seq_lens[b];
  if (len < 0 || len > cap) {
    if (report && A.K.stats) atomicCAS(&A.K.stats->status, 0u, (uint32_t)HQ_ERR_INVALID_ARG);
    len = len < 0 ? 0 : cap;
  }
  return len;
}

// Tokens of a sequence read from the coded streams: all but the residual
// window's last min(window, len).
__device__ __forceinline__ int64_t attn_coded_len(const hq_attn_args& A, int64_t len) {
  return len - (len < A.window ? len : (int64_t)A.window);
}

// 8 consecutive values (16-byte aligned) of a bf16 or fp32 array as fp32.
__device__ __forceinline__ void load8(const void* p, int64_t i, bool bf16, float* v) {
  if (bf16) {
    const uint4 raw = *(const uint4*)((const uint16_t*)p + i);
    const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[2 * k] = bf16_to_f32(w4[k] & 0xFFFFu);
      v[2 * k + 1] = bf16_to_f32(w4[k] >> 16);
    }
  } else {
    const float4 a = *(const float4*)((const float*)p + i);
    const float4 b = *(const float4*)((const float*)p + i + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

// qt = (S H D q) * scale * log2(e) per query head, with the key plan's signs
// (D of the head's own columns); one lane group of 16 per head.
__global__ __launch_bounds__(256) void hq_attn_prep_kernel(hq_attn_args A) {
  __shared__ float s_stage[HQ_WAVES_PER_WG * HQ_QJL_STAGE];  // qjl keys only
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t pair = ((int64_t)blockIdx.x * HQ_WAVES_PER_WG + (tid >> 6)) * 4 + (lane >> 4);
  if (pair >= A.batch * A.heads_q) return;  // whole lane groups
  const int32_t kvh = (int32_t)(pair % A.heads_q) / A.group;
  const int c0 = (lane & 15) * 8;
  float v[8];
  load8(A.q, pair * HQ_TILE + c0, A.q_bf16, v);
  const uint32_t dbits = sign_bits8(A.K.dmask, (int64_t)kvh * HQ_TILE + c0);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = flip(v[i], dbits, i);
  const XSigns sg(lane);
  fwht128(v, sg);
  if (A.K.rotation == HQ_ROT_QJL) qjl_tile(A.K.qjlt, s_stage + (tid >> 6) * HQ_QJL_STAGE, lane, v);
  const uint32_t sbits = A.K.rotation == HQ_ROT_SIGNS ? sign_bits8(A.K.smask, c0) : 0u;
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = flip(v[i], sbits, i) * A.qscale;
  float* o = A.qt + pair * HQ_TILE + c0;
  *(float4*)o = make_float4(v[0], v[1], v[2], v[3]);
  *(float4*)(o + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

// The lane's 8 coordinates of one coded tile, code - U (U the stream's
// dither at that row).
template <int LAT>
__device__ __forceinline__ bool attn_tile(const hq_decode_args& S, const DecHead& head, int lane,
                                          uint32_t* buf, uint32_t* starts, const uint32_t* sel,
                                          uint32_t row, uint32_t j, float* y) {
  uint32_t sym[8];
  const bool ok = decode_symbols<LAT>(S, head, lane, buf, starts, sel, sym);
  int32_t c[8];
  unstrip8<LAT>(sym, c);
#pragma unroll
  for (int i = 0; i < 8; ++i) y[i] = code_coord<LAT>(c[i], i);
  if (S.dither) {
    float u[8];
    dither8<LAT>(S.dither_seed, row, (int64_t)j * HQ_SUB + 8 * lane, u);
#pragma unroll
    for (int i = 0; i < 8; ++i) y[i] = y[i] - u[i];
  }
  if (__ballot(!ok) != 0ull) {  // a corrupt sub-stream contributes zeros
#pragma unroll
    for (int i = 0; i < 8; ++i) y[i] = 0.0f;
  }
  return ok;
}

// Stored tile norm r of the lane's tile in `row` (fp32 or fp16).
__device__ __forceinline__ float attn_norm(const hq_decode_args& S, uint32_t row, uint32_t j,
                                           int lane) {
  const int64_t t = (int64_t)row * S.tpr + 4 * (int64_t)j + (lane >> 4);
  return S.norm_fp16 ? (float)((const _Float16*)S.norms)[t] : ((const float*)S.norms)[t];
}

// Table entry (start, end, k) of one token's sub-stream, fetched earlier by
// lane i of the wave for the i-th token of a run of 64.
struct AttnMeta {
  uint32_t s, e, k;
};

__device__ __forceinline__ uint32_t lane_val(uint32_t v, uint32_t i) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, (int)i);
}

// Two passes over the same grid and token chunks.  The key pass (VAL =
// false) decodes each key tile and stores its G scores per KV head, base 2,
// at scores[(b, j, t), 4 G] plus every wave's largest score per head.  The
// value pass (VAL = true) decodes each value tile and adds p g (code - U)
// with p = 2^(s - m), m that wave's largest score, so no sum is ever
// rescaled inside the token loop; the four waves then rescale to their
// common maximum and write one partial per workgroup.  Each pass holds one
// stream's decode state: the single-pass form held both plus the value sums
// (163 registers, three waves per SIMD).  Scores, maxima and weights are
// per lane: lane l of a row of 16 handles query head hl = (l mod 16) /
// (16 / G) of the row's G, and the value pass broadcasts each head's weight
// p across the row.
// The value pass at G <= 4 is held to 128 registers (four waves per SIMD);
// what that moves to scratch is saved before the token loop and restored
// after it.
template <int LAT, int G, bool VAL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(VAL && G <= 4 ? 4 : 1)))
void hq_attn_kernel(hq_attn_args A) {
  extern __shared__ uint32_t smem[];
  __shared__ uint32_t s_sel[256];
  __shared__ float s_m[HQ_WAVES_PER_WG][4 * G];
  __shared__ float s_l[HQ_WAVES_PER_WG][4 * G];
  __shared__ float4 s_q[VAL ? 1 : 4 * G * 32];  // key pass: the query tiles, coded coordinates
  const int tid = threadIdx.x, lane = tid & 63;
  const uint32_t wave = readfirst((uint32_t)(tid >> 6));
  const uint32_t spr = (uint32_t)A.K.spr;
  const uint32_t x = blockIdx.x % (uint32_t)A.nx;
  const uint32_t bj = blockIdx.x / (uint32_t)A.nx;
  const uint32_t b = bj / spr, j = bj - b * spr;
  const int64_t len =
      attn_coded_len(A, attn_seq_len(A, b, !VAL && tid == 0 && x == 0 && j == 0));
  const int64_t wg_t0 = (int64_t)x * HQ_WAVES_PER_WG * A.chunk;
  if (wg_t0 >= len) return;  // the whole workgroup, before any barrier
  const hq_decode_args& S = VAL ? A.V : A.K;
  s_sel[tid] = kByteSelect.e[tid];
  // KV heads 4j .. 4j+3 read query heads (4j) G .. (4j + 4) G - 1: one block
  const int64_t hq0 = (int64_t)b * A.heads_q + (int64_t)j * 4 * G;
  if constexpr (!VAL) {
    for (int i = tid; i < 4 * G * 32; i += 256) s_q[i] = ((const float4*)(A.qt + hq0 * HQ_TILE))[i];
  }
  __syncthreads();
  uint32_t* buf = smem + wave * (A.lds_words + 66);
  uint32_t* starts = buf + A.lds_words + 2;
  float* comb = (float*)(smem + HQ_WAVES_PER_WG * (A.lds_words + 66));

  const int q4 = lane >> 4, c0 = (lane & 15) * 8;
  const int hl = (lane & 15) / (16 / G);
  const bool lead = (lane & (16 / G - 1)) == 0;  // first lane of its head's run
  const float4* qrow = s_q + (q4 * G) * 32 + (lane & 15) * 2;  // head g: + 32 g
  // scores of (b, j): token t's 4 G heads at + 4 G t, this lane group's at + G q4
  float* srow =
      A.scores + (int64_t)bj * ((int64_t)A.max_blocks * A.block_tokens) * (4 * G) + q4 * G + hl;
  float* wmax = A.wmax + ((int64_t)blockIdx.x * HQ_WAVES_PER_WG + wave) * (4 * G) + q4 * G + hl;
  float acc[VAL ? G : 1][8];
  float m = -__builtin_inff(), l = 0.0f;  // head hl's
  if constexpr (VAL) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[g][i] = 0.0f;
    }
  }

  const int64_t t0 = wg_t0 + (int64_t)wave * A.chunk;
  const int64_t t1 = t0 + A.chunk < len ? t0 + A.chunk : len;
  if (VAL && t0 < t1) m = *wmax;  // written by the key pass for these tokens
  const uint32_t bt = (uint32_t)A.block_tokens;
  const int32_t* trow = A.table + (int64_t)b * A.max_blocks;
  bool bad = false;
  for (int64_t tb = t0; tb < t1; tb += 64) {
    // lane i fetches token tb + i's row and table entry (rows past the
    // streams or a negative block id: row ~0u, the token is skipped)
    const uint32_t n = (uint32_t)(t1 - tb < 64 ? t1 - tb : 64);
    uint32_t rv = ~0u;
    AttnMeta me = {0u, 0u, 0u};
    if ((uint32_t)lane < n) {
      const uint32_t t = (uint32_t)(tb + lane);
      const uint32_t bi = t / bt;
      const int32_t blk = trow[bi];
      const int64_t r = (int64_t)blk * bt + (t - bi * bt);
      if (blk >= 0 && r < A.rows) {
        rv = (uint32_t)r;
        const int64_t sub = r * spr + j;
        me = {S.offsets[sub], S.offsets[sub + 1], S.kparam[sub]};
      }
    }
    if (!VAL && __ballot(rv == ~0u && (uint32_t)lane < n) && lane == 0 && A.K.stats)
      atomicCAS(&A.K.stats->status, 0u, (uint32_t)HQ_ERR_INVALID_ARG);  // block id out of range
    // token i's head, norm and (value pass) scores, each loaded one token ahead
    auto fetch = [&](uint32_t i, uint32_t& row, DecHead& h, float& nr, float& sc) {
      row = lane_val(rv, i);
      if (row != ~0u) {
        h = dec_head<LAT>(S, true, lane_val(me.s, i), lane_val(me.e, i), lane_val(me.k, i), lane);
        nr = attn_norm(S, row, j, lane);
        if constexpr (VAL) sc = srow[(tb + i) * (4 * G)];
      }
    };
    uint32_t row;
    DecHead hd;
    float nr = 0.0f, sc = 0.0f;
    fetch(0, row, hd, nr, sc);
    for (uint32_t i = 0; i < n; ++i) {
      uint32_t nrow = ~0u;
      DecHead nhd;
      float nnr = 0.0f, nsc = 0.0f;
      if (i + 1 < n) fetch(i + 1, nrow, nhd, nnr, nsc);
      if (row != ~0u) {
        float y[8];
        bad |= !attn_tile<LAT>(S, hd, lane, buf, starts, s_sel, row, j, y);
        const float gs = nr / S.alpha_n;
        if constexpr (!VAL) {
          float d[G];
#pragma unroll
          for (int g = 0; g < G; ++g) {
            const float4 qa = qrow[32 * g], qb = qrow[32 * g + 1];
            float e = qa.x * y[0];
            e = __builtin_fmaf(qa.y, y[1], e);
            e = __builtin_fmaf(qa.z, y[2], e);
            e = __builtin_fmaf(qa.w, y[3], e);
            e = __builtin_fmaf(qb.x, y[4], e);
            e = __builtin_fmaf(qb.y, y[5], e);
            e = __builtin_fmaf(qb.z, y[6], e);
            e = __builtin_fmaf(qb.w, y[7], e);
            d[g] = e;
          }
          const float sl = gs * row16_sums<G>(d, lane);
          m = __builtin_fmaxf(m, sl);
          if (lead) srow[(tb + i) * (4 * G)] = sl;
        } else {
          const float p = exp2f(sc - m);
          l += p;
          float pg[G];
          bcast_heads<G>(p * gs, pg);
#pragma unroll
          for (int g = 0; g < G; ++g) {
#pragma unroll
            for (int i2 = 0; i2 < 8; ++i2) acc[g][i2] = __builtin_fmaf(pg[g], y[i2], acc[g][i2]);
          }
        }
      }
      row = nrow;
      hd = nhd;
      nr = nnr;
      sc = nsc;
    }
  }
  if (bad && A.K.stats) {
    const unsigned long long anyb = __ballot(bad);
    if ((unsigned)lane == (unsigned)__builtin_ctzll(anyb)) {
      atomicAdd(&A.K.stats->corrupt_substreams, 1u);
      atomicCAS(&A.K.stats->status, 0u, (uint32_t)HQ_ERR_CORRUPT);
    }
  }
  if constexpr (!VAL) {
    if (t0 < t1 && lead) *wmax = m;
    return;
  } else {
    // the four waves' sums, rescaled to their common maximum, in wave order
    if (lead) s_m[wave][q4 * G + hl] = m;
    __syncthreads();
    float M = s_m[0][q4 * G + hl];
#pragma unroll
    for (int w = 1; w < HQ_WAVES_PER_WG; ++w) M = __builtin_fmaxf(M, s_m[w][q4 * G + hl]);
    const float f = m == -__builtin_inff() ? 0.0f : exp2f(m - M);
    l *= f;
    m = M;
    float fg[G];
    bcast_heads<G>(f, fg);
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[g][i] *= fg[g];
    }
    if (wave > 0) {
      float* cw = comb + ((wave - 1) * 64 + lane) * 8 * G;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        *(float4*)(cw + 8 * g) = make_float4(acc[g][0], acc[g][1], acc[g][2], acc[g][3]);
        *(float4*)(cw + 8 * g + 4) = make_float4(acc[g][4], acc[g][5], acc[g][6], acc[g][7]);
      }
      if (lead) s_l[wave][q4 * G + hl] = l;
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int w = 1; w < HQ_WAVES_PER_WG; ++w) {
        const float* cw = comb + ((w - 1) * 64 + lane) * 8 * G;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const float4 a = *(const float4*)(cw + 8 * g);
          const float4 c = *(const float4*)(cw + 8 * g + 4);
          acc[g][0] += a.x; acc[g][1] += a.y; acc[g][2] += a.z; acc[g][3] += a.w;
          acc[g][4] += c.x; acc[g][5] += c.y; acc[g][6] += c.z; acc[g][7] += c.w;
        }
        l += s_l[w][q4 * G + hl];
      }
      const int64_t h0 = hq0 + (int64_t)q4 * G;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int64_t pi = (h0 + g) * A.nx + x;
        float* o = A.part_acc + pi * HQ_TILE + c0;
        *(float4*)o = make_float4(acc[g][0], acc[g][1], acc[g][2], acc[g][3]);
        *(float4*)(o + 4) = make_float4(acc[g][4], acc[g][5], acc[g][6], acc[g][7]);
      }
      if (lead) {
        const int64_t pi = (h0 + hl) * A.nx + x;
        A.part_m[pi] = m;
        A.part_l[pi] = l;
      }
    }
  }
}

// out = (D H S sum_x f_x acc_x + sum_i p_i v_i) / (sum_x f_x l_x + sum_i p_i):
// the coded splits that hold tokens (f_x = 2^(m_x - M)) with the value
// plan's signs, plus the residual window's exact tokens i (p_i = 2^(s_i - M),
// s_i = q . k_i scaled in natural coordinates), M the maximum over both; an
// empty sequence gives zeros.  One workgroup per query head: lane group k of
// 16 takes splits k, k + 16, ... and window tokens k, k + 16, ..., and the 16
// groups' sums meet in LDS in group order.
__global__ __launch_bounds__(256) void hq_attn_combine_kernel(hq_attn_args A) {
  __shared__ float s_red[16];
  __shared__ float s_win[HQ_ATTN_WINDOW_MAX];
  __shared__ float4 s_acc[16][32];
  __shared__ float4 s_nat[16][32];
  const int tid = threadIdx.x, lane = tid & 63, grp = tid >> 4;
  const int64_t pair = blockIdx.x;
  const int64_t b = pair / A.heads_q;
  const int32_t kvh = (int32_t)(pair - b * A.heads_q) / A.group;
  const int c0 = (lane & 15) * 8;
  const int64_t len = attn_seq_len(A, b, false);
  const int64_t clen = attn_coded_len(A, len);
  const int32_t w = (int32_t)(len - clen);
  const int64_t per = (int64_t)HQ_WAVES_PER_WG * A.chunk;
  const int32_t n = (int32_t)((clen + per - 1) / per);
  const float* pm = A.part_m + pair * A.nx;
  const float* pl = A.part_l + pair * A.nx;
  const int64_t hkv = (int64_t)A.heads_q / A.group;
  float M = -__builtin_inff();
  if (w > 0) {
    float q[8];
    load8(A.q, pair * HQ_TILE + c0, A.q_bf16, q);
    for (int32_t i = grp; i < w; i += 16) {
      const int64_t slot = (clen + i) % A.window;
      float k[8];
      load8(A.win_k, ((b * A.window + slot) * hkv + kvh) * HQ_TILE + c0, A.win_bf16, k);
      float d = q[0] * k[0];
#pragma unroll
      for (int e = 1; e < 8; ++e) d = __builtin_fmaf(q[e], k[e], d);
      const float si = row16_sum(d) * A.qscale;
      if ((tid & 15) == 0) s_win[i] = si;
      M = __builtin_fmaxf(M, si);
    }
  }
  for (int32_t x = grp; x < n; x += 16) M = __builtin_fmaxf(M, pm[x]);
  if ((tid & 15) == 0) s_red[grp] = M;
  __syncthreads();
  M = s_red[0];
#pragma unroll
  for (int k = 1; k < 16; ++k) M = __builtin_fmaxf(M, s_red[k]);
  float L = 0.0f, v[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  float vn[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  if (M != -__builtin_inff()) {
    for (int32_t x = grp; x < n; x += 16) {
      const float mx = pm[x];
      const float f = mx == -__builtin_inff() ? 0.0f : exp2f(mx - M);
      L = __builtin_fmaf(f, pl[x], L);
      const float* a = A.part_acc + (pair * A.nx + x) * HQ_TILE + c0;
      const float4 a0 = *(const float4*)a;
      const float4 a1 = *(const float4*)(a + 4);
      v[0] = __builtin_fmaf(f, a0.x, v[0]); v[1] = __builtin_fmaf(f, a0.y, v[1]);
      v[2] = __builtin_fmaf(f, a0.z, v[2]); v[3] = __builtin_fmaf(f, a0.w, v[3]);
      v[4] = __builtin_fmaf(f, a1.x, v[4]); v[5] = __builtin_fmaf(f, a1.y, v[5]);
      v[6] = __builtin_fmaf(f, a1.z, v[6]); v[7] = __builtin_fmaf(f, a1.w, v[7]);
    }
    for (int32_t i = grp; i < w; i += 16) {
      const int64_t slot = (clen + i) % A.window;
      const float p = exp2f(s_win[i] - M);
      L += p;
      float val[8];
      load8(A.win_v, ((b * A.window + slot) * hkv + kvh) * HQ_TILE + c0, A.win_bf16, val);
#pragma unroll
      for (int e = 0; e < 8; ++e) vn[e] = __builtin_fmaf(p, val[e], vn[e]);
    }
  }
  __syncthreads();  // every group has read s_red
  s_acc[grp][(lane & 15) * 2] = make_float4(v[0], v[1], v[2], v[3]);
  s_acc[grp][(lane & 15) * 2 + 1] = make_float4(v[4], v[5], v[6], v[7]);
  s_nat[grp][(lane & 15) * 2] = make_float4(vn[0], vn[1], vn[2], vn[3]);
  s_nat[grp][(lane & 15) * 2 + 1] = make_float4(vn[4], vn[5], vn[6], vn[7]);
  if ((tid & 15) == 0) s_red[grp] = L;
  __syncthreads();
  if (tid >= 16) return;  // group 0 finishes: no barrier follows
  L = 0.0f;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const float4 a0 = s_acc[k][tid * 2], a1 = s_acc[k][tid * 2 + 1];
    const float4 n0 = s_nat[k][tid * 2], n1 = s_nat[k][tid * 2 + 1];
    if (k == 0) {
      v[0] = a0.x; v[1] = a0.y; v[2] = a0.z; v[3] = a0.w;
      v[4] = a1.x; v[5] = a1.y; v[6] = a1.z; v[7] = a1.w;
      vn[0] = n0.x; vn[1] = n0.y; vn[2] = n0.z; vn[3] = n0.w;
      vn[4] = n1.x; vn[5] = n1.y; vn[6] = n1.z; vn[7] = n1.w;
    } else {
      v[0] += a0.x; v[1] += a0.y; v[2] += a0.z; v[3] += a0.w;
      v[4] += a1.x; v[5] += a1.y; v[6] += a1.z; v[7] += a1.w;
      vn[0] += n0.x; vn[1] += n0.y; vn[2] += n0.z; vn[3] += n0.w;
      vn[4] += n1.x; vn[5] += n1.y; vn[6] += n1.z; vn[7] += n1.w;
    }
    L += s_red[k];
  }
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  const uint32_t sbits = A.V.rotation == HQ_ROT_SIGNS ? sign_bits8(A.V.smask, c0) : 0u;
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = flip(v[i] * inv, sbits, i);
  if (A.V.rotation == HQ_ROT_QJL) qjl_tile(A.V.qjl, (float*)s_acc, lane, v);  // v <- S^T v
  const XSigns sg(lane);
  fwht128(v, sg);
  const uint32_t dbits = sign_bits8(A.V.dmask, (int64_t)kvh * HQ_TILE + c0);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = __builtin_fmaf(vn[i], inv, flip(v[i], dbits, i));
  if (A.out_bf16) {
    uint4 o;
    o.x = cvt_pk_bf16(v[0], v[1]);
    o.y = cvt_pk_bf16(v[2], v[3]);
    o.z = cvt_pk_bf16(v[4], v[5]);
    o.w = cvt_pk_bf16(v[6], v[7]);
    *(uint4*)((uint16_t*)A.out + pair * HQ_TILE + c0) = o;
  } else {
    float* o = (float*)A.out + pair * HQ_TILE + c0;
    *(float4*)o = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)(o + 4) = make_float4(v[4], v[5], v[6], v[7]);
  }
}

// ------------------------------------------------------------ activation prep
// One workgroup per token row: per tile y = H D a (canonical stage order, the
// weights' signs: stages h = 1 .. 64 in registers per 128 columns, then for a
// longer tile h = 128 .. tile / 2 in LDS), amax over the row, then the cast.

__global__ __launch_bounds__(256) void hq_act_prep_kernel(hq_actprep_args A) {
  extern __shared__ float ybuf[];
  __shared__ float s_max[4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t row = blockIdx.x;
  const uint16_t* arow = (const uint16_t*)A.a + row * A.lda;
  const XSigns sg(lane);
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
    fwht128(v, sg);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      amax = __builtin_fmaxf(amax, __builtin_fabsf(v[i]));
      ybuf[col + i] = v[i];
    }
  }
  if (A.tile > HQ_TILE) {
    // the remaining butterflies of a long tile, one stage at a time over the
    // row: pair p of stage h is (j, j + h) with j = (p / h) 2h + p % h
    for (int64_t h = HQ_TILE; h < A.tile; h <<= 1) {
      __syncthreads();
      for (int64_t p2 = tid; p2 < A.K / 2; p2 += 256) {
        const int64_t j = (p2 / h) * 2 * h + p2 % h;
        const float a = ybuf[j], b = ybuf[j + h];
        ybuf[j] = a + b;
        ybuf[j + h] = a - b;
      }
    }
    __syncthreads();
    amax = 0.0f;
    for (int64_t c = tid; c < A.K; c += 256) amax = __builtin_fmaxf(amax, __builtin_fabsf(ybuf[c]));
  }
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) amax = __builtin_fmaxf(amax, __shfl_xor(amax, m, 64));
  if (lane == 0) s_max[wave] = amax;
  __syncthreads();
  if (A.fp8 == 2) {
    // MXFP4: blocks of 32 (eight threads of four values each) share
    // X = floor(log2 amax) - 2 and hold E2M1(y / 2^X); no per-token factor
    for (int64_t base = 0; base < A.K; base += 1024) {
      const int64_t col = base + (int64_t)tid * 4;
      const bool in = col < A.K;  // whole 32-blocks are in or out (K is a multiple of 512)
      float q[4], am = 0.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        q[i] = in ? ybuf[col + i] : 0.0f;
        am = __builtin_fmaxf(am, __builtin_fabsf(q[i]));
      }
      am = __builtin_fmaxf(am, __shfl_xor(am, 1, 64));
      am = __builtin_fmaxf(am, __shfl_xor(am, 2, 64));
      am = __builtin_fmaxf(am, __shfl_xor(am, 4, 64));
      const int32_t X = mx_exponent(am);
      uint32_t packed = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) packed |= e2m1_code(__builtin_ldexpf(q[i], -X)) << (4 * i);
      if (in) {
        *(uint16_t*)((uint8_t*)A.xq + row * (A.K / 2) + col / 2) = (uint16_t)packed;
        if ((tid & 7) == 0) A.mxs[row * (A.K / 32) + col / 32] = (uint8_t)(X + 127);
      }
    }
    return;
  }
  amax = __builtin_fmaxf(__builtin_fmaxf(s_max[0], s_max[1]), __builtin_fmaxf(s_max[2], s_max[3]));
  const float top = A.fp8 ? 448.0f : 127.0f;  // E4M3's largest magnitude, or int8's
  const float inv = (amax == 0.0f) ? 0.0f : top / amax;
  int8_t* xrow = A.xq + row * A.K;
  for (int64_t col = (int64_t)tid * 4; col < A.K; col += 1024) {
    uint32_t packed = 0;
    if (A.fp8) {
      float q[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) q[i] = __builtin_fminf(__builtin_fmaxf(ybuf[col + i] * inv, -448.0f), 448.0f);
      packed = e4m3x4(q[0], q[1], q[2], q[3]);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float qv = __builtin_rintf(ybuf[col + i] * inv);
        qv = __builtin_fminf(__builtin_fmaxf(qv, -127.0f), 127.0f);
        packed |= ((uint32_t)(int32_t)qv & 0xFFu) << (8 * i);
      }
    }
    *(uint32_t*)(xrow + col) = packed;
  }
  if (tid == 0) A.sx[row] = amax / top;
}


// ------------------------------------------------------------ block-scaled GEMM
// int8 and E4M3: out[m, n] = s_x[m] * sum_t g[n, t] * P_t[m, n], P_t the sum
// over one factor tile of K: exact int32 on the int8 matrix cores
// (v_mfma_i32_32x32x32_i8), fp32 on the f8f6f4 ones for E4M3
// (v_mfma_scale_f32_32x32x64_f8f6f4 with unit scales).  MXFP4: out[m, n] =
// sum_k X[m, k] W[n, k] over the element-times-block-scale values on the
// same instruction, whose E8M0 scales carry every factor.
// Workgroup tile 256 (tokens) x 128 (weight rows), eight waves in 4 x 2, each
// 64 x 64 = 2 x 2 MFMA blocks, one workgroup per CU.  An LDS stage is 128
// bytes of every A and B row (one K tile of int8 / E4M3, two of MXFP4) plus
// its side data (tile factors, MX block scales), in a ring of three filled
// straight from global memory by direct-to-LDS loads, with no register
// staging: stage t + 2 streams in while stage t is multiplied, by eight
// waves in two groups half a stage apart (gemm_body_pp).
// LDS rows are 128 bytes with the 16-byte chunk c of row r at position
// c ^ ((r / 2) % 8): a wave's 1 KB direct load fills rows 8q .. 8q + 7 (lane
// l at row 8q + l / 8, position l % 8), and the 16 lanes of one LDS cycle
// reading one chunk of 16 consecutive rows cover the 64 banks exactly once.
// Both operands are K-contiguous rows and every lane reads the same k range
// of A and B, so the contraction pairs identical k whatever order the
// instruction assigns inside a step.  Output lane l of a 32 x 32 block holds
// column l % 32 and rows 8 (r / 4) + 4 (l / 32) + r % 4.

typedef int v4i_t __attribute__((ext_vector_type(4)));
typedef int v8i_t __attribute__((ext_vector_type(8)));
typedef int v16i_t __attribute__((ext_vector_type(16)));
typedef float v16f_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef const __attribute__((address_space(1))) void gbl_void_t;

constexpr int kGemmM = 256, kGemmN = 128;  // the loads below assume 256 x 128 and 8 waves
constexpr int kGemmThreads = 512;           // 8 waves, 4 (m) x 2 (n)
constexpr int kGemmNB = kGemmN / 64;        // 32 x 32 blocks per wave along n
constexpr int kGemmStageA = kGemmM * 128, kGemmStageB = kGemmN * 128;
// side data of a stage: for int8 and E4M3 the weight rows' factors of the
// stage's factor tile (float n for weight row n0 + n); for MXFP4 the 8 scale
// bytes of each A row and of each B row
constexpr int kGemmSideG = 0, kGemmSideXs = 1024, kGemmSideWs = 3072;
constexpr int kGemmStages = 3;  // LDS ring: stage t + 2 loads while stage t is multiplied
template <int MODE> constexpr int gemm_stage_bytes() {
  return kGemmStageA + kGemmStageB + (MODE == 2 ? 4096 : 512);
}
template <int MODE> constexpr int gemm_lds_bytes() { return kGemmStages * gemm_stage_bytes<MODE>(); }
static_assert(gemm_lds_bytes<2>() <= 160 * 1024, "the LDS ring fits one CU");

template <bool C, class T, class F> struct gemm_pick { using type = T; };
template <class T, class F> struct gemm_pick<false, T, F> { using type = F; };
template <int MODE> struct GemmMode {
  static constexpr int U = MODE == 2 ? 2 : 1;  // 128-deep K units per stage
  using acc_t = typename gemm_pick<MODE == 0, v16i_t, v16f_t>::type;
};

// The direct-to-LDS loads go through buffer resources based at the
// workgroup's first A row, B row, factor row and scale rows: a lane's 32-bit
// offset within them is fixed for the whole K loop and the stage's offset is
// a scalar.  4 A and 2 B row groups per wave (16 bytes a lane, lane l at row
// 8q + l / 8 and K chunk (l % 8) ^ ((4q + l / 16) % 8)), then the side data
// (4 bytes a lane): for int8 and E4M3 factor dword j * 64 + l = g[n0 + 64 j +
// l, t >> lm] with j = w % 2, for MXFP4 scale dword d = w * 64 + l of the A
// rows and d = (w % 4) * 64 + l of the B rows (row d / 2, half d % 2).  Waves
// with equal j (or w % 4) load the same values to the same place, so every
// wave issues the same loads and the loop has no branch.  Rows past M or N
// read the last valid row: they only feed outputs that are never stored,
// and every access stays inside its resource.
struct GemmLoads {
  __amdgpu_buffer_rsrc_t ra, rb, rg, rxs, rws;
  uint32_t a[4], b[2], g, xs, ws;
  int lm;  // log2 of the 128-deep K units per factor tile
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t gemm_rsrc(const void* base, int64_t bytes) {
  // raw buffer (stride 0); the third descriptor word of gfx9 data buffers.
  // The operands are workgroup-uniform: read them into scalar registers.
  const uint64_t p = (uint64_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
  const int n = __builtin_amdgcn_readfirstlane((int)bytes);
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), (short)0, n, 0x00020000);
}

template <int MODE>
__device__ __forceinline__ GemmLoads gemm_loads(const hq_gemm_args& A, int64_t m0, int64_t n0,
                                                int wave, int lane) {
  const int64_t rb = MODE == 2 ? A.K / 2 : A.K;  // row bytes
  const int64_t T = A.K / A.tile, ks = A.K / 32;  // factors and MX scale bytes per row
  const int64_t ma = min<int64_t>(A.M - m0, kGemmM), nb = min<int64_t>(A.N - n0, kGemmN);
  GemmLoads L;
  L.ra = gemm_rsrc(A.xq + m0 * rb, ma * rb);
  L.rb = gemm_rsrc(A.w + n0 * rb, nb * rb);
  L.rg = gemm_rsrc(MODE != 2 ? A.g + n0 * T : nullptr, MODE != 2 ? nb * T * 4 : 0);
  L.rxs = gemm_rsrc(MODE == 2 ? A.xs + m0 * ks : nullptr, MODE == 2 ? ma * ks : 0);
  L.rws = gemm_rsrc(MODE == 2 ? A.ws + n0 * ks : nullptr, MODE == 2 ? nb * ks : 0);
  const int rr = lane >> 3;
  // row 8q + rr holds chunk (lane % 8) ^ ((4q + lane / 16) % 8) at position lane % 8
  auto kc = [&](int q) { return (uint32_t)(((lane & 7) ^ ((4 * q + (lane >> 4)) & 7)) << 4); };
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int q = wave * 4 + i;
    L.a[i] = (uint32_t)(min<int64_t>(8 * q + rr, ma - 1) * rb) + kc(q);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q = wave * 2 + i;
    L.b[i] = (uint32_t)(min<int64_t>(8 * q + rr, nb - 1) * rb) + kc(q);
  }
  L.lm = __builtin_ctz((uint32_t)(A.tile / HQ_TILE));
  L.g = (uint32_t)(min<int64_t>((wave & 1) * 64 + lane, nb - 1) * T * 4);
  const int d = wave * 64 + lane, e = (wave & 3) * 64 + lane;
  L.xs = (uint32_t)(min<int64_t>(d >> 1, ma - 1) * ks + (d & 1) * 4);
  L.ws = (uint32_t)(min<int64_t>(e >> 1, nb - 1) * ks + (e & 1) * 4);
  return L;
}

// Direct-to-LDS loads of stage t into `stage` (wave is wave-uniform).
template <int MODE>
__device__ __forceinline__ void gemm_fetch(const GemmLoads& L, int64_t t, int wave, int8_t* stage) {
  const uint32_t so = (uint32_t)(t * 128);
#pragma unroll
  for (int i = 0; i < 4; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(L.ra, (lds_void_t*)(stage + (wave * 4 + i) * 1024), 16,
                                             L.a[i], so, 0, 0);
#pragma unroll
  for (int i = 0; i < 2; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(L.rb, (lds_void_t*)(stage + kGemmStageA + (wave * 2 + i) * 1024),
                                             16, L.b[i], so, 0, 0);
  int8_t* const side = stage + kGemmStageA + kGemmStageB;
  if constexpr (MODE != 2) {
    // the stage's factor tile; MXFP4 blocks carry the factors in their scales
    __builtin_amdgcn_raw_ptr_buffer_load_lds(L.rg, (lds_void_t*)(side + kGemmSideG + (wave & 1) * 256), 4,
                                             L.g, (uint32_t)((t >> L.lm) * 4), 0, 0);
  } else {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(L.rxs, (lds_void_t*)(side + kGemmSideXs + wave * 256), 4,
                                             L.xs, (uint32_t)(t * 8), 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(L.rws, (lds_void_t*)(side + kGemmSideWs + (wave & 3) * 256),
                                             4, L.ws, (uint32_t)(t * 8), 0, 0);
  }
}

// 16 bytes of row `row`, K chunk c (0..7) of a stage operand
__device__ __forceinline__ v4i_t gemm_frag(const int8_t* base, int row, int c) {
  return *(const v4i_t*)(base + row * 128 + ((c ^ ((row >> 1) & 7)) << 4));
}

// MXFP4: a lane's scale words from the side data: the 8 scale bytes of its
// row, shifted so that byte 0 / byte 2 of the low word are the lane's blocks
// of the stage's first / second 64-deep step and those of the high word its
// third / fourth (the lane's half of step s is block 2 s + l / 32).
__device__ __forceinline__ uint2 mx_scales(const int8_t* side, int row, int lane) {
  const uint2 w = *(const uint2*)(side + row * 8);
  const uint32_t sh = 8u * (uint32_t)(lane >> 5);
  return make_uint2(w.x >> sh, w.y >> sh);
}

template <int OPSEL>
__device__ __forceinline__ v16f_t mfma_mxfp4(v4i_t a, v4i_t b, v16f_t c, uint32_t sa, uint32_t sb) {
  const v8i_t a8 = {a[0], a[1], a[2], a[3], 0, 0, 0, 0};
  const v8i_t b8 = {b[0], b[1], b[2], b[3], 0, 0, 0, 0};
  // cbsz = blgp = 4: both operands E2M1; the scales are E8M0 bytes
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, c, 4, 4, OPSEL, (int)sa, OPSEL,
                                                         (int)sb);
}

// A lane's factors for its kGemmNB weight columns (int8 and E4M3).
__device__ __forceinline__ void gemm_side_g(const int8_t* side, int wn, int lane, float (&gv)[kGemmNB]) {
#pragma unroll
  for (int b = 0; b < kGemmNB; ++b)
    gv[b] = ((const float*)(side + kGemmSideG))[wn * (kGemmN / 2) + b * 32 + (lane & 31)];
}

// Rescale elements [e0, e0 + E) of a finished tile's partials (block
// j = e / 16 = 2 a + b, register r = e % 16) into the fp32 accumulators.
template <int MODE, int E>
__device__ __forceinline__ void gemm_rescale(int e0, const typename GemmMode<MODE>::acc_t (&p)[2][kGemmNB],
                                             const float (&gv)[kGemmNB], float (&accf)[2][kGemmNB][16]) {
#pragma unroll
  for (int e = e0; e < e0 + E; ++e) {
    const int j = e >> 4, r = e & 15, a = j / kGemmNB, b = j % kGemmNB;
    accf[a][b][r] = __builtin_fmaf((float)p[a][b][r], gv[b], accf[a][b][r]);
  }
}

// MFMA steps per stage: int8 32-deep (four), E4M3 64-deep (two), MXFP4
// 64-deep over its two K units (four), and 16-byte chunks per fragment.
template <int MODE> constexpr int gemm_pp_steps() { return MODE == 1 ? 2 : 4; }
template <int MODE> constexpr int gemm_pp_fw() { return MODE == 1 ? 2 : 1; }

// The MFMA phase of a stage: its steps into `cur`, from zero when FRESH (the
// first stage of a factor tile, or of the whole product for MXFP4).
template <int MODE, bool FRESH>
__device__ __forceinline__ void gemm_mfma_pp(const v4i_t (&fa)[gemm_pp_steps<MODE>()][2][gemm_pp_fw<MODE>()],
                                             const v4i_t (&fb)[gemm_pp_steps<MODE>()][kGemmNB][gemm_pp_fw<MODE>()],
                                             const uint2 (&xs)[2], const uint2 (&ws)[kGemmNB],
                                             typename GemmMode<MODE>::acc_t (&cur)[2][kGemmNB]) {
  using acc_t = typename GemmMode<MODE>::acc_t;
#pragma unroll
  for (int s = 0; s < gemm_pp_steps<MODE>(); ++s)
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < kGemmNB; ++b) {
        const acc_t c0 = (FRESH && s == 0) ? (acc_t){} : cur[a][b];
        if constexpr (MODE == 0) {
          cur[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[s][a][0], fb[s][b][0], c0, 0, 0, 0);
        } else if constexpr (MODE == 1) {
          const v8i_t x = {fa[s][a][0][0], fa[s][a][0][1], fa[s][a][0][2], fa[s][a][0][3],
                           fa[s][a][1][0], fa[s][a][1][1], fa[s][a][1][2], fa[s][a][1][3]};
          const v8i_t y = {fb[s][b][0][0], fb[s][b][0][1], fb[s][b][0][2], fb[s][b][0][3],
                           fb[s][b][1][0], fb[s][b][1][1], fb[s][b][1][2], fb[s][b][1][3]};
          // cbsz = blgp = 0: both operands E4M3; scale bytes 127 (2^0)
          cur[a][b] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(x, y, c0, 0, 0, 0, 127, 0, 127);
        } else {
          // step s of the stage is K unit s / 2: its scale word, byte 2 (s % 2)
          const uint32_t xa = s < 2 ? xs[a].x : xs[a].y, wb = s < 2 ? ws[b].x : ws[b].y;
          cur[a][b] = (s & 1) ? mfma_mxfp4<2>(fa[s][a][0], fb[s][b][0], c0, xa, wb)
                              : mfma_mxfp4<0>(fa[s][a][0], fb[s][b][0], c0, xa, wb);
        }
      }
}

// Output staging: a wave's 64 x 64 tile in LDS with rows of 64 values plus
// 16 bytes of padding (rows 4 apart, written by the two lane halves, then
// fall in different banks), 8 regions filling less than the stage ring.
template <bool BF16> constexpr int gemm_out_row() { return BF16 ? 144 : 272; }
constexpr int kGemmOutRegion = 64 * 272;
static_assert(8 * kGemmOutRegion <= gemm_lds_bytes<0>(), "the output tiles fit the ring");

// out rows r0 .. r0 + 63, columns c0 .. c0 + 63 of the wave's tile: each
// value (s_x times the accumulator for int8 / E4M3; MXFP4's accumulator as
// is) into LDS at its MFMA position, then 16-byte row pieces to global
// memory (element stores at a ragged right edge).
template <int MODE, bool BF16>
__device__ __forceinline__ void gemm_store_tile(const hq_gemm_args& A, int8_t* tile,
                                                const typename GemmMode<MODE>::acc_t (&cur)[2][kGemmNB],
                                                const float (&accf)[2][kGemmNB][16], int64_t r0,
                                                int64_t c0, int lane) {
  constexpr bool RESCALE = MODE != 2;
  constexpr int RS = gemm_out_row<BF16>();
  constexpr int ES = BF16 ? 2 : 4;  // bytes per value
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      const int64_t m = r0 + row;
      const float sxm = RESCALE && m < A.M ? A.sx[m] : 1.0f;
#pragma unroll
      for (int b = 0; b < kGemmNB; ++b) {
        float v;
        if constexpr (RESCALE)
          v = sxm * accf[a][b][r];
        else
          v = cur[a][b][r];
        int8_t* const p = tile + row * RS + (b * 32 + (lane & 31)) * ES;
        if constexpr (BF16)
          *(uint16_t*)p = (uint16_t)f32_to_bf16(v);
        else
          *(float*)p = v;
      }
    }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  constexpr int VPL = 16 / ES;            // values per 16-byte piece
  constexpr int LPR = 64 / VPL;           // lanes per row
  constexpr int ROWS = 64 / LPR;          // rows per pass
#pragma unroll
  for (int i = 0; i < 64 / ROWS; ++i) {
    const int row = i * ROWS + lane / LPR, col = (lane % LPR) * VPL;
    const int64_t m = r0 + row, n = c0 + col;
    if (m >= A.M || n >= A.N) continue;
    const uint4 v = *(const uint4*)(tile + row * RS + col * ES);
    char* const dst = (char*)A.out + (m * A.N + n) * ES;
    if (n + VPL <= A.N && ((m * A.N + n) * ES) % 16 == 0) {
      *(uint4*)dst = v;
    } else {
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < VPL; ++e)
        if (n + e < A.N) {
          if constexpr (BF16)
            ((uint16_t*)dst)[e] = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
          else
            ((uint32_t*)dst)[e] = w[e];
        }
    }
  }
}

// The block-scaled GEMM, all three operand types: the eight waves in two
// groups of four (waves 0-3 and 4-7: with a workgroup's waves placed on the
// four SIMDs in turn, each SIMD holds one wave of each group; the results
// do not depend on the placement) that run half a stage apart.  A wave's stage t has two phases: in V(t) it
// issues the direct-to-LDS loads of stage t + 2, reads every fragment (and
// for MXFP4 the block scale words) of stage t into registers and, for int8
// and E4M3 when stage t starts a factor tile, rescales the previous tile's
// partial sums into its fp32 accumulators; in M(t) it only issues MFMAs (a
// long tile's stages accumulate into the same partials; MXFP4's scales
// carry every factor, so its MFMAs accumulate the whole product).  Group 0
// runs V(t) in phase 2t and M(t) in phase 2t + 1, group 1 one phase later,
// and every phase ends at a workgroup barrier, so on each SIMD one wave's
// MFMAs run while the other wave's LDS reads and rescale issue.  The barrier
// waits leave only this wave's newest stage of loads in flight and no LDS
// read outstanding: a stage is complete in LDS before either group reads
// it, and its slot is refilled (stage t + 3, issued in phase 2t + 2) only
// after group 1's reads of phase 2t + 1 have returned.  Every wave executes
// the same 2 TS + 1 barriers: group 1 one before its first V phase, group 0
// one after its last M phase.
template <int MODE>
__device__ __forceinline__ void gemm_body_pp(const hq_gemm_args& A) {
  using acc_t = typename GemmMode<MODE>::acc_t;
  constexpr bool RESCALE = MODE != 2;
  constexpr int SB = gemm_stage_bytes<MODE>();
  constexpr int NS = gemm_pp_steps<MODE>();
  constexpr int FW = gemm_pp_fw<MODE>();
  extern __shared__ __attribute__((aligned(16))) int8_t gsm[];
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5;
  const int wsc = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, in a scalar register
  const int wm = wsc >> 1, wn = wsc & 1, grp = wsc >> 2;
  const int64_t m0 = (int64_t)blockIdx.y * kGemmM, n0 = (int64_t)blockIdx.x * kGemmN;
  const int64_t TS = A.K / HQ_TILE / GemmMode<MODE>::U;  // LDS stages
  const uint32_t tmask = (uint32_t)(A.tile / HQ_TILE) - 1u;  // stages per factor tile, less one

  float accf[2][kGemmNB][16];
  if constexpr (RESCALE) {
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < kGemmNB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) accf[a][b][r] = 0.0f;
  }
  acc_t cur[2][kGemmNB];
  float gcur[kGemmNB];
  uint2 xs[2], ws[kGemmNB];
  v4i_t fa[NS][2][FW], fb[NS][kGemmNB][FW];

  const GemmLoads gl = gemm_loads<MODE>(A, m0, n0, wsc, lane);
  constexpr int NL = MODE == 2 ? 8 : 7;  // buffer loads per wave and stage
  gemm_fetch<MODE>(gl, 0, wsc, gsm);
  gemm_fetch<MODE>(gl, min<int64_t>(1, TS - 1), wsc, gsm + SB);
  // a phase boundary: the waits, the barrier, and no instruction scheduled
  // across it (the MFMAs of M(t) would otherwise rise into V(t))
  auto phase = [&]() {
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(NL) : "memory");
    __builtin_amdgcn_sched_barrier(0);
  };
  if (grp == 1) phase();  // group 1 starts one phase late
  for (int64_t t = 0; t < TS; ++t) {
    phase();
    // V(t)
    const int8_t* const stage = gsm + (t % 3) * SB;
    const int8_t* const side = stage + kGemmStageA + kGemmStageB;
    gemm_fetch<MODE>(gl, min(t + 2, TS - 1), wsc, gsm + ((t + 2) % 3) * SB);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      // int8: 32-deep step, chunk 2 s + h; E4M3: 64-deep step, chunks 4 s + 2 h
      // and the next; MXFP4: 64-deep step s of the stage, chunk 2 s + h (32
      // E2M1 values, one MX block)
#pragma unroll
      for (int f = 0; f < FW; ++f) {
        const int c = MODE == 1 ? 4 * s + 2 * h + f : 2 * s + h;
#pragma unroll
        for (int a = 0; a < 2; ++a) fa[s][a][f] = gemm_frag(stage, wm * 64 + a * 32 + (lane & 31), c);
#pragma unroll
        for (int b = 0; b < kGemmNB; ++b)
          fb[s][b][f] = gemm_frag(stage + kGemmStageA, wn * (kGemmN / 2) + b * 32 + (lane & 31), c);
      }
    }
    if constexpr (MODE == 2) {
#pragma unroll
      for (int a = 0; a < 2; ++a) xs[a] = mx_scales(side + kGemmSideXs, wm * 64 + a * 32 + (lane & 31), lane);
#pragma unroll
      for (int b = 0; b < kGemmNB; ++b)
        ws[b] = mx_scales(side + kGemmSideWs, wn * (kGemmN / 2) + b * 32 + (lane & 31), lane);
    }
    __builtin_amdgcn_sched_barrier(0);  // the reads issue first; the rescale runs under them
    // int8 / E4M3: a factor tile of tmask + 1 stages accumulates into the
    // partials, rescaled once, in the V phase that starts the next tile
    const bool first = RESCALE ? ((uint32_t)t & tmask) == 0u : t == 0;  // wave-uniform
    if constexpr (RESCALE) {
      if (first) {
        if (t > 0) gemm_rescale<MODE, 64>(0, cur, gcur, accf);
        gemm_side_g(side, wn, lane, gcur);
      }
    }
    phase();
    // M(t)
    if (first)
      gemm_mfma_pp<MODE, true>(fa, fb, xs, ws, cur);
    else
      gemm_mfma_pp<MODE, false>(fa, fb, xs, ws, cur);
  }
  if (grp == 0) phase();  // the same barrier count in both groups
  if constexpr (RESCALE) gemm_rescale<MODE, 64>(0, cur, gcur, accf);  // the last tile
  // every wave's re-fetches of the last stage have landed: the ring is free
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // The wave's 64 x 64 outputs, staged in LDS (its own region of the ring)
  // in the MFMA layout, then written out 16 bytes a lane along whole rows.
  int8_t* const tile = gsm + wsc * kGemmOutRegion;
  if (A.out_bf16)
    gemm_store_tile<MODE, true>(A, tile, cur, accf, m0 + wm * 64, n0 + wn * 64, lane);
  else
    gemm_store_tile<MODE, false>(A, tile, cur, accf, m0 + wm * 64, n0 + wn * 64, lane);
}

__global__ __launch_bounds__(kGemmThreads, 1) void hq_gemm_i8_kernel(hq_gemm_args A) {
  gemm_body_pp<0>(A);
}

__global__ __launch_bounds__(kGemmThreads, 1) void hq_gemm_f8_kernel(hq_gemm_args A) {
  gemm_body_pp<1>(A);
}

__global__ __launch_bounds__(kGemmThreads, 1) void hq_gemm_mx4_kernel(hq_gemm_args A) {
  gemm_body_pp<2>(A);
}

// ------------------------------------------------------------ utilities

__global__ void hq_zero_kernel(uint32_t* p, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

// Dynamic LDS above 64 KB needs a per-kernel opt-in, a costly runtime call:
// made when a launch needs more than the kernel's largest opt-in so far.
inline void allow_lds(const void* kernel, size_t bytes, size_t& granted) {
  if (bytes > 65536 && bytes > granted &&
      hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) ==
          hipSuccess)
    granted = bytes;
}

// One encode launch: a single matrix (hq_encode_args + thresholds; four or
// one sub-streams per wave) or a group (four per wave).
template <int LAT, int XT, bool KV>
void launch_encode_kernel(const hq_encode_args& a, const hq_rice_thr& t, uint32_t nwg,
                          uint32_t lds_words, hipStream_t st) {
  const size_t per_sub = (size_t)(lds_words + 2) * sizeof(uint32_t);
  const size_t lds = per_sub * HQ_ENC_SUBS_PER_WG;
  // the qjl rotation stages four tiles per wave after the sub-stream buffers
  const size_t stage = a.qjlt ? (size_t)HQ_QJL_STAGE * sizeof(float) : 0;
  if (a.spw == 1)
    hipLaunchKernelGGL((hq_encode_kernel<LAT, XT, KV, 1>), dim3(nwg), dim3(64 * HQ_ENC_SUBS_PER_WG),
                       lds + stage * HQ_ENC_SUBS_PER_WG, st, a, t);
  else
    hipLaunchKernelGGL((hq_encode_kernel<LAT, XT, KV, HQ_ENC_SUBS_PER_WAVE>), dim3(nwg),
                       dim3(64 * HQ_ENC_WAVES), lds + stage * HQ_ENC_WAVES, st, a, t);
}

template <int LAT, int XT, bool KV>
void launch_encode_kernel(const hq_encode_group_args& g, const hq_rice_thr&, uint32_t nwg,
                          uint32_t lds_words, hipStream_t st) {
  const size_t lds = (size_t)(lds_words + 2) * HQ_ENC_SUBS_PER_WG * sizeof(uint32_t);
  hipLaunchKernelGGL((hq_encode_group_kernel<LAT, XT, KV>), dim3(nwg), dim3(64 * HQ_ENC_WAVES), lds, st, g);
}

template <int LAT, typename Args>
int launch_encode_lat(const Args& a, const hq_rice_thr& t, uint32_t nwg, uint32_t lds_words, int xt,
                      bool kv, hipStream_t st) {
  if (xt == HQ_BF16) {
    if (kv)
      launch_encode_kernel<LAT, HQ_BF16, true>(a, t, nwg, lds_words, st);
    else
      launch_encode_kernel<LAT, HQ_BF16, false>(a, t, nwg, lds_words, st);
  } else {
    if (kv)
      launch_encode_kernel<LAT, HQ_FP32, true>(a, t, nwg, lds_words, st);
    else
      launch_encode_kernel<LAT, HQ_FP32, false>(a, t, nwg, lds_words, st);
  }
  return (int)hipGetLastError();
}

// One decode launch: a single matrix (hq_decode_args) or a group.
template <int LAT, int MODE, bool KV, typename Args>
void launch_decode_kernel(const Args& a, uint32_t nwg, size_t lds, hipStream_t st) {
  static size_t granted = 0;
  allow_lds(sizeof(Args) == sizeof(hq_decode_args) ? (const void*)hq_decode_kernel<LAT, MODE, KV>
                                                   : (const void*)hq_decode_group_kernel<LAT, MODE, KV>,
            lds, granted);
  if constexpr (sizeof(Args) == sizeof(hq_decode_args))
    hipLaunchKernelGGL((hq_decode_kernel<LAT, MODE, KV>), dim3(nwg), dim3(256), lds, st, a);
  else
    hipLaunchKernelGGL((hq_decode_group_kernel<LAT, MODE, KV>), dim3(nwg), dim3(256), lds, st, a);
}

template <int LAT, typename Args>
int launch_decode_lat(const Args& a, uint32_t nwg, uint32_t lds_words, int mode, bool kv,
                      hipStream_t st) {
  size_t lds = (size_t)(lds_words + 66) * HQ_WAVES_PER_WG * sizeof(uint32_t);
  if constexpr (sizeof(Args) == sizeof(hq_decode_args))
    if (a.qjl)  // qjl: the waves' stages, then a copy of S (over 64 KB in all: opt in)
      lds += ((size_t)HQ_QJL_STAGE * HQ_WAVES_PER_WG + (size_t)HQ_TILE * HQ_TILE) * sizeof(float);
  if (mode == 0) {
    if (kv) launch_decode_kernel<LAT, 0, true>(a, nwg, lds, st);
    else launch_decode_kernel<LAT, 0, false>(a, nwg, lds, st);
  } else if (mode == 1) {
    if (kv) launch_decode_kernel<LAT, 1, true>(a, nwg, lds, st);
    else launch_decode_kernel<LAT, 1, false>(a, nwg, lds, st);
  } else {
    if (kv) launch_decode_kernel<LAT, 2, true>(a, nwg, lds, st);
    else launch_decode_kernel<LAT, 2, false>(a, nwg, lds, st);
  }
  return (int)hipGetLastError();
}

// Long tiles, or sub-streams of several blocks (weight plans): four
// consecutive 512-symbol blocks per wave.
template <int LAT, int XT, int MB>
int launch_encode_tiled_mb(const hq_encode_args& a, const hq_rice_thr& t, hipStream_t st) {
  const size_t lds = (size_t)(a.lds_words + 2) * HQ_ENC_SUBS_PER_WG * sizeof(uint32_t);
  static size_t granted = 0;
  allow_lds((const void*)hq_encode_tiled_kernel<LAT, XT, MB>, lds, granted);
  hipLaunchKernelGGL((hq_encode_tiled_kernel<LAT, XT, MB>), dim3(a.nwg), dim3(64 * HQ_ENC_WAVES), lds, st,
                     a, t);
  return (int)hipGetLastError();
}

template <int LAT>
int launch_encode_tiled(const hq_encode_args& a, const hq_rice_thr& t, int xt, hipStream_t st) {
  if (xt == HQ_BF16) {
    if (a.mb == 4) return launch_encode_tiled_mb<LAT, HQ_BF16, 4>(a, t, st);
    if (a.mb == 2) return launch_encode_tiled_mb<LAT, HQ_BF16, 2>(a, t, st);
    return launch_encode_tiled_mb<LAT, HQ_BF16, 1>(a, t, st);
  }
  if (a.mb == 4) return launch_encode_tiled_mb<LAT, HQ_FP32, 4>(a, t, st);
  if (a.mb == 2) return launch_encode_tiled_mb<LAT, HQ_FP32, 2>(a, t, st);
  return launch_encode_tiled_mb<LAT, HQ_FP32, 1>(a, t, st);
}

template <int LAT>
int launch_decode_tiled(const hq_decode_args& a, uint32_t nwg, int mode, hipStream_t st) {
  const size_t lds = (size_t)(a.lds_words + 66) * HQ_WAVES_PER_WG * sizeof(uint32_t);
  static size_t granted_0 = 0, granted_1 = 0;
  if (mode == 0) {
    allow_lds((const void*)hq_decode_tiled_kernel<LAT, 0>, lds, granted_0);
    hipLaunchKernelGGL((hq_decode_tiled_kernel<LAT, 0>), dim3(nwg), dim3(256), lds, st, a);
  } else {
    allow_lds((const void*)hq_decode_tiled_kernel<LAT, 1>, lds, granted_1);
    hipLaunchKernelGGL((hq_decode_tiled_kernel<LAT, 1>), dim3(nwg), dim3(256), lds, st, a);
  }
  return (int)hipGetLastError();
}

}  // namespace

static bool kv_variant(const hq_plan_s* p) { return p->rotation || p->dither || p->norm_fp16; }

int hq_launch_encode(const hq_plan_s* p, const hq_encode_args& a, const hq_rice_thr& t, int xt,
                     void* stream) {
  hipStream_t st = (hipStream_t)stream;
  if (p->tile != HQ_TILE || p->substream != HQ_SUB) {  // long tiles, or sub-streams of 2 or 4 blocks
    switch (p->lattice) {
      case HQ_E8: return launch_encode_tiled<kE8>(a, t, xt, st);
      case HQ_D4: return launch_encode_tiled<kD4>(a, t, xt, st);
      case HQ_A2: return launch_encode_tiled<kA2>(a, t, xt, st);
      default: return launch_encode_tiled<kZ>(a, t, xt, st);
    }
  }
  const bool kv = kv_variant(p);
  const uint32_t lw = a.lds_words;
  switch (p->lattice) {
    case HQ_E8: return launch_encode_lat<kE8>(a, t, a.nwg, lw, xt, kv, st);
    case HQ_D4: return launch_encode_lat<kD4>(a, t, a.nwg, lw, xt, kv, st);
    case HQ_A2: return launch_encode_lat<kA2>(a, t, a.nwg, lw, xt, kv, st);
    default: return launch_encode_lat<kZ>(a, t, a.nwg, lw, xt, kv, st);
  }
}

int hq_launch_encode_group(const hq_plan_s* p, const hq_encode_group_args& g, uint32_t nwg,
                           uint32_t lds_words, int xt, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const bool kv = kv_variant(p);
  switch (p->lattice) {
    case HQ_E8: return launch_encode_lat<kE8>(g, g.thr, nwg, lds_words, xt, kv, st);
    case HQ_D4: return launch_encode_lat<kD4>(g, g.thr, nwg, lds_words, xt, kv, st);
    case HQ_A2: return launch_encode_lat<kA2>(g, g.thr, nwg, lds_words, xt, kv, st);
    default: return launch_encode_lat<kZ>(g, g.thr, nwg, lds_words, xt, kv, st);
  }
}

static uint32_t decode_wgs(int64_t nsub) {
  constexpr int per_wg = HQ_WAVES_PER_WG * HQ_DEC_SUBS_PER_WAVE;
  return (uint32_t)((nsub + per_wg - 1) / per_wg);
}

// qjl streams of tile 128: the matrix-core decode, a grid of workgroups
// that each take every gridDim-th pass of 16 sub-streams.
template <int LAT>
int launch_decode_qjl(const hq_decode_args& a, int mode, hipStream_t st) {
  const int64_t ngroups = (a.nsub + 15) / 16;
  if (ngroups == 0) return 0;
  const uint32_t nwg = (uint32_t)std::min<int64_t>(ngroups, 2048);
  const size_t lds = (size_t)(a.lds_words + 66) * HQ_WAVES_PER_WG * sizeof(uint32_t) +
                     (size_t)kQjlTiles * kQjlRow * sizeof(float);
  static size_t granted0 = 0, granted1 = 0;
  if (mode == 0) {
    allow_lds((const void*)hq_decode_qjl_kernel<LAT, 0>, lds, granted0);
    hipLaunchKernelGGL((hq_decode_qjl_kernel<LAT, 0>), dim3(nwg), dim3(256), lds, st, a);
  } else {
    allow_lds((const void*)hq_decode_qjl_kernel<LAT, 1>, lds, granted1);
    hipLaunchKernelGGL((hq_decode_qjl_kernel<LAT, 1>), dim3(nwg), dim3(256), lds, st, a);
  }
  return (int)hipGetLastError();
}

// A single matrix of fewer than HQ_DEC_SMALL sub-streams, fp32 or bf16 out:
// one sub-stream per wave, so that its workgroups spread over more of the
// chip than four per wave would.
template <int LAT>
int launch_decode_small(const hq_decode_args& a, int mode, bool kv, hipStream_t st) {
  const uint32_t nwg = (uint32_t)((a.nsub + HQ_WAVES_PER_WG - 1) / HQ_WAVES_PER_WG);
  const size_t lds = (size_t)(a.lds_words + 66) * HQ_WAVES_PER_WG * sizeof(uint32_t);
  static size_t granted[4] = {0, 0, 0, 0};
#define HQ_SMALL_CASE(M, K, I)                                                             \
  allow_lds((const void*)hq_decode_small_kernel<LAT, M, K>, lds, granted[I]);              \
  hipLaunchKernelGGL((hq_decode_small_kernel<LAT, M, K>), dim3(nwg), dim3(256), lds, st, a)
  if (mode == 0) {
    if (kv) { HQ_SMALL_CASE(0, true, 0); } else { HQ_SMALL_CASE(0, false, 1); }
  } else {
    if (kv) { HQ_SMALL_CASE(1, true, 2); } else { HQ_SMALL_CASE(1, false, 3); }
  }
#undef HQ_SMALL_CASE
  return (int)hipGetLastError();
}

int hq_launch_decode(const hq_plan_s* p, const hq_decode_args& a, int yt, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const int mode = (yt == HQ_FP32) ? 0 : 1;
  const bool kv = kv_variant(p);
  const uint32_t nwg = decode_wgs(a.nsub * a.mb), lw = a.lds_words;
  if (a.qjl && p->tile == HQ_TILE && p->substream == HQ_SUB) {
    switch (p->lattice) {
      case HQ_E8: return launch_decode_qjl<kE8>(a, mode, st);
      case HQ_D4: return launch_decode_qjl<kD4>(a, mode, st);
      case HQ_A2: return launch_decode_qjl<kA2>(a, mode, st);
      default: return launch_decode_qjl<kZ>(a, mode, st);
    }
  }
  if (!a.qjl && a.nsub < HQ_DEC_SMALL && p->tile == HQ_TILE && p->substream == HQ_SUB) {
    if (a.nsub == 0) return 0;
    switch (p->lattice) {
      case HQ_E8: return launch_decode_small<kE8>(a, mode, kv, st);
      case HQ_D4: return launch_decode_small<kD4>(a, mode, kv, st);
      case HQ_A2: return launch_decode_small<kA2>(a, mode, kv, st);
      default: return launch_decode_small<kZ>(a, mode, kv, st);
    }
  }
  if (p->tile != HQ_TILE || p->substream != HQ_SUB) {
    switch (p->lattice) {
      case HQ_E8: return launch_decode_tiled<kE8>(a, nwg, mode, st);
      case HQ_D4: return launch_decode_tiled<kD4>(a, nwg, mode, st);
      case HQ_A2: return launch_decode_tiled<kA2>(a, nwg, mode, st);
      default: return launch_decode_tiled<kZ>(a, nwg, mode, st);
    }
  }
  switch (p->lattice) {
    case HQ_E8: return launch_decode_lat<kE8>(a, nwg, lw, mode, kv, st);
    case HQ_D4: return launch_decode_lat<kD4>(a, nwg, lw, mode, kv, st);
    case HQ_A2: return launch_decode_lat<kA2>(a, nwg, lw, mode, kv, st);
    default: return launch_decode_lat<kZ>(a, nwg, lw, mode, kv, st);
  }
}

int hq_launch_decode_group(const hq_plan_s* p, const hq_decode_group_args& g, uint32_t nwg,
                           uint32_t lds_words, int yt, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const int mode = (yt == HQ_FP32) ? 0 : 1;
  const bool kv = kv_variant(p);
  switch (p->lattice) {
    case HQ_E8: return launch_decode_lat<kE8>(g, nwg, lds_words, mode, kv, st);
    case HQ_D4: return launch_decode_lat<kD4>(g, nwg, lds_words, mode, kv, st);
    case HQ_A2: return launch_decode_lat<kA2>(g, nwg, lds_words, mode, kv, st);
    default: return launch_decode_lat<kZ>(g, nwg, lds_words, mode, kv, st);
  }
}

uint32_t hq_decode_workgroups(int64_t nsub) { return decode_wgs(nsub); }

int hq_launch_decode_int8(const hq_plan_s* p, const hq_decode_args& a, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const bool kv = kv_variant(p);
  switch (p->lattice) {
    case HQ_E8: return launch_decode_lat<kE8>(a, decode_wgs(a.nsub), a.lds_words, 2, kv, st);
    case HQ_D4: return launch_decode_lat<kD4>(a, decode_wgs(a.nsub), a.lds_words, 2, kv, st);
    default: return launch_decode_lat<kZ>(a, decode_wgs(a.nsub), a.lds_words, 2, kv, st);
  }
}

int hq_launch_act_prep(const hq_actprep_args& a, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const size_t lds = (size_t)a.K * sizeof(float);
  hipLaunchKernelGGL(hq_act_prep_kernel, dim3((uint32_t)a.M), dim3(256), lds, st, a);
  return (int)hipGetLastError();
}

int hq_launch_gemm(const hq_gemm_args& a, void* stream) {
  if (a.K % 256 != 0) return -1;  // an even number of 128-deep K tiles
  static bool lds_set = false;  // more than 64 KB of dynamic LDS needs an opt-in
  if (!lds_set) {
    hipError_t e = hipFuncSetAttribute((const void*)hq_gemm_i8_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, gemm_lds_bytes<0>());
    if (e == hipSuccess)
      e = hipFuncSetAttribute((const void*)hq_gemm_f8_kernel,
                              hipFuncAttributeMaxDynamicSharedMemorySize, gemm_lds_bytes<1>());
    if (e == hipSuccess)
      e = hipFuncSetAttribute((const void*)hq_gemm_mx4_kernel,
                              hipFuncAttributeMaxDynamicSharedMemorySize, gemm_lds_bytes<2>());
    if (e != hipSuccess) return (int)e;
    lds_set = true;
  }
  const dim3 grid((uint32_t)((a.N + kGemmN - 1) / kGemmN), (uint32_t)((a.M + kGemmM - 1) / kGemmM));
  hipStream_t st = (hipStream_t)stream;
  if (a.fp8 == 2)
    hipLaunchKernelGGL(hq_gemm_mx4_kernel, grid, dim3(kGemmThreads), gemm_lds_bytes<2>(), st, a);
  else if (a.fp8)
    hipLaunchKernelGGL(hq_gemm_f8_kernel, grid, dim3(kGemmThreads), gemm_lds_bytes<1>(), st, a);
  else
    hipLaunchKernelGGL(hq_gemm_i8_kernel, grid, dim3(kGemmThreads), gemm_lds_bytes<0>(), st, a);
  return (int)hipGetLastError();
}

int hq_launch_decode_mxfp4(const hq_plan_s* p, const hq_decode_args& a, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const size_t lds = (size_t)(a.lds_words + 66) * HQ_WAVES_PER_WG * sizeof(uint32_t);
  const uint32_t nwg = decode_wgs(a.nsub);
  switch (p->lattice) {
    case HQ_E8: launch_decode_kernel<kE8, 4, false>(a, nwg, lds, st); break;
    case HQ_D4: launch_decode_kernel<kD4, 4, false>(a, nwg, lds, st); break;
    default: launch_decode_kernel<kZ, 4, false>(a, nwg, lds, st);
  }
  return (int)hipGetLastError();
}

int hq_launch_decode_fp8(const hq_plan_s* p, const hq_decode_args& a, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const size_t lds = (size_t)(a.lds_words + 66) * HQ_WAVES_PER_WG * sizeof(uint32_t);
  const uint32_t nwg = decode_wgs(a.nsub);
  switch (p->lattice) {
    case HQ_E8: launch_decode_kernel<kE8, 3, false>(a, nwg, lds, st); break;
    case HQ_D4: launch_decode_kernel<kD4, 3, false>(a, nwg, lds, st); break;
    default: launch_decode_kernel<kZ, 3, false>(a, nwg, lds, st);
  }
  return (int)hipGetLastError();
}

int hq_launch_zero(void* ptr, size_t bytes, void* stream) {
  const size_t n = bytes / 4;
  if (n == 0) return 0;
  hipLaunchKernelGGL(hq_zero_kernel, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0,
                     (hipStream_t)stream, (uint32_t*)ptr, n);
  return (int)hipGetLastError();
}

// ------------------------------------------------------------ fixed scratch
// The look-back scratch of hq_encode_noalloc, for callers that cannot
// allocate: one array per device, alive until the process ends.  Host code
// never passes the array's name to a kernel (on the host it is a stand-in,
// not a device address); it uses the address hipGetSymbolAddress returns for
// the current device, looked up once per device.
static __device__ __align__(256) unsigned char scratch[HQ_NOALLOC_SCAN_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];
}  // namespace

int hq_noalloc_scan(void** ptr, void* stream) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return -1;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return -1;
    // the epoch word and every status word start at zero (a fill kernel, so
    // a first call under graph capture records no memset node)
    if (hq_launch_zero(p, HQ_NOALLOC_SCAN_BYTES, stream) != 0) return -1;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return 0;
}

int hq_launch_decode_gemv(const hq_plan_s* p, const hq_decode_args& a, const void* x, int xt,
                          float* xtr, void* y, int yt, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const int64_t K = p->cols;
  hipLaunchKernelGGL(hq_gemv_prep_kernel, dim3((uint32_t)((K + 4 * HQ_SUB - 1) / (4 * HQ_SUB))),
                     dim3(256), 0, st, x, xt == HQ_BF16 ? 1 : 0, K, a.dmask, xtr);
  const int64_t rows = a.nsub / a.spr;
  const size_t lds = (size_t)(a.lds_words + 66) * HQ_WAVES_PER_WG * sizeof(uint32_t);
  const int yb = yt == HQ_BF16 ? 1 : 0;
  if (rows >= HQ_GEMV_WAVE_ROWS) {  // enough rows to fill the chip one wave each
    const uint32_t nwr = (uint32_t)((rows + HQ_WAVES_PER_WG - 1) / HQ_WAVES_PER_WG);
    switch (p->lattice) {
      case HQ_E8:
        hipLaunchKernelGGL(hq_decode_gemv_rows_kernel<kE8>, dim3(nwr), dim3(256), lds, st, a, xtr, y, yb, rows);
        break;
      case HQ_D4:
        hipLaunchKernelGGL(hq_decode_gemv_rows_kernel<kD4>, dim3(nwr), dim3(256), lds, st, a, xtr, y, yb, rows);
        break;
      case HQ_A2:
        hipLaunchKernelGGL(hq_decode_gemv_rows_kernel<kA2>, dim3(nwr), dim3(256), lds, st, a, xtr, y, yb, rows);
        break;
      default:
        hipLaunchKernelGGL(hq_decode_gemv_rows_kernel<kZ>, dim3(nwr), dim3(256), lds, st, a, xtr, y, yb, rows);
    }
    return (int)hipGetLastError();
  }
  const uint32_t nwg = (uint32_t)rows;  // one workgroup per row
  switch (p->lattice) {
    case HQ_E8:
      hipLaunchKernelGGL(hq_decode_gemv_kernel<kE8>, dim3(nwg), dim3(256), lds, st, a, xtr, y, yb);
      break;
    case HQ_D4:
      hipLaunchKernelGGL(hq_decode_gemv_kernel<kD4>, dim3(nwg), dim3(256), lds, st, a, xtr, y, yb);
      break;
    case HQ_A2:
      hipLaunchKernelGGL(hq_decode_gemv_kernel<kA2>, dim3(nwg), dim3(256), lds, st, a, xtr, y, yb);
      break;
    default:
      hipLaunchKernelGGL(hq_decode_gemv_kernel<kZ>, dim3(nwg), dim3(256), lds, st, a, xtr, y, yb);
  }
  return (int)hipGetLastError();
}

int hq_launch_decode_attention(const hq_attn_args& a, int lattice, void* stream) {
  const hipStream_t st = (hipStream_t)stream;
  const uint32_t heads = (uint32_t)((a.batch * a.heads_q + 15) / 16);
  hipLaunchKernelGGL(hq_attn_prep_kernel, dim3(heads), dim3(256), 0, st, a);
  const uint32_t nwg = (uint32_t)(a.batch * a.K.spr * a.nx);
  const size_t lds_k = (size_t)HQ_WAVES_PER_WG * (a.lds_words + 66) * 4;
  const size_t lds_v = lds_k + (size_t)(HQ_WAVES_PER_WG - 1) * 64 * 8 * a.group * 4;
#define HQ_ATTN_CASE(L, GG)                                                                  \
  hipLaunchKernelGGL((hq_attn_kernel<L, GG, false>), dim3(nwg), dim3(256), lds_k, st, a); \
  hipLaunchKernelGGL((hq_attn_kernel<L, GG, true>), dim3(nwg), dim3(256), lds_v, st, a)
#define HQ_ATTN_GROUPS(L)           \
  switch (a.group) {                \
    case 1: HQ_ATTN_CASE(L, 1); break; \
    case 2: HQ_ATTN_CASE(L, 2); break; \
    case 4: HQ_ATTN_CASE(L, 4); break; \
    default: HQ_ATTN_CASE(L, 8);    \
  }
  switch (lattice) {
    case HQ_E8: HQ_ATTN_GROUPS(kE8); break;
    case HQ_D4: HQ_ATTN_GROUPS(kD4); break;
    case HQ_A2: HQ_ATTN_GROUPS(kA2); break;
    default: HQ_ATTN_GROUPS(kZ);
  }
#undef HQ_ATTN_GROUPS
#undef HQ_ATTN_CASE
  hipLaunchKernelGGL(hq_attn_combine_kernel, dim3((uint32_t)(a.batch * a.heads_q)), dim3(256), 0,
                     st, a);
  return (int)hipGetLastError();
}
