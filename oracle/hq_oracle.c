/*
 * HyperQuant codec oracle.  TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU statement of what the HyperQuant codec
 * computes ("HyperQuant: A Rate-Distortion-Optimal Quantization Pipeline for
 * Large Language and Diffusion Models"), written step by step in the order of
 * the paper's pipeline figure (Sec. 4, Fig. 1):
 *
 *   encode:  RHT (eq. rht, Sec. 3.1, 4.1) -> Rotate (Sec. 4.2) -> Normalize
 *            (Sec. 4.3) -> Add dither (Sec. 4.4, App. A) -> Quantize to the
 *            integer lattice realization (Sec. 4.5, Tab. lattices-int) ->
 *            Strip + zig-zag (Sec. 4.6) -> Rice (Sec. 3.3, 4.7) grouped into
 *            offset-indexed sub-streams (Sec. 5.3)
 *   decode:  the exact inverse of every block, then the inverse RHT
 *   GEMM:    block-scaled int8 product on post-RHT lattice codes (Sec. 4.8,
 *            Sec. 6.3), in exact integer / fp64 arithmetic.
 *
 * Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
 * load this library.  It shares no code, header, table or helper with the HIP
 * path, and nothing here is tuned: every step is the plain definition.
 *
 * Readings of points the paper leaves open (the per-tile floating-point
 * order, the seed hash, the bitstream layout, the k policy, the dither
 * counter) are listed in the design notes; each function below says which
 * passage it follows.
 *
 * Parity unpinned (no paper value to check against, only self-consistency):
 * the seed-to-sign hash, the dither counter layout, and the sub-stream bit
 * layout.  Everything else is pinned by the tests under tests/.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define HQO_E8 0
#define HQO_D4 1
#define HQO_A2 2
#define HQO_Z 3

#define HQO_OK 0
#define HQO_ERR_ARG -1
#define HQO_ERR_CAPACITY -3
#define HQO_ERR_OVERFLOW -4
#define HQO_ERR_CORRUPT -6

#define HQO_KMAX 15

/* fp32 nearest value of sqrt(3) and of 1/(2 sqrt(3)) (Sec. 4.5: the A2
   realization scales its y axis by sqrt(3)). */
#define HQO_SQRT3F 1.7320508075688772f
#define HQO_INV2SQRT3F 0.28867513459481287f

typedef struct {
  int32_t tile;        /* n_tile, a power of two (Sec. 4.1) */
  int32_t lattice;     /* HQO_E8 / D4 / A2 / Z */
  int32_t substream;   /* S symbols per sub-stream (Sec. 5.3) */
  int32_t rice_k;      /* >= 0 fixed, -1 = per-sub-stream optimum (Sec. 3.3) */
  float alpha;         /* scale realizing the SNR (App. B eq. alpha-calib) */
  int32_t norm_fp16;   /* store per-tile norms as fp16 (Sec. 6.6 KV) */
  uint64_t rht_seed;   /* sign diagonal D of eq. rht */
  int32_t rotation;    /* 0 = none, 1 = signs, 2 = qjl (Sec. 4.2) */
  int32_t dither;      /* subtractive dither on/off (Sec. 4.4) */
  uint64_t rot_seed;
  uint64_t dither_seed;
  const float* qjl;    /* rotation 2: the n x n orthogonal S, row-major (the
                          Haar draw of Sec. 4.2, supplied by the caller) */
} hqo_params;

/* ------------------------------------------------------------------------ */
/* Lattice constants (Sec. 3.2 Tab. lattice-constants; Sec. 4.5).           */
/* ------------------------------------------------------------------------ */

int hqo_lattice_dim(int lat) {
  switch (lat) {
    case HQO_E8: return 8;
    case HQO_D4: return 4;
    case HQO_A2: return 2;
    case HQO_Z: return 1;
  }
  return 0;
}

/* Normalized second moment G of the lattice (Tab. lattice-constants), the
   textbook closed forms whose 4-digit roundings the table prints. */
double hqo_nsm(int lat) {
  switch (lat) {
    case HQO_E8: return 929.0 / 12960.0;
    case HQO_D4: return 13.0 / (120.0 * sqrt(2.0));
    case HQO_A2: return 5.0 / (36.0 * sqrt(3.0));
    case HQO_Z: return 1.0 / 12.0;
  }
  return 0.0;
}

/* Covolume of the integer realization (Sec. 4.5): 2E8 has 2^8, D4 has 2,
   {(sqrt3 ny, nx): ny = nx mod 2} has 2 sqrt3, Z has 1. */
double hqo_covolume(int lat) {
  switch (lat) {
    case HQO_E8: return 256.0;
    case HQO_D4: return 2.0;
    case HQO_A2: return 2.0 * sqrt(3.0);
    case HQO_Z: return 1.0;
  }
  return 0.0;
}

/* App. B eq. alpha-calib: alpha = sqrt(SNR_lin * G * V^(2/N)), N the lattice
   dimension, evaluated in fp64 and rounded once to fp32. */
double hqo_alpha64(int lat, double snr_db) {
  double snr_lin = pow(10.0, snr_db / 10.0);
  double m = (double)hqo_lattice_dim(lat);
  return sqrt(snr_lin * hqo_nsm(lat) * pow(hqo_covolume(lat), 2.0 / m));
}

float hqo_alpha(int lat, double snr_db) { return (float)hqo_alpha64(lat, snr_db); }

/* ------------------------------------------------------------------------ */
/* Counter-based generators, each from its published definition.            */
/* ------------------------------------------------------------------------ */

/* SplitMix64 (Steele, Lea, Flood, OOPSLA 2014): the j-th output (j >= 0) of
   the generator seeded with `seed` is mix(seed + (j+1) * golden_gamma). */
uint64_t hqo_splitmix64(uint64_t seed, uint64_t j) {
  uint64_t z = seed + (j + 1) * 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* The iid uniform +-1 diagonal of eq. rht, indexed by global column j:
   -1 when the top bit of the j-th SplitMix64 output is set. */
int hqo_sign(uint64_t seed, int64_t j) {
  return (hqo_splitmix64(seed, (uint64_t)j) >> 63) ? -1 : 1;
}

/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11), the counter-based
   generator that draws the dither (Sec. 4.4). */
void hqo_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
  uint32_t k[2] = {key_in[0], key_in[1]};
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k[0] += 0x9E3779B9u;
      k[1] += 0xBB67AE85u;
    }
    uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c[0];
    uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c[2];
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c[1] ^ k[0];
    uint32_t n2 = hi0 ^ c[3] ^ k[1];
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
  out[0] = c[0];
  out[1] = c[1];
  out[2] = c[2];
  out[3] = c[3];
}

/* 24 random bits for coordinate (row, col): Philox word (col mod 4) of the
   block with counter (col / 4, row_lo, row_hi, 0) and key (seed_lo, seed_hi). */
static uint32_t dither_bits24(uint64_t seed, int64_t row, int64_t col) {
  uint32_t ctr[4] = {(uint32_t)((uint64_t)col >> 2), (uint32_t)(uint64_t)row,
                     (uint32_t)((uint64_t)row >> 32), 0u};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t out[4];
  hqo_philox4x32_10(ctr, key, out);
  return out[col & 3] >> 8;
}

/* ------------------------------------------------------------------------ */
/* RHT (eq. rht): unnormalized Sylvester Walsh-Hadamard, natural order,     */
/* butterfly stages h = 1, 2, ..., n/2 with (a, b) -> (a + b, a - b).       */
/* ------------------------------------------------------------------------ */

void hqo_fwht_f32(float* v, int n) {
  for (int h = 1; h < n; h <<= 1)
    for (int i = 0; i < n; i += 2 * h)
      for (int j = i; j < i + h; ++j) {
        float a = v[j], b = v[j + h];
        v[j] = a + b;
        v[j + h] = a - b;
      }
}

void hqo_fwht_f64(double* v, int n) {
  for (int h = 1; h < n; h <<= 1)
    for (int i = 0; i < n; i += 2 * h)
      for (int j = i; j < i + h; ++j) {
        double a = v[j], b = v[j + h];
        v[j] = a + b;
        v[j + h] = a - b;
      }
}

void hqo_fwht_i64(int64_t* v, int n) {
  for (int h = 1; h < n; h <<= 1)
    for (int i = 0; i < n; i += 2 * h)
      for (int j = i; j < i + h; ++j) {
        int64_t a = v[j], b = v[j + h];
        v[j] = a + b;
        v[j + h] = a - b;
      }
}

/* Sum of buf[0..n) as a pairwise tree in index order:
   ((b0 + b1) + (b2 + b3)) + ...; buf is overwritten. */
static float tree_sum_f32(float* buf, int n) {
  for (int w = 1; w < n; w <<= 1)
    for (int i = 0; i < n; i += 2 * w) buf[i] = buf[i] + buf[i + w];
  return buf[0];
}

/* ------------------------------------------------------------------------ */
/* fp16 storage of KV norms (Sec. 6.6: float16 per-vector L2 norm).         */
/* ------------------------------------------------------------------------ */

/* IEEE binary16 encoding of a non-negative finite float, round to nearest
   even; returns 0x7C00 (inf) on overflow. */
uint16_t hqo_f32_to_f16(float f) {
  double x = (double)f; /* exact */
  if (x != x) return 0x7E00;
  int sign = x < 0;
  if (sign) x = -x;
  uint16_t s = sign ? 0x8000 : 0;
  if (x == 0.0) return s;
  /* Candidates on the binary16 grid: the spacing is 2^(e-10) for normal
     exponents e in [-14, 15], and 2^-24 below 2^-14. */
  int e;
  frexp(x, &e); /* x = f * 2^e, f in [0.5, 1) -> x in [2^(e-1), 2^e) */
  int ex = e - 1;
  if (ex < -14) ex = -14;
  double ulp = ldexp(1.0, ex - 10);
  double q = x / ulp; /* exact: power-of-two division */
  double r = floor(q);
  double frac = q - r;
  if (frac > 0.5 || (frac == 0.5 && fmod(r, 2.0) != 0.0)) r += 1.0;
  double v = r * ulp;
  if (v >= 65520.0 || v > 65504.0) return (uint16_t)(s | 0x7C00);
  /* re-encode v */
  if (v < ldexp(1.0, -14)) {
    return (uint16_t)(s | (uint16_t)(v / ldexp(1.0, -24)));
  }
  int e2;
  double f2 = frexp(v, &e2);
  int bexp = e2 - 1 + 15;
  uint16_t mant = (uint16_t)((f2 * 2.0 - 1.0) * 1024.0);
  return (uint16_t)(s | (uint16_t)(bexp << 10) | mant);
}

float hqo_f16_to_f32(uint16_t h) {
  int sign = h >> 15;
  int e = (h >> 10) & 31;
  int m = h & 1023;
  double v;
  if (e == 0)
    v = ldexp((double)m, -24);
  else if (e == 31)
    v = m ? NAN : INFINITY;
  else
    v = ldexp(1024.0 + m, e - 25);
  return (float)(sign ? -v : v);
}

/* ------------------------------------------------------------------------ */
/* Nearest-point decoders (Sec. 3.2 "Nearest-neighbor decoding",            */
/* Conway & Sloane ch. 20) on the integer realizations of Sec. 4.5.          */
/* Every rint is round-half-even; argmax ties go to the lowest index.        */
/* ------------------------------------------------------------------------ */

static int argmax_abs(const float* e, int m) {
  int j = 0;
  float best = fabsf(e[0]);
  for (int i = 1; i < m; ++i)
    if (fabsf(e[i]) > best) {
      best = fabsf(e[i]);
      j = i;
    }
  return j;
}

/* Z: nearest integer. */
void hqo_q_z(const float* z, int32_t* c) { c[0] = (int32_t)rintf(z[0]); }

/* D4 = {c in Z^4 : sum c even}: round every coordinate; if the sum is odd,
   re-round the coordinate with the largest rounding error the other way. */
void hqo_q_d4(const float* z, int32_t* c) {
  float k[4], e[4];
  int32_t s = 0;
  for (int i = 0; i < 4; ++i) {
    k[i] = rintf(z[i]);
    e[i] = z[i] - k[i];
    c[i] = (int32_t)k[i];
    s += c[i];
  }
  if (s & 1) {
    int j = argmax_abs(e, 4);
    c[j] += (e[j] >= 0.0f) ? 1 : -1;
  }
}

/* 2E8 = 2D8 u (2D8 + 1), with 2D8 = {2k : k in Z^8, sum k even}.  The
   nearest point of each coset is found as for D_n (round, then fix the parity
   on the worst coordinate); the nearer of the two wins, the even coset on a
   tie. */
void hqo_q_e8(const float* z, int32_t* c) {
  int32_t ka[8], fb[8];
  float ea[8], eb[8];
  int32_t sa = 0, sb = 0;
  for (int i = 0; i < 8; ++i) {
    float h = z[i] * 0.5f;
    float k = rintf(h);
    float f = floorf(h);
    ka[i] = (int32_t)k;
    fb[i] = (int32_t)f;
    ea[i] = z[i] - 2.0f * k;
    eb[i] = z[i] - (2.0f * f + 1.0f);
    sa += ka[i];
    sb += fb[i];
  }
  if (sa & 1) {
    int j = argmax_abs(ea, 8);
    ka[j] += (ea[j] >= 0.0f) ? 1 : -1;
    ea[j] = z[j] - 2.0f * (float)ka[j];
  }
  if (sb & 1) {
    int j = argmax_abs(eb, 8);
    fb[j] += (eb[j] >= 0.0f) ? 1 : -1;
    eb[j] = z[j] - (2.0f * (float)fb[j] + 1.0f);
  }
  float sqa[8], sqb[8];
  for (int i = 0; i < 8; ++i) {
    sqa[i] = ea[i] * ea[i];
    sqb[i] = eb[i] * eb[i];
  }
  float da = tree_sum_f32(sqa, 8);
  float db = tree_sum_f32(sqb, 8);
  if (da <= db)
    for (int i = 0; i < 8; ++i) c[i] = 2 * ka[i];
  else
    for (int i = 0; i < 8; ++i) c[i] = 2 * fb[i] + 1;
}

/* A2 = {(sqrt3 ny, nx) : ny = nx mod 2}, the union of two rectangular
   cosets with spacing (2 sqrt3, 2); input (y, x) = (z0, z1); returns
   (ny, nx).  Coset 0 (both even) wins a tie. */
void hqo_q_a2(const float* z, int32_t* c) {
  float y = z[0], x = z[1];
  float a0 = rintf(y * HQO_INV2SQRT3F);
  float b0 = rintf(x * 0.5f);
  float a1 = rintf((y - HQO_SQRT3F) * HQO_INV2SQRT3F);
  float b1 = rintf((x - 1.0f) * 0.5f);
  int32_t ny0 = 2 * (int32_t)a0, nx0 = 2 * (int32_t)b0;
  int32_t ny1 = 2 * (int32_t)a1 + 1, nx1 = 2 * (int32_t)b1 + 1;
  float ey0 = y - HQO_SQRT3F * (float)ny0, ex0 = x - (float)nx0;
  float ey1 = y - HQO_SQRT3F * (float)ny1, ex1 = x - (float)nx1;
  float d0 = ey0 * ey0 + ex0 * ex0;
  float d1 = ey1 * ey1 + ex1 * ex1;
  if (d0 <= d1) {
    c[0] = ny0;
    c[1] = nx0;
  } else {
    c[0] = ny1;
    c[1] = nx1;
  }
}

void hqo_quantize_block(int lat, const float* z, int32_t* c) {
  switch (lat) {
    case HQO_E8: hqo_q_e8(z, c); break;
    case HQO_D4: hqo_q_d4(z, c); break;
    case HQO_A2: hqo_q_a2(z, c); break;
    case HQO_Z: hqo_q_z(z, c); break;
  }
}

/* Batch form: nblocks blocks of hqo_lattice_dim(lat) coordinates. */
void hqo_quantize(int lat, const float* z, int64_t nblocks, int32_t* c) {
  int m = hqo_lattice_dim(lat);
  for (int64_t b = 0; b < nblocks; ++b) hqo_quantize_block(lat, z + b * m, c + b * m);
}

/* Coordinates of a lattice code as a point of R^m, in fp64. */
static void point_f64(int lat, const int32_t* c, double* p) {
  int m = hqo_lattice_dim(lat);
  for (int i = 0; i < m; ++i) p[i] = (double)c[i];
  if (lat == HQO_A2) p[0] = sqrt(3.0) * (double)c[0];
}

/* ------------------------------------------------------------------------ */
/* Voronoi margin, fp64: the distance from z to the nearest face of the      */
/* Voronoi cell around the chosen point, min over the Voronoi-relevant       */
/* vectors v of (|v|^2 / 2 - <z - c, v>) / |v|.  Negative means c is not the */
/* nearest point.  Relevant vectors: the 240 minimal vectors of 2E8, the 24  */
/* of D4, the 6 of A2, and +-1 for Z.                                        */
/* ------------------------------------------------------------------------ */

static int relevant_vectors(int lat, double* out /* cap 240*8 */) {
  int m = hqo_lattice_dim(lat), cnt = 0;
  if (lat == HQO_E8) {
    for (int i = 0; i < 8; ++i)
      for (int j = i + 1; j < 8; ++j)
        for (int si = -1; si <= 1; si += 2)
          for (int sj = -1; sj <= 1; sj += 2) {
            double* v = out + cnt * m;
            memset(v, 0, sizeof(double) * m);
            v[i] = 2.0 * si;
            v[j] = 2.0 * sj;
            ++cnt;
          }
    for (int mask = 0; mask < 256; ++mask) {
      int neg = __builtin_popcount((unsigned)mask);
      if (neg & 1) continue;
      double* v = out + cnt * m;
      for (int i = 0; i < 8; ++i) v[i] = ((mask >> i) & 1) ? -1.0 : 1.0;
      ++cnt;
    }
  } else if (lat == HQO_D4) {
    for (int i = 0; i < 4; ++i)
      for (int j = i + 1; j < 4; ++j)
        for (int si = -1; si <= 1; si += 2)
          for (int sj = -1; sj <= 1; sj += 2) {
            double* v = out + cnt * m;
            memset(v, 0, sizeof(double) * m);
            v[i] = si;
            v[j] = sj;
            ++cnt;
          }
  } else if (lat == HQO_A2) {
    double s3 = sqrt(3.0);
    double vv[6][2] = {{0, 2}, {0, -2}, {s3, 1}, {s3, -1}, {-s3, 1}, {-s3, -1}};
    for (int i = 0; i < 6; ++i) {
      out[2 * i] = vv[i][0];
      out[2 * i + 1] = vv[i][1];
    }
    cnt = 6;
  } else {
    out[0] = 1.0;
    out[1] = -1.0;
    cnt = 2;
  }
  return cnt;
}

double hqo_margin(int lat, const float* z, const int32_t* c) {
  static double rv[4][240 * 8];
  static int nrv[4] = {0, 0, 0, 0};
  if (!nrv[lat]) nrv[lat] = relevant_vectors(lat, rv[lat]);
  int m = hqo_lattice_dim(lat);
  double p[8], d[8];
  point_f64(lat, c, p);
  for (int i = 0; i < m; ++i) d[i] = (double)z[i] - p[i];
  double best = INFINITY;
  for (int r = 0; r < nrv[lat]; ++r) {
    const double* v = rv[lat] + r * m;
    double vv = 0, dv = 0;
    for (int i = 0; i < m; ++i) {
      vv += v[i] * v[i];
      dv += d[i] * v[i];
    }
    double mg = (0.5 * vv - dv) / sqrt(vv);
    if (mg < best) best = mg;
  }
  return best;
}

void hqo_margins(int lat, const float* z, const int32_t* c, int64_t nblocks, double* out) {
  int m = hqo_lattice_dim(lat);
  for (int64_t b = 0; b < nblocks; ++b) out[b] = hqo_margin(lat, z + b * m, c + b * m);
}

/* ------------------------------------------------------------------------ */
/* Strip / unstrip (Sec. 4.6 table) and zig-zag.                             */
/* ------------------------------------------------------------------------ */

static uint32_t zz(int32_t v) { return v >= 0 ? 2u * (uint32_t)v : (uint32_t)(-2 * (int64_t)v - 1); }
static int32_t unzz(uint32_t m) { return (m & 1u) ? -(int32_t)((m + 1u) / 2u) : (int32_t)(m / 2u); }

uint32_t hqo_zigzag(int32_t v) { return zz(v); }
int32_t hqo_unzigzag(uint32_t m) { return unzz(m); }

/* One block of lattice codes -> the same number of non-negative symbols.
   E8: c = c0 mod 2, s_i = (c_i - c)/2, p = (s0+..+s6) mod 2, t = (s7 - p)/2,
   symbols zz(s0..s6) and comb = 2 zz(t) + c (the coset bit folded into the
   low bit freed by halving).  D4: p = (c0+c1+c2) mod 2, t = (c3 - p)/2.
   A2: p = nx mod 2, ty = (ny - p)/2, symbols (zz(ty), zz(nx)).  Z: zz(n). */
void hqo_strip_block(int lat, const int32_t* c, uint32_t* sym) {
  if (lat == HQO_E8) {
    int32_t cb = c[0] & 1, s[8], p = 0;
    for (int i = 0; i < 8; ++i) s[i] = (c[i] - cb) / 2;
    for (int i = 0; i < 7; ++i) p += s[i];
    p &= 1;
    int32_t t = (s[7] - p) / 2;
    for (int i = 0; i < 7; ++i) sym[i] = zz(s[i]);
    sym[7] = 2u * zz(t) + (uint32_t)cb;
  } else if (lat == HQO_D4) {
    int32_t p = (c[0] + c[1] + c[2]) & 1;
    int32_t t = (c[3] - p) / 2;
    sym[0] = zz(c[0]);
    sym[1] = zz(c[1]);
    sym[2] = zz(c[2]);
    sym[3] = zz(t);
  } else if (lat == HQO_A2) {
    int32_t p = c[1] & 1;
    int32_t ty = (c[0] - p) / 2;
    sym[0] = zz(ty);
    sym[1] = zz(c[1]);
  } else {
    sym[0] = zz(c[0]);
  }
}

void hqo_unstrip_block(int lat, const uint32_t* sym, int32_t* c) {
  if (lat == HQO_E8) {
    int32_t cb = (int32_t)(sym[7] & 1u);
    int32_t t = unzz(sym[7] >> 1);
    int32_t s[8], p = 0;
    for (int i = 0; i < 7; ++i) {
      s[i] = unzz(sym[i]);
      p += s[i];
    }
    p &= 1;
    s[7] = 2 * t + p;
    for (int i = 0; i < 8; ++i) c[i] = 2 * s[i] + cb;
  } else if (lat == HQO_D4) {
    c[0] = unzz(sym[0]);
    c[1] = unzz(sym[1]);
    c[2] = unzz(sym[2]);
    int32_t p = (c[0] + c[1] + c[2]) & 1;
    c[3] = 2 * unzz(sym[3]) + p;
  } else if (lat == HQO_A2) {
    c[1] = unzz(sym[1]);
    int32_t p = c[1] & 1;
    c[0] = 2 * unzz(sym[0]) + p;
  } else {
    c[0] = unzz(sym[0]);
  }
}

void hqo_strip(int lat, const int32_t* c, int64_t nblocks, uint32_t* sym) {
  int m = hqo_lattice_dim(lat);
  for (int64_t b = 0; b < nblocks; ++b) hqo_strip_block(lat, c + b * m, sym + b * m);
}

void hqo_unstrip(int lat, const uint32_t* sym, int64_t nblocks, int32_t* c) {
  int m = hqo_lattice_dim(lat);
  for (int64_t b = 0; b < nblocks; ++b) hqo_unstrip_block(lat, sym + b * m, c + b * m);
}

/* ------------------------------------------------------------------------ */
/* Rice parameter (Sec. 3.3): the optimum for a geometric source with        */
/* parameter p is floor(log2(ceil(-ln(2-p) / ln(1-p)))).                     */
/* ------------------------------------------------------------------------ */

int hqo_rice_kstar(double p) {
  if (p >= 1.0) return 0;
  double ratio = -log(2.0 - p) / log(1.0 - p);
  double c = ceil(ratio);
  if (!(c >= 1.0)) return 0;
  if (c > 9.0e15) return HQO_KMAX;
  int64_t ci = (int64_t)c;
  int k = 0;
  while (((int64_t)1 << (k + 1)) <= ci) ++k; /* floor(log2(ci)) */
  return k > HQO_KMAX ? HQO_KMAX : k;
}

/* Per-sub-stream automatic k: the geometric parameter is estimated from
   the class's symbol mean as p = count / (count + sum). */
int hqo_rice_k_auto(int64_t count, int64_t sum) {
  if (count <= 0) return 0;
  return hqo_rice_kstar((double)count / ((double)count + (double)sum));
}

/* Rice length of a symbol: floor(m / 2^k) in unary plus k raw bits. */
int64_t hqo_rice_length(uint32_t m, int k) { return (int64_t)(m >> k) + 1 + k; }

/* Rice class of the symbol at position `pos` inside its block: D4 codes its
   halved symbol t with its own level, A2 codes ty and nx separately. */
static int sym_class(int lat, int pos) {
  if (lat == HQO_D4) return pos == 3 ? 1 : 0;
  if (lat == HQO_A2) return pos == 1 ? 1 : 0;
  return 0;
}

/* Rice length of the symbols of class `cl` in one sub-stream at parameter k. */
static int64_t class_length(int lat, const uint32_t* sym, int S, int cl, int k) {
  int m = hqo_lattice_dim(lat);
  int64_t len = 0;
  for (int i = 0; i < S; ++i)
    if (sym_class(lat, i % m) == cl) len += hqo_rice_length(sym[i], k);
  return len;
}

static int class_kstar(int lat, const uint32_t* sym, int S, int cl) {
  int m = hqo_lattice_dim(lat);
  int64_t cnt = 0, sum = 0;
  for (int i = 0; i < S; ++i)
    if (sym_class(lat, i % m) == cl) {
      cnt += 1;
      sum += sym[i];
    }
  return hqo_rice_k_auto(cnt, sum);
}

/* Rice parameters of one sub-stream of S symbols; returns the kparam byte
   (low nibble k of class 0, high nibble k of class 1 for A2).
   Automatic k ("empirically calibrated", Sec. 3.3 and App. B): start from
   the geometric optimum k* of the class's symbol mean, then keep whichever
   of k* and k* + 1 codes the sub-stream's symbols in fewer bits (k* on a
   tie).  The stripped post-RHT symbols have lighter tails than a geometric
   source, which biases k* low by one step at some rates.  D4 ties its halved
   symbol to k_t = max(k_s - 1, 0) (Sec. 4.6), so its two classes move
   together; A2's two classes are chosen independently. */
static int choose_k(const hqo_params* P, const uint32_t* sym, int S, int k_out[2]) {
  int lat = P->lattice;
  if (P->rice_k >= 0) {
    k_out[0] = P->rice_k;
    if (lat == HQO_D4)
      k_out[1] = P->rice_k > 0 ? P->rice_k - 1 : 0;
    else
      k_out[1] = P->rice_k;
  } else if (lat == HQO_D4) {
    int k0 = class_kstar(lat, sym, S, 0);
    int k1 = k0 < HQO_KMAX ? k0 + 1 : k0;
    int64_t f0 = class_length(lat, sym, S, 0, k0) + class_length(lat, sym, S, 1, k0 > 0 ? k0 - 1 : 0);
    int64_t f1 = class_length(lat, sym, S, 0, k1) + class_length(lat, sym, S, 1, k1 > 0 ? k1 - 1 : 0);
    k_out[0] = f1 < f0 ? k1 : k0;
    k_out[1] = k_out[0] > 0 ? k_out[0] - 1 : 0;
  } else {
    int ncls = (lat == HQO_A2) ? 2 : 1;
    for (int cl = 0; cl < ncls; ++cl) {
      int k0 = class_kstar(lat, sym, S, cl);
      int k1 = k0 < HQO_KMAX ? k0 + 1 : k0;
      k_out[cl] = class_length(lat, sym, S, cl, k1) < class_length(lat, sym, S, cl, k0) ? k1 : k0;
    }
    if (ncls == 1) k_out[1] = k_out[0];
  }
  if (lat == HQO_A2) return k_out[0] | (k_out[1] << 4);
  return k_out[0];
}

static void decode_kparam(int lat, uint8_t kp, int k_out[2]) {
  if (lat == HQO_A2) {
    k_out[0] = kp & 15;
    k_out[1] = kp >> 4;
  } else if (lat == HQO_D4) {
    k_out[0] = kp;
    k_out[1] = kp > 0 ? kp - 1 : 0;
  } else {
    k_out[0] = kp;
    k_out[1] = kp;
  }
}

/* Bit i of the stream is bit (i mod 32) of word i / 32: LSB-first inside
   little-endian 32-bit words. */
static void put_bit(uint32_t* w, uint64_t pos) { w[pos >> 5] |= 1u << (pos & 31); }
static int get_bit(const uint32_t* w, uint64_t pos) { return (int)((w[pos >> 5] >> (pos & 31)) & 1u); }


/* One sub-stream, split layout: the S remainder fields (m mod 2^k, k bits,
   LSB first) in symbol order, then the S unary codes (q zeros and a
   terminating one) in symbol order, then zero padding to a 32-bit word.
   Writes into `w` (zeroed by the caller); returns the unpadded bit count. */
int64_t hqo_rice_put_substream(const hqo_params* P, const uint32_t* sym, int S, const int k[2],
                               uint32_t* w) {
  int m = hqo_lattice_dim(P->lattice);
  uint64_t pos = 0;
  for (int i = 0; i < S; ++i) {
    int kk = k[sym_class(P->lattice, i % m)];
    for (int b = 0; b < kk; ++b) {
      if ((sym[i] >> b) & 1u) put_bit(w, pos);
      ++pos;
    }
  }
  for (int i = 0; i < S; ++i) {
    int kk = k[sym_class(P->lattice, i % m)];
    pos += sym[i] >> kk;
    put_bit(w, pos);
    ++pos;
  }
  return (int64_t)pos;
}

/* Inverse of hqo_rice_put_substream; returns the bits consumed or -1 if
   the words run out (nwords bounds every read). */
int64_t hqo_rice_get_substream(const hqo_params* P, const uint32_t* w, int64_t nwords, int S,
                               const int k[2], uint32_t* sym) {
  int m = hqo_lattice_dim(P->lattice);
  uint64_t pos = 0, limit = (uint64_t)nwords * 32u;
  for (int i = 0; i < S; ++i) {
    int kk = k[sym_class(P->lattice, i % m)];
    uint32_t r = 0;
    for (int b = 0; b < kk; ++b) {
      if (pos >= limit) return -1;
      r |= (uint32_t)get_bit(w, pos) << b;
      ++pos;
    }
    sym[i] = r;
  }
  for (int i = 0; i < S; ++i) {
    int kk = k[sym_class(P->lattice, i % m)];
    uint32_t q = 0;
    for (;;) {
      if (pos >= limit) return -1;
      if (get_bit(w, pos)) break;
      ++q;
      ++pos;
    }
    ++pos;
    sym[i] |= q << kk;
  }
  return (int64_t)pos;
}

/* ------------------------------------------------------------------------ */
/* Dither sample (App. A "Practical sampler"): a uniform point of a box that */
/* is a fundamental domain of a sublattice, reduced mod the lattice.  For    */
/* 2E8, D4 and Z the cube [-2, 2)^m is such a box (4Z^m lies in each); for   */
/* A2 the box is [-sqrt3, sqrt3) x [-1, 1) ((2 sqrt3, 0) and (0, 2) lie in   */
/* it).  U = b - Q(b).                                                       */
/* ------------------------------------------------------------------------ */

void hqo_dither_block(int lat, uint64_t seed, int64_t row, int64_t col0, float* u) {
  int m = hqo_lattice_dim(lat);
  float b[8];
  for (int i = 0; i < m; ++i) {
    float centered = (float)((int32_t)dither_bits24(seed, row, col0 + i) - 8388608);
    if (lat == HQO_A2)
      b[i] = (i == 0) ? (centered * 0x1p-23f) * HQO_SQRT3F : centered * 0x1p-23f;
    else
      b[i] = centered * 0x1p-22f;
  }
  int32_t c[8];
  hqo_quantize_block(lat, b, c);
  for (int i = 0; i < m; ++i) {
    float p = (lat == HQO_A2 && i == 0) ? HQO_SQRT3F * (float)c[0] : (float)c[i];
    u[i] = b[i] - p;
  }
}

/* ------------------------------------------------------------------------ */
/* The codec.                                                                */
/* ------------------------------------------------------------------------ */

static int check_params(const hqo_params* P, int64_t cols) {
  int n = P->tile, m = hqo_lattice_dim(P->lattice);
  if (m == 0 || n < m || (n & (n - 1)) != 0) return HQO_ERR_ARG;
  if (P->rotation < 0 || P->rotation > 2 || (P->rotation == 2 && !P->qjl)) return HQO_ERR_ARG;
  if (cols % n != 0) return HQO_ERR_ARG;
  /* a sub-stream holds whole tiles, or a tile spans whole sub-streams */
  if (P->substream <= 0 || (P->substream % n != 0 && n % P->substream != 0) ||
      cols % P->substream != 0)
    return HQO_ERR_ARG;
  if (P->rice_k > HQO_KMAX) return HQO_ERR_ARG;
  return HQO_OK;
}

/* The qjl rotation (Sec. 4.2): y = S v (transpose 0, encode) or S^T v
   (transpose 1, decode) for the n x n row-major S; each output is the
   left-to-right fp32 sum of the rounded products, starting from the first. */
static void qjl_apply(const float* S, int transpose, const float* v, float* y, int n) {
  for (int i = 0; i < n; ++i) {
    float acc = (transpose ? S[i] : S[(int64_t)i * n]) * v[0];
    for (int k = 1; k < n; ++k) {
      const float sk = transpose ? S[(int64_t)k * n + i] : S[(int64_t)i * n + k];
      const float p = sk * v[k];
      acc = acc + p;
    }
    y[i] = acc;
  }
}

/* Front end, one tile at a time: norm, RHT, rotate, normalize, dither,
   quantize.  x is rows x cols (row stride ld, fp32), row0 the global index
   of its first row.  Outputs the lattice codes (rows x cols int32), the
   stored per-tile norm (fp32 or fp16 bits), and optionally the decoder input
   z (rows x cols fp32) for margin checks. */
int hqo_frontend(const hqo_params* P, const float* x, int64_t rows, int64_t cols, int64_t ld,
                 int64_t row0, int32_t* codes, void* norms, float* zin) {
  int rc = check_params(P, cols);
  if (rc) return rc;
  int n = P->tile, lat = P->lattice, m = hqo_lattice_dim(lat);
  int64_t tpr = cols / n;
  float* v = (float*)malloc(sizeof(float) * n);
  float* sq = (float*)malloc(sizeof(float) * n);
  int status = HQO_OK;
  for (int64_t r = 0; r < rows; ++r) {
    for (int64_t t = 0; t < tpr; ++t) {
      const float* xt = x + r * ld + t * n;
      /* Normalize (Sec. 4.3): r = ||x|| over the tile, the radius the
         unnormalized FWHT scales by sqrt(n). */
      for (int i = 0; i < n; ++i) sq[i] = xt[i] * xt[i];
      float nrm = sqrtf(tree_sum_f32(sq, n));
      /* A tile whose norm is not finite (an infinite or NaN input) has no
         scale: it is coded as if its transform were zero and reported, the
         way an fp16 norm overflow is (an error path the paper does not
         define). */
      const int nonfinite = !isfinite(nrm);
      if (nonfinite) status = HQO_ERR_OVERFLOW;
      float rs;
      if (P->norm_fp16) {
        uint16_t h = hqo_f32_to_f16(nrm);
        if ((h & 0x7C00) == 0x7C00) status = HQO_ERR_OVERFLOW;
        ((uint16_t*)norms)[r * tpr + t] = h;
        rs = hqo_f16_to_f32(h);
      } else {
        ((float*)norms)[r * tpr + t] = nrm;
        rs = nrm;
      }
      float scale = (rs == 0.0f || nonfinite) ? 0.0f : P->alpha / rs;
      /* RHT (eq. rht): v = H D x. */
      for (int i = 0; i < n; ++i) {
        int64_t col = t * n + i;
        v[i] = (hqo_sign(P->rht_seed, col) < 0) ? -xt[i] : xt[i];
      }
      hqo_fwht_f32(v, n);
      if (nonfinite)
        for (int i = 0; i < n; ++i) v[i] = 0.0f;
      /* z = alpha sqrt(n) S y / ||y|| = (alpha / r) S y. */
      for (int i = 0; i < n; ++i) {
        float zi = v[i] * scale;
        if (P->rotation == 1 && hqo_sign(P->rot_seed, i) < 0) zi = -zi;
        v[i] = zi;
      }
      if (P->rotation == 2) {
        qjl_apply(P->qjl, 0, v, sq, n);
        for (int i = 0; i < n; ++i) v[i] = sq[i];
      }
      /* Add dither (Sec. 4.4) then quantize (Sec. 4.5), block by block. */
      for (int b = 0; b < n / m; ++b) {
        float* zb = v + b * m;
        if (P->dither) {
          float u[8];
          hqo_dither_block(lat, P->dither_seed, row0 + r, t * n + b * m, u);
          for (int i = 0; i < m; ++i) zb[i] = zb[i] + u[i];
        }
        hqo_quantize_block(lat, zb, codes + r * cols + t * n + b * m);
        if (zin)
          for (int i = 0; i < m; ++i) zin[r * cols + t * n + b * m + i] = zb[i];
      }
    }
  }
  free(v);
  free(sq);
  return status;
}

/* Strip + Rice into offset-indexed sub-streams (Sec. 5.3).  Sub-stream s of
   the stream covers S consecutive symbols in row-major tile order; the rows
   given here are global rows row0 .. row0 + rows - 1 and the first one
   starts at payload word word0.  offsets[] is indexed by global sub-stream
   and holds absolute 32-bit word offsets; offsets[first + count] is written
   as the new end.  *payload_bits receives the unpadded Rice bits. */
int hqo_pack(const hqo_params* P, const int32_t* codes, int64_t rows, int64_t cols, int64_t row0,
             uint32_t* payload, int64_t cap_words, int64_t word0, uint32_t* offsets,
             uint8_t* kparam, int64_t* payload_bits) {
  int rc = check_params(P, cols);
  if (rc) return rc;
  int S = P->substream, lat = P->lattice, m = hqo_lattice_dim(lat);
  int64_t spr = cols / S, first = row0 * spr, nsub = rows * spr;
  uint32_t* sym = (uint32_t*)malloc(sizeof(uint32_t) * S);
  /* worst-case words of one sub-stream; grown on demand */
  int64_t wcap = 4096;
  uint32_t* w = (uint32_t*)malloc(sizeof(uint32_t) * wcap);
  int64_t pos_words = word0, bits = 0;
  offsets[first] = (uint32_t)word0;
  for (int64_t s = 0; s < nsub; ++s) {
    const int32_t* cs = codes + s * S; /* rows are contiguous, S divides cols */
    for (int b = 0; b < S / m; ++b) hqo_strip_block(lat, cs + b * m, sym + b * m);
    int k[2];
    kparam[first + s] = (uint8_t)choose_k(P, sym, S, k);
    int64_t need = 0;
    for (int i = 0; i < S; ++i) need += hqo_rice_length(sym[i], k[sym_class(lat, i % m)]);
    int64_t nw = (need + 31) / 32;
    if (nw > wcap) {
      wcap = nw;
      w = (uint32_t*)realloc(w, sizeof(uint32_t) * wcap);
    }
    memset(w, 0, sizeof(uint32_t) * nw);
    int64_t got = hqo_rice_put_substream(P, sym, S, k, w);
    if (got != need) {
      free(sym);
      free(w);
      return HQO_ERR_ARG;
    }
    if (pos_words + nw > cap_words || pos_words + nw > 0xFFFFFFFFLL) {
      free(sym);
      free(w);
      return HQO_ERR_CAPACITY;
    }
    memcpy(payload + pos_words, w, sizeof(uint32_t) * nw);
    pos_words += nw;
    bits += need;
    offsets[first + s + 1] = (uint32_t)pos_words;
  }
  free(sym);
  free(w);
  if (payload_bits) *payload_bits = bits;
  return HQO_OK;
}

/* Inverse of hqo_pack for global rows row0 .. row0 + rows - 1. */
int hqo_unpack(const hqo_params* P, const uint32_t* payload, const uint32_t* offsets,
               const uint8_t* kparam, int64_t rows, int64_t cols, int64_t row0, int32_t* codes) {
  int rc = check_params(P, cols);
  if (rc) return rc;
  int S = P->substream, lat = P->lattice, m = hqo_lattice_dim(lat);
  int64_t spr = cols / S, first = row0 * spr, nsub = rows * spr;
  uint32_t* sym = (uint32_t*)malloc(sizeof(uint32_t) * S);
  int status = HQO_OK;
  for (int64_t s = 0; s < nsub; ++s) {
    int k[2];
    decode_kparam(lat, kparam[first + s], k);
    int64_t a = offsets[first + s], e = offsets[first + s + 1];
    if (e < a || hqo_rice_get_substream(P, payload + a, e - a, S, k, sym) < 0) {
      status = HQO_ERR_CORRUPT;
      memset(sym, 0, sizeof(uint32_t) * S);
    }
    int32_t* cs = codes + s * S;
    for (int b = 0; b < S / m; ++b) hqo_unstrip_block(lat, sym + b * m, cs + b * m);
  }
  free(sym);
  return status;
}

/* Back end, one tile at a time: dequantize, undither, derotate, inverse RHT,
   denormalize.  x_hat = D H c_hat * r / (alpha n), since H^-1 = H / n and
   y = H D x carries the factor sqrt(n) ||x|| that the scale alpha / r
   normalized away.  Without dither the codes of E8/D4/Z are integers and
   H c is evaluated exactly in integer arithmetic. */
int hqo_backend(const hqo_params* P, const int32_t* codes, const void* norms, int64_t rows,
                int64_t cols, int64_t row0, float* y) {
  int rc = check_params(P, cols);
  if (rc) return rc;
  int n = P->tile, lat = P->lattice, m = hqo_lattice_dim(lat);
  int64_t tpr = cols / n;
  float* v = (float*)malloc(sizeof(float) * n);
  float* vq = (float*)malloc(sizeof(float) * n);
  int64_t* vi = (int64_t*)malloc(sizeof(int64_t) * n);
  int exact = !P->dither && lat != HQO_A2 && P->rotation != 2;
  float an = P->alpha * (float)n; /* exact: n is a power of two */
  for (int64_t r = 0; r < rows; ++r) {
    for (int64_t t = 0; t < tpr; ++t) {
      const int32_t* ct = codes + r * cols + t * n;
      float rs = P->norm_fp16 ? hqo_f16_to_f32(((const uint16_t*)norms)[r * tpr + t])
                              : ((const float*)norms)[r * tpr + t];
      float g = rs / an;
      if (exact) {
        /* the rotation signs commute with nothing else here, apply first */
        for (int i = 0; i < n; ++i)
          vi[i] = (P->rotation == 1 && hqo_sign(P->rot_seed, i) < 0) ? -(int64_t)ct[i] : ct[i];
        hqo_fwht_i64(vi, n);
        for (int i = 0; i < n; ++i) {
          int64_t w = (hqo_sign(P->rht_seed, t * n + i) < 0) ? -vi[i] : vi[i];
          y[r * cols + t * n + i] = (float)w * g;
        }
      } else {
        for (int b = 0; b < n / m; ++b) {
          for (int i = 0; i < m; ++i) {
            int32_t ci = ct[b * m + i];
            v[b * m + i] = (lat == HQO_A2 && i == 0) ? HQO_SQRT3F * (float)ci : (float)ci;
          }
          if (P->dither) {
            float u[8];
            hqo_dither_block(lat, P->dither_seed, row0 + r, t * n + b * m, u);
            for (int i = 0; i < m; ++i) v[b * m + i] = v[b * m + i] - u[i];
          }
        }
        if (P->rotation == 1)
          for (int i = 0; i < n; ++i)
            if (hqo_sign(P->rot_seed, i) < 0) v[i] = -v[i];
        if (P->rotation == 2) {
          qjl_apply(P->qjl, 1, v, vq, n);
          for (int i = 0; i < n; ++i) v[i] = vq[i];
        }
        hqo_fwht_f32(v, n);
        for (int i = 0; i < n; ++i) {
          float w = (hqo_sign(P->rht_seed, t * n + i) < 0) ? -v[i] : v[i];
          y[r * cols + t * n + i] = w * g;
        }
      }
    }
  }
  free(v);
  free(vq);
  free(vi);
  return HQO_OK;
}

/* ------------------------------------------------------------------------ */
/* Whole-stream encode and decode (front end + pack, unpack + back end).     */
/* ------------------------------------------------------------------------ */

int hqo_encode(const hqo_params* P, const float* x, int64_t rows, int64_t cols, int64_t ld,
               int64_t row0, uint32_t* payload, int64_t cap_words, int64_t word0,
               uint32_t* offsets, uint8_t* kparam, void* norms, int64_t* payload_bits) {
  int32_t* codes = (int32_t*)malloc(sizeof(int32_t) * (size_t)(rows * cols + 1));
  int64_t tpr = cols / P->tile;
  void* nb = P->norm_fp16 ? (void*)((uint16_t*)norms + row0 * tpr) : (void*)((float*)norms + row0 * tpr);
  int rc = hqo_frontend(P, x, rows, cols, ld, row0, codes, nb, NULL);
  int rc2 = (rc == HQO_OK || rc == HQO_ERR_OVERFLOW)
                ? hqo_pack(P, codes, rows, cols, row0, payload, cap_words, word0, offsets, kparam,
                           payload_bits)
                : rc;
  free(codes);
  return rc2 != HQO_OK ? rc2 : rc;
}

int hqo_decode(const hqo_params* P, const uint32_t* payload, const uint32_t* offsets,
               const uint8_t* kparam, const void* norms, int64_t rows, int64_t cols, int64_t row0,
               float* y) {
  int32_t* codes = (int32_t*)malloc(sizeof(int32_t) * (size_t)(rows * cols + 1));
  int rc = hqo_unpack(P, payload, offsets, kparam, rows, cols, row0, codes);
  int64_t tpr = cols / P->tile;
  const void* nb = P->norm_fp16 ? (const void*)((const uint16_t*)norms + row0 * tpr)
                                : (const void*)((const float*)norms + row0 * tpr);
  int rc2 = hqo_backend(P, codes, nb, rows, cols, row0, y);
  free(codes);
  return rc != HQO_OK ? rc : rc2;
}

/* ------------------------------------------------------------------------ */
/* int8 GEMM on post-RHT lattice codes (Sec. 4.8 Cast, Sec. 6.3).           */
/* ------------------------------------------------------------------------ */

/* Per-tile weight factor g[r, t] = r_s / (alpha n) that multiplies the
   integer code tile (the same division as the back end). */
void hqo_weight_factors(const hqo_params* P, const void* norms, int64_t rows, int64_t cols,
                        float* g) {
  int n = P->tile;
  int64_t tpr = cols / n;
  float an = P->alpha * (float)n;
  for (int64_t i = 0; i < rows * tpr; ++i) {
    float rs = P->norm_fp16 ? hqo_f16_to_f32(((const uint16_t*)norms)[i]) : ((const float*)norms)[i];
    g[i] = rs / an;
  }
}

/* Activation preparation: per K-tile y = H D a (the weights' signs, indexed
   by global K column, so that the two rotations cancel: w.a = sum_t g c.(H D a)),
   then per-token symmetric int8: amax over the whole rotated row,
   x_q = clamp(rint(y * (127 / amax)), -127, 127), s_x = amax / 127. */
void hqo_act_prep(const float* a, int64_t M, int64_t K, int tile, uint64_t rht_seed, int8_t* xq,
                  float* sx) {
  float* y = (float*)malloc(sizeof(float) * K);
  for (int64_t i = 0; i < M; ++i) {
    for (int64_t j = 0; j < K; ++j) y[j] = (hqo_sign(rht_seed, j) < 0) ? -a[i * K + j] : a[i * K + j];
    for (int64_t t = 0; t < K / tile; ++t) hqo_fwht_f32(y + t * tile, tile);
    float amax = 0.0f;
    for (int64_t j = 0; j < K; ++j)
      if (fabsf(y[j]) > amax) amax = fabsf(y[j]);
    float inv = (amax == 0.0f) ? 0.0f : 127.0f / amax;
    for (int64_t j = 0; j < K; ++j) {
      float q = rintf(y[j] * inv);
      if (q > 127.0f) q = 127.0f;
      if (q < -127.0f) q = -127.0f;
      xq[i * K + j] = (int8_t)q;
    }
    sx[i] = amax / 127.0f;
  }
  free(y);
}

/* Y[i, r] = s_x[i] * sum_t g[r, t] * sum_{j in t} c[r, j] * x_q[i, j]:
   exact int64 tile sums, fp64 scaling.  Y is M x N. */
void hqo_gemm_blockscaled(const int32_t* codes, const float* g, const int8_t* xq, const float* sx,
                          int64_t M, int64_t N, int64_t K, int tile, double* out) {
  int64_t T = K / tile;
  for (int64_t i = 0; i < M; ++i)
    for (int64_t r = 0; r < N; ++r) {
      double acc = 0.0;
      for (int64_t t = 0; t < T; ++t) {
        int64_t s = 0;
        for (int64_t j = t * tile; j < (t + 1) * tile; ++j) s += (int64_t)codes[r * K + j] * xq[i * K + j];
        acc += (double)g[r * T + t] * (double)s;
      }
      out[i * N + r] = (double)sx[i] * acc;
    }
}
