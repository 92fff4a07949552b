// Host side of libhq.so: plan construction, argument validation and the
// C ABI declared in include/hq.h.  All codec arithmetic runs in the gfx950
// kernels of hq_kernels.hip; this file derives constants and launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

#include "hq_internal.h"

namespace {

#include "calib_table.inc"

// Lattice dimension, normalized second moment G (the closed forms behind the
// four-digit values of the paper's lattice-constant table) and covolume of
// the integer realization (Sec. 4.5).
int lattice_dim(int lat) { return lat == HQ_E8 ? 8 : lat == HQ_D4 ? 4 : lat == HQ_A2 ? 2 : 1; }

double lattice_nsm(int lat) {
  switch (lat) {
    case HQ_E8: return 929.0 / 12960.0;
    case HQ_D4: return 13.0 / (120.0 * std::sqrt(2.0));
    case HQ_A2: return 5.0 / (36.0 * std::sqrt(3.0));
    default: return 1.0 / 12.0;
  }
}

double lattice_covolume(int lat) {
  switch (lat) {
    case HQ_E8: return 256.0;
    case HQ_D4: return 2.0;
    case HQ_A2: return 2.0 * std::sqrt(3.0);
    default: return 1.0;
  }
}

// Covering radius of the integer realization: how far the nearest point can
// be from any input.
double lattice_rho(int lat) {
  switch (lat) {
    case HQ_E8: return 2.0;
    case HQ_D4: return 1.0;
    case HQ_A2: return 2.0 / std::sqrt(3.0);
    default: return 0.5;
  }
}

// App. B, eq. alpha-calib: alpha = sqrt(SNR_lin G V^(2/N)).
double alpha_for_snr(int lat, double snr_db) {
  const double snr_lin = std::pow(10.0, snr_db / 10.0);
  return std::sqrt(snr_lin * lattice_nsm(lat) *
                   std::pow(lattice_covolume(lat), 2.0 / (double)lattice_dim(lat)));
}

// The sign of column j: -1 iff the top bit of SplitMix64's j-th output is set
// (SplitMix64: Steele, Lea and Flood, 2014).
bool splitmix_negative(uint64_t seed, uint64_t j) {
  uint64_t z = seed + (j + 1) * 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  z ^= z >> 31;
  return (z >> 63) != 0;
}

// Sec. 3.3: optimal Rice parameter of a geometric source, with the
// parameter estimated from `count` symbols summing to `sum`.
int kstar_formula(int64_t count, int64_t sum) {
  if (count <= 0) return 0;
  const double p = (double)count / ((double)count + (double)sum);
  if (p >= 1.0) return 0;
  const double ratio = -std::log(2.0 - p) / std::log(1.0 - p);
  const double c = std::ceil(ratio);
  if (!(c >= 1.0)) return 0;
  if (c > 9.0e15) return HQ_KMAX;
  const int k = 63 - __builtin_clzll((unsigned long long)(int64_t)c);
  return std::min(k, HQ_KMAX);
}

// thr[t] = smallest sum with kstar_formula(count, sum) >= t (k* is
// non-decreasing in the sum); 0xFFFFFFFF when no 32-bit sum reaches t.
void kstar_thresholds(int64_t count, uint32_t* thr) {
  thr[0] = 0;
  for (int t = 1; t <= HQ_KMAX; ++t) {
    int64_t lo = 0, hi = 0xFFFFFFFFLL;
    if (kstar_formula(count, hi) < t) {
      thr[t] = 0xFFFFFFFFu;
      continue;
    }
    while (lo < hi) {
      const int64_t mid = lo + (hi - lo) / 2;
      if (kstar_formula(count, mid) >= t) hi = mid; else lo = mid + 1;
    }
    thr[t] = (uint32_t)lo;
  }
}

int kstar_from_thresholds(const uint32_t* thr, int64_t sum) {
  int k = 0;
  for (int t = 1; t <= HQ_KMAX; ++t) k += (sum >= (int64_t)thr[t]) ? 1 : 0;
  return k;
}

// Class sizes of one sub-stream (Rice class 0 and 1).
void class_counts(int lat, int S, int64_t* n0, int64_t* n1) {
  if (lat == HQ_D4) {
    *n0 = 3 * S / 4;
    *n1 = S / 4;
  } else if (lat == HQ_A2) {
    *n0 = S / 2;
    *n1 = S / 2;
  } else {
    *n0 = S;
    *n1 = 0;
  }
}

// Deterministic bound on the words of one sub-stream.  Per tile the lattice
// code satisfies |c| <= |z| + rho sqrt(n/m) (plus rho sqrt(n/m) again with
// dither), |z| = alpha sqrt(n) r / r_s (r_s the stored norm; fp16 can round a
// tiny norm down by up to a third); each stripped symbol is at most
// 2 |coordinate| + 2, so a class sums to M <= T (2 sqrt(n) |c| + 2 n).  A
// class with parameter k costs count (1 + k) + sum / 2^k bits, and the
// encoder's k never costs more than the geometric k* of that sum.
// Bound on the norm of one tile's lattice code (hence on every |c_i|).
double code_norm_bound(const hq_plan_s& p) {
  const int n = p.tile, m = p.dim;
  const double fac = p.norm_fp16 ? 1.5 : 1.0;
  return fac * (double)p.alpha * std::sqrt((double)n) * 1.001 +
         lattice_rho(p.lattice) * std::sqrt((double)n / m) * (p.dither ? 2.0 : 1.0);
}

int64_t substream_word_bound(const hq_plan_s& p) {
  const int n = p.tile, S = p.substream;
  const double T = (double)S / n;
  const double cn = code_norm_bound(p);
  // a sub-stream of whole tiles sums T tiles' bounds; a sub-stream inside a
  // longer tile may hold all of that tile's code norm on its S coordinates
  const double M = S >= n ? T * (2.0 * std::sqrt((double)n) * cn + 2.0 * n)
                          : 2.0 * std::sqrt((double)S) * cn + 2.0 * S;
  const int64_t Mi = (int64_t)std::ceil(M) + 1;
  int64_t n0, n1;
  class_counts(p.lattice, S, &n0, &n1);
  auto cost = [&](int64_t count, int k, int64_t sum) -> double {
    return (double)count * (1 + k) + std::ldexp((double)sum, -k);
  };
  double worst = 0.0;
  if (p.rice_k >= 0) {
    const int k0 = p.rice_k;
    const int k1 = (p.lattice == HQ_D4) ? std::max(k0 - 1, 0) : k0;
    worst = cost(n0, k0, Mi) + (n1 ? cost(n1, k1, Mi) : 0.0);
  } else {
    // worst case over every class sum up to M, at the k the sum selects
    double w0 = 0.0, w1 = 0.0;
    const int64_t step = std::max<int64_t>(1, Mi / 200000);
    for (int64_t s = 0; s <= Mi; s += step) {
      const int64_t ss = std::min(Mi, s + step - 1);  // the sum is at most this in the bin
      const int k0 = kstar_from_thresholds(p.thr[0], s);
      w0 = std::max(w0, cost(n0, k0, ss));
      if (p.lattice == HQ_D4) {
        w1 = std::max(w1, cost(n1, std::max(k0 - 1, 0), ss));
      } else if (p.lattice == HQ_A2) {
        const int k1 = kstar_from_thresholds(p.thr[1], s);
        w1 = std::max(w1, cost(n1, k1, ss));
      }
    }
    if (p.lattice == HQ_D4) {
      // the class-1 sum can be large while class 0 selects k = 0
      w1 = std::max(w1, cost(n1, 0, Mi));
    }
    worst = w0 + w1;
  }
  return (int64_t)std::ceil(worst * 1.02 / 32.0) + 2;
}

bool lookup_calibration(int lat, int rice_k, double bps, double* snr) {
  for (const hq_calib_curve& c : kCalib) {
    if (c.lattice != lat || c.rice_k != rice_k || c.n < 2) continue;
    for (int i = 0; i + 1 < c.n; ++i) {
      const double b0 = c.bps[i], b1 = c.bps[i + 1];
      if (b0 <= bps && bps <= b1 && b1 > b0) {
        const double f = (bps - b0) / (b1 - b0);
        *snr = c.snr0 + c.step * (i + f);
        return true;
      }
    }
    return false;
  }
  return false;
}

bool has_calibration(int lat, int rice_k) {
  for (const hq_calib_curve& c : kCalib)
    if (c.lattice == lat && c.rice_k == rice_k && c.n >= 2) return true;
  return false;
}

hq_status hip_status(int e) { return e == 0 ? HQ_OK : HQ_ERR_HIP; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

extern "C" {

const char* hq_status_string(int32_t status) {
  switch (status) {
    case HQ_OK: return "ok";
    case HQ_ERR_INVALID_ARG: return "invalid argument";
    case HQ_ERR_UNSUPPORTED: return "unsupported configuration";
    case HQ_ERR_CAPACITY: return "buffer capacity exceeded";
    case HQ_ERR_OVERFLOW: return "norm overflow or non-finite input";
    case HQ_ERR_HIP: return "HIP runtime error";
    case HQ_ERR_CORRUPT: return "corrupt sub-stream";
    case HQ_ERR_NO_CALIBRATION: return "no calibration table for this lattice / Rice setting";
  }
  return "unknown status";
}

int32_t hq_rice_kstar(int64_t count, int64_t sum) {
  uint32_t thr[HQ_KMAX + 1];
  kstar_thresholds(count, thr);
  return kstar_from_thresholds(thr, sum);
}

hq_status hq_calibrated_snr(int32_t lattice, int32_t rice_k, float bps, double* snr_db) {
  if (!snr_db || lattice < HQ_E8 || lattice > HQ_Z) return HQ_ERR_INVALID_ARG;
  if (!has_calibration(lattice, rice_k)) return HQ_ERR_NO_CALIBRATION;
  if (!lookup_calibration(lattice, rice_k, (double)bps, snr_db)) return HQ_ERR_INVALID_ARG;
  return HQ_OK;
}

hq_status hq_plan(int32_t tile, int32_t lattice, float bps, uint64_t rht_seed, int32_t rice_k,
                  int64_t cols, const hq_options* opt, hq_plan_t* out, hq_plan_info* info) {
  if (!out) return HQ_ERR_INVALID_ARG;
  *out = nullptr;
  hq_options o;
  std::memset(&o, 0, sizeof(o));
  if (opt) o = *opt;
  if (lattice < HQ_E8 || lattice > HQ_Z) return HQ_ERR_INVALID_ARG;
  const int m = lattice_dim(lattice);
  if (tile < m || tile <= 0 || (tile & (tile - 1)) != 0) return HQ_ERR_INVALID_ARG;
  const int S = o.substream ? o.substream : HQ_SUB;
  // a sub-stream holds whole tiles, or a tile spans whole sub-streams
  if (S <= 0 || (S % tile != 0 && tile % S != 0) || cols <= 0 || cols % tile != 0 || cols % S != 0)
    return HQ_ERR_INVALID_ARG;
  if (rice_k < -1 || rice_k > HQ_KMAX) return HQ_ERR_INVALID_ARG;
  if (o.rotation != HQ_ROT_NONE && o.rotation != HQ_ROT_SIGNS && o.rotation != HQ_ROT_QJL)
    return HQ_ERR_INVALID_ARG;
  if (o.rotation == HQ_ROT_QJL && !o.qjl) return HQ_ERR_INVALID_ARG;
  if (o.norm_dtype != 0 && o.norm_dtype != HQ_FP32 && o.norm_dtype != HQ_FP16)
    return HQ_ERR_INVALID_ARG;
  // sub-streams of 1024 or 2048 symbols (two or four 512-symbol blocks) are
  // built for weight plans: no rotation, no dither, fp32 norms
  if (S != HQ_SUB && ((S != 2 * HQ_SUB && S != 4 * HQ_SUB) || o.rotation != HQ_ROT_NONE ||
                      o.dither || o.norm_dtype == HQ_FP16))
    return HQ_ERR_UNSUPPORTED;
  // tiles of 256 .. 2048 (the sweep of Sec. 7.2) are built for weight plans:
  // no rotation, no dither, fp32 norms
  if (tile != HQ_TILE &&
      (tile < 256 || tile > HQ_TILE_MAX || o.rotation != HQ_ROT_NONE || o.dither ||
       o.norm_dtype == HQ_FP16))
    return HQ_ERR_UNSUPPORTED;
  if (cols > (int64_t)1 << 28) return HQ_ERR_UNSUPPORTED;  // per-lane byte offsets stay 32-bit

  double snr;
  if (o.use_snr) {
    snr = o.snr_db;
    if (!std::isfinite(snr) || snr < -30.0 || snr > 80.0) return HQ_ERR_INVALID_ARG;
  } else {
    if (!(bps > 0.0f) || !std::isfinite(bps)) return HQ_ERR_INVALID_ARG;
    if (!has_calibration(lattice, rice_k)) return HQ_ERR_NO_CALIBRATION;
    if (!lookup_calibration(lattice, rice_k, (double)bps, &snr)) return HQ_ERR_INVALID_ARG;
  }

  hq_plan_s* p = new (std::nothrow) hq_plan_s();
  if (!p) return HQ_ERR_INVALID_ARG;
  p->tile = tile;
  p->lattice = lattice;
  p->dim = m;
  p->substream = S;
  p->rice_k = rice_k;
  p->cols = cols;
  p->tpr = cols / tile;
  p->spr = cols / S;
  p->snr_db = snr;
  p->alpha = (float)alpha_for_snr(lattice, snr);
  p->rotation = o.rotation;
  p->dither = o.dither ? 1 : 0;
  p->norm_fp16 = (o.norm_dtype == HQ_FP16) ? 1 : 0;
  p->rht_seed = rht_seed;
  p->rot_seed = o.rot_seed;
  p->dither_seed = o.dither_seed;
  int64_t n0, n1;
  class_counts(lattice, S, &n0, &n1);
  kstar_thresholds(n0, p->thr[0]);
  if (n1) kstar_thresholds(n1, p->thr[1]); else kstar_thresholds(1, p->thr[1]);
  p->max_words_sub = substream_word_bound(*p);
  // qjl decodes also hold S (64 KB) and 2 KB of stage per wave in LDS, next to
  // the four sub-stream buffers; keep the workgroup within 160 KB
  if (p->max_words_sub > 8192 || (o.rotation == HQ_ROT_QJL && p->max_words_sub > 4096)) {
    delete p;
    return HQ_ERR_UNSUPPORTED;
  }
  if (hipGetDevice(&p->device) != hipSuccess) {
    delete p;
    return HQ_ERR_HIP;
  }

  // sign bitmasks: bit j set means the sign is -1
  const int64_t nw = (cols + 31) / 32;
  const int64_t snw = ((int64_t)tile + 31) / 32;  // words of the rotation mask (one bit per coordinate)
  std::vector<uint32_t> dm((size_t)nw, 0u), sm((size_t)snw, 0u);
  for (int64_t j = 0; j < cols; ++j)
    if (splitmix_negative(rht_seed, (uint64_t)j)) dm[(size_t)(j >> 5)] |= 1u << (j & 31);
  for (int j = 0; j < tile; ++j)
    if (splitmix_negative(o.rot_seed, (uint64_t)j)) sm[(size_t)(j >> 5)] |= 1u << (j & 31);
  const int64_t npairs = (cols + 1) / 2;
  std::vector<uint32_t> ds((size_t)npairs, 0u);
  for (int64_t j = 0; j < cols; ++j)
    if ((dm[(size_t)(j >> 5)] >> (j & 31)) & 1u) ds[(size_t)(j >> 1)] |= (j & 1) ? 0x80000000u : 0x8000u;
  p->d_dmask = nullptr;
  p->d_smask = nullptr;
  p->d_dsign16 = nullptr;
  p->d_qjl = nullptr;
  p->d_qjlt = nullptr;
  bool ok = hipMalloc((void**)&p->d_dmask, sizeof(uint32_t) * (size_t)nw) == hipSuccess &&
            hipMalloc((void**)&p->d_smask, sizeof(uint32_t) * (size_t)snw) == hipSuccess &&
            hipMalloc((void**)&p->d_dsign16, sizeof(uint32_t) * (size_t)npairs) == hipSuccess;
  if (ok && o.rotation == HQ_ROT_QJL) {
    const size_t nn = (size_t)tile * tile;
    std::vector<float> st(nn);
    for (int i = 0; i < tile; ++i)
      for (int k = 0; k < tile; ++k) st[(size_t)k * tile + i] = o.qjl[(size_t)i * tile + k];
    ok = hipMalloc((void**)&p->d_qjl, sizeof(float) * nn) == hipSuccess &&
         hipMalloc((void**)&p->d_qjlt, sizeof(float) * nn) == hipSuccess &&
         hipMemcpy(p->d_qjl, o.qjl, sizeof(float) * nn, hipMemcpyHostToDevice) == hipSuccess &&
         hipMemcpy(p->d_qjlt, st.data(), sizeof(float) * nn, hipMemcpyHostToDevice) == hipSuccess;
  }
  ok = ok &&
       hipMemcpy(p->d_dmask, dm.data(), sizeof(uint32_t) * (size_t)nw, hipMemcpyHostToDevice) ==
           hipSuccess &&
       hipMemcpy(p->d_smask, sm.data(), sizeof(uint32_t) * (size_t)snw, hipMemcpyHostToDevice) ==
           hipSuccess &&
       hipMemcpy(p->d_dsign16, ds.data(), sizeof(uint32_t) * (size_t)npairs,
                 hipMemcpyHostToDevice) == hipSuccess;
  if (!ok) {
    // the error reported is the failed allocation or copy; the frees are
    // best effort
    for (void* d : {(void*)p->d_dmask, (void*)p->d_smask, (void*)p->d_dsign16, (void*)p->d_qjl,
                    (void*)p->d_qjlt})
      if (d) (void)hipFree(d);
    delete p;
    return HQ_ERR_HIP;
  }
  *out = p;
  if (info) hq_plan_get_info(p, info);
  return HQ_OK;
}

hq_status hq_plan_get_info(hq_plan_t p, hq_plan_info* info) {
  if (!p || !info) return HQ_ERR_INVALID_ARG;
  std::memset(info, 0, sizeof(*info));
  info->alpha = p->alpha;
  info->snr_db = (float)p->snr_db;
  info->tile = p->tile;
  info->lattice = p->lattice;
  info->substream = p->substream;
  info->rice_k = p->rice_k;
  info->cols = p->cols;
  info->tiles_per_row = p->tpr;
  info->subs_per_row = p->spr;
  info->max_words_per_substream = p->max_words_sub;
  info->max_words_per_row = p->max_words_sub * p->spr;
  return HQ_OK;
}

hq_status hq_plan_destroy(hq_plan_t p) {
  if (!p) return HQ_ERR_INVALID_ARG;
  bool ok = true;
  for (void* d : {(void*)p->d_dmask, (void*)p->d_smask, (void*)p->d_dsign16, (void*)p->d_qjl,
                  (void*)p->d_qjlt})
    if (d) ok = hipFree(d) == hipSuccess && ok;
  delete p;
  return ok ? HQ_OK : HQ_ERR_HIP;
}

// Sub-streams per wave of an encode of nsub sub-streams: one for small
// launches (unless the caller needs the four of a group launch).
static int32_t encode_spw(int64_t nsub, bool allow_small) {
  return (allow_small && nsub <= HQ_ENC_SMALL_SUBS) ? 1 : HQ_ENC_SUBS_PER_WAVE;
}

size_t hq_scan_bytes(hq_plan_t p, int64_t rows) {
  if (!p || rows < 0) return 0;
  // one workgroup per 16 blocks of 512 symbols
  const int64_t nwg = (rows * p->spr * (p->substream / HQ_SUB) + HQ_ENC_SUBS_PER_WG - 1) / HQ_ENC_SUBS_PER_WG;
  // the epoch word, then a look-back status word and a stats word per workgroup
  return (size_t)HQ_SCAN_STATUS_OFFSET +
         2 * sizeof(unsigned long long) * (size_t)std::max<int64_t>(nwg, 1);
}

// Validates one encode and fills its kernel arguments.  Returns HQ_OK with
// *nwg = 0 when there is nothing to launch (rows == 0; the stream is then
// already up to date).
static hq_status encode_prepare(hq_plan_t p, const void* x, int32_t xt, int64_t rows, int64_t ld,
                                hq_stream* s, int32_t append, bool allow_small, hq_encode_args* out,
                                int64_t* nwg_out, void* stream) {
  *nwg_out = 0;
  if (!p || !s || rows < 0) return HQ_ERR_INVALID_ARG;
  if (xt != HQ_BF16 && xt != HQ_FP32) return HQ_ERR_INVALID_ARG;
  if (!s->payload || !s->offsets || !s->kparam || !s->norms || !s->scan) return HQ_ERR_INVALID_ARG;
  if (((uintptr_t)s->scan & 7u) != 0) return HQ_ERR_INVALID_ARG;
  const int64_t row0 = append ? s->rows : 0;
  if (row0 < 0 || row0 + rows > s->rows_capacity) return HQ_ERR_CAPACITY;
  if (rows > 0) {
    if (!x || ld < p->cols) return HQ_ERR_INVALID_ARG;
    const int64_t esz = (xt == HQ_BF16) ? 2 : 4;
    if (!aligned16(x) || (ld * esz) % 16 != 0) return HQ_ERR_INVALID_ARG;
  }
  const int64_t nsub = rows * p->spr;
  const int64_t first_sub = row0 * p->spr;
  if (first_sub + nsub > (int64_t)0xFFFFFFFF) return HQ_ERR_UNSUPPORTED;
  if (rows == 0) {
    if (!append) {
      s->rows = 0;
      return hip_status(hq_launch_zero(s->offsets, sizeof(uint32_t), stream));
    }
    return HQ_OK;
  }
  const int32_t mb = p->substream / HQ_SUB;  // 512-symbol blocks per sub-stream
  const int32_t spw = (p->tile != HQ_TILE || mb > 1) ? HQ_ENC_SUBS_PER_WAVE : encode_spw(nsub, allow_small);
  const int64_t nwg = (nsub * mb + HQ_ENC_SUBS_PER_WG - 1) / HQ_ENC_SUBS_PER_WG;
  if (nwg > 0x7FFFFFFF) return HQ_ERR_UNSUPPORTED;
  if ((size_t)s->scan_bytes < hq_scan_bytes(p, rows)) return HQ_ERR_CAPACITY;

  hq_encode_args& a = *out;
  std::memset(&a, 0, sizeof(a));
  a.x = x;
  a.ld = ld;
  a.first_row = row0;
  a.first_sub = first_sub;
  a.nsub = nsub;
  a.spr = p->spr;
  a.tpr = p->tpr;
  a.payload = s->payload;
  a.cap_words = s->capacity_words;
  a.offsets = s->offsets;
  a.kparam = s->kparam;
  a.norms = s->norms;
  a.dmask = p->d_dmask;
  a.dsign16 = p->d_dsign16;
  a.smask = p->d_smask;
  a.qjlt = p->d_qjlt;
  a.stats = s->stats;
  a.epoch = (unsigned long long*)s->scan;
  a.status = (unsigned long long*)((char*)s->scan + HQ_SCAN_STATUS_OFFSET);
  a.wgstat = a.status + nwg;
  a.nwg = (uint32_t)nwg;
  a.spw = (uint32_t)spw;
  a.append = append ? 1 : 0;
  a.rice_k = p->rice_k;
  a.rotation = p->rotation;
  a.dither = p->dither;
  a.norm_fp16 = p->norm_fp16;
  a.lds_words = (uint32_t)p->max_words_sub;
  a.dither_seed = p->dither_seed;
  a.alpha = p->alpha;
  a.alpha_half = 0.5f * p->alpha;
  a.tile = p->tile;
  a.mb = mb;
  *nwg_out = nwg;
  return HQ_OK;
}

// The plan's Rice-k thresholds as the kernel compares them.  Class sums stay
// below 2^26 (512 symbols of at most 2^17), so thresholds past 2^30 are
// unreachable; the kernel compares in signed 32-bit.
static hq_rice_thr rice_thresholds(const hq_plan_s* p) {
  hq_rice_thr t;
  for (int k = 0; k <= HQ_KMAX; ++k) {
    t.thr0[k] = std::min<uint32_t>(p->thr[0][k], 1u << 30);
    t.thr1[k] = std::min<uint32_t>(p->thr[1][k], 1u << 30);
  }
  return t;
}

hq_status hq_encode(hq_plan_t p, const void* x, int32_t xt, int64_t rows, int64_t ld,
                    hq_stream* s, int32_t append, void* stream) {
  hq_encode_args a;
  int64_t nwg;
  const hq_status st = encode_prepare(p, x, xt, rows, ld, s, append, true, &a, &nwg, stream);
  if (st != HQ_OK || nwg == 0) return st;
  if (hq_launch_encode(p, a, rice_thresholds(p), xt, stream)) return HQ_ERR_HIP;
  s->rows = a.first_row + rows;
  return HQ_OK;
}

hq_status hq_encode_noalloc(hq_plan_t p, const void* x, int32_t xt, int64_t rows, int64_t ld,
                            hq_stream* s, int32_t append, void* stream) {
  if (!p || !s || rows < 0) return HQ_ERR_INVALID_ARG;
  if (hq_scan_bytes(p, rows) > (size_t)HQ_NOALLOC_SCAN_BYTES) return HQ_ERR_CAPACITY;
  void* scan = nullptr;
  if (hq_noalloc_scan(&scan, stream) != 0) return HQ_ERR_HIP;
  hq_stream t = *s;  // the caller's stream with the fixed scratch in place of s->scan
  t.scan = scan;
  t.scan_bytes = (int64_t)HQ_NOALLOC_SCAN_BYTES;
  const hq_status st = hq_encode(p, x, xt, rows, ld, &t, append, stream);
  s->rows = t.rows;
  return st;
}

static bool same_kernel_family(const hq_plan_s* a, const hq_plan_s* b) {
  const bool kva = a->rotation || a->dither || a->norm_fp16;
  const bool kvb = b->rotation || b->dither || b->norm_fp16;
  return a->lattice == b->lattice && kva == kvb && a->tile == b->tile && a->substream == b->substream;
}

hq_status hq_encode_group(const hq_plan_t* plans, const void* const* x, int32_t xt,
                          const int64_t* rows, const int64_t* ld, hq_stream* const* s,
                          int32_t count, void* stream) {
  if (count < 0 || (count > 0 && (!plans || !x || !rows || !ld || !s))) return HQ_ERR_INVALID_ARG;
  for (int32_t i = 0; i < count; ++i) {
    if (!plans[i] || !s[i] || !same_kernel_family(plans[0], plans[i])) return HQ_ERR_INVALID_ARG;
    if (plans[i]->rotation == HQ_ROT_QJL || plans[i]->tile != HQ_TILE || plans[i]->substream != HQ_SUB)
      return HQ_ERR_UNSUPPORTED;  // single calls only
    for (int32_t j = 0; j < i; ++j)
      if (s[j] == s[i] || s[j]->scan == s[i]->scan) return HQ_ERR_INVALID_ARG;
  }
  for (int32_t b = 0; b < count; b += HQ_GROUP_MAX) {
    hq_encode_group_args g;
    std::memset(&g, 0, sizeof(g));
    int64_t total = 0;
    uint32_t lds_words = 0;
    int32_t members[HQ_GROUP_MAX];
    for (int32_t i = b; i < std::min(count, b + HQ_GROUP_MAX); ++i) {
      int64_t nwg;
      const hq_status st =
          encode_prepare(plans[i], x[i], xt, rows[i], ld[i], s[i], 0, false, &g.m[g.count], &nwg, stream);
      if (st != HQ_OK) return st;
      if (nwg == 0) continue;
      g.wg_begin[g.count] = (uint32_t)total;
      lds_words = std::max(lds_words, g.m[g.count].lds_words);
      members[g.count++] = i;
      total += nwg;
    }
    if (g.count == 0) continue;
    if (total > 0x7FFFFFFF) return HQ_ERR_UNSUPPORTED;
    g.thr = rice_thresholds(plans[members[0]]);  // one lattice and sub-stream length
    if (hq_launch_encode_group(plans[members[0]], g, (uint32_t)total, lds_words, xt, stream))
      return HQ_ERR_HIP;
    for (int32_t k = 0; k < g.count; ++k) s[members[k]]->rows = rows[members[k]];
  }
  return HQ_OK;
}

static void fill_decode_args(const hq_plan_s* p, const hq_stream* s, int64_t row0, int64_t rows,
                             hq_decode_args* a) {
  std::memset(a, 0, sizeof(*a));
  a->payload = s->payload;
  a->cap_words = s->capacity_words;
  a->offsets = s->offsets;
  a->kparam = s->kparam;
  a->norms = s->norms;
  a->first_row = row0;
  a->first_sub = row0 * p->spr;
  a->nsub = rows * p->spr;
  a->spr = p->spr;
  a->tpr = p->tpr;
  a->dmask = p->d_dmask;
  a->dsign16 = p->d_dsign16;
  a->smask = p->d_smask;
  a->qjl = p->d_qjl;
  a->qjlt = p->d_qjlt;
  a->stats = s->stats;
  a->rotation = p->rotation;
  a->dither = p->dither;
  a->norm_fp16 = p->norm_fp16;
  a->lds_words = (uint32_t)p->max_words_sub;
  a->dither_seed = p->dither_seed;
  a->alpha = p->alpha;
  a->alpha_n = p->alpha * (float)p->tile;
  a->tile = p->tile;
  a->mb = p->substream / HQ_SUB;
}

hq_status hq_decode(hq_plan_t p, const hq_stream* s, int64_t row0, int64_t rows, void* y,
                    int32_t yt, int64_t ld, void* stream) {
  if (!p || !s || row0 < 0 || rows < 0) return HQ_ERR_INVALID_ARG;
  if (yt != HQ_BF16 && yt != HQ_FP32) return HQ_ERR_INVALID_ARG;
  if (row0 + rows > s->rows) return HQ_ERR_INVALID_ARG;
  if (rows == 0) return HQ_OK;
  if (!y || ld < p->cols || !s->payload || !s->offsets || !s->kparam || !s->norms)
    return HQ_ERR_INVALID_ARG;
  const int64_t esz = (yt == HQ_BF16) ? 2 : 4;
  if (!aligned16(y) || (ld * esz) % 16 != 0) return HQ_ERR_INVALID_ARG;
  hq_decode_args a;
  fill_decode_args(p, s, row0, rows, &a);
  a.y = y;
  a.ld = ld;
  return hip_status(hq_launch_decode(p, a, yt, stream));
}

size_t hq_gemv_workspace_bytes(hq_plan_t p) { return p ? (size_t)p->cols * sizeof(float) : 0; }

hq_status hq_decode_gemv(hq_plan_t p, const hq_stream* s, int64_t row0, int64_t rows,
                         const void* x, int32_t xt, void* y, int32_t yt, void* workspace,
                         size_t ws_bytes, void* stream) {
  if (!p || !s || row0 < 0 || rows < 0) return HQ_ERR_INVALID_ARG;
  if ((xt != HQ_BF16 && xt != HQ_FP32) || (yt != HQ_BF16 && yt != HQ_FP32)) return HQ_ERR_INVALID_ARG;
  if (row0 + rows > s->rows) return HQ_ERR_INVALID_ARG;
  if (p->rotation || p->dither || p->tile != HQ_TILE || p->substream != HQ_SUB)
    return HQ_ERR_UNSUPPORTED;
  if (rows == 0) return HQ_OK;
  if (!x || !y || !workspace || !s->payload || !s->offsets || !s->kparam || !s->norms)
    return HQ_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(workspace) || ws_bytes < hq_gemv_workspace_bytes(p))
    return HQ_ERR_INVALID_ARG;
  hq_decode_args a;
  fill_decode_args(p, s, row0, rows, &a);
  return hip_status(hq_launch_decode_gemv(p, a, x, xt, (float*)workspace, y, yt, stream));
}

// Tokens per wave of the fused attention: about 16384 waves over the call
// (several rounds of the waves that fit at once, so the last round is a
// small share), from 16 to 1024 tokens each.
static int64_t attn_chunk(const hq_plan_s* k, int64_t batch, int64_t max_tokens) {
  const int64_t work = batch * k->spr * max_tokens;
  return std::min<int64_t>(1024, std::max<int64_t>(16, (work + 16383) / 16384));
}

static int64_t attn_splits(int64_t max_tokens, int64_t chunk) {
  const int64_t per = HQ_WAVES_PER_WG * chunk;
  return (max_tokens + per - 1) / per;
}

// The key pass's scores, one per query head and token, rounded up to 16
// bytes so that what follows stays aligned.
static int64_t attn_scores_floats(int64_t heads, int64_t max_tokens) {
  return (heads * max_tokens + 3) & ~(int64_t)3;
}

size_t hq_attention_workspace_bytes(hq_plan_t k, int64_t batch, int32_t heads_q,
                                    int64_t max_tokens) {
  if (!k || batch < 0 || heads_q <= 0 || max_tokens <= 0) return 0;
  const int64_t nx = attn_splits(max_tokens, attn_chunk(k, batch, max_tokens));
  const int64_t heads = batch * heads_q;
  return (size_t)(heads * HQ_TILE + heads * nx * HQ_TILE + attn_scores_floats(heads, max_tokens) +
                  heads * nx * (HQ_WAVES_PER_WG + 2)) *
         sizeof(float);
}

hq_status hq_decode_attention(hq_plan_t pk, const hq_stream* k, hq_plan_t pv, const hq_stream* v,
                              const void* q, int32_t qt, int64_t batch, int32_t heads_q,
                              float scale, const int32_t* block_table, int32_t max_blocks,
                              int32_t block_tokens, const int32_t* seq_lens,
                              const void* window_k, const void* window_v, int32_t wt,
                              int32_t window, void* out, int32_t ot, void* workspace,
                              size_t ws_bytes, void* stream) {
  if (!pk || !k || !pv || !v || batch < 0) return HQ_ERR_INVALID_ARG;
  if ((qt != HQ_BF16 && qt != HQ_FP32) || (ot != HQ_BF16 && ot != HQ_FP32)) return HQ_ERR_INVALID_ARG;
  if (pk->lattice != pv->lattice || pk->cols != pv->cols || pk->tile != HQ_TILE ||
      pv->tile != HQ_TILE || pk->substream != HQ_SUB || pv->substream != HQ_SUB)
    return HQ_ERR_INVALID_ARG;
  const int64_t hkv = pk->cols / HQ_TILE;
  if (heads_q <= 0 || heads_q % hkv != 0) return HQ_ERR_INVALID_ARG;
  const int64_t group = heads_q / hkv;
  if (group != 1 && group != 2 && group != 4 && group != 8) return HQ_ERR_UNSUPPORTED;
  if (max_blocks <= 0 || block_tokens <= 0 || !std::isfinite(scale)) return HQ_ERR_INVALID_ARG;
  if (window < 0 || window > HQ_ATTN_WINDOW_MAX) return HQ_ERR_INVALID_ARG;
  if (window > 0 && (!window_k || !window_v || !aligned16(window_k) || !aligned16(window_v) ||
                     (wt != HQ_BF16 && wt != HQ_FP32)))
    return HQ_ERR_INVALID_ARG;
  const int64_t max_tokens = (int64_t)max_blocks * block_tokens;
  if (max_tokens > 0x7FFFFFFF) return HQ_ERR_UNSUPPORTED;
  if (batch == 0) return HQ_OK;
  if (!q || !out || !block_table || !seq_lens || !workspace || !aligned16(q) || !aligned16(out) ||
      !aligned16(workspace))
    return HQ_ERR_INVALID_ARG;
  if (ws_bytes < hq_attention_workspace_bytes(pk, batch, heads_q, max_tokens))
    return HQ_ERR_INVALID_ARG;
  if (!k->payload || !k->offsets || !k->kparam || !k->norms || !v->payload || !v->offsets ||
      !v->kparam || !v->norms)
    return HQ_ERR_INVALID_ARG;
  const int64_t chunk = attn_chunk(pk, batch, max_tokens);
  const int64_t nx = attn_splits(max_tokens, chunk);
  if (batch * pk->spr * nx > 0x7FFFFFFF || batch * heads_q > 0x7FFFFFFF) return HQ_ERR_UNSUPPORTED;
  hq_attn_args a;
  std::memset(&a, 0, sizeof(a));
  fill_decode_args(pk, k, 0, k->rows, &a.K);
  fill_decode_args(pv, v, 0, v->rows, &a.V);
  a.q = q;
  a.out = out;
  a.table = block_table;
  a.seq_lens = seq_lens;
  const int64_t heads = batch * heads_q;
  a.qt = (float*)workspace;
  a.part_acc = a.qt + heads * HQ_TILE;
  a.scores = a.part_acc + heads * nx * HQ_TILE;
  a.wmax = a.scores + attn_scores_floats(heads, max_tokens);
  a.part_m = a.wmax + heads * nx * HQ_WAVES_PER_WG;
  a.part_l = a.part_m + heads * nx;
  a.batch = batch;
  a.rows = std::min(k->rows, v->rows);
  if (a.rows > 0x7FFFFFFF) return HQ_ERR_UNSUPPORTED;  // rows travel as 32-bit lane values
  a.heads_q = heads_q;
  a.group = (int32_t)group;
  a.max_blocks = max_blocks;
  a.block_tokens = block_tokens;
  a.chunk = (int32_t)chunk;
  a.nx = (int32_t)nx;
  a.q_bf16 = qt == HQ_BF16;
  a.out_bf16 = ot == HQ_BF16;
  a.lds_words = std::max(a.K.lds_words, a.V.lds_words);
  a.qscale = scale * 1.4426950408889634f;  // log2(e): the softmax runs in base 2
  a.win_k = window_k;
  a.win_v = window_v;
  a.window = window;
  a.win_bf16 = wt == HQ_BF16;
  return hip_status(hq_launch_decode_attention(a, pk->lattice, stream));
}

hq_status hq_decode_group(const hq_plan_t* plans, const hq_stream* const* s, void* const* y,
                          int32_t yt, const int64_t* ld, int32_t count, void* stream) {
  if (count < 0 || (count > 0 && (!plans || !s || !y || !ld))) return HQ_ERR_INVALID_ARG;
  if (yt != HQ_BF16 && yt != HQ_FP32) return HQ_ERR_INVALID_ARG;
  for (int32_t i = 0; i < count; ++i)
    if (!plans[i] || !s[i] || !same_kernel_family(plans[0], plans[i])) return HQ_ERR_INVALID_ARG;
  for (int32_t i = 0; i < count; ++i)
    if (plans[i]->rotation == HQ_ROT_QJL || plans[i]->tile != HQ_TILE || plans[i]->substream != HQ_SUB)
      return HQ_ERR_UNSUPPORTED;  // single calls only
  const int64_t esz = (yt == HQ_BF16) ? 2 : 4;
  for (int32_t b = 0; b < count; b += HQ_GROUP_MAX) {
    hq_decode_group_args g;
    std::memset(&g, 0, sizeof(g));
    int64_t total = 0;
    uint32_t lds_words = 0;
    int32_t first = -1;
    for (int32_t i = b; i < std::min(count, b + HQ_GROUP_MAX); ++i) {
      const hq_plan_s* p = plans[i];
      const int64_t rows = s[i]->rows;
      if (rows == 0) continue;
      if (!y[i] || ld[i] < p->cols || !s[i]->payload || !s[i]->offsets || !s[i]->kparam ||
          !s[i]->norms || !aligned16(y[i]) || (ld[i] * esz) % 16 != 0)
        return HQ_ERR_INVALID_ARG;
      hq_decode_args& a = g.m[g.count];
      fill_decode_args(p, s[i], 0, rows, &a);
      a.y = y[i];
      a.ld = ld[i];
      g.wg_begin[g.count] = (uint32_t)total;
      total += hq_decode_workgroups(a.nsub);
      lds_words = std::max(lds_words, a.lds_words);
      if (first < 0) first = i;
      ++g.count;
    }
    if (g.count == 0) continue;
    if (total > 0x7FFFFFFF) return HQ_ERR_UNSUPPORTED;
    if (hq_launch_decode_group(plans[first], g, (uint32_t)total, lds_words, yt, stream))
      return HQ_ERR_HIP;
  }
  return HQ_OK;
}

hq_status hq_decode_int8(hq_plan_t p, const hq_stream* s, int64_t row0, int64_t rows,
                         int8_t* codes, int64_t ldc, float* g, void* stream) {
  // sub-streams of 512 (any tile: the codes carry no transform)
  if (p && p->substream != HQ_SUB) return HQ_ERR_UNSUPPORTED;
  if (!p || !s || row0 < 0 || rows < 0) return HQ_ERR_INVALID_ARG;
  if (p->lattice == HQ_A2 || p->dither || p->rotation) return HQ_ERR_UNSUPPORTED;
  if (row0 + rows > s->rows) return HQ_ERR_INVALID_ARG;
  if (rows == 0) return HQ_OK;
  if (!codes || !g || ldc < p->cols || ldc % 8 != 0 || ((uintptr_t)codes & 7u) != 0)
    return HQ_ERR_INVALID_ARG;
  hq_decode_args a;
  fill_decode_args(p, s, row0, rows, &a);
  a.y = codes;
  a.ld = ldc;
  a.g = g;
  return hip_status(hq_launch_decode_int8(p, a, stream));
}

hq_status hq_decode_fp8(hq_plan_t p, const hq_stream* s, int64_t row0, int64_t rows,
                        uint8_t* codes, int64_t ldc, float* g, void* stream) {
  // sub-streams of 512 (any tile: the codes carry no transform)
  if (p && p->substream != HQ_SUB) return HQ_ERR_UNSUPPORTED;
  if (!p || !s || row0 < 0 || rows < 0) return HQ_ERR_INVALID_ARG;
  if (p->lattice == HQ_A2 || p->dither || p->rotation) return HQ_ERR_UNSUPPORTED;
  if (row0 + rows > s->rows) return HQ_ERR_INVALID_ARG;
  if (rows == 0) return HQ_OK;
  if (!codes || !g || ldc < p->cols || ldc % 8 != 0 || ((uintptr_t)codes & 7u) != 0)
    return HQ_ERR_INVALID_ARG;
  hq_decode_args a;
  fill_decode_args(p, s, row0, rows, &a);
  a.y = codes;
  a.ld = ldc;
  a.g = g;
  return hip_status(hq_launch_decode_fp8(p, a, stream));
}

hq_status hq_decode_mxfp4(hq_plan_t p, const hq_stream* s, int64_t row0, int64_t rows,
                          uint8_t* codes, uint8_t* scales, void* stream) {
  // sub-streams of 512 (any tile: the codes carry no transform)
  if (p && p->substream != HQ_SUB) return HQ_ERR_UNSUPPORTED;
  if (!p || !s || row0 < 0 || rows < 0) return HQ_ERR_INVALID_ARG;
  if (p->lattice == HQ_A2 || p->dither || p->rotation) return HQ_ERR_UNSUPPORTED;
  if (row0 + rows > s->rows) return HQ_ERR_INVALID_ARG;
  if (rows == 0) return HQ_OK;
  if (!codes || !scales || ((uintptr_t)codes & 3u) != 0) return HQ_ERR_INVALID_ARG;
  hq_decode_args a;
  fill_decode_args(p, s, row0, rows, &a);
  a.y = codes;
  a.ld = p->cols / 2;  // contiguous rows of cols / 2 bytes
  a.g = nullptr;       // the tile factors go into the cast
  a.mxs = scales;
  return hip_status(hq_launch_decode_mxfp4(p, a, stream));
}

static hq_status act_prep(hq_plan_t p, const void* a, int64_t M, int64_t lda, int8_t* xq,
                          float* sx, int fp8, void* stream, uint8_t* mxs = nullptr) {
  if (!p || M < 0) return HQ_ERR_INVALID_ARG;
  if (M == 0) return HQ_OK;
  if (!a || !xq || (fp8 == 2 ? !mxs : !sx) || lda < p->cols || !aligned16(a) ||
      (lda * 2) % 16 != 0 || ((uintptr_t)xq & 3u) != 0)
    return HQ_ERR_INVALID_ARG;
  if (p->cols > 16384 || M > 0x7FFFFFFF) return HQ_ERR_UNSUPPORTED;
  hq_actprep_args args;
  args.a = a;
  args.lda = lda;
  args.M = M;
  args.K = p->cols;
  args.xq = xq;
  args.sx = sx;
  args.dmask = p->d_dmask;
  args.fp8 = fp8;
  args.mxs = mxs;
  args.tile = p->tile;
  return hip_status(hq_launch_act_prep(args, stream));
}

hq_status hq_act_prep_mxfp4(hq_plan_t p, const void* a, int64_t M, int64_t lda, uint8_t* xq,
                            uint8_t* scales, void* stream) {
  return act_prep(p, a, M, lda, (int8_t*)xq, nullptr, 2, stream, scales);
}

hq_status hq_act_prep(hq_plan_t p, const void* a, int64_t M, int64_t lda, int8_t* xq, float* sx,
                      void* stream) {
  return act_prep(p, a, M, lda, xq, sx, 0, stream);
}

hq_status hq_act_prep_fp8(hq_plan_t p, const void* a, int64_t M, int64_t lda, uint8_t* xq,
                          float* sx, void* stream) {
  return act_prep(p, a, M, lda, (int8_t*)xq, sx, 1, stream);
}

static hq_status gemm_blockscaled(hq_plan_t p, const int8_t* xq, const float* sx, int64_t M,
                                  const int8_t* codes, const float* g, int64_t N, void* out,
                                  int32_t ot, int fp8, void* stream, const uint8_t* xs = nullptr,
                                  const uint8_t* ws = nullptr) {
  if (!p || M < 0 || N < 0) return HQ_ERR_INVALID_ARG;
  if (ot != HQ_BF16 && ot != HQ_FP32) return HQ_ERR_INVALID_ARG;
  if (M == 0 || N == 0) return HQ_OK;
  if (!xq || (fp8 == 2 ? (!xs || !ws) : (!sx || !g)) || !codes || !out) return HQ_ERR_INVALID_ARG;
  if (fp8 == 2 && (((uintptr_t)xs & 7u) != 0 || ((uintptr_t)ws & 7u) != 0)) return HQ_ERR_INVALID_ARG;
  if (!aligned16(xq) || !aligned16(codes) || !aligned16(out)) return HQ_ERR_INVALID_ARG;
  hq_gemm_args a;
  a.xq = xq;
  a.sx = sx;
  a.w = codes;
  a.g = g;
  a.out = out;
  a.M = M;
  a.N = N;
  a.K = p->cols;
  a.out_bf16 = (ot == HQ_BF16) ? 1 : 0;
  a.fp8 = fp8;
  a.xs = xs;
  a.ws = ws;
  a.tile = p->tile;
  const int e = hq_launch_gemm(a, stream);
  if (e == -1) return HQ_ERR_UNSUPPORTED;
  return hip_status(e);
}

hq_status hq_gemm_int8_blockscaled(hq_plan_t p, const int8_t* xq, const float* sx, int64_t M,
                                   const int8_t* codes, const float* g, int64_t N, void* out,
                                   int32_t ot, void* stream) {
  return gemm_blockscaled(p, xq, sx, M, codes, g, N, out, ot, 0, stream);
}

hq_status hq_gemm_fp8_blockscaled(hq_plan_t p, const uint8_t* xq, const float* sx, int64_t M,
                                  const uint8_t* codes, const float* g, int64_t N, void* out,
                                  int32_t ot, void* stream) {
  return gemm_blockscaled(p, (const int8_t*)xq, sx, M, (const int8_t*)codes, g, N, out, ot, 1,
                          stream);
}

hq_status hq_gemm_mxfp4_blockscaled(hq_plan_t plan, const uint8_t* xq, const uint8_t* xs, int64_t M,
                                    const uint8_t* codes, const uint8_t* ws, int64_t N, void* out,
                                    int32_t ot, void* stream) {
  return gemm_blockscaled(plan, (const int8_t*)xq, nullptr, M, (const int8_t*)codes, nullptr, N, out,
                          ot, 2, stream, xs, ws);
}

size_t hq_gemm_workspace_bytes(hq_plan_t p, int64_t M, int64_t N) {
  if (!p || M < 0 || N < 0) return 0;
  const size_t K = (size_t)p->cols;
  const auto up = [](size_t v) { return (v + 255) & ~(size_t)255; };
  return up((size_t)M * K) + up((size_t)M * 4) + up((size_t)N * K) + up((size_t)N * (K / 128) * 4);
}

hq_status hq_dequant_gemm_int8(hq_plan_t p, const hq_stream* w, int64_t N, const void* a,
                               int64_t M, void* out, int32_t ot, void* workspace,
                               size_t ws_bytes, void* stream) {
  if (!p || !w || !a || !out || M < 0 || N < 0) return HQ_ERR_INVALID_ARG;
  if (ws_bytes < hq_gemm_workspace_bytes(p, M, N) || !workspace) return HQ_ERR_CAPACITY;
  const size_t K = (size_t)p->cols;
  const auto up = [](size_t v) { return (v + 255) & ~(size_t)255; };
  char* ws = (char*)workspace;
  int8_t* xq = (int8_t*)ws;
  float* sx = (float*)(ws + up((size_t)M * K));
  int8_t* codes = (int8_t*)(ws + up((size_t)M * K) + up((size_t)M * 4));
  float* g = (float*)(ws + up((size_t)M * K) + up((size_t)M * 4) + up((size_t)N * K));
  hq_status st = hq_act_prep(p, a, M, (int64_t)K, xq, sx, stream);
  if (st != HQ_OK) return st;
  st = hq_decode_int8(p, w, 0, N, codes, (int64_t)K, g, stream);
  if (st != HQ_OK) return st;
  return hq_gemm_int8_blockscaled(p, xq, sx, M, codes, g, N, out, ot, stream);
}

}  // extern "C"
