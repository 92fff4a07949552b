// Internal declarations shared by the host plan (hq_host.cpp) and the gfx950
// kernels (hq_kernels.hip) of libhq.so.  Not part of the public ABI.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/hq.h"

#define HQ_KMAX 15
#define HQ_TILE 128              // tile length of the fused and GEMM kernels
#define HQ_TILE_MAX 2048         // longest tile of the codec kernels (four sub-streams)
#define HQ_SUB 512               // symbols per sub-stream the kernels are built for
#define HQ_WAVES_PER_WG 4        // wave64s per workgroup
#define HQ_ENC_SUBS_PER_WAVE 4   // encode: sub-streams per wave, one after another
#define HQ_ENC_WAVES 4           // encode: wave64s per workgroup
#define HQ_ENC_SUBS_PER_WG (HQ_ENC_WAVES * HQ_ENC_SUBS_PER_WAVE)
// Launches of at most this many sub-streams take one sub-stream per wave
// (sixteen waves per workgroup): four times the waves for the same work, so
// a small matrix or a KV append does not leave each SIMD a single long wave.
#define HQ_ENC_SMALL_SUBS 16384
#define HQ_DEC_SUBS_PER_WAVE 4   // decode: consecutive sub-streams per wave
#define HQ_DEC_SMALL 16384       // single decodes below this many sub-streams: one per wave
#define HQ_SCAN_STATUS_OFFSET 128  // bytes before the look-back status array

// Plan: immutable after hq_plan returns.
struct hq_plan_s {
  int32_t tile, lattice, dim, substream, rice_k;
  int64_t cols, tpr, spr;
  float alpha;
  double snr_db;
  int32_t rotation, dither, norm_fp16;
  uint64_t rht_seed, rot_seed, dither_seed;
  // Automatic Rice k of a class with `count` symbols summing to `sum`:
  // k0 = #{t in 1..KMAX : sum >= thr[c][t]} (thr[c][0] unused).
  uint32_t thr[2][HQ_KMAX + 1];
  int64_t max_words_sub;   // capacity bound of one sub-stream, in 32-bit words
  uint32_t* d_dmask;       // device: RHT sign bit per global column (1 = -1)
  uint32_t* d_dsign16;     // device: per column pair, the RHT signs as bf16 sign
                           // bits (bit 15: even column, bit 31: odd column)
  uint32_t* d_smask;       // device: rotation sign bit per tile coordinate
  float* d_qjl;            // device: qjl rotation S (128 x 128, row-major), or null
  float* d_qjlt;           // device: its transpose
  int device;
};

// Arguments of the encode kernel (passed by value).
struct hq_encode_args {
  const void* x;
  int64_t ld;
  int64_t first_row;      // global row of x's first row
  int64_t first_sub;      // global sub-stream index of x's first sub-stream
  int64_t nsub;           // sub-streams in this call
  int64_t spr;            // sub-streams per row
  int64_t tpr;            // tiles per row
  uint32_t* payload;
  int64_t cap_words;
  uint32_t* offsets;
  uint8_t* kparam;
  void* norms;
  const uint32_t* dmask;
  const uint32_t* dsign16;  // RHT signs as bf16 XOR words, one per column pair
  const uint32_t* smask;
  hq_stats* stats;
  unsigned long long* epoch;   // scan scratch: the launch epoch
  unsigned long long* status;  // scan scratch: one look-back word per workgroup
  unsigned long long* wgstat;  // scan scratch: one stats word per workgroup
  uint32_t nwg;
  int32_t append;
  int32_t rice_k;
  int32_t rotation, dither, norm_fp16;
  uint32_t lds_words;     // per-sub-stream assembly buffer, in words
  uint32_t spw;           // sub-streams per wave: HQ_ENC_SUBS_PER_WAVE, or 1 for small launches
  int32_t tile;           // RHT tile (128, or 256 .. 2048 for weight plans)
  int32_t mb;             // 512-symbol blocks per sub-stream (S / 512: 1, 2 or 4)
  uint64_t dither_seed;
  float alpha;
  float alpha_half;       // alpha / 2, exact (the E8 decision works on z / 2)
  const float* qjlt;      // qjl rotation: S^T (row k = column k of S), or null
};

// Automatic Rice-k thresholds of the two symbol classes (the same for every
// plan of one lattice and sub-stream length).
struct hq_rice_thr {
  uint32_t thr0[HQ_KMAX + 1];
  uint32_t thr1[HQ_KMAX + 1];
};

struct hq_decode_args {
  const uint32_t* payload;
  int64_t cap_words;
  const uint32_t* offsets;
  const uint8_t* kparam;
  const void* norms;
  int64_t first_row;
  int64_t first_sub;
  int64_t nsub;
  int64_t spr, tpr;
  void* y;                 // decode: output rows; decode_int8: int8 codes
  int64_t ld;
  float* g;                // decode_int8: per-tile factors (rows x tpr)
  uint8_t* mxs;            // decode_mxfp4: E8M0 scale bytes (rows x cols / 32)
  const uint32_t* dmask;
  const uint32_t* dsign16;  // RHT signs as bf16 XOR words, one per column pair
  const uint32_t* smask;
  hq_stats* stats;
  int32_t rotation, dither, norm_fp16;
  uint32_t lds_words;
  uint64_t dither_seed;
  float alpha;
  float alpha_n;           // alpha * tile, exact
  int32_t tile;            // RHT tile (128, or 256 .. 2048 for weight plans)
  int32_t mb;              // 512-symbol blocks per sub-stream (S / 512: 1, 2 or 4)
  const float* qjl;        // qjl rotation: S (row-major) and S^T, or null
  const float* qjlt;
};

// One-token attention over coded K and V streams (fused decode + attention).
// Workspace: qt [batch * heads_q * 128] query in coded coordinates, then per
// (sequence, query head, token split) the running sum of 128 values, its
// running maximum and its weight.
struct hq_attn_args {
  hq_decode_args K, V;
  const void* q;
  void* out;
  const int32_t* table;     // batch x max_blocks block ids
  const int32_t* seq_lens;  // batch token counts
  float* qt;
  float* part_acc;
  float* part_m;
  float* part_l;
  float* scores;            // key pass: [batch, spr, max tokens, 4 G] base-2 scores
  float* wmax;              // key pass: every wave's largest score per query head
  int64_t batch;
  int64_t rows;             // rows present in both streams
  int32_t heads_q, group;   // query heads, query heads per KV head
  int32_t max_blocks, block_tokens;
  int32_t chunk;            // tokens per wave
  int32_t nx;               // token splits per sequence (4 waves each)
  int32_t q_bf16, out_bf16;
  uint32_t lds_words;       // decode buffer words (the larger of K's and V's)
  float qscale;             // softmax scale times log2(e)
  const void* win_k;        // residual window rings [batch, window, H_kv * 128]
  const void* win_v;
  int32_t window;           // 0: none
  int32_t win_bf16;
};

#define HQ_ATTN_WINDOW_MAX 256  // residual window tokens a call may keep exact
#define HQ_GEMV_WAVE_ROWS 8192  // fused GEMV: one wave per row from this many rows
#define HQ_QJL_STAGE 512        // qjl rotation: LDS floats per wave (four tiles)

// Several matrices in one launch (kernel arguments, by value): member i owns
// workgroups wg_begin[i] .. wg_begin[i + 1] - 1 (the last one to the grid end).
#define HQ_GROUP_MAX 16
struct hq_encode_group_args {
  hq_rice_thr thr;
  hq_encode_args m[HQ_GROUP_MAX];
  uint32_t wg_begin[HQ_GROUP_MAX];
  int32_t count;
};
struct hq_decode_group_args {
  hq_decode_args m[HQ_GROUP_MAX];
  uint32_t wg_begin[HQ_GROUP_MAX];
  int32_t count;
};

struct hq_actprep_args {
  const void* a;
  int64_t lda;
  int64_t M, K;
  int8_t* xq;             // int8, or E4M3 bytes when fp8
  float* sx;
  const uint32_t* dmask;
  int32_t fp8;            // 1: E4M3 at 448 / amax instead of int8 at 127 / amax;
                          // 2: MXFP4 (E2M1 pairs per byte, E8M0 scale per 32 in mxs)
  uint8_t* mxs;           // MXFP4: scale bytes (M x K / 32)
  int32_t tile;           // RHT tile (128 .. 2048)
};

struct hq_gemm_args {
  const int8_t* xq;   // M x K
  const float* sx;    // M
  const int8_t* w;    // N x K
  const float* g;     // N x (K / tile)
  void* out;          // M x N
  int64_t M, N, K;
  int32_t out_bf16;
  int32_t fp8;        // 1: xq and w are E4M3 bytes (fp32 tile sums on the fp8 matrix cores);
                      // 2: MXFP4 (E2M1 pairs per byte, rows of K / 2 bytes)
  const uint8_t* xs;  // MXFP4: activation scale bytes (M x K / 32)
  const uint8_t* ws;  // MXFP4: weight scale bytes (N x K / 32)
  int32_t tile;       // RHT tile: the weight factors' K span (128 .. 2048)
};

// Kernel launchers (hq_kernels.hip); return a hipError_t as int.
int hq_launch_encode(const hq_plan_s* p, const hq_encode_args& a, const hq_rice_thr& t, int xt,
                     void* stream);
int hq_launch_decode(const hq_plan_s* p, const hq_decode_args& a, int yt, void* stream);
int hq_launch_decode_fp8(const hq_plan_s* p, const hq_decode_args& a, void* stream);
int hq_launch_decode_mxfp4(const hq_plan_s* p, const hq_decode_args& a, void* stream);
// Fused decode + GEMV: xtr (cols fp32) receives H D x per tile, then y (rows)
// the decoded rows' products with x.
int hq_launch_decode_attention(const hq_attn_args& a, int lattice, void* stream);
int hq_launch_decode_gemv(const hq_plan_s* p, const hq_decode_args& a, const void* x, int xt,
                          float* xtr, void* y, int yt, void* stream);
int hq_launch_encode_group(const hq_plan_s* p, const hq_encode_group_args& g, uint32_t nwg,
                           uint32_t lds_words, int xt, void* stream);
int hq_launch_decode_group(const hq_plan_s* p, const hq_decode_group_args& g, uint32_t nwg,
                           uint32_t lds_words, int yt, void* stream);
uint32_t hq_decode_workgroups(int64_t nsub);
int hq_launch_decode_int8(const hq_plan_s* p, const hq_decode_args& a, void* stream);
int hq_launch_act_prep(const hq_actprep_args& a, void* stream);
int hq_launch_gemm(const hq_gemm_args& a, void* stream);
int hq_launch_zero(void* ptr, size_t bytes, void* stream);
// Device address of the current device's fixed encode scratch
// (HQ_NOALLOC_SCAN_BYTES); the first call on a device looks it up and clears
// it on `stream`.  0 on success.
int hq_noalloc_scan(void** ptr, void* stream);
