/*
 * hq.h -- C ABI of the MI355X (gfx950) HyperQuant codec library, libhq.so.
 *
 * HyperQuant ("HyperQuant: A Rate-Distortion-Optimal Quantization Pipeline
 * for Large Language and Diffusion Models") encodes every tile of n_tile
 * consecutive scalars along a row as:
 *   RHT (eq. rht, Sec. 3.1 / 4.1) -> [signs rotation, Sec. 4.2] ->
 *   Normalize (Sec. 4.3) -> [subtractive dither, Sec. 4.4 / App. A] ->
 *   nearest point of the E8 / D4 / A2 / Z integer realization (Sec. 4.5) ->
 *   Strip + zig-zag (Sec. 4.6) -> Rice code (Sec. 3.3 / 4.7) in
 *   offset-indexed sub-streams (Sec. 5.3),
 * and decodes by the exact inverse.  The int8 GEMM path (Sec. 4.8, 6.3)
 * multiplies post-RHT lattice codes with per-token int8 activations.
 *
 * Conventions for every entry point:
 *  - Every call returns hq_status; 0 is success, negative values are errors.
 *    No C++ exception crosses this boundary.
 *  - Pointers named d_* or documented as "device" are device memory of the
 *    current HIP device, allocated and owned by the caller.  The library
 *    allocates device memory only inside hq_plan (small constants: sign
 *    bitmasks), released by hq_plan_destroy.
 *  - `stream` is a hipStream_t passed as void*.  All device work is enqueued
 *    on it asynchronously; no call synchronizes the device.  Errors found on
 *    the device (capacity, fp16 norm overflow, corrupt sub-stream) are
 *    reported in the optional hq_stats block and become visible when the
 *    caller synchronizes.
 *  - Matrices are row-major; tiles run along a row (the input/contraction
 *    dimension of a weight, the head dimension of a KV vector).
 */
#ifndef HQ_H
#define HQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HQ_OK = 0,
  HQ_ERR_INVALID_ARG = -1,   /* bad shape, null pointer, out-of-range knob */
  HQ_ERR_UNSUPPORTED = -2,   /* valid for the method, not built for gfx950 here */
  HQ_ERR_CAPACITY = -3,      /* caller buffers too small */
  HQ_ERR_OVERFLOW = -4,      /* fp16 norm overflow or a non-finite input tile */
  HQ_ERR_HIP = -5,           /* a HIP runtime call failed */
  HQ_ERR_CORRUPT = -6,       /* a sub-stream does not decode within its words */
  HQ_ERR_NO_CALIBRATION = -7 /* no SNR <-> bps table for this lattice / k */
} hq_status;

typedef enum { HQ_E8 = 0, HQ_D4 = 1, HQ_A2 = 2, HQ_Z = 3 } hq_lattice;
typedef enum { HQ_BF16 = 0, HQ_FP32 = 1, HQ_FP16 = 2, HQ_INT8 = 3 } hq_dtype;
typedef enum { HQ_ROT_NONE = 0, HQ_ROT_SIGNS = 1, HQ_ROT_QJL = 2 } hq_rotation;

/* Options beyond the five knobs of hq_plan; all-zero means the weight-path
   defaults (no rotation, no dither, fp32 norms, 512-symbol sub-streams, SNR
   from the calibration table). */
typedef struct {
  int32_t rotation;     /* hq_rotation: the KV pre-rotation of Sec. 4.2 */
  int32_t dither;       /* 1 = subtractive dither (Sec. 4.4), KV only */
  uint64_t rot_seed;    /* seed of the +-1 rotation diagonal S */
  uint64_t dither_seed; /* key of the dither generator, fixed for the life of a
                           stream: decode regenerates U from this seed and the
                           global row index, so a stream's rows must all be
                           written and read with one seed.  The fresh draw per
                           forward call (Sec. 4.4, App. A) comes from the row
                           index, which keeps counting across appends. */
  int32_t norm_dtype;   /* HQ_FP32 (default) or HQ_FP16 (KV, Sec. 6.6) */
  int32_t substream;    /* symbols per sub-stream S (Sec. 5.3): 0 = 512; 1024 and
                           2048 for weight plans (no rotation, no dither, fp32
                           norms; any tile), whose encode / decode keep one
                           Rice k and one word offset per S symbols.  The casts
                           (int8 / fp8 / MXFP4), the fused GEMV and attention,
                           and the group calls take S = 512 only
                           (HQ_ERR_UNSUPPORTED otherwise). */
  int32_t use_snr;      /* 1 = take snr_db below instead of the table lookup */
  int32_t reserved0;
  double snr_db;        /* quantization SNR in dB (App. B) when use_snr = 1 */
  const float* qjl;     /* HQ_ROT_QJL: host, tile x tile row-major orthogonal S
                           (the caller's Haar draw, Sec. 4.2); the plan keeps
                           its own device copy.  Encode applies S after the
                           normalization, decode S^T after the undither; each
                           coordinate is the left-to-right fp32 sum of the
                           rounded products. */
} hq_options;

typedef struct hq_plan_s* hq_plan_t;

/* Host-side values derived by hq_plan. */
typedef struct {
  float alpha;                 /* App. B eq. alpha-calib, rounded to fp32 */
  float snr_db;                /* the SNR realizing the target bps */
  int32_t tile, lattice, substream, rice_k;
  int64_t cols, tiles_per_row, subs_per_row;
  int64_t max_words_per_substream; /* deterministic capacity bound */
  int64_t max_words_per_row;       /* = subs_per_row * max_words_per_substream */
} hq_plan_info;

/* hq_plan -- validate the knobs of the paper's problem statement (Sec. 4.9,
 * Tab. params) and derive the codec constants.
 *   tile      n_tile, a power of two: 128 (Sec. 4.1 default), or 256 .. 2048
 *             for weight plans (the sweep of Sec. 7.2; no rotation, dither or
 *             fp16 norms); HQ_ERR_UNSUPPORTED otherwise.
 *   lattice   hq_lattice (Sec. 4.5).
 *   bps       target payload bits per scalar (App. B); mapped to an SNR by the
 *             library's calibration table unless opt->use_snr is set.
 *   rht_seed  seed of the RHT sign diagonal D of eq. rht: d_j = -1 iff the top
 *             bit of the j-th SplitMix64 output for this seed is set, for the
 *             global column j.
 *   rice_k    >= 0: fixed Rice parameter for every sub-stream (D4 codes its
 *             halved symbol at max(k-1, 0), A2 both classes at k); -1: per
 *             sub-stream, the better of the geometric optimum k* of Sec. 3.3
 *             and k* + 1 on the sub-stream's own symbols.
 *   cols      row length of every matrix encoded with this plan; a multiple of
 *             the tile and of the sub-stream length, at most 2^28
 *             (HQ_ERR_UNSUPPORTED above).
 *   opt       nullable hq_options.
 * On success *out receives a plan (owned by the caller, free with
 * hq_plan_destroy) and *info (nullable) its derived values.  Plans are
 * immutable and may be shared by concurrent calls on different streams.
 * Errors: HQ_ERR_INVALID_ARG, HQ_ERR_UNSUPPORTED, HQ_ERR_NO_CALIBRATION,
 * HQ_ERR_HIP. */
hq_status hq_plan(int32_t tile, int32_t lattice, float bps, uint64_t rht_seed, int32_t rice_k,
                  int64_t cols, const hq_options* opt, hq_plan_t* out, hq_plan_info* info);
hq_status hq_plan_destroy(hq_plan_t plan);
hq_status hq_plan_get_info(hq_plan_t plan, hq_plan_info* info);

/* Device-side counters of an encode or decode (all fields device memory of
 * one hq_stats block; the caller zeroes it when it wants fresh counts). */
typedef struct {
  unsigned long long payload_bits;  /* unpadded Rice bits written */
  unsigned long long pad_bits;      /* padding bits to 32-bit word boundaries */
  uint32_t status;                  /* first device error (hq_status, as uint) */
  uint32_t overflow_tiles;          /* fp16 norm overflow / non-finite tiles */
  uint32_t corrupt_substreams;      /* decode: sub-streams that failed to parse */
  uint32_t clamps;                  /* int8 decode: codes clamped to +-127 */
} hq_stats;

/* An encoded matrix (Sec. 5.1 / 5.2): Rice payload plus the per-sub-stream
 * table of Sec. 5.3 (32-bit start offsets and k) and per-tile norms.  All
 * array members are caller-owned device memory; the scalar members are host
 * values the library reads and advances.
 *   payload       capacity_words 32-bit words; sub-streams are word aligned,
 *                 bits LSB-first.  capacity_words >= rows_capacity *
 *                 info.max_words_per_row makes HQ_ERR_CAPACITY impossible.
 *   offsets       rows_capacity * subs_per_row + 1 absolute word offsets:
 *                 sub-stream i occupies [offsets[i], offsets[i+1]).
 *   kparam        rows_capacity * subs_per_row Rice parameter bytes (A2: low
 *                 nibble k of t_y, high nibble k of n_x).
 *   norms         rows_capacity * tiles_per_row stored tile norms (fp32, or
 *                 fp16 bits when the plan's norm_dtype is HQ_FP16).
 *   rows          rows encoded so far; hq_encode sets or advances it.
 *   scan          device scratch (8-byte aligned) of scan_bytes >=
 *                 hq_scan_bytes(plan, rows) bytes for the encoder's
 *                 single-pass cross-workgroup prefix scan.  Zero it once before
 *                 first use; afterwards the kernels keep it consistent
 *                 themselves (an encode can be captured in a HIP graph and
 *                 replayed).  Encodes that run concurrently need their own.
 *   stats         nullable device hq_stats. */
typedef struct {
  uint32_t* payload;
  int64_t capacity_words;
  uint32_t* offsets;
  uint8_t* kparam;
  void* norms;
  int64_t rows_capacity;
  int64_t rows;
  void* scan;
  int64_t scan_bytes;
  hq_stats* stats;
} hq_stream;

/* Bytes of encoder scan scratch needed to encode up to `rows` rows per call. */
size_t hq_scan_bytes(hq_plan_t plan, int64_t rows);

/* hq_encode -- the encode path of Fig. 1 on `rows` rows of x.
 *   x       device, rows x plan.cols, element type xt (HQ_BF16 or HQ_FP32),
 *           row stride ld elements (ld >= cols).
 *   append  0: the rows become rows 0 .. rows-1 of s (s->rows = rows);
 *           1: the rows continue the stream after s->rows (KV
 *           quantize-on-append, Sec. 5.2); their dither keys use the global
 *           row index, and the payload continues at offsets[first sub-stream]
 *           as written by the previous encode on the same stream.  An append
 *           to an empty stream (s->rows = 0) starts at word 0 and writes
 *           offsets[0] = 0 itself, like append = 0.
 * Errors (synchronous): HQ_ERR_INVALID_ARG, HQ_ERR_CAPACITY (rows_capacity),
 * HQ_ERR_HIP.  Device-side: payload capacity and fp16 overflow in s->stats. */
hq_status hq_encode(hq_plan_t plan, const void* x, int32_t xt, int64_t rows, int64_t ld,
                    hq_stream* s, int32_t append, void* stream);

/* hq_encode_noalloc -- hq_encode for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops (the KV
 * quantize-on-append of every forward step), harnesses that forbid it.  The
 * same kernels and bit-identical results, with the look-back scratch taken
 * from a fixed array inside the library (HQ_NOALLOC_SCAN_BYTES = 1 MiB on
 * each device the library runs on, held until the process ends) instead of
 * s->scan, which is ignored and may be null.  The caller still provides
 * every input and output buffer of s.
 *   Limit: hq_scan_bytes(plan, rows) <= 1 MiB, i.e. at most 65528
 *   workgroups of 16 sub-streams = 1048448 sub-streams (536,805,376 scalars
 *   at 512 per sub-stream) per call; larger calls return HQ_ERR_CAPACITY
 *   before any work is enqueued.
 *   The first call on a device looks the array up and clears it on `stream`.
 *   Every call on one device shares that array and leaves its contents for
 *   the next, so calls that overlap on one GPU (two streams, two host
 *   threads) race; the caller serializes them.
 * Allocates nothing (no hipMalloc, hipFree or allocating library call).
 * Errors: as hq_encode, plus HQ_ERR_CAPACITY for the limit above. */
#define HQ_NOALLOC_SCAN_BYTES (1u << 20)
hq_status hq_encode_noalloc(hq_plan_t plan, const void* x, int32_t xt, int64_t rows, int64_t ld,
                            hq_stream* s, int32_t append, void* stream);

/* hq_encode_group -- hq_encode (append = 0) of `count` matrices in as few
 * launches as possible (up to 16 per launch): member i encodes rows[i] rows of
 * x[i] (element type xt, row stride ld[i]) with plans[i] into s[i], exactly
 * as hq_encode would, bit for bit.  Whole-model quantization (Sec. 6.1 codes
 * every linear layer) calls it on a layer's matrices at once, so the small
 * ones share the machine instead of each filling only part of it.
 *   plans   host array of count plans; all of one lattice, tile, sub-stream
 *           length and variant (rotation / dither / fp16 norms on or off
 *           together); seeds, columns and rates may differ.
 *   s       host array of count distinct streams, each with its own scan
 *           scratch.
 * Errors: as hq_encode, plus HQ_ERR_INVALID_ARG for mixed plans or a stream
 * (or scan scratch) given twice, and HQ_ERR_UNSUPPORTED for a qjl plan (a KV
 * rotation: those streams are appended with hq_encode).  Members before a
 * failing one may already have been launched. */
hq_status hq_encode_group(const hq_plan_t* plans, const void* const* x, int32_t xt,
                          const int64_t* rows, const int64_t* ld, hq_stream* const* s,
                          int32_t count, void* stream);

/* hq_decode -- the decode path of Fig. 1, including the explicit inverse RHT,
 * for rows row0 .. row0+rows-1 of s into y (device, element type yt =
 * HQ_BF16 or HQ_FP32, row stride ld).  A sub-stream whose offsets or bits are
 * inconsistent is decoded as zeros and counted in s->stats (never read out of
 * bounds).  With a qjl plan (Sec. 4.2) the product S^T y of each tile runs on
 * the fp32 matrix cores, whose summation order differs from a left-to-right
 * sum by rounding only.  Errors: HQ_ERR_INVALID_ARG, HQ_ERR_HIP. */
hq_status hq_decode(hq_plan_t plan, const hq_stream* s, int64_t row0, int64_t rows, void* y,
                    int32_t yt, int64_t ld, void* stream);
/* (A corrupt sub-stream's 512 outputs are all +-0, dithered streams too: the
   whole sub-stream is dropped, not just the symbols that failed to parse.) */

/* hq_decode_group -- hq_decode of all rows of `count` streams in as few
 * launches as possible (up to 16 per launch): member i decodes s[i] (all
 * s[i]->rows rows) with plans[i] into y[i] (device, element type yt, row
 * stride ld[i]), with the same results as hq_decode.  Plans as for
 * hq_encode_group.  Errors: as hq_decode, plus HQ_ERR_INVALID_ARG for mixed
 * plans and HQ_ERR_UNSUPPORTED for a qjl plan (single calls only, as for
 * hq_encode_group). */
hq_status hq_decode_group(const hq_plan_t* plans, const hq_stream* const* s, void* const* y,
                          int32_t yt, const int64_t* ld, int32_t count, void* stream);

/* hq_decode_int8 -- Rice decode and unstrip without the inverse RHT (Sec. 4.8
 * Cast): the int8 lattice codes c (device, rows x cols, row stride ldc) and
 * the per-tile factors g = r / (alpha n) (device fp32, rows x tiles_per_row),
 * so that a decoded weight row is D H c g.  Codes beyond +-127 are clamped
 * and counted.  E8, D4 and Z only (A2 has a sqrt3 axis): HQ_ERR_UNSUPPORTED
 * otherwise; dithered or rotated streams are HQ_ERR_UNSUPPORTED too (their
 * codes are not D H-coordinates of the weights alone).  Any tile; sub-streams
 * of 512 only (HQ_ERR_UNSUPPORTED otherwise). */
hq_status hq_decode_int8(hq_plan_t plan, const hq_stream* s, int64_t row0, int64_t rows,
                         int8_t* codes, int64_t ldc, float* g, void* stream);

/* hq_act_prep -- activation side of the GEMM: per K-tile y = H D a with the
 * weight plan's signs (so the two rotations cancel), then per token
 * symmetric int8 over the whole row: x_q = clamp(rint(y * 127 / amax), +-127),
 * s_x = amax / 127.  a: device bf16 M x cols (row stride lda); xq: device
 * int8 M x cols; sx: device fp32 [M]. */
hq_status hq_act_prep(hq_plan_t plan, const void* a, int64_t M, int64_t lda, int8_t* xq,
                      float* sx, void* stream);

/* hq_gemm_int8_blockscaled -- out[i, r] = s_x[i] * sum_t g[r, t] *
 * sum_{j in tile t} c[r, j] * x_q[i, j] with exact int32 tile sums on the
 * int8 matrix cores and fp32 accumulation (N = weight rows, K = plan.cols;
 * the tile is the plan's, 128 .. 2048: a longer tile rescales less often).
 * Every operand is contiguous: xq is M x K and codes N x K with row stride
 * K = plan.cols (decode the codes with ldc = plan.cols), g is N x K/tile and
 * out is M x N, HQ_BF16 or HQ_FP32.  The same holds for the fp8 variant. */
hq_status hq_gemm_int8_blockscaled(hq_plan_t plan, const int8_t* xq, const float* sx, int64_t M,
                                   const int8_t* codes, const float* g, int64_t N, void* out,
                                   int32_t ot, void* stream);

/* The fp8 cast path (Sec. 4.8 Cast, Sec. 6.3: E4M3 at the matrix-core
 * boundary; int8 is the path the paper finds better on post-RHT data).  E4M3
 * is the OCP FP8 format (bias 7, 3 fraction bits, largest magnitude 448);
 * every cast rounds to nearest even.
 * hq_decode_fp8 -- as hq_decode_int8, with the codes as E4M3 bytes (exact up
 *   to |c| = 16, then the nearest E4M3 value; beyond 448 saturated and
 *   counted in clamps).  Same plans and errors as hq_decode_int8.
 * hq_act_prep_fp8 -- as hq_act_prep, with x = E4M3(y * 448 / amax) and
 *   s_x = amax / 448.
 * hq_gemm_fp8_blockscaled -- as hq_gemm_int8_blockscaled over the E4M3
 *   values: fp32 tile sums on the f8f6f4 matrix cores (v_mfma_scale_f32_32x32x64_f8f6f4),
 *   each rescaled by g into fp32 accumulators. */
hq_status hq_decode_fp8(hq_plan_t plan, const hq_stream* s, int64_t row0, int64_t rows,
                        uint8_t* codes, int64_t ldc, float* g, void* stream);
hq_status hq_act_prep_fp8(hq_plan_t plan, const void* a, int64_t M, int64_t lda, uint8_t* xq,
                          float* sx, void* stream);
hq_status hq_gemm_fp8_blockscaled(hq_plan_t plan, const uint8_t* xq, const float* sx, int64_t M,
                                  const uint8_t* codes, const float* g, int64_t N, void* out,
                                  int32_t ot, void* stream);

/* The MXFP4 cast path (Sec. 4.8 Cast, Sec. 6.4: the lattice output fed to
 * MXFP4).  MXFP4 is the OCP Microscaling format: blocks of 32 consecutive
 * values along a row (K) share an E8M0 scale 2^X, stored as the byte X + 127,
 * with X = floor(log2 amax) - 2 over the block (-127 for an all-zero block);
 * each element is FP4 E2M1 (magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6), the
 * nearest value to v / 2^X with ties to the even code and saturation at 6.
 * Two elements per byte, the even k in the low nibble.
 * hq_decode_mxfp4 -- as hq_decode_int8, with the reconstruction cast to
 *   MXFP4 (Sec. 4.8 Cast: the reconstruction is cast at the matmul
 *   boundary): in the rotated coordinates, v = g[r, t] c[r, k] (the int8
 *   path's tile factor times the lattice code, one fp32 product), cast per
 *   32-block.  A block lies inside one tile, so the block scales carry the
 *   tile factor and no factor array is returned.  codes device
 *   [rows, cols / 2] bytes (contiguous), scales device [rows, cols / 32]
 *   bytes.  Same plans and errors as hq_decode_int8.
 * hq_act_prep_mxfp4 -- activation side: per K-tile y = H D a as hq_act_prep,
 *   then the MXFP4 cast of y: xq device [M, cols / 2], scales [M, cols / 32];
 *   the block scales carry the magnitude, so there is no per-token factor.
 * hq_gemm_mxfp4_blockscaled -- out[i, r] = sum_k X[i, k] W[r, k] over the
 *   MXFP4 values (element times block scale), accumulated in fp32 on the
 *   gfx950 scaled matrix cores (v_mfma_scale_f32_32x32x64_f8f6f4, E2M1
 *   operands with per-32 E8M0 scales, which carry every factor).  Operands
 *   contiguous, scale arrays 8-byte aligned; out M x N, HQ_BF16 or HQ_FP32. */
hq_status hq_decode_mxfp4(hq_plan_t plan, const hq_stream* s, int64_t row0, int64_t rows,
                          uint8_t* codes, uint8_t* scales, void* stream);
hq_status hq_act_prep_mxfp4(hq_plan_t plan, const void* a, int64_t M, int64_t lda, uint8_t* xq,
                            uint8_t* scales, void* stream);
hq_status hq_gemm_mxfp4_blockscaled(hq_plan_t plan, const uint8_t* xq, const uint8_t* xs, int64_t M,
                                    const uint8_t* codes, const uint8_t* ws, int64_t N, void* out,
                                    int32_t ot, void* stream);

/* Workspace bytes for hq_dequant_gemm_int8 with M tokens and N weight rows. */
size_t hq_gemm_workspace_bytes(hq_plan_t plan, int64_t M, int64_t N);

/* hq_dequant_gemm_int8 -- Y = A W^T from a Rice-coded weight stream w (N rows
 * of plan.cols) and bf16 activations a (device M x cols, unrotated): act
 * prep, decode to int8, then the block-scaled int8 GEMM (Sec. 6.3).
 * workspace: device, >= hq_gemm_workspace_bytes(plan, M, N) bytes.
 * Errors as the three stages. */
hq_status hq_dequant_gemm_int8(hq_plan_t plan, const hq_stream* w, int64_t N, const void* a,
                               int64_t M, void* out, int32_t ot, void* workspace,
                               size_t ws_bytes, void* stream);

/* Workspace bytes for hq_decode_gemv: one fp32 per column (the transformed x). */
size_t hq_gemv_workspace_bytes(hq_plan_t plan);

/* hq_decode_gemv -- y[r] = sum_k W^[row0 + r, k] x[k] for r < rows: the
 * decode of a weight stream fused with a matrix-vector product (the fused
 * decode-GEMV of Sec. 6.6, for one token).  The RHT moves onto x (Sec. 4.1:
 * H is symmetric, so each tile's product is g coord(c) . (H D x)), and the
 * decoded rows never reach memory.
 *   x          device, plan.cols values, HQ_BF16 or HQ_FP32, 16-byte aligned.
 *   y          device, rows values, HQ_FP32 or HQ_BF16 (round to nearest even).
 *   workspace  device, 16-byte aligned, >= hq_gemv_workspace_bytes(plan).
 * The sums run in fp32 in a fixed order (per lane along the row, then a
 * butterfly over the wave; below 8192 rows a row's four waves split its
 * sub-streams and meet in wave order), so they differ from a
 * decode-then-multiply by rounding only and repeat bit for bit for a given
 * row count.
 * Plans with a rotation or a dither (KV streams): HQ_ERR_UNSUPPORTED.  A
 * corrupt sub-stream contributes zero and is reported in s->stats. */
hq_status hq_decode_gemv(hq_plan_t plan, const hq_stream* s, int64_t row0, int64_t rows,
                         const void* x, int32_t xt, void* y, int32_t yt, void* workspace,
                         size_t ws_bytes, void* stream);

/* Workspace bytes for hq_decode_attention with `batch` sequences of at most
 * max_tokens = max_blocks * block_tokens tokens and heads_q query heads:
 * the query in coded coordinates, one score per query head and token, and
 * per query head and token split one partial sum (128 values, a maximum and
 * a weight) and four wave maxima; 0 for invalid arguments. */
size_t hq_attention_workspace_bytes(hq_plan_t k_plan, int64_t batch, int32_t heads_q,
                                    int64_t max_tokens);

/* hq_decode_attention -- one query token per sequence attending over a coded
 * KV cache: out[b, h] = sum_t softmax_t(scale q[b, h] . k^_t) v^_t, k^ and
 * v^ the rows hq_decode would return for the key and value streams (the KV
 * path of Sec. 5.2 read as in Sec. 5.3, for the one-token decoding of Sec.
 * 6.6).  The decoded keys and values never reach memory: a key tile is
 * g D H S (code - U) (Sec. 4.1, 4.2, 4.4, H symmetric), so the query is
 * moved once into those coordinates, each score is g (S H D q) . (code - U),
 * the value sum stays in the same coordinates and one inverse transform per
 * head ends it.
 *   k_plan, k / v_plan, v   key and value plans and streams: one lattice,
 *               tile 128, sub-stream 512 and column count (H_kv * 128: row r
 *               of a stream holds token r's H_kv head vectors); seeds,
 *               rates, rotation, dither and norm precision may differ.  Rows
 *               are used up to min(k->rows, v->rows).
 *   q           device [batch, heads_q, 128], HQ_BF16 or HQ_FP32, 16-byte
 *               aligned; head h reads KV head h / (heads_q / H_kv), a group
 *               of 1, 2, 4 or 8 (HQ_ERR_UNSUPPORTED otherwise).
 *   scale       softmax scale (1 / sqrt(128) for standard attention).
 *   block_table device int32 [batch, max_blocks]: token t of sequence b is
 *               row block_table[b, t / block_tokens] * block_tokens
 *               + t % block_tokens of both streams (a paged cache; one block
 *               per sequence with block_tokens = its length is a plain one).
 *   seq_lens    device int32 [batch] token counts; an empty sequence gives
 *               zeros.
 *   window      residual window W, 0 .. 256 (0: none): the last
 *               min(W, seq_len) tokens of each sequence are read exact from
 *               window_k / window_v instead of the streams (the most recent
 *               tokens kept exact, as in the KV comparison of Sec. 6.7.2).
 *   window_k, window_v  device rings [batch, W, H_kv * 128] of element type
 *               wt (HQ_BF16 or HQ_FP32), 16-byte aligned: token t sits in
 *               slot t % W.  Ignored (may be null) when window = 0.
 *   out         device [batch, heads_q, 128], HQ_FP32 or HQ_BF16 (round to
 *               nearest even), 16-byte aligned.
 *   workspace   device, 16-byte aligned, >= hq_attention_workspace_bytes(
 *               k_plan, batch, heads_q, max_blocks * block_tokens).
 * Sums run in fp32 in an order fixed by the call's shape (batch, heads,
 * max_blocks * block_tokens), so results repeat bit for bit and differ from
 * decode-then-attend by rounding only.  Device-side errors go to k->stats:
 * a length outside 0 .. max_blocks * block_tokens is clamped and a block id
 * whose rows lie outside the streams is skipped (both HQ_ERR_INVALID_ARG);
 * a corrupt sub-stream counts as HQ_ERR_CORRUPT.  Host errors:
 * HQ_ERR_INVALID_ARG, HQ_ERR_UNSUPPORTED, HQ_ERR_HIP. */
hq_status hq_decode_attention(hq_plan_t k_plan, const hq_stream* k, hq_plan_t v_plan,
                              const hq_stream* v, const void* q, int32_t qt, int64_t batch,
                              int32_t heads_q, float scale, const int32_t* block_table,
                              int32_t max_blocks, int32_t block_tokens, const int32_t* seq_lens,
                              const void* window_k, const void* window_v, int32_t wt,
                              int32_t window, void* out, int32_t ot, void* workspace,
                              size_t ws_bytes, void* stream);

/* The library's automatic Rice-k rule for `count` symbols summing to `sum`
 * (the geometric optimum k* of Sec. 3.3), as the kernels evaluate it. */
int32_t hq_rice_kstar(int64_t count, int64_t sum);

/* Calibration lookup (App. B): the SNR whose realized payload rate is `bps`
 * for this lattice and Rice setting; HQ_ERR_NO_CALIBRATION if no table. */
hq_status hq_calibrated_snr(int32_t lattice, int32_t rice_k, float bps, double* snr_db);

const char* hq_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* HQ_H */
