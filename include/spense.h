/*
 * libspense - the Spense hybrid 2:4-sparse / dense linear layer on AMD Instinct MI355X
 * (gfx950), hand-written HIP kernels behind a plain C ABI.
 *
 * The layer computes Y = X W^T (PyTorch's convention, paper sec. 3.1.1) where the weight
 * W (N x K, out x in) is stored in the Spense format of sec. 3.2: two contiguous regions,
 * one pruned to 2:4 (Eq. (1): at most two non-zeros in every aligned group of four
 * input-dimension entries of a row) and stored compressed as values plus 2-bit
 * positions (sec. 3.1.1), the other kept dense.  The dense region is the trailing one
 * (sec. 3.3.2, Table "front_back"):
 *   - output-split (SPENSE_SPLIT_OUTPUT): rows [0, dense_begin) are 2:4, rows
 *     [dense_begin, N) are dense; the two parts produce disjoint output columns.
 *   - input-split (SPENSE_SPLIT_INPUT): columns [0, dense_begin) are 2:4, columns
 *     [dense_begin, K) are dense; both parts accumulate into the same outputs.
 * Gate/up-style projections use output-split and down-style ones input-split (sec. 3.2).
 *
 * Conventions for every call:
 *   - All int return values are SPENSE_OK (0) or a negative spense_status.  On error
 *     nothing has been launched and no output buffer has been written, except where a
 *     call says otherwise.  spense_last_error() returns a thread-local message.
 *   - Matrices are row-major with an explicit leading dimension in elements.
 *   - Device pointers are plain HIP device addresses; the caller allocates and frees
 *     every buffer.  The library allocates no device or host memory of its own (the
 *     one exception, spense_gemm_noalloc's file-scope scratch array, is described
 *     there).  The only other state it keeps is set once per device and never changes
 *     afterwards (the gfx950 check, the large-M kernels' LDS attributes, both under
 *     std::call_once or atomics), a per-thread cache of recent execution plans and the
 *     dispatch-log level (spense_set_log, an atomic); none of it changes a result.  The
 *     only environment variable read is SPENSE_LOG, once, when the library loads.
 *   - Calls take a hipStream_t (0 = the null stream) and are asynchronous on it unless
 *     stated otherwise.
 */
#ifndef SPENSE_H_
#define SPENSE_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPENSE_ABI_VERSION 13

typedef enum spense_status {
  SPENSE_OK = 0,
  SPENSE_ERR_ARG = -1,    /* NULL pointer, negative size, unknown enum, bad split point */
  SPENSE_ERR_ALIGN = -2,  /* a size or pointer misses the alignment the kernels need */
  SPENSE_ERR_MASK = -3,   /* the mask keeps more than 2 of 4 in some sparse-region group */
  SPENSE_ERR_WS = -4,     /* workspace missing or too small */
  SPENSE_ERR_HIP = -5,    /* a HIP runtime call or kernel launch failed */
  SPENSE_ERR_DEVICE = -6, /* the current device is not a gfx950 */
  SPENSE_ERR_NUMERIC = -7 /* a Hessian is not positive definite even after damping */
} spense_status;

typedef enum spense_dtype {
  SPENSE_FP8_E4M3FN = 1, /* OCP fp8 e4m3fn, 1 byte; NaN = 0x7f/0xff, max 448 */
  SPENSE_BF16 = 2,       /* bfloat16, 2 bytes */
  SPENSE_F32 = 3         /* fp32, 4 bytes: inputs of the quantisation calls only */
} spense_dtype;

typedef enum spense_split {
  SPENSE_SPLIT_OUTPUT = 0, /* split along N: 2:4 rows first, dense rows last */
  SPENSE_SPLIT_INPUT = 1   /* split along K: 2:4 columns first, dense columns last */
} spense_split;

/* Storage order of a packed weight's three buffers (spense_packed_t.layout). */
typedef enum spense_layout_kind {
  SPENSE_LAYOUT_ROWMAJOR = 0, /* the canonical layout of spense_layout_t */
  SPENSE_LAYOUT_TILED = 1     /* the gfx950 execution layout of spense_tiled_layout_t */
} spense_layout_kind;

/* Output flags for spense_gemm / spense_dense_gemm. */
#define SPENSE_OUT_BF16 0u /* Y is bfloat16, round to nearest even (default) */
#define SPENSE_OUT_F32 1u  /* Y is fp32 (the value before the bf16 rounding; for tests) */

/*
 * Geometry of a packed weight, filled by spense_layout.  All counts are in elements
 * of the weight dtype, except meta_* which count 32-bit words.
 *
 * Sparse region (sparse_rows x sparse_cols logical entries):
 *   values: sparse_rows x values_ld elements; entry (r, 2g + j), j in {0, 1}, is the
 *           j-th kept value of group g (logical columns 4g..4g+3 of the region) in
 *           ascending position order.
 *   meta:   sparse_rows x meta_ld uint32 words; group g of row r owns bits
 *           [4(g%8), 4(g%8)+4) of word (r, g/8): i0 | i1 << 2 with 0 <= i0 < i1 <= 3 the
 *           positions of the two stored values inside the group.  Unused bits are 0.
 * Dense region: dense_rows x dense_ld elements, row-major, the trailing rows (output-
 *   split) or the trailing columns of every row (input-split) of W unchanged.
 */
typedef struct spense_layout_t {
  int64_t sparse_rows, sparse_cols; /* logical extent of the 2:4 region */
  int64_t values_ld;                /* = sparse_cols / 2 */
  int64_t meta_ld;                  /* = sparse_cols / 32 */
  int64_t dense_rows, dense_cols;
  int64_t dense_ld; /* = dense_cols */
  size_t values_bytes, meta_bytes, dense_bytes;
} spense_layout_t;

/*
 * Tiled execution layout (fp8 only), filled by spense_tiled_layout.  The same bytes as
 * the row-major layout, reordered so that every 16-byte load of the GEMM kernel's wave
 * comes from one contiguous kilobyte (row-major storage makes each load instruction read
 * sixteen 64-byte pieces of sixteen rows).  Each region is cut into tiles of 16 rows
 * (the last one padded with zero rows) and chunks of 512 logical columns (the last one
 * padded with zero columns).  With i in [0,16), q, j in [0,4), p in {0,1}, b in [0,16):
 *   values: 4096 bytes per (tile t, chunk c) at byte (t * sparse_chunks + c) * 4096;
 *           byte 1024 j + 16 (i + 16 q) + b is row-major value byte 256 c + 64 j + 16 q + b
 *           of row 16 t + i of the 2:4 region.
 *   meta:   1024 bytes per (t, c) at byte (t * sparse_chunks + c) * 1024; bytes
 *           16 (i + 16 q) .. +15 are metadata words 16 c + 4 q .. +3 of row 16 t + i.
 *   dense:  8192 bytes per (t, c) at byte (t * dense_chunks + c) * 8192; byte
 *           1024 (2 j + p) + 16 (i + 16 q) + b is dense byte 512 c + 128 j + 64 p + 16 q + b
 *           of row 16 t + i of the dense region.
 * Positions past a region's rows or columns hold zero.  (cuSPARSELt likewise keeps its
 * compressed matrices in a device-specific order.)
 */
typedef struct spense_tiled_layout_t {
  int64_t sparse_tiles, sparse_chunks; /* 16-row tiles x 512-column chunks, 2:4 region */
  int64_t dense_tiles, dense_chunks;   /* the same for the dense region */
  size_t values_bytes, meta_bytes, dense_bytes;
} spense_tiled_layout_t;

/*
 * A packed weight: POD descriptor plus three caller-owned device buffers laid out as in
 * spense_layout_t (layout = SPENSE_LAYOUT_ROWMAJOR, with the leading dimensions) or as
 * in spense_tiled_layout_t (layout = SPENSE_LAYOUT_TILED; the leading dimensions are
 * ignored).  The library never takes ownership of the buffers.
 */
typedef struct spense_packed_t {
  int32_t dtype;       /* spense_dtype */
  int32_t split;       /* spense_split */
  int64_t N, K;        /* logical weight shape (out x in) */
  int64_t dense_begin; /* first dense row (output-split) or column (input-split) */
  void* values;
  int64_t values_ld;
  uint32_t* meta;
  int64_t meta_ld;
  void* dense;
  int64_t dense_ld;
  int32_t layout; /* spense_layout_kind; 0 (row-major) when the field is left zero */
} spense_packed_t;

/*
 * Fill *out with the packed geometry of an N x K weight split at dense_begin.
 * Pure host call.  Requirements (SPENSE_ERR_ALIGN otherwise): K % 32 == 0, and for
 * input-split dense_begin % 32 == 0.  0 <= dense_begin <= N (output) or K (input),
 * else SPENSE_ERR_ARG.  Sec. 3.2 (format), sec. 3.1.1 (compressed storage).
 */
int spense_layout(int64_t N, int64_t K, int32_t dtype, int32_t split, int64_t dense_begin,
                  spense_layout_t* out);

/*
 * Fill *out with the tiled execution layout of the same weight (see
 * spense_tiled_layout_t).  Pure host call; the same requirements as spense_layout, and
 * dtype must be SPENSE_FP8_E4M3FN (SPENSE_ERR_ARG otherwise).
 */
int spense_tiled_layout(int64_t N, int64_t K, int32_t dtype, int32_t split, int64_t dense_begin,
                        spense_tiled_layout_t* out);

/* Device workspace (bytes) needed by spense_compress: a counter. */
size_t spense_compress_workspace_size(void);

/*
 * Pack W (N x K device matrix, leading dimension ldw elements, dtype codes) into the
 * Spense format.  mask is an optional N x K device byte matrix (leading dimension ldm);
 * non-zero means keep.  With mask == NULL an entry is kept when its bit pattern is not
 * all zeros.  The mask is ignored in the dense region.  A sparse-region group that keeps
 * fewer than two entries is padded with its smallest non-kept positions holding +0.
 *
 * `packed` must have dtype, split, N, K, dense_begin and the three buffer pointers and
 * leading dimensions set as spense_layout describes (leading dimensions may be larger).
 * ws: device memory of spense_compress_workspace_size() bytes.
 *
 * SYNCHRONOUS: waits for `stream` to finish, to read the count of groups that keep more
 * than two entries.  If that count is non-zero the call returns SPENSE_ERR_MASK, stores
 * the count in *bad_groups (if not NULL) and the packed buffers hold unspecified data.
 * Sec. 3.1.1 (Eq. (1), compressed storage), sec. 3.2 (regions).
 */
int spense_compress(const void* W, int64_t ldw, const uint8_t* mask, int64_t ldm, const spense_packed_t* packed,
                    int64_t* bad_groups, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Inverse of spense_compress: W_out (N x K, leading dimension ldw) receives the dense
 * matrix, with +0 at every sparse-region position the metadata does not name.
 * Asynchronous.  A test aid; sec. 3.1.1.
 */
int spense_decompress(const spense_packed_t* packed, void* W_out, int64_t ldw, hipStream_t stream);

/*
 * Reorder a row-major packed weight (src, as written by spense_compress) into the tiled
 * execution layout (dst: the same dtype, split, N, K and dense_begin, layout =
 * SPENSE_LAYOUT_TILED, buffers of the sizes spense_tiled_layout gives, not overlapping
 * src).  Every destination byte is written, padding included.  Asynchronous; fp8 only.
 * An offline step like spense_compress: the format is the one of sec. 3.1.1 and 3.2, in
 * the order the gfx950 kernels read it.
 */
int spense_tile(const spense_packed_t* src, const spense_packed_t* dst, hipStream_t stream);

/*
 * Device workspace (bytes) that spense_gemm needs for this M and weight; 0 means none.
 * It is non-zero when the plan cuts K into slices run by separate workgroups (weights
 * with fewer than 1024 16-row tiles at up to 64 tokens, when every slice keeps enough of
 * K: e.g. k / v and down from one token on, o from 17 tokens; few-row or long-K weights
 * at two or three 64-token blocks; long-K weights of fewer than 768 tiles at 65-128 and
 * 193-320 tokens, as 128-token blocks in 2 to 6 slices): S x M x N fp32 partial sums,
 * added in slice order by a second kernel of the same call.  The workspace is only
 * scratch between the two kernels of one call; calls that overlap on one workspace race.
 */
size_t spense_gemm_workspace_size(int64_t M, const spense_packed_t* packed);

/*
 * Y = X W^T for a packed Spense weight (either layout), in one kernel launch (two when
 * the plan slices K, see spense_gemm_workspace_size):
 *   Y[m, n] = round((sum_k x[m, k] * w[n, k]) * w_scale[n] * x_scale[m])
 * X: M x K device matrix of the weight's dtype, leading dimension ldx (elements).
 * w_scale: N fp32 per-output-channel scales; x_scale: M fp32 per-token scales; either
 *   may be NULL, meaning 1.0.  The two multiplications are separate fp32 roundings in
 *   the order shown.
 * Y: M x N device matrix, leading dimension ldy (elements), bf16 (round to nearest even)
 *   or fp32 with SPENSE_OUT_F32.
 * The sparse region runs on gfx950 structured-sparse matrix instructions, the dense
 * region on dense ones; with output-split they write disjoint columns, with input-split
 * one fp32 accumulator crosses the region boundary (no rounding between the regions).
 * Accumulation is fp32; the summation order differs from a sequential sum.
 * Alignment (SPENSE_ERR_ALIGN): X, values, meta, dense 16-byte aligned; ldx, values_ld,
 * dense_ld multiples of 16 bytes; K % 32 == 0 (and dense_begin % 32 for input-split).
 * Sec. 3.2 (output-split / input-split), sec. 3.1.1.
 */
int spense_gemm(const void* X, int64_t M, int64_t ldx, const spense_packed_t* packed, const float* w_scale,
                const float* x_scale, void* Y, int64_t ldy, uint32_t out_flags, void* ws, size_t ws_bytes,
                hipStream_t stream);

/* Scratch that spense_gemm_noalloc holds on each device it runs on (16 MiB). */
#define SPENSE_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

/*
 * spense_gemm for callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops and harnesses that forbid allocation): the same arguments
 * without the workspace, the same plan and kernels, results bit for bit equal to
 * spense_gemm's.  The fp32 partial sums of K-sliced plans go to a scratch array of
 * SPENSE_NOALLOC_SCRATCH_BYTES that the library keeps on each device it runs on until the
 * process ends (a K-sliced plan needs slices x M x N x 4 bytes: 15.7 MB for a 5120-row
 * down projection at 65-128 tokens, 6 slices, or at 193-256, 3).  Every call on a device shares that array, which keeps the last call's
 * partial sums (each call writes every partial it reads): calls that overlap on one
 * device, from any stream or thread, race and must be serialised by the caller.
 * SPENSE_ERR_WS if the plan would need more scratch than the array holds.  No hipMalloc,
 * hipFree or other allocation on any path.  Errors otherwise as spense_gemm.
 */
int spense_gemm_noalloc(const void* X, int64_t M, int64_t ldx, const spense_packed_t* packed, const float* w_scale,
                        const float* x_scale, void* Y, int64_t ldy, uint32_t out_flags, hipStream_t stream);

/*
 * Parts of spense_gemm's execution plan forced by the caller, for tests that check every
 * kernel and workgroup shape bit for bit, and for tuning sweeps.  spense_gemm itself
 * reads no such setting: its plan depends only on the dtype, M and the weight geometry.
 * A zero field (or -1 where stated) leaves that choice to the planner.  A forced plan
 * changes the order of the fp32 sums, not what is summed.
 */
typedef struct spense_plan_override_t {
  int32_t kernel;           /* 0 planner; 1 K split over a workgroup's waves (row-major
                               layout only); 2 rows split, activations staged in LDS;
                               3 large-M tiles of 128 rows x 256 tokens; 4 large-M tiles
                               of 256 x 256 (tiled layout; a row-major weight runs 3)
                               (3 and 4 fp8 only); 5 rows split with two 64-token halves
                               per workgroup, 128 tokens a block (tiled fp8; no shape
                               fields; ksplit allowed) */
  int32_t row_tiles;        /* K-split kernel: 16-row tiles per workgroup (1, 2, 4); with
                               kernel 2: 1 or 2 (with 4 waves) */
  int32_t waves;            /* K-split kernel: 4, 8 or 16 waves per workgroup (row_tiles
                               1 allows all three, 2 allows 4 and 8, 4 allows 4); row-split:
                               4 or 8; kernel 3: 4 or 8; kernel 4: 8 */
  int32_t act_tiles;        /* at most this many 16-token activation tiles per token block
                               (1 or 2) */
  int32_t ksplit;           /* row-split kernel: K slices, 1 .. 8 (capped at the chunk count) */
  int32_t waves_used;       /* row-split kernel: waves owning rows, every region */
  int32_t waves_used_dense; /* row-split kernel: the same for the dense region only */
  int32_t waves_used_24;    /* row-split kernel: the same for the 2:4 region only */
  int32_t block_order;      /* row-split kernel with several token blocks: -1 planner, 0 grid
                               of (row group, token block), 1 a row group's blocks adjacent,
                               2 a row group's blocks on one XCD */
  int32_t xcd_order;        /* large-M kernel: -1 planner, 0 plain order, 1 XCD-aware where
                               the grid allows it */
  int32_t u8;               /* K-split kernel, one activation tile, one row tile, 4 or 8
                               waves: 1 = eight instruction steps per batch of loads */
  int32_t half_row_blocks;  /* 256 x 256 kernel: -1 planner, else this many 256-row blocks
                               at the end of the last region run as 256 x 128 tiles, after
                               all 256 x 256 tiles (capped at the region's row blocks) */
  int32_t resident_x;       /* row-split kernel with one or two token tiles, tiled fp8, 8
                               waves, no K slices: 0 planner, 1 activations staged chunk by
                               chunk, 2 the whole K range of activations kept in LDS (where
                               it fits: 160 KB, i.e. 20 chunks of 512 columns with one token
                               tile, 10 with two) */
} spense_plan_override_t;

/*
 * spense_gemm with parts of the plan forced (plan may be NULL: exactly spense_gemm).
 * Arguments, results and errors as spense_gemm; SPENSE_ERR_ARG also for an override the
 * weight or dtype cannot run (e.g. the K-split kernel on a tiled weight, the large-M
 * kernel on bf16, a workgroup shape outside the lists above).
 * spense_gemm_planned_workspace_size: the workspace this plan needs (0 also when the
 * override is rejected).
 */
size_t spense_gemm_planned_workspace_size(int64_t M, const spense_packed_t* packed,
                                          const spense_plan_override_t* plan);
int spense_gemm_planned(const void* X, int64_t M, int64_t ldx, const spense_packed_t* packed, const float* w_scale,
                        const float* x_scale, void* Y, int64_t ldy, uint32_t out_flags, void* ws, size_t ws_bytes,
                        const spense_plan_override_t* plan, hipStream_t stream);

/*
 * Several Spense weights that share the activations X and K, in one launch: Y[i] =
 * X W_i^T for i < count (sec. 3.2, output-split, as spense_gemm for each weight; e.g.
 * the q, k and v projections of a layer, or gate and up).  Each weight keeps its own
 * 2:4 and dense regions and its own output; together they fill the GPU where one small
 * weight alone would need K slices and a second pass.  Up to 64 tokens it runs the
 * row-split kernel over all weights; where the weights' 256-row blocks times the 256-token
 * blocks of M fill the GPU (at least 160 tiles) one 256 x 256 tile grid covers all
 * weights; in between it issues one launch per weight with that weight's own plan held
 * to one K slice (several launches).  Weights: fp8 e4m3fn, output-split, tiled layout
 * (spense_tile), equal K; count in [1, 4].  w_scales (array of count
 * pointers, or NULL for none) and x_scale as in spense_gemm; Y[i] (bf16 or fp32 per
 * out_flags) with leading dimension ldy[i] >= N_i.  Results equal spense_gemm's up to the
 * order of the fp32 sum (no K slices here).  Allocates nothing; asynchronous.
 * SPENSE_ERR_ARG for NULL arrays or pointers, count outside [1, 4], mixed K, dtype,
 * split or layout; SPENSE_ERR_ALIGN as spense_gemm.
 */
int spense_gemm_grouped(const void* X, int64_t M, int64_t ldx, int32_t count, const spense_packed_t* const* packed,
                        const float* const* w_scales, const float* x_scale, void* const* Y, const int64_t* ldy,
                        uint32_t out_flags, hipStream_t stream);

/*
 * The gate and up projections of a GLU MLP and the GLU step between them, in one launch
 * (sec. 3.2 output-split weights; sec. 3.3.1, Eq. (4), the activation read as SiLU):
 *   g = X Wg^T, u = X Wu^T, each scaled as in spense_gemm ((acc * w_scale[n]) *
 *   x_scale[m], fp32), then H[m, n] = u * g / (1 + exp(-g)) in fp32 with the same
 *   arithmetic as spense_glu_quantize_fp8 (so quantising H with spense_quantize_fp8
 *   gives the codes and scales that spense_glu_quantize_fp8 gives for the G and U of
 *   spense_gemm_grouped, bit for bit).  A workgroup computes gate and up tiles of the
 *   same rows and pairs them on chip, so G and U are never written.  Like
 *   spense_gemm_grouped it runs the row-split kernel, which pays for up to 64 tokens;
 *   for more, two spense_gemm calls (fp32 out) and spense_glu_quantize_fp8 are faster.
 * gate, up: fp8 e4m3fn, output-split, tiled layout, with equal N, K and dense_begin.
 * X: M x K fp8 codes (ldx bytes, 16-byte aligned, ldx a multiple of 16).  w_scale_gate /
 * w_scale_up: N fp32 each or NULL; x_scale: M fp32 or NULL.  H: M x N fp32, leading
 * dimension ldh >= N (caller-owned).  Allocates nothing; asynchronous.
 * SPENSE_ERR_ARG for NULL pointers, mismatched or unsupported weights, K = 0, ldh < N;
 * SPENSE_ERR_ALIGN for a misaligned X or H.
 */
int spense_gemm_glu(const void* X, int64_t M, int64_t ldx, const spense_packed_t* gate, const spense_packed_t* up,
                    const float* w_scale_gate, const float* w_scale_up, const float* x_scale, float* H, int64_t ldh,
                    hipStream_t stream);

/* Device workspace (bytes) that spense_gemm_glu_fp8 needs for M tokens and N gate / up
 * rows (0 for sizes below 1 or above 2^31-1). */
size_t spense_gemm_glu_fp8_workspace_size(int64_t M, int64_t N);

/*
 * The producer half of the GLU MLP (sec. 3.3.1, Eq. (4)) in two launches: gate and up
 * with the GLU step in their epilogue, as spense_gemm_glu, writing H into the workspace
 * together with each workgroup's per-token maximum of |h|; then the per-token fp8
 * quantisation of H from those maxima (one workgroup per 2048 columns of a token row).
 * q (M x N e4m3fn codes, ldq bytes) and scales (M fp32) equal, bit for bit, those of
 * spense_quantize_fp8 applied to spense_gemm_glu's H, and of spense_glu_quantize_fp8
 * applied to the fp32 G and U of spense_gemm_grouped: the input of the down projection.
 * Weights, X and scales as spense_gemm_glu.  ws: device workspace of at least
 * spense_gemm_glu_fp8_workspace_size(M, N) bytes, 256-byte aligned, caller-owned, its
 * contents not kept.  Asynchronous; allocates nothing.  Errors as spense_gemm_glu,
 * SPENSE_ERR_ARG for a NULL q or scales or ldq < N, SPENSE_ERR_WS for a missing or small
 * workspace, SPENSE_ERR_ALIGN for a misaligned one.
 */
int spense_gemm_glu_fp8(const void* X, int64_t M, int64_t ldx, const spense_packed_t* gate, const spense_packed_t* up,
                        const float* w_scale_gate, const float* w_scale_up, const float* x_scale, uint8_t* q,
                        int64_t ldq, float* scales, void* ws, size_t ws_bytes, hipStream_t stream);

/* Device workspace (bytes) that spense_dense_gemm needs; same rules as above. */
size_t spense_dense_gemm_workspace_size(int64_t M, int64_t N, int64_t K, int32_t dtype);

/*
 * The dense baseline: Y = X W^T for a plain N x K weight W (leading dimension ldw), with
 * the same scales, epilogue, alignment rules and dense kernel as spense_gemm.  Used as
 * the speed reference for the Spense format (every weight byte stored).
 */
int spense_dense_gemm(const void* X, int64_t M, int64_t ldx, const void* W, int64_t ldw, int64_t N, int64_t K,
                      int32_t dtype, const float* w_scale, const float* x_scale, void* Y, int64_t ldy,
                      uint32_t out_flags, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Per-token fp8 quantisation of activations, as spense_gemm consumes them (the inputs of
 * the GLU MLP's GEMMs, sec. 3.3.1 Eq. (4)):
 *   scales[m] = max_k |a[m, k]| / 448 (1.0 for an all-zero row),
 *   q[m, k] = e4m3fn(a[m, k] / scales[m]),
 * in fp32 with a correctly rounded division; the encode rounds to nearest, ties to an
 * even mantissa, and saturates to +-448; NaN stays NaN (0xff, whatever its sign).
 * src: M x K device matrix of src_type (SPENSE_BF16 or SPENSE_F32), leading dimension
 *   ld_src (elements).  q: M x K fp8 codes, leading dimension ldq (bytes).  scales: M
 *   fp32.  Caller-owned device buffers; q and scales must not overlap src.
 * One workgroup per row.  Asynchronous.  SPENSE_ERR_ARG for NULL pointers, negative
 * sizes, ld below K, M above 2^31-1 or another src_type.
 */
int spense_quantize_fp8(const void* src, int32_t src_type, int64_t M, int64_t K, int64_t ld_src, uint8_t* q,
                        int64_t ldq, float* scales, hipStream_t stream);

/*
 * The GLU step of the MLP between the output-split gate / up GEMMs and the input-split
 * down GEMM (sec. 3.2 and sec. 3.3.1, Eq. (4), the activation read as SiLU), fused with
 * the per-token fp8 quantisation of its result:
 *   h[m, i] = u[m, i] * g[m, i] / (1 + exp(-g[m, i])) in fp32 (exp and the reciprocal
 *   from the hardware approximations, within a few ulp), then scales / q of h as in
 *   spense_quantize_fp8.
 * g, u: M x I device matrices of gu_type (SPENSE_BF16 or SPENSE_F32), leading dimensions
 *   ldg, ldu (elements), with the same intermediate-index order (the order of the down
 *   weight's input columns).  q: M x I codes (ldq bytes); scales: M fp32.  Caller-owned.
 * Asynchronous.  Errors as spense_quantize_fp8.
 */
int spense_glu_quantize_fp8(const void* g, int64_t ldg, const void* u, int64_t ldu, int32_t gu_type, int64_t M,
                            int64_t I, uint8_t* q, int64_t ldq, float* scales, hipStream_t stream);

/*
 * SpenseGPT+ dense-index priorities of a GLU MLP (sec. 3.3.1: the Wanda-style element
 * score |W_ij| sqrt(H_jj) of Eq. (8) averaged per intermediate index, Eq. (9), each
 * projection's vector divided by its mean plus eps, Eq. (10), the three summed, Eq. (11);
 * for down the index is a column, so its scores average over that column):
 *   raw[0*I + i] = mean_j |w_gate[i, j]| sqrt(h_in[j]),   raw[1*I + i] likewise for w_up,
 *   raw[2*I + i] = mean_n |w_down[n, i]| sqrt(h_mid[i]),
 *   total[i] = sum_v raw[v*I + i] / (mean_i raw[v*I + i] + eps).
 * w_gate, w_up: I x D (leading dimension ld_gu elements); w_down: D x I (ld_down); all of
 * wtype SPENSE_BF16 or SPENSE_F32 (the weights before quantisation).  h_in: D fp32, the
 * diagonal of X^T X for the MLP input; h_mid: I fp32, the same for the down projection's
 * input.  raw: 3 x I fp32, total: I fp32 (outputs).  fp32 sums in a fixed order
 * (deterministic).  Offline, asynchronous.  SPENSE_ERR_ARG for NULL pointers, sizes
 * below 1, ld below the row length, I or D above 2^31-1.
 */
int spense_index_scores(const void* w_gate, const void* w_up, int64_t ld_gu, const void* w_down, int64_t ld_down,
                        int32_t wtype, int64_t I, int64_t D, const float* h_in, const float* h_mid, float eps,
                        float* raw, float* total, hipStream_t stream);

/*
 * TopK of the priorities (Eq. (12)) and the permutation that moves the chosen indices
 * to the back (sec. 3.3.1): flags[i] = 1 for the n_dense indices with the largest total (ties: the
 * lower index first; NaN below every number), 0 otherwise; perm[new] = old lists the
 * unflagged indices in ascending order, then the flagged ones.  perm applies to the rows
 * of Wgate and Wup (spense_gather_rows) and the columns of Wdown (spense_gather_cols),
 * after which the dense region is the trailing one of all three (Eq. (4) keeps the MLP
 * unchanged).  total: I fp32; flags: I bytes; perm: I int32 (outputs).  Asynchronous.
 * SPENSE_ERR_ARG for NULL pointers, I < 1 or above 2^31-1, n_dense outside [0, I].
 */
int spense_dense_permutation(const float* total, int64_t I, int64_t n_dense, uint8_t* flags, int32_t* perm,
                             hipStream_t stream);

/*
 * dst[r, :] = src[perm[r], :] for r < rows (row_bytes bytes per row; leading dimensions
 * in bytes).  perm must hold indices in [0, rows) (others are clamped into that range).
 * src and dst must not overlap.  Asynchronous.
 */
int spense_gather_rows(const void* src, int64_t ld_src_b, void* dst, int64_t ld_dst_b, int64_t rows,
                       int64_t row_bytes, const int32_t* perm, hipStream_t stream);

/*
 * dst[n, c] = src[n, perm[c]] for n < rows, c < cols, elements of elem_bytes (1, 2 or 4)
 * bytes, leading dimensions in elements.  perm must hold indices in [0, cols) (others
 * are clamped).  src and dst must not overlap.  Asynchronous.
 */
int spense_gather_cols(const void* src, int64_t ld_src, void* dst, int64_t ld_dst, int64_t rows, int64_t cols,
                       int32_t elem_bytes, const int32_t* perm, hipStream_t stream);

/*
 * SparseGPT 2:4 pruning with the dense region kept last (sec. 3.1.2, Eqs. (2)-(3); sec.
 * 3.3.1: the dense columns stay a compensation buffer while the 2:4 columns before them
 * are pruned).  Two offline calls, both on fp32 weights before quantisation.
 *
 * spense_obs_factor: from H = X^T X (K x K fp32, leading dimension ldh; only the lower
 * triangle is read, so a lower-only accumulation suffices), the damped Hessian
 * Hd = H + lambda I with lambda = percdamp * mean(diag H), where a zero diagonal entry
 * (a column no calibration input excites) is read as 1 and flagged in dead[j] (K bytes,
 * output).  Writes U (K x K fp32, ldu, upper triangular, zeros below the diagonal) with
 * Hd^{-1} = U^T U: U_jj^2 is the OBS denominator [H^{-1}]_mm of Eq. (3) for column j and
 * U[j, j:] / U_jj its compensation direction, the inverse Hessian of the columns j..K-1.
 * ws: spense_obs_factor_workspace_size(K) bytes, 16-byte aligned.  U must not overlap H.
 * Synchronous (reads back a failure flag).  SPENSE_ERR_NUMERIC if a pivot is not
 * positive; SPENSE_ERR_ARG for NULL pointers, K < 1 or above 2^31-1, ld < K, percdamp
 * negative or not finite, overlapping H and U; SPENSE_ERR_ALIGN for unaligned pointers.
 */
size_t spense_obs_factor_workspace_size(int64_t K);
int spense_obs_factor(const float* H, int64_t ldh, int64_t K, float percdamp, float* U, int64_t ldu, uint8_t* dead,
                      void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * spense_obs_prune_24: prunes W (N x K fp32, ldw; in place) to 2:4 on the columns
 * [0, dense_begin) and compensates, keeping the columns [dense_begin, K) dense.  Columns
 * are processed left to right and frozen once processed.  At the first column of each
 * group of four, each row prunes the two weights with the smallest OBS error w^2 / U_mm^2
 * (the weights as updated so far; equal errors prune the lower index first); each
 * processed column's change is then compensated on the later columns along U's row
 * (Eq. (3)).  dead (K bytes from spense_obs_factor, or NULL): those columns are zeroed
 * first.  keep (N x K bytes, ldk, output): 1 where a weight is kept (every dense column),
 * 0 where pruned.  dense_begin % 4 == 0.  For an output-split matrix pass the 2:4 rows
 * only, with dense_begin = K (the dense rows are not touched).  ws:
 * spense_obs_prune_workspace_size(N) bytes, 16-byte aligned.  Asynchronous.  U as written
 * by spense_obs_factor for this K.  SPENSE_ERR_ARG for NULL pointers, sizes below 0 or
 * above 2^31-1, ld below the row length, dense_begin not a multiple of 4 or outside
 * [0, K]; SPENSE_ERR_WS for a missing or small workspace.
 */
size_t spense_obs_prune_workspace_size(int64_t N);
int spense_obs_prune_24(float* W, int64_t ldw, int64_t N, int64_t K, const float* U, int64_t ldu, const uint8_t* dead,
                        int64_t dense_begin, uint8_t* keep, int64_t ldk, void* ws, size_t ws_bytes,
                        hipStream_t stream);

/* Thread-local description of the last error raised on this thread ("" if none). */
const char* spense_last_error(void);

/* SPENSE_ABI_VERSION of the built library. */
int spense_abi_version(void);

/*
 * Dispatch log (no paper passage: an aid for reading what the planner chose).  With level
 * >= 1 every call that makes a new plan for a single weight (the planner's choice for one
 * dtype, M and weight geometry; later calls with the same key reuse it) writes one line to
 * stderr naming the kernel and its shape; with level >= 2 every grouped and paired call
 * does too.  The level starts at the value of the environment variable SPENSE_LOG when
 * the library is loaded (0 when unset or not a number); it is read there only.  The log
 * never changes a plan or a result.  Returns the previous level; thread-safe.
 */
int spense_set_log(int32_t level);

#ifdef __cplusplus
}
#endif

#endif /* SPENSE_H_ */
