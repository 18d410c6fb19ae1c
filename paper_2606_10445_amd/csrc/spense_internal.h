// Internal declarations shared by the libspense translation units (host + device).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spense {

enum : int32_t { kFP8 = 1, kBF16 = 2 };
enum : int32_t { kSplitOutput = 0, kSplitInput = 1 };

constexpr int kMaxWaves = 16;
constexpr int kMaxMats = 4;                  // weights of one grouped launch
constexpr int kMaxRegions = 2 * kMaxMats;    // 2:4 rows and dense rows of each

// One contiguous part of the weight: a range of output rows and the logical K range
// [0, K) whose columns below kbound are stored 2:4 and the rest dense.  Output-split has
// up to two regions (2:4 rows with kbound = K, dense rows with kbound = 0); input-split
// has one region with kbound = the first dense column.  A workgroup owns 16*RT rows of
// one region; its waves split K at cut[0..waves] (cost-balanced), each wave running the
// 2:4 loop over its part below kbound and the dense loop over the rest into one fp32
// accumulator; the waves' partial sums are added in LDS in wave order.  The row-split
// kernel instead gives each of the first `wused` waves of a workgroup 16 rows over a
// slice of K (fewer rows per workgroup where rows carry more bytes, to balance the CUs;
// several slices where the weight has too few rows to fill the CUs, their fp32 partial
// sums added afterwards in slice order by splitk_reduce).
struct Region {
  int32_t row0, rows;          // output rows [row0, row0 + rows)
  int32_t kbound;              // first dense column (K for all-2:4, 0 for all-dense)
  int32_t kend;                // K
  int32_t dense_row_off;       // dense storage row = n - dense_row_off
  int32_t dense_col_off;       // dense storage column = k - dense_col_off
  int32_t nrb;                 // row groups (workgroups per activation block)
  int32_t wg0;                 // first workgroup of this region
  int32_t wused;               // row-split kernel: waves of a workgroup that own rows here
  int32_t ksplit;              // row-split kernel: K slices (1 = none); >1 writes fp32 partials
  int32_t mat;                 // row-split kernel: the weight (GemmArgs::mat) these rows belong to
  int32_t cut[kMaxWaves + 1];  // K-split kernel: K boundaries of the waves' parts;
                               // row-split kernel: chunk boundaries of the K slices
};

// One weight of a launch as the row-split kernel reads it: its buffers, output and
// per-row scales.  A plain launch has one (the same buffers as GemmArgs); a grouped launch
// (several weights sharing X and K) has up to kMaxMats.
struct MatDesc {
  const uint8_t* values;
  const uint32_t* meta;
  const uint8_t* dense;
  uint32_t v_bytes, m_bytes, d_bytes;
  void* Y;
  int64_t ldy;  // elements
  const float* sw;
  int32_t vec_store;
};

struct GemmArgs {
  const uint8_t* X;
  int64_t ldx_b;  // bytes
  const uint8_t* values;
  int64_t v_ld_b;  // bytes per 2:4 row
  const uint32_t* meta;
  int64_t m_ld_b;  // bytes per 2:4 row of metadata
  const uint8_t* dense;
  int64_t d_ld_b;  // bytes per dense row
  const float* sw;
  const float* sx;
  void* Y;
  int64_t ldy;  // elements
  uint32_t x_bytes, v_bytes, m_bytes, d_bytes;  // buffer extents for range-checked loads
  int32_t M, N;
  int32_t out_f32;
  int32_t vec_store;  // 4 consecutive outputs may be stored as one vector
  int32_t nreg;
  int32_t groups;
  int32_t tiled;  // weight buffers in the tiled execution layout (fp8, row-split kernel)
  float* part;    // fp32 partial sums of K-sliced regions: part[(slice * M + m) * N + n]
  int32_t tblocks;  // large-M kernel: 256-token blocks (workgroups of a row block are adjacent)
  int32_t btok;     // 256 x 256 kernel: tokens of a full tile's block, 192 or 256 (0 = 256)
  // 256 x 256 kernel: workgroups from hg0 on (the last ones) compute 256 x 128 tiles of
  // the last region's row blocks hrb0 .., hper of them per row block (hg0 = groups: none)
  int32_t hg0, hrb0, hper;
  int32_t xgt, xrc;  // large-M kernel, XCD-aware order (0 = off): token blocks per XCD, row classes
  int32_t xg1;       // the XCD-aware order covers workgroups [0, xg1); the rest keep their place
  int32_t nmat;
  // row-split kernel, several token blocks: 0 = grid (row groups, token blocks); 1 = one
  // dimension, the token blocks of a row group adjacent; 2 = one dimension, the token
  // blocks of a row group on one XCD (row groups a multiple of 8)
  int32_t rorder, mblk;
  float* hmax;  // paired gate / up launch: per-workgroup maxima of |h| per token, hmax[m * groups + g] (or NULL)
  MatDesc mat[kMaxMats];
  Region reg[kMaxRegions];
};

// The GLU step h = u * silu(g) = u * g / (1 + e^-g) as every kernel computes it (the
// hardware exponential and reciprocal), so that the fused and the separate MLP paths give
// the same bits.
__device__ __forceinline__ float glu_silu(float g, float u) {
  return u * (g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)));
}

struct LaunchShape {
  int ct;       // 16-column tiles of M per workgroup (1, 2, 4)
  int rt;       // 16-row tiles per workgroup (1, 2, 4)
  int waves;    // waves per workgroup (4, 8, 16): they split K
  int mblocks;  // grid.y
  int u8;       // eight instruction steps per batch of loads (single activation tile only)
  int rows;     // row-split workgroups with activations staged in LDS
  int big;      // large-M kernels (fp8): 1 = 128-row x 256-token workgroup tiles, 2 = 256 x 256
  int glu;      // row-split kernel, gate and up paired: waves 0-3 gate tiles, 4-7 the same up tiles
  int xres;     // row-split kernel, one token tile: >0 = the activations of all xres chunks stay in LDS
};

hipError_t launch_gemm(int dtype, const LaunchShape& ls, const GemmArgs& a, hipStream_t s);

// Record an error message for spense_last_error (printf format) and return code.
int api_fail(int code, const char* fmt, ...);

// Y for the rows of K-sliced regions: the sum of their fp32 partials in slice order, then
// the epilogue (after launch_gemm, on the same stream).
hipError_t launch_splitk_reduce(const GemmArgs& a, hipStream_t s);

hipError_t launch_compress(int dtype, const uint8_t* W, int64_t ldw_b, const uint8_t* mask, int64_t ldm,
                           int64_t s_rows, int64_t s_cols, uint8_t* values, int64_t v_ld_b, uint32_t* meta,
                           int64_t m_ld, const uint8_t* dsrc, int64_t d_rows, int64_t d_cols_b, uint8_t* dense,
                           int64_t d_ld_b, unsigned long long* bad, hipStream_t s);

hipError_t launch_decompress(int dtype, const uint8_t* values, int64_t v_ld_b, const uint32_t* meta, int64_t m_ld,
                             int64_t s_rows, int64_t s_cols, uint8_t* W, int64_t ldw_b, const uint8_t* dense,
                             int64_t d_ld_b, int64_t d_rows, int64_t d_cols_b, uint8_t* ddst, hipStream_t s);

hipError_t launch_zero_u64(unsigned long long* p, hipStream_t s);

// Per-token fp8 quantisation (type = SPENSE_BF16 / SPENSE_F32; leading dimensions in bytes
// for the sources) and the GLU step fused with it.
hipError_t launch_quantize(int type, const void* src, int64_t ld_b, int64_t M, int64_t K, uint8_t* q, int64_t ldq,
                           float* scales, hipStream_t st);
hipError_t launch_glu_quantize(int type, const void* g, int64_t ldg_b, const void* u, int64_t ldu_b, int64_t M,
                               int64_t I, uint8_t* q, int64_t ldq, float* scales, hipStream_t st);
// Per-token fp8 quantisation of an fp32 M x N matrix H (ldh elements, rows 16-byte
// aligned) whose row maxima come as partial maxima of |h|: pmax[m * P + p], p < P.
hipError_t launch_quantize_rowmax(const float* H, int64_t ldh, int64_t M, int64_t N, const float* pmax, int P,
                                  uint8_t* q, int64_t ldq, float* scales, hipStream_t st);

// Dense-index selection (SpenseGPT+): priorities, TopK permutation, row / column gathers.
hipError_t launch_index_scores(int type, const void* wg, const void* wu, int64_t ld_gu_b, int64_t I, int64_t D,
                               const void* wd, int64_t ld_d_b, const float* h_in, const float* h_mid, float eps,
                               float* raw, float* total, hipStream_t st);
hipError_t launch_dense_permutation(const float* total, int64_t I, int64_t n_dense, uint8_t* flag, int32_t* perm,
                                    hipStream_t st);
hipError_t launch_gather_rows(const void* src, int64_t ld_src_b, void* dst, int64_t ld_dst_b, int64_t rows,
                              int64_t cols_b, const int32_t* perm, hipStream_t st);
hipError_t launch_gather_cols(int es, const void* src, int64_t ld_src_b, void* dst, int64_t ld_dst_b, int64_t rows,
                              int64_t cols, const int32_t* perm, hipStream_t st);

// SparseGPT 2:4 with a protected dense region: the inverse-Hessian factor and the sweep.
size_t obs_factor_workspace(int64_t K);
int* obs_factor_fail_flag(void* ws, int64_t K);
hipError_t launch_obs_factor(const float* H, int64_t ldh, int64_t K, float percdamp, float* U, int64_t ldu,
                             uint8_t* dead, void* ws, hipStream_t st);
size_t obs_prune_workspace(int64_t N);
hipError_t launch_obs_prune(float* W, int64_t ldw, int64_t N, int64_t K, const float* U, int64_t ldu,
                            const uint8_t* dead, int64_t dense_begin, uint8_t* keep, int64_t ldk, void* ws,
                            hipStream_t st);

// Tiled execution layout: kind 0 values, 1 metadata, 2 dense (fp8).  src is one row-major
// region (rows x row_bytes, pitch src_ld_b); dst receives tiles x chunks blocks.
hipError_t launch_tile(int kind, const uint8_t* src, int64_t src_ld_b, int64_t rows, int64_t row_bytes, int64_t tiles,
                       int64_t chunks, uint8_t* dst, hipStream_t s);

}  // namespace spense
