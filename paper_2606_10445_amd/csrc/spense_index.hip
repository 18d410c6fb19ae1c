// SpenseGPT+ dense-index selection on the GPU (paper sec. 3.3.1, Eqs. (8)-(12)): each
// intermediate index i of a GLU MLP gets a Wanda-style priority from its row of Wgate and
// Wup and its column of Wdown,
//   s_gate[i] = mean_j |Wgate[i, j]| sqrt(h_in[j]),   s_up likewise,
//   s_down[i] = mean_n |Wdown[n, i]| sqrt(h_mid[i]),
// with h the diagonals of the input Hessians X^T X; each vector is divided by its mean
// (plus eps) and the three are summed.  The pN indices with the largest priority (ties:
// lower index first) are kept dense and permuted to the back, the others keep their
// order in front (Eq. (4): the MLP is unchanged when the rows of Wgate, Wup and the
// columns of Wdown move together).  Offline tooling next to spense_compress; every sum runs in a fixed
// order, so results are deterministic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "spense.h"
#include "spense_internal.h"

namespace spense {
namespace {

template <int TYPE>
__device__ __forceinline__ float wval(const uint8_t* row, int64_t j) {
  if constexpr (TYPE == SPENSE_BF16)
    return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(row)[j] << 16);
  else
    return reinterpret_cast<const float*>(row)[j];
}

template <int THREADS>
__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  const int w = threadIdx.x >> 6;
  __syncthreads();  // red may still be read by a previous call
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = 0.0f;
#pragma unroll
  for (int i = 0; i < THREADS / 64; ++i) r += red[i];
  return r;
}

// Row scores of Wgate and Wup, general form: one workgroup per row (blockIdx.y = 0 gate,
// 1 up), element loads.  Used when a row does not split into 16-byte pieces.
template <int TYPE>
__global__ __launch_bounds__(256) void row_scores_kernel(const uint8_t* __restrict__ wg, const uint8_t* __restrict__ wu,
                                                         int64_t ld_b, int64_t D, const float* __restrict__ h_in,
                                                         float* __restrict__ out, int64_t I) {
  __shared__ float red[4];
  const int64_t i = blockIdx.x;
  const uint8_t* row = (blockIdx.y == 0 ? wg : wu) + i * ld_b;
  float acc = 0.0f;
  for (int64_t j = threadIdx.x; j < D; j += 256) acc += fabsf(wval<TYPE>(row, j)) * sqrtf(h_in[j]);
  acc = block_sum<256>(acc, red);
  if (threadIdx.x == 0) out[blockIdx.y * I + i] = acc / (float)D;
}

// Row scores, streaming form: a wave per row (rows 0..I-1 of Wgate, then of Wup, shared
// out among the waves of the grid).  Lane l owns the 16-byte pieces l, l + 64, ... of
// every row (T of them, T <= TMAX) and keeps sqrt(h_in) of their elements in registers,
// so each wave computes those square roots once; all T loads of a row are issued before
// the first is used.  Each lane sums its pieces in order, then the wave adds its lanes
// with a fixed butterfly.
template <int TYPE, int TMAX>
__global__ __launch_bounds__(256) void row_scores_wave_kernel(const uint8_t* __restrict__ wg,
                                                              const uint8_t* __restrict__ wu, int64_t ld_b, int64_t D,
                                                              int T, const float* __restrict__ h_in,
                                                              float* __restrict__ out, int64_t I) {
  constexpr int EP = TYPE == SPENSE_BF16 ? 8 : 4;  // elements per 16-byte piece
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6;
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  float sh[TMAX][EP];
#pragma unroll
  for (int t = 0; t < TMAX; ++t) {
    const int64_t j = ((int64_t)t * 64 + lane) * EP;
#pragma unroll
    for (int e = 0; e < EP; ++e) sh[t][e] = (t < T && j < D) ? sqrtf(h_in[j + e]) : 0.0f;
  }
  for (int64_t r = wave; r < 2 * I; r += nwaves) {
    const uint8_t* row = (r < I ? wg + r * ld_b : wu + (r - I) * ld_b);
    int4 v[TMAX];
#pragma unroll
    for (int t = 0; t < TMAX; ++t) {
      const int64_t j = ((int64_t)t * 64 + lane) * EP;
      v[t] = (t < T && j < D) ? *reinterpret_cast<const int4*>(row + j * (16 / EP)) : make_int4(0, 0, 0, 0);
    }
    float acc = 0.0f;
#pragma unroll
    for (int t = 0; t < TMAX; ++t) {
      const uint32_t w[4] = {(uint32_t)v[t].x, (uint32_t)v[t].y, (uint32_t)v[t].z, (uint32_t)v[t].w};
#pragma unroll
      for (int e = 0; e < EP; ++e) {
        float x;
        if constexpr (TYPE == SPENSE_BF16)
          x = __uint_as_float(e & 1 ? (w[e >> 1] & 0xffff0000u) : (w[e >> 1] << 16));
        else
          x = __uint_as_float(w[e]);
        acc += fabsf(x) * sh[t][e];
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (lane == 0) out[r] = acc / (float)D;
  }
}

// Column scores of Wdown (D x I), general form: a workgroup covers 64 columns; its 4
// waves each sum a quarter of the rows of every column (rows n = wave, wave + 4, ...),
// then the four partial sums are added in wave order.
template <int TYPE>
__global__ __launch_bounds__(256) void col_scores_kernel(const uint8_t* __restrict__ wd, int64_t ld_b, int64_t D,
                                                         int64_t I, const float* __restrict__ h_mid,
                                                         float* __restrict__ out) {
  __shared__ float part[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t i = (int64_t)blockIdx.x * 64 + lane;
  float acc = 0.0f;
  if (i < I)
    for (int64_t n = wave; n < D; n += 4) acc += fabsf(wval<TYPE>(wd + n * ld_b, i));
  part[wave][lane] = acc;
  __syncthreads();
  if (wave == 0 && i < I) {
    const float s = ((part[0][lane] + part[1][lane]) + part[2][lane]) + part[3][lane];
    out[2 * I + i] = s / (float)D * sqrtf(h_mid[i]);
  }
}

// Column scores, streaming form: a workgroup of 16 waves covers 256 columns, lane l the
// four columns 4l..4l+3 (one 8- or 16-byte load per row); wave w sums rows w, w + 16, ...
// (UNR rows' loads in flight at a time), then the 16 partial sums of each column are
// added in wave order.  Needs I % 4 == 0 and 4-element-aligned rows.
template <int TYPE>
__global__ __launch_bounds__(1024) void col_scores_wide_kernel(const uint8_t* __restrict__ wd, int64_t ld_b,
                                                               int64_t D, int64_t I, const float* __restrict__ h_mid,
                                                               float* __restrict__ out) {
  constexpr int UNR = 8;
  typedef typename std::conditional<TYPE == SPENSE_BF16, uint2, uint4>::type V;
  __shared__ float part[16][256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t c0 = (int64_t)blockIdx.x * 256 + lane * 4;
  const bool live = c0 < I;
  const uint8_t* base = wd + c0 * (TYPE == SPENSE_BF16 ? 2 : 4);
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  auto add = [&](const V& v) __attribute__((always_inline)) {
    if constexpr (TYPE == SPENSE_BF16) {
      acc[0] += fabsf(__uint_as_float(v.x << 16));
      acc[1] += fabsf(__uint_as_float(v.x & 0xffff0000u));
      acc[2] += fabsf(__uint_as_float(v.y << 16));
      acc[3] += fabsf(__uint_as_float(v.y & 0xffff0000u));
    } else {
      acc[0] += fabsf(__uint_as_float(v.x));
      acc[1] += fabsf(__uint_as_float(v.y));
      acc[2] += fabsf(__uint_as_float(v.z));
      acc[3] += fabsf(__uint_as_float(v.w));
    }
  };
  if (live) {
    int64_t n = wave;
    for (; n + 16 * (UNR - 1) < D; n += 16 * UNR) {
      V v[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) v[u] = *reinterpret_cast<const V*>(base + (n + 16 * u) * ld_b);
#pragma unroll
      for (int u = 0; u < UNR; ++u) add(v[u]);
    }
    for (; n < D; n += 16) add(*reinterpret_cast<const V*>(base + n * ld_b));
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) part[wave][lane * 4 + k] = acc[k];
  __syncthreads();
  if (threadIdx.x < 256) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < I) {
      float s = 0.0f;
#pragma unroll
      for (int w = 0; w < 16; ++w) s += part[w][threadIdx.x];
      out[2 * I + i] = s / (float)D * sqrtf(h_mid[i]);
    }
  }
}

// total[i] = sum over the three vectors of raw[v][i] / (mean(raw[v]) + eps); one
// workgroup, means summed in a fixed order.
__global__ __launch_bounds__(1024) void normalize_kernel(const float* __restrict__ raw, int64_t I, float eps,
                                                         float* __restrict__ total) {
  __shared__ float red[16];
  float inv[3];
  for (int v = 0; v < 3; ++v) {
    float acc = 0.0f;
    for (int64_t i = threadIdx.x; i < I; i += 1024) acc += raw[v * I + i];
    const float mean = block_sum<1024>(acc, red) / (float)I;
    inv[v] = 1.0f / (mean + eps);
  }
  for (int64_t i = threadIdx.x; i < I; i += 1024)
    total[i] = (raw[i] * inv[0] + raw[I + i] * inv[1]) + raw[2 * I + i] * inv[2];
}

// Order-preserving 32-bit key of a priority: larger priority, larger key; -0 equals +0;
// every NaN gets key 0, below every number (-inf included).
__device__ __forceinline__ uint32_t order_key(float x) {
  if (x != x) return 0u;
  const uint32_t u = x == 0.0f ? 0u : __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix count of `pred` over the 1024 threads in thread order, and the total
// (ballot per wave, wave counts through LDS).
__device__ __forceinline__ uint32_t block_prefix(bool pred, uint32_t* wcnt, uint32_t* total) {
  const uint64_t m = __ballot(pred);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
  __syncthreads();  // wcnt may still be read by a previous call
  if (lane == 0) wcnt[wave] = (uint32_t)__popcll(m);
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < 16; ++w) {
    const uint32_t c = wcnt[w];
    before += w < wave ? c : 0u;
    all += c;
  }
  *total = all;
  return before + below;
}

// TopK and permutation in one workgroup of 1024 threads.
// 1. Radix select, 8 bits a pass from the top: the key T of the n_dense-th largest
//    priority and the number k of indices with key T that still belong to the TopK.
// 2. One pass over the indices in 1024-index blocks: flag = key > T, or key == T among
//    the first k such indices (ties: the lower index first); the flagged indices are
//    written to the back of perm and the others to the front, each in ascending order.
__global__ __launch_bounds__(1024) void select_kernel(const float* __restrict__ t, int64_t I, int64_t n_dense,
                                                     uint8_t* __restrict__ flag, int32_t* __restrict__ perm) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t wcnt[16];
  __shared__ uint32_t sel[2];  // chosen digit, remaining count
  uint32_t prefix = 0, mask = 0;
  uint32_t k = (uint32_t)n_dense;
  if (n_dense > 0) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (threadIdx.x < 256) hist[threadIdx.x] = 0;
      __syncthreads();
      for (int64_t i = threadIdx.x; i < I; i += 1024) {
        const uint32_t key = order_key(t[i]);
        if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (threadIdx.x < 64) {
        // lane l holds digits 4l..4l+3; above(d) = candidates with a larger digit
        const int l = threadIdx.x;
        const uint32_t h0 = hist[4 * l], h1 = hist[4 * l + 1], h2 = hist[4 * l + 2], h3 = hist[4 * l + 3];
        const uint32_t mine = h0 + h1 + h2 + h3;
        uint32_t suf = mine;  // inclusive sum over lanes >= l
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t x = __shfl_down(suf, o, 64);
          suf += l + o < 64 ? x : 0u;
        }
        uint32_t above = suf - mine;
        const uint32_t hs[4] = {h3, h2, h1, h0};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (above < k && k <= above + hs[q]) {
            sel[0] = (uint32_t)(4 * l + 3 - q);
            sel[1] = k - above;
          }
          above += hs[q];
        }
      }
      __syncthreads();
      prefix |= sel[0] << shift;
      mask |= 255u << shift;
      k = sel[1];
      __syncthreads();  // sel and hist are rewritten by the next pass
    }
  }
  const bool any = n_dense > 0;
  uint32_t eq_before = 0;     // indices with key T in earlier blocks
  int64_t dense_before = 0;   // flagged indices in earlier blocks
  for (int64_t b = 0; b < I; b += 1024) {
    const int64_t i = b + threadIdx.x;
    const bool in = i < I;
    const uint32_t key = in ? order_key(t[i]) : 0u;
    const bool eq = any && in && key == prefix;
    uint32_t eq_all;
    const uint32_t eq_rank = eq_before + block_prefix(eq, wcnt, &eq_all);
    const bool f = any && in && (key > prefix || (eq && eq_rank < k));
    uint32_t f_all;
    const int64_t d = dense_before + block_prefix(f, wcnt, &f_all);  // flagged indices before i
    if (in) {
      flag[i] = f ? 1 : 0;
      const int64_t pos = f ? (I - n_dense) + d : i - d;
      if (pos >= 0 && pos < I) perm[pos] = (int32_t)i;
    }
    eq_before += eq_all;
    dense_before += f_all;
  }
}

// dst[r] = src[perm[r]] row by row (bytes per row `cols_b`; source rows = destination
// rows, indices clamped into range), a wave per row.  vec: 16-byte pieces, up to 8 of a
// row's loads in flight before their stores; else bytes.
__global__ __launch_bounds__(256) void gather_rows_kernel(const uint8_t* __restrict__ src, int64_t ld_src_b,
                                                          uint8_t* __restrict__ dst, int64_t ld_dst_b, int64_t rows,
                                                          int64_t cols_b, const int32_t* __restrict__ perm, int vec) {
  const int lane = threadIdx.x & 63;
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  for (int64_t r = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6; r < rows; r += nwaves) {
    const int64_t pr = min(max((int64_t)perm[r], (int64_t)0), rows - 1);
    const uint8_t* s = src + pr * ld_src_b;
    uint8_t* d = dst + r * ld_dst_b;
    if (vec) {
      for (int64_t c0 = 0; c0 < cols_b; c0 += 8 * 64 * 16) {
        int4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int64_t c = c0 + ((int64_t)u * 64 + lane) * 16;
          v[u] = c < cols_b ? *reinterpret_cast<const int4*>(s + c) : make_int4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int64_t c = c0 + ((int64_t)u * 64 + lane) * 16;
          if (c < cols_b) *reinterpret_cast<int4*>(d + c) = v[u];
        }
      }
    } else {
      for (int64_t c = lane; c < cols_b; c += 64) d[c] = s[c];
    }
  }
}

// dst[n][c] = src[n][perm[c]] (elements of ES bytes); blockIdx.y walks the rows.  Each
// thread writes V consecutive outputs, one 16-byte store when vec (V = 16 / ES), else
// element stores.
template <int ES>
__global__ __launch_bounds__(256) void gather_cols_kernel(const uint8_t* __restrict__ src, int64_t ld_src_b,
                                                          uint8_t* __restrict__ dst, int64_t ld_dst_b, int64_t rows,
                                                          int64_t cols, const int32_t* __restrict__ perm, int vec) {
  typedef typename std::conditional<ES == 1, uint8_t, typename std::conditional<ES == 2, uint16_t, uint32_t>::type>::type T;
  constexpr int V = 16 / ES;
  const int64_t c0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * V;
  if (c0 >= cols) return;
  int32_t p[V];
#pragma unroll
  for (int e = 0; e < V; ++e) p[e] = c0 + e < cols ? min(max(perm[c0 + e], 0), (int32_t)(cols - 1)) : 0;
  for (int64_t n = blockIdx.y; n < rows; n += gridDim.y) {
    const T* s = reinterpret_cast<const T*>(src + n * ld_src_b);
    T* d = reinterpret_cast<T*>(dst + n * ld_dst_b);
    if (vec) {
      union {
        T e[V];
        int4 v;
      } o;
#pragma unroll
      for (int e = 0; e < V; ++e) o.e[e] = s[p[e]];
      *reinterpret_cast<int4*>(d + c0) = o.v;
    } else {
#pragma unroll
      for (int e = 0; e < V; ++e)
        if (c0 + e < cols) d[c0 + e] = s[p[e]];
    }
  }
}

}  // namespace

namespace {
int grid_for(int64_t waves) {  // workgroups of 4 waves, at most 8 per CU's worth
  const int64_t g = (waves + 3) / 4;
  return (int)(g < 2048 ? (g < 1 ? 1 : g) : 2048);
}
}  // namespace

hipError_t launch_index_scores(int type, const void* wg, const void* wu, int64_t ld_gu_b, int64_t I, int64_t D,
                               const void* wd, int64_t ld_d_b, const float* h_in, const float* h_mid, float eps,
                               float* raw, float* total, hipStream_t st) {
  const uint8_t* g = static_cast<const uint8_t*>(wg);
  const uint8_t* u = static_cast<const uint8_t*>(wu);
  const uint8_t* d = static_cast<const uint8_t*>(wd);
  const int64_t es = type == SPENSE_BF16 ? 2 : 4, ep = 16 / es;
  const int64_t T = (D + 64 * ep - 1) / (64 * ep);
  const bool row_vec = D % ep == 0 && ld_gu_b % 16 == 0 && (uintptr_t)g % 16 == 0 && (uintptr_t)u % 16 == 0 && T <= 16;
  const bool col_vec = I % 4 == 0 && ld_d_b % (4 * es) == 0 && (uintptr_t)d % (4 * es) == 0;
  const dim3 rg((unsigned)I, 2), cg((unsigned)((I + 63) / 64)), wg_grid((unsigned)grid_for(2 * I));
  const dim3 cwg((unsigned)((I + 255) / 256));
  if (type == SPENSE_BF16) {
    if (row_vec)
      hipLaunchKernelGGL((row_scores_wave_kernel<SPENSE_BF16, 16>), wg_grid, dim3(256), 0, st, g, u, ld_gu_b, D, (int)T,
                         h_in, raw, I);
    else
      hipLaunchKernelGGL(row_scores_kernel<SPENSE_BF16>, rg, dim3(256), 0, st, g, u, ld_gu_b, D, h_in, raw, I);
    if (col_vec)
      hipLaunchKernelGGL(col_scores_wide_kernel<SPENSE_BF16>, cwg, dim3(1024), 0, st, d, ld_d_b, D, I, h_mid, raw);
    else
      hipLaunchKernelGGL(col_scores_kernel<SPENSE_BF16>, cg, dim3(256), 0, st, d, ld_d_b, D, I, h_mid, raw);
  } else {
    if (row_vec)
      hipLaunchKernelGGL((row_scores_wave_kernel<SPENSE_F32, 16>), wg_grid, dim3(256), 0, st, g, u, ld_gu_b, D, (int)T,
                         h_in, raw, I);
    else
      hipLaunchKernelGGL(row_scores_kernel<SPENSE_F32>, rg, dim3(256), 0, st, g, u, ld_gu_b, D, h_in, raw, I);
    if (col_vec)
      hipLaunchKernelGGL(col_scores_wide_kernel<SPENSE_F32>, cwg, dim3(1024), 0, st, d, ld_d_b, D, I, h_mid, raw);
    else
      hipLaunchKernelGGL(col_scores_kernel<SPENSE_F32>, cg, dim3(256), 0, st, d, ld_d_b, D, I, h_mid, raw);
  }
  hipLaunchKernelGGL(normalize_kernel, dim3(1), dim3(1024), 0, st, raw, I, eps, total);
  return hipGetLastError();
}

hipError_t launch_dense_permutation(const float* total, int64_t I, int64_t n_dense, uint8_t* flag, int32_t* perm,
                                    hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3(1), dim3(1024), 0, st, total, I, n_dense, flag, perm);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void* src, int64_t ld_src_b, void* dst, int64_t ld_dst_b, int64_t rows,
                              int64_t cols_b, const int32_t* perm, hipStream_t st) {
  const int vec = ((uintptr_t)src % 16 == 0) && ((uintptr_t)dst % 16 == 0) && ld_src_b % 16 == 0 &&
                  ld_dst_b % 16 == 0 && cols_b % 16 == 0;
  hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)grid_for(rows)), dim3(256), 0, st,
                     static_cast<const uint8_t*>(src), ld_src_b, static_cast<uint8_t*>(dst), ld_dst_b, rows, cols_b,
                     perm, vec);
  return hipGetLastError();
}

hipError_t launch_gather_cols(int es, const void* src, int64_t ld_src_b, void* dst, int64_t ld_dst_b, int64_t rows,
                              int64_t cols, const int32_t* perm, hipStream_t st) {
  const uint8_t* s = static_cast<const uint8_t*>(src);
  uint8_t* d = static_cast<uint8_t*>(dst);
  const int64_t V = 16 / es;
  const int vec = (uintptr_t)d % 16 == 0 && ld_dst_b % 16 == 0 && cols % V == 0;
  const dim3 grid((unsigned)((cols + 256 * V - 1) / (256 * V)), (unsigned)(rows < 65535 ? rows : 65535));
  if (es == 1)
    hipLaunchKernelGGL(gather_cols_kernel<1>, grid, dim3(256), 0, st, s, ld_src_b, d, ld_dst_b, rows, cols, perm, vec);
  else if (es == 2)
    hipLaunchKernelGGL(gather_cols_kernel<2>, grid, dim3(256), 0, st, s, ld_src_b, d, ld_dst_b, rows, cols, perm, vec);
  else
    hipLaunchKernelGGL(gather_cols_kernel<4>, grid, dim3(256), 0, st, s, ld_src_b, d, ld_dst_b, rows, cols, perm, vec);
  return hipGetLastError();
}

}  // namespace spense
