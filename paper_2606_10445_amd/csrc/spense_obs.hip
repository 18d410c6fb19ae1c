// SparseGPT 2:4 pruning with a protected dense region, on the GPU (paper sec. 3.1.2,
// Eqs. (2)-(3); sec. 3.3.1: the dense columns are placed last so that they absorb the
// compensation of the 2:4 columns processed before them).
//
// Two offline steps:
//  1. The factor.  U upper triangular with Hd^{-1} = U^T U, Hd = H + lambda I (plus
//     H_jj = 1 for columns no input excites).  Row j of U scaled by U_jj is row j of the
//     inverse Hessian of the columns j..K-1, so U_jj^2 is the OBS denominator of Eq. (3)
//     for column j and U[j, j:] / U_jj its compensation direction.  With P the index
//     reversal, P Hd P = L L^T (lower Cholesky) gives Hd = (P L P)(P L P)^T with P L P
//     upper, hence U = (P L P)^{-1} = P L^{-1} P: one Cholesky factorisation and one
//     triangular inverse of the reversed matrix, then a reversal back.  Both are blocked
//     (64-wide diagonal blocks factored and inverted in LDS, everything else as fp32
//     matrix-core products).
//  2. The sweep, 64 columns at a time: a thread per row keeps the row's 64 weights of
//     the block in registers and processes the columns in order (2:4 choice at each
//     group's first column by the OBS error w^2 / U_mm^2, then the compensation inside
//     the block); the block's scaled errors E then update every later column at once,
//     W[:, j0+64:] -= E U[j0:j0+64, j0+64:], on the matrix cores.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "spense.h"
#include "spense_internal.h"

namespace spense {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int NB = 64;  // diagonal block of the factorisations, sweep block, GEMM tile

template <typename F, int... I>
__device__ __forceinline__ void unrolled_impl(F& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>()), ...);
}
// f(integral_constant<int, i>) for i = 0 .. N-1: every index a compile-time constant.
template <int N, typename F>
__device__ __forceinline__ void unrolled(F&& f) {
  unrolled_impl(f, std::make_integer_sequence<int, N>());
}

// ------------------------------------------------------------------ fp32 matrix-core GEMM
// C[i][j] = beta C[i][j] + alpha sum_k A[i][k] B(k, j) over an m x n output, row-major
// operands, B(k, j) = TB ? B[j][k] : B[k][j].
// LOWER: only output tiles on or below the diagonal (tile column <= tile row) are formed.
// TRI (bit mask) marks triangular operands whose other half is read as 0 (and holds
// anything in memory): 1 = A lower (A[i][k] = 0 for k > i), 2 = B(k, j) = 0 for k > j,
// 4 = B(k, j) = 0 for k < j; the k loop is cut to the range they leave.
// BT x BT output tile per workgroup of 4 waves (2 x 2; each BT/2 x BT/2 as TW x TW
// v_mfma_f32_16x16x4_f32 tiles), k staged through LDS 16 deep in two buffers, 16-byte
// loads when the operands allow.
// Operand lanes (measured): A lane l = A[l % 16][l / 16], B lane l = B[l / 16][l % 16],
// D lane l, element r = D[4 (l / 16) + r][l % 16].
struct GemmF32 {
  const float* A;
  int64_t lda;
  const float* B;
  int64_t ldb;
  float* C;
  int64_t ldc;
  int64_t m, n, k;
  float alpha, beta;
};

template <int BT, bool TB, bool LOWER, int TRI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmF32 g, int vec) {
  constexpr int P = BT + 4;        // LDS row pitch (floats)
  constexpr int TW = BT / 32;      // MFMA tiles per wave and dimension
  constexpr int NQ = BT / 64;      // 16-byte pieces per thread and operand per step
  __shared__ float As[2][16][P];   // As[kk][i]
  __shared__ float Bs[2][16][P];   // Bs[kk][j]
  const int tr = blockIdx.y, tc = blockIdx.x;
  if (LOWER && tc > tr) return;
  const int64_t i0 = (int64_t)tr * BT, j0 = (int64_t)tc * BT;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wi = (wave >> 1) * (BT / 2), wj = (wave & 1) * (BT / 2);
  int64_t klo = 0, khi = g.k;
  if (TRI & 1) khi = khi < i0 + BT ? khi : i0 + BT;
  if (TRI & 2) khi = khi < j0 + BT ? khi : j0 + BT;
  if (TRI & 4) klo = j0;
  const int s0 = (int)(klo / 16), s1 = (int)((khi + 15) / 16);

  float ra[NQ][4], rb[NQ][4];
  // four consecutive elements of a row-major operand at (row, k), zero outside
  // [klo, khi), past `rows` and where `keep(k)` says the triangular half is empty
  auto quad = [&](const float* base, int64_t ld, int64_t row, int64_t rows, int64_t kq, float* out, auto keep)
      __attribute__((always_inline)) {
    const bool full = vec && row < rows && kq >= klo && kq + 3 < khi;
    if (full) {
      const float4 v = *reinterpret_cast<const float4*>(base + row * ld + kq);
      out[0] = v.x;
      out[1] = v.y;
      out[2] = v.z;
      out[3] = v.w;
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int64_t kk = kq + c;
        out[c] = (row < rows && kk >= klo && kk < khi) ? base[row * ld + kk] : 0.0f;
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (!keep(kq + c)) out[c] = 0.0f;
  };
  auto load = [&](int s) __attribute__((always_inline)) {
    const int64_t k0 = (int64_t)s * 16;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int slot = t + 256 * q;
      const int64_t i = i0 + (slot >> 2), kq = k0 + (slot & 3) * 4;
      quad(g.A, g.lda, i, g.m, kq, ra[q], [&](int64_t kk) { return !(TRI & 1) || kk <= i; });
      if (TB) {
        const int64_t j = j0 + (slot >> 2);
        quad(g.B, g.ldb, j, g.n, kq, rb[q], [&](int64_t kk) {
          return (!(TRI & 2) || kk <= j) && (!(TRI & 4) || kk >= j);
        });
      } else {
        const int64_t kk = k0 + slot / (BT / 4), jq = j0 + (slot % (BT / 4)) * 4;
        const bool full = vec && kk >= klo && kk < khi && jq + 3 < g.n;
        if (full) {
          const float4 v = *reinterpret_cast<const float4*>(g.B + kk * g.ldb + jq);
          rb[q][0] = v.x;
          rb[q][1] = v.y;
          rb[q][2] = v.z;
          rb[q][3] = v.w;
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c)
            rb[q][c] = (kk >= klo && kk < khi && jq + c < g.n) ? g.B[kk * g.ldb + jq + c] : 0.0f;
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int64_t j = jq + c;
          if (((TRI & 2) && kk > j) || ((TRI & 4) && kk < j)) rb[q][c] = 0.0f;
        }
      }
    }
  };
  auto store = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int slot = t + 256 * q;
#pragma unroll
      for (int c = 0; c < 4; ++c) As[buf][(slot & 3) * 4 + c][slot >> 2] = ra[q][c];
      if (TB) {
#pragma unroll
        for (int c = 0; c < 4; ++c) Bs[buf][(slot & 3) * 4 + c][slot >> 2] = rb[q][c];
      } else {
        *reinterpret_cast<float4*>(&Bs[buf][slot / (BT / 4)][(slot % (BT / 4)) * 4]) =
            make_float4(rb[q][0], rb[q][1], rb[q][2], rb[q][3]);
      }
    }
  };

  f4 acc[TW][TW];
#pragma unroll
  for (int a = 0; a < TW; ++a)
#pragma unroll
    for (int b = 0; b < TW; ++b) acc[a][b] = f4{0.0f, 0.0f, 0.0f, 0.0f};

  if (s0 < s1) {
    load(s0);
    store(0);
  }
  __syncthreads();
  for (int s = s0; s < s1; ++s) {
    const int buf = (s - s0) & 1;
    if (s + 1 < s1) load(s + 1);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int kk = q * 4 + (lane >> 4);
      float av[TW], bv[TW];
#pragma unroll
      for (int a = 0; a < TW; ++a) av[a] = As[buf][kk][wi + a * 16 + (lane & 15)];
#pragma unroll
      for (int b = 0; b < TW; ++b) bv[b] = Bs[buf][kk][wj + b * 16 + (lane & 15)];
#pragma unroll
      for (int a = 0; a < TW; ++a)
#pragma unroll
        for (int b = 0; b < TW; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a], bv[b], acc[a][b], 0, 0, 0);
    }
    if (s + 1 < s1) store(buf ^ 1);
    __syncthreads();
  }
#pragma unroll
  for (int a = 0; a < TW; ++a)
#pragma unroll
    for (int b = 0; b < TW; ++b) {
      const int64_t j = j0 + wj + b * 16 + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t i = i0 + wi + a * 16 + 4 * (lane >> 4) + r;
        if (i < g.m && j < g.n) {
          float* c = g.C + i * g.ldc + j;
          const float v = g.alpha * acc[a][b][r];
          *c = g.beta == 0.0f ? v : g.beta * *c + v;
        }
      }
    }
}

template <bool TB, bool LOWER, int TRI>
hipError_t gemm_f32(const GemmF32& g, hipStream_t st) {
  if (g.m <= 0 || g.n <= 0) return hipSuccess;
  const int vec = (g.lda % 4 == 0) && (g.ldb % 4 == 0) && ((uintptr_t)g.A % 16 == 0) && ((uintptr_t)g.B % 16 == 0);
  if (g.m >= 128 && g.n >= 128) {
    const dim3 grid((unsigned)((g.n + 127) / 128), (unsigned)((g.m + 127) / 128));
    hipLaunchKernelGGL((gemm_f32_kernel<128, TB, LOWER, TRI>), grid, dim3(256), 0, st, g, vec);
  } else {
    const dim3 grid((unsigned)((g.n + 63) / 64), (unsigned)((g.m + 63) / 64));
    hipLaunchKernelGGL((gemm_f32_kernel<64, TB, LOWER, TRI>), grid, dim3(256), 0, st, g, vec);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ the factor
// Damping: lambda = percdamp * mean(diag H) with H_jj = 0 read as 1 (and flagged dead).
// One workgroup; the sum runs in a fixed order.  st[0] = lambda.
__global__ __launch_bounds__(1024) void damp_kernel(const float* __restrict__ H, int64_t ldh, int64_t K,
                                                   float percdamp, uint8_t* __restrict__ dead,
                                                   float* __restrict__ st) {
  __shared__ float red[16];
  float acc = 0.0f;
  for (int64_t j = threadIdx.x; j < K; j += 1024) {
    const float h = H[j * ldh + j];
    dead[j] = h == 0.0f ? 1 : 0;
    acc += h == 0.0f ? 1.0f : h;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    float s = 0.0f;
    for (int w = 0; w < 16; ++w) s += red[w];
    st[0] = percdamp * (s / (float)K);
  }
}

// A[a][b] = Hd[K-1-a][K-1-b] for a >= b, read from the lower triangle of H (the reversed
// pair (K-1-a, K-1-b) has its larger index first when swapped).  64 x 64 tiles.
__global__ __launch_bounds__(256) void reverse_damp_kernel(const float* __restrict__ H, int64_t ldh, int64_t K,
                                                           const uint8_t* __restrict__ dead,
                                                           const float* __restrict__ st, float* __restrict__ A,
                                                           int64_t lda) {
  const int64_t a0 = (int64_t)blockIdx.y * 64, b0 = (int64_t)blockIdx.x * 64;
  if (b0 > a0) return;
  const float lambda = st[0];
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int64_t a = a0 + (e >> 6), b = b0 + (e & 63);
    if (a >= K || b > a) continue;
    const int64_t r = K - 1 - b, c = K - 1 - a;  // r >= c: the lower triangle of H
    float v = H[r * ldh + c];
    if (a == b) v = (dead[r] ? 1.0f : v) + lambda;
    A[a * lda + b] = v;
  }
}

// A diagonal block (n x n, n <= 64) of the lower Cholesky factorisation, in place: L is
// factored and replaced by its inverse X = L^{-1} (lower, zeros above the diagonal
// inside the block).  One wave; lane t holds row t of L and of the running right-hand
// side R of L X = I in registers (every index a compile-time constant).  Step j: the
// pivot L_jj and column j's entries reach every lane through readlane (no barriers);
// lanes below j scale their L_tj and update their row; row j of X is R_j / L_jj and the
// rows below subtract L_tj X_j.  A non-positive or NaN pivot sets *fail and continues
// with pivot 1 so that the rest stays finite.
__device__ __forceinline__ float lane_value(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

__global__ __launch_bounds__(64) void potrf_block_kernel(float* __restrict__ A, int64_t lda, int n,
                                                         int* __restrict__ fail) {
  const int t = threadIdx.x;
  float L[64], R[64];
  unrolled<64>([&](auto cc) __attribute__((always_inline)) {
    constexpr int c = decltype(cc)::value;
    float v = 0.0f;
    if (t < n && c <= t && c < n) v = A[t * lda + c];
    else if (t == c) v = 1.0f;  // padding of a partial block: identity
    L[c] = v;
    R[c] = t == c ? 1.0f : 0.0f;
  });
  bool bad = false;
  unrolled<64>([&](auto jj) __attribute__((always_inline)) {
    constexpr int j = decltype(jj)::value;
    float d = lane_value(L[j], j);
    if (!(d > 0.0f)) {
      bad = bad || j < n;
      d = 1.0f;
    }
    const float s = sqrtf(d), inv = 1.0f / s;
    L[j] = t == j ? s : (t > j ? L[j] * inv : L[j]);
    const float ltj = t > j ? L[j] : 0.0f;
    // trailing columns of this lane's row
    unrolled<63 - j>([&](auto oo) __attribute__((always_inline)) {
      constexpr int c = j + 1 + decltype(oo)::value;
      L[c] -= ltj * lane_value(L[j], c);
    });
    // row j of X, then the rows below
    unrolled<j + 1>([&](auto cc) __attribute__((always_inline)) {
      constexpr int c = decltype(cc)::value;
      if (t == j) R[c] *= inv;
      R[c] -= ltj * lane_value(R[c], j);
    });
  });
  if (bad && t == 0) atomicOr(fail, 1);
  unrolled<64>([&](auto cc) __attribute__((always_inline)) {
    constexpr int c = decltype(cc)::value;
    if (t < n && c < n) A[t * lda + c] = c <= t ? R[c] : 0.0f;
  });
}

// The reversal back: U[K-1-a][K-1-b] = X[a][b] for a > b (lower -> upper), and the
// diagonal reversed (pairs swapped).  Reads only the lower triangle, writes only the
// upper triangle and the diagonal pairs each thread owns.
__global__ __launch_bounds__(256) void reverse_out_kernel(float* __restrict__ A, int64_t lda, int64_t K) {
  const int64_t a0 = (int64_t)blockIdx.y * 64, b0 = (int64_t)blockIdx.x * 64;
  if (b0 > a0) return;
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int64_t a = a0 + (e >> 6), b = b0 + (e & 63);
    if (a >= K || b > a) continue;
    if (a > b) {
      A[(K - 1 - a) * lda + (K - 1 - b)] = A[a * lda + b];
    } else if (a < K - 1 - a) {
      const int64_t z = K - 1 - a;
      const float x = A[a * lda + a], y = A[z * lda + z];
      A[a * lda + a] = y;
      A[z * lda + z] = x;
    }
  }
}

__global__ __launch_bounds__(256) void zero_lower_kernel(float* __restrict__ A, int64_t lda, int64_t K) {
  const int64_t a0 = (int64_t)blockIdx.y * 64, b0 = (int64_t)blockIdx.x * 64;
  if (b0 > a0) return;
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int64_t a = a0 + (e >> 6), b = b0 + (e & 63);
    if (a < K && b < a) A[a * lda + b] = 0.0f;
  }
}

// ------------------------------------------------------------------ the sweep
__global__ __launch_bounds__(256) void zero_dead_kernel(float* __restrict__ W, int64_t ldw, int64_t N, int64_t K,
                                                        const uint8_t* __restrict__ dead) {
  for (int64_t n = blockIdx.y; n < N; n += gridDim.y)
    for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < K; j += (int64_t)gridDim.x * 256)
      if (dead[j]) W[n * ldw + j] = 0.0f;
}

// One 64-column block [j0, j0 + 64) of the sweep; columns j0 .. j0+cnt-1 are 2:4 columns
// (cnt a multiple of 4), the rest of the block (dense columns, or past K) only take
// updates.  A thread per row n: its 64 weights in registers (every index a compile-time
// constant, so nothing spills), U's block (upper; 1 on the diagonal past K) in LDS.
// Writes the block back, the kept flags of the whole block (1 for the columns past the
// 2:4 ones) and E[n][c] = (w_c - q_c) / U_cc (0 where nothing changed).
__global__ __launch_bounds__(256) void sweep_block_kernel(float* __restrict__ W, int64_t ldw, int64_t N, int64_t K,
                                                          const float* __restrict__ U, int64_t ldu, int64_t j0, int cnt,
                                                          uint8_t* __restrict__ keep, int64_t ldk,
                                                          float* __restrict__ E, int64_t lde) {
  __shared__ float Ub[64][64];
  const int width = (int)(K - j0 < 64 ? K - j0 : 64);
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int r = e >> 6, c = e & 63;
    float v = 0.0f;
    if (r < width && c < width && c >= r) v = U[(j0 + r) * ldu + (j0 + c)];
    else if (r == c) v = 1.0f;
    Ub[r][c] = v;
  }
  __syncthreads();
  const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (n >= N) return;
  float* wr = W + n * ldw + j0;
  float w[64];
#pragma unroll
  for (int c = 0; c < 64; ++c) w[c] = c < width ? wr[c] : 0.0f;
  uint32_t kept[2] = {0xffffffffu, 0xffffffffu};
  float* er = E + n * lde;
  unrolled<64>([&](auto cc) __attribute__((always_inline)) {
    constexpr int c = decltype(cc)::value;
    if constexpr (c % 4 == 0) {
      // OBS error of each weight of the group (Eq. (3)); prune the two smallest, ties
      // pruning the lower index; only inside the 2:4 columns
      const bool active = c < cnt;
      float s[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const float d = Ub[c + m][c + m];
        s[m] = (w[c + m] * w[c + m]) / (d * d);
      }
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        int rank = 0;
#pragma unroll
        for (int o = 0; o < 4; ++o) rank += (s[o] < s[m]) || (s[o] == s[m] && o < m);
        if (active && rank < 2) kept[(c + m) >> 5] &= ~(1u << ((c + m) & 31));
      }
    }
    const bool k = (kept[c >> 5] >> (c & 31)) & 1u;
    const float q = k ? w[c] : 0.0f;
    const float ec = (w[c] - q) / Ub[c][c];
#pragma unroll
    for (int c2 = c + 1; c2 < 64; ++c2) w[c2] -= ec * Ub[c][c2];
    w[c] = q;
    er[c] = ec;
  });
#pragma unroll
  for (int c = 0; c < 64; ++c)
    if (c < width) wr[c] = w[c];
  uint8_t* kr = keep + n * ldk + j0;
#pragma unroll
  for (int c = 0; c < 64; ++c)
    if (c < width) kr[c] = (kept[c >> 5] >> (c & 31)) & 1u;
}

// keep = 1 on the columns [from, K) of every row.
__global__ __launch_bounds__(256) void keep_dense_kernel(uint8_t* __restrict__ keep, int64_t ldk, int64_t N,
                                                         int64_t from, int64_t K) {
  for (int64_t n = blockIdx.y; n < N; n += gridDim.y)
    for (int64_t j = from + (int64_t)blockIdx.x * 256 + threadIdx.x; j < K; j += (int64_t)gridDim.x * 256)
      keep[n * ldk + j] = 1;
}

__global__ __launch_bounds__(256) void copy_f32_kernel(const float* __restrict__ src, int64_t lds, float* __restrict__ dst,
                                                       int64_t ldd, int64_t rows, int64_t cols) {
  for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) {
    const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (c < cols) dst[r * ldd + c] = src[r * lds + c];
  }
}

dim3 lower_tiles(int64_t K) {
  const unsigned t = (unsigned)((K + 63) / 64);
  return dim3(t, t);
}

// Recursive factor-and-invert of the lower part of A (n x n, in place): on return A holds
// X = L^{-1} with L L^T = A.  With A = [[A11, .], [A21, A22]] split at n1 (a multiple of
// 64): X11 = (L11)^{-1} recursively, L21 = A21 X11^T, A22 -= L21 L21^T, X22 recursively,
// X21 = -X22 (L21 X11).  Every product is a large, square-ish matrix-core GEMM.
// Workspace: L21 (n2 x n1) plus the second recursion's, behind it.
int64_t chol_inv_ws(int64_t n) {
  if (n <= NB) return 0;
  const int64_t n1 = (n / 2 + NB - 1) / NB * NB, n2 = n - n1;
  const int64_t a = chol_inv_ws(n1), b = n2 * n1 + chol_inv_ws(n2);
  return a > b ? a : b;
}

hipError_t chol_inv(float* A, int64_t lda, int64_t n, float* ws, int* fail, hipStream_t st) {
  if (n <= NB) {
    hipLaunchKernelGGL(potrf_block_kernel, dim3(1), dim3(64), 0, st, A, lda, (int)n, fail);
    return hipGetLastError();
  }
  const int64_t n1 = (n / 2 + NB - 1) / NB * NB, n2 = n - n1;
  float* A11 = A;
  float* A21 = A + n1 * lda;
  float* A22 = A21 + n1;
  float* L21 = ws;
  hipError_t e = chol_inv(A11, lda, n1, ws, fail, st);
  // L21 = A21 X11^T (X11 lower: B(k, j) = X11[j][k] vanishes for k > j)
  if (e == hipSuccess) e = gemm_f32<true, false, 2>(GemmF32{A21, lda, A11, lda, L21, n1, n2, n1, n1, 1.0f, 0.0f}, st);
  // A22 -= L21 L21^T, lower tiles
  if (e == hipSuccess) e = gemm_f32<true, true, 0>(GemmF32{L21, n1, L21, n1, A22, lda, n2, n2, n1, -1.0f, 1.0f}, st);
  if (e == hipSuccess) e = chol_inv(A22, lda, n2, ws + n2 * n1, fail, st);
  // T = L21 X11 into A21's place (X11 lower: B(k, j) = X11[k][j] vanishes for k < j)
  if (e == hipSuccess) e = gemm_f32<false, false, 4>(GemmF32{L21, n1, A11, lda, A21, lda, n2, n1, n1, 1.0f, 0.0f}, st);
  // X21 = -X22 T into the workspace (X22 lower), then back into A21's place
  if (e == hipSuccess) e = gemm_f32<false, false, 1>(GemmF32{A22, lda, A21, lda, L21, n1, n2, n1, n2, -1.0f, 0.0f}, st);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(copy_f32_kernel, dim3((unsigned)((n1 + 255) / 256), (unsigned)(n2 < 65535 ? n2 : 65535)),
                       dim3(256), 0, st, L21, n1, A21, lda, n2, n1);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

// Workspace: lambda at float 0, the failure flag at float 16, the recursion's from
// float 64 on.
size_t obs_factor_workspace(int64_t K) { return (size_t)(64 + chol_inv_ws(K)) * sizeof(float); }

int* obs_factor_fail_flag(void* ws, int64_t) { return reinterpret_cast<int*>(static_cast<float*>(ws) + 16); }

hipError_t launch_obs_factor(const float* H, int64_t ldh, int64_t K, float percdamp, float* U, int64_t ldu,
                             uint8_t* dead, void* ws, hipStream_t st) {
  float* stat = static_cast<float*>(ws);  // lambda
  int* fail = obs_factor_fail_flag(ws, K);
  hipLaunchKernelGGL(damp_kernel, dim3(1), dim3(1024), 0, st, H, ldh, K, percdamp, dead, stat);
  hipLaunchKernelGGL(reverse_damp_kernel, lower_tiles(K), dim3(256), 0, st, H, ldh, K, dead, stat, U, ldu);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) e = chol_inv(U, ldu, K, stat + 64, fail, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(reverse_out_kernel, lower_tiles(K), dim3(256), 0, st, U, ldu, K);
  hipLaunchKernelGGL(zero_lower_kernel, lower_tiles(K), dim3(256), 0, st, U, ldu, K);
  return hipGetLastError();
}

// The sweep in two levels: 64-column blocks inside 256-column outer blocks.  Inside an
// outer block each 64-block's errors update only the rest of the outer block (k = 64);
// at its end the outer block's errors update every later column at once (k = 256), so
// the trailing columns are read and written once per 256 columns instead of per 64.
constexpr int OB = 256;

size_t obs_prune_workspace(int64_t N) { return (size_t)N * OB * sizeof(float); }

hipError_t launch_obs_prune(float* W, int64_t ldw, int64_t N, int64_t K, const float* U, int64_t ldu,
                            const uint8_t* dead, int64_t dense_begin, uint8_t* keep, int64_t ldk, void* ws,
                            hipStream_t st) {
  float* E = static_cast<float*>(ws);  // N x OB: the outer block's scaled errors
  const unsigned rows_y = (unsigned)(N < 65535 ? N : 65535);
  if (dead) hipLaunchKernelGGL(zero_dead_kernel, dim3((unsigned)((K + 255) / 256 < 64 ? (K + 255) / 256 : 64), rows_y),
                               dim3(256), 0, st, W, ldw, N, K, dead);
  hipError_t e = hipGetLastError();
  int64_t pe = 0;  // end of the processed 64-blocks
  for (int64_t o0 = 0; o0 < dense_begin && e == hipSuccess; o0 += OB) {
    const int64_t last = o0 + OB < dense_begin ? o0 + OB : dense_begin;  // 2:4 columns of this outer block end here
    pe = o0 + (last - o0 + NB - 1) / NB * NB;                             // processed blocks end here
    for (int64_t j0 = o0; j0 < last && e == hipSuccess; j0 += NB) {
      const int cnt = (int)(last - j0 < NB ? last - j0 : NB);
      hipLaunchKernelGGL(sweep_block_kernel, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, st, W, ldw, N, K, U,
                         ldu, j0, cnt, keep, ldk, E + (j0 - o0), (int64_t)OB);
      e = hipGetLastError();
      const int64_t c0 = j0 + NB, c1 = pe < K ? pe : K;  // the rest of the processed blocks
      if (e == hipSuccess && c0 < c1)
        e = gemm_f32<false, false, 0>(GemmF32{E + (j0 - o0), OB, U + j0 * ldu + c0, ldu, W + c0, ldw, N, c1 - c0, NB,
                                              -1.0f, 1.0f}, st);
    }
    if (e == hipSuccess && pe < K)
      e = gemm_f32<false, false, 0>(GemmF32{E, OB, U + o0 * ldu + pe, ldu, W + pe, ldw, N, K - pe, pe - o0, -1.0f,
                                            1.0f}, st);
  }
  if (e != hipSuccess) return e;
  const int64_t from = pe < K ? pe : K;  // the sweep blocks wrote the flags of [0, pe)
  if (from < K)
    hipLaunchKernelGGL(keep_dense_kernel, dim3((unsigned)((K - from + 255) / 256 < 64 ? (K - from + 255) / 256 : 64), rows_y),
                       dim3(256), 0, st, keep, ldk, N, from, K);
  return hipGetLastError();
}

}  // namespace spense
