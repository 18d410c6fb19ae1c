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
// C[i][j] = beta C[i][j] + alpha sum_k A(i, k) B(k, j) over an m x n output, with
//   A(i, k) = TA ? A[k][i] : A[i][k],   B(k, j) = TB ? B[j][k] : B[k][j]  (row-major, ld).
// LOWER: only output tiles on or below the diagonal (tile column <= tile row) are formed.
// TRIA: A is lower triangular (A(i, k) = 0 for k > i): k stops at the tile's last row and
// entries above the diagonal are read as 0.
// 64 x 64 output tile per workgroup of 4 waves (2 x 2, 32 x 32 each as 2 x 2
// v_mfma_f32_16x16x4_f32 tiles), k in steps of 16 staged through LDS (two buffers).
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

constexpr int GP = 68;  // LDS row pitch (floats) of the k-major operand tiles

template <bool TA, bool TB, bool LOWER, bool TRIA>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmF32 g) {
  __shared__ float As[2][16][GP];  // As[kk][i]
  __shared__ float Bs[2][16][GP];  // Bs[kk][j]
  const int tr = blockIdx.y, tc = blockIdx.x;
  if (LOWER && tc > tr) return;
  const int64_t i0 = (int64_t)tr * 64, j0 = (int64_t)tc * 64;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wi = (wave >> 1) * 32, wj = (wave & 1) * 32;
  int64_t kend = g.k;
  if (TRIA) kend = kend < i0 + 64 ? kend : i0 + 64;
  const int nsteps = (int)((kend + 15) / 16);

  // global -> register staging of one 16-deep step
  float ra[4], rb[4];
  auto load = [&](int s) __attribute__((always_inline)) {
    const int64_t k0 = (int64_t)s * 16;
    // A: 64 rows (i) x 16 k
    if (!TA) {
      const int64_t i = i0 + (t >> 2), kq = k0 + (t & 3) * 4;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int64_t kk = kq + c;
        bool ok = i < g.m && kk < kend;
        if (TRIA) ok = ok && kk <= i;
        ra[c] = ok ? g.A[i * g.lda + kk] : 0.0f;
      }
    } else {  // A[k][i]: 16 k-rows of 64 i
      const int64_t kk = k0 + (t >> 4), iq = i0 + (t & 15) * 4;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int64_t i = iq + c;
        ra[c] = (i < g.m && kk < kend) ? g.A[kk * g.lda + i] : 0.0f;
      }
    }
    if (!TB) {  // B[k][j]: 16 k-rows of 64 j
      const int64_t kk = k0 + (t >> 4), jq = j0 + (t & 15) * 4;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int64_t j = jq + c;
        rb[c] = (j < g.n && kk < kend) ? g.B[kk * g.ldb + j] : 0.0f;
      }
    } else {  // B[j][k]
      const int64_t j = j0 + (t >> 2), kq = k0 + (t & 3) * 4;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int64_t kk = kq + c;
        rb[c] = (j < g.n && kk < kend) ? g.B[j * g.ldb + kk] : 0.0f;
      }
    }
  };
  auto store = [&](int buf) __attribute__((always_inline)) {
    if (!TA) {
#pragma unroll
      for (int c = 0; c < 4; ++c) As[buf][(t & 3) * 4 + c][t >> 2] = ra[c];
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) As[buf][t >> 4][(t & 15) * 4 + c] = ra[c];
    }
    if (!TB) {
#pragma unroll
      for (int c = 0; c < 4; ++c) Bs[buf][t >> 4][(t & 15) * 4 + c] = rb[c];
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) Bs[buf][(t & 3) * 4 + c][t >> 2] = rb[c];
    }
  };

  f4 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f4{0.0f, 0.0f, 0.0f, 0.0f};

  if (nsteps > 0) {
    load(0);
    store(0);
  }
  __syncthreads();
  for (int s = 0; s < nsteps; ++s) {
    const int buf = s & 1;
    if (s + 1 < nsteps) load(s + 1);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int kk = q * 4 + (lane >> 4);
      float av[2], bv[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) av[a] = As[buf][kk][wi + a * 16 + (lane & 15)];
#pragma unroll
      for (int b = 0; b < 2; ++b) bv[b] = Bs[buf][kk][wj + b * 16 + (lane & 15)];
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a], bv[b], acc[a][b], 0, 0, 0);
    }
    if (s + 1 < nsteps) store(buf ^ 1);
    __syncthreads();
  }
  // epilogue
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
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

template <bool TA, bool TB, bool LOWER, bool TRIA>
hipError_t gemm_f32(const GemmF32& g, hipStream_t st) {
  if (g.m <= 0 || g.n <= 0) return hipSuccess;
  const dim3 grid((unsigned)((g.n + 63) / 64), (unsigned)((g.m + 63) / 64));
  hipLaunchKernelGGL((gemm_f32_kernel<TA, TB, LOWER, TRIA>), grid, dim3(256), 0, st, g);
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

// Diagonal block k0 of the lower Cholesky factorisation, in place: L_kk (nb x nb, nb <=
// 64) is factored in LDS, then replaced by its inverse L_kk^{-1} (lower, zeros above
// the diagonal inside the block).  A non-positive or NaN pivot sets *fail and continues
// with pivot 1 so that the remaining steps stay finite.
__global__ __launch_bounds__(256) void potrf_block_kernel(float* __restrict__ A, int64_t lda, int64_t k0, int nb,
                                                          int* __restrict__ fail) {
  __shared__ float L[64][65];
  __shared__ float X[64][65];
  const int t = threadIdx.x;
  for (int e = t; e < 64 * 64; e += 256) {
    const int i = e >> 6, j = e & 63;
    float v = 0.0f;
    if (i < nb && j <= i) v = A[(k0 + i) * lda + (k0 + j)];
    else if (i == j) v = 1.0f;  // padding of a partial block: identity
    L[i][j] = v;
  }
  __syncthreads();
  for (int j = 0; j < 64; ++j) {
    float d = L[j][j];
    if (!(d > 0.0f)) {
      if (t == 0 && j < nb) atomicOr(fail, 1);
      d = 1.0f;
    }
    const float s = sqrtf(d);
    __syncthreads();  // everyone has read L[j][j]
    if (t == 0) L[j][j] = s;
    if (t > j && t < 64) L[t][j] = L[t][j] / s;
    __syncthreads();
    // trailing update of the lower part: rows and columns j+1..63
    for (int e = t; e < 64 * 64; e += 256) {
      const int i = e >> 6, c = e & 63;
      if (c > j && i >= c) L[i][c] -= L[i][j] * L[c][j];
    }
    __syncthreads();
  }
  // inverse by forward substitution, one column per thread
  if (t < 64) {
    const int c = t;
    for (int i = 0; i < 64; ++i) {
      float v;
      if (i < c) v = 0.0f;
      else if (i == c) v = 1.0f / L[c][c];
      else {
        float s = 0.0f;
        for (int k = c; k < i; ++k) s += L[i][k] * X[k][c];
        v = -s / L[i][i];
      }
      X[i][c] = v;
    }
  }
  __syncthreads();
  for (int e = t; e < 64 * 64; e += 256) {
    const int i = e >> 6, j = e & 63;
    if (i < nb && j < nb) A[(k0 + i) * lda + (k0 + j)] = X[i][j];
  }
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
                                                          float* __restrict__ E) {
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
  float* er = E + n * 64;
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

dim3 lower_tiles(int64_t K) {
  const unsigned t = (unsigned)((K + 63) / 64);
  return dim3(t, t);
}

}  // namespace

size_t obs_factor_workspace(int64_t K) { return (size_t)(K * NB + 64) * sizeof(float); }

int* obs_factor_fail_flag(void* ws, int64_t K) { return reinterpret_cast<int*>(static_cast<float*>(ws) + K * NB + 16); }

// Workspace: T (K x 64 fp32), lambda at float K*64, the failure flag at float K*64 + 16
// (zeroed by the caller before the launch).
hipError_t launch_obs_factor(const float* H, int64_t ldh, int64_t K, float percdamp, float* U, int64_t ldu,
                             uint8_t* dead, void* ws, hipStream_t st) {
  float* T = static_cast<float*>(ws);  // K x 64 staging of the triangular inverse
  float* stat = T + K * NB;            // lambda
  int* fail = obs_factor_fail_flag(ws, K);
  hipLaunchKernelGGL(damp_kernel, dim3(1), dim3(1024), 0, st, H, ldh, K, percdamp, dead, stat);
  hipLaunchKernelGGL(reverse_damp_kernel, lower_tiles(K), dim3(256), 0, st, H, ldh, K, dead, stat, U, ldu);
  const int64_t nblk = (K + NB - 1) / NB;
  hipError_t e = hipGetLastError();
  // Cholesky, right-looking; each diagonal block is left holding its inverse
  for (int64_t b = 0; b < nblk && e == hipSuccess; ++b) {
    const int64_t k0 = b * NB, nb = K - k0 < NB ? K - k0 : NB, r0 = k0 + nb, rows = K - r0;
    hipLaunchKernelGGL(potrf_block_kernel, dim3(1), dim3(256), 0, st, U, ldu, k0, (int)nb, fail);
    if (rows > 0) {
      // panel: L[r0:, k0:k0+nb] = A[r0:, k0:k0+nb] L_kk^{-T} (in place: a workgroup owns its rows)
      GemmF32 g{U + r0 * ldu + k0, ldu, U + k0 * ldu + k0, ldu, U + r0 * ldu + k0, ldu, rows, nb, nb, 1.0f, 0.0f};
      e = gemm_f32<false, true, false, false>(g, st);
      // trailing lower part: A[r0:, r0:] -= L_panel L_panel^T
      GemmF32 s{U + r0 * ldu + k0, ldu, U + r0 * ldu + k0, ldu, U + r0 * ldu + r0, ldu, rows, rows, nb, -1.0f, 1.0f};
      if (e == hipSuccess) e = gemm_f32<false, true, true, false>(s, st);
    }
    if (e == hipSuccess) e = hipGetLastError();
  }
  // triangular inverse, right to left: X[r0:, k0:] = -X[r0:, r0:] (L[r0:, k0:] X_kk)
  for (int64_t b = nblk - 1; b >= 0 && e == hipSuccess; --b) {
    const int64_t k0 = b * NB, nb = K - k0 < NB ? K - k0 : NB, r0 = k0 + nb, rows = K - r0;
    if (rows <= 0) continue;
    GemmF32 g1{U + r0 * ldu + k0, ldu, U + k0 * ldu + k0, ldu, T, NB, rows, nb, nb, 1.0f, 0.0f};
    e = gemm_f32<false, false, false, false>(g1, st);
    GemmF32 g2{U + r0 * ldu + r0, ldu, T, NB, U + r0 * ldu + k0, ldu, rows, nb, rows, -1.0f, 0.0f};
    if (e == hipSuccess) e = gemm_f32<false, false, false, true>(g2, st);
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(reverse_out_kernel, lower_tiles(K), dim3(256), 0, st, U, ldu, K);
  hipLaunchKernelGGL(zero_lower_kernel, lower_tiles(K), dim3(256), 0, st, U, ldu, K);
  return hipGetLastError();
}

size_t obs_prune_workspace(int64_t N) { return (size_t)N * NB * sizeof(float); }

hipError_t launch_obs_prune(float* W, int64_t ldw, int64_t N, int64_t K, const float* U, int64_t ldu,
                            const uint8_t* dead, int64_t dense_begin, uint8_t* keep, int64_t ldk, void* ws,
                            hipStream_t st) {
  float* E = static_cast<float*>(ws);
  const unsigned rows_y = (unsigned)(N < 65535 ? N : 65535);
  if (dead) hipLaunchKernelGGL(zero_dead_kernel, dim3((unsigned)((K + 255) / 256 < 64 ? (K + 255) / 256 : 64), rows_y),
                               dim3(256), 0, st, W, ldw, N, K, dead);
  hipError_t e = hipGetLastError();
  int64_t j0 = 0;
  for (; j0 < dense_begin && e == hipSuccess; j0 += NB) {
    const int cnt = (int)(dense_begin - j0 < NB ? dense_begin - j0 : NB);
    hipLaunchKernelGGL(sweep_block_kernel, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, st, W, ldw, N, K, U, ldu,
                       j0, cnt, keep, ldk, E);
    e = hipGetLastError();
    const int64_t c0 = j0 + NB;
    if (e == hipSuccess && c0 < K) {
      GemmF32 g{E, NB, U + j0 * ldu + c0, ldu, W + c0, ldw, N, K - c0, NB, -1.0f, 1.0f};
      e = gemm_f32<false, false, false, false>(g, st);
    }
  }
  if (e != hipSuccess) return e;
  const int64_t from = j0 < K ? j0 : K;  // the sweep blocks wrote the flags of [0, j0)
  if (from < K)
    hipLaunchKernelGGL(keep_dense_kernel, dim3((unsigned)((K - from + 255) / 256 < 64 ? (K - from + 255) / 256 : 64), rows_y),
                       dim3(256), 0, st, keep, ldk, N, from, K);
  return hipGetLastError();
}

}  // namespace spense
