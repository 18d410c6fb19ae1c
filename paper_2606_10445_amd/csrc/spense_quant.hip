// Activation quantisation on either side of the Spense GEMMs of a GLU MLP (paper sec.
// 3.3.1, Eq. (4): MLP(X) = ((X Wup^T) .* sigma(X Wgate^T)) Wdown^T, sigma = SiLU here):
//   - per-token fp8 quantisation of activations;
//   - the GLU step h = u * silu(g) fused with the per-token fp8 quantisation of h.
// Both produce what spense_gemm consumes: e4m3fn codes and one fp32 scale per token,
//   s[m] = max_k |a[m,k]| / 448 (1.0 for an all-zero row),  q[m,k] = e4m3fn(a[m,k] / s[m]),
// in fp32 with a correctly rounded division; the encode rounds to nearest, ties to an
// even mantissa, and saturates to +-448.
//
// One workgroup per token row.  Rows of up to 32768 fp32 / 65536 bf16 elements with
// 16-byte aligned rows are held in registers (1024 threads, one read); other rows take
// two passes (the maximum, then the codes, re-reading the row from L2), the GLU value
// computed by the same instructions in both, so the maximum is always the maximum of
// exactly the values that are encoded (it is exact in any order).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "spense.h"
#include "spense_internal.h"

namespace spense {
namespace {

constexpr int kQuantThreads = 256;

// fp32 -> e4m3fn codes with the gfx950 conversion instruction (OCP e4m3fn, round to
// nearest even): two values per instruction, into the low (HI = false) or high half of
// `old`.  Inputs here are at most 448 * (1 + 2^-23) in magnitude (a / s with s = max/448),
// which round to 448, so the saturation of the definition is never needed; NaN stays
// NaN.  The GPU tests check the codes bit for bit against the oracle's encoder written
// from the format definition (ties, the subnormal range, NaN included).
template <bool HI>
__device__ __forceinline__ uint32_t cvt2_e4m3fn(float a, float b, uint32_t old) {
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)old, HI);
}

__device__ __forceinline__ uint32_t encode_e4m3fn(float f) { return cvt2_e4m3fn<false>(f, 0.0f, 0u) & 0xFFu; }

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Element i of a row of type T (float or bf16 bits).
template <int TYPE>
__device__ __forceinline__ float load_elem(const void* row, int64_t i) {
  if constexpr (TYPE == SPENSE_BF16)
    return bf16_to_f32(reinterpret_cast<const uint16_t*>(row)[i]);
  else
    return reinterpret_cast<const float*>(row)[i];
}

// h = u * silu(g) = u * (g * sigmoid(g)), fp32, exp and the reciprocal of 1 + exp(-g)
// from the hardware approximations (about 1 ulp each); the same helper as the fused
// gate / up epilogue.
__device__ __forceinline__ float glu(float g, float u) { return glu_silu(g, u); }

template <int THREADS>
__device__ __forceinline__ float block_max(float v, float* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < THREADS / 64; ++i) r = fmaxf(r, red[i]);
  return r;
}

typedef int v4i __attribute__((ext_vector_type(4)));

// GLU = false: a = src0; GLU = true: a = glu(src0, src1) (src0 = g, src1 = u).
// Two-pass version for any row length and alignment: pass 1 finds the maximum, pass 2
// re-reads the row and writes the codes.
template <int TYPE, bool GLU>
__global__ __launch_bounds__(kQuantThreads) void quantize_rows_kernel(const uint8_t* __restrict__ src0, int64_t ld0_b,
                                                                      const uint8_t* __restrict__ src1, int64_t ld1_b,
                                                                      int64_t K, uint8_t* __restrict__ q, int64_t ldq,
                                                                      float* __restrict__ scales) {
  __shared__ float red[kQuantThreads / 64];
  const int64_t m = blockIdx.x;
  const uint8_t* r0 = src0 + m * ld0_b;
  const uint8_t* r1 = GLU ? src1 + m * ld1_b : nullptr;
  auto value = [&](int64_t k) {
    const float x = load_elem<TYPE>(r0, k);
    if constexpr (GLU)
      return glu(x, load_elem<TYPE>(r1, k));
    else
      return x;
  };
  float amax = 0.0f;
  for (int64_t k = threadIdx.x; k < K; k += kQuantThreads) amax = fmaxf(amax, fabsf(value(k)));
  amax = block_max<kQuantThreads>(amax, red);
  const float s = amax > 0.0f ? amax / 448.0f : 1.0f;
  if (threadIdx.x == 0) scales[m] = s;
  uint8_t* qr = q + m * ldq;
  for (int64_t k = threadIdx.x; k < K; k += kQuantThreads) qr[k] = (uint8_t)encode_e4m3fn(value(k) / s);
}

// Rows held in registers (rows of up to NJ * E * kRowThreads elements, 16-byte aligned):
// thread t owns the 16-byte pieces t + kRowThreads * j (E = 4 fp32 or 8 bf16 elements
// each), loads them all at once, keeps the activation values, reduces the maximum over
// the workgroup and encodes from registers, one 4- or 8-byte store of codes per piece.
constexpr int kRowThreads = 1024;

template <int TYPE, bool GLU, int NJ>
__global__ __launch_bounds__(kRowThreads) void quantize_rows_reg_kernel(const uint8_t* __restrict__ src0, int64_t ld0_b,
                                                                        const uint8_t* __restrict__ src1, int64_t ld1_b,
                                                                        int64_t K, uint8_t* __restrict__ q, int64_t ldq,
                                                                        float* __restrict__ scales) {
  constexpr int E = TYPE == SPENSE_BF16 ? 8 : 4;
  __shared__ float red[kRowThreads / 64];
  const int64_t m = blockIdx.x;
  const uint8_t* r0 = src0 + m * ld0_b;
  const uint8_t* r1 = GLU ? src1 + m * ld1_b : nullptr;
  // all loads first (pieces past the row read its first piece instead, and are masked
  // below), so that they are in flight together
  constexpr int ES = TYPE == SPENSE_BF16 ? 2 : 4;
  v4i ra[NJ], rb[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int64_t k0 = (int64_t)E * (threadIdx.x + kRowThreads * j);
    const int64_t ks = k0 + E <= K ? k0 : 0;
    ra[j] = *reinterpret_cast<const v4i*>(r0 + ks * ES);
    if constexpr (GLU) rb[j] = *reinterpret_cast<const v4i*>(r1 + ks * ES);
  }
  float v[NJ][E];
  float amax = 0.0f;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int64_t k0 = (int64_t)E * (threadIdx.x + kRowThreads * j);
    if (k0 + E <= K) {  // a whole piece
      const v4i a = ra[j];
      v4i b = {0, 0, 0, 0};
      if constexpr (GLU) b = rb[j];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        float x, y = 0.0f;
        if constexpr (TYPE == SPENSE_BF16) {
          x = bf16_to_f32((uint16_t)((uint32_t)a[e / 2] >> (16 * (e & 1))));
          if constexpr (GLU) y = bf16_to_f32((uint16_t)((uint32_t)b[e / 2] >> (16 * (e & 1))));
        } else {
          x = __int_as_float(a[e]);
          if constexpr (GLU) y = __int_as_float(b[e]);
        }
        v[j][e] = GLU ? glu(x, y) : x;
      }
    } else {  // the row's ragged end (at most one piece per row), element by element
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int64_t k = k0 + e;
        float x = 0.0f;
        if (k < K) {
          x = load_elem<TYPE>(r0, k);
          if constexpr (GLU) x = glu(x, load_elem<TYPE>(r1, k));
        }
        v[j][e] = x;
      }
    }
#pragma unroll
    for (int e = 0; e < E; ++e) amax = fmaxf(amax, fabsf(v[j][e]));
  }
  amax = block_max<kRowThreads>(amax, red);
  const float s = amax > 0.0f ? amax / 448.0f : 1.0f;
  if (threadIdx.x == 0) scales[m] = s;
  uint8_t* qr = q + m * ldq;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int64_t k0 = (int64_t)E * (threadIdx.x + kRowThreads * j);
    float t[E];
#pragma unroll
    for (int e = 0; e < E; ++e) t[e] = v[j][e] / s;
    uint32_t w[E / 4];
#pragma unroll
    for (int h = 0; h < E / 4; ++h)
      w[h] = cvt2_e4m3fn<true>(t[4 * h + 2], t[4 * h + 3], cvt2_e4m3fn<false>(t[4 * h], t[4 * h + 1], 0u));
    if (k0 + E <= K) {
      if constexpr (E == 8) {
        typedef uint32_t u2 __attribute__((ext_vector_type(2)));
        *reinterpret_cast<u2*>(qr + k0) = (u2){w[0], w[1]};
      } else {
        *reinterpret_cast<uint32_t*>(qr + k0) = w[0];
      }
    } else {
#pragma unroll
      for (int e = 0; e < E; ++e)
        if (k0 + e < K) qr[k0 + e] = (uint8_t)(w[e / 4] >> (8 * (e % 4)));
    }
  }
}

// fp32 rows whose maxima come as partial maxima (pmax[m * P + p], each the maximum of |h|
// over some of the row's columns, together all of them; written by the producing GEMM):
// a workgroup takes 2048 columns of one row, so that a matrix of few, long rows still
// fills the GPU.  It reduces the row's P partials (exact in any order), forms the scale
// as the row kernels do, and encodes its columns (16-byte loads, 4-byte code stores).
constexpr int kPieceThreads = 256, kPieceCols = 8 * kPieceThreads;

__global__ __launch_bounds__(kPieceThreads) void quantize_rowmax_kernel(const float* __restrict__ H, int64_t ldh,
                                                                        int64_t N, const float* __restrict__ pmax, int P,
                                                                        uint8_t* __restrict__ q, int64_t ldq,
                                                                        float* __restrict__ scales, int vec_q,
                                                                        int pieces) {
  __shared__ float red[kPieceThreads / 64];
  const int64_t m = blockIdx.x / pieces;
  const int piece = blockIdx.x % pieces;
  const float* hr = H + m * ldh;
  // the two 4-column pieces of this thread: loads first
  int64_t k[2];
  float v[2][4];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    k[j] = (int64_t)piece * kPieceCols + 4 * (threadIdx.x + kPieceThreads * j);
    if (k[j] + 4 <= N) {
      const v4i x = *reinterpret_cast<const v4i*>(hr + k[j]);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[j][e] = __int_as_float(x[e]);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[j][e] = k[j] + e < N ? hr[k[j] + e] : 0.0f;
    }
  }
  float amax = 0.0f;
  const float* pr = pmax + m * P;
  for (int p = threadIdx.x; p < P; p += kPieceThreads) amax = fmaxf(amax, pr[p]);
  amax = block_max<kPieceThreads>(amax, red);
  const float s = amax > 0.0f ? amax / 448.0f : 1.0f;
  if (piece == 0 && threadIdx.x == 0) scales[m] = s;
  uint8_t* qr = q + m * ldq;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (k[j] >= N) continue;
    const uint32_t w =
        cvt2_e4m3fn<true>(v[j][2] / s, v[j][3] / s, cvt2_e4m3fn<false>(v[j][0] / s, v[j][1] / s, 0u));
    if (vec_q && k[j] + 4 <= N) {
      *reinterpret_cast<uint32_t*>(qr + k[j]) = w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (k[j] + e < N) qr[k[j] + e] = (uint8_t)(w >> (8 * e));
    }
  }
}

template <int TYPE, bool GLU>
hipError_t launch_quant_type(const uint8_t* a, int64_t ld0_b, const uint8_t* b, int64_t ld1_b, int64_t M, int64_t K,
                             uint8_t* q, int64_t ldq, float* scales, hipStream_t st) {
  constexpr int E = TYPE == SPENSE_BF16 ? 8 : 4;
  // the register path needs 16-byte aligned source rows and 4- / 8-byte aligned code rows
  const bool aligned = ((uintptr_t)a % 16 == 0) && (ld0_b % 16 == 0) && (!GLU || ((uintptr_t)b % 16 == 0 && ld1_b % 16 == 0)) &&
                       ((uintptr_t)q % E == 0) && (ldq % E == 0);
  const int64_t pieces = (K + E - 1) / E;
  const int64_t nj = (pieces + kRowThreads - 1) / kRowThreads;
  const dim3 grid((unsigned)M);
  if (aligned && nj <= 8) {
    if (nj <= 1)
      hipLaunchKernelGGL((quantize_rows_reg_kernel<TYPE, GLU, 1>), grid, dim3(kRowThreads), 0, st, a, ld0_b, b, ld1_b, K,
                         q, ldq, scales);
    else if (nj <= 2)
      hipLaunchKernelGGL((quantize_rows_reg_kernel<TYPE, GLU, 2>), grid, dim3(kRowThreads), 0, st, a, ld0_b, b, ld1_b, K,
                         q, ldq, scales);
    else if (nj <= 4)
      hipLaunchKernelGGL((quantize_rows_reg_kernel<TYPE, GLU, 4>), grid, dim3(kRowThreads), 0, st, a, ld0_b, b, ld1_b, K,
                         q, ldq, scales);
    else
      hipLaunchKernelGGL((quantize_rows_reg_kernel<TYPE, GLU, 8>), grid, dim3(kRowThreads), 0, st, a, ld0_b, b, ld1_b, K,
                         q, ldq, scales);
  } else {
    hipLaunchKernelGGL((quantize_rows_kernel<TYPE, GLU>), grid, dim3(kQuantThreads), 0, st, a, ld0_b, b, ld1_b, K, q,
                       ldq, scales);
  }
  return hipGetLastError();
}

template <bool GLU>
hipError_t launch_quant_t(int type, const void* s0, int64_t ld0_b, const void* s1, int64_t ld1_b, int64_t M, int64_t K,
                          uint8_t* q, int64_t ldq, float* scales, hipStream_t st) {
  const uint8_t* a = static_cast<const uint8_t*>(s0);
  const uint8_t* b = static_cast<const uint8_t*>(s1);
  if (type == SPENSE_BF16) return launch_quant_type<SPENSE_BF16, GLU>(a, ld0_b, b, ld1_b, M, K, q, ldq, scales, st);
  return launch_quant_type<SPENSE_F32, GLU>(a, ld0_b, b, ld1_b, M, K, q, ldq, scales, st);
}

}  // namespace

hipError_t launch_quantize_rowmax(const float* H, int64_t ldh, int64_t M, int64_t N, const float* pmax, int P,
                                  uint8_t* q, int64_t ldq, float* scales, hipStream_t st) {
  const int vec_q = (uintptr_t)q % 4 == 0 && ldq % 4 == 0;
  const int64_t pieces = (N + kPieceCols - 1) / kPieceCols;
  if (M <= 0 || pieces <= 0 || M * pieces > INT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(quantize_rowmax_kernel, dim3((unsigned)(M * pieces)), dim3(kPieceThreads), 0, st, H, ldh, N, pmax,
                     P, q, ldq, scales, vec_q, (int)pieces);
  return hipGetLastError();
}

hipError_t launch_quantize(int type, const void* src, int64_t ld_b, int64_t M, int64_t K, uint8_t* q, int64_t ldq,
                           float* scales, hipStream_t st) {
  return launch_quant_t<false>(type, src, ld_b, nullptr, 0, M, K, q, ldq, scales, st);
}

hipError_t launch_glu_quantize(int type, const void* g, int64_t ldg_b, const void* u, int64_t ldu_b, int64_t M,
                               int64_t I, uint8_t* q, int64_t ldq, float* scales, hipStream_t st) {
  return launch_quant_t<true>(type, g, ldg_b, u, ldu_b, M, I, q, ldq, scales, st);
}

}  // namespace spense
