// Activation quantisation on either side of the Spense GEMMs of a GLU MLP (paper sec.
// 3.3.1, Eq. (4): MLP(X) = ((X Wup^T) .* sigma(X Wgate^T)) Wdown^T, sigma = SiLU here):
//   - per-token fp8 quantisation of activations;
//   - the GLU step h = u * silu(g) fused with the per-token fp8 quantisation of h.
// Both produce what spense_gemm consumes: e4m3fn codes and one fp32 scale per token,
//   s[m] = max_k |a[m,k]| / 448 (1.0 for an all-zero row),  q[m,k] = e4m3fn(a[m,k] / s[m]),
// in fp32 with a correctly rounded division; the encode rounds to nearest, ties to an
// even mantissa, and saturates to +-448.
//
// One workgroup per token row: pass 1 finds the row's absolute maximum (exact in any
// order), pass 2 re-reads the row (from L2) and writes the codes.  The GLU value is
// computed by the same instructions in both passes, so the maximum is the maximum of
// exactly the values that are encoded.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "spense.h"
#include "spense_internal.h"

namespace spense {
namespace {

constexpr int kQuantThreads = 256;

// fp32 -> e4m3fn from the format definition (1 sign, 4 exponent bits with bias 7, 3
// mantissa bits; exponent field 0 holds multiples of 2^-9; 0x7f / 0xff are NaN).
__device__ __forceinline__ uint32_t encode_e4m3fn(float f) {
  const uint32_t bits = __float_as_uint(f);
  const uint32_t sign = (bits >> 24) & 0x80u;
  const float a = fabsf(f);
  if (!(a == a)) return sign | 0x7Fu;       // NaN
  if (a >= 464.0f) return sign | 0x7Eu;     // rounds past 448 (464 is the midpoint to 480)
  if (a < 0.015625f) {                      // below 2^-6: multiples of 2^-9
    const float q = __builtin_rintf(a * 512.0f);  // exact scaling, ties to even
    return sign | (uint32_t)q;              // 8 -> 0x08, the smallest normal
  }
  int e = (int)((bits >> 23) & 0xFFu) - 127;  // a >= 2^-6 is a normal fp32 value
  const float frac = __uint_as_float((bits & 0x007FFFFFu) | 0x3F800000u);  // a / 2^e in [1, 2)
  float m = __builtin_rintf((frac - 1.0f) * 8.0f);
  if (m >= 8.0f) {
    m = 0.0f;
    e += 1;
  }
  uint32_t code = (uint32_t)((e + 7) << 3) | (uint32_t)m;
  if (code > 0x7Eu) code = 0x7Eu;
  return sign | code;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Element i of a row of type T (float or bf16 bits).
template <int TYPE>
__device__ __forceinline__ float load_elem(const void* row, int64_t i) {
  if constexpr (TYPE == SPENSE_BF16)
    return bf16_to_f32(reinterpret_cast<const uint16_t*>(row)[i]);
  else
    return reinterpret_cast<const float*>(row)[i];
}

// h = u * silu(g) = u * (g / (1 + exp(-g))), fp32.
__device__ __forceinline__ float glu(float g, float u) { return u * (g / (1.0f + __expf(-g))); }

__device__ __forceinline__ float block_max(float v, float* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < kQuantThreads / 64; ++i) r = fmaxf(r, red[i]);
  return r;
}

// GLU = false: a = src0; GLU = true: a = glu(src0, src1) (src0 = g, src1 = u).
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
  amax = block_max(amax, red);
  const float s = amax > 0.0f ? amax / 448.0f : 1.0f;
  if (threadIdx.x == 0) scales[m] = s;
  uint8_t* qr = q + m * ldq;
  for (int64_t k = threadIdx.x; k < K; k += kQuantThreads) qr[k] = (uint8_t)encode_e4m3fn(value(k) / s);
}

template <bool GLU>
hipError_t launch_quant_t(int type, const void* s0, int64_t ld0_b, const void* s1, int64_t ld1_b, int64_t M, int64_t K,
                          uint8_t* q, int64_t ldq, float* scales, hipStream_t st) {
  const uint8_t* a = static_cast<const uint8_t*>(s0);
  const uint8_t* b = static_cast<const uint8_t*>(s1);
  if (type == SPENSE_BF16)
    hipLaunchKernelGGL((quantize_rows_kernel<SPENSE_BF16, GLU>), dim3((unsigned)M), dim3(kQuantThreads), 0, st, a,
                       ld0_b, b, ld1_b, K, q, ldq, scales);
  else
    hipLaunchKernelGGL((quantize_rows_kernel<SPENSE_F32, GLU>), dim3((unsigned)M), dim3(kQuantThreads), 0, st, a,
                       ld0_b, b, ld1_b, K, q, ldq, scales);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize(int type, const void* src, int64_t ld_b, int64_t M, int64_t K, uint8_t* q, int64_t ldq,
                           float* scales, hipStream_t st) {
  return launch_quant_t<false>(type, src, ld_b, nullptr, 0, M, K, q, ldq, scales, st);
}

hipError_t launch_glu_quantize(int type, const void* g, int64_t ldg_b, const void* u, int64_t ldu_b, int64_t M,
                               int64_t I, uint8_t* q, int64_t ldq, float* scales, hipStream_t st) {
  return launch_quant_t<true>(type, g, ldg_b, u, ldu_b, M, I, q, ldq, scales, st);
}

}  // namespace spense
