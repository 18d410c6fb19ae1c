/*
 * Plain CPU oracle for the Spense hybrid 2:4-sparse / dense linear layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link or call this
 * file; it exists so that tests, the smoke check and the benchmark's CPU baseline can
 * compare the GPU library against a slow, obviously correct implementation.  It shares
 * no code, header, table or constant with the GPU library.
 *
 * What it computes (paper: "SpenseGPT", sec. 3.1.1 and sec. 3.2):
 *   - the 2:4 constraint of Eq. (1): in every row of W (N x K, PyTorch's X W^T
 *     convention) each aligned group of 4 consecutive input-dimension entries holds at
 *     most 2 non-zeros;
 *   - 2:4 compressed storage (sec. 3.1.1): only the kept values plus a few position bits
 *     per group;
 *   - the Spense format (sec. 3.2): W is split into a 2:4 region and a dense region.
 *     Output-split cuts the output dimension N (rows [0,Ns) sparse, [Ns,N) dense);
 *     input-split cuts the input dimension K (cols [0,Ks) sparse, [Ks,K) dense).  The
 *     dense region is the last one (sec. 3.3.2, Table "front_back": "Back").
 *   - Both variants are an exact re-association of one GEMM: output-split concatenates
 *     disjoint output columns, input-split sums two partial products into one output.
 *     Hence the result has a plain definition, which is what the GEMM below computes:
 *         Y[m,n] = bf16_rne( (sum_k xhat[m,k] * what[n,k]) * sw[n] * sx[m] )
 *     with what = decompress(packed) and xhat = decode(X).
 *
 * Readings where the paper is silent (fp8 flavour, scales, metadata bit order, padding
 * of groups with fewer than two kept values, accumulation precision) are fixed here and
 * listed in the design notes of the repository.  Accumulation is fp32 in ascending k
 * starting from +0; a second entry point accumulates in fp64.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared spense_oracle.c -o liboracle.so
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Harness only (no arithmetic): the number of OpenMP threads of the parallel loops below,
 * for the benchmark's single-thread figure; returns the previous maximum. */
int or_set_threads(int n) {
  const int prev = omp_get_max_threads();
  if (n > 0) omp_set_num_threads(n);
  return prev;
}

#define OR_FP8 1  /* OCP fp8 e4m3fn: 1 sign, 4 exponent (bias 7), 3 mantissa bits */
#define OR_BF16 2 /* bfloat16: the top 16 bits of an IEEE-754 binary32 */
#define OR_AXIS_OUTPUT 0
#define OR_AXIS_INPUT 1

/* ---------------------------------------------------------------- number formats */

/* e4m3fn decode from the format definition: exponent field 0 is subnormal
 * (m * 2^-9), exponent/mantissa all-ones is NaN, there is no infinity. */
double or_decode_e4m3fn(uint8_t c) {
  int s = (c >> 7) & 1, e = (c >> 3) & 15, m = c & 7;
  double v;
  if (e == 15 && m == 7) return NAN;
  if (e == 0)
    v = ldexp((double)m, -9);
  else
    v = ldexp(1.0 + m / 8.0, e - 7);
  return s ? -v : v;
}

float or_decode_bf16(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* binary32 -> bfloat16, round to nearest, ties to even, on the 16 dropped bits.
 * NaN stays NaN (quiet bit forced).  Overflow rounds to +-inf as IEEE requires. */
uint16_t or_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x0040u);
  uint32_t lower = u & 0xffffu;
  uint32_t upper = u >> 16;
  if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u))) upper += 1u;
  return (uint16_t)upper;
}

void or_decode_e4m3fn_array(const uint8_t* c, int64_t n, double* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = or_decode_e4m3fn(c[i]);
}
void or_decode_bf16_array(const uint16_t* c, int64_t n, float* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = or_decode_bf16(c[i]);
}
void or_bf16_rne_array(const float* f, int64_t n, uint16_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = or_bf16_rne(f[i]);
}

/* ---------------------------------------------------------------- format geometry */

/* Sizes of the three packed buffers, in elements (values, dense) and 32-bit words
 * (meta).  One meta word holds 8 groups (32 logical K) of one row. */
static int region(int64_t N, int64_t K, int axis, int64_t dense_begin, int64_t* s_rows, int64_t* s_cols,
                  int64_t* d_rows, int64_t* d_cols) {
  if (axis == OR_AXIS_OUTPUT) {
    if (dense_begin < 0 || dense_begin > N) return -1;
    *s_rows = dense_begin;
    *s_cols = K;
    *d_rows = N - dense_begin;
    *d_cols = K;
  } else if (axis == OR_AXIS_INPUT) {
    if (dense_begin < 0 || dense_begin > K) return -1;
    *s_rows = N;
    *s_cols = dense_begin;
    *d_rows = N;
    *d_cols = K - dense_begin;
  } else {
    return -1;
  }
  return 0;
}

int or_layout(int64_t N, int64_t K, int axis, int64_t dense_begin, int64_t* out6) {
  int64_t sr, sc, dr, dc;
  if (region(N, K, axis, dense_begin, &sr, &sc, &dr, &dc)) return -1;
  out6[0] = sr;             /* sparse rows */
  out6[1] = sc / 2;         /* values per sparse row */
  out6[2] = (sc + 31) / 32; /* meta words per sparse row */
  out6[3] = dr;             /* dense rows */
  out6[4] = dc;             /* dense elements per row */
  out6[5] = sc;             /* logical K of the sparse region */
  return 0;
}

/* ---------------------------------------------------------------- compress */

/* Canonical compression of the sparse region.  For each row and each group of 4:
 *   kept = mask != 0 (or, with no mask, a non-zero bit pattern of W);
 *   more than 2 kept -> the group is counted as bad and stored as if nothing was kept;
 *   fewer than 2 kept -> padded with the smallest non-kept positions, value +0;
 *   the two positions i0 < i1 are stored in ascending order, their values in the same
 *   order, and the 4-bit code (i0 | i1 << 2) goes to bits [4*(g%8), 4*(g%8)+4) of
 *   meta word g/8 of the row.
 * The dense region is copied unchanged.  Returns the number of bad groups, or -1 on a
 * bad argument (K % 4 != 0 in the sparse region). */
int64_t or_compress(const void* W, const uint8_t* mask, int64_t N, int64_t K, int es, int axis,
                    int64_t dense_begin, void* values, uint32_t* meta, void* dense) {
  int64_t L[6];
  if (or_layout(N, K, axis, dense_begin, L)) return -1;
  const int64_t s_rows = L[0], v_ld = L[1], m_ld = L[2], d_rows = L[3], d_ld = L[4], s_cols = L[5];
  if (s_cols % 4) return -1;
  const uint8_t* w = (const uint8_t*)W;
  uint8_t* v = (uint8_t*)values;
  int64_t bad = 0;
  for (int64_t r = 0; r < s_rows; ++r) {
    for (int64_t wd = 0; wd < m_ld; ++wd) meta[r * m_ld + wd] = 0;
    for (int64_t g = 0; g < s_cols / 4; ++g) {
      int kept[4], nk = 0;
      for (int i = 0; i < 4; ++i) {
        int64_t col = 4 * g + i;
        const uint8_t* src = w + (r * K + col) * es;
        int keep;
        if (mask)
          keep = mask[r * K + col] != 0;
        else {
          keep = 0;
          for (int b = 0; b < es; ++b) keep |= src[b] != 0;
        }
        if (keep) kept[nk++] = i;
      }
      int pos[2], fromw[2];
      if (nk > 2) {
        ++bad;
        nk = 0;
      }
      /* take the kept positions, then pad with the smallest non-kept ones */
      int np = 0;
      for (int i = 0; i < 4 && np < 2; ++i) {
        int is_kept = 0;
        for (int t = 0; t < nk; ++t) is_kept |= kept[t] == i;
        if (is_kept) {
          pos[np] = i;
          fromw[np] = 1;
          ++np;
        }
      }
      for (int i = 0; i < 4 && np < 2; ++i) {
        int is_kept = 0;
        for (int t = 0; t < nk; ++t) is_kept |= kept[t] == i;
        if (!is_kept) {
          pos[np] = i;
          fromw[np] = 0;
          ++np;
        }
      }
      if (pos[0] > pos[1]) { /* ascending order */
        int t = pos[0];
        pos[0] = pos[1];
        pos[1] = t;
        t = fromw[0];
        fromw[0] = fromw[1];
        fromw[1] = t;
      }
      for (int j = 0; j < 2; ++j) {
        uint8_t* dst = v + (r * v_ld + 2 * g + j) * es;
        if (fromw[j])
          memcpy(dst, w + (r * K + 4 * g + pos[j]) * es, es);
        else
          memset(dst, 0, es);
      }
      meta[r * m_ld + g / 8] |= (uint32_t)(pos[0] | (pos[1] << 2)) << (4 * (g % 8));
    }
  }
  uint8_t* d = (uint8_t*)dense;
  for (int64_t r = 0; r < d_rows; ++r) {
    const uint8_t* src;
    if (axis == OR_AXIS_OUTPUT)
      src = w + ((dense_begin + r) * K) * es;
    else
      src = w + (r * K + dense_begin) * es;
    memcpy(d + r * d_ld * es, src, d_ld * es);
  }
  return bad;
}

/* Inverse of compress: every position not named by the metadata becomes +0. */
int or_decompress(const void* values, const uint32_t* meta, const void* dense, int64_t N, int64_t K, int es,
                  int axis, int64_t dense_begin, void* W_out) {
  int64_t L[6];
  if (or_layout(N, K, axis, dense_begin, L)) return -1;
  const int64_t s_rows = L[0], v_ld = L[1], m_ld = L[2], d_rows = L[3], d_ld = L[4], s_cols = L[5];
  const uint8_t* v = (const uint8_t*)values;
  const uint8_t* d = (const uint8_t*)dense;
  uint8_t* w = (uint8_t*)W_out;
  memset(w, 0, (size_t)(N * K * es));
  for (int64_t r = 0; r < s_rows; ++r)
    for (int64_t g = 0; g < s_cols / 4; ++g) {
      uint32_t code = (meta[r * m_ld + g / 8] >> (4 * (g % 8))) & 15u;
      int p0 = code & 3, p1 = (code >> 2) & 3;
      memcpy(w + (r * K + 4 * g + p0) * es, v + (r * v_ld + 2 * g) * es, es);
      memcpy(w + (r * K + 4 * g + p1) * es, v + (r * v_ld + 2 * g + 1) * es, es);
    }
  for (int64_t r = 0; r < d_rows; ++r) {
    uint8_t* dst;
    if (axis == OR_AXIS_OUTPUT)
      dst = w + ((dense_begin + r) * K) * es;
    else
      dst = w + (r * K + dense_begin) * es;
    memcpy(dst, d + r * d_ld * es, d_ld * es);
  }
  return 0;
}

/* ---------------------------------------------------------------- GEMM */

static void decode_row(const uint8_t* src, int64_t n, int dtype, float* out) {
  if (dtype == OR_FP8)
    for (int64_t i = 0; i < n; ++i) out[i] = (float)or_decode_e4m3fn(src[i]);
  else
    for (int64_t i = 0; i < n; ++i) out[i] = or_decode_bf16(((const uint16_t*)src)[i]);
}

/* Y = X W^T on decoded values.  X is M x K, W is N x K (both row-major codes).
 * acc  (M x N fp32, may be NULL): sum over k = 0..K-1 in ascending order from +0, fp32;
 * yf   (M x N fp32, may be NULL): (acc * sw[n]) * sx[m], two fp32 roundings;
 * ybf  (M x N bf16 bits, may be NULL): bf16_rne(yf).
 * sw / sx may be NULL, meaning 1.0. */
int or_gemm_f32(const void* X, const void* W, int64_t M, int64_t N, int64_t K, int dtype, const float* sw,
                const float* sx, float* acc, float* yf, uint16_t* ybf) {
  if (dtype != OR_FP8 && dtype != OR_BF16) return -1;
  const int es = dtype == OR_FP8 ? 1 : 2;
  float* xd = (float*)malloc(sizeof(float) * (size_t)(M * K > 0 ? M * K : 1));
  if (!xd) return -2;
  for (int64_t m = 0; m < M; ++m) decode_row((const uint8_t*)X + m * K * es, K, dtype, xd + m * K);
#pragma omp parallel
  {
    float* wd = (float*)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1));
#pragma omp for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
      decode_row((const uint8_t*)W + n * K * es, K, dtype, wd);
      for (int64_t m = 0; m < M; ++m) {
        const float* xr = xd + m * K;
        float a = 0.0f;
        for (int64_t k = 0; k < K; ++k) a += xr[k] * wd[k];
        float t = a * (sw ? sw[n] : 1.0f);
        t = t * (sx ? sx[m] : 1.0f);
        if (acc) acc[m * N + n] = a;
        if (yf) yf[m * N + n] = t;
        if (ybf) ybf[m * N + n] = or_bf16_rne(t);
      }
    }
    free(wd);
  }
  free(xd);
  return 0;
}

/* Same contraction with fp64 accumulation; y = acc * sw[n] * sx[m] in fp64, no
 * rounding to the output type.  Products of two fp8 or two bf16 values are exact. */
int or_gemm_f64(const void* X, const void* W, int64_t M, int64_t N, int64_t K, int dtype, const float* sw,
                const float* sx, double* acc, double* y, double* abs_dot) {
  if (dtype != OR_FP8 && dtype != OR_BF16) return -1;
  const int es = dtype == OR_FP8 ? 1 : 2;
  float* xd = (float*)malloc(sizeof(float) * (size_t)(M * K > 0 ? M * K : 1));
  if (!xd) return -2;
  for (int64_t m = 0; m < M; ++m) decode_row((const uint8_t*)X + m * K * es, K, dtype, xd + m * K);
#pragma omp parallel
  {
    float* wd = (float*)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1));
#pragma omp for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
      decode_row((const uint8_t*)W + n * K * es, K, dtype, wd);
      for (int64_t m = 0; m < M; ++m) {
        const float* xr = xd + m * K;
        double a = 0.0, b = 0.0;
        for (int64_t k = 0; k < K; ++k) {
          a += (double)xr[k] * (double)wd[k];
          b += fabs((double)xr[k] * (double)wd[k]);
        }
        if (acc) acc[m * N + n] = a;
        if (y) y[m * N + n] = a * (sw ? (double)sw[n] : 1.0) * (sx ? (double)sx[m] : 1.0);
        if (abs_dot) abs_dot[m * N + n] = b;
      }
    }
    free(wd);
  }
  free(xd);
  return 0;
}

/* ---------------------------------------------------------------- activation quantisation
 *
 * The steps on either side of the GEMMs in the GLU MLP the paper prunes (sec. 3.3.1,
 * Eq. (4)): MLP(X) = ((X Wup^T) .* sigma(X Wgate^T)) Wdown^T, with Wgate / Wup
 * output-split and Wdown input-split (sec. 3.2).  The activation function sigma is read
 * as SiLU (x * sigmoid(x)), the SwiGLU of the Qwen3 and Seed-OSS models the paper
 * evaluates.  Each GEMM consumes fp8 e4m3fn activations with one fp32 scale per token:
 * s[m] = max_k |a[m,k]| / 448 (1.0 for an all-zero row) and q[m,k] = e4m3fn(a[m,k] / s[m]),
 * both in fp32, the encode rounding to nearest-even and saturating to +-448.
 */

/* fp32 -> e4m3fn code from the format definition: round to nearest, ties to an even
 * mantissa; magnitudes that round past 448 saturate to 448 (the format has no infinity;
 * its all-ones pattern is NaN); NaN maps to 0x7F with the input's sign. */
uint8_t or_encode_e4m3fn(float f) {
  const uint8_t sign = signbit(f) ? 0x80 : 0x00;
  if (isnan(f)) return (uint8_t)(sign | 0x7F);
  double a = fabs((double)f);
  if (a >= 464.0) return (uint8_t)(sign | 0x7E); /* 464 is halfway from 448 to 480 */
  if (a < ldexp(1.0, -6)) {                      /* subnormal range: multiples of 2^-9 */
    double q = nearbyint(a * 512.0);             /* exact scaling; rounds half to even */
    return (uint8_t)(sign | (uint8_t)q);         /* q = 8 is the smallest normal, 0x08 */
  }
  int e = 0;
  double fr = frexp(a, &e); /* a = fr * 2^e, fr in [0.5, 1) */
  int ex = e - 1;           /* a = (1 + m) * 2^ex, m in [0, 1) */
  double m = nearbyint((fr * 2.0 - 1.0) * 8.0);
  if (m >= 8.0) {
    m = 0.0;
    ex += 1;
  }
  int code = ((ex + 7) << 3) | (int)m;
  if (code > 0x7E) code = 0x7E;
  return (uint8_t)(sign | code);
}

void or_encode_e4m3fn_array(const float* f, int64_t n, uint8_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = or_encode_e4m3fn(f[i]);
}

/* Per-token quantisation of an M x K fp32 matrix (row stride ld). */
void or_quantize_rows(const float* a, int64_t M, int64_t K, int64_t ld, uint8_t* q, float* s) {
  for (int64_t m = 0; m < M; ++m) {
    const float* r = a + m * ld;
    float amax = 0.0f;
    for (int64_t k = 0; k < K; ++k) amax = fmaxf(amax, fabsf(r[k]));
    const float sc = amax > 0.0f ? amax / 448.0f : 1.0f;
    s[m] = sc;
    for (int64_t k = 0; k < K; ++k) q[m * K + k] = or_encode_e4m3fn(r[k] / sc);
  }
}

/* GLU: h = u * silu(g) = u * g / (1 + exp(-g)), in fp64. */
void or_glu_f64(const double* g, const double* u, int64_t n, double* h) {
  for (int64_t i = 0; i < n; ++i) h[i] = u[i] * (g[i] / (1.0 + exp(-g[i])));
}
