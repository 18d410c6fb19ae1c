// Fused Spense GEMM for gfx950: Y = X W^T with W in the hybrid 2:4 / dense format
// (paper sec. 3.2), one kernel launch for both regions.
//
//   - 2:4 region: v_smfmac_f32_16x16x128_fp8_fp8 / v_smfmac_f32_16x16x64_bf16, the
//     compressed weight as the sparse A operand, one metadata word as the index register
//     (sec. 3.1.1: kept values + 2-bit positions);
//   - dense region: v_mfma_f32_16x16x128_f8f6f4 / v_mfma_f32_16x16x32_bf16;
//   - output-split: a workgroup lies in one region, so the regions write disjoint output
//     columns; input-split: a wave's fp32 accumulator runs over its 2:4 columns and then
//     its dense columns, with no rounding between the two partial products;
//   - epilogue: y = (acc * w_scale[n]) * x_scale[m], rounded to bf16 (or kept fp32).
//
// Operand layouts (measured on gfx950 with one-hot and random-integer probes):
//   A row = lane % 16 for all four instructions; D[lane][r] = (row 4*(lane/16) + r,
//   column lane % 16).  Dense: lane group q = lane/16 holds K [32q, 32q+32) (fp8) or
//   [8q, 8q+8) (bf16) of both A and B.  Sparse fp8: lane group q holds the 16 kept values
//   of logical K [32q, 32q+32) with their 2-bit positions in bits [2c, 2c+2) of the
//   index register, i.e. exactly one canonical metadata word; B holds K [16q, 16q+16) in
//   bytes 0..15 and [64+16q, 64+16q+16) in bytes 16..31.  Sparse bf16: lane group q
//   holds logical K [16q, 16q+16) (half a metadata word, chosen by shifting); B holds K
//   [8q, 8q+8) and [32+8q, 32+8q+8).
//
// Memory path (the layer is HBM-bound for small M): a workgroup owns 16*RT weight rows;
// its W waves split the K range (cost-balanced on the host) and stream their part with
// range-checked buffer loads, U instruction steps per batch of loads.  A lane whose chunk
// lies past the end of its range gets an out-of-range offset and reads zeros, so the
// loop has no divergent branches.  At the end the waves add their accumulators in LDS
// in wave order (deterministic) and the workgroup applies the epilogue.
#include "spense_internal.h"

namespace spense {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v16bf __attribute__((ext_vector_type(16)));

constexpr uint32_t kOOB = 0x80000000u;  // any offset past every buffer extent
// Cache policy of the weight loads.  Measured on MI355X: for rows read as 16 x 64-byte
// segments per instruction the default policy streams ~15% faster than non-temporal.
constexpr int kNT = 0;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
template <int AUX>
__device__ __forceinline__ v4i bl16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, AUX));
}
template <int AUX>
__device__ __forceinline__ int bl4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return (int)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, AUX);
}
__device__ __forceinline__ v8i cat8(v4i a, v4i b) { return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7); }
__device__ __forceinline__ uint32_t sel(bool ok, uint32_t off) { return ok ? off : kOOB; }

template <int DT>
struct Traits;
template <>
struct Traits<kFP8> {
  static constexpr int KS = 128;  // logical K per sparse instruction
  static constexpr int KD = 128;  // K per dense instruction
  static constexpr int ES = 1;
};
template <>
struct Traits<kBF16> {
  static constexpr int KS = 64;
  static constexpr int KD = 32;
  static constexpr int ES = 2;
};

__device__ __forceinline__ v4f mma_sparse(v4i a, v8i b, v4f c, int idx, std::integral_constant<int, kFP8>) {
  return __builtin_amdgcn_smfmac_f32_16x16x128_fp8_fp8(a, b, c, idx, 0, 0);
}
__device__ __forceinline__ v4f mma_sparse(v4i a, v8i b, v4f c, int idx, std::integral_constant<int, kBF16>) {
  return __builtin_amdgcn_smfmac_f32_16x16x64_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v16bf, b), c,
                                                   idx, 0, 0);
}
__device__ __forceinline__ v4f mma_dense(v8i a, v8i b, v4f c, std::integral_constant<int, kFP8>) {
  // fp8 e4m3 for both operands (format selectors 0), no block scales
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}
__device__ __forceinline__ v4f mma_dense(v8i a, v8i b, v4f c, std::integral_constant<int, kBF16>) {
  const v4i a4 = {a[0], a[1], a[2], a[3]}, b4 = {b[0], b[1], b[2], b[3]};
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a4), __builtin_bit_cast(v8bf, b4), c, 0,
                                                 0, 0);
}

// ---------------------------------------------------------------- pipeline stages
// One stage = U instruction steps of one wave.  Offsets are byte offsets into the
// buffers; masked lanes use kOOB and read zeros.
template <int DT, int CT, int RT, int U>
struct SparseStage {
  v4i a[U][RT];
  int ix[U][RT];
  v8i b[U][CT];
};
template <int DT, int CT, int RT, int U>
struct DenseStage {
  v8i a[U][RT];
  v8i b[U][CT];
};

struct LaneCtx {
  __amdgpu_buffer_rsrc_t rx, rv, rm, rd;
  int lq;
};

template <int DT, int CT, int RT, int U, bool WM>
__device__ __forceinline__ void load_sparse(SparseStage<DT, CT, RT, U>& st, const LaneCtx& L, const uint32_t (&vrow)[RT],
                                            const uint32_t (&mrow)[RT], const uint32_t (&xrow)[CT],
                                            const bool (&xok)[CT], int k, int kend) {
  const int lq = L.lq;
#pragma unroll
  for (int j = 0; j < U; ++j) {
    const int kk = k + j * Traits<DT>::KS;
    if constexpr (DT == kFP8) {
      const bool oka = kk + 32 * lq < kend;  // this lane group's 32 logical K
#pragma unroll
      for (int t = 0; t < RT; ++t) {
        st.a[j][t] = bl16<kNT>(L.rv, sel(oka, vrow[t] + (kk >> 1)));
        if constexpr (!WM) st.ix[j][t] = bl4<kNT>(L.rm, sel(oka, mrow[t] + 4 * (kk >> 5)));
      }
      const bool ok0 = kk + 16 * lq < kend, ok1 = kk + 64 + 16 * lq < kend;
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const v4i p0 = bl16<0>(L.rx, sel(ok0 && xok[c], xrow[c] + kk));
        const v4i p1 = bl16<0>(L.rx, sel(ok1 && xok[c], xrow[c] + kk + 64));
        st.b[j][c] = cat8(p0, p1);
      }
    } else {
      const bool oka = kk + 16 * lq < kend;
#pragma unroll
      for (int t = 0; t < RT; ++t) {
        st.a[j][t] = bl16<kNT>(L.rv, sel(oka, vrow[t] + kk));
        st.ix[j][t] = (int)((uint32_t)bl4<kNT>(L.rm, sel(oka, mrow[t] + 4 * (kk >> 5))) >> (16 * (lq & 1)));
      }
      const bool ok0 = kk + 8 * lq < kend, ok1 = kk + 32 + 8 * lq < kend;
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const v4i p0 = bl16<0>(L.rx, sel(ok0 && xok[c], xrow[c] + 2 * kk));
        const v4i p1 = bl16<0>(L.rx, sel(ok1 && xok[c], xrow[c] + 2 * (kk + 32)));
        st.b[j][c] = cat8(p0, p1);
      }
    }
  }
  if constexpr (WM) {
    static_assert(DT == kFP8 && U % 4 == 0, "wide metadata loads cover four fp8 steps");
    // Metadata for four steps at once: lane group q loads the 16 bytes holding words
    // 4q..4q+3 of those steps' 16 words (one line segment per row), then a 4x4 transpose
    // across lane groups hands step j's word 4j+q to lane group q.  Words of steps past
    // kend only meet zeroed A and B operands.
#pragma unroll
    for (int j0 = 0; j0 < U; j0 += 4) {
      const int kk = k + j0 * Traits<DT>::KS;
#pragma unroll
      for (int t = 0; t < RT; ++t) {
        const v4i w = bl16<kNT>(L.rm, sel(kk + 128 * lq < kend, mrow[t] + 4 * (kk >> 5) + 12 * lq));
        const auto s02 = __builtin_amdgcn_permlane32_swap((unsigned)w[0], (unsigned)w[2], false, false);
        const auto s13 = __builtin_amdgcn_permlane32_swap((unsigned)w[1], (unsigned)w[3], false, false);
        const auto s01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
        const auto s23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
        st.ix[j0 + 0][t] = (int)s01[0];
        st.ix[j0 + 1][t] = (int)s01[1];
        st.ix[j0 + 2][t] = (int)s23[0];
        st.ix[j0 + 3][t] = (int)s23[1];
      }
    }
  }
}

template <int DT, int CT, int RT, int U>
__device__ __forceinline__ void load_dense(DenseStage<DT, CT, RT, U>& st, const LaneCtx& L, const uint32_t (&drow)[RT],
                                           const uint32_t (&xrow)[CT], const bool (&xok)[CT], int k, int kend,
                                           int dco) {
  const int lq = L.lq;
  const v4i z = {0, 0, 0, 0};
#pragma unroll
  for (int j = 0; j < U; ++j) {
    const int kk = k + j * Traits<DT>::KD;
    if constexpr (DT == kFP8) {
      const bool ok = kk + 32 * lq < kend;
#pragma unroll
      for (int t = 0; t < RT; ++t) {
        const uint32_t o = sel(ok, drow[t] + (uint32_t)(kk - dco));
        st.a[j][t] = cat8(bl16<kNT>(L.rd, o), bl16<kNT>(L.rd, o + 16));
      }
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const uint32_t o = sel(ok && xok[c], xrow[c] + kk);
        st.b[j][c] = cat8(bl16<0>(L.rx, o), bl16<0>(L.rx, o + 16));
      }
    } else {
      const bool ok = kk + 8 * lq < kend;
#pragma unroll
      for (int t = 0; t < RT; ++t) st.a[j][t] = cat8(bl16<kNT>(L.rd, sel(ok, drow[t] + 2 * (uint32_t)(kk - dco))), z);
#pragma unroll
      for (int c = 0; c < CT; ++c) st.b[j][c] = cat8(bl16<0>(L.rx, sel(ok && xok[c], xrow[c] + 2 * kk)), z);
    }
  }
}

template <int DT, int CT, int RT, int U>
__device__ __forceinline__ void mma_stage(v4f (&acc)[RT][CT], const SparseStage<DT, CT, RT, U>& st) {
#pragma unroll
  for (int j = 0; j < U; ++j)
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int c = 0; c < CT; ++c)
        acc[t][c] = mma_sparse(st.a[j][t], st.b[j][c], acc[t][c], st.ix[j][t], std::integral_constant<int, DT>());
}
template <int DT, int CT, int RT, int U>
__device__ __forceinline__ void mma_stage(v4f (&acc)[RT][CT], const DenseStage<DT, CT, RT, U>& st) {
#pragma unroll
  for (int j = 0; j < U; ++j)
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int c = 0; c < CT; ++c)
        acc[t][c] = mma_dense(st.a[j][t], st.b[j][c], acc[t][c], std::integral_constant<int, DT>());
}

// One stage at a time: issue all loads of U steps, then feed the matrix cores.  Latency
// is hidden by the many resident waves rather than by register double buffering, which
// measured slower on MI355X for this access pattern.
template <typename Stage, typename LoadFn, int RT, int CT>
__device__ __forceinline__ void run_pipeline(v4f (&acc)[RT][CT], int k0, int kend, int step, LoadFn load) {
  for (int k = k0; k < kend; k += step) {
    Stage st;
    load(st, k);
    mma_stage(acc, st);
  }
}

// ---------------------------------------------------------------- epilogue
__device__ __forceinline__ uint32_t bf16_bits(float v) {
  __bf16 h = (__bf16)v;  // round to nearest even
  return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

// Four consecutive outputs n0..n0+3 of activation row m.
__device__ __forceinline__ void store4(const GemmArgs& a, v4f acc, int m, int n0, int rowend) {
  const float xs = a.sx ? a.sx[m] : 1.0f;
  float v[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int n = n0 + r < rowend ? n0 + r : rowend - 1;
    float y = acc[r];
    if (a.sw) y = y * a.sw[n];
    v[r] = y * xs;
  }
  if (a.out_f32) {
    float* yp = reinterpret_cast<float*>(a.Y) + (int64_t)m * a.ldy + n0;
    if (a.vec_store && n0 + 3 < rowend) {
      *reinterpret_cast<v4f*>(yp) = (v4f){v[0], v[1], v[2], v[3]};
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (n0 + r < rowend) yp[r] = v[r];
    }
  } else {
    uint16_t* yp = reinterpret_cast<uint16_t*>(a.Y) + (int64_t)m * a.ldy + n0;
    const uint32_t b0 = bf16_bits(v[0]), b1 = bf16_bits(v[1]), b2 = bf16_bits(v[2]), b3 = bf16_bits(v[3]);
    if (a.vec_store && n0 + 3 < rowend) {
      typedef uint32_t u2 __attribute__((ext_vector_type(2)));
      *reinterpret_cast<u2*>(yp) = (u2){b0 | (b1 << 16), b2 | (b3 << 16)};
    } else {
      const uint32_t bb[4] = {b0, b1, b2, b3};
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (n0 + r < rowend) yp[r] = (uint16_t)bb[r];
    }
  }
}

// ---------------------------------------------------------------- kernel
template <int DT, int CT, int RT, int W, int U, bool WM>
__global__ __launch_bounds__(64 * W) void spense_gemm_kernel(GemmArgs a) {
  typedef Traits<DT> T;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int li = lane & 15, lq = lane >> 4;
  const int g = blockIdx.x, mb = blockIdx.y;
  const int ri = (a.nreg > 1 && g >= a.reg[1].wg0) ? 1 : 0;
  const Region& R = a.reg[ri];
  const int nbase = R.row0 + (g - R.wg0) * 16 * RT;
  const int rowend = R.row0 + R.rows;
  const int m0 = mb * 16 * CT;
  const int ka = R.cut[wave], kb = R.cut[wave + 1];
  const int ks_end = min(kb, R.kbound);  // 2:4 columns of this wave: [ka, ks_end)
  const int kd_beg = max(ka, R.kbound);  // dense columns of this wave: [kd_beg, kb)

  LaneCtx L;
  L.lq = lq;
  L.rx = rsrc(a.X, a.x_bytes);
  L.rv = rsrc(a.values, a.v_bytes);
  L.rm = rsrc(a.meta, a.m_bytes);
  L.rd = rsrc(a.dense, a.d_bytes);

  v4f acc[RT][CT];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int c = 0; c < CT; ++c) acc[t][c] = (v4f){0.f, 0.f, 0.f, 0.f};

  uint32_t xrow[CT];
  bool xok[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const int m = m0 + 16 * c + li;
    xok[c] = m < a.M;
    // lane group offset inside a step: sparse B pieces start at 16q (fp8) / 8q (bf16)
    // logical K, dense B at 32q / 8q; both are encoded at load time from kk.
    xrow[c] = (uint32_t)((int64_t)(xok[c] ? m : 0) * a.ldx_b);
  }

  if (ka < ks_end) {
    uint32_t vrow[RT], mrow[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      const int n = min(nbase + 16 * t + li, rowend - 1);
      vrow[t] = (uint32_t)((int64_t)n * a.v_ld_b) + (DT == kFP8 ? 16u : 16u) * lq;
      mrow[t] = (uint32_t)((int64_t)n * a.m_ld_b) + (DT == kFP8 ? 4u * lq : 4u * (lq >> 1));
    }
    uint32_t xr[CT];
#pragma unroll
    for (int c = 0; c < CT; ++c) xr[c] = xrow[c] + (DT == kFP8 ? 16u * lq : 16u * lq);
    run_pipeline<SparseStage<DT, CT, RT, U>>(acc, ka, ks_end, U * T::KS, [&](SparseStage<DT, CT, RT, U>& st, int k) {
      load_sparse<DT, CT, RT, U, WM>(st, L, vrow, mrow, xr, xok, k, ks_end);
    });
  }
  if (kd_beg < kb) {
    uint32_t drow[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      const int n = min(nbase + 16 * t + li, rowend - 1);
      drow[t] = (uint32_t)((int64_t)(n - R.dense_row_off) * a.d_ld_b) + (DT == kFP8 ? 32u * lq : 16u * lq);
    }
    uint32_t xr[CT];
#pragma unroll
    for (int c = 0; c < CT; ++c) xr[c] = xrow[c] + (DT == kFP8 ? 32u * lq : 16u * lq);
    const int dco = R.dense_col_off;
    run_pipeline<DenseStage<DT, CT, RT, U>>(acc, kd_beg, kb, U * T::KD, [&](DenseStage<DT, CT, RT, U>& st, int k) {
      load_dense<DT, CT, RT, U>(st, L, drow, xr, xok, k, kb, dco);
    });
  }

  // ---- add the waves' partial sums in LDS (wave order), then the epilogue
  __shared__ v4f red[W * RT * CT * 64];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int c = 0; c < CT; ++c) red[((wave * RT + t) * CT + c) * 64 + lane] = acc[t][c];
  __syncthreads();
  for (int e = threadIdx.x; e < RT * CT * 64; e += 64 * W) {
    const int ln = e & 63, tc = e >> 6;
    const int t = tc / CT, c = tc - t * CT;
    v4f s = red[e];
#pragma unroll
    for (int w = 1; w < W; ++w) s += red[w * RT * CT * 64 + e];
    const int m = m0 + 16 * c + (ln & 15);
    const int n0 = nbase + 16 * t + 4 * (ln >> 4);
    if (m < a.M && n0 < rowend) store4(a, s, m, n0, rowend);
  }
}

template <int DT, int CT, int RT, int W, int UMAX = 0>
hipError_t launch_t(const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  // steps per pipeline stage: keep two stages of operands within the register budget
  constexpr int per_step = 8 * RT + 8 * CT;  // VGPRs of one dense step (the larger kind)
  constexpr int budget = W >= 16 ? 80 : (W >= 8 ? 100 : 128);
  constexpr int U0 = budget / per_step;
  constexpr int U = UMAX ? UMAX : (U0 < 1 ? 1 : (U0 > 4 ? 4 : U0));
  dim3 grid(a.groups, ls.mblocks), block(64 * W);
  // metadata rows 16-byte aligned -> one 16-byte load covers four steps of a row
  constexpr bool kWide = DT == kFP8 && U % 4 == 0;
  if (kWide && a.m_ld_b % 16 == 0)
    hipLaunchKernelGGL((spense_gemm_kernel<DT, CT, RT, W, U, kWide>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((spense_gemm_kernel<DT, CT, RT, W, U, false>), grid, block, 0, s, a);
  return hipGetLastError();
}

template <int DT, int CT>
hipError_t launch_ct(const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  // W * RT * CT <= 64 keeps the LDS reduction buffer at 64 KB
  switch (ls.rt * 100 + ls.waves + (ls.u8 && CT == 1 ? 10000 : 0)) {
    case 104: return launch_t<DT, CT, 1, 4>(ls, a, s);
    case 108: return launch_t<DT, CT, 1, 8>(ls, a, s);
    case 116: return launch_t<DT, CT, 1, 16>(ls, a, s);
    case 204: return launch_t<DT, CT, 2, 4>(ls, a, s);
    case 208: return launch_t<DT, CT, 2, 8>(ls, a, s);
    case 404: return launch_t<DT, CT, 4, 4>(ls, a, s);
    case 10104: return launch_t<DT, CT, 1, 4, 8>(ls, a, s);
    case 10108: return launch_t<DT, CT, 1, 8, 8>(ls, a, s);
    default: return hipErrorInvalidValue;
  }
}

template <int DT>
hipError_t launch_dt(const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  if (ls.ct == 1) return launch_ct<DT, 1>(ls, a, s);
  if (ls.ct == 2) return launch_ct<DT, 2>(ls, a, s);
  return launch_ct<DT, 4>(ls, a, s);
}

}  // namespace

hipError_t launch_gemm(int dtype, const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  return dtype == kFP8 ? launch_dt<kFP8>(ls, a, s) : launch_dt<kBF16>(ls, a, s);
}

}  // namespace spense
