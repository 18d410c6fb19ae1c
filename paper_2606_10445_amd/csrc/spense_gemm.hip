// Fused Spense GEMM for gfx950: Y = X W^T with W in the hybrid 2:4 / dense format
// (paper sec. 3.2).  One launch covers both regions:
//   - 2:4 region: v_smfmac_f32_16x16x128_fp8_fp8 / v_smfmac_f32_16x16x64_bf16 with the
//     compressed weight as the sparse A operand and the metadata word as the index
//     register (sec. 3.1.1: values + 2-bit positions);
//   - dense region: v_mfma_f32_16x16x128_f8f6f4 / v_mfma_f32_16x16x32_bf16;
//   - output-split: a work unit lies in one region, so the two regions write disjoint
//     output columns; input-split: the same fp32 accumulator runs over the 2:4 columns
//     and then the dense columns (no rounding between the two partial products);
//   - epilogue: y = ((acc * w_scale[n]) * x_scale[m]) rounded to bf16 (or fp32).
//
// Operand layouts (measured on gfx950 with one-hot and random-integer probes):
//   A row  = lane % 16 for all four instructions, D[lane, r] = (row 4*(lane/16) + r,
//   column lane % 16).  Dense: lane group q = lane/16 holds K [32q, 32q+32) (fp8) or
//   [8q, 8q+8) (bf16) of A and of B.  Sparse fp8: lane group q holds the 16 compressed
//   values of logical K [32q, 32q+32) and their 2-bit positions in bits [2c, 2c+2) of
//   the index register - exactly one canonical metadata word; B holds K
//   [16q, 16q+16) in bytes 0..15 and [64+16q, 64+16q+16) in bytes 16..31.  Sparse
//   bf16: lane group q holds logical K [16q, 16q+16) (half a metadata word, selected by
//   shifting), B holds K [8q, 8q+8) and [32+8q, 32+8q+8).
//
// Work decomposition: a unit is (region, block of 16*RT*WAVES output rows, K range,
// block of 16*CT activation rows).  When a region's K is split over several units, each
// writes fp32 partials to the workspace and the last one to arrive (counter) sums them
// in split order, so results do not depend on scheduling.
#include "spense_internal.h"

namespace spense {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v16bf __attribute__((ext_vector_type(16)));

__device__ __forceinline__ v4i ld16(const uint8_t* p) { return *reinterpret_cast<const v4i*>(p); }
__device__ __forceinline__ v8i cat8(v4i a, v4i b) { return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7); }

template <int DT>
struct Traits;
template <>
struct Traits<kFP8> {
  static constexpr int KS = 128;  // logical K per sparse instruction
  static constexpr int KD = 128;  // K per dense instruction
  typedef v8i DenseA;
  typedef v8i DenseB;
};
template <>
struct Traits<kBF16> {
  static constexpr int KS = 64;
  static constexpr int KD = 32;
  typedef v4i DenseA;
  typedef v4i DenseB;
};

__device__ __forceinline__ v4f mma_sparse(v4i a, v8i b, v4f c, int idx, std::integral_constant<int, kFP8>) {
  return __builtin_amdgcn_smfmac_f32_16x16x128_fp8_fp8(a, b, c, idx, 0, 0);
}
__device__ __forceinline__ v4f mma_sparse(v4i a, v8i b, v4f c, int idx, std::integral_constant<int, kBF16>) {
  return __builtin_amdgcn_smfmac_f32_16x16x64_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v16bf, b), c,
                                                   idx, 0, 0);
}
__device__ __forceinline__ v4f mma_dense(v8i a, v8i b, v4f c) {
  // fp8 e4m3 for both operands (format selectors 0), no block scales
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}
__device__ __forceinline__ v4f mma_dense(v4i a, v4i b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c, 0, 0,
                                                 0);
}

// ---------------------------------------------------------------- fragment loads
// Sparse A: compressed values of logical K [k + span*q, ...) of one row plus the index.
template <int DT>
__device__ __forceinline__ void load_sparse_a(const uint8_t* vrow, const uint32_t* mrow, int k, int lq, bool ok,
                                              v4i& a, int& idx) {
  if constexpr (DT == kFP8) {
    // logical K [k + 32q, +32) -> 16 compressed bytes at k/2 + 16q, metadata word k/32 + q
    if (ok) {
      a = ld16(vrow + (k >> 1) + 16 * lq);
      idx = (int)mrow[(k >> 5) + lq];
    } else {
      a = (v4i){0, 0, 0, 0};
      idx = 0;
    }
  } else {
    // logical K [k + 16q, +16) -> 8 bf16 at element k/2 + 8q, half of word k/32 + q/2
    if (ok) {
      a = ld16(vrow + k + 16 * lq);
      idx = (int)(mrow[(k >> 5) + (lq >> 1)] >> (16 * (lq & 1)));
    } else {
      a = (v4i){0, 0, 0, 0};
      idx = 0;
    }
  }
}

// Sparse B (activations): two 16-byte pieces of one activation row.
template <int DT>
__device__ __forceinline__ v8i load_sparse_b(const uint8_t* xrow, int k, int lq, bool ok0, bool ok1) {
  const v4i z = {0, 0, 0, 0};
  if constexpr (DT == kFP8) {
    v4i p0 = ok0 ? ld16(xrow + k + 16 * lq) : z;
    v4i p1 = ok1 ? ld16(xrow + k + 64 + 16 * lq) : z;
    return cat8(p0, p1);
  } else {
    v4i p0 = ok0 ? ld16(xrow + 2 * (k + 8 * lq)) : z;
    v4i p1 = ok1 ? ld16(xrow + 2 * (k + 32 + 8 * lq)) : z;
    return cat8(p0, p1);
  }
}

template <int DT>
__device__ __forceinline__ typename Traits<DT>::DenseA load_dense_a(const uint8_t* drow, int kc, int lq, bool ok) {
  if constexpr (DT == kFP8) {
    const v4i z = {0, 0, 0, 0};
    if (!ok) return cat8(z, z);
    const uint8_t* p = drow + kc + 32 * lq;
    return cat8(ld16(p), ld16(p + 16));
  } else {
    if (!ok) return (v4i){0, 0, 0, 0};
    return ld16(drow + 2 * (kc + 8 * lq));
  }
}

template <int DT>
__device__ __forceinline__ typename Traits<DT>::DenseB load_dense_b(const uint8_t* xrow, int k, int lq, bool ok) {
  if constexpr (DT == kFP8) {
    const v4i z = {0, 0, 0, 0};
    if (!ok) return cat8(z, z);
    const uint8_t* p = xrow + k + 32 * lq;
    return cat8(ld16(p), ld16(p + 16));
  } else {
    if (!ok) return (v4i){0, 0, 0, 0};
    return ld16(xrow + 2 * (k + 8 * lq));
  }
}

// ---------------------------------------------------------------- epilogue
__device__ __forceinline__ uint32_t bf16_bits(float v) {
  __bf16 h = (__bf16)v;  // round to nearest even
  return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

template <int RT, int CT>
__device__ __forceinline__ void store_tile(const GemmArgs& a, const v4f (&acc)[RT][CT], int nbase, int rowend, int m0,
                                           int li, int lq) {
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const int m = m0 + 16 * c + li;
    if (m >= a.M) continue;
    const float xs = a.sx ? a.sx[m] : 1.0f;
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      const int n0 = nbase + 16 * t + 4 * lq;
      if (n0 >= rowend) continue;
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int n = n0 + r < rowend ? n0 + r : rowend - 1;
        float y = acc[t][c][r];
        if (a.sw) y = y * a.sw[n];
        y = y * xs;
        v[r] = y;
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
  }
}

// ---------------------------------------------------------------- kernel
template <int DT, int CT, int RT, int WAVES, int U>
__global__ __launch_bounds__(64 * WAVES) void spense_gemm_kernel(GemmArgs a) {
  typedef Traits<DT> T;
  constexpr int KS = T::KS, KD = T::KD;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int li = lane & 15, lq = lane >> 4;
  const int u = blockIdx.x, mb = blockIdx.y;
  const int ri = (a.nreg > 1 && u >= a.reg[1].unit0) ? 1 : 0;
  const Region& R = a.reg[ri];
  const int S = R.splits;
  const int local = u - R.unit0;
  const int rb = local / S, s = local - rb * S;
  const int ka = R.cut[s], kb = R.cut[s + 1];
  const int ks_end = min(kb, R.kbound);    // 2:4 columns of this unit: [ka, ks_end)
  const int kd_beg = max(ka, R.kbound);    // dense columns of this unit: [kd_beg, kb)
  const int rowend = R.row0 + R.rows;
  const int nbase = R.row0 + rb * (16 * RT * WAVES) + wave * 16 * RT;
  const int m0 = mb * 16 * CT;

  v4f acc[RT][CT];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int c = 0; c < CT; ++c) acc[t][c] = (v4f){0.f, 0.f, 0.f, 0.f};

  const uint8_t* xrow[CT];
  bool xok[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const int m = m0 + 16 * c + li;
    xok[c] = m < a.M;
    xrow[c] = a.X + (int64_t)(xok[c] ? m : 0) * a.ldx_b;
  }

  if (nbase < rowend && ka < ks_end) {
    const uint8_t* vrow[RT];
    const uint32_t* mrow[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      const int n = min(nbase + 16 * t + li, rowend - 1);
      vrow[t] = a.values + (int64_t)n * a.v_ld_b;
      mrow[t] = a.meta + (int64_t)n * a.m_ld;
    }
    const int kb2 = ks_end;
    int k = ka;
    for (; k + U * KS <= kb2; k += U * KS) {
      v4i av[U][RT];
      int ix[U][RT];
      v8i bv[U][CT];
#pragma unroll
      for (int j = 0; j < U; ++j) {
#pragma unroll
        for (int t = 0; t < RT; ++t) load_sparse_a<DT>(vrow[t], mrow[t], k + j * KS, lq, true, av[j][t], ix[j][t]);
#pragma unroll
        for (int c = 0; c < CT; ++c) bv[j][c] = load_sparse_b<DT>(xrow[c], k + j * KS, lq, xok[c], xok[c]);
      }
#pragma unroll
      for (int j = 0; j < U; ++j)
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
          for (int c = 0; c < CT; ++c)
            acc[t][c] = mma_sparse(av[j][t], bv[j][c], acc[t][c], ix[j][t], std::integral_constant<int, DT>());
    }
    for (; k < kb2; k += KS) {  // ragged tail: lanes past kb2 contribute zeros
      constexpr int qa = DT == kFP8 ? 32 : 16, pb = DT == kFP8 ? 16 : 8, hb = DT == kFP8 ? 64 : 32;
      v4i av[RT];
      int ix[RT];
      v8i bv[CT];
#pragma unroll
      for (int t = 0; t < RT; ++t) load_sparse_a<DT>(vrow[t], mrow[t], k, lq, k + qa * lq < kb2, av[t], ix[t]);
#pragma unroll
      for (int c = 0; c < CT; ++c)
        bv[c] = load_sparse_b<DT>(xrow[c], k, lq, xok[c] && k + pb * lq < kb2, xok[c] && k + hb + pb * lq < kb2);
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int c = 0; c < CT; ++c)
          acc[t][c] = mma_sparse(av[t], bv[c], acc[t][c], ix[t], std::integral_constant<int, DT>());
    }
  }
  if (nbase < rowend && kd_beg < kb) {
    const uint8_t* drow[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      const int n = min(nbase + 16 * t + li, rowend - 1);
      drow[t] = a.dense + (int64_t)(n - R.dense_row_off) * a.d_ld_b;
    }
    const int dco = R.dense_col_off;
    int k = kd_beg;
    for (; k + U * KD <= kb; k += U * KD) {
      typename T::DenseA av[U][RT];
      typename T::DenseB bv[U][CT];
#pragma unroll
      for (int j = 0; j < U; ++j) {
#pragma unroll
        for (int t = 0; t < RT; ++t) av[j][t] = load_dense_a<DT>(drow[t], k + j * KD - dco, lq, true);
#pragma unroll
        for (int c = 0; c < CT; ++c) bv[j][c] = load_dense_b<DT>(xrow[c], k + j * KD, lq, xok[c]);
      }
#pragma unroll
      for (int j = 0; j < U; ++j)
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
          for (int c = 0; c < CT; ++c) acc[t][c] = mma_dense(av[j][t], bv[j][c], acc[t][c]);
    }
    for (; k < kb; k += KD) {
      constexpr int qa = DT == kFP8 ? 32 : 8;
      const bool ok = k + qa * lq < kb;
      typename T::DenseA av[RT];
      typename T::DenseB bv[CT];
#pragma unroll
      for (int t = 0; t < RT; ++t) av[t] = load_dense_a<DT>(drow[t], k - dco, lq, ok);
#pragma unroll
      for (int c = 0; c < CT; ++c) bv[c] = load_dense_b<DT>(xrow[c], k, lq, ok && xok[c]);
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int c = 0; c < CT; ++c) acc[t][c] = mma_dense(av[t], bv[c], acc[t][c]);
    }
  }

  if (S == 1) {
    if (nbase < rowend) store_tile<RT, CT>(a, acc, nbase, rowend, m0, li, lq);
    return;
  }

  // ---- split K: write partials, the last unit of this (row block, M block) reduces
  const int64_t MN = (int64_t)a.M * a.N;
  if (nbase < rowend) {
    float* P = a.part + (int64_t)s * MN;
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      const int m = m0 + 16 * c + li;
      if (m >= a.M) continue;
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = nbase + 16 * t + 4 * lq + r;
          if (n < rowend) P[(int64_t)m * a.N + n] = acc[t][c][r];
        }
    }
  }
  __threadfence();
  __syncthreads();
  __shared__ uint32_t s_last;
  const int ctr = R.ctr0 + rb + mb * a.counters_per_mb;
  if (threadIdx.x == 0) {
    const uint32_t prev = atomicAdd(&a.counters[ctr], 1u);
    s_last = prev == (uint32_t)(S - 1);
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  if (nbase < rowend) {
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      const int m = m0 + 16 * c + li;
      if (m >= a.M) continue;
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = nbase + 16 * t + 4 * lq + r;
          float sum = 0.f;
          if (n < rowend) {
            const float* P = a.part + (int64_t)m * a.N + n;
            for (int j = 0; j < S; ++j) sum += P[(int64_t)j * MN];
          }
          acc[t][c][r] = sum;
        }
    }
    store_tile<RT, CT>(a, acc, nbase, rowend, m0, li, lq);
  }
  if (threadIdx.x == 0) atomicExch(&a.counters[ctr], 0u);
}

template <int DT, int CT, int RT>
hipError_t launch_t(const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  constexpr int U = CT == 1 ? 4 : 2;
  dim3 grid(a.units, ls.mblocks), block(64 * 4);
  hipLaunchKernelGGL((spense_gemm_kernel<DT, CT, RT, 4, U>), grid, block, 0, s, a);
  return hipGetLastError();
}

template <int DT>
hipError_t launch_dt(const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  if (ls.rt == 1) {
    if (ls.ct == 1) return launch_t<DT, 1, 1>(ls, a, s);
    if (ls.ct == 2) return launch_t<DT, 2, 1>(ls, a, s);
    return launch_t<DT, 4, 1>(ls, a, s);
  }
  if (ls.ct == 1) return launch_t<DT, 1, 2>(ls, a, s);
  if (ls.ct == 2) return launch_t<DT, 2, 2>(ls, a, s);
  return launch_t<DT, 4, 2>(ls, a, s);
}

}  // namespace

hipError_t launch_gemm(int dtype, const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  if (ls.waves != 4) return hipErrorInvalidValue;
  return dtype == kFP8 ? launch_dt<kFP8>(ls, a, s) : launch_dt<kBF16>(ls, a, s);
}

}  // namespace spense
