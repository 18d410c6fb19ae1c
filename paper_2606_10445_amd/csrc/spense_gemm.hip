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
//   [8q, 8q+8) (bf16) of both A and B.  Any permutation of K applied to both operands
//   gives the same dot products, so the dense fp8 step feeds lane group q the K range
//   [16q, 16q+16) in bytes 0..15 and [64+16q, 64+16q+16) in bytes 16..31 (the sparse B
//   order): each 16-byte load instruction then covers 64 contiguous bytes of a row.  Sparse fp8: lane group q holds the 16 kept values
//   of logical K [32q, 32q+32) with their 2-bit positions in bits [2c, 2c+2) of the
//   index register, i.e. exactly one canonical metadata word; B holds K [16q, 16q+16) in
//   bytes 0..15 and [64+16q, 64+16q+16) in bytes 16..31.  Sparse bf16: lane group q
//   holds logical K [16q, 16q+16) (half a metadata word, chosen by shifting); B holds K
//   [8q, 8q+8) and [32+8q, 32+8q+8).
//
// Five GEMM kernels; the host planner picks one per call from M and the weight geometry:
//   - spense_gemm_rows_kernel (decode, HBM-bound): each wave owns 16 weight rows over all
//     of K; the waves of a workgroup share every chunk of activations through LDS (or
//     keep all of them resident) and keep two chunks of weights in flight; K slices, where
//     the weight has few rows, go through splitk_reduce_kernel;
//   - spense_gemm_rows2_kernel (65-256 tokens): the same with two 64-token halves per
//     workgroup, each weight chunk feeding both;
//   - spense_gemm_kernel: a workgroup owns 16*RT weight rows and its W waves split the K
//     range (cost-balanced on the host), U instruction steps per batch of loads; at the
//     end the waves add their accumulators in LDS in wave order (deterministic);
//   - spense_gemm_big_kernel / spense_gemm_big2_kernel (many tokens): 128 x 256 and
//     256 x 256 (or 256 x 192) workgroup tiles with both operands copied into LDS a few
//     steps ahead; their bf16 output tile leaves through LDS as whole token rows.
// All loads are range-checked buffer loads: a lane whose chunk lies past the end of its
// range gets an out-of-range offset and reads zeros, so the loops have no divergent
// branches.
#include <mutex>

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
// segments per instruction the default policy streams ~15% faster than non-temporal;
// for the tiled layout (1 KB contiguous per instruction) non-temporal is 5-9% faster.
constexpr int kNT = 0;
constexpr int kTiledNT = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
// voffset: per-lane byte offset; soffset: wave-uniform byte offset (scalar register)
template <int AUX>
__device__ __forceinline__ v4i bl16(__amdgpu_buffer_rsrc_t r, uint32_t off, int soff = 0) {
  return __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, soff, AUX));
}
template <int AUX>
__device__ __forceinline__ int bl4(__amdgpu_buffer_rsrc_t r, uint32_t off, int soff = 0) {
  return (int)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, soff, AUX);
}
__device__ __forceinline__ v8i cat8(v4i a, v4i b) { return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7); }
__device__ __forceinline__ uint32_t sel(bool ok, uint32_t off) { return ok ? off : kOOB; }

// Matrix-core results are written several cycles after the instruction issues (up to
// about a dozen wait states for the 8-pass fp8 instruction), and the hardware does not
// interlock a later non-matrix read (or a matrix read of a different register) against
// that write.  Where such a read sits in another basic block than the producing matrix
// instruction (loop exits, the 2:4 -> dense switch, the epilogue), the compiler's own
// padding was measured to fall short on gfx950, so these points get 20 explicit wait
// states.  The scheduling barriers keep instructions from moving across them.
__device__ __forceinline__ void xdl_fence() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

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

// FULL: every step of the stage lies inside [k, kend): no per-lane masks, the step's K
// offset travels in the scalar offset.  Otherwise lanes past kend read zeros.
template <int DT, int CT, int RT, int U, bool WM, bool FULL>
__device__ __forceinline__ void load_sparse(SparseStage<DT, CT, RT, U>& st, const LaneCtx& L, const uint32_t (&vrow)[RT],
                                            const uint32_t (&mrow)[RT], const uint32_t (&xrow)[CT],
                                            const bool (&xok)[CT], int k, int kend) {
  const int lq = L.lq;
#pragma unroll
  for (int j = 0; j < U; ++j) {
    const int kk = k + j * Traits<DT>::KS;
    if constexpr (DT == kFP8 && FULL) {
#pragma unroll
      for (int t = 0; t < RT; ++t) {
        st.a[j][t] = bl16<kNT>(L.rv, vrow[t], kk >> 1);
        if constexpr (!WM) st.ix[j][t] = bl4<kNT>(L.rm, mrow[t], 4 * (kk >> 5));
      }
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const uint32_t o = xok[c] ? xrow[c] : kOOB;
        st.b[j][c] = cat8(bl16<0>(L.rx, o, kk), bl16<0>(L.rx, o, kk + 64));
      }
    } else if constexpr (DT == kFP8) {
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
        const v4i w = FULL ? bl16<kNT>(L.rm, mrow[t] + 12 * lq, 4 * (kk >> 5))
                           : bl16<kNT>(L.rm, sel(kk + 128 * lq < kend, mrow[t] + 4 * (kk >> 5) + 12 * lq));
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

template <int DT, int CT, int RT, int U, bool FULL>
__device__ __forceinline__ void load_dense(DenseStage<DT, CT, RT, U>& st, const LaneCtx& L, const uint32_t (&drow)[RT],
                                           const uint32_t (&xrow)[CT], const bool (&xok)[CT], int k, int kend,
                                           int dco) {
  const int lq = L.lq;
  const v4i z = {0, 0, 0, 0};
#pragma unroll
  for (int j = 0; j < U; ++j) {
    const int kk = k + j * Traits<DT>::KD;
    if constexpr (DT == kFP8 && FULL) {
#pragma unroll
      for (int t = 0; t < RT; ++t) st.a[j][t] = cat8(bl16<kNT>(L.rd, drow[t], kk - dco), bl16<kNT>(L.rd, drow[t], kk - dco + 64));
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const uint32_t o = xok[c] ? xrow[c] : kOOB;
        st.b[j][c] = cat8(bl16<0>(L.rx, o, kk), bl16<0>(L.rx, o, kk + 64));
      }
    } else if constexpr (DT == kFP8) {
      const bool ok0 = kk + 16 * lq < kend, ok1 = kk + 64 + 16 * lq < kend;
#pragma unroll
      for (int t = 0; t < RT; ++t) {
        const uint32_t o = drow[t] + (uint32_t)(kk - dco);
        st.a[j][t] = cat8(bl16<kNT>(L.rd, sel(ok0, o)), bl16<kNT>(L.rd, sel(ok1, o + 64)));
      }
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const uint32_t o = xrow[c] + kk;
        st.b[j][c] = cat8(bl16<0>(L.rx, sel(ok0 && xok[c], o)), bl16<0>(L.rx, sel(ok1 && xok[c], o + 64)));
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
// measured slower on MI355X for this access pattern.  Whole stages run unmasked with
// wave-uniform offsets; the last, partial stage masks lanes past kend.
template <typename Stage, typename LoadFull, typename LoadTail, int RT, int CT>
__device__ __forceinline__ void run_stages(v4f (&acc)[RT][CT], int k0, int kend, int step, LoadFull full,
                                           LoadTail tail) {
  int k = k0;
  for (; k + step <= kend; k += step) {
    Stage st;
    full(st, k);
    mma_stage(acc, st);
  }
  if (k < kend) {
    Stage st;
    tail(st, k);
    xdl_fence();
    mma_stage(acc, st);
  }
  xdl_fence();
}

// ---------------------------------------------------------------- epilogue
__device__ __forceinline__ uint32_t bf16_bits(float v) {
  __bf16 h = (__bf16)v;  // round to nearest even
  return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

// Epilogue of 4 consecutive output rows n0.. of token m: (acc * w_scale[n]) * x_scale[m],
// bf16 (round to nearest even) or fp32, one vector store where allowed.
// Y[m, n0 + r] = v[r] for r < 4 (rows before rowend), bf16 RNE or fp32 per a.out_f32.
__device__ __forceinline__ void put4(void* Y, int64_t ldy, int vec_store, const GemmArgs& a, const float (&v)[4], int m,
                                     int n0, int rowend) {
  if (a.out_f32) {
    float* yp = reinterpret_cast<float*>(Y) + (int64_t)m * ldy + n0;
    if (vec_store && n0 + 3 < rowend) {
      *reinterpret_cast<v4f*>(yp) = (v4f){v[0], v[1], v[2], v[3]};
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (n0 + r < rowend) yp[r] = v[r];
    }
  } else {
    uint16_t* yp = reinterpret_cast<uint16_t*>(Y) + (int64_t)m * ldy + n0;
    const uint32_t b0 = bf16_bits(v[0]), b1 = bf16_bits(v[1]), b2 = bf16_bits(v[2]), b3 = bf16_bits(v[3]);
    if (vec_store && n0 + 3 < rowend) {
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

// The epilogue of one output quad: Y[m, n0 + r] = (acc[r] * w_scale[n]) * x_scale[m]
// (each factor only where given), fp32, then put4.
__device__ __forceinline__ void store4(void* Y, int64_t ldy, const float* sw, int vec_store, const GemmArgs& a,
                                       v4f acc, int m, int n0, int rowend) {
  const float xs = a.sx ? a.sx[m] : 1.0f;
  float v[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int n = n0 + r < rowend ? n0 + r : rowend - 1;
    float y = acc[r];
    if (sw) y = y * sw[n];
    v[r] = y * xs;
  }
  put4(Y, ldy, vec_store, a, v, m, n0, rowend);
}

// The scales of one wave's RT x CT output quads (rows n0 + 16 t + [0, 4), token m0 +
// 16 c), loaded together before any output store: read next to each store, a scale load
// would follow stores that may alias it and wait for their acknowledgement, one memory
// round trip per quad.  Rows past the region and tokens past M read the last valid one
// (their stores are skipped); a missing scale reads as 1.
template <int RT, int CT>
struct EpiScales {
  float w[RT][4];
  float x[CT];
};

template <int RT, int CT>
__device__ __forceinline__ void epi_scales(EpiScales<RT, CT>& e, const float* sw, const float* sx, int M, int n0, int m0,
                                           int rowend) {
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) e.w[t][r] = sw ? sw[min(n0 + 16 * t + r, rowend - 1)] : 1.0f;
#pragma unroll
  for (int c = 0; c < CT; ++c) e.x[c] = sx ? sx[min(m0 + 16 * c, M - 1)] : 1.0f;
}

// store4 of quad (t, c) with its scales from epi_scales: the same arithmetic, bit for bit.
template <int RT, int CT>
__device__ __forceinline__ void store4e(void* Y, int64_t ldy, bool wscaled, int vec_store, const GemmArgs& a,
                                        const EpiScales<RT, CT>& e, int t, int c, v4f acc, int m, int n0, int rowend) {
  float v[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float y = acc[r];
    if (wscaled) y = y * e.w[t][r];
    v[r] = y * e.x[c];
  }
  put4(Y, ldy, vec_store, a, v, m, n0, rowend);
}

__device__ __forceinline__ void store4(const GemmArgs& a, v4f acc, int m, int n0, int rowend) {
  store4(a.Y, a.ldy, a.sw, a.vec_store, a, acc, m, n0, rowend);
}

// A large-M workgroup's bf16 output tile through LDS, so that it leaves as whole token
// rows: stored straight from the accumulators, each instruction would write 16 token rows
// 32 bytes apiece, four times the write requests of whole rows (measured on the 256 x 256
// kernel: about 9 us of store issue per tile against 2).  Token row r of the tile (NB
// 16-byte blocks of eight outputs) sits at byte r * 16 NB, its block b stored at block
// b ^ (r % NB), so that neither the quad writes nor the row reads meet in a bank.
// out_tile_write: a wave's RT x CT quads (rows 16 (RT wr + t) + 4 lq + [0, 4) of the tile,
// token 16 (CT wc + c) + li), scaled and rounded as store4e does.
template <int RT, int CT, int NB>
__device__ __forceinline__ void out_tile_write(uint8_t* ot, const v4f (&acc)[RT][CT], const EpiScales<RT, CT>& es,
                                               bool wscaled, int wr, int wc, int li, int lq) {
  typedef uint32_t u2 __attribute__((ext_vector_type(2)));
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float y = acc[t][c][r];
        if (wscaled) y = y * es.w[t][r];
        v[r] = y * es.x[c];
      }
      const int r = 16 * (CT * wc + c) + li, n = 16 * (RT * wr + t) + 4 * lq;
      *reinterpret_cast<u2*>(ot + r * (16 * NB) + (((n >> 3) ^ (r % NB)) << 4) + (n & 7) * 2) =
          (u2){bf16_bits(v[0]) | (bf16_bits(v[1]) << 16), bf16_bits(v[2]) | (bf16_bits(v[3]) << 16)};
    }
}

// out_tile_store: the tile's first ntok token rows to Y (tile row 0 = output row rblk,
// token 0 = m0), 16 bytes per thread; Y 16-byte aligned, ldy and rblk multiples of 8.
template <int NB, int NTHR>
__device__ __forceinline__ void out_tile_store(const uint8_t* ot, int ntok, int m0, int M, int rblk, int rowend, void* Y,
                                               int64_t ldy) {
  for (int q = threadIdx.x; q < ntok * NB; q += NTHR) {
    const int r = q / NB, b = q % NB;
    const int m = m0 + r, n = rblk + 8 * b;
    if (m >= M || n >= rowend) continue;
    const v4i d = *reinterpret_cast<const v4i*>(ot + r * (16 * NB) + ((b ^ (r % NB)) << 4));
    uint16_t* yp = reinterpret_cast<uint16_t*>(Y) + (int64_t)m * ldy + n;
    if (n + 8 <= rowend) {
      *reinterpret_cast<v4i*>(yp) = d;
    } else {
      for (int e = 0; e < rowend - n; ++e) yp[e] = (uint16_t)((uint32_t)d[e >> 1] >> (16 * (e & 1)));
    }
  }
}

// ---------------------------------------------------------------- kernel
template <int DT, int CT, int RT, int W, int U, bool WM>
__global__ __launch_bounds__(64 * W) void spense_gemm_kernel(GemmArgs a) {
  typedef Traits<DT> T;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
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
    // the lane group's offset inside a step (16 bytes per group for every kind of step)
    // is added per region below
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
    run_stages<SparseStage<DT, CT, RT, U>>(
        acc, ka, ks_end, U * T::KS,
        [&](SparseStage<DT, CT, RT, U>& st, int k) {
          load_sparse<DT, CT, RT, U, WM, true>(st, L, vrow, mrow, xr, xok, k, ks_end);
        },
        [&](SparseStage<DT, CT, RT, U>& st, int k) {
          load_sparse<DT, CT, RT, U, WM, false>(st, L, vrow, mrow, xr, xok, k, ks_end);
        });
  }
  if (kd_beg < kb) {
    uint32_t drow[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      const int n = min(nbase + 16 * t + li, rowend - 1);
      drow[t] = (uint32_t)((int64_t)(n - R.dense_row_off) * a.d_ld_b) + 16u * lq;
    }
    uint32_t xr[CT];
#pragma unroll
    for (int c = 0; c < CT; ++c) xr[c] = xrow[c] + 16u * lq;
    const int dco = R.dense_col_off;
    run_stages<DenseStage<DT, CT, RT, U>>(
        acc, kd_beg, kb, U * T::KD,
        [&](DenseStage<DT, CT, RT, U>& st, int k) { load_dense<DT, CT, RT, U, true>(st, L, drow, xr, xok, k, kb, dco); },
        [&](DenseStage<DT, CT, RT, U>& st, int k) {
          load_dense<DT, CT, RT, U, false>(st, L, drow, xr, xok, k, kb, dco);
        });
  }

  // ---- add the waves' partial sums in LDS (wave order), then the epilogue; one
  // activation tile at a time keeps the buffer at W * RT KB
  __shared__ v4f red[W * RT * 64];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    if (c) __syncthreads();  // the previous tile's reads are done
#pragma unroll
    for (int t = 0; t < RT; ++t) red[(wave * RT + t) * 64 + lane] = acc[t][c];
    __syncthreads();
    for (int e = threadIdx.x; e < RT * 64; e += 64 * W) {
      const int ln = e & 63, t = e >> 6;
      v4f s = red[e];
#pragma unroll
      for (int w = 1; w < W; ++w) s += red[w * RT * 64 + e];
      const int m = m0 + 16 * c + (ln & 15);
      const int n0 = nbase + 16 * t + 4 * (ln >> 4);
      if (m < a.M && n0 < rowend) store4(a, s, m, n0, rowend);
    }
  }
}

// ---------------------------------------------------------------- row-split kernel
// For several activation tiles the activations are the reused operand.  Here each of the
// first `wused` waves of a workgroup owns 16 weight rows and all of K; the waves walk K
// together in chunks of four instruction steps.  Each chunk of activations (16*CT rows)
// is copied once per workgroup from global memory straight into LDS (buffer loads with
// an LDS destination; 16-byte blocks XOR-swizzled by row so the fragment reads are
// conflict-free; two buffers), and every wave reads its B fragments from there.  The
// weights are requested D chunks ahead into registers; the barrier that publishes the
// next activation chunk waits only for the activation loads, so the weight loads stay
// in flight across it.  No wave splits K: the epilogue stores from the accumulators.
template <int DT, int CT>
struct XTile {
  static constexpr int KS = Traits<DT>::KS;
  static constexpr int CHUNK_K = 4 * KS;                  // logical K per chunk
  static constexpr int ROW_B = CHUNK_K * Traits<DT>::ES;  // bytes per activation row (512)
  static constexpr int ROWS = 16 * CT;
  static constexpr int BYTES = ROWS * ROW_B;
  // LDS byte address of 16-byte block b of row r
  __device__ static __forceinline__ int addr(int r, int b) { return r * ROW_B + ((b ^ (r & 31)) << 4); }
};

template <int DT, int CT>
__device__ __forceinline__ v4i xlds(const uint8_t* lds, int r, int byte) {
  return *reinterpret_cast<const v4i*>(lds + XTile<DT, CT>::addr(r, byte >> 4) + (byte & 15));
}

// B fragments of one step from the LDS tile (step_b: byte offset of the step in a row).
// 2:4 steps and dense fp8 steps read K [16q, 16q+16) and [64+16q, 64+16q+16) of the
// step; dense bf16 steps read K [8q, 8q+8).
template <int DT, int CT>
__device__ __forceinline__ void frag_pair(v8i (&b)[CT], const uint8_t* lds, int li, int lq, int step_b) {
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const int r = 16 * c + li;
    b[c] = cat8(xlds<DT, CT>(lds, r, step_b + 16 * lq), xlds<DT, CT>(lds, r, step_b + 64 + 16 * lq));
  }
}
template <int DT, int CT>
__device__ __forceinline__ void frag_one(v8i (&b)[CT], const uint8_t* lds, int li, int lq, int step_b) {
  const v4i z = {0, 0, 0, 0};
#pragma unroll
  for (int c = 0; c < CT; ++c) b[c] = cat8(xlds<DT, CT>(lds, 16 * c + li, step_b + 16 * lq), z);
}

// Copy activations [m0, m0+16CT) x [kc, kc+CHUNK_K) into an LDS tile: each wave fills XI
// consecutive 1 KB blocks (lane l writes bytes 16l..16l+15 of its block; the source
// address applies the swizzle).  Rows past M and columns past kend are written as zeros.
template <int DT, int CT, int XI>
__device__ __forceinline__ void x_to_lds(uint8_t* lds, const GemmArgs& a, __amdgpu_buffer_rsrc_t rx, int m0, int kc,
                                         int kend, int wave, int lane) {
  typedef XTile<DT, CT> XT;
#pragma unroll
  for (int i = 0; i < XI; ++i) {
    const int blk = wave * XI + i;                           // 1 KB block of the tile
    const int r = (blk * 1024 + 16 * lane) / XT::ROW_B;      // tile row
    const int pb = ((blk * 1024 + 16 * lane) % XT::ROW_B) >> 4;  // physical 16-byte slot
    const int b = pb ^ (r & 31);                             // logical block stored there
    const int kcol = kc + b * 16 / Traits<DT>::ES;
    const int m = m0 + r;
    const uint32_t off = sel(m < a.M && kcol < kend, (uint32_t)((int64_t)m * a.ldx_b + (int64_t)kcol * Traits<DT>::ES));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (__attribute__((address_space(3))) void*)(lds + blk * 1024), 16, off,
                                             0, 0, 0);
  }
}

// Weights of one chunk in registers: eight 16-byte fragments and four metadata words.
// fp8 (both kinds of chunk have four 128-wide steps): w[j] is step j's 2:4 value fragment
// or the first half of its dense fragment, w[4+j] the dense second half.  bf16: w[j] is
// step j's value fragment (2:4, j < 4) or dense fragment (eight 32-wide steps).
struct WChunk {
  v4i w[8];
  int ix[4];
};

// Load instructions one chunk issues; the same for 2:4 and dense chunks (the unused ones
// get out-of-range offsets), so the loads need no branches and the compiler keeps the
// fragments in place while they are in flight.
template <bool WM>
struct ChunkLoads {
  static constexpr int N = 8 + (WM ? 1 : 4);
};

// ok = false masks every lane (past the last chunk, or a wave that owns no rows).
template <int DT, bool WM>
__device__ __forceinline__ void load_chunk(WChunk& W, bool sparse, bool ok, int kc, int ke, int lq, uint32_t vrow,
                                           uint32_t mrow, uint32_t drow, int dco, __amdgpu_buffer_rsrc_t rv,
                                           __amdgpu_buffer_rsrc_t rm, __amdgpu_buffer_rsrc_t rd) {
  const __amdgpu_buffer_rsrc_t rw = sparse ? rv : rd;
  if constexpr (DT == kFP8) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int kk = kc + 128 * j;
      // 2:4: 16 kept values of logical K [kk+32q, kk+32q+32); dense: K [kk+16q, +16) and
      // [kk+64+16q, +16)
      const bool oka = ok && kk + (sparse ? 32 : 16) * lq < ke;
      const bool okb = ok && !sparse && kk + 64 + 16 * lq < ke;
      const uint32_t oa = sparse ? vrow + (uint32_t)(kk >> 1) : drow + (uint32_t)(kk - dco);
      W.w[j] = bl16<kNT>(rw, sel(oka, oa));
      W.w[4 + j] = bl16<kNT>(rd, sel(okb, oa + 64));
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int kk = kc + (sparse ? 64 : 32) * j;
      const bool okj = ok && (!sparse || j < 4) && kk + (sparse ? 16 : 8) * lq < ke;
      const uint32_t o = sparse ? vrow + (uint32_t)kk : drow + 2 * (uint32_t)(kk - dco);
      W.w[j] = bl16<kNT>(rw, sel(okj, o));
    }
  }
  if constexpr (WM) {
    // lane group q loads step q's four words (16 bytes of the row); they are transposed
    // when the chunk is consumed (meta_words), not here, so the load stays in flight
    const v4i w = bl16<kNT>(rm, sel(ok && sparse && kc + 128 * lq < ke, mrow + 4 * (kc >> 5) + 12 * lq));
#pragma unroll
    for (int j = 0; j < 4; ++j) W.ix[j] = w[j];
  } else {
    constexpr int KS = Traits<DT>::KS;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int kk = kc + j * KS;
      W.ix[j] = bl4<kNT>(rm, sel(ok && sparse && kk + (DT == kFP8 ? 32 : 16) * lq < ke, mrow + 4 * (kk >> 5)));
    }
  }
}

// Tiled layout (fp8): each fragment of the chunk is one contiguous kilobyte.  vt, mt, dt:
// this lane's byte offset in its tile's first 2:4 / metadata / dense chunk (16 * lane
// included); cs, cd >= 0: the chunk's index within the 2:4 / dense part.  The chunk part
// of the address travels in the scalar offset; ok = false masks every lane.
__device__ __forceinline__ void load_chunk_tiled(WChunk& W, bool sparse, bool ok, int cs, int cd, uint32_t vt,
                                                 uint32_t mt, uint32_t dt, __amdgpu_buffer_rsrc_t rv,
                                                 __amdgpu_buffer_rsrc_t rm, __amdgpu_buffer_rsrc_t rd) {
  const __amdgpu_buffer_rsrc_t rw = sparse ? rv : rd;
  const uint32_t base = sel(ok, sparse ? vt : dt);
  const uint32_t dbase = sel(ok && !sparse, dt);
  const int s0 = sparse ? cs * 4096 : cd * 8192, sj = sparse ? 1024 : 2048;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    W.w[j] = bl16<kTiledNT>(rw, base, s0 + sj * j);
    W.w[4 + j] = bl16<kTiledNT>(rd, dbase, cd * 8192 + 2048 * j + 1024);
  }
  const v4i w = bl16<kTiledNT>(rm, sel(ok && sparse, mt), cs * 1024);
#pragma unroll
  for (int j = 0; j < 4; ++j) W.ix[j] = w[j];
}

// The metadata word of each step for this lane group.  Wide loads: lane group q holds
// step q's four words; a 4x4 transpose across lane groups (two lane swaps) gives lane
// group q word 4j+q of every step j.
template <bool WM>
__device__ __forceinline__ void meta_words(int (&ix)[4], const WChunk& W) {
  if constexpr (WM) {
    const auto s02 = __builtin_amdgcn_permlane32_swap((unsigned)W.ix[0], (unsigned)W.ix[2], false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap((unsigned)W.ix[1], (unsigned)W.ix[3], false, false);
    const auto s01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
    const auto s23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
    ix[0] = (int)s01[0];
    ix[1] = (int)s01[1];
    ix[2] = (int)s23[0];
    ix[3] = (int)s23[1];
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) ix[j] = W.ix[j];
  }
}

// MMAs of one chunk.  The B fragments of P steps are read from LDS before their MMAs,
// so the LDS latency is paid once per group rather than once per step.
template <int DT, int CT, int RT, bool WM, int P>
__device__ __forceinline__ void mma_chunk(v4f (&acc)[RT][CT], const WChunk (&W)[RT], bool sparse, const uint8_t* lds,
                                          int li, int lq) {
  static_assert(P == 1 || P == 2 || P == 4, "fragment group size");
  // each B fragment read from LDS feeds the RT row tiles of this wave
  if (sparse) {
    int mw[RT][4];
#pragma unroll
    for (int t = 0; t < RT; ++t) meta_words<WM>(mw[t], W[t]);
#pragma unroll
    for (int j0 = 0; j0 < 4; j0 += P) {
      v8i b[P][CT];
#pragma unroll
      for (int j = 0; j < P; ++j) frag_pair<DT, CT>(b[j], lds, li, lq, (j0 + j) * 128);
      if constexpr (P > 1) __builtin_amdgcn_sched_barrier(0);  // all reads of the group before its MMAs
#pragma unroll
      for (int j = 0; j < P; ++j)
#pragma unroll
        for (int t = 0; t < RT; ++t) {
          const int ix = DT == kFP8 ? mw[t][j0 + j] : (int)((uint32_t)mw[t][j0 + j] >> (16 * (lq & 1)));
#pragma unroll
          for (int c = 0; c < CT; ++c)
            acc[t][c] = mma_sparse(W[t].w[j0 + j], b[j][c], acc[t][c], ix, std::integral_constant<int, DT>());
        }
    }
  } else if constexpr (DT == kFP8) {
#pragma unroll
    for (int j0 = 0; j0 < 4; j0 += P) {
      v8i b[P][CT];
#pragma unroll
      for (int j = 0; j < P; ++j) frag_pair<DT, CT>(b[j], lds, li, lq, (j0 + j) * 128);
      if constexpr (P > 1) __builtin_amdgcn_sched_barrier(0);  // all reads of the group before its MMAs
#pragma unroll
      for (int j = 0; j < P; ++j)
#pragma unroll
        for (int t = 0; t < RT; ++t) {
          const v8i av = cat8(W[t].w[j0 + j], W[t].w[4 + j0 + j]);
#pragma unroll
          for (int c = 0; c < CT; ++c) acc[t][c] = mma_dense(av, b[j][c], acc[t][c], std::integral_constant<int, DT>());
        }
    }
  } else {
    const v4i z = {0, 0, 0, 0};
#pragma unroll
    for (int j0 = 0; j0 < 8; j0 += 2 * P) {
      v8i b[2 * P][CT];
#pragma unroll
      for (int j = 0; j < 2 * P; ++j) frag_one<DT, CT>(b[j], lds, li, lq, (j0 + j) * 64);
      if constexpr (P > 1) __builtin_amdgcn_sched_barrier(0);  // all reads of the group before its MMAs
#pragma unroll
      for (int j = 0; j < 2 * P; ++j)
#pragma unroll
        for (int t = 0; t < RT; ++t) {
          const v8i av = cat8(W[t].w[j0 + j], z);
#pragma unroll
          for (int c = 0; c < CT; ++c) acc[t][c] = mma_dense(av, b[j][c], acc[t][c], std::integral_constant<int, DT>());
        }
    }
  }
}

// Workgroup barrier that first waits until at most N of this wave's vector-memory
// operations are outstanding (loads complete in issue order, so every older one is
// done).  The wait is the builtin, which the compiler's own wait insertion takes into
// account; the barrier's memory clobber keeps LDS accesses from moving across it.
template <int N>
__device__ __forceinline__ void barrier_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // s_waitcnt fields: vmcnt[3:0] and [15:14], expcnt [6:4] and lgkmcnt [11:8] left at max
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
  asm volatile("s_barrier" ::: "memory");
}

// As barrier_vm, and also wait for this wave's LDS accesses (lgkmcnt(0)).
template <int N>
__device__ __forceinline__ void barrier_vm_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (0 << 8));
  asm volatile("s_barrier" ::: "memory");
}

// Pipeline with NS register slots and NS LDS buffers, D = NS-1 chunks ahead (per wave,
// in issue order within chunk step c): activations of chunk c+D -> LDS buffer
// (c+D) % NS, weights of chunk c+D -> register slot (c+D) % NS, MMAs of chunk c (buffer
// and slot c % NS), then a barrier that waits for the activations of chunk c+1 (issued
// in step c+1-D, before that step's weights), so D chunks of weights stay in flight
// across it.  The buffer being filled held chunk c-1, which every wave has finished.
//
// XR (one or two token tiles): the activations of every chunk of the workgroup's K range
// are copied into dynamic LDS once, behind one barrier, and each wave then streams its
// weights with no further barrier, as far ahead as its register slots allow.
template <int DT, int CT, int RT, int WR, bool WM, int NS, int P, bool TL, int GM, bool XR = false>
__global__ __launch_bounds__(64 * WR) void spense_gemm_rows_kernel(GemmArgs a) {
  constexpr bool GR = GM == 1;   // grouped launch
  constexpr bool GLU = GM == 2;  // gate and up paired, the GLU step in the epilogue
  static_assert(!GLU || (RT == 1 && WR == 8), "paired gate / up: four waves per weight");
  static_assert(NS == 3 || NS == 4, "three or four pipeline slots");
  static_assert(!TL || (DT == kFP8 && WM), "the tiled layout is fp8 with whole-chunk metadata loads");
  static_assert(!XR || (CT <= 2 && GM <= 1), "resident activations: one or two token tiles, plain or grouped launch");
  constexpr int D = NS - 1;
  typedef XTile<DT, CT> XT;
  constexpr int KC = XT::CHUNK_K;
  constexpr int XI = XT::BYTES / 1024 / WR;  // 1 KB activation blocks per wave per chunk
  static_assert(XI >= 1 && XI * 1024 * WR == XT::BYTES, "activation tile must split evenly");
  constexpr int NL = ChunkLoads<WM>::N;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int li = lane & 15, lq = lane >> 4;
  int g = blockIdx.x, mb = blockIdx.y;
  if (a.rorder == 2) {  // XCD x (= id % 8) runs the token blocks of row groups x, x + 8, ...
    const int x = (int)blockIdx.x & 7, l = (int)blockIdx.x >> 3;
    g = (l / a.mblk) * 8 + x;
    mb = l % a.mblk;
  } else if (a.rorder == 1) {
    g = (int)blockIdx.x / a.mblk;
    mb = (int)blockIdx.x % a.mblk;
  }
  // GR (grouped launch): up to kMaxRegions regions in workgroup order, each of one weight
  // (its buffers, output and scales in a.mat); otherwise one weight (GLU: two weights,
  // gate and up, of equal geometry), up to two regions, buffers in a or a.mat (GLU).
  int ri = 0;
  if constexpr (GR) {
    for (int i = 1; i < a.nreg; ++i)
      if (g >= a.reg[i].wg0) ri = i;
  } else {
    ri = (a.nreg > 1 && g >= a.reg[1].wg0) ? 1 : 0;
  }
  const Region& R = a.reg[ri];
  // GLU: waves 0-3 own gate tiles, waves 4-7 the up tiles of the same rows
  const int wsel = GLU ? (wave & 3) : wave;
  const MatDesc& MD = a.mat[GR ? R.mat : (GLU ? wave >> 2 : 0)];
  const int rowend = R.row0 + R.rows;
  // workgroups of a region: (row group, K slice), slices of one row group adjacent
  const int slice = (g - R.wg0) % R.ksplit, rgroup = (g - R.wg0) / R.ksplit;
  const int nbase = R.row0 + (rgroup * R.wused + wsel) * 16 * RT;  // first row of the wave's RT tiles
  const int m0 = mb * 16 * CT;
  const int K = R.kend;
  const int kbound = R.kbound;
  const bool active = wsel < R.wused && nbase < rowend;

  __shared__ __attribute__((aligned(1024))) uint8_t xbuf[NS][XT::BYTES];
  extern __shared__ __attribute__((aligned(1024))) uint8_t xres[];  // XR: chunk c at (c - c_lo) * XT::BYTES
  constexpr bool FROM_MAT = GR || GLU;
  const __amdgpu_buffer_rsrc_t rx = rsrc(a.X, a.x_bytes),
                               rv = FROM_MAT ? rsrc(MD.values, MD.v_bytes) : rsrc(a.values, a.v_bytes),
                               rm = FROM_MAT ? rsrc(MD.meta, MD.m_bytes) : rsrc(a.meta, a.m_bytes),
                               rd = FROM_MAT ? rsrc(MD.dense, MD.d_bytes) : rsrc(a.dense, a.d_bytes);

  v4f acc[RT][CT];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int c = 0; c < CT; ++c) acc[t][c] = (v4f){0.f, 0.f, 0.f, 0.f};

  bool tok[RT];  // tile t of this wave holds rows of the region
  uint32_t vrow[RT], mrow[RT], drow[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    tok[t] = nbase + 16 * t < rowend;
    const int n = min(nbase + 16 * t + li, rowend - 1);
    vrow[t] = (uint32_t)((int64_t)n * a.v_ld_b) + 16u * lq;
    mrow[t] = (uint32_t)((int64_t)n * a.m_ld_b) + (DT == kFP8 ? 4u * lq : 4u * (lq >> 1));
    drow[t] = (uint32_t)((int64_t)max(n - R.dense_row_off, 0) * a.d_ld_b) + 16u * lq;
  }

  // chunk list: 2:4 chunks start at 0 and cover [0, kbound); dense chunks start at kbound;
  // this workgroup's K slice is chunks [c_lo, c_hi)
  const int n_sp = (kbound + KC - 1) / KC;
  const int n_de = (K - kbound + KC - 1) / KC;
  const int c_lo = R.cut[slice], c_hi = R.cut[slice + 1];
  auto chunk_k = [&](int c) { return c < n_sp ? c * KC : kbound + (c - n_sp) * KC; };
  auto chunk_end = [&](int c) { return c < n_sp ? kbound : K; };
  // tiled layout: offsets of this lane in its tiles' first chunk of each part
  uint32_t vt[RT], mt[RT], dt[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    vt[t] = mt[t] = dt[t] = 0;
    if constexpr (TL) {
      const uint32_t ts = (uint32_t)(nbase / 16 + t), td = (uint32_t)((nbase - R.dense_row_off) / 16 + t);
      vt[t] = ts * (uint32_t)n_sp * 4096u + 16u * lane;
      mt[t] = ts * (uint32_t)n_sp * 1024u + 16u * lane;
      dt[t] = td * (uint32_t)n_de * 8192u + 16u * lane;
    }
  }
  auto load = [&](WChunk (&W)[RT], int c) {
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      if constexpr (TL)
        load_chunk_tiled(W[t], c < n_sp, tok[t] && c < c_hi, c, max(c - n_sp, 0), vt[t], mt[t], dt[t], rv, rm, rd);
      else
        load_chunk<DT, WM>(W[t], c < n_sp, tok[t] && c < c_hi, chunk_k(c), chunk_end(c), lq, vrow[t], mrow[t],
                           drow[t], R.dense_col_off, rv, rm, rd);
    }
  };
  auto xload = [&](int buf, int c) {
    x_to_lds<DT, CT, XI>(xbuf[buf], a, rx, m0, chunk_k(c), c < c_hi ? chunk_end(c) : -1, wave, lane);
  };
  auto xtile = [&](int s, int c) -> const uint8_t* {
    if constexpr (XR)
      return xres + (c - c_lo) * XT::BYTES;
    else
      return xbuf[s];
  };

  // A wave that owns rows loads weights and runs the MMAs; the others only stage
  // activations and take part in the barriers.  The two loops are separate so that no
  // path leaves a weight load pending where the compiler would have to wait for it.
  auto run = [&](auto act_const) {
    constexpr bool ACT = decltype(act_const)::value;
    // loads issued after the activations of chunk c+1, at the barrier of chunk c: that
    // step's weights, then D-1 further steps of activations and weights
    constexpr int AFTER = ACT ? RT * NL + (D - 1) * (XI + RT * NL) : (D - 1) * XI;
    WChunk slot[NS][RT];
    if constexpr (XR) {
      // every chunk's activations, then the first D chunks of weights; the barrier waits
      // for the activations only (loads complete in issue order)
      for (int c = c_lo; c < c_hi; ++c)
        x_to_lds<DT, CT, XI>(xres + (c - c_lo) * XT::BYTES, a, rx, m0, chunk_k(c), chunk_end(c), wave, lane);
      if constexpr (ACT) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
          __builtin_amdgcn_sched_barrier(0);  // each chunk's weights before the next chunk's
          load(slot[d], c_lo + d);
        }
      }
      barrier_vm<ACT ? D * RT * NL : 0>();
      if constexpr (!ACT) return;
    } else {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        xload(d, c_lo + d);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (ACT) load(slot[d], c_lo + d);
        __builtin_amdgcn_sched_barrier(0);
      }
      // the first chunk's activations only: the loads issued after them (D chunks of
      // weights, D - 1 of activations, in this order: the scheduling barriers keep a
      // chunk's weight loads from sinking below the next chunk's) stay in flight while the
      // next ones are requested
      barrier_vm<AFTER>();
    }
    auto step = [&](auto s_const, int c) {
      constexpr int S = decltype(s_const)::value;
      constexpr int SD = (S + D) % NS;
      if constexpr (!XR) {
        xload(SD, c + D);
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (ACT) {
        load(slot[SD], c + D);
        __builtin_amdgcn_sched_barrier(0);
        mma_chunk<DT, CT, RT, WM, P>(acc, slot[S], c < n_sp, xtile(S, c), li, lq);
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (!XR) barrier_vm<AFTER>();
    };
    int c = c_lo;
    for (; c + NS <= c_hi; c += NS) {
      step(std::integral_constant<int, 0>(), c);
      step(std::integral_constant<int, 1>(), c + 1);
      step(std::integral_constant<int, 2>(), c + 2);
      if constexpr (NS == 4) step(std::integral_constant<int, 3 % NS>(), c + 3);
    }
    if (c < c_hi) step(std::integral_constant<int, 0>(), c);
    if (c + 1 < c_hi) step(std::integral_constant<int, 1>(), c + 1);
    if constexpr (NS == 4)
      if (c + 2 < c_hi) step(std::integral_constant<int, 2>(), c + 2);
  };
  // the epilogue's scales, requested before any weight or activation so that they have
  // long arrived when the stores begin (K slices write unscaled partials and need none)
  EpiScales<RT, CT> es, eu;  // GLU: gate scales and token scales in es, up scales in eu
  if constexpr (GLU) {
    if (wave >= 4 && active) {
      epi_scales(es, a.mat[0].sw, a.sx, a.M, nbase + 4 * lq, m0 + li, rowend);
      epi_scales(eu, a.mat[1].sw, nullptr, a.M, nbase + 4 * lq, m0 + li, rowend);
    }
  } else {
    if (active && R.ksplit == 1) epi_scales(es, MD.sw, a.sx, a.M, nbase + 4 * lq, m0 + li, rowend);
  }
  if (active)
    run(std::true_type());
  else
    run(std::false_type());

  if constexpr (GLU) {
    // h = glu(g, u) with g, u each scaled as the plain epilogue scales them: the gate waves
    // pass their accumulators through the (now idle) staging buffers to the up waves of
    // the same rows, which write H (fp32).  Every wave takes both barriers.
    xdl_fence();
    barrier_vm<0>();  // all staging loads of every wave have landed
    static_assert(XT::BYTES >= 4 * CT * 64 * 16, "gate accumulators fit one staging buffer");
    float* ex = reinterpret_cast<float*>(&xbuf[0][0]);
    if (wave < 4 && active) {
#pragma unroll
      for (int cc = 0; cc < CT; ++cc) *reinterpret_cast<v4f*>(ex + ((wsel * CT + cc) * 64 + lane) * 4) = acc[0][cc];
    }
    barrier_vm_lgkm0<63>();
    float tmax[CT];  // per token: the maximum of |h| over this lane's stored rows
#pragma unroll
    for (int cc = 0; cc < CT; ++cc) tmax[cc] = 0.0f;
    if (wave >= 4 && active) {
      const MatDesc& G = a.mat[0];
      const MatDesc& Up = a.mat[1];
#pragma unroll
      for (int cc = 0; cc < CT; ++cc) {
        const int m = m0 + 16 * cc + li;
        const int n0 = nbase + 4 * lq;
        if (m >= a.M || n0 >= rowend) continue;
        const v4f gv = *reinterpret_cast<const v4f*>(ex + ((wsel * CT + cc) * 64 + lane) * 4);
        const float xs = es.x[cc];
        float h[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float gg = gv[r], uu = acc[0][cc][r];
          if (G.sw) gg = gg * es.w[0][r];
          if (Up.sw) uu = uu * eu.w[0][r];
          h[r] = glu_silu(gg * xs, uu * xs);
          if (n0 + r < rowend) tmax[cc] = fmaxf(tmax[cc], fabsf(h[r]));
        }
        float* hp = reinterpret_cast<float*>(G.Y) + (int64_t)m * G.ldy + n0;
        if (G.vec_store && n0 + 3 < rowend) {
          *reinterpret_cast<v4f*>(hp) = (v4f){h[0], h[1], h[2], h[3]};
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (n0 + r < rowend) hp[r] = h[r];
        }
      }
    }
    if (a.hmax) {
      // per token, the maximum over the workgroup's rows: the four row groups of a lane
      // column (lanes li, li + 16, li + 32, li + 48), then the four up waves through LDS
      float* red = reinterpret_cast<float*>(&xbuf[1][0]);
      if (wave >= 4) {
#pragma unroll
        for (int cc = 0; cc < CT; ++cc) {
          float v = fmaxf(tmax[cc], __shfl_xor(tmax[cc], 16, 64));
          v = fmaxf(v, __shfl_xor(v, 32, 64));
          if (lq == 0) red[wsel * 16 * CT + 16 * cc + li] = v;
        }
      }
      barrier_vm_lgkm0<63>();
      if (wave == 4 && lane < 16 * CT) {
        const int m = m0 + lane;
        const float v = fmaxf(fmaxf(red[lane], red[16 * CT + lane]), fmaxf(red[32 * CT + lane], red[48 * CT + lane]));
        if (m < a.M) a.hmax[(int64_t)m * a.groups + g] = v;
      }
    }
    return;
  }
  if (!active) return;
  xdl_fence();
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int cc = 0; cc < CT; ++cc) {
      const int m = m0 + 16 * cc + li;
      const int n0 = nbase + 16 * t + 4 * lq;
      if (m >= a.M || n0 >= rowend) continue;
      if (R.ksplit == 1) {
        store4e(MD.Y, MD.ldy, MD.sw != nullptr, MD.vec_store, a, es, t, cc, acc[t][cc], m, n0, rowend);
      } else {  // unscaled fp32 partial of this K slice, one 16-byte store where it can
        float* pp = a.part + ((int64_t)slice * a.M + m) * a.N + n0;
        if (n0 + 3 < rowend && a.N % 4 == 0 && (uintptr_t)a.part % 16 == 0) {
          *reinterpret_cast<v4f*>(pp) = acc[t][cc];
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (n0 + r < rowend) pp[r] = acc[t][cc][r];
        }
      }
    }
}

// Row-split kernel for two 64-token halves per workgroup (65-128 tokens per block): each
// wave's weights of a chunk, in registers, feed the MMAs of both halves, so a weight row
// is streamed once for up to 128 tokens instead of once per 64.  The activations of a
// chunk (both halves, 64 KB) take two LDS buffers: chunk c + 1 is copied during step c
// into the buffer chunk c - 1 left (every wave finished with it at the previous barrier),
// and the barrier at the end of step c waits for it; the weights run NS - 1 chunks ahead
// in NS register slots.  Plain launches of tiled fp8 weights, one row tile and eight
// waves per workgroup; with K slices (workgroups (row group, slice), slices of a row
// group adjacent) each writes its unscaled fp32 partial sums for the reduction launch.
template <int WR, int NS>
__global__ __launch_bounds__(64 * WR) void spense_gemm_rows2_kernel(GemmArgs a) {
  constexpr int DT = kFP8, CT = 4, RT = 1, D = NS - 1;
  static_assert(NS == 2 || NS == 3, "two or three weight slots");
  typedef XTile<DT, CT> XT;  // one 64-token half
  constexpr int KC = XT::CHUNK_K;
  constexpr int XI = XT::BYTES / 1024 / WR;  // 1 KB activation blocks per wave per half
  static_assert(XI >= 1 && XI * 1024 * WR == XT::BYTES, "activation tile must split evenly");
  constexpr int NL = ChunkLoads<true>::N;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int li = lane & 15, lq = lane >> 4;
  const int g = blockIdx.x;
  const int ri = (a.nreg > 1 && g >= a.reg[1].wg0) ? 1 : 0;
  const Region& R = a.reg[ri];
  const MatDesc& MD = a.mat[0];
  const int rowend = R.row0 + R.rows;
  const int slice = (g - R.wg0) % R.ksplit, rgroup = (g - R.wg0) / R.ksplit;
  const int nbase = R.row0 + (rgroup * R.wused + wave) * 16;
  const int m0 = blockIdx.y * 32 * CT;
  const int K = R.kend, kbound = R.kbound;
  const bool active = wave < R.wused && nbase < rowend;

  __shared__ __attribute__((aligned(1024))) uint8_t xbuf[2][2 * XT::BYTES];
  const __amdgpu_buffer_rsrc_t rx = rsrc(a.X, a.x_bytes), rv = rsrc(a.values, a.v_bytes),
                               rm = rsrc(a.meta, a.m_bytes), rd = rsrc(a.dense, a.d_bytes);
  v4f acc0[RT][CT], acc1[RT][CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) acc0[0][c] = acc1[0][c] = (v4f){0.f, 0.f, 0.f, 0.f};

  const int n_sp = (kbound + KC - 1) / KC, n_de = (K - kbound + KC - 1) / KC;
  const int c_lo = R.cut[slice], c_hi = R.cut[slice + 1];  // this workgroup's chunks
  auto chunk_k = [&](int c) { return c < n_sp ? c * KC : kbound + (c - n_sp) * KC; };
  auto chunk_end = [&](int c) { return c < n_sp ? kbound : K; };
  const bool tok = nbase < rowend;
  const uint32_t ts = (uint32_t)(nbase / 16), td = (uint32_t)((nbase - R.dense_row_off) / 16);
  const uint32_t vt = ts * (uint32_t)n_sp * 4096u + 16u * lane, mt = ts * (uint32_t)n_sp * 1024u + 16u * lane,
                 dt = td * (uint32_t)n_de * 8192u + 16u * lane;
  auto load = [&](WChunk& W, int c) {
    load_chunk_tiled(W, c < n_sp, tok && c < c_hi, c, max(c - n_sp, 0), vt, mt, dt, rv, rm, rd);
  };
  auto xload = [&](int c) {  // both halves of chunk c into buffer c % 2
    uint8_t* b = xbuf[c & 1];
    const int ke = c < c_hi ? chunk_end(c) : -1;
    x_to_lds<DT, CT, XI>(b, a, rx, m0, chunk_k(c), ke, wave, lane);
    x_to_lds<DT, CT, XI>(b + XT::BYTES, a, rx, m0 + 16 * CT, chunk_k(c), ke, wave, lane);
  };

  auto run = [&](auto act_const) {
    constexpr bool ACT = decltype(act_const)::value;
    WChunk slot[NS][RT];
    // the first chunk's activations, then D chunks of weights; the barrier waits for the
    // activations only (loads complete in issue order)
    xload(c_lo);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (ACT) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        load(slot[d][0], c_lo + d);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    barrier_vm<ACT ? D * NL : 0>();
    // step c: activations of chunk c + 1, weights of chunk c + 2, the MMAs of chunk c for
    // both halves, then a barrier that waits for chunk c + 1's activations (issued before
    // this step's weights, the only loads younger than them)
    auto step = [&](auto s_const, int c) {
      constexpr int S = decltype(s_const)::value;
      xload(c + 1);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (ACT) {
        load(slot[(S + D) % NS][0], c + D);
        __builtin_amdgcn_sched_barrier(0);
        const uint8_t* xb = xbuf[c & 1];
        mma_chunk<DT, CT, RT, true, 1>(acc0, slot[S], c < n_sp, xb, li, lq);
        mma_chunk<DT, CT, RT, true, 1>(acc1, slot[S], c < n_sp, xb + XT::BYTES, li, lq);
        __builtin_amdgcn_sched_barrier(0);
      }
      barrier_vm<ACT ? NL : 0>();
    };
    int c = c_lo;
    for (; c + NS <= c_hi; c += NS) {
      step(std::integral_constant<int, 0>(), c);
      step(std::integral_constant<int, 1>(), c + 1);
      if constexpr (NS == 3) step(std::integral_constant<int, 2 % NS>(), c + 2);
    }
    if (c < c_hi) step(std::integral_constant<int, 0>(), c);
    if constexpr (NS == 3)
      if (c + 1 < c_hi) step(std::integral_constant<int, 1>(), c + 1);
  };
  if (active)
    run(std::true_type());
  else
    run(std::false_type());
  if (!active) return;
  if (R.ksplit > 1) {  // unscaled fp32 partials of this K slice, one 16-byte store where it can
    xdl_fence();
#pragma unroll
    for (int c = 0; c < 2 * CT; ++c) {
      const int m = m0 + 16 * c + li;
      const int n0 = nbase + 4 * lq;
      if (m >= a.M || n0 >= rowend) continue;
      const v4f v = c < CT ? acc0[0][c] : acc1[0][c - CT];
      float* pp = a.part + ((int64_t)slice * a.M + m) * a.N + n0;
      if (n0 + 3 < rowend && a.N % 4 == 0 && (uintptr_t)a.part % 16 == 0) {
        *reinterpret_cast<v4f*>(pp) = v;
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (n0 + r < rowend) pp[r] = v[r];
      }
    }
    return;
  }
  // the epilogue's scales only now: held through the loop they would push the kernel
  // past the register file
  EpiScales<RT, 2 * CT> es;
  epi_scales(es, MD.sw, a.sx, a.M, nbase + 4 * lq, m0 + li, rowend);
  xdl_fence();
#pragma unroll
  for (int c = 0; c < 2 * CT; ++c) {
    const int m = m0 + 16 * c + li;
    const int n0 = nbase + 4 * lq;
    if (m >= a.M || n0 >= rowend) continue;
    store4e(MD.Y, MD.ldy, MD.sw != nullptr, MD.vec_store, a, es, 0, c, c < CT ? acc0[0][c] : acc1[0][c - CT], m, n0,
            rowend);
  }
}

// Y of a K-sliced GEMM (the planner slices every region of a weight alike, KS slices):
// the sum of the slices' fp32 partials in slice order, then the epilogue of store4
// ((sum * w_scale[n]) * x_scale[m], bf16 or fp32).  One thread per output element; its
// KS loads and the scales are issued before the first add, so their latencies overlap.
template <int KS>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs a) {
  const int64_t total = (int64_t)a.M * a.N;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const bool narrow = total < ((int64_t)1 << 31);
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += stride) {
    const int m = narrow ? (int)e / a.N : (int)(e / a.N);
    const int n = (int)(e - (int64_t)m * a.N);
    const float* pe = a.part + e;  // slice sl's partial of this element: pe[sl * M * N]
    float p[KS];
#pragma unroll
    for (int sl = 0; sl < KS; ++sl) p[sl] = pe[sl * total];
    const float sw = a.sw ? a.sw[n] : 1.0f, sx = a.sx ? a.sx[m] : 1.0f;
    float v = p[0];
#pragma unroll
    for (int sl = 1; sl < KS; ++sl) v += p[sl];
    if (a.sw) v = v * sw;
    v = v * sx;
    if (a.out_f32)
      reinterpret_cast<float*>(a.Y)[(int64_t)m * a.ldy + n] = v;
    else
      reinterpret_cast<uint16_t*>(a.Y)[(int64_t)m * a.ldy + n] = (uint16_t)bf16_bits(v);
  }
}

// Pipeline depth and fragment grouping per instance, chosen to stay within the register
// file: four slots and whole-chunk fragment groups for up to two activation tiles, three
// slots and two-step groups for four; fp8 without wide metadata loads (metadata rows not
// 16-byte aligned, four separately masked loads per chunk) one step lighter, and even so
// its four-tile, eight-wave instance spills a few registers.
// The resident-activation instances' dynamic LDS above the default limit: a per-device
// function attribute, set once per (device, instance) under std::call_once.
constexpr int kXresMaxBytes = 160 * 1024;

template <int DT, int CT, int RT, int WR, bool WM, bool TL, int GM = 0>
hipError_t launch_rows_wm(const dim3& grid, const dim3& block, const GemmArgs& a, hipStream_t s, int xres = 0) {
  constexpr bool light = DT == kFP8 && !WM;
  constexpr int NS = CT <= 2 && RT == 1 && !light ? 4 : 3;
  constexpr int P = CT == 1 && RT == 1 ? 4 : 1;
  if constexpr (DT == kFP8 && CT <= 2 && RT == 1 && WR == 8 && TL && GM <= 1) {
    if (xres > 0) {
      const int lds = xres * XTile<DT, CT>::BYTES;
      if (lds > kXresMaxBytes) return hipErrorInvalidValue;
      auto k = spense_gemm_rows_kernel<DT, CT, RT, WR, WM, NS, P, TL, GM, true>;
      int dev = 0;
      hipError_t e = hipGetDevice(&dev);
      if (e != hipSuccess) return e;
      if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
      static std::once_flag once[64];  // one set per instance of this function
      static hipError_t rc[64];
      std::call_once(once[dev], [&] {
        rc[dev] = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                      kXresMaxBytes);
      });
      if (rc[dev] != hipSuccess) return rc[dev];
      hipLaunchKernelGGL(k, grid, block, lds, s, a);
      return hipGetLastError();
    }
  }
  if (xres > 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL((spense_gemm_rows_kernel<DT, CT, RT, WR, WM, NS, P, TL, GM>), grid, block, 0, s, a);
  return hipGetLastError();
}

template <int DT, int CT, int RT, int WR>
hipError_t launch_rows(const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  dim3 grid = a.rorder ? dim3(a.groups * ls.mblocks) : dim3(a.groups, ls.mblocks), block(64 * WR);
  if constexpr (DT == kFP8) {
    if (a.tiled && (a.nmat > 1 || ls.glu)) {  // grouped or paired launch: tiled fp8, 8 waves
      if constexpr (RT == 1 && WR == 8) {
        if (ls.glu) return launch_rows_wm<DT, CT, RT, WR, true, true, 2>(grid, block, a, s);
        return launch_rows_wm<DT, CT, RT, WR, true, true, 1>(grid, block, a, s, ls.xres);
      }
      return hipErrorInvalidValue;
    }
    if (a.tiled) return launch_rows_wm<DT, CT, RT, WR, true, true>(grid, block, a, s, ls.xres);
    if (ls.xres) return hipErrorInvalidValue;
    if (a.m_ld_b % 16 == 0) return launch_rows_wm<DT, CT, RT, WR, true, false>(grid, block, a, s);
  }
  if (a.tiled || ls.xres) return hipErrorInvalidValue;
  return launch_rows_wm<DT, CT, RT, WR, false, false>(grid, block, a, s);
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
  // the LDS reduction buffer is W * RT KB
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

template <int DT, int CT>
hipError_t launch_rows_ct(const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  switch (ls.rt * 100 + ls.waves) {
    case 104: return launch_rows<DT, CT, 1, 4>(ls, a, s);
    case 108: return launch_rows<DT, CT, 1, 8>(ls, a, s);
    case 204: return launch_rows<DT, CT, 2, 4>(ls, a, s);
    default: return hipErrorInvalidValue;
  }
}

// ---------------------------------------------------------------- large-M kernel
// For many tokens the matrix cores become the bound, and every byte moved should feed
// many MMAs.  A workgroup computes 128 weight rows x 256 tokens; its waves form a grid of
// 2 row halves x 2 or 4 token parts, each wave 64 rows (4 row tiles) x 128 or 64 tokens
// (with 8 waves, two per SIMD, one wave's stalls are covered by the other's MMAs).  Both
// operands of a step (128 columns) are copied once into LDS by direct loads
// (activations 256 x 128 bytes, with 16-byte blocks swizzled so that the fragment reads
// of 16 rows are conflict-free; the weight fragments of the 8 row tiles in lane order),
// three stages deep, so that two steps of loads are in flight without holding
// registers.  Each B fragment read feeds 4 MMAs, each A fragment 4 or 8.  The barrier of
// a step sits before its last MMA group, and the fragments of the next step are read
// from LDS right after it, under that group, so that no wave starts a step waiting for
// LDS.  Workgroups of one row block are adjacent (token block fastest), so with 8 token
// blocks each XCD keeps one activation block in its L2.  fp8 only.
constexpr int kBigTokens = 256, kBigRowTiles = 8;

struct BigStage {
  static constexpr int X_B = kBigTokens * 128;       // activations: 256 tokens x 128 bytes
  static constexpr int W_B = kBigRowTiles * 2048;    // per row tile: 2:4 values or dense halves
  static constexpr int M_B = kBigRowTiles * 256;     // per row tile: metadata words
  static constexpr int BYTES = X_B + W_B + M_B;
  __device__ static __forceinline__ int xaddr(int r, int b) { return r * 128 + ((b ^ ((r >> 1) & 7)) << 4); }
};

template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>()), ...);
}
// f(integral_constant<int, i>) for i = 0 .. N-1, each index a compile-time constant.
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>());
}

// Where the loads of one step go and what they cover.
struct BigStepLd {
  uint8_t* st;                 // stage buffer
  int ks, ke, cs, js, cd, jd;  // first column, column end, tiled-layout chunk and step
  bool in, sparse;
};

// Step kinds for the fragment reads of the next step.
constexpr int kStepSparse = 0, kStepDense = 1, kStepNone = 2;

template <bool TL, int WV>
__global__ __launch_bounds__(64 * WV) void spense_gemm_big_kernel(GemmArgs a) {
  static_assert(WV == 4 || WV == 8, "4 or 8 waves");
  constexpr int RPW = 4, NT = kBigRowTiles;
  typedef BigStage St;
  constexpr int NS = 3, D = NS - 1;
  constexpr int TC = 32 / WV;                    // token tiles per wave
  constexpr int TU = NT / WV;                    // row tiles whose weights a wave copies
  constexpr int XI = St::X_B / 1024 / WV;        // 1 KB activation blocks per wave per step
  constexpr int NL = XI + 3 * TU;                // loads per wave per step
  constexpr int PER = (NL + TC - 1) / TC;        // loads issued after each MMA group
  constexpr int NL_AT_BAR = (TC - 1) * PER < NL ? (TC - 1) * PER : NL;  // issued before the barrier
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int li = lane & 15, lq = lane >> 4;
  const int wr = wave & 1, wc = wave >> 1;
  int g = blockIdx.x;
  if (a.xgt > 0 && g < a.xg1) {
    // XCD-aware order: XCD x (= id % 8) takes token group x % (T / GT) (GT blocks) and
    // the row blocks of class x / (T / GT) (every RC-th); a bijection on [0, xg1)
    const int T = a.tblocks, GT = a.xgt, RC = a.xrc, TGc = T / GT;
    const int x = g & 7, l = g >> 3, tg = x % TGc, rc = x / TGc;
    g = ((l / GT) * RC + rc) * T + tg * GT + l % GT;
  }
  const int ri = (a.nreg > 1 && g >= a.reg[1].wg0) ? 1 : 0;
  const Region& R = a.reg[ri];
  const int rowend = R.row0 + R.rows;
  const int rb = (g - R.wg0) / a.tblocks, tb = (g - R.wg0) % a.tblocks;
  const int rblk = R.row0 + rb * 16 * NT;  // first row of the workgroup
  const int m0 = tb * kBigTokens;
  const int K = R.kend, kbound = R.kbound;

  extern __shared__ __attribute__((aligned(1024))) uint8_t big_lds[];
  const __amdgpu_buffer_rsrc_t rx = rsrc(a.X, a.x_bytes), rv = rsrc(a.values, a.v_bytes),
                               rm = rsrc(a.meta, a.m_bytes), rd = rsrc(a.dense, a.d_bytes);
  v4f acc[RPW][TC];
#pragma unroll
  for (int t = 0; t < RPW; ++t)
#pragma unroll
    for (int c = 0; c < TC; ++c) acc[t][c] = (v4f){0.f, 0.f, 0.f, 0.f};

  // steps of 128 columns: 2:4 steps cover [0, kbound), dense steps start at kbound
  const int n_sp = (kbound + 127) / 128, n_de = (K - kbound + 127) / 128, nst = n_sp + n_de;
  const int nch_sp = (n_sp + 3) / 4, nch_de = (n_de + 3) / 4;  // tiled layout chunks
  auto step_k = [&](int s) __attribute__((always_inline)) { return s < n_sp ? 128 * s : kbound + 128 * (s - n_sp); };

  // This wave copies the weights of row tiles TU wave .. TU wave + TU - 1.
  bool tok[TU];
  uint32_t vb[TU], mb[TU], db[TU];
#pragma unroll
  for (int u = 0; u < TU; ++u) {
    const int r0 = rblk + 16 * (TU * wave + u);
    tok[u] = r0 < rowend;
    if constexpr (TL) {
      const uint32_t ts = (uint32_t)(r0 / 16), td = (uint32_t)((r0 - R.dense_row_off) / 16);
      vb[u] = ts * (uint32_t)nch_sp * 4096u + 16u * lane;
      mb[u] = ts * (uint32_t)nch_sp * 1024u + 16u * li + 4u * lq;
      db[u] = td * (uint32_t)nch_de * 8192u + 16u * lane;
    } else {
      const int n = min(r0 + li, rowend - 1);
      vb[u] = (uint32_t)((int64_t)n * a.v_ld_b) + 16u * lq;
      mb[u] = (uint32_t)((int64_t)n * a.m_ld_b) + 4u * lq;
      db[u] = (uint32_t)((int64_t)max(n - R.dense_row_off, 0) * a.d_ld_b) + 16u * lq;
    }
  }

  // Loads of step s into a stage buffer, numbered 0 .. NL-1: the activation blocks, then
  // for each of the wave's row tiles the value (or first dense) fragment, the second
  // dense fragment and the metadata word.  The ones a step does not use get out-of-range
  // offsets, so every step issues the same loads.
  auto prep = [&](int buf, int s) __attribute__((always_inline)) {
    BigStepLd p;
    p.st = big_lds + buf * St::BYTES;
    // wave-uniform (readfirstlane), so that the buffer resources chosen by them stay scalar
    p.in = __builtin_amdgcn_readfirstlane(s < nst ? 1 : 0) != 0;
    p.sparse = __builtin_amdgcn_readfirstlane(s < n_sp ? 1 : 0) != 0;
    p.ks = step_k(s);
    p.ke = !p.in ? -1 : (p.sparse ? kbound : K);
    const int sd = max(s - n_sp, 0);
    p.cs = s / 4;
    p.js = s & 3;
    p.cd = sd / 4;
    p.jd = sd & 3;
    return p;
  };
  auto load_one = [&](auto i_const, const BigStepLd& p) __attribute__((always_inline)) {
    constexpr int i = decltype(i_const)::value;
    if constexpr (i < XI) {
      const int blk = wave * XI + i;
      const int r = 8 * blk + (lane >> 3), pb = lane & 7, b = pb ^ ((r >> 1) & 7);
      const int m = m0 + r, kcol = p.ks + 16 * b;
      const uint32_t off = sel(m < a.M && kcol < p.ke, (uint32_t)((int64_t)m * a.ldx_b + kcol));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (__attribute__((address_space(3))) void*)(p.st + blk * 1024), 16, off,
                                               0, 0, 0);
    } else {
      constexpr int u = (i - XI) / 3, kind = (i - XI) % 3;
      const int tile = TU * wave + u;
      const bool ok = p.in && tok[u];
      if constexpr (kind == 0) {
        uint32_t off;
        bool k;
        if constexpr (TL) {
          off = p.sparse ? vb[u] + (uint32_t)(p.cs * 4096 + 1024 * p.js) : db[u] + (uint32_t)(p.cd * 8192 + 2048 * p.jd);
          k = ok;
        } else {
          off = p.sparse ? vb[u] + (uint32_t)(p.ks >> 1) : db[u] + (uint32_t)(p.ks - R.dense_col_off);
          k = ok && p.ks + (p.sparse ? 32 : 16) * lq < p.ke;
        }
        __builtin_amdgcn_raw_ptr_buffer_load_lds(p.sparse ? rv : rd,
                                                 (__attribute__((address_space(3))) void*)(p.st + St::X_B + tile * 2048),
                                                 16, sel(k, off), 0, 0, TL ? kTiledNT : kNT);
      } else if constexpr (kind == 1) {
        uint32_t off;
        bool k;
        if constexpr (TL) {
          off = db[u] + (uint32_t)(p.cd * 8192 + 2048 * p.jd + 1024);
          k = ok;
        } else {
          off = db[u] + (uint32_t)(p.ks - R.dense_col_off) + 64;
          k = ok && p.ks + 64 + 16 * lq < p.ke;
        }
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rd, (__attribute__((address_space(3))) void*)(p.st + St::X_B + tile * 2048 + 1024), 16,
            sel(k && !p.sparse, off), 0, 0, TL ? kTiledNT : kNT);
      } else {
        uint32_t off;
        bool k;
        if constexpr (TL) {
          off = mb[u] + (uint32_t)(p.cs * 1024 + 256 * p.js);
          k = ok;
        } else {
          off = mb[u] + 4u * (uint32_t)(p.ks >> 5);
          k = ok && p.ks + 32 * lq < p.ke;
        }
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rm, (__attribute__((address_space(3))) void*)(p.st + St::X_B + St::W_B + tile * 256), 4,
            sel(k && p.sparse, off), 0, 0, TL ? kTiledNT : kNT);
      }
    }
  };

  // Fragments.  A of the wave's 4 row tiles (2:4: value fragment and metadata word; dense:
  // both halves) in two sets that alternate between steps (set P holds the current step's,
  // the other receives the next step's); B, one register per token tile (the next step's
  // first two land in registers the current step's last group no longer reads).
  static_assert(TC >= 3, "the last group must not use B registers 0 and 1");
  v4i alo[2][RPW], ahi[2][RPW];
  int aix[2][RPW];
  v8i bq[TC];
  auto bfrag = [&](const uint8_t* st, int c) __attribute__((always_inline)) {
    const int r = 16 * (TC * wc + c) + li;
    return cat8(*reinterpret_cast<const v4i*>(st + St::xaddr(r, lq)),
                *reinterpret_cast<const v4i*>(st + St::xaddr(r, 4 + lq)));
  };
  auto read_a = [&](auto kind_const, auto set_const, const uint8_t* st) __attribute__((always_inline)) {
    constexpr int KIND = decltype(kind_const)::value, Q = decltype(set_const)::value;
    const uint8_t* wl = st + St::X_B + (RPW * wr) * 2048 + 16 * lane;
    const int* ml = reinterpret_cast<const int*>(st + St::X_B + St::W_B + (RPW * wr) * 256) + lane;
#pragma unroll
    for (int t = 0; t < RPW; ++t) {
      alo[Q][t] = *reinterpret_cast<const v4i*>(wl + t * 2048);
      if constexpr (KIND == kStepSparse) aix[Q][t] = ml[t * 64];
      if constexpr (KIND == kStepDense) ahi[Q][t] = *reinterpret_cast<const v4i*>(wl + t * 2048 + 1024);
    }
    bq[0] = bfrag(st, 0);
    bq[1] = bfrag(st, 1);
  };

  // One step: MMA group c uses B fragment c; fragment c + 2 is read before it.  Before the
  // last group: wait for this wave's reads of the stage and for its loads of step s + 1
  // (the loads of step s + D issued so far are younger), meet the other waves, and read the
  // first fragments of step s + 1 into the other set, under the last group.  The loads of
  // step s + D into stage (s + D) % NS (it held step s - 1, which every wave had finished
  // reading at the previous barrier) follow the MMA groups, PER at a time.
  int s = 0, cur = 0;  // cur = s % NS
  auto step = [&](auto kind_const, auto next_const, auto set_const) __attribute__((always_inline)) {
    constexpr bool SPARSE = decltype(kind_const)::value == kStepSparse;
    constexpr int NEXT = decltype(next_const)::value, P = decltype(set_const)::value;
    const int nxt = cur == 0 ? D : cur - 1;  // (s + D) % NS
    const int nx1 = cur == NS - 1 ? 0 : cur + 1;
    const uint8_t* st = big_lds + cur * St::BYTES;
    const BigStepLd ld = prep(nxt, s + D);
    static_for<TC>([&](auto c_const) {
      constexpr int c = decltype(c_const)::value;
      if constexpr (c == TC - 1) {
        barrier_vm_lgkm0<NL_AT_BAR>();
        if constexpr (NEXT != kStepNone)
          read_a(std::integral_constant<int, NEXT>(), std::integral_constant<int, 1 - P>(), big_lds + nx1 * St::BYTES);
      } else if constexpr (c + 2 < TC) {
        bq[c + 2] = bfrag(st, c + 2);
      }
#pragma unroll
      for (int t = 0; t < RPW; ++t) {
        if constexpr (SPARSE)
          acc[t][c] = mma_sparse(alo[P][t], bq[c], acc[t][c], aix[P][t], std::integral_constant<int, kFP8>());
        else
          acc[t][c] = mma_dense(cat8(alo[P][t], ahi[P][t]), bq[c], acc[t][c], std::integral_constant<int, kFP8>());
      }
      static_for<PER>([&](auto j_const) {
        constexpr int i = c * PER + decltype(j_const)::value;
        if constexpr (i < NL) load_one(std::integral_constant<int, i>(), ld);
      });
      __builtin_amdgcn_sched_barrier(0);
    });
    ++s;
    cur = nx1;
  };
  const std::integral_constant<int, 0> S0;
  const std::integral_constant<int, 1> S1;
  // Steps [s, e) of one kind, entered with the current fragments in set 0 and left with
  // the next part's first fragments (kind NEXT) in set 0.
  auto part = [&](auto kind_const, auto next_const, int e) __attribute__((always_inline)) {
    while (s + 2 < e) {
      step(kind_const, kind_const, S0);
      step(kind_const, kind_const, S1);
    }
    if (s + 2 == e) {
      step(kind_const, kind_const, S0);
      step(kind_const, next_const, S1);
    } else {
      step(kind_const, next_const, S0);
      if constexpr (decltype(next_const)::value != kStepNone) {
#pragma unroll
        for (int t = 0; t < RPW; ++t) {
          alo[0][t] = alo[1][t];
          ahi[0][t] = ahi[1][t];
          aix[0][t] = aix[1][t];
        }
      }
    }
  };

  // Prologue: loads of steps 0 .. D-1, then the first fragments of step 0.
#pragma unroll
  for (int d = 0; d < D; ++d) {
    const BigStepLd p = prep(d, d);
    static_for<NL>([&](auto i_const) { load_one(i_const, p); });
  }
  barrier_vm<NL>();  // step 0 is in LDS (only step 1's loads may be outstanding)
  const std::integral_constant<int, kStepSparse> SP;
  const std::integral_constant<int, kStepDense> DE;
  const std::integral_constant<int, kStepNone> NO;
  if (n_sp > 0)
    read_a(SP, S0, big_lds);
  else
    read_a(DE, S0, big_lds);

  // 2:4 steps, then dense steps.
  if (n_sp > 0) {
    if (n_de > 0)
      part(SP, DE, n_sp);
    else
      part(SP, NO, n_sp);
  }
  if (n_de > 0) part(DE, NO, nst);

  xdl_fence();
  EpiScales<RPW, TC> es;
  epi_scales(es, a.sw, a.sx, a.M, rblk + 16 * RPW * wr + 4 * lq, m0 + 16 * TC * wc + li, rowend);
  if (!a.out_f32 && ((uintptr_t)a.Y % 16 == 0) && (a.ldy % 8 == 0) && (rblk % 8 == 0)) {
    // whole token rows through LDS (out_tile_write)
    static_assert(16 * NT * 2 * kBigTokens <= 3 * St::BYTES, "the output tile fits the stages");
    barrier_vm_lgkm0<0>();  // every wave's last operand reads and copies are done
    out_tile_write<RPW, TC, 2 * NT>(big_lds, acc, es, a.sw != nullptr, wr, wc, li, lq);
    barrier_vm_lgkm0<0>();
    out_tile_store<2 * NT, 64 * WV>(big_lds, kBigTokens, m0, a.M, rblk, rowend, a.Y, a.ldy);
    return;
  }
#pragma unroll
  for (int t = 0; t < RPW; ++t)
#pragma unroll
    for (int c = 0; c < TC; ++c) {
      const int m = m0 + 16 * (TC * wc + c) + li;
      const int n0 = rblk + 16 * (RPW * wr + t) + 4 * lq;
      if (m < a.M && n0 < rowend) store4e(a.Y, a.ldy, a.sw != nullptr, a.vec_store, a, es, t, c, acc[t][c], m, n0, rowend);
    }
}

// ---------------------------------------------------------------- large-M kernel, 256 x 256 tiles
// Both operands through LDS as in spense_gemm_big_kernel, with twice the rows per
// workgroup and per wave: a workgroup computes 256 weight rows x 256 tokens, its 8 waves a
// grid of 2 row halves x 4 token quarters, each wave 128 rows (8 row tiles) x 64 tokens (4
// token tiles, 128 accumulators).  Each B fragment read from LDS feeds 8 MMAs, each A
// fragment 4.  Tiled weight layout only.
//
// The CU's load path moves about 57 bytes per clock from L2 with 16-byte-per-lane loads,
// into registers or straight into LDS alike, but a load instruction costs at least ~18
// clocks however few bytes it moves (a 4-byte-per-lane load moves 256 bytes in ~32; all
// measured on MI355X).  So every load here moves 1 KB: per 128-column step a wave issues 4
// activation blocks and, for its 2 row tiles, the 2:4 value blocks or both dense halves;
// a 2:4 step's metadata (256 bytes per row tile) takes 4 more loads, one on each of waves
// 0-3, each gathering the pieces of 4 row tiles.  6.5 loads per 2:4 step (52 KB per
// workgroup) against ~1.07k clocks of its 256 MMAs.
//
// Per-wave timelines showed every wave waiting at the barrier for the loads when they had
// one step to land in, so the 2:4 steps run three stages deep (loads two steps ahead; a
// stage is 52 KB: activations, values, metadata) and the dense steps, whose stage is 64 KB
// and whose MMAs take twice as long, two.  Within a step the loads go out early: the
// activation blocks before the first group of 4 MMAs, the weight blocks before the third.
// An input-split weight switches from the first layout to the second once, after a
// barrier.  The per-lane offsets are loop-invariant; the step's offset travels in the
// scalar offset.  The barrier at the start of a step waits for this wave's loads of the
// step and for its LDS reads of the previous step.
constexpr int kB2Rows = 256, kB2Tokens = 256, kB2RowTiles = 16;
constexpr int kB2XSlot = kB2Tokens * 128;                                      // activations of one step
constexpr int kB2SStage = kB2XSlot + kB2RowTiles * 1024 + kB2RowTiles * 256;  // + 2:4 values, metadata
constexpr int kB2DStage = kB2XSlot + kB2RowTiles * 2048;                       // + both dense halves
constexpr int kB2Lds = 3 * kB2SStage > 2 * kB2DStage ? 3 * kB2SStage : 2 * kB2DStage;

template <int AUX>
__device__ __forceinline__ void lds_load16(__amdgpu_buffer_rsrc_t r, uint8_t* dst, uint32_t voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)dst, 16, voff, soff, 0, AUX);
}

// GR: a grouped launch (several weights sharing X and K): up to kMaxRegions regions, each
// reading its weight's buffers, output and scales from a.mat[R.mat].
template <bool GR>
__global__ __launch_bounds__(512) void spense_gemm_big2_kernel(GemmArgs a) {
  constexpr int WV = 8, NT = kB2RowTiles, RPW = 8, TC = 4;
  constexpr int TU = NT / WV;                // row tiles whose weights a wave copies
  constexpr int XI = kB2XSlot / 1024 / WV;  // 1 KB activation blocks per wave per step
  constexpr int MW = NT * 256 / 1024;       // waves that copy a 2:4 step's metadata
  static_assert(XI + 2 * TU == RPW, "eight loads per dense step");
  static_assert(XI == 4 && TU == 2 && MW <= WV, "load schedule");
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int li = lane & 15, lq = lane >> 4;
  const int wr = wave & 1, wc = wave >> 1;
  // Workgroups [0, hg0): 256 x 256 tiles, in the XCD-aware order when it is on.  From
  // hg0 on (dispatched last, so that they fill the tail of the grid): the row blocks
  // hrb0 .. of the last region as 256 x 128 tiles, hper per row block; their waves of
  // token quarters 2 and 3 only copy and take part in the barriers.
  int g = blockIdx.x, ri, rb, m0;
  bool half = false;
  if (g < a.hg0) {
    if (a.xgt > 0 && g < a.xg1) {  // XCD-aware order, as in spense_gemm_big_kernel
      const int T = a.tblocks, GT = a.xgt, RC = a.xrc, TGc = T / GT;
      const int x = g & 7, l = g >> 3, tg = x % TGc, rc = x / TGc;
      g = ((l / GT) * RC + rc) * T + tg * GT + l % GT;
    }
    ri = 0;
    if constexpr (GR) {
      for (int i = 1; i < a.nreg; ++i)
        if (g >= a.reg[i].wg0) ri = i;
    } else {
      ri = (a.nreg > 1 && g >= a.reg[1].wg0) ? 1 : 0;
    }
    rb = (g - a.reg[ri].wg0) / a.tblocks;
    m0 = (g - a.reg[ri].wg0) % a.tblocks * (a.btok > 0 ? a.btok : kB2Tokens);
  } else {
    const int h = g - a.hg0;
    ri = a.nreg - 1;
    rb = a.hrb0 + h / a.hper;
    m0 = h % a.hper * (kB2Tokens / 2);
    half = true;
  }
  const Region& R = a.reg[ri];
  const int rowend = R.row0 + R.rows;
  const int rblk = R.row0 + rb * kB2Rows;
  // tokens of this tile: 256, or 192 (full tiles of a 192-token block), or 128 (half tiles)
  const int ntok = half ? kB2Tokens / 2 : (a.btok > 0 ? a.btok : kB2Tokens);
  const int K = R.kend, kbound = R.kbound;

  extern __shared__ __attribute__((aligned(1024))) uint8_t big_lds[];
  const MatDesc& MD = a.mat[GR ? R.mat : 0];
  const __amdgpu_buffer_rsrc_t rx = rsrc(a.X, a.x_bytes),
                               rv = GR ? rsrc(MD.values, MD.v_bytes) : rsrc(a.values, a.v_bytes),
                               rm = GR ? rsrc(MD.meta, MD.m_bytes) : rsrc(a.meta, a.m_bytes),
                               rd = GR ? rsrc(MD.dense, MD.d_bytes) : rsrc(a.dense, a.d_bytes);
  v4f acc[RPW][TC];
#pragma unroll
  for (int t = 0; t < RPW; ++t)
#pragma unroll
    for (int c = 0; c < TC; ++c) acc[t][c] = (v4f){0.f, 0.f, 0.f, 0.f};

  const int n_sp = (kbound + 127) / 128, n_de = (K - kbound + 127) / 128, nst = n_sp + n_de;
  const int nch_sp = (n_sp + 3) / 4, nch_de = (n_de + 3) / 4;

  // loop-invariant per-lane offsets (kOOB for rows past M or row tiles past the region)
  uint32_t xo[XI];
  int xb[XI];  // the column (bytes) of this lane's 16-byte block inside the step
#pragma unroll
  for (int i = 0; i < XI; ++i) {
    const int blk = wave * XI + i;
    const int r = 8 * blk + (lane >> 3), b = (lane & 7) ^ ((r >> 1) & 7);
    const int m = m0 + r;
    xb[i] = 16 * b;
    xo[i] = m < a.M && r < ntok ? (uint32_t)((int64_t)m * a.ldx_b + 16 * b) : kOOB;
  }
  uint32_t vo[TU], dlo[TU];
#pragma unroll
  for (int u = 0; u < TU; ++u) {
    const int r0 = rblk + 16 * (TU * wave + u);
    const bool ok = r0 < rowend;
    vo[u] = ok ? (uint32_t)(r0 / 16) * (uint32_t)nch_sp * 4096u + 16u * lane : kOOB;
    dlo[u] = ok && r0 >= R.dense_row_off ? (uint32_t)((r0 - R.dense_row_off) / 16) * (uint32_t)nch_de * 8192u + 16u * lane
                                          : kOOB;
  }
  // a 2:4 step's metadata: wave w < MW copies the 256-byte pieces of row tiles 4w .. 4w + 3
  // (lane l: 16 bytes of tile 4w + l / 16); a tile's piece for step s sits 256 s bytes into
  // its metadata
  uint32_t mo1 = kOOB;
  if (wave < MW) {
    const int r0 = rblk + 16 * (4 * wave + (lane >> 4));
    if (r0 < rowend) mo1 = (uint32_t)(r0 / 16) * (uint32_t)nch_sp * 1024u + 16u * li;
  }

  // Load j of this wave for 2:4 step sn into stage stg: activation blocks (j < 4), the value
  // blocks of its two row tiles (j = 4, 5), the metadata gather (j = 6, waves 0-3).
  auto sp_load = [&](auto j_const, int sn, uint8_t* stg) __attribute__((always_inline)) {
    constexpr int j = decltype(j_const)::value;
    if (sn >= n_sp) return;  // uniform
    if constexpr (j < XI) {
      const int ks = 128 * sn;
      uint32_t off = xo[j];
      if (ks + 128 > kbound) off = ks + xb[j] < kbound ? off : kOOB;  // the region's last, partial step
      lds_load16<0>(rx, stg + (wave * XI + j) * 1024, off, ks);
    } else if constexpr (j < XI + TU) {
      constexpr int u = j - XI;
      lds_load16<kTiledNT>(rv, stg + kB2XSlot + (TU * wave + u) * 1024, vo[u], 1024 * sn);
    } else {
      if (wave < MW) lds_load16<kTiledNT>(rm, stg + kB2XSlot + NT * 1024 + wave * 1024, mo1, 256 * sn);
    }
  };
  // Load j of this wave for dense step sn into stage stg: activation blocks (j < 4), then
  // the two halves of its two row tiles.
  auto de_load = [&](auto j_const, int sn, uint8_t* stg) __attribute__((always_inline)) {
    constexpr int j = decltype(j_const)::value;
    if (sn >= nst) return;  // uniform
    if constexpr (j < XI) {
      const int ks = kbound + 128 * (sn - n_sp);
      uint32_t off = xo[j];
      if (ks + 128 > K) off = ks + xb[j] < K ? off : kOOB;
      lds_load16<0>(rx, stg + (wave * XI + j) * 1024, off, ks);
    } else {
      constexpr int u = (j - XI) % TU, half = (j - XI) / TU;
      lds_load16<kTiledNT>(rd, stg + kB2XSlot + (TU * wave + u) * 2048 + 1024 * half, dlo[u],
                           2048 * (sn - n_sp) + 1024 * half);
    }
  };

  // B fragments of the wave's 4 token tiles from a stage
  auto read_b = [&](v8i (&bq)[TC], const uint8_t* xs) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < TC; ++c) {
      const int r = 16 * (TC * wc + c) + li;
      bq[c] = cat8(*reinterpret_cast<const v4i*>(xs + r * 128 + ((lq ^ ((r >> 1) & 7)) << 4)),
                   *reinterpret_cast<const v4i*>(xs + r * 128 + (((4 + lq) ^ ((r >> 1) & 7)) << 4)));
    }
  };

  // 2:4 step s from stage cur; the loads of step s + 2 go to stage nxt.  Per row tile t the
  // A fragment of tile t + 1 is read (other register set) before the 4 MMAs of tile t.
  // ACT = false: a wave without tokens (token quarters past a 128- or 192-token tile) only copies.
  auto sp_step = [&](auto act_const, int s, const uint8_t* cur, uint8_t* nxt) __attribute__((always_inline)) {
    constexpr bool ACT = decltype(act_const)::value;
    // this wave's loads of step s have landed once at most those of step s + 1 are pending
    if (s + 1 < n_sp) {
      if (wave < MW)
        barrier_vm_lgkm0<XI + TU + 1>();
      else
        barrier_vm_lgkm0<XI + TU>();
    } else {
      barrier_vm_lgkm0<0>();
    }
    v8i bq[TC];
    const uint8_t* vl = cur + kB2XSlot + (RPW * wr) * 1024 + 16 * lane;
    const uint8_t* ml = cur + kB2XSlot + NT * 1024 + (RPW * wr) * 256 + 16 * li + 4 * lq;
    v4i av[2];
    int aix[2];
    if constexpr (ACT) {
      read_b(bq, cur);
      av[0] = *reinterpret_cast<const v4i*>(vl);
      aix[0] = *reinterpret_cast<const int*>(ml);
    }
    static_for<RPW>([&](auto t_const) {
      constexpr int t = decltype(t_const)::value;
      constexpr int q = t & 1;
      if constexpr (ACT && t + 1 < RPW) {
        av[1 - q] = *reinterpret_cast<const v4i*>(vl + (t + 1) * 1024);
        aix[1 - q] = *reinterpret_cast<const int*>(ml + (t + 1) * 256);
      }
      if constexpr (t == 0) static_for<XI>([&](auto j) { sp_load(j, s + 2, nxt); });
      if constexpr (t == 2) {
        sp_load(std::integral_constant<int, XI>(), s + 2, nxt);
        sp_load(std::integral_constant<int, XI + 1>(), s + 2, nxt);
        sp_load(std::integral_constant<int, XI + 2>(), s + 2, nxt);
      }
      if constexpr (ACT) {
#pragma unroll
        for (int c = 0; c < TC; ++c)
          acc[t][c] = mma_sparse(av[q], bq[c], acc[t][c], aix[q], std::integral_constant<int, kFP8>());
      }
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  // dense step s from stage cur; the loads of step s + 1 go to stage nxt
  auto de_step = [&](auto act_const, int s, const uint8_t* cur, uint8_t* nxt) __attribute__((always_inline)) {
    constexpr bool ACT = decltype(act_const)::value;
    barrier_vm_lgkm0<0>();
    v8i bq[TC];
    const uint8_t* wl = cur + kB2XSlot + (RPW * wr) * 2048 + 16 * lane;
    v4i alo[2], ahi[2];
    if constexpr (ACT) {
      read_b(bq, cur);
      alo[0] = *reinterpret_cast<const v4i*>(wl);
      ahi[0] = *reinterpret_cast<const v4i*>(wl + 1024);
    }
    static_for<RPW>([&](auto t_const) {
      constexpr int t = decltype(t_const)::value;
      constexpr int q = t & 1;
      if constexpr (ACT && t + 1 < RPW) {
        alo[1 - q] = *reinterpret_cast<const v4i*>(wl + (t + 1) * 2048);
        ahi[1 - q] = *reinterpret_cast<const v4i*>(wl + (t + 1) * 2048 + 1024);
      }
      if constexpr (t == 0 || t == 2) {
        de_load(std::integral_constant<int, 2 * t>(), s + 1, nxt);
        de_load(std::integral_constant<int, 2 * t + 1>(), s + 1, nxt);
        de_load(std::integral_constant<int, 2 * t + 2>(), s + 1, nxt);
        de_load(std::integral_constant<int, 2 * t + 3>(), s + 1, nxt);
      }
      if constexpr (ACT) {
#pragma unroll
        for (int c = 0; c < TC; ++c)
          acc[t][c] = mma_dense(cat8(alo[q], ahi[q]), bq[c], acc[t][c], std::integral_constant<int, kFP8>());
      }
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  auto run = [&](auto act_const) __attribute__((always_inline)) {
    int s = 0;
    if (n_sp > 0) {
      static_for<XI + TU + 1>([&](auto j) { sp_load(j, 0, big_lds); });
      static_for<XI + TU + 1>([&](auto j) { sp_load(j, 1, big_lds + kB2SStage); });
      int k = 0;  // stage of step s
      for (; s < n_sp; ++s) {
        const int k2 = k == 0 ? 2 : k - 1;  // stage of step s + 2
        sp_step(act_const, s, big_lds + k * kB2SStage, big_lds + k2 * kB2SStage);
        k = k == 2 ? 0 : k + 1;
      }
      xdl_fence();
    }
    if (n_de > 0) {
      if (n_sp > 0) barrier_vm_lgkm0<0>();  // every wave is done with the 2:4 stages
      static_for<RPW>([&](auto j) { de_load(j, s, big_lds); });
      for (; s < nst; ++s) {
        const int k = (s - n_sp) & 1;
        de_step(act_const, s, big_lds + k * kB2DStage, big_lds + (1 - k) * kB2DStage);
      }
      xdl_fence();
    }
  };
  // bf16 output with 16-byte aligned rows leaves through LDS as whole token rows
  // (out_tile_write); the waves of token quarters past the tile's tokens (2 and 3 of a 256
  // x 128 tile, 3 of a 256 x 192 one) then only help with the stores
  const bool idle = wc * (kB2Tokens / 4) >= ntok;
  const bool via_lds = !a.out_f32 && ((uintptr_t)MD.Y % 16 == 0) && (MD.ldy % 8 == 0) && (rblk % 8 == 0);
  if (idle) {
    run(std::false_type());
    if (!via_lds) return;
  } else {
    run(std::true_type());
  }
  EpiScales<RPW, TC> es;
  if (!idle) epi_scales(es, MD.sw, a.sx, a.M, rblk + 16 * RPW * wr + 4 * lq, m0 + 16 * TC * wc + li, rowend);
  if (!via_lds) {
#pragma unroll
    for (int t = 0; t < RPW; ++t)
#pragma unroll
      for (int c = 0; c < TC; ++c) {
        const int m = m0 + 16 * (TC * wc + c) + li;
        const int n0 = rblk + 16 * (RPW * wr + t) + 4 * lq;
        if (m < a.M && n0 < rowend) store4e(MD.Y, MD.ldy, MD.sw != nullptr, MD.vec_store, a, es, t, c, acc[t][c], m, n0, rowend);
      }
    return;
  }
  barrier_vm_lgkm0<0>();  // every wave's last operand reads and copies are done
  if (!idle) out_tile_write<RPW, TC, kB2Rows / 8>(big_lds, acc, es, MD.sw != nullptr, wr, wc, li, lq);
  barrier_vm_lgkm0<0>();
  out_tile_store<kB2Rows / 8, 512>(big_lds, ntok, m0, a.M, rblk, rowend, MD.Y, MD.ldy);
}

// The large-M kernels' dynamic LDS above the default limit is a per-device function
// attribute: set once per (device, kernel instance), under std::call_once, so that host
// threads making their first large-M call together do not race.
constexpr int kMaxDevices = 64;
std::once_flag g_big_lds_once[kMaxDevices][2][4];  // [device][tiled][kernel instance]
hipError_t g_big_lds_rc[kMaxDevices][2][4];

template <typename KernelT>
hipError_t set_big_lds(KernelT k, int tiled, int which, int lds) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::call_once(g_big_lds_once[dev][tiled][which], [&] {
    g_big_lds_rc[dev][tiled][which] =
        hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  });
  return g_big_lds_rc[dev][tiled][which];
}

hipError_t launch_big2(const GemmArgs& a, hipStream_t s) {
  static_assert(kB2Lds <= 160 * 1024, "LDS of a CU");
  if (!a.tiled) return hipErrorInvalidValue;  // the planner sends row-major weights to the 128 x 256 kernel
  const bool gr = a.nmat > 1;
  auto k = gr ? spense_gemm_big2_kernel<true> : spense_gemm_big2_kernel<false>;
  hipError_t e = set_big_lds(k, 1, gr ? 3 : 2, kB2Lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k, dim3(a.groups), dim3(512), kB2Lds, s, a);
  return hipGetLastError();
}

template <int WV>
hipError_t launch_big_wv(const GemmArgs& a, hipStream_t s) {
  constexpr int lds = 3 * BigStage::BYTES;
  static_assert(lds <= 160 * 1024, "LDS of a CU");
  auto k = a.tiled ? spense_gemm_big_kernel<true, WV> : spense_gemm_big_kernel<false, WV>;
  hipError_t e = set_big_lds(k, a.tiled ? 1 : 0, WV == 8 ? 1 : 0, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k, dim3(a.groups), dim3(64 * WV), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_big(const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  if (ls.big == 2) return launch_big2(a, s);
  return ls.waves == 4 ? launch_big_wv<4>(a, s) : launch_big_wv<8>(a, s);
}

template <int DT>
hipError_t launch_dt(const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  if (ls.big) return DT == kFP8 ? launch_big(ls, a, s) : hipErrorInvalidValue;
  if (a.tiled && !ls.rows) return hipErrorInvalidValue;  // the K-split kernel reads the row-major layout only
  if (ls.rows == 2) {  // two 64-token halves per workgroup: tiled fp8, 8 waves, one row tile
    if constexpr (DT == kFP8) {
      if (!a.tiled || ls.rt != 1 || ls.waves != 8 || a.nmat != 1) return hipErrorInvalidValue;
      for (int i = 0; i < a.nreg; ++i)
        if (a.reg[i].ksplit > 1 && !a.part) return hipErrorInvalidValue;
      // two weight slots: with three the kernel spills past the register file
      hipLaunchKernelGGL((spense_gemm_rows2_kernel<8, 2>), dim3(a.groups, ls.mblocks), dim3(512), 0, s, a);
      return hipGetLastError();
    }
    return hipErrorInvalidValue;
  }
  if (ls.rows) {
    if (ls.ct == 1) return launch_rows_ct<DT, 1>(ls, a, s);
    if (ls.ct == 2) return launch_rows_ct<DT, 2>(ls, a, s);
    return launch_rows_ct<DT, 4>(ls, a, s);
  }
  if (ls.ct == 1) return launch_ct<DT, 1>(ls, a, s);
  if (ls.ct == 2) return launch_ct<DT, 2>(ls, a, s);
  return launch_ct<DT, 4>(ls, a, s);
}

}  // namespace

hipError_t launch_splitk_reduce(const GemmArgs& a, hipStream_t s) {
  const int64_t total = (int64_t)a.M * a.N;
  int64_t g = (total + 255) / 256;
  if (g > 4096) g = 4096;
  const dim3 grid((unsigned)(g < 1 ? 1 : g)), block(256);
  for (int i = 1; i < a.nreg; ++i)
    if (a.reg[i].ksplit != a.reg[0].ksplit) return hipErrorInvalidValue;  // one slice count per weight
  switch (a.reg[0].ksplit) {
    case 2: hipLaunchKernelGGL(splitk_reduce_kernel<2>, grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL(splitk_reduce_kernel<3>, grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL(splitk_reduce_kernel<4>, grid, block, 0, s, a); break;
    case 5: hipLaunchKernelGGL(splitk_reduce_kernel<5>, grid, block, 0, s, a); break;
    case 6: hipLaunchKernelGGL(splitk_reduce_kernel<6>, grid, block, 0, s, a); break;
    case 7: hipLaunchKernelGGL(splitk_reduce_kernel<7>, grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL(splitk_reduce_kernel<8>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(int dtype, const LaunchShape& ls, const GemmArgs& a, hipStream_t s) {
  return dtype == kFP8 ? launch_dt<kFP8>(ls, a, s) : launch_dt<kBF16>(ls, a, s);
}

}  // namespace spense
