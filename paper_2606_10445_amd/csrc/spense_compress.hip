// 2:4 compressor / decompressor and dense-region copies (paper sec. 3.1.1: keep only the
// non-zeros of each group of four plus their positions; sec. 3.2: the dense region is
// stored unchanged).
//
// One thread owns one 32-entry slice of a 2:4 row: it reads 32 weights and 32 mask
// bytes, emits 16 kept values and one 32-bit metadata word (8 groups x 4 bits).
#include "spense_internal.h"

namespace spense {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

template <int ES>
struct Slice {
  v4i q[2 * ES];  // 32 * ES bytes
};

template <int ES>
__device__ inline Slice<ES> load_slice(const uint8_t* p) {
  Slice<ES> s;
#pragma unroll
  for (int i = 0; i < 2 * ES; ++i) s.q[i] = *reinterpret_cast<const v4i*>(p + 16 * i);
  return s;
}

template <int ES>
__device__ inline uint32_t elem(const Slice<ES>& s, int e) {
  const uint8_t* b = reinterpret_cast<const uint8_t*>(s.q);
  if constexpr (ES == 1)
    return b[e];
  else
    return reinterpret_cast<const uint16_t*>(b)[e];
}

// The two selected positions of a group: the kept ones, padded with the lowest free
// positions, in ascending order.  sel has exactly two bits set.
__device__ inline uint32_t fill_to_two(uint32_t keep) {
  uint32_t sel = keep;
  while (__popc(sel) < 2) sel |= (~sel) & (sel + 1u) & 15u;  // lowest clear bit
  return sel;
}

template <int ES>
__global__ __launch_bounds__(256) void compress_kernel(const uint8_t* __restrict__ W, int64_t ldw_b,
                                                       const uint8_t* __restrict__ mask, int64_t ldm,
                                                       int64_t rows, int64_t words, uint8_t* __restrict__ values,
                                                       int64_t v_ld_b, uint32_t* __restrict__ meta, int64_t m_ld,
                                                       unsigned long long* bad) {
  const int64_t total = rows * words;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t nbad = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int64_t r = i / words, w = i - r * words;
    const Slice<ES> s = load_slice<ES>(W + r * ldw_b + w * 32 * ES);
    uint32_t keepmask = 0;  // bit e set: entry e of the slice is kept
    if (mask) {
      const uint8_t* mp = mask + r * ldm + w * 32;
      const v4i m0 = *reinterpret_cast<const v4i*>(mp);
      const v4i m1 = *reinterpret_cast<const v4i*>(mp + 16);
      const uint8_t* mb0 = reinterpret_cast<const uint8_t*>(&m0);
      const uint8_t* mb1 = reinterpret_cast<const uint8_t*>(&m1);
#pragma unroll
      for (int e = 0; e < 16; ++e) keepmask |= (mb0[e] != 0 ? 1u : 0u) << e;
#pragma unroll
      for (int e = 0; e < 16; ++e) keepmask |= (mb1[e] != 0 ? 1u : 0u) << (16 + e);
    } else {
#pragma unroll
      for (int e = 0; e < 32; ++e) keepmask |= (elem<ES>(s, e) != 0 ? 1u : 0u) << e;
    }
    uint32_t word = 0;
    uint32_t out[4 * ES];  // 16 values of ES bytes packed into 32-bit words
#pragma unroll
    for (int j = 0; j < 4 * ES; ++j) out[j] = 0;
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      uint32_t keep = (keepmask >> (4 * g)) & 15u;
      if (__popc(keep) > 2) {
        ++nbad;
        keep = 0;
      }
      const uint32_t sel = fill_to_two(keep);
      const uint32_t i0 = __builtin_ctz(sel);
      const uint32_t i1 = __builtin_ctz(sel & (sel - 1u));
      const uint32_t v0 = (keep >> i0) & 1u ? elem<ES>(s, 4 * g + i0) : 0u;
      const uint32_t v1 = (keep >> i1) & 1u ? elem<ES>(s, 4 * g + i1) : 0u;
      word |= (i0 | (i1 << 2)) << (4 * g);
      if constexpr (ES == 1) {
        out[g / 2] |= (v0 | (v1 << 8)) << (16 * (g & 1));
      } else {
        out[g] = v0 | (v1 << 16);
      }
    }
    uint8_t* vp = values + r * v_ld_b + w * 16 * ES;
#pragma unroll
    for (int j = 0; j < ES; ++j) {
      v4i o = {(int)out[4 * j], (int)out[4 * j + 1], (int)out[4 * j + 2], (int)out[4 * j + 3]};
      *reinterpret_cast<v4i*>(vp + 16 * j) = o;
    }
    meta[r * m_ld + w] = word;
  }
  if (nbad) atomicAdd(bad, (unsigned long long)nbad);
}

template <int ES>
__global__ __launch_bounds__(256) void decompress_kernel(const uint8_t* __restrict__ values, int64_t v_ld_b,
                                                         const uint32_t* __restrict__ meta, int64_t m_ld,
                                                         int64_t rows, int64_t words, uint8_t* __restrict__ W,
                                                         int64_t ldw_b) {
  const int64_t total = rows * words;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int64_t r = i / words, w = i - r * words;
    const uint8_t* vp = values + r * v_ld_b + w * 16 * ES;
    uint32_t in[4 * ES];
#pragma unroll
    for (int j = 0; j < ES; ++j) {
      v4i t = *reinterpret_cast<const v4i*>(vp + 16 * j);
      in[4 * j + 0] = t[0];
      in[4 * j + 1] = t[1];
      in[4 * j + 2] = t[2];
      in[4 * j + 3] = t[3];
    }
    const uint32_t word = meta[r * m_ld + w];
    uint32_t out[8 * ES];
#pragma unroll
    for (int j = 0; j < 8 * ES; ++j) out[j] = 0;
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      const uint32_t code = (word >> (4 * g)) & 15u;
      const int p0 = 4 * g + (code & 3u), p1 = 4 * g + (code >> 2);
      uint32_t v0, v1;
      if constexpr (ES == 1) {
        v0 = (in[(2 * g) / 4] >> (8 * ((2 * g) & 3))) & 0xffu;
        v1 = (in[(2 * g + 1) / 4] >> (8 * ((2 * g + 1) & 3))) & 0xffu;
        out[p0 / 4] |= v0 << (8 * (p0 & 3));
        out[p1 / 4] |= v1 << (8 * (p1 & 3));
      } else {
        v0 = in[g] & 0xffffu;
        v1 = in[g] >> 16;
        out[p0 / 2] |= v0 << (16 * (p0 & 1));
        out[p1 / 2] |= v1 << (16 * (p1 & 1));
      }
    }
    uint8_t* wp = W + r * ldw_b + w * 32 * ES;
#pragma unroll
    for (int j = 0; j < 8 * ES; j += 4) {
      v4i o = {(int)out[j], (int)out[j + 1], (int)out[j + 2], (int)out[j + 3]};
      *reinterpret_cast<v4i*>(wp + 4 * j) = o;
    }
  }
}

// rows x cols_b bytes, 16-byte chunks, strided source and destination.
__global__ __launch_bounds__(256) void copy2d_kernel(const uint8_t* __restrict__ src, int64_t src_ld,
                                                     uint8_t* __restrict__ dst, int64_t dst_ld, int64_t rows,
                                                     int64_t chunks) {
  const int64_t total = rows * chunks;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int64_t r = i / chunks, c = i - r * chunks;
    *reinterpret_cast<v4i*>(dst + r * dst_ld + 16 * c) = *reinterpret_cast<const v4i*>(src + r * src_ld + 16 * c);
  }
}

__global__ void zero_u64_kernel(unsigned long long* p) { *p = 0ull; }

// Reorder one region of a row-major packed fp8 weight into the tiled execution layout
// (one thread per 16-byte destination block; positions past the region are zero).
// Destination block g lies in tile-chunk tc = g / per (tile t = tc / chunks, chunk
// c = tc % chunks); within it, instruction n = (g % per) / 64 and lane l = g % 64 =
// i + 16 q read 16 bytes of row 16 t + i:
//   kind 0 (2:4 values, per = 256): value bytes 256 c + 64 n + 16 q;
//   kind 1 (metadata, per = 64):   words 16 c + 4 q .. +3 (copied one word at a time);
//   kind 2 (dense, per = 512):     bytes 512 c + 128 (n / 2) + 64 (n % 2) + 16 q.
__global__ __launch_bounds__(256) void tile_kernel(int kind, const uint8_t* __restrict__ src, int64_t src_ld_b,
                                                   int64_t rows, int64_t row_bytes, int64_t chunks,
                                                   uint8_t* __restrict__ dst, int64_t nblocks) {
  const int per = kind == 0 ? 256 : (kind == 1 ? 64 : 512);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nblocks; g += stride) {
    const int64_t tc = g / per;
    const int w = (int)(g - tc * per);
    const int64_t t = tc / chunks, c = tc - t * chunks;
    const int l = w & 63, n = w >> 6, i = l & 15, q = l >> 4;
    const int64_t row = 16 * t + i;
    const int64_t byte = kind == 0 ? 256 * c + 64 * n + 16 * q
                                   : (kind == 1 ? 4 * (16 * c + 4 * q) : 512 * c + 128 * (n >> 1) + 64 * (n & 1) + 16 * q);
    v4i v = {0, 0, 0, 0};
    if (row < rows) {
      const uint8_t* sp = src + row * src_ld_b + byte;
      if (kind == 1) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (byte + 4 * k + 4 <= row_bytes) v[k] = reinterpret_cast<const int*>(sp)[k];
      } else if (byte + 16 <= row_bytes) {
        v = *reinterpret_cast<const v4i*>(sp);
      }
    }
    *reinterpret_cast<v4i*>(dst + 16 * g) = v;
  }
}

inline unsigned grid_for(int64_t n) {
  int64_t g = (n + 255) / 256;
  if (g > 8192) g = 8192;
  return (unsigned)(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_tile(int kind, const uint8_t* src, int64_t src_ld_b, int64_t rows, int64_t row_bytes, int64_t tiles,
                       int64_t chunks, uint8_t* dst, hipStream_t s) {
  const int64_t per = kind == 0 ? 256 : (kind == 1 ? 64 : 512);
  const int64_t nblocks = tiles * chunks * per;
  if (nblocks == 0) return hipSuccess;
  hipLaunchKernelGGL(tile_kernel, dim3(grid_for(nblocks)), dim3(256), 0, s, kind, src, src_ld_b, rows, row_bytes,
                     chunks, dst, nblocks);
  return hipGetLastError();
}

hipError_t launch_zero_u64(unsigned long long* p, hipStream_t s) {
  hipLaunchKernelGGL(zero_u64_kernel, dim3(1), dim3(1), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_compress(int dtype, const uint8_t* W, int64_t ldw_b, const uint8_t* mask, int64_t ldm,
                           int64_t s_rows, int64_t s_cols, uint8_t* values, int64_t v_ld_b, uint32_t* meta,
                           int64_t m_ld, const uint8_t* dsrc, int64_t d_rows, int64_t d_cols_b, uint8_t* dense,
                           int64_t d_ld_b, unsigned long long* bad, hipStream_t s) {
  const int64_t words = s_cols / 32;
  if (s_rows > 0 && words > 0) {
    const unsigned g = grid_for(s_rows * words);
    if (dtype == kFP8)
      hipLaunchKernelGGL(compress_kernel<1>, dim3(g), dim3(256), 0, s, W, ldw_b, mask, ldm, s_rows, words, values,
                         v_ld_b, meta, m_ld, bad);
    else
      hipLaunchKernelGGL(compress_kernel<2>, dim3(g), dim3(256), 0, s, W, ldw_b, mask, ldm, s_rows, words, values,
                         v_ld_b, meta, m_ld, bad);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (d_rows > 0 && d_cols_b > 0) {
    const int64_t chunks = d_cols_b / 16;
    hipLaunchKernelGGL(copy2d_kernel, dim3(grid_for(d_rows * chunks)), dim3(256), 0, s, dsrc, ldw_b, dense, d_ld_b,
                       d_rows, chunks);
    return hipGetLastError();
  }
  return hipSuccess;
}

hipError_t launch_decompress(int dtype, const uint8_t* values, int64_t v_ld_b, const uint32_t* meta, int64_t m_ld,
                             int64_t s_rows, int64_t s_cols, uint8_t* W, int64_t ldw_b, const uint8_t* dense,
                             int64_t d_ld_b, int64_t d_rows, int64_t d_cols_b, uint8_t* ddst, hipStream_t s) {
  const int64_t words = s_cols / 32;
  if (s_rows > 0 && words > 0) {
    const unsigned g = grid_for(s_rows * words);
    if (dtype == kFP8)
      hipLaunchKernelGGL(decompress_kernel<1>, dim3(g), dim3(256), 0, s, values, v_ld_b, meta, m_ld, s_rows, words,
                         W, ldw_b);
    else
      hipLaunchKernelGGL(decompress_kernel<2>, dim3(g), dim3(256), 0, s, values, v_ld_b, meta, m_ld, s_rows, words,
                         W, ldw_b);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (d_rows > 0 && d_cols_b > 0) {
    const int64_t chunks = d_cols_b / 16;
    hipLaunchKernelGGL(copy2d_kernel, dim3(grid_for(d_rows * chunks)), dim3(256), 0, s, dense, d_ld_b, ddst, ldw_b,
                       d_rows, chunks);
    return hipGetLastError();
  }
  return hipSuccess;
}

}  // namespace spense
