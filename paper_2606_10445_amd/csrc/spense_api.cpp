// Host side of libspense: argument validation (no device synchronisation except in
// spense_compress), work planning and kernel dispatch.  See include/spense.h.
#include <hip/hip_runtime.h>

#include <cmath>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "../../include/spense.h"
#include "spense_internal.h"

namespace {

// The last error message of this thread (a fixed buffer: no call allocates host memory).
thread_local char g_err[512];

int vfail(int code, const char* fmt, va_list ap) {
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  return code;
}

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vfail(code, fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return SPENSE_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int esize(int32_t dtype) { return dtype == SPENSE_FP8_E4M3FN ? 1 : 2; }

// Per-device cache of "is this a gfx950" (0 unknown, 1 yes, 2 no).
std::atomic<int> g_arch[64];

int check_device();

// Arguments of the quantisation calls.
int check_quant_args(const void* src, int32_t type, int64_t M, int64_t K, int64_t ld, const uint8_t* q, int64_t ldq,
                     const float* scales, const char* what) {
  if (type != SPENSE_BF16 && type != SPENSE_F32) return fail(SPENSE_ERR_ARG, "%s type %d is not bf16 or f32", what, type);
  if (M < 0 || K < 0) return fail(SPENSE_ERR_ARG, "negative size");
  if (M > INT32_MAX) return fail(SPENSE_ERR_ARG, "M too large");
  if (M == 0) return SPENSE_OK;
  if (!scales) return fail(SPENSE_ERR_ARG, "scales is NULL");
  if (K > 0 && (!src || !q)) return fail(SPENSE_ERR_ARG, "%s or q is NULL", what);
  if (ld < K || ldq < K) return fail(SPENSE_ERR_ARG, "leading dimension below K");
  return SPENSE_OK;
}

int check_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(SPENSE_ERR_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= 64) return fail(SPENSE_ERR_DEVICE, "device index %d out of range", dev);
  int st = g_arch[dev].load(std::memory_order_relaxed);
  if (st == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return fail(SPENSE_ERR_HIP, "hipGetDeviceProperties failed");
    st = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
    g_arch[dev].store(st, std::memory_order_relaxed);
  }
  if (st != 1) return fail(SPENSE_ERR_DEVICE, "libspense needs a gfx950 (MI355X) device");
  return SPENSE_OK;
}

int layout_impl(int64_t N, int64_t K, int32_t dtype, int32_t split, int64_t dense_begin, spense_layout_t* L) {
  if (!L) return fail(SPENSE_ERR_ARG, "layout: out is NULL");
  if (dtype != SPENSE_FP8_E4M3FN && dtype != SPENSE_BF16) return fail(SPENSE_ERR_ARG, "unknown dtype %d", dtype);
  if (split != SPENSE_SPLIT_OUTPUT && split != SPENSE_SPLIT_INPUT)
    return fail(SPENSE_ERR_ARG, "unknown split %d", split);
  if (N < 0 || K < 0) return fail(SPENSE_ERR_ARG, "negative shape N=%lld K=%lld", (long long)N, (long long)K);
  if (N > INT32_MAX || K > INT32_MAX) return fail(SPENSE_ERR_ARG, "shape too large");
  if (K % 32) return fail(SPENSE_ERR_ALIGN, "K=%lld is not a multiple of 32", (long long)K);
  const int64_t extent = split == SPENSE_SPLIT_OUTPUT ? N : K;
  if (dense_begin < 0 || dense_begin > extent)
    return fail(SPENSE_ERR_ARG, "dense_begin=%lld outside [0, %lld]", (long long)dense_begin, (long long)extent);
  if (split == SPENSE_SPLIT_INPUT && dense_begin % 32)
    return fail(SPENSE_ERR_ALIGN, "input-split dense_begin=%lld is not a multiple of 32", (long long)dense_begin);
  const int es = esize(dtype);
  if (split == SPENSE_SPLIT_OUTPUT) {
    L->sparse_rows = dense_begin;
    L->sparse_cols = K;
    L->dense_rows = N - dense_begin;
    L->dense_cols = K;
  } else {
    L->sparse_rows = N;
    L->sparse_cols = dense_begin;
    L->dense_rows = N;
    L->dense_cols = K - dense_begin;
  }
  L->values_ld = L->sparse_cols / 2;
  L->meta_ld = L->sparse_cols / 32;
  L->dense_ld = L->dense_cols;
  L->values_bytes = (size_t)(L->sparse_rows * L->values_ld * es);
  L->meta_bytes = (size_t)(L->sparse_rows * L->meta_ld * 4);
  L->dense_bytes = (size_t)(L->dense_rows * L->dense_ld * es);
  return ok();
}

constexpr int64_t kTileRows = 16, kTileCols = 512;  // tiled layout: rows x logical columns

int tiled_impl(int64_t N, int64_t K, int32_t dtype, int32_t split, int64_t dense_begin, spense_tiled_layout_t* T) {
  if (!T) return fail(SPENSE_ERR_ARG, "tiled layout: out is NULL");
  spense_layout_t L;
  int rc = layout_impl(N, K, dtype, split, dense_begin, &L);
  if (rc) return rc;
  if (dtype != SPENSE_FP8_E4M3FN) return fail(SPENSE_ERR_ARG, "the tiled layout is defined for fp8 weights only");
  auto cdiv = [](int64_t a, int64_t b) { return (a + b - 1) / b; };
  const bool sp = L.sparse_rows > 0 && L.sparse_cols > 0, de = L.dense_rows > 0 && L.dense_cols > 0;
  T->sparse_tiles = sp ? cdiv(L.sparse_rows, kTileRows) : 0;
  T->sparse_chunks = sp ? cdiv(L.sparse_cols, kTileCols) : 0;
  T->dense_tiles = de ? cdiv(L.dense_rows, kTileRows) : 0;
  T->dense_chunks = de ? cdiv(L.dense_cols, kTileCols) : 0;
  T->values_bytes = (size_t)(T->sparse_tiles * T->sparse_chunks * 4096);
  T->meta_bytes = (size_t)(T->sparse_tiles * T->sparse_chunks * 1024);
  T->dense_bytes = (size_t)(T->dense_tiles * T->dense_chunks * 8192);
  return ok();
}

// Validate a packed descriptor against its own geometry (either layout).
int check_packed(const spense_packed_t* P, spense_layout_t* L) {
  if (!P) return fail(SPENSE_ERR_ARG, "packed is NULL");
  int rc = layout_impl(P->N, P->K, P->dtype, P->split, P->dense_begin, L);
  if (rc) return rc;
  if (P->layout == SPENSE_LAYOUT_TILED) {
    spense_tiled_layout_t T;
    rc = tiled_impl(P->N, P->K, P->dtype, P->split, P->dense_begin, &T);
    if (rc) return rc;
    if (T.values_bytes && (!P->values || !P->meta))
      return fail(SPENSE_ERR_ARG, "values/meta NULL with a non-empty 2:4 region");
    if (T.dense_bytes && !P->dense) return fail(SPENSE_ERR_ARG, "dense NULL with a non-empty dense region");
    if ((T.values_bytes && (!aligned16(P->values) || !aligned16(P->meta))) || (T.dense_bytes && !aligned16(P->dense)))
      return fail(SPENSE_ERR_ALIGN, "tiled buffers must be 16-byte aligned");
    return SPENSE_OK;
  }
  if (P->layout != SPENSE_LAYOUT_ROWMAJOR) return fail(SPENSE_ERR_ARG, "unknown layout %d", P->layout);
  const int es = esize(P->dtype);
  if (L->sparse_rows > 0 && L->sparse_cols > 0) {
    if (!P->values || !P->meta) return fail(SPENSE_ERR_ARG, "values/meta NULL with a non-empty 2:4 region");
    if (P->values_ld < L->values_ld || P->meta_ld < L->meta_ld)
      return fail(SPENSE_ERR_ARG, "values_ld/meta_ld smaller than the region");
    if (!aligned16(P->values) || (P->values_ld * es) % 16)
      return fail(SPENSE_ERR_ALIGN, "values must be 16-byte aligned with a 16-byte multiple row pitch");
    if ((reinterpret_cast<uintptr_t>(P->meta) & 3u)) return fail(SPENSE_ERR_ALIGN, "meta must be 4-byte aligned");
  }
  if (L->dense_rows > 0 && L->dense_cols > 0) {
    if (!P->dense) return fail(SPENSE_ERR_ARG, "dense NULL with a non-empty dense region");
    if (P->dense_ld < L->dense_ld) return fail(SPENSE_ERR_ARG, "dense_ld smaller than the region");
    if (!aligned16(P->dense) || (P->dense_ld * es) % 16)
      return fail(SPENSE_ERR_ALIGN, "dense must be 16-byte aligned with a 16-byte multiple row pitch");
  }
  return SPENSE_OK;
}

// ------------------------------------------------------------------ planning
struct Plan {
  spense::LaunchShape ls;
  spense::GemmArgs args;  // geometry part filled
  size_t ws_bytes;        // device workspace needed (none at present)
};

// Parts of the plan a caller forced (spense_gemm_planned); the defaults leave every
// choice to the planner.
struct Override {
  int kernel = 0, rt = 0, waves = 0, ct = 0, ksplit = 0, wused = 0, wused_d = 0, wused_s = 0, order = -1, xcd = -1,
      u8 = 0, halfrb = -1, xres = 0;
  bool operator==(const Override& o) const {
    return kernel == o.kernel && rt == o.rt && waves == o.waves && ct == o.ct && ksplit == o.ksplit &&
           wused == o.wused && wused_d == o.wused_d && wused_s == o.wused_s && order == o.order && xcd == o.xcd &&
           u8 == o.u8 && halfrb == o.halfrb && xres == o.xres;
  }
};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

constexpr int kMaxWavesUsed = 8;  // row-split kernel: waves per workgroup

// Workgroup shapes the kernels are built for: (row tiles, waves).
const int kShapes[][2] = {{2, 4}, {1, 4}, {2, 8}, {1, 8}, {1, 16}, {4, 4}};

// Check a caller's override against what the kernels are built for and this weight can
// run; fills *o (the planner's defaults for ov == NULL).
int read_override(const spense_plan_override_t* ov, int32_t dtype, bool tiled, Override* o) {
  *o = Override();
  if (!ov) return SPENSE_OK;
  o->kernel = ov->kernel;
  o->rt = ov->row_tiles;
  o->waves = ov->waves;
  o->ct = ov->act_tiles;
  o->ksplit = ov->ksplit;
  o->wused = ov->waves_used;
  o->wused_d = ov->waves_used_dense;
  o->wused_s = ov->waves_used_24;
  o->order = ov->block_order;
  o->xcd = ov->xcd_order;
  o->u8 = ov->u8;
  o->halfrb = ov->half_row_blocks;
  o->xres = ov->resident_x;
  if (o->kernel < 0 || o->kernel > 5) return fail(SPENSE_ERR_ARG, "plan: unknown kernel %d", o->kernel);
  if (o->kernel == 5 && (!tiled || dtype != SPENSE_FP8_E4M3FN))
    return fail(SPENSE_ERR_ARG, "plan: the two-half row-split kernel reads tiled fp8 weights only");
  if (o->kernel == 5 && (o->rt || o->waves || o->ct || o->xres == 2))
    return fail(SPENSE_ERR_ARG, "plan: the two-half row-split kernel has one shape (1 row tile, 8 waves)");
  if (o->kernel == 1 && tiled) return fail(SPENSE_ERR_ARG, "plan: the K-split kernel reads the row-major layout only");
  if (o->kernel >= 3 && dtype != SPENSE_FP8_E4M3FN) return fail(SPENSE_ERR_ARG, "plan: the large-M kernels are fp8 only");
  if (o->ct < 0 || o->ct > 2) return fail(SPENSE_ERR_ARG, "plan: act_tiles %d (0, 1 or 2)", o->ct);
  if (o->ksplit < 0 || o->ksplit > 8) return fail(SPENSE_ERR_ARG, "plan: ksplit %d outside [0, 8]", o->ksplit);
  for (int w : {o->wused, o->wused_d, o->wused_s})
    if (w < 0 || w > kMaxWavesUsed) return fail(SPENSE_ERR_ARG, "plan: waves used %d outside [0, 8]", w);
  if (o->order < -1 || o->order > 2) return fail(SPENSE_ERR_ARG, "plan: block_order %d", o->order);
  if (o->xcd < -1 || o->xcd > 1) return fail(SPENSE_ERR_ARG, "plan: xcd_order %d", o->xcd);
  if (o->u8 < 0 || o->u8 > 1) return fail(SPENSE_ERR_ARG, "plan: u8 %d", o->u8);
  if (o->halfrb < -1) return fail(SPENSE_ERR_ARG, "plan: half_row_blocks %d", o->halfrb);
  if (o->xres < 0 || o->xres > 2) return fail(SPENSE_ERR_ARG, "plan: resident_x %d", o->xres);
  if (o->rt || o->waves) {
    bool okshape = false;
    if (o->kernel == 1) {
      for (const auto& sh : kShapes) okshape = okshape || (sh[0] == o->rt && sh[1] == o->waves);
    } else if (o->kernel == 2) {
      okshape = (o->rt == 1 && (o->waves == 4 || o->waves == 8)) || (o->rt == 2 && o->waves == 4);
    } else if (o->kernel == 3) {
      okshape = o->rt == 0 && (o->waves == 4 || o->waves == 8);
    } else if (o->kernel == 4) {
      okshape = o->rt == 0 && o->waves == 8;
    }
    if (!okshape)
      return fail(SPENSE_ERR_ARG, "plan: no kernel %d built for %d row tiles x %d waves", o->kernel, o->rt, o->waves);
  }
  return SPENSE_OK;
}

constexpr int kCUs = 256;  // compute units of an MI355X
// XCD-aware order of the large-M grids: each XCD takes GT of the T token blocks (the
// divisor of T nearest 4 whose token groups T / GT divide the 8 XCDs; 0 = none) and every
// RC-th row block (RC = 8 / (T / GT)).
int64_t xcd_token_group(int64_t T) {
  int64_t GT = 0;
  for (int64_t d = 1; d <= T; ++d)
    if (T % d == 0 && 8 % (T / d) == 0 && (GT == 0 || std::llabs(d - 4) < std::llabs(GT - 4))) GT = d;
  return GT;
}

// 256 x 256 kernel: the row blocks at the end of the last region that run as 256 x 128
// tiles after every full tile.  With whole tiles the last round of the grid leaves CUs
// idle: gate / up at M = 2048 is 800 tiles of 65 (2:4) and 84 us (dense) on 256 CUs, so
// some CUs run four tiles while the average load is 218 us (per-workgroup timestamps on
// MI355X).  Smaller tiles dispatched last fill that round.  Measured (us, half tiles'
// row blocks 0 -> the best): gate / up M = 2048 277 -> 248 (12-24), down and o at M =
// 2048 240 -> 220 and 92 -> 87 (4), Seed-OSS gate 278 -> 257 (12); q at M = 2048 (one
// round of 256 tiles) only loses.  The rule: with more than one round, half tiles worth
// about an eighth of the work (a dense step costing 1.28 2:4 steps, a half tile 0.6 of a
// full one), rounded up to whole XCD row classes.
int64_t choose_half_rows(const spense::Region* regs, int nreg, int64_t T, int64_t M, int64_t rc) {
  double W = 0;
  int64_t rbtot = 0;
  double wl = 0;
  int64_t rbl = 0;
  for (int i = 0; i < nreg; ++i) {
    const int64_t rb = ceil_div(regs[i].rows, 256);
    const double w = (double)ceil_div(regs[i].kbound, 128) + 1.28 * (double)ceil_div(regs[i].kend - regs[i].kbound, 128);
    W += (double)(rb * T) * w;
    rbtot += rb;
    wl = w;
    rbl = rb;
  }
  if (rbtot * T <= kCUs || wl <= 0) return 0;
  const double per_rb = (double)ceil_div(M, 128) * 0.6 * wl;
  int64_t rh = (int64_t)std::ceil(W / 8.0 / per_rb);
  if (rc > 1) rh = ceil_div(rh, rc) * rc;
  return std::min(rh, rbl);
}

constexpr int64_t kBigMinM = 65;       // tokens from which the large-M kernel is used (fp8)
constexpr int64_t kBigMinTiles = 120;  // and workgroup tiles (128 rows x 256 tokens) it needs

// Waves (16-row tiles) per workgroup for each kind of region, w[kind] in [1, wmax]:
// region i (rows[i] rows, kind[i] in {0, 1}, tile[i] the weight bytes one wave streams)
// gets ceil(rows / (16 rt w)) workgroups per token block and K slice (mult).  Model: with
// W workgroups on kCUs CUs the time is ceil(W / kCUs) rounds of the largest workgroup,
// whose cost is its waves' weight bytes plus the activation staging (x_cost); one active
// wave costs as two (alone it keeps too few loads in flight for the CU's share of HBM).
// Ties go to more workgroups (more CUs streaming), then to more waves in the smallest
// workgroup.  Measured on MI355X (graph replay, tiled fp8, M = 1 / 32 / 64, us): q 8192 x
// 5120 with (dense 1, 2:4 3) waves 8.85 / 11.71 / 14.40, with (2, 2) 7.95 / 10.79 / 13.40;
// gate / up with (5, 8) 18.04 / 20.40 / 23.72, with (5, 7) 17.82 / 19.89 / 23.13.
void pick_waves(int n, const int64_t* rows, const int* kind, const double* tile, int rt, int wmax, int64_t mult,
                double x_cost, int w_out[2]) {
  bool has1 = false;
  for (int i = 0; i < n; ++i) has1 = has1 || kind[i] == 1;
  double best = 0;
  int64_t best_wg = 0;
  int best_min = 0;
  w_out[0] = w_out[1] = wmax;
  for (int w0 = 1; w0 <= wmax; ++w0)
    for (int w1 = 1; w1 <= (has1 ? wmax : 1); ++w1) {
      const int wk[2] = {w0, w1};
      int64_t wg = 0;
      double big = 0;
      int wmin = wmax;
      for (int i = 0; i < n; ++i) {
        const int w = wk[kind[i]];
        wg += ceil_div(rows[i], 16 * rt * w) * mult;
        big = std::max(big, std::max(w, 2) * tile[i]);
        wmin = std::min(wmin, w);
      }
      const double t = (double)ceil_div(wg, kCUs) * (big + x_cost);
      const bool tie = best_wg != 0 && t <= best * (1 + 1e-9) && t >= best * (1 - 1e-9);
      if (best_wg == 0 || t < best * (1 - 1e-9) || (tie && (wg > best_wg || (wg == best_wg && wmin > best_min)))) {
        best = t;
        best_wg = wg;
        best_min = wmin;
        w_out[0] = w0;
        w_out[1] = w1;
      }
    }
}

// Row-split kernel: 16-row tiles per workgroup, per region (pick_waves; the dense region
// of an output-split weight, whose rows carry more bytes, gets fewer, so that the
// workgroups are alike in bytes).
void choose_rows_per_group(spense::Region* regs, int nreg, int rt, int waves, int ct, int mblocks, int64_t K, int es,
                           double sparse_cost, int ksplit, const Override& ov) {
  double tile_b[2];
  int64_t rows[2];
  const int kind[2] = {0, 1};  // one kind per region
  for (int i = 0; i < nreg; ++i) {
    tile_b[i] = 16.0 * rt * (sparse_cost * regs[i].kbound + (double)es * (K - regs[i].kbound)) / ksplit;
    rows[i] = regs[i].rows;
  }
  const double x_cost = 0.25 * 16.0 * ct * K * es / ksplit;
  int bw[2];
  pick_waves(nreg, rows, kind, tile_b, rt, waves, (int64_t)mblocks * ksplit, x_cost, bw);
  const int ew = ov.wused, ewd = ov.wused_d, ews = ov.wused_s;  // forced: every region / per kind
  for (int i = 0; i < nreg; ++i) {
    const int ek = regs[i].kbound == 0 ? ewd : ews;
    regs[i].wused = ew > 0 ? std::min(ew, waves) : (ek > 0 ? std::min(ek, waves) : bw[i]);
    regs[i].nrb = (int32_t)(ceil_div(regs[i].rows, 16 * rt * regs[i].wused) * ksplit);
  }
}

// Row-split kernel: number of K slices.  Slicing K multiplies the waves of a weight with
// few 16-row tiles, at the price of an fp32 partial-sum pass (the reduction launch).
// Measured on the q / k / o / down shapes (tiled fp8, graph replay, with the reduction
// that issues every slice's load before adding): it pays for one block of tokens
// (several blocks already multiply the workgroups) on weights with fewer than 1024
// tiles, when each slice keeps enough chunks.  k / v (64 tiles, 10 chunks): 4 slices,
// 5-8% faster at every M.  o (320 tiles, 16 chunks): 3 slices from 17 tokens, 3-9%
// (Seed-OSS o, 20 chunks: 4 slices, 7-13%); none at 1-16.  down (320 tiles, 50 chunks):
// 4 slices, up to 1.5x at 17-64 tokens and 4-12% at 1-16 (all dense: 2 or 4 slices
// within run-to-run noise from 17 tokens; 4 kept).
// q (512 tiles, 10 chunks): 2 slices lose 12-15% at 32-64 tokens, so none.
int choose_ksplit(const spense::Region* regs, int nreg, int ct, int mblocks, int64_t chunks, int64_t M,
                  const Override& ov) {
  int64_t tiles = 0;
  bool has_24 = false;
  for (int i = 0; i < nreg; ++i) {
    tiles += ceil_div(regs[i].rows, 16);
    has_24 = has_24 || (regs[i].kbound > 0 && regs[i].rows > 0);
  }
  int S = 1;
  const int64_t by_tiles = ceil_div(1024, std::max<int64_t>(tiles, 1));
  // Weights of 128 tiles or more with one activation tile (M <= 16): only if every slice
  // keeps at least 12 chunks; a weight with a 2:4 part takes up to 4 slices (its chunks
  // carry fewer bytes, so the waves of one tile keep too few in flight), an all-dense one
  // 2 and only above 8 tokens.  Measured on down (5120 x 25600, us, slices 1 / 2 / 4):
  // 25% dense M = 1: 23.6 / 21.4 / 21.0, M = 16: 23.3 / 21.7 / 21.6; all dense M = 1:
  // 25.1 / 25.5 / 26.3, M = 4: 23.9 / 24.6 / 26.3, M = 16: 27.7 / 25.6 / 27.3.  More
  // activation tiles: slices of at least 5 chunks, below 512 tiles.
  if (mblocks == 1 && tiles < 1024) {
    if (tiles < 128) {
      // few rows (k / v): slices of two or more chunks pay at every M
      S = (int)std::max<int64_t>(1, std::min<int64_t>({4, by_tiles, chunks / 2}));
    } else if (ct == 1) {
      S = (int)std::max<int64_t>(1, std::min<int64_t>({4, by_tiles, chunks / 12}));
      if (!has_24) S = M > 8 ? std::min(S, 2) : 1;
    } else if (tiles < 512) {
      S = (int)std::max<int64_t>(1, std::min<int64_t>({4, by_tiles, chunks / 5}));
    }
  } else if (mblocks == 2 && tiles < 512) {
    // Two token blocks (65-128 tokens), tiled layout, measured (us, slices 1 / 2 / 3 / 4):
    // down (320 tiles, 50 chunks) M = 80: 48.3 / 38.5 / 37.0 / 43.8, M = 128: 50.6 /
    // 40.6 / 38.9 / 45.9; k (64 tiles, 10 chunks) M = 80: 10.8 / 9.7 / 9.4 / 8.8, M = 128:
    // 10.9 / 9.9 / 9.8 / 8.9; o (320 tiles, 16 chunks) M = 128: 19.0 / 19.8 / 21.4 / 25.1.
    // Few rows: slices of two or more chunks; otherwise slices of at least 16 chunks.
    S = (int)std::max<int64_t>(1, tiles < 128 ? std::min<int64_t>({4, by_tiles, chunks / 2})
                                              : std::min<int64_t>({3, by_tiles, chunks / 16}));
  } else if (mblocks == 3 && tiles < 512 && chunks >= 32) {
    // 129-192 tokens: two slices of a long K only (down M = 192: 53.3 / 50.2 / 70.9; o,
    // 16 chunks, M = 192: 20.4 / 23.6; four token blocks lose with any slices)
    S = 2;
  }
  if (ov.ksplit >= 1) S = (int)std::max<int64_t>(1, std::min<int64_t>(ov.ksplit, chunks));
  return S;
}

// Chunk boundaries of S slices of a row-split region with equal byte cost (2:4 chunks
// cost sparse_cost bytes per logical column, dense chunks es).
void slice_cuts(spense::Region& r, int S, int64_t kc, int es, double sparse_cost) {
  const int64_t n_sp = ceil_div(r.kbound, kc), n_de = ceil_div(r.kend - r.kbound, kc);
  const int64_t nch = n_sp + n_de;
  const double cs = sparse_cost * n_sp, total = cs + (double)es * n_de;
  r.cut[0] = 0;
  for (int s = 1; s < S; ++s) {
    const double c = total * s / S;
    const double k = c <= cs ? c / sparse_cost : n_sp + (c - cs) / es;
    int64_t cut = std::llround(k);
    cut = std::max<int64_t>(r.cut[s - 1] + 1, std::min<int64_t>(cut, nch - (S - s)));
    r.cut[s] = (int32_t)cut;
  }
  r.cut[S] = (int32_t)nch;
  r.ksplit = S;
}

// The plan depends only on the dtype, M and the weight geometry, so equal geometry gets
// the same decomposition and summation order (the dense baseline and a Spense weight
// with no 2:4 part are planned identically).
void make_plan(int32_t dtype, int64_t M, int64_t N, int32_t split, int64_t K, int64_t dense_begin, bool tiled,
               const Override& ov, Plan* pl) {
  using spense::Region;
  memset(pl, 0, sizeof *pl);
  const int es = esize(dtype);
  const int64_t gran = dtype == SPENSE_FP8_E4M3FN ? 128 : 64;  // K per 2:4 instruction
  const double sparse_cost = 0.5 * es + 0.125;                 // bytes per logical 2:4 entry
  int ct = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  if (ov.ct == 1 || ov.ct == 2) ct = std::min(ct, ov.ct);
  pl->ls.ct = ct;
  pl->ls.mblocks = (int)ceil_div(M, 16 * ct);

  // Workgroup shape (measured on MI355X with the gate/up and down shapes):
  //  - one activation tile (M <= 16): 16 rows per workgroup; 4 waves when that gives
  //    >= 4096 waves, else 8 (the waves split K);
  //  - more activation tiles: more rows per workgroup so that each activation fragment
  //    feeds more weight rows, as long as enough workgroups remain.
  int rt, waves;
  auto groups_for = [&](int r) { return ceil_div(N, 16 * r) * pl->ls.mblocks; };
  if (ct == 1) {
    rt = 1;
    waves = groups_for(1) * 4 >= 4096 ? 4 : 8;
  } else {
    rt = groups_for(4) >= 300 ? 4 : 2;
    waves = 4;
  }
  // Row-split workgroups (activations staged once per workgroup in LDS, weights
  // prefetched two chunks ahead) measured faster than K-split on the q/k/o/gate/down
  // shapes at every M > 16, and at M <= 16 whenever there are at least as many 16-row
  // tiles as CUs; with fewer rows the K split gives the single activation tile more
  // parallelism (only the row-split kernel reads the tiled layout).  Eight waves per
  // workgroup: with warmed weights and interleaved repeats they measured as fast as four
  // for one activation tile and up to 1.6x faster for several (q/k/o/gate/down); two row
  // tiles per wave won only on q at M = 256.
  int rows_mode = (tiled || ct > 1 || ceil_div(N, 16) * pl->ls.mblocks >= kCUs) ? 1 : 0;
  if (rows_mode) {
    rt = 1;
    waves = 8;
  }
  if (ov.kernel == 1) rows_mode = 0;  // forced (checked against the layout by read_override)
  if (ov.kernel == 2 || ov.kernel == 5) rows_mode = 1;
  if (rows_mode) {
    rt = 1;
    waves = 8;
  }
  if (ov.rt && ov.kernel < 3) {  // a shape checked against the kernel's list
    rt = ov.rt;
    waves = ov.waves;
  }
  pl->ls.rt = rt;
  pl->ls.waves = waves;
  pl->ls.rows = rows_mode;
  pl->ls.u8 = (ct == 1 && rt == 1 && (waves == 4 || waves == 8) && ov.u8) ? 1 : 0;
  // Many tokens (fp8): 128-row x 256-token workgroup tiles.  Measured on MI355X (q / k /
  // o / gate / down shapes, M = 65 .. 2048, XCD-aware order): it wins above one row-split
  // token block (64 tokens) once there are at least 128 such tiles (gate / up at M = 96 /
  // 128 / 192: 42.5 / 43.2 / 46.0 vs 45.3 / 47.9 / 71.4 us; q at M = 512: 45 vs 54 us; o
  // and down at M = 1024: 60 vs 97 and 156 vs 265 us); with fewer (q below 257 tokens, o
  // and down below 513), the row-split kernel's finer grid keeps more CUs busy.  Since the
  // output tile goes through LDS, 120 tiles suffice (o, down and Seed-OSS o at M = 513 /
  // 576 / 700, 120 tiles: 50.7 / 50.6 / 51.5, 140.9 / 140.3 / 143.8 and 62.8 / 61.3 /
  // 63.2 us against 58.6 / 57.4 / 62.7, 154.0 / 154.3 / 171.9 and 70.7 / 70.1 / 77.4 on
  // row-split; at 80 tiles, M = 257-512, row-split stays ahead: o 33 against 50).
  // Up to five 64-token blocks the row-split kernel also beats a grid of fewer than 160
  // such tiles (q, 128 tiles, at M = 257 / 320: 31.7 / 31.9 against 35.7 / 35.1 us; at
  // 384, six blocks, 45.1 against 35.6).
  const int64_t tiles128 = ceil_div(N, 128) * ceil_div(M, 256);
  int big = (dtype == SPENSE_FP8_E4M3FN && M >= kBigMinM && tiles128 >= kBigMinTiles &&
             !(tiles128 < 160 && ceil_div(M, 64) <= 5))
                ? 1
                : 0;
  // 256-row x 256-token tiles (tiled weights) once that grid has at least 160 workgroups:
  // measured on MI355X (us, 128 x 256 tiles -> 256 x 256): gate / up at M = 1024 / 2048
  // 177 / 312 -> 159 / 291, Seed-OSS gate 178 / 316 -> 168 / 290, down and o at M = 2048
  // (160 workgroups) 313 -> 267 and 120 -> 100, q at M = 2048 95 -> 91; with fewer
  // workgroups it loses (q at M = 1024, 128 workgroups: 49 -> 84; down at M = 1024, 80: 159
  // -> 279).  A ragged last token block used to favour the 128 x 256 kernel at two or
  // three blocks; since both kernels write their output tile through LDS and the 256 x
  // 256 grid ends in 256 x 128 tiles, the 256 x 256 kernel wins there too (gate / up at
  // M = 257 / 300 / 513 / 576 / 700: 65.8 / 66.7 / 82.9 / 84.4 / 87.0 against 68.2 / 67.9
  // / 100.3 / 102.8 / 108.8 us; Seed-OSS gate alike).
  if (big && tiled) {
    const int64_t rb256 = split == SPENSE_SPLIT_OUTPUT
                              ? ceil_div(dense_begin, 256) + ceil_div(N - dense_begin, 256)
                              : ceil_div(N, 256);
    const int64_t tb256 = ceil_div(M, 256);
    if (rb256 * tb256 >= 160) big = 2;
  }
  // Two 64-token halves per row-split workgroup (spense_gemm_rows2_kernel: 128 tokens a
  // block, four token tiles, one row tile, eight waves).  Each weight chunk
  // feeds twice the tokens of the row-split kernel's, but the 128 KB of staged
  // activations leave one workgroup per CU, so it needs several rounds of workgroups.
  // Measured on MI355X (graph replay, us, planner's choice -> two halves): with one
  // 128-token block (M = 65 / 100 / 128) it wins from 768 row tiles of 16 (gate / up
  // 25600 x 5120 37.1 / 37.0 / 37.3 -> 29.1 / 29.5 / 31.2; 16384 x 5120 29.7 / 29.8 /
  // 30.1 -> 23.7 / 24.1 / 25.8; 12288 x 5120 22.0 / 21.6 / 22.1 -> 21.3 / 20.5 / 20.8;
  // 20480 x 4096 and the input-split 25600 x 5120 alike) and loses below (q, 512 tiles:
  // 15.9 / 16.4 / 16.2 -> 18.2 / 19.0 / 19.2; 10240 x 5120 by 2-3 us).  With two blocks
  // (M = 129 .. 256) the weight is read twice, so it only replaces row-split grids of
  // three or four token blocks (q at M = 224 / 256 29.7 / 29.6 -> 24.0 / 24.0, at 160 /
  // 192 21.9 / 22.2 -> 23.6 / 23.8; 10240 x 5120 at 160 / 192 / 224 25.1 / 26.5 / 31.0
  // -> 25.1 / 25.1 / 25.2; 12288 x 5120 at 160 / 224 30.9 / 43.5 -> 28.4 / 29.7; the
  // input-split 16384 x 8192 at 160 / 256 55.5 / 54.1 -> 40.8 / 45.2), not the large-M
  // kernels (gate / up at M = 160 / 256: 37.7 / 43.5 against 56.3 / 59.6).
  // On weights with fewer row tiles but a long K it runs with K slices instead (partials
  // reduced as for the row-split kernel): down 5120 x 25600 (50 chunks) at M = 65 / 100 /
  // 128 39.4 / 37.7 / 39.0 -> 33.3 / 36.2 / 37.4 with 6 slices (4: 35.9 / 37.6 / 38.9),
  // at M = 256 61.2 -> 57.4 with 3; Seed-OSS down 5120 x 27648 41.1 / 39.6 / 41.1 -> 33.8
  // / 36.3 / 38.1 and 64.9 -> 59.5; Seed-OSS o 5120 x 10240 (20 chunks) at M = 65 / 100
  // 24.4 / 22.1 -> 20.1 / 21.8 with 4 (M = 128: 22.8 against 23.0).  At 129-192 tokens the
  // row-split kernel's three blocks stay ahead (down at M = 160 / 192 49.0 / 50.3 against
  // 55.6 / 55.6), as they do on o (16 chunks), q and k at every M here.
  // Past 256 tokens (to 768), on weights of 256 to 767 row tiles (the large-M grids have
  // too few tiles there), it halves the row-split kernel's token blocks (us, planner's
  // choice -> two halves): down 5120 x 25600 at M = 448 / 512 / 640 / 768 118.6 / 119.1 /
  // 143.4 / 150.7 -> 100.8 / 102.9 / 124.2 / 120.8, at M = 300 with 2 slices 91.5 ->
  // 74.8; Seed-OSS down alike; o 5120 x 8192 at M = 448 / 512 / 640 / 768 43.7 / 44.5 /
  // 50.7 / 53.1 -> 37.5 / 38.7 / 44.5 / 43.9; q (512 tiles) at M = 300 / 384 33.0 / 35.6
  // -> 30.7 / 31.5, also against the 128 x 256 kernel.  Not o and down at 321-384 tokens
  // (six 64-token blocks: down 76.4 against 78.0) nor from 769 (seven 128-token blocks:
  // down at 896 149.6 against 201.2), nor q from 385 on (the 128 x 256 kernel, 36.6 /
  // 39.4 at 448 / 512 against 47.7 / 48.6).
  bool rows2 = ov.kernel == 5;
  int rows2_ks = 1;
  if (ov.kernel == 0 && !ov.rt && !ov.waves && !ov.ct && ov.ksplit <= 1 && !ov.wused && !ov.wused_d &&
      !ov.wused_s && !ov.u8 && !ov.xres && tiled && dtype == SPENSE_FP8_E4M3FN && M > 64 && M <= 768) {
    const int64_t rtiles = ceil_div(N, 16);
    const int64_t kch = split == SPENSE_SPLIT_INPUT ? ceil_div(dense_begin, 512) + ceil_div(K - dense_begin, 512)
                                                    : ceil_div(K, 512);
    if (M <= 256) {
      rows2 = M <= 128 ? rtiles >= 768 : (!big && rtiles >= (M <= 192 ? 640 : 512));
      if (!rows2 && ov.ksplit < 1 && rtiles < 768) {
        if (kch >= 40 && (M <= 128 || (M > 192 && !big))) {
          rows2 = true;
          rows2_ks = M <= 128 ? 6 : 3;
        } else if (kch >= 20 && M <= 96) {
          rows2 = true;
          rows2_ks = 4;
        }
      }
    } else if (rtiles >= 256 && rtiles < 768) {
      if (M > 384) {
        rows2 = !big || rtiles < 512;  // down at 640 (128 x 256, 120 tiles) 143.9 against 124.2
      } else if (rtiles >= 512) {
        rows2 = true;
      } else if (M <= 320 && kch >= 40 && ov.ksplit < 1) {
        rows2 = true;
        rows2_ks = 2;
      }
    }
  }
  if (ov.kernel == 1 || ov.kernel == 2 || rows2) big = 0;
  if (ov.kernel == 3) big = 1;  // fp8 (checked by read_override)
  if (ov.kernel == 4) big = tiled ? 2 : 1;  // the 256 x 256 kernel reads the tiled layout
  pl->ls.big = big;
  if (rows2) {
    pl->ls.ct = 4;
    pl->ls.mblocks = (int)ceil_div(M, 128);
    pl->ls.rt = 1;
    pl->ls.waves = 8;
  }
  const int big_rows = big == 2 ? 256 : 128;  // rows of a large-M workgroup tile
  if (big) pl->ls.waves = (big == 1 && ov.waves == 4) ? 4 : 8;
  const int64_t tblocks = ceil_div(M, 256);

  Region regs[2];
  int nreg = 0;
  auto add = [&](int64_t row0, int64_t rows, int64_t kbound, int64_t dro, int64_t dco) {
    Region r;
    memset(&r, 0, sizeof r);
    r.row0 = (int32_t)row0;
    r.rows = (int32_t)rows;
    r.kbound = (int32_t)kbound;
    r.dense_row_off = (int32_t)dro;
    r.dense_col_off = (int32_t)dco;
    r.kend = (int32_t)K;
    r.wused = waves;
    r.ksplit = 1;
    r.nrb = (int32_t)(big ? ceil_div(rows, big_rows) * tblocks : ceil_div(rows, 16 * rt));
    // cut [0, K) into `waves` parts of equal byte cost, on multiples of the instruction K
    const double cs = sparse_cost * kbound, total = cs + es * (double)(K - kbound);
    r.cut[0] = 0;
    for (int w = 1; w < waves; ++w) {
      const double c = total * w / waves;
      const double k = c <= cs ? c / sparse_cost : kbound + (c - cs) / es;
      int64_t kr = (int64_t)std::llround(k / gran) * gran;
      kr = std::max<int64_t>(r.cut[w - 1], std::min<int64_t>(kr, K));
      r.cut[w] = (int32_t)kr;
    }
    r.cut[waves] = (int32_t)K;
    regs[nreg++] = r;
  };
  if (split == SPENSE_SPLIT_OUTPUT) {
    // dense rows first: their workgroups carry more bytes, so dispatching them early
    // keeps them out of the tail
    if (N - dense_begin > 0) add(dense_begin, N - dense_begin, 0, dense_begin, 0);
    if (dense_begin > 0) add(0, dense_begin, K, 0, 0);
  } else if (N > 0) {
    add(0, N, dense_begin, 0, dense_begin);
  }
  int ksplit = 1;
  if (rows_mode && !big) {
    // chunks of 4 instruction steps: 512 logical columns (fp8), 256 (bf16)
    const int64_t kc = dtype == SPENSE_FP8_E4M3FN ? 512 : 256;
    int64_t chunks = 0;
    for (int i = 0; i < nreg; ++i) chunks = std::max(chunks, ceil_div(regs[i].kbound, kc) + ceil_div(K - regs[i].kbound, kc));
    if (rows2)
      ksplit = (int)std::max<int64_t>(1, std::min<int64_t>(ov.ksplit >= 1 ? ov.ksplit : rows2_ks, chunks));
    else
      ksplit = chunks > 0 ? choose_ksplit(regs, nreg, pl->ls.ct, pl->ls.mblocks, chunks, M, ov) : 1;
    for (int i = 0; i < nreg; ++i) slice_cuts(regs[i], ksplit, kc, es, sparse_cost);
    choose_rows_per_group(regs, nreg, rt, waves, pl->ls.ct, pl->ls.mblocks, K, es, sparse_cost, ksplit, ov);
    // One or two token tiles, tiled fp8, 8 waves, no K slices: the activations of the
    // whole K range stay in LDS (at most 160 KB: 20 chunks with one token tile, 10 with
    // two) and each wave streams its weights with no barrier after the first.  Measured
    // on MI355X (graph replay, us, staged -> resident): gate / up at M = 1 / 8 / 16 17.9 /
    // 17.6 / 17.9 -> 16.9 / 17.0 / 17.3, at M = 17 / 24 / 32 19.1 / 19.4 / 20.0 -> 18.6 /
    // 18.7 / 19.3; k
    // at M = 1 5.8 -> 5.5 (but K-sliced), q and o at M = 16 8.7 / 9.8 -> 8.4 / 9.6.  Where
    // a workgroup has few active waves the first barrier is not repaid (q and o at M = 1
    // 8.0 / 9.2 -> 8.2 / 9.5), nor on down's K slices (M = 1 / 16: 19.4 / 20.4 -> 19.9 /
    // 20.8), so it is used where every region gives a workgroup at least 4 waves.
    if (!rows2 && ct <= 2 && rt == 1 && waves == 8 && tiled && dtype == SPENSE_FP8_E4M3FN && ksplit == 1 && ov.xres != 1 &&
        chunks * 8192 * ct <= 160 * 1024) {
      bool wide = true;
      for (int i = 0; i < nreg; ++i) wide = wide && regs[i].wused >= 4;
      if (wide || ov.xres == 2) pl->ls.xres = (int)chunks;
    }
  }
  // 256 x 256 kernel: the last row blocks of the last region may run as 256 x 128 tiles
  // after every 256 x 256 tile, to fill the grid's last round
  int64_t half_rb = 0, rbl = 0;
  if (big == 2 && nreg > 0) {
    rbl = ceil_div(regs[nreg - 1].rows, 256);
    const int64_t GT = xcd_token_group(tblocks);
    const int64_t rc = GT > 0 ? 8 / (tblocks / GT) : 1;
    half_rb = ov.halfrb >= 0 ? std::min<int64_t>(ov.halfrb, rbl) : choose_half_rows(regs, nreg, tblocks, M, rc);
    regs[nreg - 1].nrb = (int32_t)((rbl - half_rb) * tblocks);
  }
  spense::GemmArgs& a = pl->args;
  a.nreg = nreg;
  int32_t groups = 0;
  for (int i = 0; i < nreg; ++i) {
    regs[i].wg0 = groups;
    groups += regs[i].nrb;
    a.reg[i] = regs[i];
  }
  a.groups = groups;
  a.tiled = tiled ? 1 : 0;
  a.tblocks = (int32_t)tblocks;
  // 256 x 256 kernel: blocks of 192 tokens where they need no more blocks than 256-token
  // ones (257-384, 513-576, ... tokens): the same grid, a quarter of each tile's MMAs and
  // activation copies fewer.  Measured on MI355X (graph replay, us, one box, 256 -> 192):
  // gate / up at M = 257 / 300 / 384 / 540 / 576 65.8 / 65.7 / 66.4 / 86.1 / 87.0 -> 62.8 /
  // 63.3 / 65.1 / 81.9 / 82.8; Seed-OSS gate 66.8 / 66.8 / 67.4 / 95.5 / 96.0 -> 63.3 /
  // 63.6 / 65.9 / 88.0 / 89.3.
  a.btok = big == 2 && M > 256 && ceil_div(M, 192) == tblocks ? 192 : 0;
  a.hg0 = groups;
  a.hrb0 = (int32_t)(rbl - half_rb);
  a.hper = (int32_t)ceil_div(M, 128);
  a.groups = (int32_t)(groups + half_rb * a.hper);
  // Large-M kernel, XCD-aware order: workgroups are dealt to the 8 XCDs round-robin
  // (XCD = id % 8).  Each XCD is given GT token blocks (up to 4) and every RC-th row
  // block, so a weight block is fetched into an XCD's L2 once for GT token blocks and
  // the activations of those blocks stay there.  Needs T / GT to divide 8 and the row
  // blocks to split evenly into RC classes; otherwise the plain order.  Measured on
  // MI355X (gate / up and down at M = 2048): 9% faster than one token block per XCD.
  a.xgt = a.xrc = a.xg1 = 0;
  if (big && ov.xcd != 0) {
    // GT: the divisor of T nearest 4 whose token groups (T / GT) divide the 8 XCDs; the
    // row blocks beyond the last whole set of RC classes keep the plain order after the
    // others
    const int64_t T = tblocks;
    const int64_t GT = xcd_token_group(T);
    int64_t rbtot = -half_rb;  // row blocks of the full-size tiles
    for (int i = 0; i < nreg; ++i) rbtot += ceil_div(regs[i].rows, big_rows);
    if (GT > 0) {
      const int64_t RC = 8 / (T / GT), rbx = rbtot / RC * RC;
      if (rbx > 0) {
        a.xgt = (int32_t)GT;
        a.xrc = (int32_t)RC;
        a.xg1 = (int32_t)(rbx * T);
      }
    }
  }
  // Row-split kernel with several token blocks: the blocks of a row group on one XCD
  // (workgroups are dealt to the 8 XCDs round-robin), so that they share its L2 for the
  // weight rows.  Measured on MI355X (tiled, M = 128 / 256 / 512, us): down 53.8 / 65.6 /
  // 125.5 -> 50.5 / 65.0 / 123.2; q 18.3 / 34.7 / 46.0 -> 18.2 / 33.3 / 45.8; Seed-OSS q
  // 19.3 / 38.0 / 47.6 -> 19.2 / 35.5 / 47.0; o and k within 1%.  Needs the row groups
  // to split evenly over the XCDs.
  a.mblk = pl->ls.mblocks;
  a.rorder = pl->ls.rows && !big && !rows2 && pl->ls.mblocks > 1 ? (ov.order >= 0 ? ov.order : 2) : 0;
  if (a.rorder == 2 && a.groups % 8) a.rorder = 0;
  if (rows2) pl->ls.rows = 2;
  // K-sliced regions keep fp32 partial sums: slices x M x N floats
  pl->ws_bytes = ksplit > 1 ? (size_t)ksplit * (size_t)M * (size_t)N * sizeof(float) : 0;
}

// The plans of the last few calls of this thread, keyed by everything make_plan reads
// (the plan depends on nothing else): a decode loop that repeats one geometry plans once.
struct PlanKey {
  int32_t dtype, split;
  int64_t M, N, K, dense_begin;
  bool tiled;
  Override ov;
  bool operator==(const PlanKey& o) const {
    return dtype == o.dtype && split == o.split && M == o.M && N == o.N && K == o.K && dense_begin == o.dense_begin &&
           tiled == o.tiled && ov == o.ov;
  }
};
constexpr int kPlanCache = 8;
struct PlanCache {
  PlanKey key[kPlanCache];
  Plan plan[kPlanCache];
  int used = 0, next = 0;
};
thread_local PlanCache g_plans;

// Dispatch log level (spense_set_log); the environment is read once, at load.
std::atomic<int> g_log{0};
__attribute__((constructor)) void read_log_env() {
  const char* e = getenv("SPENSE_LOG");
  if (e) g_log.store(atoi(e));
}

const char* kernel_name(const spense::LaunchShape& ls) {
  if (ls.big == 2) return "large-M 256x256";
  if (ls.big == 1) return "large-M 128x256";
  if (ls.glu) return "row-split, gate/up paired";
  if (ls.rows == 2) return "row-split, two 64-token halves";
  return ls.rows ? "row-split" : "K-split";
}

void log_plan(const char* what, int32_t dtype, int64_t M, int64_t N, int32_t split, int64_t K, int64_t dense_begin,
              bool tiled, const spense::LaunchShape& ls, const spense::GemmArgs& a, size_t ws_bytes) {
  fprintf(stderr,
          "spense: %s dtype=%s M=%lld N=%lld K=%lld split=%s dense_begin=%lld layout=%s -> %s act_tiles=%d "
          "row_tiles=%d waves=%d token_blocks=%d block_tokens=%d workgroups=%d regions=%d k_slices=%d "
          "resident_x=%d half_tile_groups=%d workspace=%zu\n",
          what, dtype == SPENSE_FP8_E4M3FN ? "fp8" : "bf16", (long long)M, (long long)N, (long long)K,
          split == SPENSE_SPLIT_OUTPUT ? "output" : "input", (long long)dense_begin, tiled ? "tiled" : "row-major",
          kernel_name(ls), ls.ct, ls.rt, ls.waves, ls.big ? a.tblocks : ls.mblocks,
          ls.big == 2 ? (a.btok > 0 ? a.btok : 256) : (ls.big ? 256 : (ls.rows == 2 ? 128 : 16 * ls.ct)), a.groups,
          a.nreg, a.nreg > 0 ? a.reg[0].ksplit : 1,
          ls.xres, ls.big == 2 ? a.groups - a.hg0 : 0, ws_bytes);
}

const Plan& cached_plan(int32_t dtype, int64_t M, int64_t N, int32_t split, int64_t K, int64_t dense_begin, bool tiled,
                        const Override& ov) {
  PlanCache& c = g_plans;
  const PlanKey k{dtype, split, M, N, K, dense_begin, tiled, ov};
  for (int i = 0; i < c.used; ++i)
    if (c.key[i] == k) return c.plan[i];
  const int slot = c.next;
  c.next = (c.next + 1) % kPlanCache;
  if (c.used < kPlanCache) ++c.used;
  c.key[slot] = k;
  make_plan(dtype, M, N, split, K, dense_begin, tiled, ov, &c.plan[slot]);
  if (g_log.load(std::memory_order_relaxed) >= 1)
    log_plan("plan", dtype, M, N, split, K, dense_begin, tiled, c.plan[slot].ls, c.plan[slot].args,
             c.plan[slot].ws_bytes);
  return c.plan[slot];
}

int gemm_common(const void* X, int64_t M, int64_t ldx, int32_t dtype, int32_t split, int64_t N, int64_t K,
                int64_t dense_begin, int32_t layout, const void* values, int64_t values_ld, const uint32_t* meta,
                int64_t meta_ld, const void* dense, int64_t dense_ld, const float* w_scale, const float* x_scale,
                void* Y, int64_t ldy, uint32_t out_flags, void* ws, size_t ws_bytes, const Override& ov,
                hipStream_t stream) {
  const bool tiled = layout == SPENSE_LAYOUT_TILED;
  if (M < 0) return fail(SPENSE_ERR_ARG, "negative M");
  if (M > INT32_MAX) return fail(SPENSE_ERR_ARG, "M too large");
  if (out_flags & ~1u) return fail(SPENSE_ERR_ARG, "unknown out_flags 0x%x", out_flags);
  if (M == 0 || N == 0) return ok();
  const int es = esize(dtype);
  if (!Y) return fail(SPENSE_ERR_ARG, "Y is NULL");
  if (ldy < N) return fail(SPENSE_ERR_ARG, "ldy=%lld < N=%lld", (long long)ldy, (long long)N);
  if (K > 0) {
    if (!X) return fail(SPENSE_ERR_ARG, "X is NULL");
    if (ldx < K) return fail(SPENSE_ERR_ARG, "ldx=%lld < K=%lld", (long long)ldx, (long long)K);
    if (!aligned16(X) || (ldx * es) % 16)
      return fail(SPENSE_ERR_ALIGN, "X must be 16-byte aligned with a 16-byte multiple row pitch");
  }
  const int out_es = (out_flags & SPENSE_OUT_F32) ? 4 : 2;
  if ((reinterpret_cast<uintptr_t>(Y) % out_es)) return fail(SPENSE_ERR_ALIGN, "Y misaligned");
  if ((int64_t)M * ldy > (int64_t)1 << 40) return fail(SPENSE_ERR_ARG, "Y too large");
  Plan pl = cached_plan(dtype, M, N, split, K, dense_begin, tiled, ov);
  if (pl.ws_bytes > 0) {
    if (!ws || ws_bytes < pl.ws_bytes)
      return fail(SPENSE_ERR_WS, "workspace of %zu bytes needed, %zu given", pl.ws_bytes, ws ? ws_bytes : (size_t)0);
    if (!aligned16(ws)) return fail(SPENSE_ERR_ALIGN, "workspace must be 16-byte aligned");
  }
  int rc = check_device();
  if (rc) return rc;
  spense::GemmArgs& a = pl.args;
  a.X = static_cast<const uint8_t*>(X);
  a.ldx_b = ldx * es;
  a.values = static_cast<const uint8_t*>(values);
  a.v_ld_b = values_ld * es;
  a.meta = meta;
  a.m_ld_b = meta_ld * 4;
  a.dense = static_cast<const uint8_t*>(dense);
  a.d_ld_b = dense_ld * es;
  a.sw = w_scale;
  a.sx = x_scale;
  a.Y = Y;
  a.ldy = ldy;
  a.M = (int32_t)M;
  a.N = (int32_t)N;
  a.out_f32 = (out_flags & SPENSE_OUT_F32) ? 1 : 0;
  bool vec = (ldy % 4 == 0) && (reinterpret_cast<uintptr_t>(Y) % (4 * out_es) == 0);
  for (int i = 0; i < a.nreg; ++i) vec = vec && (a.reg[i].row0 % 4 == 0);
  a.vec_store = vec ? 1 : 0;
  // extents of the range-checked loads; every one must stay below 2^31
  int64_t sparse_rows = split == SPENSE_SPLIT_OUTPUT ? dense_begin : N;
  int64_t sparse_cols = split == SPENSE_SPLIT_OUTPUT ? K : dense_begin;
  int64_t dense_rows = split == SPENSE_SPLIT_OUTPUT ? N - dense_begin : N;
  int64_t dense_cols = split == SPENSE_SPLIT_OUTPUT ? K : K - dense_begin;
  const int64_t xb = K > 0 ? ((M - 1) * ldx + K) * es : 0;
  int64_t vb = sparse_rows > 0 && sparse_cols > 0 ? ((sparse_rows - 1) * values_ld + sparse_cols / 2) * es : 0;
  int64_t mb = sparse_rows > 0 && sparse_cols > 0 ? ((sparse_rows - 1) * meta_ld + sparse_cols / 32) * 4 : 0;
  int64_t db = dense_rows > 0 && dense_cols > 0 ? ((dense_rows - 1) * dense_ld + dense_cols) * es : 0;
  if (tiled) {
    spense_tiled_layout_t T;
    tiled_impl(N, K, dtype, split, dense_begin, &T);  // validated by check_packed
    vb = (int64_t)T.values_bytes;
    mb = (int64_t)T.meta_bytes;
    db = (int64_t)T.dense_bytes;
  }
  const int64_t lim = (int64_t)1 << 31;
  if (xb >= lim || vb >= lim || mb >= lim || db >= lim)
    return fail(SPENSE_ERR_ARG, "an operand spans 2 GiB or more; split the layer");
  a.x_bytes = (uint32_t)xb;
  a.v_bytes = (uint32_t)vb;
  a.m_bytes = (uint32_t)mb;
  a.d_bytes = (uint32_t)db;
  // the row-split kernel reads the weight through its descriptor
  a.nmat = 1;
  a.mat[0] = spense::MatDesc{a.values, a.meta, a.dense, a.v_bytes, a.m_bytes, a.d_bytes, a.Y, a.ldy, a.sw,
                             a.vec_store};
  if (a.groups == 0) return ok();
  a.part = static_cast<float*>(ws);
  hipError_t e = spense::launch_gemm(dtype, pl.ls, a, stream);
  if (e == hipSuccess && pl.ws_bytes > 0) e = spense::launch_splitk_reduce(a, stream);
  if (e != hipSuccess) return fail(SPENSE_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

// Checks of the gate / up pair and X shared by the GLU calls.
int check_glu_pair(const void* X, int64_t M, int64_t ldx, const spense_packed_t* gate, const spense_packed_t* up) {
  if (!gate || !up) return fail(SPENSE_ERR_ARG, "gate or up is NULL");
  if (M < 0 || M > INT32_MAX) return fail(SPENSE_ERR_ARG, "bad M");
  for (const spense_packed_t* P : {gate, up}) {
    spense_layout_t L;
    int rc = check_packed(P, &L);
    if (rc) return rc;
    if (P->dtype != SPENSE_FP8_E4M3FN || P->layout != SPENSE_LAYOUT_TILED || P->split != SPENSE_SPLIT_OUTPUT)
      return fail(SPENSE_ERR_ARG, "gate and up must be fp8, output-split, in the tiled layout");
  }
  if (gate->N != up->N || gate->K != up->K || gate->dense_begin != up->dense_begin)
    return fail(SPENSE_ERR_ARG, "gate and up must have the same N, K and dense_begin");
  const int64_t N = gate->N, K = gate->K;
  if (M == 0 || N == 0) return SPENSE_OK;
  if (K == 0) return fail(SPENSE_ERR_ARG, "K = 0 (H would be glu(0, 0) = 0; not a GEMM)");
  if (!X) return fail(SPENSE_ERR_ARG, "X is NULL");
  if (ldx < K) return fail(SPENSE_ERR_ARG, "ldx=%lld < K=%lld", (long long)ldx, (long long)K);
  if (!aligned16(X) || ldx % 16) return fail(SPENSE_ERR_ALIGN, "X must be 16-byte aligned with a 16-byte multiple row pitch");
  if ((M - 1) * ldx + K >= ((int64_t)1 << 31)) return fail(SPENSE_ERR_ARG, "X spans 2 GiB or more");
  spense_tiled_layout_t T;
  tiled_impl(N, K, SPENSE_FP8_E4M3FN, SPENSE_SPLIT_OUTPUT, gate->dense_begin, &T);
  if ((int64_t)T.values_bytes >= ((int64_t)1 << 31) || (int64_t)T.meta_bytes >= ((int64_t)1 << 31) ||
      (int64_t)T.dense_bytes >= ((int64_t)1 << 31))
    return fail(SPENSE_ERR_ARG, "weights span 2 GiB or more");
  return SPENSE_OK;
}

// The paired gate / up launch (arguments checked, M, N > 0): H (fp32, ldh) and, when hmax
// is given, the per-workgroup maxima of |h| per token, hmax[m * groups + g]; *groups_out
// receives the number of workgroups along N.
int launch_glu_pair(const void* X, int64_t M, int64_t ldx, const spense_packed_t* gate, const spense_packed_t* up,
                    const float* w_scale_gate, const float* w_scale_up, const float* x_scale, float* H, int64_t ldh,
                    float* hmax, int32_t* groups_out, hipStream_t stream) {
  using spense::Region;
  const int64_t N = gate->N, K = gate->K, db = gate->dense_begin;
  spense_tiled_layout_t T;
  tiled_impl(N, K, SPENSE_FP8_E4M3FN, SPENSE_SPLIT_OUTPUT, db, &T);
  // Plan: the row-split kernel with 8 waves, waves 0-3 on gate tiles and 4-7 on the up
  // tiles of the same rows, no K slices; the dense rows first, then the 2:4 rows; row
  // tiles per workgroup (1-4) per kind from the same cost model as the grouped launch,
  // each tile counted twice (gate and up).
  spense::LaunchShape ls;
  memset(&ls, 0, sizeof ls);
  ls.ct = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  ls.mblocks = (int)ceil_div(M, 16 * ls.ct);
  ls.rt = 1;
  ls.waves = 8;
  ls.rows = 1;
  ls.glu = 1;
  spense::GemmArgs a;
  memset(&a, 0, sizeof a);
  const double sparse_cost = 0.625;  // fp8 bytes per logical 2:4 entry
  Region regs[2];
  int nreg = 0;
  for (int pass = 0; pass < 2; ++pass) {
    const int64_t r0 = pass == 0 ? db : 0, rows = pass == 0 ? N - db : db;
    if (rows <= 0) continue;
    Region r;
    memset(&r, 0, sizeof r);
    r.row0 = (int32_t)r0;
    r.rows = (int32_t)rows;
    r.kbound = pass == 0 ? 0 : (int32_t)K;
    r.kend = (int32_t)K;
    r.dense_row_off = (int32_t)db;
    slice_cuts(r, 1, 512, 1, sparse_cost);
    regs[nreg++] = r;
  }
  const double tile_d = 2 * 16.0 * K, tile_s = 2 * 16.0 * sparse_cost * K, x_cost = 0.25 * 16.0 * ls.ct * K;
  int64_t rows[2];
  int kind[2];
  double tile[2];
  for (int i = 0; i < nreg; ++i) {
    rows[i] = regs[i].rows;
    kind[i] = regs[i].kbound == 0 ? 0 : 1;
    tile[i] = regs[i].kbound == 0 ? tile_d : tile_s;
  }
  int bw[2];
  pick_waves(nreg, rows, kind, tile, 1, 4, ls.mblocks, x_cost, bw);
  int32_t groups = 0;
  for (int i = 0; i < nreg; ++i) {
    regs[i].wused = bw[kind[i]];
    regs[i].nrb = (int32_t)ceil_div(regs[i].rows, 16 * regs[i].wused);
    regs[i].wg0 = groups;
    groups += regs[i].nrb;
    a.reg[i] = regs[i];
  }
  a.nreg = nreg;
  a.groups = groups;
  a.tiled = 1;
  a.X = static_cast<const uint8_t*>(X);
  a.ldx_b = ldx;
  a.x_bytes = (uint32_t)((M - 1) * ldx + K);
  a.sx = x_scale;
  a.M = (int32_t)M;
  a.N = (int32_t)N;
  a.out_f32 = 1;
  a.nmat = 2;
  const bool vec = ldh % 4 == 0 && reinterpret_cast<uintptr_t>(H) % 16 == 0 && db % 4 == 0;
  const spense_packed_t* const PW[2] = {gate, up};
  const float* const SW[2] = {w_scale_gate, w_scale_up};
  for (int i = 0; i < 2; ++i)
    a.mat[i] = spense::MatDesc{static_cast<const uint8_t*>(PW[i]->values), PW[i]->meta,
                               static_cast<const uint8_t*>(PW[i]->dense), (uint32_t)T.values_bytes,
                               (uint32_t)T.meta_bytes, (uint32_t)T.dense_bytes, H, ldh, SW[i], vec ? 1 : 0};
  // the row maxima take one slot per workgroup along N: at most ceil(rows / 16) per region
  if (hmax && groups > ceil_div(N, 16) + 1) return fail(SPENSE_ERR_HIP, "internal: %d workgroups along N", groups);
  a.hmax = hmax;
  *groups_out = groups;
  if (g_log.load(std::memory_order_relaxed) >= 2)
    log_plan("paired gate/up", SPENSE_FP8_E4M3FN, M, N, SPENSE_SPLIT_OUTPUT, K, db, true, ls, a, 0);
  hipError_t e = spense::launch_gemm(SPENSE_FP8_E4M3FN, ls, a, stream);
  if (e != hipSuccess) return fail(SPENSE_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return SPENSE_OK;
}

// Workspace of spense_gemm_glu_fp8: H (fp32, rows padded to 64 elements), then the
// per-workgroup row maxima (at least 16 weight rows per workgroup, in each of the two
// regions).
int64_t glu_ldh(int64_t N) { return (N + 63) / 64 * 64; }
int64_t glu_hmax_offset(int64_t M, int64_t N) { return (M * glu_ldh(N) * 4 + 255) / 256 * 256; }

}  // namespace

namespace spense {
int api_fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vfail(code, fmt, ap);
  va_end(ap);
  return code;
}
}  // namespace spense

extern "C" {

int spense_abi_version(void) { return SPENSE_ABI_VERSION; }

int spense_set_log(int32_t level) { return g_log.exchange(level); }

const char* spense_last_error(void) { return g_err; }

int spense_quantize_fp8(const void* src, int32_t src_type, int64_t M, int64_t K, int64_t ld_src, uint8_t* q,
                        int64_t ldq, float* scales, hipStream_t stream) {
  int rc = check_quant_args(src, src_type, M, K, ld_src, q, ldq, scales, "src");
  if (rc) return rc;
  if (M == 0) return ok();
  rc = check_device();
  if (rc) return rc;
  const int64_t es = src_type == SPENSE_BF16 ? 2 : 4;
  if (spense::launch_quantize(src_type, src, ld_src * es, M, K, q, ldq, scales, stream) != hipSuccess)
    return fail(SPENSE_ERR_HIP, "quantize launch failed");
  return ok();
}

size_t spense_obs_factor_workspace_size(int64_t K) { return K < 1 ? 0 : spense::obs_factor_workspace(K); }

int spense_obs_factor(const float* H, int64_t ldh, int64_t K, float percdamp, float* U, int64_t ldu, uint8_t* dead,
                      void* ws, size_t ws_bytes, hipStream_t stream) {
  if (K < 1 || K > INT32_MAX) return fail(SPENSE_ERR_ARG, "bad K=%lld", (long long)K);
  if (!H || !U || !dead) return fail(SPENSE_ERR_ARG, "NULL pointer");
  if (ldh < K || ldu < K) return fail(SPENSE_ERR_ARG, "leading dimension below K");
  if (!(percdamp >= 0.0f) || !std::isfinite(percdamp)) return fail(SPENSE_ERR_ARG, "percdamp must be >= 0 and finite");
  const uintptr_t h0 = reinterpret_cast<uintptr_t>(H), h1 = h0 + (uintptr_t)(((K - 1) * ldh + K) * 4);
  const uintptr_t u0 = reinterpret_cast<uintptr_t>(U), u1 = u0 + (uintptr_t)(((K - 1) * ldu + K) * 4);
  if (h0 < u1 && u0 < h1) return fail(SPENSE_ERR_ARG, "U overlaps H");
  if (h0 % 4 || u0 % 4) return fail(SPENSE_ERR_ALIGN, "H and U must be 4-byte aligned");
  if (!ws || ws_bytes < spense::obs_factor_workspace(K) || !aligned16(ws))
    return fail(SPENSE_ERR_WS, "a 16-byte aligned workspace of %zu bytes is needed", spense::obs_factor_workspace(K));
  int rc = check_device();
  if (rc) return rc;
  int* flag = spense::obs_factor_fail_flag(ws, K);
  hipError_t e = spense::launch_zero_u64(reinterpret_cast<unsigned long long*>(flag), stream);
  if (e == hipSuccess) e = spense::launch_obs_factor(H, ldh, K, percdamp, U, ldu, dead, ws, stream);
  if (e != hipSuccess) return fail(SPENSE_ERR_HIP, "launch failed: %s", hipGetErrorString(e));
  int host_fail = 0;
  e = hipMemcpyAsync(&host_fail, flag, sizeof host_fail, hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return fail(SPENSE_ERR_HIP, "factor failed: %s", hipGetErrorString(e));
  if (host_fail) return fail(SPENSE_ERR_NUMERIC, "the damped Hessian is not positive definite");
  return ok();
}

size_t spense_obs_prune_workspace_size(int64_t N) { return N < 1 ? 0 : spense::obs_prune_workspace(N); }

int spense_obs_prune_24(float* W, int64_t ldw, int64_t N, int64_t K, const float* U, int64_t ldu, const uint8_t* dead,
                        int64_t dense_begin, uint8_t* keep, int64_t ldk, void* ws, size_t ws_bytes,
                        hipStream_t stream) {
  if (N < 0 || K < 0 || N > INT32_MAX || K > INT32_MAX) return fail(SPENSE_ERR_ARG, "bad size");
  if (dense_begin < 0 || dense_begin > K || dense_begin % 4)
    return fail(SPENSE_ERR_ARG, "dense_begin=%lld must be a multiple of 4 in [0, K]", (long long)dense_begin);
  if (N == 0 || K == 0) return ok();
  if (!W || !U || !keep) return fail(SPENSE_ERR_ARG, "NULL pointer");
  if (ldw < K || ldu < K || ldk < K) return fail(SPENSE_ERR_ARG, "leading dimension below K");
  if (reinterpret_cast<uintptr_t>(W) % 4 || reinterpret_cast<uintptr_t>(U) % 4)
    return fail(SPENSE_ERR_ALIGN, "W and U must be 4-byte aligned");
  if (!ws || ws_bytes < spense::obs_prune_workspace(N) || !aligned16(ws))
    return fail(SPENSE_ERR_WS, "a 16-byte aligned workspace of %zu bytes is needed", spense::obs_prune_workspace(N));
  int rc = check_device();
  if (rc) return rc;
  if (spense::launch_obs_prune(W, ldw, N, K, U, ldu, dead, dense_begin, keep, ldk, ws, stream) != hipSuccess)
    return fail(SPENSE_ERR_HIP, "prune launch failed");
  return ok();
}

int spense_index_scores(const void* w_gate, const void* w_up, int64_t ld_gu, const void* w_down, int64_t ld_down,
                        int32_t wtype, int64_t I, int64_t D, const float* h_in, const float* h_mid, float eps,
                        float* raw, float* total, hipStream_t stream) {
  if (wtype != SPENSE_BF16 && wtype != SPENSE_F32) return fail(SPENSE_ERR_ARG, "wtype %d is not bf16 or f32", wtype);
  if (I < 1 || D < 1 || I > INT32_MAX || D > INT32_MAX) return fail(SPENSE_ERR_ARG, "bad I=%lld D=%lld", (long long)I, (long long)D);
  if (!w_gate || !w_up || !w_down || !h_in || !h_mid || !raw || !total) return fail(SPENSE_ERR_ARG, "NULL pointer");
  if (ld_gu < D || ld_down < I) return fail(SPENSE_ERR_ARG, "leading dimension below the row length");
  int rc = check_device();
  if (rc) return rc;
  const int64_t es = wtype == SPENSE_BF16 ? 2 : 4;
  if (spense::launch_index_scores(wtype, w_gate, w_up, ld_gu * es, I, D, w_down, ld_down * es, h_in, h_mid, eps, raw,
                                  total, stream) != hipSuccess)
    return fail(SPENSE_ERR_HIP, "index score launch failed");
  return ok();
}

int spense_dense_permutation(const float* total, int64_t I, int64_t n_dense, uint8_t* flags, int32_t* perm,
                             hipStream_t stream) {
  if (I < 1 || I > INT32_MAX) return fail(SPENSE_ERR_ARG, "bad I=%lld", (long long)I);
  if (n_dense < 0 || n_dense > I) return fail(SPENSE_ERR_ARG, "n_dense=%lld outside [0, I]", (long long)n_dense);
  if (!total || !flags || !perm) return fail(SPENSE_ERR_ARG, "NULL pointer");
  int rc = check_device();
  if (rc) return rc;
  if (spense::launch_dense_permutation(total, I, n_dense, flags, perm, stream) != hipSuccess)
    return fail(SPENSE_ERR_HIP, "permutation launch failed");
  return ok();
}

int spense_gather_rows(const void* src, int64_t ld_src_b, void* dst, int64_t ld_dst_b, int64_t rows,
                       int64_t row_bytes, const int32_t* perm, hipStream_t stream) {
  if (rows < 0 || row_bytes < 0 || rows > INT32_MAX) return fail(SPENSE_ERR_ARG, "bad size");
  if (rows == 0 || row_bytes == 0) return ok();
  if (!src || !dst || !perm) return fail(SPENSE_ERR_ARG, "NULL pointer");
  if (ld_src_b < row_bytes || ld_dst_b < row_bytes) return fail(SPENSE_ERR_ARG, "leading dimension below the row");
  int rc = check_device();
  if (rc) return rc;
  if (spense::launch_gather_rows(src, ld_src_b, dst, ld_dst_b, rows, row_bytes, perm, stream) != hipSuccess)
    return fail(SPENSE_ERR_HIP, "gather launch failed");
  return ok();
}

int spense_gather_cols(const void* src, int64_t ld_src, void* dst, int64_t ld_dst, int64_t rows, int64_t cols,
                       int32_t elem_bytes, const int32_t* perm, hipStream_t stream) {
  if (elem_bytes != 1 && elem_bytes != 2 && elem_bytes != 4) return fail(SPENSE_ERR_ARG, "elem_bytes %d", elem_bytes);
  if (rows < 0 || cols < 0 || rows > INT32_MAX || cols > INT32_MAX) return fail(SPENSE_ERR_ARG, "bad size");
  if (rows == 0 || cols == 0) return ok();
  if (!src || !dst || !perm) return fail(SPENSE_ERR_ARG, "NULL pointer");
  if (ld_src < cols || ld_dst < cols) return fail(SPENSE_ERR_ARG, "leading dimension below the row");
  if ((uintptr_t)src % elem_bytes || (uintptr_t)dst % elem_bytes) return fail(SPENSE_ERR_ALIGN, "misaligned matrix");
  int rc = check_device();
  if (rc) return rc;
  if (spense::launch_gather_cols(elem_bytes, src, ld_src * elem_bytes, dst, ld_dst * elem_bytes, rows, cols, perm,
                                 stream) != hipSuccess)
    return fail(SPENSE_ERR_HIP, "gather launch failed");
  return ok();
}

int spense_glu_quantize_fp8(const void* g, int64_t ldg, const void* u, int64_t ldu, int32_t gu_type, int64_t M,
                            int64_t I, uint8_t* q, int64_t ldq, float* scales, hipStream_t stream) {
  int rc = check_quant_args(g, gu_type, M, I, ldg, q, ldq, scales, "g");
  if (rc) return rc;
  rc = check_quant_args(u, gu_type, M, I, ldu, q, ldq, scales, "u");
  if (rc) return rc;
  if (M == 0) return ok();
  rc = check_device();
  if (rc) return rc;
  const int64_t es = gu_type == SPENSE_BF16 ? 2 : 4;
  if (spense::launch_glu_quantize(gu_type, g, ldg * es, u, ldu * es, M, I, q, ldq, scales, stream) != hipSuccess)
    return fail(SPENSE_ERR_HIP, "glu quantize launch failed");
  return ok();
}

int spense_layout(int64_t N, int64_t K, int32_t dtype, int32_t split, int64_t dense_begin, spense_layout_t* out) {
  return layout_impl(N, K, dtype, split, dense_begin, out);
}

size_t spense_compress_workspace_size(void) { return 256; }

int spense_tiled_layout(int64_t N, int64_t K, int32_t dtype, int32_t split, int64_t dense_begin,
                        spense_tiled_layout_t* out) {
  return tiled_impl(N, K, dtype, split, dense_begin, out);
}

int spense_tile(const spense_packed_t* src, const spense_packed_t* dst, hipStream_t stream) {
  spense_layout_t L, Ld;
  int rc = check_packed(src, &L);
  if (rc) return rc;
  rc = check_packed(dst, &Ld);
  if (rc) return rc;
  if (src->layout != SPENSE_LAYOUT_ROWMAJOR || dst->layout != SPENSE_LAYOUT_TILED)
    return fail(SPENSE_ERR_ARG, "spense_tile reorders a row-major weight into a tiled one");
  if (src->dtype != dst->dtype || src->split != dst->split || src->N != dst->N || src->K != dst->K ||
      src->dense_begin != dst->dense_begin)
    return fail(SPENSE_ERR_ARG, "source and destination describe different weights");
  spense_tiled_layout_t T;
  rc = tiled_impl(src->N, src->K, src->dtype, src->split, src->dense_begin, &T);
  if (rc) return rc;
  auto overlaps = [](const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return na && nb && x < y + nb && y < x + na;
  };
  const void* srcs[3] = {src->values, src->meta, src->dense};
  const size_t srcn[3] = {L.values_bytes, L.meta_bytes, L.dense_bytes};
  const void* dsts[3] = {dst->values, dst->meta, dst->dense};
  const size_t dstn[3] = {T.values_bytes, T.meta_bytes, T.dense_bytes};
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j)
      if (overlaps(srcs[i], srcn[i], dsts[j], dstn[j])) return fail(SPENSE_ERR_ARG, "source and destination overlap");
  rc = check_device();
  if (rc) return rc;
  hipError_t e = spense::launch_tile(0, static_cast<const uint8_t*>(src->values), src->values_ld, L.sparse_rows,
                                     L.sparse_cols / 2, T.sparse_tiles, T.sparse_chunks,
                                     static_cast<uint8_t*>(dst->values), stream);
  if (e == hipSuccess)
    e = spense::launch_tile(1, reinterpret_cast<const uint8_t*>(src->meta), src->meta_ld * 4, L.sparse_rows,
                            L.sparse_cols / 32 * 4, T.sparse_tiles, T.sparse_chunks,
                            reinterpret_cast<uint8_t*>(dst->meta), stream);
  if (e == hipSuccess)
    e = spense::launch_tile(2, static_cast<const uint8_t*>(src->dense), src->dense_ld, L.dense_rows, L.dense_cols,
                            T.dense_tiles, T.dense_chunks, static_cast<uint8_t*>(dst->dense), stream);
  if (e != hipSuccess) return fail(SPENSE_ERR_HIP, "launch failed: %s", hipGetErrorString(e));
  return ok();
}

int spense_compress(const void* W, int64_t ldw, const uint8_t* mask, int64_t ldm, const spense_packed_t* packed,
                    int64_t* bad_groups, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (bad_groups) *bad_groups = 0;
  spense_layout_t L;
  int rc = check_packed(packed, &L);
  if (rc) return rc;
  if (packed->layout != SPENSE_LAYOUT_ROWMAJOR)
    return fail(SPENSE_ERR_ARG, "spense_compress writes the row-major layout (then spense_tile)");
  const int64_t N = packed->N, K = packed->K;
  const int es = esize(packed->dtype);
  if (N == 0 || K == 0) return ok();
  if (!W) return fail(SPENSE_ERR_ARG, "W is NULL");
  if (ldw < K) return fail(SPENSE_ERR_ARG, "ldw < K");
  if (!aligned16(W) || (ldw * es) % 16) return fail(SPENSE_ERR_ALIGN, "W must be 16-byte aligned, 16-byte pitch");
  if (mask) {
    if (ldm < K) return fail(SPENSE_ERR_ARG, "ldm < K");
    if (!aligned16(mask) || ldm % 16) return fail(SPENSE_ERR_ALIGN, "mask must be 16-byte aligned, 16-byte pitch");
  }
  if (!ws || ws_bytes < spense_compress_workspace_size() || (reinterpret_cast<uintptr_t>(ws) & 7u))
    return fail(SPENSE_ERR_WS, "compress needs an 8-byte aligned workspace of %zu bytes",
                spense_compress_workspace_size());
  rc = check_device();
  if (rc) return rc;
  unsigned long long* bad = static_cast<unsigned long long*>(ws);
  hipError_t e = spense::launch_zero_u64(bad, stream);
  if (e != hipSuccess) return fail(SPENSE_ERR_HIP, "launch failed: %s", hipGetErrorString(e));
  const uint8_t* w8 = static_cast<const uint8_t*>(W);
  const uint8_t* dsrc = packed->split == SPENSE_SPLIT_OUTPUT ? w8 + packed->dense_begin * ldw * es
                                                              : w8 + packed->dense_begin * es;
  e = spense::launch_compress(packed->dtype, w8, ldw * es, mask, ldm, L.sparse_rows, L.sparse_cols,
                              static_cast<uint8_t*>(packed->values), packed->values_ld * es, packed->meta,
                              packed->meta_ld, dsrc, L.dense_rows, L.dense_cols * es,
                              static_cast<uint8_t*>(packed->dense), packed->dense_ld * es, bad, stream);
  if (e != hipSuccess) return fail(SPENSE_ERR_HIP, "launch failed: %s", hipGetErrorString(e));
  unsigned long long host_bad = 0;
  e = hipMemcpyAsync(&host_bad, bad, sizeof host_bad, hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return fail(SPENSE_ERR_HIP, "compress failed: %s", hipGetErrorString(e));
  if (bad_groups) *bad_groups = (int64_t)host_bad;
  if (host_bad) return fail(SPENSE_ERR_MASK, "%llu group(s) of the 2:4 region keep more than 2 of 4", host_bad);
  return ok();
}

int spense_decompress(const spense_packed_t* packed, void* W_out, int64_t ldw, hipStream_t stream) {
  spense_layout_t L;
  int rc = check_packed(packed, &L);
  if (rc) return rc;
  if (packed->layout != SPENSE_LAYOUT_ROWMAJOR) return fail(SPENSE_ERR_ARG, "spense_decompress reads the row-major layout");
  const int64_t N = packed->N, K = packed->K;
  const int es = esize(packed->dtype);
  if (N == 0 || K == 0) return ok();
  if (!W_out) return fail(SPENSE_ERR_ARG, "W_out is NULL");
  if (ldw < K) return fail(SPENSE_ERR_ARG, "ldw < K");
  if (!aligned16(W_out) || (ldw * es) % 16) return fail(SPENSE_ERR_ALIGN, "W_out must be 16-byte aligned");
  rc = check_device();
  if (rc) return rc;
  uint8_t* w8 = static_cast<uint8_t*>(W_out);
  uint8_t* ddst = packed->split == SPENSE_SPLIT_OUTPUT ? w8 + packed->dense_begin * ldw * es
                                                       : w8 + packed->dense_begin * es;
  hipError_t e = spense::launch_decompress(packed->dtype, static_cast<const uint8_t*>(packed->values),
                                           packed->values_ld * es, packed->meta, packed->meta_ld, L.sparse_rows,
                                           L.sparse_cols, w8, ldw * es, static_cast<const uint8_t*>(packed->dense),
                                           packed->dense_ld * es, L.dense_rows, L.dense_cols * es, ddst, stream);
  if (e != hipSuccess) return fail(SPENSE_ERR_HIP, "launch failed: %s", hipGetErrorString(e));
  return ok();
}

size_t spense_gemm_planned_workspace_size(int64_t M, const spense_packed_t* packed,
                                          const spense_plan_override_t* plan) {
  spense_layout_t L;
  if (M <= 0 || M > INT32_MAX || check_packed(packed, &L)) return 0;
  Override ov;
  if (read_override(plan, packed->dtype, packed->layout == SPENSE_LAYOUT_TILED, &ov)) return 0;
  return cached_plan(packed->dtype, M, packed->N, packed->split, packed->K, packed->dense_begin,
                     packed->layout == SPENSE_LAYOUT_TILED, ov)
      .ws_bytes;
}

size_t spense_gemm_workspace_size(int64_t M, const spense_packed_t* packed) {
  return spense_gemm_planned_workspace_size(M, packed, nullptr);
}

int spense_gemm_planned(const void* X, int64_t M, int64_t ldx, const spense_packed_t* packed, const float* w_scale,
                        const float* x_scale, void* Y, int64_t ldy, uint32_t out_flags, void* ws, size_t ws_bytes,
                        const spense_plan_override_t* plan, hipStream_t stream) {
  spense_layout_t L;
  int rc = check_packed(packed, &L);
  if (rc) return rc;
  Override ov;
  rc = read_override(plan, packed->dtype, packed->layout == SPENSE_LAYOUT_TILED, &ov);
  if (rc) return rc;
  return gemm_common(X, M, ldx, packed->dtype, packed->split, packed->N, packed->K, packed->dense_begin,
                     packed->layout, packed->values, packed->values_ld, packed->meta, packed->meta_ld, packed->dense,
                     packed->dense_ld, w_scale, x_scale, Y, ldy, out_flags, ws, ws_bytes, ov, stream);
}

int spense_gemm(const void* X, int64_t M, int64_t ldx, const spense_packed_t* packed, const float* w_scale,
                const float* x_scale, void* Y, int64_t ldy, uint32_t out_flags, void* ws, size_t ws_bytes,
                hipStream_t stream) {
  return spense_gemm_planned(X, M, ldx, packed, w_scale, x_scale, Y, ldy, out_flags, ws, ws_bytes, nullptr, stream);
}

int spense_gemm_grouped(const void* X, int64_t M, int64_t ldx, int32_t count, const spense_packed_t* const* packed,
                        const float* const* w_scales, const float* x_scale, void* const* Y, const int64_t* ldy,
                        uint32_t out_flags, hipStream_t stream) {
  using spense::Region;
  if (count < 1 || count > spense::kMaxMats) return fail(SPENSE_ERR_ARG, "count=%d outside [1, %d]", count, spense::kMaxMats);
  if (!packed || !Y || !ldy) return fail(SPENSE_ERR_ARG, "NULL array");
  if (M < 0 || M > INT32_MAX) return fail(SPENSE_ERR_ARG, "bad M");
  if (out_flags & ~1u) return fail(SPENSE_ERR_ARG, "unknown out_flags 0x%x", out_flags);
  const int out_es = (out_flags & SPENSE_OUT_F32) ? 4 : 2;
  int64_t K = -1;
  for (int i = 0; i < count; ++i) {
    spense_layout_t L;
    if (!packed[i]) return fail(SPENSE_ERR_ARG, "packed[%d] is NULL", i);
    int rc = check_packed(packed[i], &L);
    if (rc) return rc;
    const spense_packed_t& P = *packed[i];
    if (P.dtype != SPENSE_FP8_E4M3FN || P.layout != SPENSE_LAYOUT_TILED || P.split != SPENSE_SPLIT_OUTPUT)
      return fail(SPENSE_ERR_ARG, "grouped weights must be fp8, output-split, in the tiled layout");
    if (K >= 0 && P.K != K) return fail(SPENSE_ERR_ARG, "grouped weights must share K");
    K = P.K;
    if (!Y[i]) return fail(SPENSE_ERR_ARG, "Y[%d] is NULL", i);
    if (ldy[i] < P.N) return fail(SPENSE_ERR_ARG, "ldy[%d] < N", i);
    if (reinterpret_cast<uintptr_t>(Y[i]) % out_es) return fail(SPENSE_ERR_ALIGN, "Y[%d] misaligned", i);
    if ((int64_t)M * ldy[i] > (int64_t)1 << 40) return fail(SPENSE_ERR_ARG, "Y[%d] too large", i);
  }
  if (M == 0 || K == 0) return ok();
  if (!X) return fail(SPENSE_ERR_ARG, "X is NULL");
  if (ldx < K) return fail(SPENSE_ERR_ARG, "ldx=%lld < K=%lld", (long long)ldx, (long long)K);
  if (!aligned16(X) || ldx % 16) return fail(SPENSE_ERR_ALIGN, "X must be 16-byte aligned with a 16-byte multiple row pitch");
  const int64_t xb = (M - 1) * ldx + K;
  if (xb >= ((int64_t)1 << 31)) return fail(SPENSE_ERR_ARG, "X spans 2 GiB or more");

  // Plan: the row-split kernel as for one weight of this M (activation tiles, 8 waves), no
  // K slices; the dense rows of every weight first (their workgroups carry more bytes),
  // then the 2:4 rows; rows per workgroup chosen per kind as for one weight.
  spense::LaunchShape ls;
  memset(&ls, 0, sizeof ls);
  ls.ct = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  ls.mblocks = (int)ceil_div(M, 16 * ls.ct);
  ls.rt = 1;
  ls.waves = 8;
  ls.rows = 1;
  spense::GemmArgs a;
  memset(&a, 0, sizeof a);
  const double sparse_cost = 0.625;  // fp8 bytes per logical 2:4 entry
  const int64_t kc = 512;
  Region regs[spense::kMaxRegions];
  int nreg = 0;
  for (int pass = 0; pass < 2; ++pass)
    for (int i = 0; i < count; ++i) {
      const spense_packed_t& P = *packed[i];
      const int64_t r0 = pass == 0 ? P.dense_begin : 0, rows = pass == 0 ? P.N - P.dense_begin : P.dense_begin;
      if (rows <= 0) continue;
      Region r;
      memset(&r, 0, sizeof r);
      r.row0 = (int32_t)r0;
      r.rows = (int32_t)rows;
      r.kbound = pass == 0 ? 0 : (int32_t)K;
      r.kend = (int32_t)K;
      r.dense_row_off = (int32_t)P.dense_begin;
      r.mat = i;
      slice_cuts(r, 1, kc, 1, sparse_cost);
      regs[nreg++] = r;
    }
  // Many tokens: the 256 x 256 large-M kernel over every weight's regions in one grid, on
  // the single-weight rule (at least 160 tiles; with two or three token blocks the last
  // one full), with its tail tiles and XCD-aware order; small weights such as k and v then
  // ride in q's grid instead of leaving most CUs idle (alone at M = 2048 they run 37 us on
  // the row-split kernel).
  const int64_t T256 = ceil_div(M, 256);
  int64_t rb256 = 0;
  for (int i = 0; i < nreg; ++i) rb256 += ceil_div(regs[i].rows, 256);
  const bool big2 = M >= kBigMinM && rb256 * T256 >= 160;
  if (M >= kBigMinM && !big2) {
    // Between one token block and the 256 x 256 grid each weight's own plan (the 128 x
    // 256 large-M kernel on large weights) beats one row-split grid over all of them
    // (Seed-OSS q / k / v at M = 512: 75 against 95 us): one launch per weight, its plan
    // held to one K slice so that it needs no workspace.
    spense_plan_override_t one{};
    one.ksplit = 1;
    one.block_order = -1;
    one.xcd_order = -1;
    one.half_row_blocks = -1;
    for (int i = 0; i < count; ++i) {
      const int r = spense_gemm_planned(X, M, ldx, packed[i], w_scales ? w_scales[i] : nullptr, x_scale, Y[i], ldy[i],
                                        out_flags, nullptr, 0, &one, stream);
      if (r) return r;
    }
    return ok();
  }
  if (big2) {
    ls.rows = 0;
    ls.big = 2;
    ls.ct = 4;
    ls.mblocks = 1;
    const int64_t GT = xcd_token_group(T256);
    const int64_t rc = GT > 0 ? 8 / (T256 / GT) : 1;
    const int64_t rbl = ceil_div(regs[nreg - 1].rows, 256);
    const int64_t half_rb = choose_half_rows(regs, nreg, T256, M, rc);
    int32_t groups = 0;
    for (int i = 0; i < nreg; ++i) {
      regs[i].nrb = (int32_t)((ceil_div(regs[i].rows, 256) - (i == nreg - 1 ? half_rb : 0)) * T256);
      regs[i].wg0 = groups;
      groups += regs[i].nrb;
      a.reg[i] = regs[i];
    }
    a.tblocks = (int32_t)T256;
    a.btok = M > 256 && ceil_div(M, 192) == T256 ? 192 : 0;  // as for one weight
    a.hg0 = groups;
    a.hrb0 = (int32_t)(rbl - half_rb);
    a.hper = (int32_t)ceil_div(M, 128);
    a.groups = (int32_t)(groups + half_rb * a.hper);
    if (GT > 0) {
      const int64_t rbx = (rb256 - half_rb) / rc * rc;
      if (rbx > 0) {
        a.xgt = (int32_t)GT;
        a.xrc = (int32_t)rc;
        a.xg1 = (int32_t)(rbx * T256);
      }
    }
  } else {
  // rows per workgroup: w0 waves for dense regions, w1 for 2:4 regions (cost model of
  // pick_waves)
  const double tile_d = 16.0 * K, tile_s = 16.0 * sparse_cost * K, x_cost = 0.25 * 16.0 * ls.ct * K;
  int64_t rows[spense::kMaxRegions];
  int kind[spense::kMaxRegions];
  double tile[spense::kMaxRegions];
  for (int i = 0; i < nreg; ++i) {
    rows[i] = regs[i].rows;
    kind[i] = regs[i].kbound == 0 ? 0 : 1;
    tile[i] = regs[i].kbound == 0 ? tile_d : tile_s;
  }
  int bw[2];
  pick_waves(nreg, rows, kind, tile, 1, 8, ls.mblocks, x_cost, bw);
  int32_t groups = 0;
  for (int i = 0; i < nreg; ++i) {
    regs[i].wused = bw[kind[i]];
    regs[i].nrb = (int32_t)ceil_div(regs[i].rows, 16 * regs[i].wused);
    regs[i].wg0 = groups;
    groups += regs[i].nrb;
    a.reg[i] = regs[i];
  }
  // activations resident in LDS wherever they fit (one or two token tiles, K <= 5120 with
  // two): measured on MI355X (graph replay, us, staged -> resident): q / k / v grouped at
  // M = 1 / 16 / 32 9.6 / 9.7 / 13.0 -> 8.8 / 9.1 / 11.3 (Seed-OSS shapes 10.8 / 11.3 /
  // 13.6 -> 10.6 / 10.8 / 12.4), gate / up grouped 34.5 / 35.8 / 42.8 -> 34.0 / 35.0 /
  // 41.4; unlike one weight alone, also with few waves per workgroup
  const int64_t nch = ceil_div(K, kc);
  if (ls.ct <= 2 && nch * 8192 * ls.ct <= 160 * 1024) ls.xres = (int)nch;
  a.groups = groups;
  }
  a.nreg = nreg;
  a.tiled = 1;
  a.X = static_cast<const uint8_t*>(X);
  a.ldx_b = ldx;
  a.x_bytes = (uint32_t)xb;
  a.sx = x_scale;
  a.M = (int32_t)M;
  a.out_f32 = (out_flags & SPENSE_OUT_F32) ? 1 : 0;
  a.nmat = count;
  for (int i = 0; i < count; ++i) {
    const spense_packed_t& P = *packed[i];
    spense_tiled_layout_t T;
    tiled_impl(P.N, P.K, P.dtype, P.split, P.dense_begin, &T);
    if ((int64_t)T.values_bytes >= ((int64_t)1 << 31) || (int64_t)T.meta_bytes >= ((int64_t)1 << 31) ||
        (int64_t)T.dense_bytes >= ((int64_t)1 << 31))
      return fail(SPENSE_ERR_ARG, "weight %d spans 2 GiB or more", i);
    const bool vec = ldy[i] % 4 == 0 && reinterpret_cast<uintptr_t>(Y[i]) % (4 * out_es) == 0 && P.dense_begin % 4 == 0;
    a.mat[i] = spense::MatDesc{static_cast<const uint8_t*>(P.values), P.meta, static_cast<const uint8_t*>(P.dense),
                               (uint32_t)T.values_bytes, (uint32_t)T.meta_bytes, (uint32_t)T.dense_bytes, Y[i], ldy[i],
                               w_scales ? w_scales[i] : nullptr, vec ? 1 : 0};
  }
  // one weight: the plain instance, which reads its buffers from a
  const spense::MatDesc& m0 = a.mat[0];
  a.values = m0.values;
  a.meta = m0.meta;
  a.dense = m0.dense;
  a.v_bytes = m0.v_bytes;
  a.m_bytes = m0.m_bytes;
  a.d_bytes = m0.d_bytes;
  a.Y = m0.Y;
  a.ldy = m0.ldy;
  a.sw = m0.sw;
  a.vec_store = m0.vec_store;
  a.N = (int32_t)packed[0]->N;
  if (a.groups == 0) return ok();
  if (g_log.load(std::memory_order_relaxed) >= 2) {
    int64_t nsum = 0;
    for (int i = 0; i < count; ++i) nsum += packed[i]->N;
    log_plan("grouped", SPENSE_FP8_E4M3FN, M, nsum, SPENSE_SPLIT_OUTPUT, K, -1, true, ls, a, 0);
  }
  int rc = check_device();
  if (rc) return rc;
  hipError_t e = spense::launch_gemm(SPENSE_FP8_E4M3FN, ls, a, stream);
  if (e != hipSuccess) return fail(SPENSE_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

int spense_gemm_glu(const void* X, int64_t M, int64_t ldx, const spense_packed_t* gate, const spense_packed_t* up,
                    const float* w_scale_gate, const float* w_scale_up, const float* x_scale, float* H, int64_t ldh,
                    hipStream_t stream) {
  int rc = check_glu_pair(X, M, ldx, gate, up);
  if (rc) return rc;
  const int64_t N = gate->N;
  if (!H) return fail(SPENSE_ERR_ARG, "H is NULL");
  if (ldh < N) return fail(SPENSE_ERR_ARG, "ldh < N");
  if (reinterpret_cast<uintptr_t>(H) % 4) return fail(SPENSE_ERR_ALIGN, "H misaligned");
  if ((int64_t)M * ldh > (int64_t)1 << 40) return fail(SPENSE_ERR_ARG, "H too large");
  if (M == 0 || N == 0) return ok();
  rc = check_device();
  if (rc) return rc;
  int32_t groups = 0;
  rc = launch_glu_pair(X, M, ldx, gate, up, w_scale_gate, w_scale_up, x_scale, H, ldh, nullptr, &groups, stream);
  return rc ? rc : ok();
}

size_t spense_gemm_glu_fp8_workspace_size(int64_t M, int64_t N) {
  if (M <= 0 || N <= 0 || M > INT32_MAX || N > INT32_MAX) return 0;
  // workgroups along N: at most ceil(rows / 16) per region, two regions
  return (size_t)(glu_hmax_offset(M, N) + M * (ceil_div(N, 16) + 1) * 4);
}

int spense_gemm_glu_fp8(const void* X, int64_t M, int64_t ldx, const spense_packed_t* gate, const spense_packed_t* up,
                        const float* w_scale_gate, const float* w_scale_up, const float* x_scale, uint8_t* q,
                        int64_t ldq, float* scales, void* ws, size_t ws_bytes, hipStream_t stream) {
  int rc = check_glu_pair(X, M, ldx, gate, up);
  if (rc) return rc;
  const int64_t N = gate->N;
  if (M == 0) return ok();
  if (!scales) return fail(SPENSE_ERR_ARG, "scales is NULL");
  if (N > 0 && !q) return fail(SPENSE_ERR_ARG, "q is NULL");
  if (ldq < N) return fail(SPENSE_ERR_ARG, "ldq < N");
  if (N == 0) return fail(SPENSE_ERR_ARG, "N = 0");
  const size_t need = spense_gemm_glu_fp8_workspace_size(M, N);
  if (!ws || ws_bytes < need)
    return fail(SPENSE_ERR_WS, "workspace of %zu bytes needed, %zu given", need, ws ? ws_bytes : (size_t)0);
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(SPENSE_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (M * ceil_div(N, 2048) > INT32_MAX) return fail(SPENSE_ERR_ARG, "M x N too large for the quantisation grid");
  rc = check_device();
  if (rc) return rc;
  float* H = static_cast<float*>(ws);
  float* hmax = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + glu_hmax_offset(M, N));
  int32_t groups = 0;
  rc = launch_glu_pair(X, M, ldx, gate, up, w_scale_gate, w_scale_up, x_scale, H, glu_ldh(N), hmax, &groups, stream);
  if (rc) return rc;
  if (spense::launch_quantize_rowmax(H, glu_ldh(N), M, N, hmax, groups, q, ldq, scales, stream) != hipSuccess)
    return fail(SPENSE_ERR_HIP, "quantize launch failed");
  return ok();
}



size_t spense_dense_gemm_workspace_size(int64_t M, int64_t N, int64_t K, int32_t dtype) {
  spense_layout_t L;
  if (M <= 0 || M > INT32_MAX || layout_impl(N, K, dtype, SPENSE_SPLIT_OUTPUT, 0, &L)) return 0;
  return cached_plan(dtype, M, N, SPENSE_SPLIT_OUTPUT, K, 0, false, Override()).ws_bytes;
}

int spense_dense_gemm(const void* X, int64_t M, int64_t ldx, const void* W, int64_t ldw, int64_t N, int64_t K,
                      int32_t dtype, const float* w_scale, const float* x_scale, void* Y, int64_t ldy,
                      uint32_t out_flags, void* ws, size_t ws_bytes, hipStream_t stream) {
  spense_layout_t L;
  int rc = layout_impl(N, K, dtype, SPENSE_SPLIT_OUTPUT, 0, &L);
  if (rc) return rc;
  const int es = esize(dtype);
  if (N > 0 && K > 0) {
    if (!W) return fail(SPENSE_ERR_ARG, "W is NULL");
    if (ldw < K) return fail(SPENSE_ERR_ARG, "ldw < K");
    if (!aligned16(W) || (ldw * es) % 16) return fail(SPENSE_ERR_ALIGN, "W must be 16-byte aligned, 16-byte pitch");
  }
  return gemm_common(X, M, ldx, dtype, SPENSE_SPLIT_OUTPUT, N, K, 0, SPENSE_LAYOUT_ROWMAJOR, nullptr, 0, nullptr, 0, W,
                     ldw, w_scale, x_scale, Y, ldy, out_flags, ws, ws_bytes, Override(), stream);
}

}  // extern "C"
