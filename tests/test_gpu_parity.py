"""GPU parity: libspense (through its C ABI) against the CPU oracle on the same seeded
inputs.

- compression / metadata: bit-exact;
- GEMM, fp32 output: elementwise |y - y_exact| <= (delta + 2*gamma_K) * sum_k |x w| *
  |sw sx| + 4u|y_exact| against the fp64 oracle, with gamma_K = K u / (1 - K u),
  u = 2^-24, and delta = 2^-12 for fp8 (the gfx950 fp8 matrix instructions sum the
  products of one lane's K chunk with about 13 fractional bits relative to the largest
  one; measured) or 0 for bf16;
- GEMM, bf16 output: relative Frobenius <= 5e-3 (fp8) / 1e-3 (bf16 inputs) and max
  element error <= 1e-2 * max|Y_ref|, both sides rounded to bf16;
- exact-integer inputs (all partial sums exact in fp32): bit-exact in both output modes.
Full-size workloads compare sampled output rows (the oracle computes those rows only)
and run the exact-integer case on the whole output.
"""
import functools
import os
import sys

import numpy as np
import pytest
import torch

import gen
import oracle

pytestmark = pytest.mark.gpu

FP8, BF16 = 1, 2


@pytest.fixture(scope="module")
def S():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10445_amd as S
    return S


def say(*a):
    print(*a, file=sys.stderr, flush=True)


# ------------------------------------------------------------------ helpers
def tdev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(a).cuda()


def tnp(t: torch.Tensor, dt=None) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        t = t.view(torch.int16)
    a = t.cpu().numpy()
    if a.dtype == np.int16:
        a = a.view(np.uint16)
    if a.dtype == np.int32 and dt == np.uint32:
        a = a.view(np.uint32)
    return a


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def gdt(dtype):
    return gen.FP8 if dtype == FP8 else gen.BF16


def gaxis(axis):
    return gen.OUTPUT if axis == 0 else gen.INPUT


def compress_both(S, W, mask, dtype, axis, db, use_mask=True):
    """GPU compress (checked bit-exact against the oracle); returns the packed weight."""
    pw = S.compress(tdev(W), tdev(mask) if use_mask else None, axis, db)
    v, m, d, bad = oracle.compress(W, mask if use_mask else None, dtype, axis, db)
    assert bad == 0
    assert np.array_equal(tnp(pw.values), v), "values differ"
    assert np.array_equal(tnp(pw.meta, np.uint32), m), "metadata differs"
    assert np.array_equal(tnp(pw.dense), d), "dense region differs"
    return pw, (v, m, d)


def assert_bf16_close(y_bits, ref_bits, dtype):
    g, r = bf16_to_f64(y_bits), bf16_to_f64(ref_bits)
    assert not np.any(np.isnan(g)) and not np.any(np.isnan(r))
    rmax = np.abs(r).max() if r.size else 0.0
    if rmax == 0:
        assert np.all(g == 0)
        return
    rel = np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-300)
    tol = 5e-3 if dtype == FP8 else 1e-3
    assert rel <= tol, f"relative Frobenius error {rel:.3e} > {tol}"
    err = np.abs(g - r).max()
    assert err <= 1e-2 * rmax, f"max error {err:.3e} > 1e-2 * {rmax:.3e}"


U32 = 2.0 ** -24


def assert_f32_bound(y, X, Wd, dtype, sw=None, sx=None):
    """fp32 output against the fp64 oracle within the bound derived in the docstring."""
    o = oracle.gemm_f64(X, Wd, dtype, sw, sx)
    K = X.shape[1]
    gamma = K * U32 / (1 - K * U32)
    delta = 2.0 ** -12 if dtype == FP8 else 0.0
    scale = np.ones_like(o["y"])
    if sw is not None:
        scale = scale * np.abs(sw.astype(np.float64))[None, :]
    if sx is not None:
        scale = scale * np.abs(sx.astype(np.float64))[:, None]
    bound = (delta + 2 * gamma) * o["abs_dot"] * scale + 4 * U32 * np.abs(o["y"]) + 1e-38
    err = np.abs(y.astype(np.float64) - o["y"])
    worst = float((err / bound).max()) if err.size else 0.0
    assert worst <= 1.0, f"fp32 output exceeds the error bound by {worst:.2f}x"


def run_gemm(S, pw, X, sw, sx, out_f32, plan=None):
    y = S.gemm(tdev(X), pw, None if sw is None else tdev(sw), None if sx is None else tdev(sx), out_f32=out_f32,
               plan=plan)
    torch.cuda.synchronize()
    return tnp(y)


def random_case(seed, M, N, K, axis, db, dtype, allow_fewer=True):
    r = np.random.default_rng(seed)
    if dtype == FP8:
        W, sw = gen.quantize_rows_fp8(gen.draw_weight(r, N, K))
        X, sx = gen.quantize_rows_fp8(gen.draw_x(r, M, K, "student_t4"))
    else:
        W, sw = gen.to_bf16(gen.draw_weight(r, N, K)), None
        X, sx = gen.to_bf16(gen.draw_x(r, M, K)), None
    mask = gen.random_mask_24(r, N, K, gaxis(axis), db, allow_fewer)
    return W, mask, X, sw, sx


# ------------------------------------------------------------------ compression
COMPRESS_CASES = [
    (FP8, 0, 48, 256, 32), (FP8, 1, 40, 256, 160), (BF16, 0, 33, 128, 17), (BF16, 1, 16, 512, 384),
    (FP8, 0, 100, 1024, 0), (FP8, 0, 100, 1024, 100), (FP8, 1, 7, 96, 0), (FP8, 1, 7, 96, 96),
]


@pytest.mark.parametrize("dtype,axis,N,K,db", COMPRESS_CASES)
@pytest.mark.parametrize("use_mask", [True, False])
def test_compress_bit_exact(S, dtype, axis, N, K, db, use_mask):
    W, mask, _, _, _ = random_case(1, 1, N, K, axis, db, dtype)
    if not use_mask:  # zero the pruned entries so the bit pattern carries the mask
        W = W * mask.astype(W.dtype)
    compress_both(S, W, mask, dtype, axis, db, use_mask)


def test_compress_rejects_three_of_four(S):
    W = np.full((8, 64), 0x38, np.uint8)
    mask = np.ones((8, 64), np.uint8)
    mask[2, 4:8] = [1, 1, 1, 0]
    mask[5, 32:36] = [1, 1, 1, 1]
    mask[:, 8:] = 0
    mask[:, 8:10] = 1
    with pytest.raises(S.SpenseError) as e:
        S.compress(tdev(W), tdev(mask), 0, 8)
    assert e.value.code == S.SPENSE_ERR_MASK
    # every group with more than two kept entries is counted: rows 0..7 groups 0,1 keep 4
    _, _, _, bad = oracle.compress(W, mask, FP8, 0, 8)
    assert e.value.bad_groups == bad


@pytest.mark.parametrize("dtype,axis,N,K,db", COMPRESS_CASES[:4])
def test_decompress_round_trip(S, dtype, axis, N, K, db):
    W, mask, _, _, _ = random_case(2, 1, N, K, axis, db, dtype)
    pw, _ = compress_both(S, W, mask, dtype, axis, db)
    back = tnp(S.decompress(pw))
    assert np.array_equal(back, W * mask.astype(W.dtype))


# ------------------------------------------------------------------ GEMM, small shapes
GEMM_CASES = [
    # dtype, axis, M, N, K, dense_begin
    (FP8, 0, 1, 256, 512, 192), (FP8, 0, 17, 100, 544, 48), (FP8, 0, 64, 272, 1024, 208),
    (FP8, 0, 65, 96, 256, 80), (FP8, 1, 3, 128, 640, 480), (FP8, 1, 33, 200, 1056, 800),
    (FP8, 1, 100, 64, 2048, 1536), (FP8, 1, 1, 48, 160, 32), (BF16, 0, 1, 256, 512, 192),
    (BF16, 1, 1, 256, 512, 384), (BF16, 0, 40, 130, 352, 66), (BF16, 1, 20, 90, 480, 224),
    (FP8, 0, 5, 64, 128, 0), (FP8, 0, 5, 64, 128, 64), (FP8, 1, 5, 64, 128, 0), (FP8, 1, 5, 64, 128, 128),
]


@pytest.mark.parametrize("dtype,axis,M,N,K,db", GEMM_CASES)
def test_gemm_parity(S, dtype, axis, M, N, K, db):
    W, mask, X, sw, sx = random_case(3, M, N, K, axis, db, dtype)
    pw, (v, m, d) = compress_both(S, W, mask, dtype, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, dtype, axis, db, sw, sx)
    y32 = run_gemm(S, pw, X, sw, sx, True)
    assert_f32_bound(y32, X, oracle.decompress(v, m, d, N, K, dtype, axis, db), dtype, sw, sx)
    ybf = run_gemm(S, pw, X, sw, sx, False).view(np.uint16)
    assert_bf16_close(ybf, ref["y_bf16"], dtype)


@pytest.mark.parametrize("dtype,axis,M,N,K,db", GEMM_CASES)
def test_gemm_exact_integers_bit_exact(S, dtype, axis, M, N, K, db):
    W, mask, X, sw, sx = gen.make_exact_int(11, N, M, N, K, gaxis(axis), db, gdt(dtype))
    pw, (v, m, d) = compress_both(S, W, mask, dtype, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, dtype, axis, db, sw, sx)
    assert np.array_equal(run_gemm(S, pw, X, sw, sx, True), ref["y_f32"])
    assert np.array_equal(run_gemm(S, pw, X, sw, sx, False).view(np.uint16), ref["y_bf16"])


@pytest.mark.parametrize("axis", [0, 1])
@pytest.mark.parametrize("M", [1, 40])
def test_dense_fraction_one_equals_dense_gemm(S, axis, M):
    N, K = 300, 2048
    W, _, X, sw, sx = random_case(4, M, N, K, axis, 0, FP8)
    pw, _ = compress_both(S, W, np.ones_like(W), FP8, axis, 0)
    y1 = run_gemm(S, pw, X, sw, sx, True)
    y2 = S.dense_gemm(tdev(X), tdev(W), tdev(sw), tdev(sx), out_f32=True)
    torch.cuda.synchronize()
    assert np.array_equal(y1, tnp(y2))
    assert_f32_bound(y1, X, W, FP8, sw, sx)


def test_repeated_calls_are_bitwise_identical(S):
    M, N, K, db = 64, 5120, 8192, 6144  # input-split with split K
    W, mask, X, sw, sx = random_case(5, M, N, K, 1, db, FP8)
    pw = S.compress(tdev(W), tdev(mask), 1, db)
    Xd, swd, sxd = tdev(X), tdev(sw), tdev(sx)
    outs = [tnp(S.gemm(Xd, pw, swd, sxd, out_f32=True)) for _ in range(3)]
    assert all(np.array_equal(outs[0], o) for o in outs[1:])


# forced plans (spense_gemm_planned): kernel 1 = K split over a workgroup's waves, 2 = rows
# split with activations in LDS, 3 = large-M tiles; None = the planner's own choice
KSPLIT, ROWS, BIG, BIG2 = 1, 2, 3, 4
KERNEL_SHAPES = [None, dict(kernel=KSPLIT, waves=4, row_tiles=1), dict(kernel=KSPLIT, waves=16, row_tiles=1),
                 dict(kernel=KSPLIT, waves=8, row_tiles=2), dict(kernel=KSPLIT, waves=8, row_tiles=1, u8=1),
                 dict(kernel=KSPLIT, waves=4, row_tiles=2), dict(kernel=KSPLIT, waves=4, row_tiles=4),
                 dict(kernel=ROWS, waves=4, row_tiles=1),
                 dict(kernel=ROWS, waves=8, row_tiles=1),
                 dict(kernel=ROWS, waves=8, row_tiles=1, ksplit=4),
                 dict(kernel=ROWS, waves=4, row_tiles=1, ksplit=7),
                 dict(kernel=ROWS, waves=4, row_tiles=2),
                 dict(kernel=ROWS, waves=4, row_tiles=2, ksplit=3),
                 dict(kernel=BIG, waves=8), dict(kernel=BIG, waves=4), dict(kernel=BIG2, waves=8)]


def plan(S, cfg):
    return None if cfg is None else S.plan_override(**cfg)


@pytest.mark.parametrize("axis,db", [(1, 6144), (0, 1536)])
@pytest.mark.parametrize("dtype", [FP8, BF16])
def test_every_kernel_shape_is_repeatable_and_within_bound(S, dtype, axis, db):
    """Repeated calls on the same inputs are bitwise identical and inside the error bound
    for every kernel and workgroup shape, with both regions present.  This guards the
    points where a matrix-core result is read by a later instruction in another basic
    block (2:4 -> dense switch, loop tails, the reduction and the epilogue): a result read
    before the matrix core has written it shows up as run-to-run differences."""
    N, K = 2048, 8192
    W, mask, X, sw, sx = random_case(6, 64, N, K, axis, db, dtype)
    pw, (v, m, d) = compress_both(S, W, mask, dtype, axis, db)
    Wd = oracle.decompress(v, m, d, N, K, dtype, axis, db)
    for cfg in KERNEL_SHAPES:
        if cfg is not None and cfg["kernel"] in (BIG, BIG2) and dtype != FP8:
            continue
        for M in (64, 33, 7, 1):
            swd = None if sw is None else tdev(sw)
            sxd = None if sx is None else tdev(sx[:M])
            Xd = tdev(X[:M])
            outs = [tnp(S.gemm(Xd, pw, swd, sxd, out_f32=True, plan=plan(S, cfg))) for _ in range(4)]
            assert all(np.array_equal(outs[0], o) for o in outs[1:]), f"{cfg} M={M}: calls differ"
            assert_f32_bound(outs[0], X[:M], Wd, dtype, sw, None if sx is None else sx[:M])


def test_back_to_back_calls_with_smaller_second_call(S):
    N, K, db = 2048, 8192, 6144
    W, mask, X, sw, sx = random_case(6, 64, N, K, 1, db, FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, 1, db)
    ws = S.Workspace("cuda")
    for M in (64, 7):
        y = tnp(S.gemm(tdev(X[:M]), pw, tdev(sw), tdev(sx[:M]), out_f32=True, workspace=ws))
        assert_f32_bound(y, X[:M], oracle.decompress(v, m, d, N, K, FP8, 1, db), FP8, sw, sx[:M])


def test_strided_operands(S):
    """Leading dimensions larger than the logical widths."""
    M, N, K, db = 9, 80, 256, 48
    W, mask, X, sw, sx = random_case(7, M, N, K, 0, db, FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, 0, db)
    Xbig = torch.zeros((M, K + 64), dtype=torch.uint8, device="cuda")
    Xbig[:, :K] = tdev(X)
    Ybig = torch.full((M, N + 8), 7.0, dtype=torch.float32, device="cuda")
    S.gemm(Xbig[:, :K], pw, tdev(sw), tdev(sx), out=Ybig[:, :N], out_f32=True)
    torch.cuda.synchronize()
    assert_f32_bound(tnp(Ybig[:, :N]), X, oracle.decompress(v, m, d, N, K, FP8, 0, db), FP8, sw, sx)
    assert torch.all(Ybig[:, N:] == 7.0)


def test_error_paths_leave_output_untouched(S):
    M, N, K, db = 4, 64, 256, 32
    W, mask, X, sw, sx = random_case(8, M, N, K, 0, db, FP8)
    pw = S.compress(tdev(W), tdev(mask), 0, db)
    Y = torch.full((M, N), 3.0, dtype=torch.float32, device="cuda")
    Xd = tdev(X)
    rc = S.spense_gemm(Xd.data_ptr() + 1, M, K, pw.desc, None, None, Y.data_ptr(), N, 1, None, 0,
                       torch.cuda.current_stream().cuda_stream)
    assert rc == S.SPENSE_ERR_ALIGN
    rc = S.spense_gemm(Xd.data_ptr(), M, K - 32, pw.desc, None, None, Y.data_ptr(), N, 1, None, 0,
                       torch.cuda.current_stream().cuda_stream)
    assert rc == S.SPENSE_ERR_ARG
    torch.cuda.synchronize()
    assert torch.all(Y == 3.0)


# ------------------------------------------------------------------ tiled execution layout
def tiled_reference(v, m, d, N, K, axis, db):
    """The tiled layout built on the CPU from the row-major buffers, by padding and
    reshaping as the header defines it (tiles of 16 rows, chunks of 512 columns)."""
    sr, sc = (db, K) if axis == 0 else (N, db)
    dr, dc = (N - db, K) if axis == 0 else (N, K - db)

    def pad(a, rows, cols):
        out = np.zeros((rows, cols), a.dtype)
        out[:a.shape[0], :a.shape[1]] = a
        return out

    vt = mt = np.zeros(0, np.uint8)
    if sr and sc:
        T, C = -(-sr // 16), -(-sc // 512)
        vp = pad(v.reshape(sr, sc // 2), 16 * T, 256 * C)  # byte 256c + 64j + 16q + b of row 16t + i
        vt = vp.reshape(T, 16, C, 4, 4, 16).transpose(0, 2, 3, 4, 1, 5).ravel()
        mp = pad(m.reshape(sr, sc // 32), 16 * T, 16 * C)  # word 16c + 4q + k of row 16t + i
        mt = mp.reshape(T, 16, C, 4, 4).transpose(0, 2, 3, 1, 4).ravel().view(np.uint8)
    dt = np.zeros(0, np.uint8)
    if dr and dc:
        T, C = -(-dr // 16), -(-dc // 512)
        dp = pad(d.reshape(dr, dc), 16 * T, 512 * C)  # byte 512c + 128j + 64p + 16q + b
        dt = dp.reshape(T, 16, C, 4, 2, 4, 16).transpose(0, 2, 3, 4, 5, 1, 6).ravel()
    return vt, mt, dt


TILE_CASES = [(0, 256, 1024, 192), (1, 256, 1024, 768), (0, 200, 1056, 72), (1, 200, 1056, 800), (0, 17, 96, 0),
              (1, 17, 96, 96), (0, 40, 544, 40), (1, 33, 2080, 32)]


@pytest.mark.parametrize("axis,N,K,db", TILE_CASES)
def test_tile_matches_definition(S, axis, N, K, db):
    W, mask, X, sw, sx = random_case(30 + N, 4, N, K, axis, db, FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    pwt = S.tile(pw)
    torch.cuda.synchronize()
    vt, mt, dt = tiled_reference(v, m, d, N, K, axis, db)
    assert np.array_equal(tnp(pwt.values), vt)
    assert np.array_equal(tnp(pwt.meta).view(np.uint8), mt)
    assert np.array_equal(tnp(pwt.dense), dt)


@pytest.mark.parametrize("axis,N,K,db", TILE_CASES)
@pytest.mark.parametrize("M", [1, 7, 20, 64, 130])
def test_tiled_gemm_equals_row_major(S, axis, N, K, db, M):
    """The tiled weight gives bit-for-bit the output of the row-major weight under the
    same (row-split) plan, and stays inside the error bound against the oracle."""
    W, mask, X, sw, sx = random_case(40 + N, M, N, K, axis, db, FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    pwt = S.tile(pw)
    rows = S.plan_override(kernel=ROWS)
    for f32 in (True, False):
        a = run_gemm(S, pw, X, sw, sx, f32, rows)
        b = run_gemm(S, pwt, X, sw, sx, f32, rows)
        assert np.array_equal(a, b)
    Wd = oracle.decompress(v, m, d, N, K, FP8, axis, db)
    assert_f32_bound(run_gemm(S, pwt, X, sw, sx, True), X, Wd, FP8, sw, sx)


def test_tiled_exact_integers(S):
    for axis, N, K, db in TILE_CASES:
        W, mask, X, sw, sx = gen.make_exact_int(21, N, 37, N, K, gaxis(axis), db, gen.FP8)
        pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
        ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
        pwt = S.tile(pw)
        assert np.array_equal(run_gemm(S, pwt, X, sw, sx, True), ref["y_f32"])
        assert np.array_equal(run_gemm(S, pwt, X, sw, sx, False).view(np.uint16), ref["y_bf16"])


# ------------------------------------------------------------------ large-M kernel
BIG_CASES = [  # axis, M, N, K, dense_begin: ragged tokens, rows and columns around its 256 x 128 x 128 tiles
    (0, 1, 200, 1056, 72), (0, 300, 272, 1024, 208), (1, 257, 200, 1056, 800), (1, 513, 136, 640, 128),
    (0, 600, 136, 384, 0), (0, 300, 136, 384, 136), (1, 300, 64, 512, 0), (1, 300, 64, 512, 512),
    # XCD-aware order: T = 2, 4, 8 token blocks with row blocks in 8, 8, 4 classes (two regions
    # for output-split; ragged tokens)
    (0, 512, 1024, 128, 512), (0, 1024, 1024, 256, 256), (1, 2048, 512, 384, 128), (1, 1900, 512, 256, 256)]
# 256 x 256 tiles: rows around 256-row blocks (both regions ragged), XCD-aware grids with
# 2, 4 and 8 token blocks and 8 / 4 row-block classes
BIG2_CASES = [(0, 700, 784, 640, 528), (1, 300, 600, 1152, 896), (0, 512, 2048, 256, 1024),
              (0, 1024, 2048, 384, 1536), (1, 2048, 1024, 256, 128)]


LARGE_M_KERNELS = [(BIG, 4), (BIG, 8), (BIG2, 8)]


@pytest.mark.parametrize("kernel,waves", LARGE_M_KERNELS)
@pytest.mark.parametrize("axis,M,N,K,db", BIG_CASES + BIG2_CASES)
def test_large_m_kernel_exact_both_layouts(S, axis, M, N, K, db, kernel, waves):
    """The large-M kernels (128-row x 256-token tiles with 4 or 8 waves, 256 x 256 tiles
    with 8 waves), forced on at any M, on exact-integer data: bit-exact against the oracle
    with the row-major and the tiled weight."""
    W, mask, X, sw, sx = gen.make_exact_int(13, M + N, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    big = S.plan_override(kernel=kernel, waves=waves)
    for w in (pw, S.tile(pw)):
        assert np.array_equal(run_gemm(S, w, X, sw, sx, True, big), ref["y_f32"])
        assert np.array_equal(run_gemm(S, w, X, sw, sx, False, big).view(np.uint16), ref["y_bf16"])


# K slices with two or three token blocks (65-192 tokens): few-row weights with a long K
# take them from the planner; (axis, M, N, K, db) with the slice count the planner picks.
KSLICE_BLOCK_CASES = [(1, 80, 2048, 24576, 18432, 6),  # 48 chunks: the planner takes two 64-token halves, 6 slices
                      (0, 100, 1024, 5120, 768, 4), (1, 150, 2048, 16384, 12288, 2), (0, 128, 1040, 6144, 784, 4)]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("axis,M,N,K,db,slices", KSLICE_BLOCK_CASES)
def test_k_slices_with_several_token_blocks_exact(S, axis, M, N, K, db, slices):
    """The planner's K slices above 64 tokens (workspace = slices x M x N floats), and
    forced 2 and 3 slices: bit-exact against the oracle on exact-integer data."""
    say(f"[kslices blocks] axis={axis} M={M} N={N} K={K} db={db}")
    W, mask, X, sw, sx = gen.make_exact_int(29, M + N, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    pwt = S.tile(pw)
    assert S.spense_gemm_workspace_size(M, pwt.desc) == slices * M * N * 4
    for plan in (None, S.plan_override(kernel=ROWS, ksplit=2), S.plan_override(kernel=ROWS, ksplit=3)):
        assert np.array_equal(run_gemm(S, pwt, X, sw, sx, True, plan), ref["y_f32"])
        assert np.array_equal(run_gemm(S, pwt, X, sw, sx, False, plan).view(np.uint16), ref["y_bf16"])


# The row-split kernel with two 64-token halves per workgroup (128 tokens a block; forced
# through the plan override, kernel 5): (axis, N, K, db) over both regions, ragged rows and
# columns, at token counts from one to several 128-token blocks.
ROWS2_CASES = [(0, 784, 1536, 528), (1, 600, 2560, 1792), (0, 300, 512, 208), (1, 136, 1024, 1024)]


@pytest.mark.parametrize("axis,N,K,db", ROWS2_CASES)
def test_two_half_row_split_exact(S, axis, N, K, db):
    """Bit-exact against the oracle on exact-integer data (fp32 and bf16 outputs)."""
    ROWS2 = 5
    for M in (1, 37, 64, 65, 100, 128, 129, 300):
        say(f"[rows2] axis={axis} N={N} K={K} db={db} M={M}")
        W, mask, X, sw, sx = gen.make_exact_int(31, M + N, M, N, K, gaxis(axis), db, gen.FP8)
        pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
        ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
        pwt = S.tile(pw)
        for ks in (1, 2, 3) if M in (37, 100, 300) else (1,):  # K slices: fp32 partials, then the reduction
            plan = S.plan_override(kernel=ROWS2, ksplit=ks)
            assert np.array_equal(run_gemm(S, pwt, X, sw, sx, True, plan), ref["y_f32"]), ks
            assert np.array_equal(run_gemm(S, pwt, X, sw, sx, False, plan).view(np.uint16), ref["y_bf16"]), ks


# Seeded random shapes for the same kernel: either split, any 2:4 / dense boundary (input
# split: multiples of 32), ragged N and K, 65-300 tokens, 1-4 K slices.
def _rows2_random_cases(n=10, seed=2411):
    r = np.random.default_rng(seed)
    out = []
    for i in range(n):
        axis = int(r.integers(0, 2))
        N = int(r.integers(16, 1200))
        K = 32 * int(r.integers(8, 100))
        db = int(r.integers(0, N + 1)) if axis == 0 else 32 * int(r.integers(0, K // 32 + 1))
        out.append((i, axis, N, K, db, int(r.integers(65, 301)), int(r.integers(1, 5))))
    return out


@pytest.mark.parametrize("i,axis,N,K,db,M,ks", _rows2_random_cases())
def test_two_half_random_shapes_exact(S, i, axis, N, K, db, M, ks):
    """Bit-exact against the oracle on exact-integer data, fp32 and bf16 outputs."""
    say(f"[rows2 random] axis={axis} N={N} K={K} db={db} M={M} ks={ks}")
    W, mask, X, sw, sx = gen.make_exact_int(33, i, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    plan = S.plan_override(kernel=5, ksplit=ks)
    pwt = S.tile(pw)
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, True, plan), ref["y_f32"])
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, False, plan).view(np.uint16), ref["y_bf16"])


# Its epilogue with N off multiples of 4 and a padded Y (leading dimension N + 8: 16-byte
# stores where a quad fits; N + 3: scalar stores), with and without K slices (the
# partials' scalar path): (axis, M, N, K, db).
ROWS2_OUT_CASES = [(0, 100, 203, 384, 100), (1, 130, 203, 1536, 256)]


@pytest.mark.parametrize("axis,M,N,K,db", ROWS2_OUT_CASES)
def test_two_half_output_paths_exact(S, axis, M, N, K, db):
    """Bit-exact bf16 and fp32 against the oracle into padded outputs; the padding is untouched."""
    W, mask, X, sw, sx = gen.make_exact_int(27, M + N, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    pwt = S.tile(pw)
    for ks in (1, 3):
        plan = S.plan_override(kernel=5, ksplit=ks)
        for pad in (8, 3):
            for out_f32 in (False, True):
                dt = torch.float32 if out_f32 else torch.bfloat16
                Ybig = torch.full((M, N + pad), 7.0, dtype=dt, device="cuda")
                S.gemm(tdev(X), pwt, tdev(sw), tdev(sx), out=Ybig[:, :N], out_f32=out_f32, plan=plan)
                torch.cuda.synchronize()
                got = tnp(Ybig[:, :N])
                want = ref["y_f32"] if out_f32 else ref["y_bf16"]
                assert np.array_equal(got if out_f32 else got.view(np.uint16), want), (ks, pad, out_f32)
                assert torch.all(Ybig[:, N:] == 7.0)


# The same kernel as the planner's own choice (tall weights at one 128-token block; two
# blocks where the row-split kernel would take three or four): (axis, N, K, db, M).
ROWS2_AUTO_CASES = [(0, 12288, 512, 9216, 100), (1, 12288, 384, 256, 127), (0, 8192, 512, 6144, 250),
                    (0, 10240, 256, 7680, 131),
                    # short weights with a long K: with K slices (6, 3 and 4)
                    (1, 320, 20992, 15744, 100), (1, 200, 20480, 15360, 250), (1, 300, 10240, 7680, 90),
                    # 257-768 tokens on 256-767 row tiles (a long K at 300: 2 slices)
                    (1, 4096, 20480, 15360, 300), (1, 4096, 1024, 768, 450), (0, 8192, 512, 6144, 300),
                    (1, 4100, 2048, 1536, 600), (0, 5000, 768, 3750, 700)]


@pytest.mark.parametrize("axis,N,K,db,M", ROWS2_AUTO_CASES)
def test_two_half_row_split_planned_exact(S, capfd, axis, N, K, db, M):
    """Bit-exact against the oracle with no override, the dispatch log naming the kernel."""
    say(f"[rows2 auto] axis={axis} N={N} K={K} db={db} M={M}")
    W, mask, X, sw, sx = gen.make_exact_int(37, M + N, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    pwt = S.tile(pw)
    prev = S.spense_set_log(1)
    try:
        capfd.readouterr()
        y32 = run_gemm(S, pwt, X, sw, sx, True)
        log = capfd.readouterr().err
    finally:
        S.spense_set_log(prev)
    assert "row-split, two 64-token halves" in log, log
    assert np.array_equal(y32, ref["y_f32"])
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, False).view(np.uint16), ref["y_bf16"])


# Seeded random shapes for the 64-token kernels (forced): the row-split kernel on either
# layout with 1-4 K slices, the K-split kernel on the row-major layout; 1-64 tokens.
def _rows_random_cases(n=10, seed=2413):
    r = np.random.default_rng(seed)
    out = []
    for i in range(n):
        axis = int(r.integers(0, 2))
        N = int(r.integers(16, 1500))
        K = 32 * int(r.integers(4, 120))
        db = int(r.integers(0, N + 1)) if axis == 0 else 32 * int(r.integers(0, K // 32 + 1))
        out.append((i, axis, N, K, db, int(r.integers(1, 65)), int(r.integers(1, 5))))
    return out


@pytest.mark.parametrize("i,axis,N,K,db,M,ks", _rows_random_cases())
def test_rows_random_shapes_exact(S, i, axis, N, K, db, M, ks):
    """Bit-exact fp32 and bf16 against the oracle on exact-integer data: row-split (tiled
    and row-major, ks K slices) and K-split (row-major)."""
    say(f"[rows random] axis={axis} N={N} K={K} db={db} M={M} ks={ks}")
    W, mask, X, sw, sx = gen.make_exact_int(37, i, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    pwt = S.tile(pw)
    for w, plan in ((pwt, S.plan_override(kernel=ROWS, ksplit=ks)), (pw, S.plan_override(kernel=ROWS, ksplit=ks)),
                    (pw, S.plan_override(kernel=1))):
        assert np.array_equal(run_gemm(S, w, X, sw, sx, True, plan), ref["y_f32"]), plan.kernel
        assert np.array_equal(run_gemm(S, w, X, sw, sx, False, plan).view(np.uint16), ref["y_bf16"]), plan.kernel


# The 256 x 256 kernel with 192-token blocks (257-384 and 513-576 tokens): (axis, M, N, K,
# db), ragged N, the last block partly filled; bf16 through LDS (leading dimension N + 8)
# and quad by quad (N + 3), and fp32.
TILE192_CASES = [(0, 257, 700, 512, 300), (1, 300, 520, 768, 256), (0, 384, 1100, 384, 1000), (1, 560, 640, 640, 320)]


@pytest.mark.parametrize("axis,M,N,K,db", TILE192_CASES)
def test_256_row_tiles_of_192_tokens_exact(S, axis, M, N, K, db):
    """Bit-exact against the oracle; the padding of Y is untouched."""
    say(f"[tiles 192] axis={axis} M={M} N={N} K={K} db={db}")
    W, mask, X, sw, sx = gen.make_exact_int(39, M + N, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    big2 = S.plan_override(kernel=BIG2, waves=8)
    pwt = S.tile(pw)
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, True, big2), ref["y_f32"])
    for pad in (0, 8, 3):
        Ybig = torch.full((M, N + pad), 7.0, dtype=torch.bfloat16, device="cuda")
        S.gemm(tdev(X), pwt, tdev(sw), tdev(sx), out=Ybig[:, :N], plan=big2)
        torch.cuda.synchronize()
        assert np.array_equal(tnp(Ybig[:, :N]), ref["y_bf16"]), pad
        assert torch.all(Ybig[:, N:] == 7.0)


# Seeded random shapes for the large-M kernels (forced): either split, any boundary, ragged
# N and K, 200-1100 tokens (partial last token blocks of both tile heights).
def _large_m_random_cases(n=6, seed=2412):
    r = np.random.default_rng(seed)
    out = []
    for i in range(n):
        axis = int(r.integers(0, 2))
        N = int(r.integers(100, 1400))
        K = 32 * int(r.integers(8, 60))
        db = int(r.integers(0, N + 1)) if axis == 0 else 32 * int(r.integers(0, K // 32 + 1))
        out.append((i, axis, N, K, db, int(r.integers(200, 1101))))
    return out


@pytest.mark.parametrize("kernel,waves", LARGE_M_KERNELS)
@pytest.mark.parametrize("i,axis,N,K,db,M", _large_m_random_cases())
def test_large_m_random_shapes_exact(S, i, axis, N, K, db, M, kernel, waves):
    """Bit-exact fp32 and bf16 against the oracle on exact-integer data."""
    say(f"[large-M random] kernel={kernel} waves={waves} axis={axis} N={N} K={K} db={db} M={M}")
    W, mask, X, sw, sx = gen.make_exact_int(35, i, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    plan = S.plan_override(kernel=kernel, waves=waves)
    pwt = S.tile(pw)
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, True, plan), ref["y_f32"])
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, False, plan).view(np.uint16), ref["y_bf16"])


# bf16 output of the large-M kernels: through LDS as whole token rows where Y is 16-byte
# aligned with ldy and the tile's first row multiples of 8, else quad by quad; (axis, M,
# N, K, db) with N and the 2:4 / dense boundary off multiples of 8 (a partial last block,
# a region starting mid-block) and ragged M.
OUT_CASES = [(0, 300, 203, 384, 100), (1, 520, 203, 512, 256), (0, 700, 600, 256, 300)]


@pytest.mark.parametrize("kernel,waves", LARGE_M_KERNELS)
@pytest.mark.parametrize("axis,M,N,K,db", OUT_CASES)
def test_large_m_output_paths_exact(S, axis, M, N, K, db, kernel, waves):
    """Bit-exact bf16 output against the oracle with a contiguous Y and with leading
    dimensions N + 8 (rows through LDS) and N + 3 (quad stores); the padding is untouched."""
    W, mask, X, sw, sx = gen.make_exact_int(23, M + N, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    big = S.plan_override(kernel=kernel, waves=waves)
    pwt = S.tile(pw)
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, False, big).view(np.uint16), ref["y_bf16"])
    for pad in (8, 3):
        Ybig = torch.full((M, N + pad), 7.0, dtype=torch.bfloat16, device="cuda")
        S.gemm(tdev(X), pwt, tdev(sw), tdev(sx), out=Ybig[:, :N], plan=big)
        torch.cuda.synchronize()
        assert np.array_equal(tnp(Ybig[:, :N]).view(np.uint16), ref["y_bf16"])
        assert torch.all(Ybig[:, N:] == 7.0)


# 256 x 256 kernel with its last row blocks as 256 x 128 tiles at the end of the grid:
# (axis, M, N, K, db, half row blocks); ragged M (a half tile past M, a partial one),
# ragged rows in both regions, the XCD-aware order on the full tiles with leftover row
# blocks in place, and every row block split.
BIG2_HALF_CASES = [(0, 700, 784, 640, 528, 1), (0, 700, 784, 640, 528, 3), (1, 300, 600, 1152, 896, 1),
                   (0, 1024, 2048, 384, 1536, 2), (1, 2048, 1024, 256, 128, 3), (1, 2048, 1024, 256, 128, 4),
                   (0, 520, 2304, 512, 1792, 5)]


@pytest.mark.parametrize("axis,M,N,K,db,rh", BIG2_HALF_CASES)
def test_large_m_half_tiles_exact(S, axis, M, N, K, db, rh):
    """256 x 128 tail tiles (the waves of the missing token quarters only copy): bit-exact
    against the oracle on exact-integer data, and equal to the plan without them."""
    W, mask, X, sw, sx = gen.make_exact_int(17, M + N + rh, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    pwt = S.tile(pw)
    half = S.plan_override(kernel=BIG2, waves=8, half_row_blocks=rh)
    whole = S.plan_override(kernel=BIG2, waves=8, half_row_blocks=0)
    y32 = run_gemm(S, pwt, X, sw, sx, True, half)
    assert np.array_equal(y32, ref["y_f32"])
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, False, half).view(np.uint16), ref["y_bf16"])
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, True, whole), y32)


# One or two token tiles with the whole K range of activations resident in LDS: (axis, M,
# N, K, db); ragged M, N and K, both regions, up to 20 chunks of 512 columns with one
# token tile and 10 with two (the LDS limit).
XRES_CASES = [(0, 1, 300, 640, 208), (0, 16, 1040, 5120, 784), (1, 7, 520, 2080, 1536), (1, 13, 264, 10240, 7680),
              (0, 5, 2064, 10240, 1040), (1, 16, 48, 512, 256), (0, 17, 1040, 5120, 784), (1, 32, 520, 4608, 3584),
              (0, 29, 300, 640, 208)]


@pytest.mark.parametrize("axis,M,N,K,db", XRES_CASES)
def test_resident_activations_exact(S, axis, M, N, K, db):
    """The row-split kernel with every chunk's activations kept in LDS (forced on, also
    where the planner would not choose it): bit-exact against the oracle on exact-integer
    data and equal to the chunk-by-chunk staging."""
    W, mask, X, sw, sx = gen.make_exact_int(19, M + N + K, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    pwt = S.tile(pw)
    on = S.plan_override(kernel=ROWS, row_tiles=1, waves=8, ksplit=1, resident_x=2)
    off = S.plan_override(kernel=ROWS, row_tiles=1, waves=8, ksplit=1, resident_x=1)
    y32 = run_gemm(S, pwt, X, sw, sx, True, on)
    assert np.array_equal(y32, ref["y_f32"])
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, False, on).view(np.uint16), ref["y_bf16"])
    assert np.array_equal(run_gemm(S, pwt, X, sw, sx, True, off), y32)


@pytest.mark.parametrize("kernel,waves", LARGE_M_KERNELS)
@pytest.mark.parametrize("axis,db", [(0, 744), (1, 1536)])
def test_large_m_kernel_random_within_bound(S, axis, db, kernel, waves):
    """Random data through the large-M kernel: inside the error bound against the oracle,
    equal with both layouts and bitwise repeatable."""
    M, N, K = 520, 1000, 2080
    W, mask, X, sw, sx = random_case(6, M, N, K, axis, db, FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    Wd = oracle.decompress(v, m, d, N, K, FP8, axis, db)
    pwt = S.tile(pw)
    big = S.plan_override(kernel=kernel, waves=waves)
    y32 = run_gemm(S, pw, X, sw, sx, True, big)
    assert_f32_bound(y32, X, Wd, FP8, sw, sx)
    assert_bf16_close(run_gemm(S, pw, X, sw, sx, False, big).view(np.uint16), ref["y_bf16"], FP8)
    for _ in range(2):
        assert np.array_equal(run_gemm(S, pwt, X, sw, sx, True, big), y32)


# ------------------------------------------------------------------ full-size workloads
@functools.lru_cache(maxsize=4)
def _matrix(cfg, mat, name, N, K, axis, frac, dtype):
    say(f"[gen] cfg{cfg} {name} {N}x{K} {axis} p={frac}")
    return gen.make_matrix(cfg, mat, name, N, K, axis, frac, dtype)


def _full_case(S, cfg, mat, name, N, K, axis, frac, ms, xdist, sample_rows=384):
    """Both storage layouts (row-major as compressed, and tiled) against the oracle on a
    sample of weight rows (every activation row)."""
    mx = _matrix(cfg, mat, name, N, K, axis, frac, gen.FP8)
    ax = 0 if axis == gen.OUTPUT else 1
    say(f"[compress] cfg{cfg} {name} dense_begin={mx.dense_begin}")
    pw, (v, m, d) = compress_both(S, mx.W, mx.mask, FP8, ax, mx.dense_begin)
    pwt = S.tile(pw)
    Wd = oracle.decompress(v, m, d, N, K, FP8, ax, mx.dense_begin)
    rows = np.sort(np.random.default_rng(cfg * 100 + mat).choice(N, size=min(N, sample_rows), replace=False))
    for M in ms:
        X, sx = gen.make_x(cfg, mat, M, K, gen.FP8, xdist)
        ref = oracle.gemm(X, Wd[rows], FP8, mx.sw[rows], sx)
        for w, lay in ((pw, "row-major"), (pwt, "tiled")):
            say(f"[gemm] cfg{cfg} {name} M={M} {lay}")
            y = run_gemm(S, w, X, mx.sw, sx, False).view(np.uint16)
            assert_bf16_close(y[:, rows], ref["y_bf16"], FP8)
            y32 = run_gemm(S, w, X, mx.sw, sx, True)
            assert_f32_bound(y32[:, rows], X, Wd[rows], FP8, mx.sw[rows], sx)


def test_full_tiny_bf16_both_axes(S):
    """Tiny linear 256x512 bf16, 25% dense, M=1: the whole output against the oracle."""
    for name, N, K, axis in gen.WORKLOADS[1]["mats"]:
        mx = gen.make_matrix(1, 0 if axis == gen.OUTPUT else 1, name, N, K, axis, 0.25, gen.BF16)
        ax = 0 if axis == gen.OUTPUT else 1
        assert mx.dense_begin == (192 if ax == 0 else 384)
        pw, (v, m, d) = compress_both(S, mx.W, mx.mask, BF16, ax, mx.dense_begin)
        X, _ = gen.make_x(1, 0, 1, K, gen.BF16)
        ref = oracle.spense_gemm(X, v, m, d, N, K, BF16, ax, mx.dense_begin)
        assert_bf16_close(run_gemm(S, pw, X, None, None, False).view(np.uint16), ref["y_bf16"], BF16)
        Wd = oracle.decompress(v, m, d, N, K, BF16, ax, mx.dense_begin)
        assert_f32_bound(run_gemm(S, pw, X, None, None, True), X, Wd, BF16)


@pytest.mark.timeout(300)
def test_full_gate_up_25600x5120(S):
    _full_case(S, 2, 0, "gate_up", 25600, 5120, gen.OUTPUT, 0.25, [1, 8, 32, 64], "normal")


@pytest.mark.timeout(400)
@pytest.mark.parametrize("frac", [0.0, 0.125, 0.25, 0.5, 1.0])
def test_full_down_5120x25600_dense_sweep(S, frac):
    _full_case(S, 3, 0, "down", 5120, 25600, gen.INPUT, frac, [1, 16, 64], "student_t4", sample_rows=256)


@pytest.mark.timeout(400)
@pytest.mark.parametrize("layer", [4, 5])
def test_full_layer_linears(S, layer):
    ms = [64] if layer == 4 else [1, 4, 16, 64, 256, 2048]
    for i, (name, N, K, axis) in enumerate(gen.WORKLOADS[layer]["mats"]):
        if name in ("up",):  # same shape as gate, other seed; gate covers it
            continue
        _full_case(S, layer, i, name, N, K, axis, 0.25, ms if name in ("gate", "down") else [ms[-1]], "normal",
                   sample_rows=128)


SEED_DECODE_MS = [1, 4, 16, 64, 256]


@pytest.mark.timeout(400)
@pytest.mark.parametrize("name", ["q", "k", "v", "o"])
def test_full_seed_oss_attention_linears_at_decode_m(S, name):
    """Seed-OSS-36B-like q (10240 x 5120), k / v (1024 x 5120) and o (5120 x 10240,
    input-split) at every decode M the benchmark times (1, 4, 16, 64, 256): random data
    on sampled rows, both layouts, bf16 tolerance and the fp32 bound.  These run the
    plans the layer timing uses, among them k / v with 4 K slices at every M and o with
    4 K slices from 17 tokens."""
    i, (nm, N, K, axis) = next((i, m) for i, m in enumerate(gen.WORKLOADS[5]["mats"]) if m[0] == name)
    _full_case(S, 5, i, nm, N, K, axis, 0.25, SEED_DECODE_MS, "normal", sample_rows=128)


@pytest.mark.timeout(400)
@pytest.mark.parametrize("name", ["q", "k", "o"])
def test_seed_oss_decode_exact_whole_output(S, name):
    """The same weights' shapes on exact-integer data: the whole output bit for bit, in
    both layouts, at M = 256, 64, 20, 16, 4 and 1 (the activations of a smaller M are the
    first rows of the larger draw, and each output row depends on its own row only)."""
    _, N, K, axis = next(m for m in gen.WORKLOADS[5]["mats"] if m[0] == name)
    ax = 0 if axis == gen.OUTPUT else 1
    db = gen.split_point(N, K, axis, 0.25)
    Mmax = 256
    W, mask, X, sw, sx = gen.make_exact_int(22, N % 89, Mmax, N, K, axis, db, gen.FP8)
    say(f"[exact seed] {name} {N}x{K}")
    pw, (v, m, d) = compress_both(S, W, mask, FP8, ax, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, ax, db, sw, sx)
    for w in (pw, S.tile(pw)):
        for M in (256, 64, 20, 16, 4, 1):
            y32 = run_gemm(S, w, X[:M], sw, sx[:M], True)
            ybf = run_gemm(S, w, X[:M], sw, sx[:M], False).view(np.uint16)
            assert np.array_equal(y32, ref["y_f32"][:M]), f"{name} M={M} fp32"
            assert np.array_equal(ybf, ref["y_bf16"][:M]), f"{name} M={M} bf16"


@pytest.mark.timeout(400)
@pytest.mark.parametrize("name,N,K,axis,M", [("gate_up", 25600, 5120, gen.OUTPUT, 64),
                                             ("down", 5120, 25600, gen.INPUT, 64),
                                             ("seed_gate", 27648, 5120, gen.OUTPUT, 2048),
                                             ("k", 1024, 5120, gen.OUTPUT, 64),
                                             ("k", 1024, 5120, gen.OUTPUT, 1),  # 4 K slices at one token
                                             ("gate_up", 25600, 5120, gen.OUTPUT, 100),  # large-M kernel, one block
                                             ("o", 5120, 8192, gen.INPUT, 40)])  # 3 K slices
def test_full_size_exact_integers_whole_output(S, name, N, K, axis, M):
    ax = 0 if axis == gen.OUTPUT else 1
    db = gen.split_point(N, K, axis, 0.25)
    W, mask, X, sw, sx = gen.make_exact_int(20, N % 97, M, N, K, axis, db, gen.FP8)
    say(f"[exact] {name} M={M}")
    pw, (v, m, d) = compress_both(S, W, mask, FP8, ax, db)
    Wd = oracle.decompress(v, m, d, N, K, FP8, ax, db)
    sel = np.arange(M) if M <= 256 else np.sort(np.random.default_rng(1).choice(M, 64, replace=False))
    ref = oracle.gemm(X[sel], Wd, FP8, sw, sx[sel])  # a sample of activation rows past M = 256
    for w in (pw, S.tile(pw)):
        y32 = run_gemm(S, w, X, sw, sx, True)
        ybf = run_gemm(S, w, X, sw, sx, False).view(np.uint16)
        assert np.array_equal(y32[sel], ref["y_f32"]) and np.array_equal(ybf[sel], ref["y_bf16"])


@pytest.mark.parametrize("rows,rt,waves,wused,ks", [(0, 1, 4, 0, 0), (0, 2, 4, 0, 0), (0, 1, 8, 0, 0), (0, 2, 8, 0, 0),
                                                    (0, 1, 16, 0, 0), (0, 4, 4, 0, 0), (1, 1, 4, 0, 1), (1, 1, 8, 0, 1),
                                                    (1, 1, 4, 3, 1), (1, 1, 8, 5, 1), (1, 1, 8, 8, 1), (1, 1, 4, 0, 2),
                                                    (1, 1, 8, 3, 3), (1, 1, 8, 8, 2), (1, 2, 4, 0, 1), (1, 2, 4, 3, 2)])
@pytest.mark.parametrize("dtype,axis,M", [(FP8, 1, 3), (FP8, 0, 40), (BF16, 1, 20), (FP8, 1, 64), (BF16, 0, 17)])
def test_every_workgroup_shape_is_exact(S, rows, rt, waves, wused, ks, dtype, axis, M):
    """All built kernels and (row tiles, waves) shapes - K split across the waves of a
    workgroup, or rows split with activations staged in LDS, `wused` of the waves owning
    rows and K cut into `ks` slices whose partial sums are added afterwards - give
    bit-exact results on exact-integer data."""
    p = S.plan_override(kernel=ROWS if rows else KSPLIT, row_tiles=rt, waves=waves, waves_used=wused, ksplit=ks)
    N, K = 200, 1056
    db = 800 if axis == 1 else 72
    W, mask, X, sw, sx = gen.make_exact_int(12, rt * 10 + waves, M, N, K, gaxis(axis), db, gdt(dtype))
    pw, (v, m, d) = compress_both(S, W, mask, dtype, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, dtype, axis, db, sw, sx)
    assert np.array_equal(run_gemm(S, pw, X, sw, sx, True, p), ref["y_f32"])
    assert np.array_equal(run_gemm(S, pw, X, sw, sx, False, p).view(np.uint16), ref["y_bf16"])


@pytest.mark.parametrize("order", [0, 1, 2])
@pytest.mark.parametrize("axis,M,N,K,db", [(0, 200, 1024, 512, 768), (1, 150, 2048, 1024, 768), (0, 97, 640, 384, 480)])
def test_token_block_orders_exact(S, order, axis, M, N, K, db):
    """The row-split kernel's orders of (row group, token block) workgroups: a grid of
    both, one dimension with a row group's token blocks adjacent, and one dimension with
    them on one XCD (the default where the row groups split evenly over 8): every output
    bit for bit against the oracle on exact-integer data, both layouts."""
    W, mask, X, sw, sx = gen.make_exact_int(17, M + N + order, M, N, K, gaxis(axis), db, gen.FP8)
    pw, (v, m, d) = compress_both(S, W, mask, FP8, axis, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, axis, db, sw, sx)
    p = S.plan_override(kernel=ROWS, block_order=order)
    for w in (pw, S.tile(pw)):
        assert np.array_equal(run_gemm(S, w, X, sw, sx, True, p), ref["y_f32"])
        assert np.array_equal(run_gemm(S, w, X, sw, sx, False, p).view(np.uint16), ref["y_bf16"])
