"""C-ABI checks that need no GPU: every function declared in include/*.h is exported by
the built library, the layout query agrees with the oracle's geometry, and argument
validation rejects bad calls before anything touches a device."""
import ctypes
import glob
import os
import re

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for m in re.finditer(r"^[A-Za-z_][\w \*]*?\b(spense_\w+)\s*\(", text, flags=re.M):
            names.add(m.group(1))
    return sorted(names)


@pytest.fixture(scope="module")
def S():
    import paper_2606_10445_amd as S
    return S


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("spense_layout", "spense_compress", "spense_decompress", "spense_gemm", "spense_dense_gemm",
              "spense_last_error", "spense_gemm_workspace_size"):
        assert n in names


def test_library_exports_every_declared_symbol(S):
    lib = ctypes.CDLL(S.LIB_PATH)
    for n in _declared():
        assert hasattr(lib, n), f"{n} declared in include/ but not exported"
    assert set(_declared()) == set(S.EXPORTS)
    assert S.spense_abi_version() == 13


@pytest.mark.parametrize("N,K,split,db", [(256, 512, 0, 192), (256, 512, 1, 384), (25600, 5120, 0, 19200),
                                          (5120, 25600, 1, 19200), (17, 96, 0, 0), (17, 96, 1, 96), (0, 64, 0, 0)])
@pytest.mark.parametrize("dtype", [1, 2])
def test_layout_matches_oracle_geometry(S, N, K, split, db, dtype):
    L = S.spense_layout(N, K, dtype, split, db)
    o = oracle.layout(N, K, split, db)
    assert (L.sparse_rows, L.sparse_cols, L.values_ld, L.meta_ld) == (o["sparse_rows"], o["sparse_cols"],
                                                                       o["values_ld"], o["meta_ld"])
    assert (L.dense_rows, L.dense_ld) == (o["dense_rows"], o["dense_ld"])
    es = 1 if dtype == 1 else 2
    assert L.values_bytes == L.sparse_rows * L.values_ld * es
    assert L.meta_bytes == L.sparse_rows * L.meta_ld * 4
    assert L.dense_bytes == L.dense_rows * L.dense_ld * es


@pytest.mark.parametrize("args,code", [
    ((256, 500, 1, 0, 0), -2),    # K not a multiple of 32
    ((256, 512, 1, 1, 100), -2),  # input-split point not a multiple of 32
    ((256, 512, 1, 0, 300), -1),  # split point past N
    ((256, 512, 3, 0, 0), -1),    # unknown dtype
    ((256, 512, 1, 2, 0), -1),    # unknown split
    ((-1, 512, 1, 0, 0), -1),
])
def test_layout_rejects(S, args, code):
    with pytest.raises(S.SpenseError) as e:
        S.spense_layout(*args)
    assert e.value.code == code
    assert S.spense_last_error()


def test_gemm_validation_happens_before_any_device_call(S):
    """Bad arguments return an error code without a GPU (the device is queried last)."""
    L = S.spense_layout(64, 128, 1, 0, 32)
    good = S.spense_packed_t(1, 0, 64, 128, 32, 4096, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld)
    # NULL packed
    assert S._lib.spense_gemm(4096, 4, 128, None, None, None, 4096, 64, 0, None, 0, None) == S.SPENSE_ERR_ARG
    # NULL Y
    assert S.spense_gemm(4096, 4, 128, good, None, None, None, 64, 0, None, 0, None) == S.SPENSE_ERR_ARG
    # misaligned X
    assert S.spense_gemm(4097, 4, 128, good, None, None, 4096, 64, 0, None, 0, None) == S.SPENSE_ERR_ALIGN
    # ldx < K
    assert S.spense_gemm(4096, 4, 64, good, None, None, 4096, 64, 0, None, 0, None) == S.SPENSE_ERR_ARG
    # ldy < N
    assert S.spense_gemm(4096, 4, 128, good, None, None, 4096, 32, 0, None, 0, None) == S.SPENSE_ERR_ARG
    # unknown flags
    assert S.spense_gemm(4096, 4, 128, good, None, None, 4096, 64, 8, None, 0, None) == S.SPENSE_ERR_ARG
    # values pointer NULL with a non-empty 2:4 region
    bad = S.spense_packed_t(1, 0, 64, 128, 32, None, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld)
    assert S.spense_gemm(4096, 4, 128, bad, None, None, 4096, 64, 0, None, 0, None) == S.SPENSE_ERR_ARG
    # misaligned dense
    bad = S.spense_packed_t(1, 0, 64, 128, 32, 4096, L.values_ld, 8192, L.meta_ld, 16392, L.dense_ld)
    assert S.spense_gemm(4096, 4, 128, bad, None, None, 4096, 64, 0, None, 0, None) == S.SPENSE_ERR_ALIGN
    # M == 0 and N == 0 are no-ops that succeed without touching anything
    assert S.spense_gemm(None, 0, 128, good, None, None, None, 64, 0, None, 0, None) == S.SPENSE_OK
    # the current kernels split K inside a workgroup and need no workspace
    Ld = S.spense_layout(1024, 8192, 1, 1, 6144)
    big = S.spense_packed_t(1, 1, 1024, 8192, 6144, 4096, Ld.values_ld, 8192, Ld.meta_ld, 16384, Ld.dense_ld)
    assert S.spense_gemm_workspace_size(1, big) == 0
    assert S.spense_gemm_workspace_size(2048, big) == 0


def test_compress_validation(S):
    L = S.spense_layout(64, 128, 1, 0, 32)
    pk = S.spense_packed_t(1, 0, 64, 128, 32, 4096, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld)
    rc, bad = S.spense_compress(None, 128, None, 0, pk, 4096, 256, None)
    assert rc == S.SPENSE_ERR_ARG and bad == 0
    rc, _ = S.spense_compress(4096, 128, 4097, 128, pk, 4096, 256, None)
    assert rc == S.SPENSE_ERR_ALIGN
    rc, _ = S.spense_compress(4096, 128, None, 0, pk, None, 0, None)
    assert rc == S.SPENSE_ERR_WS


def test_workspace_size_is_a_pure_function_of_geometry(S):
    L = S.spense_layout(5120, 25600, 1, 1, 19200)
    pk = S.spense_packed_t(1, 1, 5120, 25600, 19200, 4096, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld)
    a = [S.spense_gemm_workspace_size(m, pk) for m in (1, 16, 64, 65)]
    b = [S.spense_gemm_workspace_size(m, pk) for m in (1, 16, 64, 65)]
    assert a == b
    # the dense baseline with all rows dense plans exactly like a Spense weight with no 2:4 part
    L0 = S.spense_layout(4096, 5120, 1, 0, 0)
    pk0 = S.spense_packed_t(1, 0, 4096, 5120, 0, None, L0.values_ld, None, L0.meta_ld, 16384, L0.dense_ld)
    for m in (1, 8, 64):
        assert S.spense_gemm_workspace_size(m, pk0) == S.spense_dense_gemm_workspace_size(m, 4096, 5120, 1)


@pytest.mark.parametrize("N,K,split,db", [(25600, 5120, 0, 19200), (5120, 25600, 1, 19200), (17, 96, 0, 0),
                                          (17, 96, 1, 96), (200, 1056, 1, 800), (200, 1056, 0, 72), (0, 64, 0, 0)])
def test_tiled_layout_geometry(S, N, K, split, db):
    """Tiles of 16 rows and chunks of 512 logical columns per region, 4096 / 1024 / 8192
    bytes per (tile, chunk) for values / metadata / dense (the header's definition)."""
    T = S.spense_tiled_layout(N, K, 1, split, db)
    sr, sc = (db, K) if split == 0 else (N, db)
    dr, dc = (N - db, K) if split == 0 else (N, K - db)
    cdiv = lambda a, b: -(-a // b)
    st, sch = (cdiv(sr, 16), cdiv(sc, 512)) if sr and sc else (0, 0)
    dt, dch = (cdiv(dr, 16), cdiv(dc, 512)) if dr and dc else (0, 0)
    assert (T.sparse_tiles, T.sparse_chunks, T.dense_tiles, T.dense_chunks) == (st, sch, dt, dch)
    assert (T.values_bytes, T.meta_bytes, T.dense_bytes) == (st * sch * 4096, st * sch * 1024, dt * dch * 8192)


def test_tiled_layout_is_fp8_only(S):
    with pytest.raises(S.SpenseError) as e:
        S.spense_tiled_layout(64, 128, 2, 0, 32)
    assert e.value.code == S.SPENSE_ERR_ARG


def test_tiled_descriptor_validation(S):
    """Tiled descriptors are checked before any device call; their leading dimensions
    are ignored."""
    good = S.spense_packed_t(1, 0, 64, 128, 32, 4096, 0, 8192, 0, 16384, 0, S.SPENSE_LAYOUT_TILED)
    assert S.spense_gemm(None, 0, 128, good, None, None, None, 64, 0, None, 0, None) == S.SPENSE_OK
    bad = S.spense_packed_t(1, 0, 64, 128, 32, None, 0, 8192, 0, 16384, 0, S.SPENSE_LAYOUT_TILED)
    assert S.spense_gemm(4096, 4, 128, bad, None, None, 4096, 64, 0, None, 0, None) == S.SPENSE_ERR_ARG
    bad = S.spense_packed_t(1, 0, 64, 128, 32, 4104, 0, 8192, 0, 16384, 0, S.SPENSE_LAYOUT_TILED)
    assert S.spense_gemm(4096, 4, 128, bad, None, None, 4096, 64, 0, None, 0, None) == S.SPENSE_ERR_ALIGN
    bad = S.spense_packed_t(2, 0, 64, 128, 32, 4096, 0, 8192, 0, 16384, 0, S.SPENSE_LAYOUT_TILED)
    assert S.spense_gemm(4096, 4, 128, bad, None, None, 4096, 64, 0, None, 0, None) == S.SPENSE_ERR_ARG
    bad = S.spense_packed_t(1, 0, 64, 128, 32, 4096, 0, 8192, 0, 16384, 0, 7)
    assert S.spense_gemm(4096, 4, 128, bad, None, None, 4096, 64, 0, None, 0, None) == S.SPENSE_ERR_ARG
    # spense_tile takes a row-major source and a tiled destination of the same weight
    L = S.spense_layout(64, 128, 1, 0, 32)
    src = S.spense_packed_t(1, 0, 64, 128, 32, 4096, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld)
    dst = S.spense_packed_t(1, 0, 64, 128, 32, 1 << 20, 0, 2 << 20, 0, 3 << 20, 0, S.SPENSE_LAYOUT_TILED)
    assert S.spense_tile(dst, src, None) == S.SPENSE_ERR_ARG
    other = S.spense_packed_t(1, 0, 64, 128, 48, 1 << 20, 0, 2 << 20, 0, 3 << 20, 0, S.SPENSE_LAYOUT_TILED)
    assert S.spense_tile(src, other, None) == S.SPENSE_ERR_ARG
    overlap = S.spense_packed_t(1, 0, 64, 128, 32, 4096 + 1024, 0, 2 << 20, 0, 3 << 20, 0, S.SPENSE_LAYOUT_TILED)
    assert S.spense_tile(src, overlap, None) == S.SPENSE_ERR_ARG
    # compress and decompress work on the row-major layout only
    assert S.spense_decompress(dst, 4096, 128, None) == S.SPENSE_ERR_ARG


def test_k_slices_need_a_workspace(S):
    """Weights with few rows (down: 5120 x 25600) are sliced along K at decode M; the
    partial sums need slices x M x N floats of workspace, checked before any device call."""
    L = S.spense_layout(5120, 25600, 1, 1, 19200)
    pk = S.spense_packed_t(1, 1, 5120, 25600, 19200, 4096, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld)
    need = S.spense_gemm_workspace_size(64, pk)
    assert need > 0 and need % (64 * 5120 * 4) == 0 and need // (64 * 5120 * 4) <= 8
    assert S.spense_gemm(4096, 64, 25600, pk, None, None, 4096, 5120, 0, None, 0, None) == S.SPENSE_ERR_WS
    assert S.spense_gemm(4096, 64, 25600, pk, None, None, 4096, 5120, 0, 4096, need - 4, None) == S.SPENSE_ERR_WS
    # a weight with many rows (gate/up) is not sliced
    Lg = S.spense_layout(25600, 5120, 1, 0, 19200)
    pg = S.spense_packed_t(1, 0, 25600, 5120, 19200, 4096, Lg.values_ld, 8192, Lg.meta_ld, 16384, Lg.dense_ld)
    assert all(S.spense_gemm_workspace_size(m, pg) == 0 for m in (1, 8, 32, 64))


def test_quantize_calls_validate_arguments_on_the_host(S):
    """Error paths of the quantisation calls return before touching the device."""
    q = S.spense_quantize_fp8
    assert q(None, S.SPENSE_BF16, 0, 16, 16, None, 16, None, None) == S.SPENSE_OK  # M = 0: nothing to do
    assert q(None, S.SPENSE_FP8_E4M3FN, 4, 16, 16, None, 16, None, None) == S.SPENSE_ERR_ARG  # fp8 input
    assert q(None, S.SPENSE_F32, -1, 16, 16, None, 16, None, None) == S.SPENSE_ERR_ARG
    assert q(None, S.SPENSE_F32, 4, 16, 16, None, 16, None, None) == S.SPENSE_ERR_ARG  # NULL pointers
    assert "NULL" in S.spense_last_error()
    assert q(8, S.SPENSE_F32, 4, 16, 15, 8, 16, 8, None) == S.SPENSE_ERR_ARG  # ld < K
    assert q(8, S.SPENSE_F32, 1 << 31, 16, 16, 8, 16, 8, None) == S.SPENSE_ERR_ARG  # M too large
    g = S.spense_glu_quantize_fp8
    assert g(None, 16, None, 16, S.SPENSE_BF16, 0, 16, None, 16, None, None) == S.SPENSE_OK
    assert g(8, 16, None, 16, S.SPENSE_BF16, 2, 16, 8, 16, 8, None) == S.SPENSE_ERR_ARG  # u NULL
    assert g(8, 16, 8, 8, S.SPENSE_F32, 2, 16, 8, 16, 8, None) == S.SPENSE_ERR_ARG  # ldu < I


def test_index_calls_validate_arguments_on_the_host(S):
    """Error paths of the dense-index selection calls return before touching the device."""
    sc = S.spense_index_scores
    assert sc(8, 8, 16, 8, 4, S.SPENSE_FP8_E4M3FN, 4, 16, 8, 8, 1e-8, 8, 8, None) == S.SPENSE_ERR_ARG  # fp8 weights
    assert sc(8, 8, 16, 8, 4, S.SPENSE_BF16, 0, 16, 8, 8, 1e-8, 8, 8, None) == S.SPENSE_ERR_ARG  # I = 0
    assert sc(8, None, 16, 8, 4, S.SPENSE_BF16, 4, 16, 8, 8, 1e-8, 8, 8, None) == S.SPENSE_ERR_ARG  # NULL
    assert sc(8, 8, 15, 8, 4, S.SPENSE_BF16, 4, 16, 8, 8, 1e-8, 8, 8, None) == S.SPENSE_ERR_ARG  # ld_gu < D
    assert sc(8, 8, 16, 8, 3, S.SPENSE_F32, 4, 16, 8, 8, 1e-8, 8, 8, None) == S.SPENSE_ERR_ARG  # ld_down < I
    dp = S.spense_dense_permutation
    assert dp(8, 4, 5, 8, 8, None) == S.SPENSE_ERR_ARG  # n_dense > I
    assert dp(8, 4, -1, 8, 8, None) == S.SPENSE_ERR_ARG
    assert dp(8, 0, 0, 8, 8, None) == S.SPENSE_ERR_ARG
    assert dp(8, 4, 2, None, 8, None) == S.SPENSE_ERR_ARG
    gr = S.spense_gather_rows
    assert gr(None, 16, None, 16, 0, 16, None, None) == S.SPENSE_OK  # nothing to do
    assert gr(8, 8, 8, 16, 4, 16, 8, None) == S.SPENSE_ERR_ARG  # ld_src < row bytes
    assert gr(8, 16, 8, 16, 4, 16, None, None) == S.SPENSE_ERR_ARG  # NULL perm
    gc = S.spense_gather_cols
    assert gc(8, 16, 8, 16, 4, 16, 3, 8, None) == S.SPENSE_ERR_ARG  # element size
    assert gc(8, 15, 8, 16, 4, 16, 2, 8, None) == S.SPENSE_ERR_ARG  # ld_src < cols
    assert gc(9, 16, 8, 16, 4, 16, 2, 8, None) == S.SPENSE_ERR_ALIGN  # misaligned source
    assert gc(None, 16, None, 16, 4, 0, 2, None, None) == S.SPENSE_OK


def test_obs_calls_validate_arguments_on_the_host(S):
    """Error paths of the SparseGPT calls return before touching the device."""
    f = S.spense_obs_factor
    ws = S.spense_obs_factor_workspace_size(64)
    assert ws == 256  # a single 64-block: no recursion workspace
    big = S.spense_obs_factor_workspace_size(25600)  # the recursion's L21 blocks, about K^2 / 3 floats
    assert 25600 ** 2 / 4 * 4 <= big <= 25600 ** 2 / 2 * 4
    assert f(None, 64, 64, 0.01, 1 << 30, 64, 16, 1 << 12, ws, None) == S.SPENSE_ERR_ARG  # NULL H
    assert f(1 << 20, 64, 0, 0.01, 1 << 30, 64, 16, 1 << 12, ws, None) == S.SPENSE_ERR_ARG  # K = 0
    assert f(1 << 20, 63, 64, 0.01, 1 << 30, 64, 16, 1 << 12, ws, None) == S.SPENSE_ERR_ARG  # ldh < K
    assert f(1 << 20, 64, 64, -1.0, 1 << 30, 64, 16, 1 << 12, ws, None) == S.SPENSE_ERR_ARG  # negative damping
    assert f(1 << 20, 64, 64, float("nan"), 1 << 30, 64, 16, 1 << 12, ws, None) == S.SPENSE_ERR_ARG
    assert f(1 << 20, 64, 64, 0.01, (1 << 20) + 4096, 64, 16, 1 << 12, ws, None) == S.SPENSE_ERR_ARG  # U overlaps H
    assert "overlaps" in S.spense_last_error()
    assert f(1 << 20, 64, 64, 0.01, 1 << 30, 64, 16, 1 << 12, ws - 1, None) == S.SPENSE_ERR_WS
    assert f(1 << 20, 64, 64, 0.01, 1 << 30, 64, 16, (1 << 12) + 8, ws, None) == S.SPENSE_ERR_WS  # unaligned
    p = S.spense_obs_prune_24
    pws = S.spense_obs_prune_workspace_size(8)
    assert p(None, 64, 0, 64, None, 64, None, 0, None, 64, None, 0, None) == S.SPENSE_OK  # N = 0
    assert p(1 << 20, 64, 8, 64, 1 << 22, 64, None, 6, 1 << 24, 64, 1 << 12, pws, None) == S.SPENSE_ERR_ARG  # % 4
    assert p(1 << 20, 64, 8, 64, 1 << 22, 64, None, 68, 1 << 24, 64, 1 << 12, pws, None) == S.SPENSE_ERR_ARG  # > K
    assert p(1 << 20, 64, 8, 64, None, 64, None, 32, 1 << 24, 64, 1 << 12, pws, None) == S.SPENSE_ERR_ARG  # NULL U
    assert p(1 << 20, 60, 8, 64, 1 << 22, 64, None, 32, 1 << 24, 64, 1 << 12, pws, None) == S.SPENSE_ERR_ARG  # ldw
    assert p(1 << 20, 64, 8, 64, 1 << 22, 64, None, 32, 1 << 24, 64, 1 << 12, pws - 4, None) == S.SPENSE_ERR_WS


def test_large_m_xcd_order_is_a_permutation_of_the_grid():
    """The large-M kernels' XCD-aware workgroup order (the same formulas as the kernels and
    the planner: GT the divisor of T nearest 4 whose token groups divide the 8 XCDs, the
    order over the whole sets of RC row classes, the remaining row blocks in place after
    them) visits every (row block, token block) pair exactly once."""
    for T in range(1, 33):
        cands = [d for d in range(1, T + 1) if T % d == 0 and 8 % (T // d) == 0]
        if not cands:
            continue  # the planner keeps the plain order
        GT = min(cands, key=lambda d: (abs(d - 4), d))
        TGc = T // GT
        RC = 8 // TGc
        for rbtot in (1, 2, 3, 8, 13, 40, 64, 100, 150, 200, 216):
            rbx = rbtot // RC * RC
            G, xg1 = rbtot * T, rbx * T
            seen = set()
            for g in range(G):
                if g < xg1:
                    x, l = g & 7, g >> 3
                    g = ((l // GT) * RC + x // TGc) * T + (x % TGc) * GT + l % GT
                seen.add(g)
            assert seen == set(range(G)), (T, rbtot)


def test_grouped_gemm_validates_arguments_on_the_host(S):
    """Error paths of spense_gemm_grouped return before touching the device."""
    import ctypes
    g = S.spense_gemm_grouped
    L = S.spense_layout(64, 256, S.SPENSE_FP8_E4M3FN, S.SPENSE_SPLIT_OUTPUT, 48)
    T = S.spense_tiled_layout(64, 256, S.SPENSE_FP8_E4M3FN, S.SPENSE_SPLIT_OUTPUT, 48)
    d = S.spense_packed_t(1, 0, 64, 256, 48, 1 << 20, L.values_ld, 2 << 20, L.meta_ld, 3 << 20, L.dense_ld,
                          S.SPENSE_LAYOUT_TILED)
    d2 = S.spense_packed_t(1, 0, 64, 512, 48, 1 << 20, L.values_ld, 2 << 20, L.meta_ld, 3 << 20, L.dense_ld,
                           S.SPENSE_LAYOUT_TILED)  # another K
    rm = S.spense_packed_t(1, 0, 64, 256, 48, 1 << 20, L.values_ld, 2 << 20, L.meta_ld, 3 << 20, L.dense_ld,
                           S.SPENSE_LAYOUT_ROWMAJOR)
    PP = ctypes.POINTER(S.spense_packed_t)
    arr = lambda *ds: (PP * len(ds))(*[ctypes.pointer(x) for x in ds])
    ys = (ctypes.c_void_p * 4)(1 << 24, 1 << 25, 1 << 26, 1 << 27)
    lds = (ctypes.c_int64 * 4)(64, 64, 64, 64)
    assert T.sparse_tiles == 3
    assert g(1 << 28, 8, 256, 0, arr(d), None, None, ys, lds, 0, None) == S.SPENSE_ERR_ARG  # count 0
    assert g(1 << 28, 8, 256, 5, arr(d, d, d, d, d), None, None, ys, lds, 0, None) == S.SPENSE_ERR_ARG  # > 4
    assert g(1 << 28, 8, 256, 2, arr(d, d2), None, None, ys, lds, 0, None) == S.SPENSE_ERR_ARG  # mixed K
    assert g(1 << 28, 8, 256, 2, arr(d, rm), None, None, ys, lds, 0, None) == S.SPENSE_ERR_ARG  # row-major
    assert g(1 << 28, 8, 256, 1, arr(d), None, None, None, lds, 0, None) == S.SPENSE_ERR_ARG  # NULL Y array
    short = (ctypes.c_int64 * 1)(32)
    assert g(1 << 28, 8, 256, 1, arr(d), None, None, ys, short, 0, None) == S.SPENSE_ERR_ARG  # ldy < N
    assert g(None, 8, 256, 1, arr(d), None, None, ys, lds, 0, None) == S.SPENSE_ERR_ARG  # NULL X
    assert g((1 << 28) + 8, 8, 256, 1, arr(d), None, None, ys, lds, 0, None) == S.SPENSE_ERR_ALIGN  # unaligned X
    assert g(1 << 28, 0, 256, 1, arr(d), None, None, ys, lds, 0, None) == S.SPENSE_OK  # M = 0


def test_gemm_glu_validates_arguments_on_the_host(S):
    """Error paths of spense_gemm_glu return before touching the device."""
    import ctypes
    f = S.spense_gemm_glu
    L = S.spense_layout(64, 256, S.SPENSE_FP8_E4M3FN, S.SPENSE_SPLIT_OUTPUT, 48)

    def desc(N=64, K=256, db=48, layout=S.SPENSE_LAYOUT_TILED, dtype=1):
        return S.spense_packed_t(dtype, 0, N, K, db, 1 << 20, L.values_ld, 2 << 20, L.meta_ld, 3 << 20, L.dense_ld,
                                 layout)
    g = desc()
    ref = ctypes.byref
    X, H = 1 << 28, 1 << 24
    assert f(X, 8, 256, ref(g), None, None, None, None, H, 64, None) == S.SPENSE_ERR_ARG  # up NULL
    assert f(X, 8, 256, ref(g), ref(desc(N=80)), None, None, None, H, 80, None) == S.SPENSE_ERR_ARG  # N differs
    assert f(X, 8, 256, ref(g), ref(desc(db=32)), None, None, None, H, 64, None) == S.SPENSE_ERR_ARG  # dense_begin
    assert f(X, 8, 256, ref(g), ref(desc(layout=S.SPENSE_LAYOUT_ROWMAJOR)), None, None, None, H, 64,
             None) == S.SPENSE_ERR_ARG  # row-major
    assert f(X, 8, 256, ref(g), ref(g), None, None, None, None, 64, None) == S.SPENSE_ERR_ARG  # H NULL
    assert f(X, 8, 256, ref(g), ref(g), None, None, None, H, 32, None) == S.SPENSE_ERR_ARG  # ldh < N
    assert f(X, 8, 256, ref(g), ref(g), None, None, None, H + 2, 64, None) == S.SPENSE_ERR_ALIGN  # H misaligned
    assert f(None, 8, 256, ref(g), ref(g), None, None, None, H, 64, None) == S.SPENSE_ERR_ARG  # X NULL
    assert f(X + 8, 8, 256, ref(g), ref(g), None, None, None, H, 64, None) == S.SPENSE_ERR_ALIGN  # X misaligned
    assert f(X, 8, 128, ref(g), ref(g), None, None, None, H, 64, None) == S.SPENSE_ERR_ARG  # ldx < K
    assert f(X, 0, 256, ref(g), ref(g), None, None, None, H, 64, None) == S.SPENSE_OK  # M = 0


def test_gemm_glu_fp8_validates_arguments_on_the_host(S):
    """Error paths of spense_gemm_glu_fp8 and its workspace size, before the device."""
    import ctypes
    f = S.spense_gemm_glu_fp8
    L = S.spense_layout(64, 256, S.SPENSE_FP8_E4M3FN, S.SPENSE_SPLIT_OUTPUT, 48)
    g = S.spense_packed_t(1, 0, 64, 256, 48, 1 << 20, L.values_ld, 2 << 20, L.meta_ld, 3 << 20, L.dense_ld,
                          S.SPENSE_LAYOUT_TILED)
    ref = ctypes.byref
    X, Q, SC, WS = 1 << 28, 1 << 24, 1 << 23, 1 << 30
    need = S.spense_gemm_glu_fp8_workspace_size(8, 64)
    # H (8 rows of 64 fp32), then per token one maximum per workgroup along N: at most
    # one per 16 rows of each of the two regions (48 + 16 rows here: 4, bounded by 5)
    assert need == 8 * 64 * 4 + 8 * 5 * 4
    assert S.spense_gemm_glu_fp8_workspace_size(0, 64) == 0
    assert S.spense_gemm_glu_fp8_workspace_size(8, 0) == 0
    assert f(X, 8, 256, ref(g), ref(g), None, None, None, Q, 64, SC, WS, need - 1, None) == S.SPENSE_ERR_WS
    assert f(X, 8, 256, ref(g), ref(g), None, None, None, Q, 64, SC, None, need, None) == S.SPENSE_ERR_WS
    assert f(X, 8, 256, ref(g), ref(g), None, None, None, Q, 64, SC, WS + 16, need, None) == S.SPENSE_ERR_ALIGN
    assert f(X, 8, 256, ref(g), ref(g), None, None, None, None, 64, SC, WS, need, None) == S.SPENSE_ERR_ARG
    assert f(X, 8, 256, ref(g), ref(g), None, None, None, Q, 64, None, WS, need, None) == S.SPENSE_ERR_ARG
    assert f(X, 8, 256, ref(g), ref(g), None, None, None, Q, 63, SC, WS, need, None) == S.SPENSE_ERR_ARG
    assert f(X, 8, 256, ref(g), None, None, None, None, Q, 64, SC, WS, need, None) == S.SPENSE_ERR_ARG
    assert f(X, 0, 256, ref(g), ref(g), None, None, None, Q, 64, SC, WS, need, None) == S.SPENSE_OK


def test_k_slice_rule_on_the_layer_shapes(S):
    """Which Qwen3-like layer weights (tiled layout) the planner slices along K (a
    workspace is needed exactly then): k / v (64 tiles) at every M up to 128, o (320 tiles,
    16 chunks) from 17 to 64 tokens, down (50 chunks, with a 2:4 part) from one token to
    192, q (512 tiles) and gate (1600 tiles) never; none from four token blocks on."""
    def ws(N, K, split, M):
        db = N * 3 // 4 if split == 0 else K * 3 // 4
        L = S.spense_layout(N, K, 1, split, db)
        p = S.spense_packed_t(1, split, N, K, db, 4096, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld,
                              S.SPENSE_LAYOUT_TILED)
        return S.spense_gemm_workspace_size(M, p)
    for M in (1, 16, 64):
        assert ws(1024, 5120, 0, M) > 0  # k / v
        assert ws(5120, 25600, 1, M) > 0  # down
        assert ws(8192, 5120, 0, M) == 0  # q
        assert ws(25600, 5120, 0, M) == 0  # gate / up
    assert ws(5120, 8192, 1, 1) == 0 and ws(5120, 8192, 1, 16) == 0  # o: one token block of 1-16
    assert ws(5120, 8192, 1, 17) > 0 and ws(5120, 8192, 1, 64) > 0  # o from 17 tokens
    for M in (65, 100, 128):  # two token blocks: k / v sliced, down as 6 slices of 128 tokens, o, q and gate not
        assert ws(1024, 5120, 0, M) > 0 and ws(5120, 25600, 1, M) == 6 * M * 5120 * 4
        assert ws(5120, 8192, 1, M) == 0 and ws(8192, 5120, 0, M) == 0 and ws(25600, 5120, 0, M) == 0
    assert ws(5120, 25600, 1, 192) > 0 and ws(1024, 5120, 0, 192) == 0  # three: only the long K
    assert ws(1024, 5120, 0, 200) == 0  # four or more token blocks
    assert ws(5120, 25600, 1, 200) == 3 * 200 * 5120 * 4  # down from 193 tokens: 3 slices of 128 tokens
    assert ws(5120, 25600, 1, 300) == 2 * 300 * 5120 * 4  # 257-320: two halves in 2 slices
    assert ws(5120, 25600, 1, 350) == 0 and ws(5120, 25600, 1, 500) == 0


def test_two_half_rule_on_the_layer_shapes(S, capfd):
    """Where the planner runs two 64-token halves per row-split workgroup (tiled fp8, seen
    through the dispatch log): one 128-token block on weights of at least 768 row tiles
    (gate / up, 1600; 12288 rows), not on q (512) or at 64 tokens; two blocks where the
    row-split kernel would take three or four (q from 193 tokens, 640 tiles from 129), not
    where the large-M kernel runs (gate / up) or above 256 tokens; the row-major layout
    never."""
    def kernel(N, K, split, M, layout=S.SPENSE_LAYOUT_TILED):
        db = N * 3 // 4 if split == 0 else K * 3 // 4
        L = S.spense_layout(N, K, 1, split, db)
        p = S.spense_packed_t(1, split, N, K, db, 4096, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld, layout)
        S.spense_gemm_workspace_size(M, p)
        err = capfd.readouterr().err.strip().splitlines()
        assert err, (N, K, split, M)  # planned once in this test; a cached plan would log nothing
        return err[-1].split(" -> ")[1].split(" act_tiles")[0]
    two = "row-split, two 64-token halves"
    prev = S.spense_set_log(1)
    try:
        # token counts other tests do not plan on these geometries (plans are cached per thread)
        capfd.readouterr()
        for M in (66, 127):
            assert kernel(25600, 5120, 0, M) == two and kernel(25600, 5120, 1, M) == two
            assert kernel(12288, 5120, 0, M) == two
            assert kernel(8192, 5120, 0, M) == "row-split" and kernel(10240, 5120, 0, M) == "row-split"
        assert kernel(25600, 5120, 0, 63) == "row-split"
        assert kernel(8192, 5120, 0, 191) == "row-split" and kernel(8192, 5120, 0, 193) == two
        assert kernel(10240, 5120, 0, 131) == two and kernel(16384, 8192, 1, 131) == two
        assert kernel(25600, 5120, 0, 131).startswith("large-M") and kernel(25600, 5120, 0, 300).startswith("large-M")
        # 257-768 tokens on 256-767 row tiles: q up to 384, o and down from 385 (and down
        # at 257-320, in 2 slices), not the 128 x 256 kernel's q above 384
        assert kernel(8192, 5120, 0, 257) == two and kernel(8192, 5120, 0, 383) == two
        assert kernel(8192, 5120, 0, 449).startswith("large-M")
        assert kernel(5120, 8192, 1, 450) == two and kernel(5120, 25600, 1, 639) == two
        assert kernel(5120, 25600, 1, 301) == two and kernel(5120, 25600, 1, 350) == "row-split"
        assert kernel(5120, 8192, 1, 301) == "row-split" and kernel(5120, 25600, 1, 700) == two
        assert kernel(5120, 25600, 1, 769) != two and kernel(5120, 8192, 1, 900) != two
        assert kernel(1024, 5120, 0, 450) != two  # k / v: 64 row tiles
        assert kernel(25600, 5120, 0, 99, layout=0) != two
        # short weights with a long K: with K slices (down 50 chunks, Seed-OSS o 20)
        assert kernel(5120, 25600, 1, 67) == two and kernel(5120, 25600, 1, 250) == two
        assert kernel(5120, 25600, 1, 170) == "row-split"
        assert kernel(5120, 10240, 1, 67) == two and kernel(5120, 10240, 1, 120) == "row-split"
        assert kernel(5120, 8192, 1, 67) == "row-split"  # o, 16 chunks
    finally:
        S.spense_set_log(prev)


def test_192_token_blocks_rule(S, capfd):
    """The 256 x 256 kernel takes 192-token blocks where they need no more blocks than
    256-token ones (257-384, 513-576 tokens), else 256, seen through the dispatch log."""
    L = S.spense_layout(25600, 5120, 1, 0, 19200)
    p = S.spense_packed_t(1, 0, 25600, 5120, 19200, 4096, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld,
                          S.SPENSE_LAYOUT_TILED)
    prev = S.spense_set_log(1)
    try:
        got = {}
        for M in (259, 383, 389, 515, 575, 577, 2047):  # token counts no other test plans on this weight
            capfd.readouterr()
            S.spense_gemm_workspace_size(M, p)
            line = capfd.readouterr().err.strip().splitlines()[-1]
            assert "large-M 256x256" in line, line
            got[M] = int(line.split("block_tokens=")[1].split()[0])
        assert got == {259: 192, 383: 192, 389: 256, 515: 192, 575: 192, 577: 256, 2047: 256}, got
    finally:
        S.spense_set_log(prev)


def _down_desc(S, layout=0, dtype=1):
    L = S.spense_layout(5120, 25600, dtype, 1, 19200)
    return S.spense_packed_t(dtype, 1, 5120, 25600, 19200, 4096, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld,
                             layout)


def test_plan_override_is_checked_on_the_host(S):
    """spense_gemm_planned: a forced plan changes what the planner would choose (seen here
    through the workspace it needs), and an override no kernel is built for, or this
    weight cannot run, is rejected with SPENSE_ERR_ARG before any device call."""
    po = S.plan_override
    rm, tl, bf = _down_desc(S), _down_desc(S, S.SPENSE_LAYOUT_TILED), _down_desc(S, dtype=2)
    assert S.spense_gemm_planned_workspace_size(64, rm, None) == S.spense_gemm_workspace_size(64, rm)
    assert S.spense_gemm_planned_workspace_size(64, tl, po(kernel=2, ksplit=3)) == 3 * 64 * 5120 * 4
    assert S.spense_gemm_planned_workspace_size(64, tl, po(kernel=2, ksplit=1)) == 0
    assert S.spense_gemm_planned_workspace_size(64, rm, po(kernel=1)) == 0  # no K slices in the K-split kernel
    assert S.spense_gemm_planned_workspace_size(64, rm, po(kernel=3)) == 0
    assert S.spense_gemm_planned_workspace_size(100, tl, po(kernel=5)) == 0  # 128 tokens a block, no slices
    assert S.spense_gemm_planned_workspace_size(100, tl, po(kernel=5, ksplit=3)) == 3 * 100 * 5120 * 4
    bad = [(tl, po(kernel=1)),                      # the K-split kernel reads the row-major layout only
           (bf, po(kernel=3)),                      # large-M is fp8 only
           (rm, po(kernel=2, row_tiles=4, waves=4)),  # no such row-split shape
           (rm, po(kernel=1, row_tiles=4, waves=8)),  # no such K-split shape
           (rm, po(kernel=3, waves=16)),
           (rm, po(waves=8)),                       # a shape needs the kernel it is for
           (rm, po(kernel=5)),                      # the two-half row-split kernel: tiled fp8 only,
           (tl, po(kernel=5, waves=8)), (tl, po(kernel=5, act_tiles=2)),  # one shape
           (rm, po(kernel=6)), (rm, po(ksplit=9)), (rm, po(act_tiles=3)), (rm, po(waves_used=9)),
           (rm, po(block_order=3)), (rm, po(xcd_order=2)), (rm, po(u8=2)), (rm, po(half_row_blocks=-2)), (rm, po(resident_x=3))]
    for desc, p in bad:
        assert S.spense_gemm_planned_workspace_size(64, desc, p) == 0
        rc = S.spense_gemm_planned(1 << 28, 64, 25600, desc, None, None, 1 << 30, 5120, 0, 1 << 31, 1 << 26, p, None)
        assert rc == S.SPENSE_ERR_ARG, (p.kernel, rc)
        assert "plan" in S.spense_last_error()


def test_environment_does_not_change_the_plan(S, monkeypatch):
    """spense_gemm's plan depends on the dtype, M and the weight geometry only: variables
    that once steered the planner in testing builds change nothing."""
    tl = _down_desc(S, S.SPENSE_LAYOUT_TILED)
    before = [S.spense_gemm_workspace_size(m, tl) for m in (1, 16, 64)]
    for k, v in (("SPENSE_KSPLIT", "2"), ("SPENSE_ROWS", "0"), ("SPENSE_BIG", "1"), ("SPENSE_CT", "1"),
                 ("SPENSE_WAVES", "4"), ("SPENSE_RT", "2"), ("SPENSE_WUSED", "3")):
        monkeypatch.setenv(k, v)
    assert [S.spense_gemm_workspace_size(m, tl) for m in (1, 16, 64)] == before


def test_binding_checks_tensors_before_the_library(S):
    """The torch wrappers reject outputs of the wrong shape, dtype or layout and
    activations of the wrong dtype before any pointer reaches the library (a short
    output would otherwise be written past its end)."""
    import torch
    N, K, db = 64, 256, 48
    pw = S.PackedWeight.empty(N, K, S.SPENSE_FP8_E4M3FN, S.SPENSE_SPLIT_OUTPUT, db, device="cpu")
    X = torch.zeros((8, K), dtype=torch.uint8)
    cases = [dict(out=torch.empty((7, N), dtype=torch.bfloat16)),                    # too few rows
             dict(out=torch.empty((8, N), dtype=torch.float32)),                     # fp32 for a bf16 output
             dict(out=torch.empty((8, N), dtype=torch.bfloat16), out_f32=True),      # bf16 for an fp32 output
             dict(out=torch.empty((N, 8), dtype=torch.bfloat16).t()),                # columns not contiguous
             dict(out=torch.empty((8, N, 1), dtype=torch.bfloat16)[:, :, 0])]        # 2-D view, fine shape: ok below
    for kw in cases[:4]:
        with pytest.raises(ValueError):
            S.gemm(X, pw, **kw)
    with pytest.raises(ValueError):
        S.gemm(X.to(torch.bfloat16), pw)  # bf16 activations for an fp8 weight
    with pytest.raises(ValueError):
        S.gemm(torch.zeros((8, K + 32), dtype=torch.uint8), pw)  # K differs
    with pytest.raises(ValueError):
        S.gemm_grouped(X, [pw, pw], outs=[torch.empty((8, N), dtype=torch.bfloat16),
                                          torch.empty((4, N), dtype=torch.bfloat16)])
    with pytest.raises(ValueError):
        S.dense_gemm(X, torch.zeros((N, K), dtype=torch.uint8), out=torch.empty((8, N - 1), dtype=torch.bfloat16))
    with pytest.raises(ValueError):
        S.dense_gemm(X.to(torch.bfloat16), torch.zeros((N, K), dtype=torch.uint8))


def test_dispatch_log_names_the_plan_and_changes_nothing(S, capfd):
    """spense_set_log(1): a new single-weight plan writes one stderr line naming its kernel
    and shape; a reused plan writes none; the plan (here its workspace) is the same with the
    log on and off."""
    L = S.spense_layout(5120, 25600, 1, 1, 19200)
    pk = S.spense_packed_t(1, 1, 5120, 25600, 19200, 4096, L.values_ld, 8192, L.meta_ld, 16384, L.dense_ld)
    M = 61  # a geometry no other test of this process plans
    prev = S.spense_set_log(0)
    try:
        capfd.readouterr()
        quiet = S.spense_gemm_workspace_size(M, pk)
        assert capfd.readouterr().err == ""
        assert S.spense_set_log(1) == 0
        Lg = S.spense_layout(9024, 5120, 1, 0, 7040)
        pg = S.spense_packed_t(1, 0, 9024, 5120, 7040, 4096, Lg.values_ld, 8192, Lg.meta_ld, 16384, Lg.dense_ld)
        S.spense_gemm_workspace_size(M, pg)  # new key: one line
        S.spense_gemm_workspace_size(M, pg)  # cached: none
        err = capfd.readouterr().err.strip().splitlines()
        assert len(err) == 1 and err[0].startswith("spense: plan dtype=fp8 M=61 N=9024 K=5120 split=output"), err
        assert "-> row-split" in err[0] and "k_slices=" in err[0]
        assert S.spense_gemm_workspace_size(M, pk) == quiet  # the log does not change the plan
    finally:
        S.spense_set_log(prev)
