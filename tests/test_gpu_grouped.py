"""GPU parity of the grouped launch (spense_gemm_grouped: several Spense weights that
share X and K in one launch, e.g. q / k / v or gate / up), through the C ABI.

- exact-integer data (values in [-3, 3], power-of-two scales: every partial sum is an
  exact integer, so any summation order gives the same fp32 value): every output bit
  for bit against the oracle, bf16 and fp32, at ragged M and weight sizes that are not
  multiples of the workgroup's rows;
- random data: each output within the fp32 error bound of the fp64 oracle;
- the Qwen3-like q, k, v at M = 64 (full size, exact-integer data) bit for bit.
"""
import sys

import numpy as np
import pytest
import torch

import gen
import oracle

pytestmark = pytest.mark.gpu

FP8 = 1
U32 = 2.0 ** -24


@pytest.fixture(scope="module")
def S():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10445_amd as S
    return S


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def tdev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def weights(cfg, shapes, M, K, exact=True):
    """Per weight: (codes, mask, sw, dense_begin); one X and sx for all (the first draw's)."""
    out, X, sx = [], None, None
    for i, (N, frac) in enumerate(shapes):
        db = gen.split_point(N, K, gen.OUTPUT, frac)
        if exact:
            W, mask, Xi, sw, sxi = gen.make_exact_int(cfg, i, M, N, K, gen.OUTPUT, db, gen.FP8)
        else:
            r = np.random.default_rng(cfg * 10 + i)
            W, sw = gen.quantize_rows_fp8(gen.draw_weight(r, N, K))
            Xi, sxi = gen.quantize_rows_fp8(gen.draw_x(r, M, K, "normal"))
            mask = gen.random_mask_24(r, N, K, gen.OUTPUT, db, True)
        if X is None:
            X, sx = Xi, sxi
        out.append((W, mask, sw, db))
    return out, X, sx


def packed(S, W, mask, db):
    return S.tile(S.compress(tdev(W), tdev(mask), 0, db))


GROUP_CASES = [  # M, K, [(N, dense fraction)]
    (1, 1024, [(320, 0.25), (64, 0.25), (64, 0.25)]),
    (17, 512, [(200, 0.25), (48, 0.5)]),
    (64, 1024, [(320, 0.25), (64, 0.25), (64, 0.25)]),
    (100, 640, [(256, 0.0), (96, 1.0), (144, 0.25), (16, 0.25)]),
    (33, 384, [(512, 0.25)]),
    (32, 5120, [(128, 0.25), (48, 0.25)]),   # two token tiles, activations resident: 160 KB
    (9, 10240, [(96, 0.25), (32, 0.5)]),     # one token tile, 20 chunks resident
    # more row groups than CUs at 33-64 tokens (two rounds of workgroups)
    (64, 1024, [(20480, 0.25), (20480, 0.25)]),
    (64, 256, [(20480, 0.25), (20480, 0.25)]),   # one chunk
    (40, 640, [(24576, 0.25), (8192, 0.5), (4096, 0.0), (1000, 1.0)]),  # four weights, all-2:4 and all-dense ones, ragged chunk
    (33, 1536, [(32768, 0.25), (4104, 0.25)]),  # ragged last row group
]


@pytest.mark.parametrize("M,K,shapes", GROUP_CASES)
def test_grouped_exact(S, M, K, shapes):
    say(f"[grouped exact] M={M} K={K} {shapes}")
    ws, X, sx = weights(5 + M, shapes, M, K)
    pws = [packed(S, W, mask, db) for (W, mask, sw, db) in ws]
    sws = [tdev(sw) for (_, _, sw, _) in ws]
    for out_f32 in (True, False):
        ys = S.gemm_grouped(tdev(X), pws, sws, tdev(sx), out_f32=out_f32)
        torch.cuda.synchronize()
        for (W, mask, sw, db), y in zip(ws, ys):
            v, m, d, bad = oracle.compress(W, mask, FP8, 0, db)
            ref = oracle.spense_gemm(X, v, m, d, W.shape[0], K, FP8, 0, db, sw, sx)
            got = y.cpu().numpy() if out_f32 else y.view(torch.int16).cpu().numpy().view(np.uint16)
            assert np.array_equal(got, ref["y_f32" if out_f32 else "y_bf16"])


# Many tokens: the grouped 256 x 256 large-M launch (at least 160 tiles), its tail tiles and
# XCD-aware order over every weight's regions; between 64 tokens and that grid, one launch
# per weight; (M, K, [(N, dense fraction)]).
GROUP_LARGE_M_CASES = [
    (4096, 256, [(1280, 0.25), (640, 0.25), (640, 0.5)]),   # 11 row blocks x 16 token blocks
    (3400, 384, [(1536, 0.25), (768, 0.25), (768, 0.25)]),  # 12 x 14, ragged M
    (520, 256, [(640, 0.25), (256, 0.25), (200, 0.5)]),     # 5 x 3: per-weight launches
    (520, 256, [(10240, 0.25), (2048, 0.25), (2048, 0.5)]),  # 56 x 3 on the grid, a ragged third block
    (65, 512, [(512, 0.25), (128, 0.25)]),                  # just above the row-split range
]


@pytest.mark.parametrize("M,K,shapes", GROUP_LARGE_M_CASES)
def test_grouped_large_m_exact(S, M, K, shapes):
    say(f"[grouped large-M exact] M={M} K={K} {shapes}")
    ws, X, sx = weights(11 + M % 7, shapes, M, K)
    pws = [packed(S, W, mask, db) for (W, mask, sw, db) in ws]
    sws = [tdev(sw) for (_, _, sw, _) in ws]
    ys = S.gemm_grouped(tdev(X), pws, sws, tdev(sx), out_f32=True)
    ys16 = S.gemm_grouped(tdev(X), pws, sws, tdev(sx))  # bf16: the output tile through LDS
    torch.cuda.synchronize()
    for (W, mask, sw, db), y, y16 in zip(ws, ys, ys16):
        v, m, d, bad = oracle.compress(W, mask, FP8, 0, db)
        ref = oracle.spense_gemm(X, v, m, d, W.shape[0], K, FP8, 0, db, sw, sx)
        assert np.array_equal(y.cpu().numpy(), ref["y_f32"])
        assert np.array_equal(y16.view(torch.int16).cpu().numpy().view(np.uint16), ref["y_bf16"])


# Seeded random groups: 1-4 output-split weights of ragged N sharing a ragged K, any
# boundary, at token counts on each of the three paths (row-split grid up to 64, one
# launch per weight, the 256 x 256 grid).
def _grouped_random_cases(n=8, seed=2414):
    r = np.random.default_rng(seed)
    out = []
    for i in range(n):
        K = 32 * int(r.integers(4, 80))
        shapes = [(int(r.integers(16, 2000)), float(r.choice([0.0, 0.25, 0.5, 1.0]))) for _ in range(int(r.integers(1, 5)))]
        M = int(r.choice([int(r.integers(1, 65)), int(r.integers(65, 300)), int(r.integers(300, 1100))]))
        out.append((i, M, K, shapes))
    return out


@pytest.mark.parametrize("i,M,K,shapes", _grouped_random_cases())
def test_grouped_random_shapes_exact(S, i, M, K, shapes):
    say(f"[grouped random] M={M} K={K} {shapes}")
    ws, X, sx = weights(60 + i, shapes, M, K)
    pws = [packed(S, W, mask, db) for (W, mask, sw, db) in ws]
    sws = [tdev(sw) for (_, _, sw, _) in ws]
    for out_f32 in (True, False):
        ys = S.gemm_grouped(tdev(X), pws, sws, tdev(sx), out_f32=out_f32)
        torch.cuda.synchronize()
        for (W, mask, sw, db), y in zip(ws, ys):
            v, m, d, bad = oracle.compress(W, mask, FP8, 0, db)
            ref = oracle.spense_gemm(X, v, m, d, W.shape[0], K, FP8, 0, db, sw, sx)
            got = y.cpu().numpy() if out_f32 else y.view(torch.int16).cpu().numpy().view(np.uint16)
            assert np.array_equal(got, ref["y_f32" if out_f32 else "y_bf16"])


def test_grouped_random_within_bound(S):
    M, K = 48, 1536
    shapes = [(640, 0.25), (128, 0.25), (128, 0.25)]
    ws, X, sx = weights(9, shapes, M, K, exact=False)
    pws = [packed(S, W, mask, db) for (W, mask, sw, db) in ws]
    ys = S.gemm_grouped(tdev(X), pws, [tdev(sw) for (_, _, sw, _) in ws], tdev(sx), out_f32=True)
    torch.cuda.synchronize()
    for (W, mask, sw, db), y in zip(ws, ys):
        v, m, d, _ = oracle.compress(W, mask, FP8, 0, db)
        Wd = oracle.decompress(v, m, d, W.shape[0], K, FP8, 0, db)
        o = oracle.gemm_f64(X, Wd, FP8, sw, sx)
        gamma = K * U32 / (1 - K * U32)
        scale = np.abs(sw.astype(np.float64))[None, :] * np.abs(sx.astype(np.float64))[:, None]
        bound = (2.0 ** -12 + 2 * gamma) * o["abs_dot"] * scale + 4 * U32 * np.abs(o["y"]) + 1e-38
        assert np.all(np.abs(y.cpu().numpy().astype(np.float64) - o["y"]) <= bound)


def test_grouped_qkv_full_size(S):
    """The q (8192 x 5120), k and v (1024 x 5120) projections of the Qwen3-like layer at
    M = 64, 25% dense rows each, in one launch: every bf16 output bit for bit."""
    M, K = 64, 5120
    ws, X, sx = weights(31, [(8192, 0.25), (1024, 0.25), (1024, 0.25)], M, K)
    pws = [packed(S, W, mask, db) for (W, mask, sw, db) in ws]
    ys = S.gemm_grouped(tdev(X), pws, [tdev(sw) for (_, _, sw, _) in ws], tdev(sx))
    torch.cuda.synchronize()
    for (W, mask, sw, db), y in zip(ws, ys):
        v, m, d, _ = oracle.compress(W, mask, FP8, 0, db)
        ref = oracle.spense_gemm(X, v, m, d, W.shape[0], K, FP8, 0, db, sw, sx)
        assert np.array_equal(y.view(torch.int16).cpu().numpy().view(np.uint16), ref["y_bf16"])


@pytest.mark.timeout(400)
@pytest.mark.parametrize("group", ["qkv", "gate_up"])
def test_grouped_seed_oss_full_size_at_decode_m(S, group):
    """The Seed-OSS-36B-like q (10240), k and v (1024 rows) or gate and up (27648 rows),
    K = 5120, 25% dense rows each, grouped in one launch at M = 64, 16, 4 and 1 (the
    benchmark's grouped layer timing): every output bit for bit, bf16 and fp32, on
    exact-integer data.  The activations of a smaller M are the first rows of the M = 64
    draw; each output row depends on its own row only."""
    shapes = [(10240, 0.25), (1024, 0.25), (1024, 0.25)] if group == "qkv" else [(27648, 0.25), (27648, 0.25)]
    K, Mmax = 5120, 64
    ws, X, sx = weights(41 if group == "qkv" else 43, shapes, Mmax, K)
    say(f"[grouped seed] {group}")
    pws = [packed(S, W, mask, db) for (W, mask, sw, db) in ws]
    sws = [tdev(sw) for (_, _, sw, _) in ws]
    refs = []
    for (W, mask, sw, db) in ws:
        v, m, d, _ = oracle.compress(W, mask, FP8, 0, db)
        refs.append(oracle.spense_gemm(X, v, m, d, W.shape[0], K, FP8, 0, db, sw, sx))
    for M in (64, 16, 4, 1):
        for out_f32 in (True, False):
            ys = S.gemm_grouped(tdev(X[:M]), pws, sws, tdev(sx[:M]), out_f32=out_f32)
            torch.cuda.synchronize()
            for ref, y in zip(refs, ys):
                got = y.cpu().numpy() if out_f32 else y.view(torch.int16).cpu().numpy().view(np.uint16)
                assert np.array_equal(got, ref["y_f32" if out_f32 else "y_bf16"][:M]), f"{group} M={M}"


def test_grouped_validates_arguments(S):
    M, K = 8, 256
    ws, X, sx = weights(3, [(64, 0.25), (32, 0.25)], M, K)
    pws = [packed(S, W, mask, db) for (W, mask, sw, db) in ws]
    other = S.tile(S.compress(tdev(ws[0][0][:, :128]), tdev(ws[0][1][:, :128]), 0, ws[0][3]))
    with pytest.raises(ValueError):
        S.gemm_grouped(tdev(X), [pws[0], other])  # K differs
    rowmajor = S.compress(tdev(ws[0][0]), tdev(ws[0][1]), 0, ws[0][3])
    with pytest.raises(S.SpenseError):
        S.gemm_grouped(tdev(X), [pws[0], rowmajor])  # not the tiled layout
    with pytest.raises(S.SpenseError):
        S.gemm_grouped(tdev(X), pws * 3)  # more than four weights
