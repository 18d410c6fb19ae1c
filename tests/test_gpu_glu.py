"""GPU parity of the gate / up GEMMs with the GLU step in their epilogue (spense_gemm_glu,
sec. 3.2 output-split weights, sec. 3.3.1 Eq. (4) with SiLU), through the C ABI:

- exact-integer data (values in [-3, 3], power-of-two scales: g and u are exact in
  fp32, so the oracle's g and u equal the kernel's bit for bit): every element of H
  against the fp64 glu of the oracle's g and u, within the error of the device exp and
  reciprocal (relative (1.5 |g| + 8) 2^-24, the exp argument's rounding growing with
  |g|), at ragged M and N, dense_begin not a multiple of 4, a dense fraction of 0 and 1,
  and a leading dimension above N (nothing written between N and ldh);
- the same data through spense_quantize_fp8: codes and scales bit for bit equal to
  spense_glu_quantize_fp8 of the separately computed G and U (spense_gemm_grouped), so
  the fused MLP is the unfused one;
- random data: H within the fp32 GEMM error bound of the fp64 oracle, carried through
  the GLU (|dh/dg| <= 1.1 |u|, |dh/du| = |silu(g)|);
- spense_gemm_glu_fp8 (the same launch writing per-workgroup row maxima, then the
  quantisation from them): codes and scales bit for bit those of spense_quantize_fp8 on
  spense_gemm_glu's H, with code rows that allow 4-byte stores and rows that do not;
- the Qwen3-like gate / up (25600 x 5120, 25% dense rows) at M = 64, full size.
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


def exact_pair(cfg, M, N, K, db):
    """Gate and up weights (codes, masks, scales) of one geometry and one X (the gate
    draw's), exact-integer data."""
    Wg, mg, X, sg, sx = gen.make_exact_int(cfg, 0, M, N, K, gen.OUTPUT, db, gen.FP8)
    Wu, mu, _, su, _ = gen.make_exact_int(cfg, 1, M, N, K, gen.OUTPUT, db, gen.FP8)
    return (Wg, mg, sg), (Wu, mu, su), X, sx


def packed(S, W, mask, db):
    return S.tile(S.compress(tdev(W), tdev(mask), 0, db))


def oracle_y(X, W, mask, sw, sx, db):
    N, K = W.shape
    v, m, d, _ = oracle.compress(W, mask, FP8, 0, db)
    return oracle.spense_gemm(X, v, m, d, N, K, FP8, 0, db, sw, sx)["y_f32"]


def glu_bound(g, u, h_ref):
    """Relative (1.5 |g| + 8) 2^-24: the exp argument g log2(e) rounded (an error that
    grows with |g|), the exp and the reciprocal (about 1 ulp each), the add and three
    products.  Below the normal range (g < -87, where 1 / (1 + exp(-g)) is subnormal or
    exp overflows and the sigmoid comes out 0) an absolute |u| (|g| + 2) 2^-125."""
    return (1.5 * np.abs(g) + 8) * U32 * np.abs(h_ref) + np.abs(u) * (np.abs(g) + 2) * 2.0 ** -125 + 2.0 ** -125


EXACT_CASES = [  # M, N, K, dense_begin (a fraction: the trailing share of rows kept dense)
    (1, 64, 512, 0.25),
    (5, 200, 1024, 0.25),
    (17, 130, 512, 0.5),
    (33, 320, 1536, 0.25),
    (64, 512, 1024, 0.0),
    (64, 256, 512, 1.0),
    (100, 452, 640, 0.25),
    (7, 200, 512, 98),  # not a multiple of 4: element stores at the region seam
    (20, 136, 640, 72),
    (3, 48, 96, 0.25),  # K below one 512-column chunk
    (40, 80, 160, 0.5),
]


@pytest.mark.parametrize("M,N,K,split", EXACT_CASES)
def test_gemm_glu_exact(S, M, N, K, split):
    db = split if isinstance(split, int) else gen.split_point(N, K, gen.OUTPUT, split)
    say(f"[gemm-glu exact] M={M} N={N} K={K} dense_begin={db}")
    (Wg, mg, sg), (Wu, mu, su), X, sx = exact_pair(7 + M + N, M, N, K, db)
    pg, pu = packed(S, Wg, mg, db), packed(S, Wu, mu, db)
    Xd, sgd, sud, sxd = tdev(X), tdev(sg), tdev(su), tdev(sx)
    ldh = N + 12  # a wider output: the columns past N stay untouched
    Hbuf = torch.full((M, ldh), 7.0, dtype=torch.float32, device="cuda")
    H = S.gemm_glu(Xd, pg, pu, sgd, sud, sxd, out=Hbuf[:, :N])
    torch.cuda.synchronize()
    g = oracle_y(X, Wg, mg, sg, sx, db).astype(np.float64)
    u = oracle_y(X, Wu, mu, su, sx, db).astype(np.float64)
    h_ref = oracle.glu_f64(g, u)
    h = H.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(h - h_ref) <= glu_bound(g, u, h_ref))
    assert torch.all(Hbuf[:, N:] == 7.0)
    # the fused path feeds the down projection what the unfused one feeds it
    G, U = S.gemm_grouped(Xd, [pg, pu], [sgd, sud], sxd, out_f32=True)
    q0, s0 = S.glu_quantize_fp8(G, U)
    q1, s1 = S.quantize_fp8(H)
    torch.cuda.synchronize()
    assert torch.equal(q0, q1)
    assert torch.equal(s0.view(torch.int32), s1.view(torch.int32))
    # the quantisation from the epilogue's row maxima, into wide code rows (ldq not a
    # multiple of 4: element stores) and into packed ones
    for ldq in (N + 3, N):
        qbuf = torch.full((M, ldq), 0xAB, dtype=torch.uint8, device="cuda")
        s2 = torch.empty(M, dtype=torch.float32, device="cuda")
        S.gemm_glu_fp8(Xd, pg, pu, sgd, sud, sxd, q=qbuf[:, :N], scales=s2)
        torch.cuda.synchronize()
        assert torch.equal(qbuf[:, :N], q1)
        assert torch.all(qbuf[:, N:] == 0xAB)
        assert torch.equal(s2.view(torch.int32), s1.view(torch.int32))


def test_gemm_glu_no_scales(S):
    """Without weight and token scales: H is glu of the raw accumulators."""
    M, N, K, db = 9, 192, 512, 144
    (Wg, mg, _), (Wu, mu, _), X, _ = exact_pair(3, M, N, K, db)
    H = S.gemm_glu(tdev(X), packed(S, Wg, mg, db), packed(S, Wu, mu, db))
    torch.cuda.synchronize()
    g = oracle_y(X, Wg, mg, None, None, db).astype(np.float64)
    u = oracle_y(X, Wu, mu, None, None, db).astype(np.float64)
    h_ref = oracle.glu_f64(g, u)
    assert np.all(np.abs(H.cpu().numpy() - h_ref) <= glu_bound(g, u, h_ref))


def test_gemm_glu_random_within_bound(S):
    M, N, K = 48, 640, 1536
    db = gen.split_point(N, K, gen.OUTPUT, 0.25)
    r = np.random.default_rng(11)
    Wg, sg = gen.quantize_rows_fp8(gen.draw_weight(r, N, K))
    Wu, su = gen.quantize_rows_fp8(gen.draw_weight(r, N, K))
    X, sx = gen.quantize_rows_fp8(gen.draw_x(r, M, K, "normal"))
    mg = gen.random_mask_24(r, N, K, gen.OUTPUT, db, True)
    mu = gen.random_mask_24(r, N, K, gen.OUTPUT, db, True)
    H = S.gemm_glu(tdev(X), packed(S, Wg, mg, db), packed(S, Wu, mu, db), tdev(sg), tdev(su), tdev(sx))
    torch.cuda.synchronize()
    gamma = K * U32 / (1 - K * U32)
    scale_x = np.abs(sx.astype(np.float64))[:, None]
    res = {}
    for name, W, mask, sw in (("g", Wg, mg, sg), ("u", Wu, mu, su)):
        v, m, d, _ = oracle.compress(W, mask, FP8, 0, db)
        o = oracle.gemm_f64(X, oracle.decompress(v, m, d, N, K, FP8, 0, db), FP8, sw, sx)
        err = (2.0 ** -12 + 2 * gamma) * o["abs_dot"] * np.abs(sw.astype(np.float64))[None, :] * scale_x \
            + 4 * U32 * np.abs(o["y"])
        res[name] = (o["y"], err)
    (g, eg), (u, eu) = res["g"], res["u"]
    h_ref = oracle.glu_f64(g, u)
    silu = np.abs(oracle.glu_f64(g, np.ones_like(g)))
    bound = 1.1 * (np.abs(u) + eu) * eg + (silu + 1.1 * eg) * eu + glu_bound(g, u, h_ref)
    assert np.all(np.abs(H.cpu().numpy().astype(np.float64) - h_ref) <= bound)


def test_gemm_glu_qwen3_gate_up_full_size(S):
    """Gate and up 25600 x 5120, 25% dense rows, M = 64 (the decode batch of the
    headline workload), exact-integer data: every H element within the GLU bound, and
    the quantised H bit for bit that of the unfused path."""
    M, N, K = 64, 25600, 5120
    db = gen.split_point(N, K, gen.OUTPUT, 0.25)
    say(f"[gemm-glu full size] M={M} N={N} K={K} dense_begin={db}")
    (Wg, mg, sg), (Wu, mu, su), X, sx = exact_pair(41, M, N, K, db)
    pg, pu = packed(S, Wg, mg, db), packed(S, Wu, mu, db)
    Xd, sgd, sud, sxd = tdev(X), tdev(sg), tdev(su), tdev(sx)
    H = S.gemm_glu(Xd, pg, pu, sgd, sud, sxd)
    G, U = S.gemm_grouped(Xd, [pg, pu], [sgd, sud], sxd, out_f32=True)
    q0, s0 = S.glu_quantize_fp8(G, U)
    q1, s1 = S.quantize_fp8(H)
    q2, s2 = S.gemm_glu_fp8(Xd, pg, pu, sgd, sud, sxd)
    torch.cuda.synchronize()
    assert torch.equal(q0, q1) and torch.equal(q1, q2)
    assert torch.equal(s0.view(torch.int32), s1.view(torch.int32))
    assert torch.equal(s2.view(torch.int32), s1.view(torch.int32))
    g = oracle_y(X, Wg, mg, sg, sx, db).astype(np.float64)
    u = oracle_y(X, Wu, mu, su, sx, db).astype(np.float64)
    h_ref = oracle.glu_f64(g, u)
    assert np.all(np.abs(H.cpu().numpy() - h_ref) <= glu_bound(g, u, h_ref))


def test_gemm_glu_fp8_random_rows(S):
    """Random data with rows of very different magnitude and an all-zero token (scale 1):
    the fused quantisation equals the two-step one bit for bit, over several token
    blocks (M = 150)."""
    M, N, K = 150, 1000, 768
    db = gen.split_point(N, K, gen.OUTPUT, 0.25)
    r = np.random.default_rng(23)
    Wg, sg = gen.quantize_rows_fp8(gen.draw_weight(r, N, K))
    Wu, su = gen.quantize_rows_fp8(gen.draw_weight(r, N, K))
    Xf = gen.draw_x(r, M, K, "normal") * np.exp(r.uniform(-6, 6, (M, 1))).astype(np.float32)
    Xf[7] = 0
    X, sx = gen.quantize_rows_fp8(Xf)
    mg = gen.random_mask_24(r, N, K, gen.OUTPUT, db, True)
    mu = gen.random_mask_24(r, N, K, gen.OUTPUT, db, True)
    pg, pu = packed(S, Wg, mg, db), packed(S, Wu, mu, db)
    args = (tdev(X), pg, pu, tdev(sg), tdev(su), tdev(sx))
    q1, s1 = S.quantize_fp8(S.gemm_glu(*args))
    q2, s2 = S.gemm_glu_fp8(*args)
    torch.cuda.synchronize()
    assert torch.equal(q1, q2)
    assert torch.equal(s1.view(torch.int32), s2.view(torch.int32))
    assert s2[7].item() == 1.0


def test_gemm_glu_validates_arguments(S):
    M, N, K, db = 8, 128, 256, 96
    (Wg, mg, _), (Wu, mu, _), X, _ = exact_pair(5, M, N, K, db)
    pg = packed(S, Wg, mg, db)
    other_db = packed(S, Wu, gen.random_mask_24(np.random.default_rng(1), N, K, gen.OUTPUT, 64), 64)
    with pytest.raises(S.SpenseError):
        S.gemm_glu(tdev(X), pg, other_db)  # dense_begin differs
    rowmajor = S.compress(tdev(Wu), tdev(mu), 0, db)
    with pytest.raises(S.SpenseError):
        S.gemm_glu(tdev(X), pg, rowmajor)  # not the tiled layout
    with pytest.raises(ValueError):
        S.gemm_glu(tdev(X[:, :128]), pg, pg)  # K differs from X
