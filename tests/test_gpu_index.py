"""GPU parity of the SpenseGPT+ dense-index selection (sec. 3.3.1), through the C ABI,
against the CPU oracle:

- priorities (spense_index_scores): each raw vector and the normalised total within a
  relative bound derived from fp32 recursive summation of positive terms: a sum of n
  positive terms carries a relative error of at most (n - 1) u, u = 2^-24, and the
  kernels sum at most D / 4 (the column scores), D / 256 + 8 (the row scores) and
  I / 1024 + 16 (the means) terms in a row, plus a few roundings for sqrt, the products
  and the divisions;
- TopK and permutation (spense_dense_permutation): an integer decision taken from fp32
  priorities, so the oracle is given the very fp32 totals the device produced and flags
  and perm must match bit for bit; separately, the chosen set must be a valid TopK of
  the oracle's fp64 totals within the priority tolerance;
- gathers (spense_gather_rows / spense_gather_cols): bit-exact against indexing.
"""
import sys

import numpy as np
import pytest
import torch

import gen
import oracle

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


@pytest.fixture(scope="module")
def S():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10445_amd as S
    return S


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def mlp_weights(seed, I, D):
    """Gate / up (I x D) and down (D x I) weights whose rows and columns have spread norms
    (log-normal per-index scales), and Hessian diagonals from synthetic calibration
    activations with a few outlier channels."""
    r = np.random.default_rng(seed)
    scale_i = np.exp(r.normal(0, 0.5, I)).astype(np.float32)
    Wg = gen.draw_weight(r, I, D) * scale_i[:, None]
    Wu = gen.draw_weight(r, I, D) * np.exp(r.normal(0, 0.3, I)).astype(np.float32)[:, None]
    Wd = gen.draw_weight(r, D, I) * scale_i[None, :]
    X = gen.draw_x(r, 64, D) * np.exp(r.normal(0, 1.0, D)).astype(np.float32)
    h_in = (X.astype(np.float64) ** 2).sum(0).astype(np.float32)
    Hm = gen.draw_x(r, 64, I) * np.exp(r.normal(0, 1.0, I)).astype(np.float32)
    h_mid = (Hm.astype(np.float64) ** 2).sum(0).astype(np.float32)
    return Wg, Wu, Wd, h_in, h_mid


def as_dtype(A, dtype):
    """(numpy fp32 values both sides see, device tensor)."""
    if dtype == "bf16":
        bits = gen.to_bf16(A)
        t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()
        return (bits.astype(np.uint32) << 16).view(np.float32), t
    return A, torch.from_numpy(np.ascontiguousarray(A)).cuda()


def score_rtol(I, D):
    return (D / 4 + D / 256 + I / 1024 + 64) * U


SCORE_CASES = [  # (I, D, dtype, n_dense)
    (1, 7, "f32", 1),
    (300, 257, "f32", 75),
    (1000, 512, "bf16", 250),
    (2049, 130, "bf16", 512),
    (3000, 1024, "bf16", 0),
    (1024, 1024, "bf16", 1024),
]


@pytest.mark.parametrize("I,D,dtype,n_dense", SCORE_CASES)
def test_index_scores_and_permutation(S, I, D, dtype, n_dense):
    say(f"index scores I={I} D={D} {dtype} n_dense={n_dense}")
    Wg, Wu, Wd, h_in, h_mid = mlp_weights(100 + I, I, D)
    (g, tg), (u, tu), (d, td) = as_dtype(Wg, dtype), as_dtype(Wu, dtype), as_dtype(Wd, dtype)
    ref = oracle.index_scores(g, u, d, h_in, h_mid)
    out = S.index_scores(tg, tu, td, torch.from_numpy(h_in).cuda(), torch.from_numpy(h_mid).cuda())
    torch.cuda.synchronize()
    rtol = score_rtol(I, D)
    for k in ("gate", "up", "down", "total"):
        got = out[k].cpu().numpy().astype(np.float64)
        err = np.max(np.abs(got - ref[k]) / np.abs(ref[k]))
        assert err <= rtol, (k, err, rtol)
    total = out["total"]
    flags, perm = S.dense_permutation(total, n_dense)
    torch.cuda.synchronize()
    t32 = total.cpu().numpy().astype(np.float64)
    pr = oracle.dense_index_permutation(t32, n_dense)
    want_flags = np.zeros(I, np.uint8)
    want_flags[pr["dense"]] = 1
    assert np.array_equal(flags.cpu().numpy(), want_flags)
    assert np.array_equal(perm.cpu().numpy(), pr["perm"])
    # a valid TopK of the fp64 priorities, up to the priority tolerance
    f = want_flags.astype(bool)
    if 0 < n_dense < I:
        lo, hi = ref["total"][f].min(), ref["total"][~f].max()
        assert lo >= hi * (1 - 4 * rtol), (lo, hi)


def test_permutation_ties_and_nan(S):
    """Equal priorities keep the lower index first; NaN ranks below every number; blocks
    of the scan (1024 indices) are crossed."""
    r = np.random.default_rng(7)
    for I, n_dense in ((2500, 900), (1024, 1), (1025, 1024), (5, 3)):
        t = r.integers(0, 6, I).astype(np.float32)
        t[r.integers(0, I, max(1, I // 50))] = np.nan
        t[r.integers(0, I, max(1, I // 100))] = np.inf
        say(f"permutation ties I={I} n_dense={n_dense}")
        flags, perm = S.dense_permutation(torch.from_numpy(t).cuda(), n_dense)
        torch.cuda.synchronize()
        pr = oracle.dense_index_permutation(t.astype(np.float64), n_dense)
        assert np.array_equal(perm.cpu().numpy(), pr["perm"])
        assert np.array_equal(np.flatnonzero(flags.cpu().numpy()), pr["dense"])


@pytest.mark.parametrize("rows,cols,dtype,ld_pad", [
    (513, 4096, torch.bfloat16, 0), (77, 123, torch.uint8, 5), (64, 33, torch.float32, 3), (1, 16, torch.uint8, 0),
    (300, 1000, torch.uint8, 24), (128, 512, torch.uint8, 32)])
def test_gathers_bit_exact(S, rows, cols, dtype, ld_pad):
    say(f"gathers {rows}x{cols} {dtype} pad={ld_pad}")
    g = torch.Generator().manual_seed(rows * 7 + cols)
    base = torch.randint(0, 256, (rows, cols + ld_pad), generator=g, dtype=torch.uint8)
    if dtype != torch.uint8:
        base = torch.randint(-2**15, 2**15, (rows, (cols + ld_pad) * dtype.itemsize // 2), generator=g,
                             dtype=torch.int16).view(dtype)
    src = base.cuda()[:, :cols]
    prow = torch.randperm(rows, generator=g).to(torch.int32)
    pcol = torch.randperm(cols, generator=g).to(torch.int32)
    out_r = S.gather_rows(src, prow.cuda())
    out_c = S.gather_cols(src, pcol.cuda())
    torch.cuda.synchronize()
    s = src.cpu()
    assert torch.equal(out_r.cpu().view(torch.uint8), s[prow.long()].contiguous().view(torch.uint8))
    assert torch.equal(out_c.cpu().view(torch.uint8), s[:, pcol.long()].contiguous().view(torch.uint8))


def test_qwen3_mlp_selection(S):
    """The whole step at the MLP size of the workload (I = 25600, D = 5120, bf16 weights,
    25% of the indices dense): priorities against the oracle, the permutation exact on the
    device's priorities, and the permuted weights equal to the oracle's indexing (Eq. (4):
    the rows of gate / up and the columns of down move together)."""
    I, D, n_dense = 25600, 5120, 6400
    say(f"qwen3 selection I={I} D={D} n_dense={n_dense}")
    Wg, Wu, Wd, h_in, h_mid = mlp_weights(3, I, D)
    (g, tg), (u, tu), (d, td) = as_dtype(Wg, "bf16"), as_dtype(Wu, "bf16"), as_dtype(Wd, "bf16")
    del Wg, Wu, Wd
    out = S.select_dense_indices(tg, tu, td, torch.from_numpy(h_in).cuda(), torch.from_numpy(h_mid).cuda(), n_dense)
    torch.cuda.synchronize()
    ref = oracle.index_scores(g, u, d, h_in, h_mid)
    rtol = score_rtol(I, D)
    got = out["scores"]["total"].cpu().numpy().astype(np.float64)
    assert np.max(np.abs(got - ref["total"]) / np.abs(ref["total"])) <= rtol
    pr = oracle.dense_index_permutation(got, n_dense)
    perm = out["perm"].cpu().numpy()
    assert np.array_equal(perm, pr["perm"])
    p = torch.from_numpy(perm.astype(np.int64))
    assert torch.equal(out["Wg"].cpu(), tg.cpu()[p])
    assert torch.equal(out["Wu"].cpu(), tu.cpu()[p])
    assert torch.equal(out["Wd"].cpu(), td.cpu()[:, p])


@pytest.mark.timeout(300)
@pytest.mark.parametrize("D,I,M", [(512, 1536, 9), (5120, 25600, 64)])
def test_permuted_mlp_is_the_same_function(S, D, I, M):
    """Eq. (4) on the device: permuting the rows of gate / up (codes and per-row scales)
    and the columns of down by the selection's perm leaves the MLP unchanged.  The gate
    and up outputs and the quantised GLU codes move with perm bit for bit (each output
    keeps its own dot product; the per-token absmax does not depend on the order).  The
    down projection sums the same K = I products in another order, so its fp32 outputs
    agree elementwise within twice the fp32 summation bound plus the epilogue roundings:
    |Y' - Y| <= 2 (K + 4) u sum_k |h_k| |w_k| (scales included).  All-dense weights: the
    identity holds before any pruning."""
    say(f"[eq4] D={D} I={I} M={M}")
    mg = gen.make_matrix(70, 0, "gate", I, D, gen.OUTPUT, 1.0, gen.FP8)
    mu = gen.make_matrix(71, 0, "up", I, D, gen.OUTPUT, 1.0, gen.FP8)
    md = gen.make_matrix(72, 1, "down", D, I, gen.INPUT, 1.0, gen.FP8)
    cg, cu, cd = (torch.from_numpy(m.W).cuda() for m in (mg, mu, md))
    sg, su, sd = (torch.from_numpy(m.sw).cuda() for m in (mg, mu, md))
    f8 = torch.float8_e4m3fn
    # master weights for the priorities: the decoded fp8 weights
    Wg = (cg.view(f8).float() * sg[:, None]).contiguous()
    Wu = (cu.view(f8).float() * su[:, None]).contiguous()
    Wd = (cd.view(f8).float() * sd[:, None]).contiguous()
    r = np.random.default_rng(I)
    h_in = torch.from_numpy(r.uniform(0.5, 50, D).astype(np.float32)).cuda()
    h_mid = torch.from_numpy(r.uniform(0.5, 50, I).astype(np.float32)).cuda()
    perm = S.select_dense_indices(Wg, Wu, Wd, h_in, h_mid, I // 4)["perm"]
    del Wg, Wu, Wd
    cg2, cu2, cd2 = S.gather_rows(cg, perm), S.gather_rows(cu, perm), S.gather_cols(cd, perm)
    sg2 = S.gather_cols(sg.view(1, I), perm).view(I)
    su2 = S.gather_cols(su.view(1, I), perm).view(I)
    pk = lambda W, ax: S.compress(W, None, ax, 0)
    X, sx = gen.make_x(70, 0, M, D, gen.FP8)
    Xd, sxd = torch.from_numpy(X).cuda(), torch.from_numpy(sx).cuda()
    outs = []
    for (c_g, c_u, c_d, s_g, s_u) in ((cg, cu, cd, sg, su), (cg2, cu2, cd2, sg2, su2)):
        G = S.gemm(Xd, pk(c_g, 0), s_g, sxd, out_f32=True)
        U_ = S.gemm(Xd, pk(c_u, 0), s_u, sxd, out_f32=True)
        Hq, sh = S.glu_quantize_fp8(G, U_)
        Y = S.gemm(Hq, pk(c_d, 1), sd, sh, out_f32=True)
        outs.append((G, U_, Hq, sh, Y))
    torch.cuda.synchronize()
    (G, U_, Hq, sh, Y), (G2, U2, Hq2, sh2, Y2) = outs
    p = perm.long()
    assert torch.equal(G2.view(torch.int32), G[:, p].view(torch.int32))
    assert torch.equal(U2.view(torch.int32), U_[:, p].view(torch.int32))
    assert torch.equal(Hq2, Hq[:, p]) and torch.equal(sh2, sh)
    habs = (Hq.view(f8).float().double() * sh.double()[:, None]).abs()
    wabs = (cd.view(f8).float().double() * sd.double()[:, None]).abs().t().contiguous()
    bound = 2 * (I + 4) * U * (habs @ wabs)
    diff = (Y2.double() - Y.double()).abs()
    assert bool((diff <= bound).all()), (diff - bound).max().item()
