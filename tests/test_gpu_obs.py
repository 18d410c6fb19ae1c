"""GPU parity of SparseGPT 2:4 pruning with the dense region kept last (sec. 3.1.2,
Eqs. (2)-(3); sec. 3.3.1), through the C ABI, against the CPU oracle (fp64).

Tolerances come from the arithmetic.  The factor U (Hd^{-1} = U^T U) is formed in fp32
by a Cholesky factorisation and a triangular inverse; both have first-order normwise
forward errors of at most about kappa(Hd) K u and sqrt(kappa(Hd)) K u, so U is checked
to relative Frobenius error <= 2 (kappa + sqrt(kappa)) K u, with kappa(Hd) computed
(or bounded above: lambda_max by the largest absolute row sum, lambda_min by the damping
plus the tridiagonal part's smallest eigenvalue) from the test's own Hessian.  The swept
weights inherit U's error through the compensation plus K roundings of their own:
relative Frobenius <= 2 tol_U + 4 K u.  The 2:4 choice is an integer decision taken from
floating-point errors computed along different paths on the two sides, so it is
compared exactly only on weights built so that the decision is never close (in each
group two weights' scores exceed the other two's by a wide margin); on random weights
the masks must be valid 2:4, and where a row's mask differs from the oracle's, the
first differing choice must be a near tie of the oracle's errors.
"""
import sys

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24


@pytest.fixture(scope="module")
def S():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10445_amd as S
    return S


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def hessian(seed, K, M=4096, rank=64, dead=()):
    """A synthetic calibration Hessian: M (C^T C + diag(d)) + F F^T, C = I + 0.3 (shift),
    d ~ U[0, 1], F a K x rank Gaussian block with variance M / (2K) (dense correlations
    whose eigenvalues stay O(M)); fp32.  Columns in `dead` are zeroed (inputs that never
    fire).  Returns (H fp32, lower bound of lambda_min(H) before damping)."""
    r = np.random.default_rng(seed)
    d = r.uniform(0, 1, K)
    H = np.zeros((K, K), np.float64)
    idx = np.arange(K)
    H[idx, idx] = M * (1.0 + (idx + 1 < K) * 0.09 + d)
    H[idx[:-1], idx[:-1] + 1] = M * 0.3
    H[idx[:-1] + 1, idx[:-1]] = M * 0.3
    F = r.standard_normal((K, rank)).astype(np.float32) * np.float32(np.sqrt(0.5 * M / K))
    H = (H + (F @ F.T).astype(np.float64)).astype(np.float32)
    for j in dead:
        H[j, :] = 0
        H[:, j] = 0
    return H, M * (1 - 0.3) ** 2


def kappa_bound(H, lam_floor, percdamp=0.01):
    """Upper bound of cond2 of the damped Hessian: Gershgorin above, damping below."""
    Hd = H.astype(np.float64)
    lam = percdamp * np.mean(np.where(np.diag(Hd) == 0, 1.0, np.diag(Hd)))
    hi = np.abs(Hd).sum(1).max() + lam + 1.0
    return hi / (lam_floor + lam)


def kappa_exact(H, percdamp=0.01):
    Hd, _ = oracle.obs_damp(H, percdamp)
    ev = np.linalg.eigvalsh(Hd)
    return ev[-1] / ev[0]


def tol_u(kappa, K):
    return 2 * (kappa + np.sqrt(kappa)) * K * U32


def rel(a, b):
    return np.linalg.norm(np.asarray(a, np.float64) - b) / max(np.linalg.norm(b), 1e-300)


def separated_weights(seed, N, K, H):
    """Each group of four holds two weights whose score w^2 H_jj is at least 400x that of
    the other two (random positions and signs); with the well-conditioned Hessians here
    the OBS errors w^2 / U_mm^2 keep a wide margin, so the 2:4 choice is never close."""
    r = np.random.default_rng(seed)
    sh = 1.0 / np.sqrt(np.maximum(np.diag(H).astype(np.float64), 1.0))
    mag = r.uniform(0.0, 0.05, (N, K))
    big = np.zeros((N, K), bool)
    for g in range(K // 4):
        pos = np.argsort(r.random((N, 4)), axis=1)[:, :2]
        big[np.arange(N)[:, None], 4 * g + pos] = True
    mag[big] = r.uniform(1.0, 2.0, big.sum())
    W = mag * sh[None, :] * np.where(r.random((N, K)) < 0.5, -1.0, 1.0)
    return W.astype(np.float32)


def gpu_factor(S, H):
    U, dead = S.obs_factor(torch.from_numpy(H).cuda())
    torch.cuda.synchronize()
    return U, dead


def test_factor_of_a_diagonal_hessian(S):
    """Uncorrelated inputs: U = diag(1 / sqrt(h_jj + lambda)), zero elsewhere; a zero
    column is flagged dead and reads 1.  Error: the square root and the reciprocal (one
    rounding each), the sum h_jj + lambda, and lambda's fp32 mean over K positive terms
    (relative error <= K u), which moves U_jj by at most (lambda / hd_jj) K u / 2."""
    r = np.random.default_rng(1)
    K = 200
    h = r.uniform(0.5, 50, K).astype(np.float32)
    h[17] = 0
    U, dead = gpu_factor(S, np.diag(h))
    U = U.cpu().numpy().astype(np.float64)
    ref, rdead = oracle.obs_factor(np.diag(h))
    assert np.array_equal(dead.cpu().numpy().astype(bool), rdead)
    assert np.array_equal(U[~np.eye(K, dtype=bool)], np.zeros(K * K - K))
    hd = np.diag(oracle.obs_damp(np.diag(h))[0])
    lam = hd[0] - h[0]
    tol = 0.5 * lam / hd * K * U32 + 4 * U32
    assert (np.abs(np.diag(U) - np.diag(ref)) / np.diag(ref) <= tol).all()


@pytest.mark.parametrize("K", [64, 98, 100, 320, 700])
def test_factor_matches_oracle(S, K):
    say(f"[obs factor] K={K}")
    H, _ = hessian(K, K, dead=(3,) if K == 100 else ())
    U, dead = gpu_factor(S, H)
    ref, rdead = oracle.obs_factor(H)
    assert np.array_equal(dead.cpu().numpy().astype(bool), rdead)
    Ug = U.cpu().numpy()
    assert np.array_equal(np.tril(Ug, -1), np.zeros((K, K), np.float32))
    err, tol = rel(Ug, ref), tol_u(kappa_exact(H), K)
    say(f"  rel {err:.2e} tol {tol:.2e}")
    assert err <= tol


def run_prune(S, W, H, dense_begin, U=None, dead=None):
    if U is None:
        U, dead = gpu_factor(S, H)
    Wd = torch.from_numpy(W).cuda()
    keep = S.obs_prune_24(Wd, U, dense_begin, dead)
    torch.cuda.synchronize()
    return Wd.cpu().numpy(), keep.cpu().numpy().astype(bool)


@pytest.mark.parametrize("N,K,dense_begin", [(300, 256, 192), (77, 200, 100), (64, 128, 128), (33, 96, 0),
                                             (260, 384, 260), (50, 98, 64), (40, 130, 128), (70, 600, 516)])
def test_prune_matches_oracle_on_clear_choices(S, N, K, dense_begin):
    say(f"[obs prune] N={N} K={K} dense_begin={dense_begin}")
    H, _ = hessian(N + K, K, dead=(5,) if K == 200 else ())
    W = separated_weights(N * K, N, K, H)
    Wg, keep = run_prune(S, W, H, dense_begin)
    ref = oracle.obs_prune_24(W, H, dense_begin)
    assert np.array_equal(keep, ref["keep"])
    tol = 2 * tol_u(kappa_exact(H), K) + 4 * K * U32
    err = rel(Wg, ref["W"])
    say(f"  rel {err:.2e} tol {tol:.2e}")
    assert err <= tol
    assert np.array_equal(Wg[:, :dense_begin] != 0, keep[:, :dense_begin])


def check_valid_masks(keep, ref, dense_begin, tol):
    """2:4 in every group of the 2:4 columns, all kept after them; rows whose mask differs
    from the oracle's must differ first at a near tie of the oracle's OBS errors."""
    N = keep.shape[0]
    assert (keep[:, :dense_begin].reshape(N, -1, 4).sum(-1) == 2).all()
    assert keep[:, dense_begin:].all()
    differ = []
    for n in range(N):
        if np.array_equal(keep[n], ref["keep"][n]):
            continue
        differ.append(n)
        g = np.flatnonzero((keep[n, :dense_begin] != ref["keep"][n, :dense_begin]).reshape(-1, 4).any(1))[0]
        e = ref["err"][n, 4 * g:4 * g + 4]
        gpu_pruned = e[~keep[n, 4 * g:4 * g + 4]]
        threshold = np.sort(e)[1]  # the oracle prunes the two smallest
        assert gpu_pruned.max() <= threshold * (1 + tol) + 1e-300, (n, g, e)
    return differ


def test_prune_random_weights_gives_valid_choices(S):
    N, K, db = 257, 320, 256
    H, _ = hessian(11, K)
    W = np.random.default_rng(12).standard_normal((N, K)).astype(np.float32) * 0.02
    Wg, keep = run_prune(S, W, H, db)
    ref = oracle.obs_prune_24(W, H, db)
    tol = 2 * tol_u(kappa_exact(H), K) + 4 * K * U32
    differ = check_valid_masks(keep, ref, db, 10 * tol)
    same = np.setdiff1d(np.arange(N), differ)
    say(f"  rows with another valid choice: {len(differ)} of {N}")
    assert len(differ) <= N // 10
    assert rel(Wg[same], ref["W"][same]) <= tol


def test_gate_up_size(S):
    """The 2:4 rows of a gate / up projection of the MLP (19200 of 25600 rows kept 2:4 at
    25% dense, K = 5120; output-split, so the dense rows are not passed): the factor
    against the oracle's, and 8 sampled rows swept by the oracle."""
    N, K = 19200, 5120
    say(f"[obs gate/up] N={N} K={K}")
    H, floor = hessian(21, K)
    U, dead = gpu_factor(S, H)
    ref_U, ref_dead = oracle.obs_factor(H)
    tolU = tol_u(kappa_bound(H, floor), K)
    errU = rel(U.cpu().numpy(), ref_U)
    say(f"  factor rel {errU:.2e} tol {tolU:.2e}")
    assert errU <= tolU
    W = separated_weights(22, N, K, H)
    Wg, keep = run_prune(S, W, H, K, U, dead)
    rows = np.random.default_rng(23).choice(N, 8, replace=False)
    ref = oracle.obs_prune_24(W[rows], H, K, factor=(ref_U, ref_dead))
    assert np.array_equal(keep[rows], ref["keep"])
    assert rel(Wg[rows], ref["W"]) <= 2 * tolU + 4 * K * U32
    assert (keep.reshape(N, -1, 4).sum(-1) == 2).all()


def test_down_size_properties(S):
    """The down projection (N = 5120, K = 25600, the last 6400 columns dense): at this size
    the fp64 oracle factor is out of reach, so properties that hold at any size are
    checked: U upper triangular with a positive diagonal; Hd U^T U e_c = e_c on sampled
    columns (a residual of first order kappa(Hd) K u: checked <= 4 kappa K u); 2:4 masks;
    and on sampled rows the dense columns equal the least-squares compensation of the
    frozen 2:4 columns, w_D - Hd_DD^{-1} Hd_DS (w_hat_S - w_S) (the property the oracle is
    pinned by), to the weights' tolerance."""
    N, K, db = 5120, 25600, 19200
    say(f"[obs down] N={N} K={K} dense_begin={db}")
    H, floor = hessian(31, K, rank=32)
    U, dead = gpu_factor(S, H)
    kap = kappa_bound(H, floor)
    Hd, _ = oracle.obs_damp(H)
    d = torch.diagonal(U).cpu().numpy()
    assert (d > 0).all() and not dead.cpu().numpy().any()
    assert not torch.tril(U, -1).any().item()
    Uh = U.cpu().numpy()
    for c in (0, 1, 777, 12800, K - 2, K - 1):
        x = (Uh[:, c] @ Uh).astype(np.float64)  # (U^T U e_c)^T
        res = np.abs(Hd @ x - np.eye(1, K, c)[0]).max()
        assert res <= 4 * kap * K * U32, (c, res)
    del Uh
    W = separated_weights(32, N, K, H)
    Wg, keep = run_prune(S, W, H, db, U, dead)
    assert (keep[:, :db].reshape(N, -1, 4).sum(-1) == 2).all() and keep[:, db:].all()
    tolW = 2 * tol_u(kappa_bound(H, floor), K) + 4 * K * U32
    Sx, Dx = slice(0, db), slice(db, K)
    rows = np.random.default_rng(33).choice(N, 4, replace=False)
    want = W[rows][:, Dx] - np.linalg.solve(Hd[Dx, Dx], Hd[Dx, Sx] @ (Wg[rows][:, Sx] - W[rows][:, Sx]).T).T
    assert rel(Wg[rows][:, Dx], want) <= tolW


def test_back_placement_on_the_device(S):
    """Sec. 3.3.1, Table "front_back", through the library: the same dense columns,
    processed last (compensation buffer) versus first (frozen before any pruning: the
    sweep over the 2:4 columns alone), on seeded correlated data; Eq. (2)'s loss."""
    K, nd, N = 256, 64, 128
    H, _ = hessian(41, K, rank=128)
    W = np.random.default_rng(42).standard_normal((N, K)).astype(np.float32)
    back, _ = run_prune(S, W, H, K - nd)
    Sx = slice(0, K - nd)
    front = W.copy()
    front[:, Sx], _ = run_prune(S, np.ascontiguousarray(W[:, Sx]), np.ascontiguousarray(H[Sx, Sx]), K - nd)
    lb, lf = oracle.reconstruction_loss(W, back, H), oracle.reconstruction_loss(W, front, H)
    say(f"  loss back {lb:.4e} front {lf:.4e}")
    assert lb < lf
