"""Plain CPU oracle for the Spense hybrid 2:4-sparse / dense linear layer.

TEST INFRASTRUCTURE ONLY: tests, the smoke check and the benchmark's CPU-baseline leg
may import this package; the product library never does.  It shares no code with the
GPU path.  The arithmetic lives in ``spense_oracle.c`` (plain C, built with gcc); this
module only marshals numpy arrays.

Paper references (SpenseGPT): the 2:4 constraint is Eq. (1) in sec. 3.1.1, compressed
2:4 storage is described in sec. 3.1.1, the output-split / input-split Spense format in
sec. 3.2, and the dense region being the last one in sec. 3.3.2 and Table "front_back".

Parity status: every function here is pinned by tests that do not re-use it (format
definition vs torch's converters, brute force over all 2:4 masks, numpy fp64 matmul
within the Higham bound, exact-integer cases, linearity of the two split variants; for
the GLU-MLP steps: every e4m3fn code's round trip and midpoint, torch's converter, the
odd and even parts of SiLU, and the permutation invariance of Eq. (4); for the
SpenseGPT+ index step: closed forms of the scores, the Wanda identity, brute-force TopK;
for the SparseGPT sweep: the factor's rows against explicit inverse Hessians, Eq. (3)
with an explicit inverse per step, the diagonal-Hessian case (magnitude pruning), the
least-squares optimality of the dense buffer, and the edge cases; the reconstruction loss
of Eq. (2) against an explicit calibration matrix; the MLP of Eq. (4) against a
composition from numpy and torch's converters that shares none of this module's code).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

FP8 = 1
BF16 = 2
AXIS_OUTPUT = 0
AXIS_INPUT = 1

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spense_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (OpenMP, no FMA contraction, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", _SRC,
               "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        p, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        lib.or_decode_e4m3fn.restype = ctypes.c_double
        lib.or_decode_e4m3fn.argtypes = [ctypes.c_uint8]
        lib.or_decode_bf16.restype = ctypes.c_float
        lib.or_decode_bf16.argtypes = [ctypes.c_uint16]
        lib.or_bf16_rne.restype = ctypes.c_uint16
        lib.or_bf16_rne.argtypes = [ctypes.c_float]
        lib.or_decode_e4m3fn_array.argtypes = [p, i64, p]
        lib.or_decode_bf16_array.argtypes = [p, i64, p]
        lib.or_bf16_rne_array.argtypes = [p, i64, p]
        lib.or_layout.restype = i32
        lib.or_layout.argtypes = [i64, i64, i32, i64, p]
        lib.or_compress.restype = i64
        lib.or_compress.argtypes = [p, p, i64, i64, i32, i32, i64, p, p, p]
        lib.or_decompress.restype = i32
        lib.or_decompress.argtypes = [p, p, p, i64, i64, i32, i32, i64, p]
        lib.or_gemm_f32.restype = i32
        lib.or_gemm_f32.argtypes = [p, p, i64, i64, i64, i32, p, p, p, p, p]
        lib.or_gemm_f64.restype = i32
        lib.or_gemm_f64.argtypes = [p, p, i64, i64, i64, i32, p, p, p, p, p]
        lib.or_encode_e4m3fn.restype = ctypes.c_uint8
        lib.or_encode_e4m3fn.argtypes = [ctypes.c_float]
        lib.or_encode_e4m3fn_array.argtypes = [p, i64, p]
        lib.or_quantize_rows.argtypes = [p, i64, i64, i64, p, p]
        lib.or_glu_f64.argtypes = [p, p, i64, p]
        lib.or_set_threads.restype = i32
        lib.or_set_threads.argtypes = [i32]
        _lib = lib
    return _lib


def set_threads(n: int) -> int:
    """OpenMP threads of the oracle's parallel loops (0 keeps them); returns the previous
    maximum.  Harness only: the results do not depend on it."""
    return _L().or_set_threads(n)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _codes(a, dtype):
    want = np.uint8 if dtype == FP8 else np.uint16
    a = np.ascontiguousarray(a)
    if a.dtype != want:
        raise TypeError(f"expected {want} codes, got {a.dtype}")
    return a


def esize(dtype: int) -> int:
    return 1 if dtype == FP8 else 2


# ------------------------------------------------------------------ number formats
def decode_e4m3fn(codes) -> np.ndarray:
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    out = np.empty(c.shape, np.float64)
    _L().or_decode_e4m3fn_array(_ptr(c), c.size, _ptr(out))
    return out


def decode_bf16(bits) -> np.ndarray:
    c = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty(c.shape, np.float32)
    _L().or_decode_bf16_array(_ptr(c), c.size, _ptr(out))
    return out


def bf16_rne(x) -> np.ndarray:
    f = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(f.shape, np.uint16)
    _L().or_bf16_rne_array(_ptr(f), f.size, _ptr(out))
    return out


def decode(codes, dtype) -> np.ndarray:
    return decode_e4m3fn(codes) if dtype == FP8 else decode_bf16(codes).astype(np.float64)


# ------------------------------------------------------------------ format
def layout(N: int, K: int, axis: int, dense_begin: int) -> dict:
    out = np.zeros(6, np.int64)
    if _L().or_layout(N, K, axis, dense_begin, _ptr(out)):
        raise ValueError("bad split")
    sr, vld, mld, dr, dld, sc = (int(v) for v in out)
    return {"sparse_rows": sr, "values_ld": vld, "meta_ld": mld, "dense_rows": dr, "dense_ld": dld,
            "sparse_cols": sc}


def compress(W, mask, dtype: int, axis: int, dense_begin: int):
    """Canonical 2:4 compression.  Returns (values, meta, dense, bad_groups)."""
    W = _codes(W, dtype)
    N, K = W.shape
    lay = layout(N, K, axis, dense_begin)
    vt = np.uint8 if dtype == FP8 else np.uint16
    values = np.zeros((lay["sparse_rows"], lay["values_ld"]), vt)
    meta = np.zeros((lay["sparse_rows"], lay["meta_ld"]), np.uint32)
    dense = np.zeros((lay["dense_rows"], lay["dense_ld"]), vt)
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    if m is not None and m.shape != W.shape:
        raise ValueError("mask shape")
    bad = _L().or_compress(_ptr(W), _ptr(m), N, K, esize(dtype), axis, dense_begin, _ptr(values), _ptr(meta),
                           _ptr(dense))
    if bad < 0:
        raise ValueError("sparse region K must be a multiple of 4")
    return values, meta, dense, int(bad)


def decompress(values, meta, dense, N: int, K: int, dtype: int, axis: int, dense_begin: int) -> np.ndarray:
    vt = np.uint8 if dtype == FP8 else np.uint16
    lay = layout(N, K, axis, dense_begin)
    values = np.ascontiguousarray(values, dtype=vt).reshape(lay["sparse_rows"], lay["values_ld"])
    meta = np.ascontiguousarray(meta, dtype=np.uint32).reshape(lay["sparse_rows"], lay["meta_ld"])
    dense = np.ascontiguousarray(dense, dtype=vt).reshape(lay["dense_rows"], lay["dense_ld"])
    W = np.empty((N, K), vt)
    if _L().or_decompress(_ptr(values), _ptr(meta), _ptr(dense), N, K, esize(dtype), axis, dense_begin, _ptr(W)):
        raise ValueError("bad split")
    return W


# ------------------------------------------------------------------ GEMM
def gemm(X, W, dtype: int, sw=None, sx=None) -> dict:
    """Y = X W^T with fp32 ascending-k accumulation and the fp32 scale epilogue.

    Returns {"acc": fp32 M x N, "y_f32": fp32 M x N, "y_bf16": uint16 M x N}."""
    X = _codes(X, dtype)
    W = _codes(W, dtype)
    M, K = X.shape
    N, K2 = W.shape
    if K != K2:
        raise ValueError("K mismatch")
    swa = None if sw is None else np.ascontiguousarray(sw, dtype=np.float32)
    sxa = None if sx is None else np.ascontiguousarray(sx, dtype=np.float32)
    acc = np.empty((M, N), np.float32)
    yf = np.empty((M, N), np.float32)
    yb = np.empty((M, N), np.uint16)
    rc = _L().or_gemm_f32(_ptr(X), _ptr(W), M, N, K, dtype, _ptr(swa), _ptr(sxa), _ptr(acc), _ptr(yf), _ptr(yb))
    if rc:
        raise RuntimeError(f"or_gemm_f32 failed {rc}")
    return {"acc": acc, "y_f32": yf, "y_bf16": yb}


def gemm_f64(X, W, dtype: int, sw=None, sx=None) -> dict:
    """Same contraction in fp64; also returns sum_k |x w| for error bounds."""
    X = _codes(X, dtype)
    W = _codes(W, dtype)
    M, K = X.shape
    N, _ = W.shape
    swa = None if sw is None else np.ascontiguousarray(sw, dtype=np.float32)
    sxa = None if sx is None else np.ascontiguousarray(sx, dtype=np.float32)
    acc = np.empty((M, N), np.float64)
    y = np.empty((M, N), np.float64)
    ad = np.empty((M, N), np.float64)
    rc = _L().or_gemm_f64(_ptr(X), _ptr(W), M, N, K, dtype, _ptr(swa), _ptr(sxa), _ptr(acc), _ptr(y), _ptr(ad))
    if rc:
        raise RuntimeError(f"or_gemm_f64 failed {rc}")
    return {"acc": acc, "y": y, "abs_dot": ad}


def spense_gemm(X, values, meta, dense, N: int, K: int, dtype: int, axis: int, dense_begin: int, sw=None,
                sx=None) -> dict:
    """The whole layer from the packed format: decompress, then the plain GEMM."""
    W = decompress(values, meta, dense, N, K, dtype, axis, dense_begin)
    return gemm(X, W, dtype, sw, sx)


# ------------------------------------------------------------------ activation quantisation
def encode_e4m3fn(x) -> np.ndarray:
    """fp32 values -> e4m3fn codes: nearest, ties to an even mantissa, saturating to
    +-448 (the definition the GLU-MLP steps use; sec. 3.3.1, Eq. (4))."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(f.shape, np.uint8)
    _L().or_encode_e4m3fn_array(_ptr(f), f.size, _ptr(out))
    return out


def quantize_rows(a):
    """Per-token fp8 quantisation of an M x K fp32 matrix: scale = absmax / 448 (1.0 for a
    zero row) and codes = e4m3fn(a / scale), all in fp32.  Returns (codes, scales)."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    M, K = f.shape
    q = np.empty((M, K), np.uint8)
    s = np.empty(M, np.float32)
    _L().or_quantize_rows(_ptr(f), M, K, K, _ptr(q), _ptr(s))
    return q, s


def glu_f64(g, u) -> np.ndarray:
    """h = u * silu(g) = u * g / (1 + exp(-g)) in fp64 (the GLU of the MLP, sec. 3.3.1
    Eq. (4), with sigma read as SiLU)."""
    ga = np.ascontiguousarray(g, dtype=np.float64)
    ua = np.ascontiguousarray(u, dtype=np.float64)
    if ga.shape != ua.shape:
        raise ValueError("g and u differ in shape")
    h = np.empty(ga.shape, np.float64)
    _L().or_glu_f64(_ptr(ga), _ptr(ua), ga.size, _ptr(h))
    return h


def mlp(X, sx, gate, up, down, dtype=FP8):
    """The GLU MLP of sec. 3.3.1 Eq. (4) through the Spense format, step by step:
    G = gate(X), U = up(X) (output-split GEMMs), H = U * silu(G), (Hq, sh) = per-token fp8
    quantisation of H (from the fp32 rounding of the fp64 H), Y = down(Hq) (input-split).
    gate / up / down are (values, meta, dense, N, K, axis, dense_begin, sw) tuples.
    Returns a dict with the intermediate results."""
    def run(Xq, s, w, out_f64=False):
        v, m, d, N, K, axis, db, sw = w
        Wd = decompress(v, m, d, N, K, dtype, axis, db)
        return gemm_f64(Xq, Wd, dtype, sw, s)["y"] if out_f64 else gemm(Xq, Wd, dtype, sw, s)["y_f32"]
    G = run(X, sx, gate, True)
    U = run(X, sx, up, True)
    H = glu_f64(G, U)
    Hq, sh = quantize_rows(H.astype(np.float32))
    Y = run(Hq, sh, down)
    return {"G": G, "U": U, "H": H, "Hq": Hq, "sh": sh, "Y": Y}


# ------------------------------------------------------------------ dense-index selection
def index_scores(Wg, Wu, Wd, h_in, h_mid, eps: float = 1e-8) -> dict:
    """SpenseGPT+ priority of each intermediate index (sec. 3.3.1: the Wanda-style
    element score S_ij = |W_ij| sqrt(H_jj) of Eq. (8) averaged per index, Eq. (9), each
    projection's score vector normalised by its mean, Eq. (10), the three summed,
    Eq. (11)).  Wg, Wu: I x D (index i = row i),
    Wd: D x I (index i = column i); h_in: diag(X^T X) of the MLP input (D), h_mid: the
    same for the down projection's input (I).  Reading for down: index i's score is the
    mean over the column's entries, |Wd[n, i]| sqrt(h_mid[i]).  fp64, plain loops over
    numpy rows.  Returns the three raw score vectors and their normalised sum."""
    Wg = np.asarray(Wg, np.float64)
    Wu = np.asarray(Wu, np.float64)
    Wd = np.asarray(Wd, np.float64)
    I, D = Wg.shape
    sx = np.sqrt(np.asarray(h_in, np.float64))
    sm = np.sqrt(np.asarray(h_mid, np.float64))
    s_gate = np.array([np.sum(np.abs(Wg[i]) * sx) / D for i in range(I)])
    s_up = np.array([np.sum(np.abs(Wu[i]) * sx) / D for i in range(I)])
    s_down = np.array([np.sum(np.abs(Wd[:, i])) * sm[i] / Wd.shape[0] for i in range(I)])

    def norm(v):
        return v / (np.sum(v) / v.size + eps)

    return {"gate": s_gate, "up": s_up, "down": s_down, "total": norm(s_gate) + norm(s_up) + norm(s_down)}


def dense_index_permutation(total, n_dense: int) -> dict:
    """TopK of the priorities, Eq. (12) (the n_dense largest; ties keep the lower index) and the
    permutation that moves them to the back (sec. 3.3.1): perm[new] = old, the sparse
    indices first and the dense ones last, each in ascending order."""
    t = np.asarray(total, np.float64)
    order = np.argsort(-t, kind="stable")  # a library sort; stable keeps lower indices first on ties
    dense = np.sort(order[:n_dense])
    is_dense = np.zeros(t.size, bool)
    is_dense[dense] = True
    perm = np.concatenate([np.flatnonzero(~is_dense), dense]).astype(np.int32)
    return {"dense": dense, "perm": perm}



# ------------------------------------------------------------------ SparseGPT 2:4 with a protected dense region
def obs_damp(H, percdamp: float = 0.01):
    """Conditioning of the Hessian H = X^T X before the OBS sweep (sec. 3.1.2 uses
    SparseGPT; the paper gives no constants, so SparseGPT's published ones are read in):
    a column that no calibration input excites (H_jj = 0) gets H_jj = 1 and is reported as
    dead (its weights are zeroed); then lambda = percdamp * mean(diag H) is added to the
    diagonal.  Returns (damped H, dead mask).  fp64."""
    H = np.array(H, np.float64, copy=True)
    dead = np.diag(H) == 0
    idx = np.flatnonzero(dead)
    H[idx, idx] = 1.0
    H[np.diag_indices_from(H)] += percdamp * np.mean(np.diag(H))
    return H, dead


def obs_factor(H, percdamp: float = 0.01):
    """The factor the column sweep reads: U upper triangular with Hd^{-1} = U^T U, Hd the
    damped Hessian.  Row j of U times U_jj is row j of the inverse Hessian of the columns
    j..K-1 (those not yet frozen when column j is processed), so U_jj^2 is the OBS
    denominator [H^{-1}]_mm of Eq. (3) for column j and U[j, j:] / U_jj its compensation
    direction.  Library primitives: the inverse and the Cholesky factor.  Returns (U, dead)."""
    Hd, dead = obs_damp(H, percdamp)
    U = np.linalg.cholesky(np.linalg.inv(Hd)).T
    return U, dead


def obs_prune_24(W, H, dense_begin: int, percdamp: float = 0.01, factor=None) -> dict:
    """SparseGPT 2:4 pruning of W (N x K) with the trailing columns [dense_begin, K) kept
    dense (sec. 3.1.2, Eqs. (2)-(3); sec. 3.3.1: the dense region placed last so that it
    stays a compensation buffer).  Columns 0 .. dense_begin-1 are processed left to right
    and frozen once processed.  At the first column of each group of four, every row
    prunes the two weights of the group with the smallest OBS error w_m^2 / [H^{-1}]_mm
    (Eq. (3); the denominator is U_mm^2, the one column m has when it is processed; the
    weights as updated so far; ties prune the lower index).  Each processed column's
    change (w_j - q_j) is compensated on the columns not yet processed along Eq. (3)'s
    direction: W[:, j:] -= ((w_j - q_j) / U_jj) U[j, j:].  The dense columns are never
    pruned and absorb the compensation.  Full updates every column (no blocking).  fp64.
    factor: (U, dead) from obs_factor of the same H and percdamp, to reuse it over row
    samples.  Returns the pruned and compensated W, the kept mask (True = kept), the OBS
    error each 2:4 weight had when its group was chosen ("err", N x dense_begin) and U."""
    W = np.array(W, np.float64, copy=True)
    N, K = W.shape
    if dense_begin % 4 or not 0 <= dense_begin <= K:
        raise ValueError("dense_begin must be a multiple of 4 in [0, K]")
    U, dead = obs_factor(H, percdamp) if factor is None else factor
    W[:, dead] = 0.0
    keep = np.ones((N, K), bool)
    errs = np.zeros((N, dense_begin))
    rows = np.arange(N)[:, None]
    for j in range(dense_begin):
        if j % 4 == 0:
            err = W[:, j:j + 4] ** 2 / np.diag(U)[j:j + 4] ** 2
            errs[:, j:j + 4] = err
            order = np.argsort(err, axis=1, kind="stable")  # a library sort; stable: lower index first on ties
            keep[rows, j + order[:, :2]] = False
        q = np.where(keep[:, j], W[:, j], 0.0)
        e = (W[:, j] - q) / U[j, j]
        W[:, j + 1:] -= np.outer(e, U[j, j + 1:])
        W[:, j] = q
    return {"W": W, "keep": keep, "err": errs, "U": U, "dead": dead}


def reconstruction_loss(W, W_hat, H) -> float:
    """The layer reconstruction error of Eq. (2), ||X W^T - X W_hat^T||_F^2, written with
    H = X^T X: sum over rows of (w - w_hat)^T H (w - w_hat).  fp64."""
    D = np.asarray(W, np.float64) - np.asarray(W_hat, np.float64)
    return float(np.einsum("nk,kl,nl->", D, np.asarray(H, np.float64), D))
