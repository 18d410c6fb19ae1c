"""Seeded synthetic inputs for the Spense linear layer.

This module is the only code shared by the GPU tests and the CPU oracle.  It holds no
part of the method's arithmetic: it draws weights and activations, prunes the sparse
region to 2:4 by magnitude (the mask is an input of the compressor), computes
per-output-channel and per-token absmax scales, and quantises with torch's own
float8_e4m3fn / bfloat16 converters.

Workloads are synthetic stand-ins for the paper's Qwen3-32B and Seed-OSS-36B layers
(sec. 4.1): their weights, calibration set and benchmarks are not available, and the
GEMM's timing does not depend on the values.  The value distributions follow the
workload descriptions: W ~ N(0, 0.02); X ~ N(0, 1) for the up/gate family, heavy
tailed (Student-t with 4 degrees of freedom) for the down projection.

Every tensor comes from its own stream ``default_rng(SeedSequence([0, cfg, mat, role]))``.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np
import torch

FP8 = "fp8"
BF16 = "bf16"
OUTPUT = "output"  # split along N (gate/up style)
INPUT = "input"  # split along K (down style)
FP8_MAX = 448.0

ROLE_W, ROLE_X, ROLE_MASK = 0, 1, 2


def rng(cfg: int, mat: int, role: int, base: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([base, cfg, mat, role]))


def sha256(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


# ------------------------------------------------------------------ splits
def split_point(N: int, K: int, axis: str, dense_frac: float, granule: int = 32) -> int:
    """First index of the dense region along the split axis.

    The dense region is the trailing ~dense_frac of the axis; the sparse extent is
    rounded to a multiple of ``granule`` along K (input-split) or 16 along N."""
    extent = N if axis == OUTPUT else K
    g = 16 if axis == OUTPUT else granule
    sparse = extent - int(round(dense_frac * extent))
    sparse = int(round(sparse / g)) * g
    return max(0, min(extent, sparse))


# ------------------------------------------------------------------ draws
def draw_weight(r: np.random.Generator, N: int, K: int, std: float = 0.02) -> np.ndarray:
    return (r.standard_normal((N, K), dtype=np.float32) * np.float32(std)).astype(np.float32)


def draw_x(r: np.random.Generator, M: int, K: int, dist: str = "normal") -> np.ndarray:
    if dist == "normal":
        return r.standard_normal((M, K), dtype=np.float32)
    if dist == "student_t4":
        z = r.standard_normal((M, K), dtype=np.float32)
        chi2 = np.zeros((M, K), np.float32)
        for _ in range(4):
            g = r.standard_normal((M, K), dtype=np.float32)
            chi2 += g * g
        return (z / np.sqrt(chi2 / np.float32(4.0))).astype(np.float32)
    raise ValueError(dist)


def magnitude_mask_24(W: np.ndarray, axis: str, dense_begin: int) -> np.ndarray:
    """uint8 N x K mask: in the sparse region keep the 2 largest |w| of every aligned
    group of 4 along K (ties keep the lower index); the dense region is all ones."""
    N, K = W.shape
    mask = np.ones((N, K), np.uint8)
    if axis == OUTPUT:
        reg = W[:dense_begin]
    else:
        reg = W[:, :dense_begin]
    rows, cols = reg.shape
    if rows == 0 or cols == 0:
        return mask
    a = np.abs(reg.astype(np.float32)).reshape(rows, cols // 4, 4)
    rank = np.zeros(a.shape, np.int8)
    for i in range(4):
        for j in range(4):
            if i == j:
                continue
            beats = a[..., j] > a[..., i]
            if j < i:
                beats |= a[..., j] == a[..., i]
            rank[..., i] += beats
    keep = (rank < 2).astype(np.uint8).reshape(rows, cols)
    if axis == OUTPUT:
        mask[:dense_begin] = keep
    else:
        mask[:, :dense_begin] = keep
    return mask


def random_mask_24(r: np.random.Generator, N: int, K: int, axis: str, dense_begin: int,
                   allow_fewer: bool = True) -> np.ndarray:
    """Random valid 2:4 mask (also groups with 0 or 1 kept when allow_fewer)."""
    mask = np.ones((N, K), np.uint8)
    rows = dense_begin if axis == OUTPUT else N
    cols = K if axis == OUTPUT else dense_begin
    if rows == 0 or cols == 0:
        return mask
    pats = [(0, 1), (0, 2), (0, 3), (1, 2), (1, 3), (2, 3)]
    table = np.zeros((len(pats) + (5 if allow_fewer else 0), 4), np.uint8)
    for t, (a, b) in enumerate(pats):
        table[t, a] = table[t, b] = 1
    if allow_fewer:
        for t in range(4):
            table[len(pats) + t, t] = 1
        # last row: nothing kept
    ch = r.integers(0, table.shape[0], size=(rows, cols // 4))
    keep = table[ch].reshape(rows, cols)
    if axis == OUTPUT:
        mask[:dense_begin] = keep
    else:
        mask[:, :dense_begin] = keep
    return mask


# ------------------------------------------------------------------ quantisation
def absmax_scale(A: np.ndarray) -> np.ndarray:
    """Per-row fp32 absmax / 448 (1.0 for an all-zero row)."""
    s = (np.abs(A).max(axis=1) if A.shape[1] else np.zeros(A.shape[0], np.float32)).astype(np.float32)
    s = s / np.float32(FP8_MAX)
    s[s == 0] = 1.0
    return s.astype(np.float32)


def to_e4m3fn(A: np.ndarray) -> np.ndarray:
    """fp32 -> e4m3fn codes via torch (round to nearest even), saturated to +-448."""
    t = torch.from_numpy(np.ascontiguousarray(A, dtype=np.float32)).clamp_(-FP8_MAX, FP8_MAX)
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy().copy()


def to_bf16(A: np.ndarray) -> np.ndarray:
    """fp32 -> bfloat16 bit patterns via torch (round to nearest even)."""
    t = torch.from_numpy(np.ascontiguousarray(A, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def quantize_rows_fp8(A: np.ndarray):
    s = absmax_scale(A)
    return to_e4m3fn(A / s[:, None]), s


# ------------------------------------------------------------------ whole matrices
@dataclass
class Matrix:
    name: str
    N: int
    K: int
    axis: str
    dense_begin: int
    dtype: str
    W: np.ndarray  # codes N x K (uint8 fp8 / uint16 bf16), dense region untouched
    mask: np.ndarray  # uint8 N x K
    sw: np.ndarray | None  # fp32 N (None for bf16)
    meta: dict = field(default_factory=dict)


def make_matrix(cfg: int, mat: int, name: str, N: int, K: int, axis: str, dense_frac: float, dtype: str,
                dense_begin: int | None = None) -> Matrix:
    r = rng(cfg, mat, ROLE_W)
    Wf = draw_weight(r, N, K)
    db = split_point(N, K, axis, dense_frac) if dense_begin is None else dense_begin
    if dtype == FP8:
        mask = magnitude_mask_24(Wf, axis, db)  # prune on the fp32 draw, then quantise
        codes, sw = quantize_rows_fp8(Wf)
    else:
        codes = to_bf16(Wf)
        vals = torch.from_numpy(codes.view(np.int16)).view(torch.bfloat16).float().numpy()
        mask = magnitude_mask_24(vals, axis, db)  # prune on the bf16 values
        sw = None
    return Matrix(name, N, K, axis, db, dtype, codes, mask, sw)


def make_x(cfg: int, mat: int, M: int, K: int, dtype: str, dist: str = "normal"):
    """Returns (codes M x K, per-token scale or None)."""
    Xf = draw_x(rng(cfg, mat, ROLE_X), M, K, dist)
    if dtype == FP8:
        return quantize_rows_fp8(Xf)
    return to_bf16(Xf), None


# exact small integers: every partial sum of K products of values in [-3, 3] is an
# integer of magnitude <= 9K < 2^24 for K <= 1.8M, so fp32 sums are exact in any order
_FP8_INT = {v: c for v, c in zip(range(-3, 4), [0xC4, 0xC0, 0xB8, 0x00, 0x38, 0x40, 0x44])}
_BF16_INT = {v: c for v, c in zip(range(-3, 4), [0xC040, 0xC000, 0xBF80, 0x0000, 0x3F80, 0x4000, 0x4040])}


def int_codes(vals: np.ndarray, dtype: str) -> np.ndarray:
    tab = _FP8_INT if dtype == FP8 else _BF16_INT
    lut = np.array([tab[v] for v in range(-3, 4)], np.uint8 if dtype == FP8 else np.uint16)
    return lut[np.asarray(vals, np.int64) + 3]


def make_exact_int(cfg: int, mat: int, M: int, N: int, K: int, axis: str, dense_begin: int, dtype: str):
    """Integer-valued inputs in [-3, 3] with power-of-two scales (exact epilogue)."""
    r = rng(cfg, mat, ROLE_MASK, base=7)
    Wv = r.integers(-3, 4, size=(N, K))
    Xv = r.integers(-3, 4, size=(M, K))
    mask = random_mask_24(r, N, K, axis, dense_begin)
    sw = (2.0 ** r.integers(-3, 2, size=N)).astype(np.float32) if dtype == FP8 else None
    sx = (2.0 ** r.integers(-3, 2, size=M)).astype(np.float32) if dtype == FP8 else None
    return int_codes(Wv, dtype), mask, int_codes(Xv, dtype), sw, sx


# ------------------------------------------------------------------ the five workloads
# (name, N, K, axis) per matrix; dense fraction 0.25 unless swept.
QWEN3_32B_LAYER = [("q", 8192, 5120, OUTPUT), ("k", 1024, 5120, OUTPUT), ("v", 1024, 5120, OUTPUT),
                   ("o", 5120, 8192, INPUT), ("gate", 25600, 5120, OUTPUT), ("up", 25600, 5120, OUTPUT),
                   ("down", 5120, 25600, INPUT)]
SEED_OSS_36B_LAYER = [("q", 10240, 5120, OUTPUT), ("k", 1024, 5120, OUTPUT), ("v", 1024, 5120, OUTPUT),
                      ("o", 5120, 10240, INPUT), ("gate", 27648, 5120, OUTPUT), ("up", 27648, 5120, OUTPUT),
                      ("down", 5120, 27648, INPUT)]

WORKLOADS = {
    1: {"name": "tiny linear 256x512 bf16", "dtype": BF16, "mats": [("w", 256, 512, OUTPUT), ("w", 256, 512, INPUT)],
        "ms": [1], "dense_fracs": [0.25], "xdist": "normal"},
    2: {"name": "qwen3-32b-like gate/up 25600x5120 fp8", "dtype": FP8, "mats": [("gate_up", 25600, 5120, OUTPUT)],
        "ms": [1, 8, 32, 64], "dense_fracs": [0.25], "xdist": "normal"},
    3: {"name": "qwen3-32b-like down 5120x25600 fp8", "dtype": FP8, "mats": [("down", 5120, 25600, INPUT)],
        "ms": [1, 16, 64], "dense_fracs": [0.0, 0.125, 0.25, 0.5, 1.0], "xdist": "student_t4"},
    4: {"name": "qwen3-32b-like layer linears fp8", "dtype": FP8, "mats": QWEN3_32B_LAYER, "ms": [64],
        "dense_fracs": [0.25], "xdist": "normal"},
    5: {"name": "seed-oss-36b-like layer linears fp8", "dtype": FP8, "mats": SEED_OSS_36B_LAYER,
        "ms": [1, 4, 16, 64, 256, 2048], "dense_fracs": [0.25], "xdist": "normal"},
}
