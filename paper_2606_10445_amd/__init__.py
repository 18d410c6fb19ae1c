"""Python binding of libspense: the Spense hybrid 2:4-sparse / dense linear layer on
MI355X (gfx950).

Argument marshalling only.  Every step of the computation runs in the HIP kernels of
``libspense.so``; there is no fallback: importing this package without the built
library raises.  PyTorch is used for device memory and streams.

Low-level functions carry the C names (``spense_layout``, ``spense_compress``,
``spense_decompress``, ``spense_gemm``, ``spense_dense_gemm``, ...) and take raw
pointers; ``PackedWeight``, ``compress``, ``gemm`` and ``dense_gemm`` wrap them for torch
tensors.  Paper: SpenseGPT, sec. 3.1.1 (2:4 storage) and sec. 3.2 (Spense format).
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspense.so")

SPENSE_OK = 0
SPENSE_ERR_ARG = -1
SPENSE_ERR_ALIGN = -2
SPENSE_ERR_MASK = -3
SPENSE_ERR_WS = -4
SPENSE_ERR_HIP = -5
SPENSE_ERR_DEVICE = -6
SPENSE_ERR_NUMERIC = -7
SPENSE_FP8_E4M3FN = 1
SPENSE_BF16 = 2
SPENSE_F32 = 3
SPENSE_SPLIT_OUTPUT = 0
SPENSE_SPLIT_INPUT = 1
SPENSE_OUT_BF16 = 0
SPENSE_OUT_F32 = 1
SPENSE_LAYOUT_ROWMAJOR = 0
SPENSE_LAYOUT_TILED = 1
SPENSE_NOALLOC_SCRATCH_BYTES = 16 << 20

EXPORTS = ["spense_abi_version", "spense_set_log", "spense_last_error", "spense_layout", "spense_tiled_layout",
           "spense_compress_workspace_size", "spense_compress", "spense_decompress", "spense_tile",
           "spense_gemm_workspace_size", "spense_gemm", "spense_dense_gemm_workspace_size", "spense_dense_gemm",
           "spense_quantize_fp8", "spense_glu_quantize_fp8", "spense_index_scores", "spense_dense_permutation",
           "spense_gather_rows", "spense_gather_cols", "spense_obs_factor_workspace_size", "spense_obs_factor",
           "spense_obs_prune_workspace_size", "spense_obs_prune_24", "spense_gemm_grouped", "spense_gemm_glu",
           "spense_gemm_glu_fp8_workspace_size", "spense_gemm_glu_fp8", "spense_gemm_planned_workspace_size",
           "spense_gemm_planned", "spense_gemm_noalloc"]


class SpenseError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"spense error {code}: {msg}")
        self.code = code


class spense_layout_t(ctypes.Structure):
    _fields_ = [("sparse_rows", ctypes.c_int64), ("sparse_cols", ctypes.c_int64), ("values_ld", ctypes.c_int64),
                ("meta_ld", ctypes.c_int64), ("dense_rows", ctypes.c_int64), ("dense_cols", ctypes.c_int64),
                ("dense_ld", ctypes.c_int64), ("values_bytes", ctypes.c_size_t), ("meta_bytes", ctypes.c_size_t),
                ("dense_bytes", ctypes.c_size_t)]


class spense_tiled_layout_t(ctypes.Structure):
    _fields_ = [("sparse_tiles", ctypes.c_int64), ("sparse_chunks", ctypes.c_int64), ("dense_tiles", ctypes.c_int64),
                ("dense_chunks", ctypes.c_int64), ("values_bytes", ctypes.c_size_t), ("meta_bytes", ctypes.c_size_t),
                ("dense_bytes", ctypes.c_size_t)]


class spense_packed_t(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("split", ctypes.c_int32), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("dense_begin", ctypes.c_int64), ("values", ctypes.c_void_p), ("values_ld", ctypes.c_int64),
                ("meta", ctypes.c_void_p), ("meta_ld", ctypes.c_int64), ("dense", ctypes.c_void_p),
                ("dense_ld", ctypes.c_int64), ("layout", ctypes.c_int32)]


class spense_plan_override_t(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32), ("row_tiles", ctypes.c_int32), ("waves", ctypes.c_int32),
                ("act_tiles", ctypes.c_int32), ("ksplit", ctypes.c_int32), ("waves_used", ctypes.c_int32),
                ("waves_used_dense", ctypes.c_int32), ("waves_used_24", ctypes.c_int32),
                ("block_order", ctypes.c_int32), ("xcd_order", ctypes.c_int32), ("u8", ctypes.c_int32),
                ("half_row_blocks", ctypes.c_int32), ("resident_x", ctypes.c_int32)]


KERNEL_KSPLIT, KERNEL_ROWS, KERNEL_LARGE_M = 1, 2, 3


def plan_override(**kw) -> spense_plan_override_t:
    """A spense_plan_override_t with the given fields forced and the rest left to the
    planner (block_order, xcd_order and half_row_blocks default to -1)."""
    p = spense_plan_override_t(block_order=-1, xcd_order=-1, half_row_blocks=-1)
    for k, v in kw.items():
        if not hasattr(p, k):
            raise TypeError(f"unknown plan field {k}")
        setattr(p, k, int(v))
    return p


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_10445_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    p, i64, i32, u32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_size_t
    P = ctypes.POINTER
    sig = {
        "spense_abi_version": (ctypes.c_int, []),
        "spense_set_log": (ctypes.c_int, [i32]),
        "spense_last_error": (ctypes.c_char_p, []),
        "spense_layout": (ctypes.c_int, [i64, i64, i32, i32, i64, P(spense_layout_t)]),
        "spense_tiled_layout": (ctypes.c_int, [i64, i64, i32, i32, i64, P(spense_tiled_layout_t)]),
        "spense_tile": (ctypes.c_int, [P(spense_packed_t), P(spense_packed_t), p]),
        "spense_compress_workspace_size": (sz, []),
        "spense_compress": (ctypes.c_int, [p, i64, p, i64, P(spense_packed_t), P(i64), p, sz, p]),
        "spense_decompress": (ctypes.c_int, [P(spense_packed_t), p, i64, p]),
        "spense_gemm_workspace_size": (sz, [i64, P(spense_packed_t)]),
        "spense_gemm": (ctypes.c_int, [p, i64, i64, P(spense_packed_t), p, p, p, i64, u32, p, sz, p]),
        "spense_dense_gemm_workspace_size": (sz, [i64, i64, i64, i32]),
        "spense_dense_gemm": (ctypes.c_int, [p, i64, i64, p, i64, i64, i64, i32, p, p, p, i64, u32, p, sz, p]),
        "spense_quantize_fp8": (ctypes.c_int, [p, i32, i64, i64, i64, p, i64, p, p]),
        "spense_glu_quantize_fp8": (ctypes.c_int, [p, i64, p, i64, i32, i64, i64, p, i64, p, p]),
        "spense_index_scores": (ctypes.c_int, [p, p, i64, p, i64, i32, i64, i64, p, p, ctypes.c_float, p, p, p]),
        "spense_dense_permutation": (ctypes.c_int, [p, i64, i64, p, p, p]),
        "spense_gather_rows": (ctypes.c_int, [p, i64, p, i64, i64, i64, p, p]),
        "spense_gather_cols": (ctypes.c_int, [p, i64, p, i64, i64, i64, i32, p, p]),
        "spense_obs_factor_workspace_size": (sz, [i64]),
        "spense_obs_factor": (ctypes.c_int, [p, i64, i64, ctypes.c_float, p, i64, p, p, sz, p]),
        "spense_obs_prune_workspace_size": (sz, [i64]),
        "spense_obs_prune_24": (ctypes.c_int, [p, i64, i64, i64, p, i64, p, i64, p, i64, p, sz, p]),
        "spense_gemm_grouped": (ctypes.c_int, [p, i64, i64, i32, p, p, p, p, p, u32, p]),
        "spense_gemm_glu": (ctypes.c_int, [p, i64, i64, p, p, p, p, p, p, i64, p]),
        "spense_gemm_glu_fp8_workspace_size": (ctypes.c_size_t, [i64, i64]),
        "spense_gemm_glu_fp8": (ctypes.c_int, [p, i64, i64, p, p, p, p, p, p, i64, p, p, ctypes.c_size_t, p]),
        "spense_gemm_planned_workspace_size": (sz, [i64, P(spense_packed_t), P(spense_plan_override_t)]),
        "spense_gemm_noalloc": (ctypes.c_int, [p, i64, i64, P(spense_packed_t), p, p, p, i64, u32, p]),
        "spense_gemm_planned": (ctypes.c_int, [p, i64, i64, P(spense_packed_t), p, p, p, i64, u32, p, sz,
                                               P(spense_plan_override_t), p]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()


# ------------------------------------------------------------------ raw C calls
def spense_abi_version() -> int:
    return _lib.spense_abi_version()


def spense_set_log(level: int) -> int:
    return _lib.spense_set_log(level)


def spense_last_error() -> str:
    return _lib.spense_last_error().decode()


def _check(rc: int):
    if rc != SPENSE_OK:
        raise SpenseError(rc, spense_last_error())


def spense_layout(N: int, K: int, dtype: int, split: int, dense_begin: int) -> spense_layout_t:
    L = spense_layout_t()
    _check(_lib.spense_layout(N, K, dtype, split, dense_begin, ctypes.byref(L)))
    return L


def spense_tiled_layout(N: int, K: int, dtype: int, split: int, dense_begin: int) -> spense_tiled_layout_t:
    T = spense_tiled_layout_t()
    _check(_lib.spense_tiled_layout(N, K, dtype, split, dense_begin, ctypes.byref(T)))
    return T


def spense_tile(src: spense_packed_t, dst: spense_packed_t, stream) -> int:
    return _lib.spense_tile(ctypes.byref(src), ctypes.byref(dst), stream)


def spense_compress_workspace_size() -> int:
    return _lib.spense_compress_workspace_size()


def spense_compress(W, ldw, mask, ldm, packed: spense_packed_t, ws, ws_bytes, stream) -> tuple[int, int]:
    """Returns (status, bad_groups); does not raise so callers can inspect the count."""
    bad = ctypes.c_int64(0)
    rc = _lib.spense_compress(W, ldw, mask, ldm, ctypes.byref(packed), ctypes.byref(bad), ws, ws_bytes, stream)
    return rc, bad.value


def spense_decompress(packed: spense_packed_t, W_out, ldw, stream) -> int:
    return _lib.spense_decompress(ctypes.byref(packed), W_out, ldw, stream)


def spense_gemm_workspace_size(M: int, packed: spense_packed_t) -> int:
    return _lib.spense_gemm_workspace_size(M, ctypes.byref(packed))


def spense_gemm(X, M, ldx, packed: spense_packed_t, w_scale, x_scale, Y, ldy, out_flags, ws, ws_bytes,
                stream) -> int:
    return _lib.spense_gemm(X, M, ldx, ctypes.byref(packed), w_scale, x_scale, Y, ldy, out_flags, ws, ws_bytes,
                            stream)


def spense_gemm_planned_workspace_size(M: int, packed: spense_packed_t, plan) -> int:
    return _lib.spense_gemm_planned_workspace_size(M, ctypes.byref(packed), None if plan is None else ctypes.byref(plan))


def spense_gemm_planned(X, M, ldx, packed: spense_packed_t, w_scale, x_scale, Y, ldy, out_flags, ws, ws_bytes, plan,
                        stream) -> int:
    return _lib.spense_gemm_planned(X, M, ldx, ctypes.byref(packed), w_scale, x_scale, Y, ldy, out_flags, ws,
                                    ws_bytes, None if plan is None else ctypes.byref(plan), stream)


def spense_gemm_noalloc(X, M, ldx, packed: spense_packed_t, w_scale, x_scale, Y, ldy, out_flags, stream) -> int:
    return _lib.spense_gemm_noalloc(X, M, ldx, ctypes.byref(packed), w_scale, x_scale, Y, ldy, out_flags, stream)


def spense_dense_gemm_workspace_size(M: int, N: int, K: int, dtype: int) -> int:
    return _lib.spense_dense_gemm_workspace_size(M, N, K, dtype)


def spense_dense_gemm(X, M, ldx, W, ldw, N, K, dtype, w_scale, x_scale, Y, ldy, out_flags, ws, ws_bytes,
                      stream) -> int:
    return _lib.spense_dense_gemm(X, M, ldx, W, ldw, N, K, dtype, w_scale, x_scale, Y, ldy, out_flags, ws, ws_bytes,
                                  stream)


def spense_quantize_fp8(src, src_type, M, K, ld_src, q, ldq, scales, stream) -> int:
    return _lib.spense_quantize_fp8(src, src_type, M, K, ld_src, q, ldq, scales, stream)


def spense_glu_quantize_fp8(g, ldg, u, ldu, gu_type, M, I, q, ldq, scales, stream) -> int:
    return _lib.spense_glu_quantize_fp8(g, ldg, u, ldu, gu_type, M, I, q, ldq, scales, stream)


def spense_index_scores(w_gate, w_up, ld_gu, w_down, ld_down, wtype, I, D, h_in, h_mid, eps, raw, total,
                        stream) -> int:
    return _lib.spense_index_scores(w_gate, w_up, ld_gu, w_down, ld_down, wtype, I, D, h_in, h_mid, eps, raw, total,
                                    stream)


def spense_dense_permutation(total, I, n_dense, flags, perm, stream) -> int:
    return _lib.spense_dense_permutation(total, I, n_dense, flags, perm, stream)


def spense_gather_rows(src, ld_src_b, dst, ld_dst_b, rows, row_bytes, perm, stream) -> int:
    return _lib.spense_gather_rows(src, ld_src_b, dst, ld_dst_b, rows, row_bytes, perm, stream)


def spense_gather_cols(src, ld_src, dst, ld_dst, rows, cols, elem_bytes, perm, stream) -> int:
    return _lib.spense_gather_cols(src, ld_src, dst, ld_dst, rows, cols, elem_bytes, perm, stream)


def spense_gemm_grouped(X, M, ldx, count, packed_array, w_scales_array, x_scale, Y_array, ldy_array, out_flags,
                        stream) -> int:
    return _lib.spense_gemm_grouped(X, M, ldx, count, packed_array, w_scales_array, x_scale, Y_array, ldy_array,
                                    out_flags, stream)


def spense_gemm_glu(X, M, ldx, gate, up, w_scale_gate, w_scale_up, x_scale, H, ldh, stream) -> int:
    return _lib.spense_gemm_glu(X, M, ldx, gate, up, w_scale_gate, w_scale_up, x_scale, H, ldh, stream)


def spense_gemm_glu_fp8_workspace_size(M: int, N: int) -> int:
    return _lib.spense_gemm_glu_fp8_workspace_size(M, N)


def spense_gemm_glu_fp8(X, M, ldx, gate, up, w_scale_gate, w_scale_up, x_scale, q, ldq, scales, ws, ws_bytes,
                        stream) -> int:
    return _lib.spense_gemm_glu_fp8(X, M, ldx, gate, up, w_scale_gate, w_scale_up, x_scale, q, ldq, scales, ws,
                                    ws_bytes, stream)


def spense_obs_factor_workspace_size(K: int) -> int:
    return _lib.spense_obs_factor_workspace_size(K)


def spense_obs_factor(H, ldh, K, percdamp, U, ldu, dead, ws, ws_bytes, stream) -> int:
    return _lib.spense_obs_factor(H, ldh, K, percdamp, U, ldu, dead, ws, ws_bytes, stream)


def spense_obs_prune_workspace_size(N: int) -> int:
    return _lib.spense_obs_prune_workspace_size(N)


def spense_obs_prune_24(W, ldw, N, K, U, ldu, dead, dense_begin, keep, ldk, ws, ws_bytes, stream) -> int:
    return _lib.spense_obs_prune_24(W, ldw, N, K, U, ldu, dead, dense_begin, keep, ldk, ws, ws_bytes, stream)


# ------------------------------------------------------------------ torch helpers
def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype in (torch.uint8, torch.float8_e4m3fn):
        return SPENSE_FP8_E4M3FN
    if t.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return SPENSE_BF16
    raise TypeError(f"unsupported weight dtype {t.dtype}")


def _storage_dtype(dtype: int):
    return torch.uint8 if dtype == SPENSE_FP8_E4M3FN else torch.int16


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _ptr(t):
    return None if t is None else t.data_ptr()


def _row_major(t: torch.Tensor, name: str):
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{name} must be a 2-D row-major tensor")


class Workspace:
    """A device buffer for spense_gemm's scratch, grown on demand and reused across calls
    (calls that overlap on one workspace race)."""

    def __init__(self, device):
        self.device = torch.device(device)
        self.buf = None

    def get(self, nbytes: int):
        if nbytes == 0:
            return None, 0
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.zeros(max(nbytes, 1 << 20), dtype=torch.uint8, device=self.device)
        return self.buf.data_ptr(), self.buf.numel()


_workspaces: dict = {}


def workspace_for(device) -> Workspace:
    d = torch.device(device)
    key = (d.type, d.index if d.index is not None else torch.cuda.current_device())
    if key not in _workspaces:
        _workspaces[key] = Workspace(torch.device("cuda", key[1]))
    return _workspaces[key]


class PackedWeight:
    """A weight in the Spense format: device buffers (values, meta, dense) + descriptor.
    ``kind`` is the storage order: SPENSE_LAYOUT_ROWMAJOR (as spense_compress writes it;
    ``layout`` is its spense_layout_t) or SPENSE_LAYOUT_TILED (``tiled`` is its
    spense_tiled_layout_t)."""

    def __init__(self, N, K, dtype, split, dense_begin, values, meta, dense, kind=SPENSE_LAYOUT_ROWMAJOR):
        self.N, self.K, self.dtype, self.split, self.dense_begin = N, K, dtype, split, dense_begin
        self.values, self.meta, self.dense = values, meta, dense
        self.kind = kind
        self.layout = spense_layout(N, K, dtype, split, dense_begin)
        self.tiled = spense_tiled_layout(N, K, dtype, split, dense_begin) if kind == SPENSE_LAYOUT_TILED else None
        self.desc = spense_packed_t(dtype, split, N, K, dense_begin, _ptr(values), self.layout.values_ld, _ptr(meta),
                                    self.layout.meta_ld, _ptr(dense), self.layout.dense_ld, kind)

    @classmethod
    def empty(cls, N, K, dtype, split, dense_begin, device="cuda"):
        L = spense_layout(N, K, dtype, split, dense_begin)
        st = _storage_dtype(dtype)
        values = torch.empty((L.sparse_rows, L.values_ld), dtype=st, device=device)
        meta = torch.empty((L.sparse_rows, L.meta_ld), dtype=torch.int32, device=device)
        dense = torch.empty((L.dense_rows, L.dense_ld), dtype=st, device=device)
        return cls(N, K, dtype, split, dense_begin, values, meta, dense)

    def weight_bytes(self) -> int:
        """Bytes of the three buffers (the tiled layout includes its zero padding)."""
        g = self.tiled if self.kind == SPENSE_LAYOUT_TILED else self.layout
        return g.values_bytes + g.meta_bytes + g.dense_bytes

    def clone(self) -> "PackedWeight":
        return PackedWeight(self.N, self.K, self.dtype, self.split, self.dense_begin, self.values.clone(),
                            self.meta.clone(), self.dense.clone(), self.kind)


def compress(W: torch.Tensor, mask: torch.Tensor | None, split: int, dense_begin: int) -> PackedWeight:
    """Pack a device weight (codes) into the Spense format with spense_compress."""
    _row_major(W, "W")
    dtype = _dtype_code(W)
    N, K = W.shape
    pw = PackedWeight.empty(N, K, dtype, split, dense_begin, device=W.device)
    if mask is not None:
        _row_major(mask, "mask")
        if mask.shape != W.shape or mask.dtype != torch.uint8 or mask.device != W.device:
            raise ValueError("mask must be a uint8 tensor of W's shape on W's device")
    ws = torch.zeros(spense_compress_workspace_size(), dtype=torch.uint8, device=W.device)
    rc, bad = spense_compress(_ptr(W), W.stride(0), _ptr(mask), 0 if mask is None else mask.stride(0), pw.desc,
                              ws.data_ptr(), ws.numel(), _stream(W.device))
    if rc != SPENSE_OK:
        err = SpenseError(rc, spense_last_error())
        err.bad_groups = bad
        raise err
    return pw


def tile(pw: PackedWeight) -> PackedWeight:
    """The same fp8 weight in the tiled execution layout (spense_tile)."""
    dev = (pw.dense if pw.dense.numel() else pw.values).device
    T = spense_tiled_layout(pw.N, pw.K, pw.dtype, pw.split, pw.dense_begin)
    values = torch.empty(T.values_bytes, dtype=torch.uint8, device=dev)
    meta = torch.empty(T.meta_bytes // 4, dtype=torch.int32, device=dev)
    dense = torch.empty(T.dense_bytes, dtype=torch.uint8, device=dev)
    out = PackedWeight(pw.N, pw.K, pw.dtype, pw.split, pw.dense_begin, values, meta, dense, SPENSE_LAYOUT_TILED)
    _check(spense_tile(pw.desc, out.desc, _stream(dev)))
    return out


def decompress(pw: PackedWeight) -> torch.Tensor:
    dev = (pw.dense if pw.dense.numel() else pw.values).device
    W = torch.empty((pw.N, pw.K), dtype=_storage_dtype(pw.dtype), device=dev)
    _check(spense_decompress(pw.desc, _ptr(W), W.stride(0), _stream(dev)))
    return W


def _check_x(X: torch.Tensor, dtype: int, K: int):
    _row_major(X, "X")
    if _act_code(X) != dtype:
        raise ValueError(f"X is {X.dtype}; this weight takes {'fp8 codes (uint8)' if dtype == SPENSE_FP8_E4M3FN else 'bfloat16'}")
    if X.shape[1] != K:
        raise ValueError(f"X.shape[1] = {X.shape[1]} != K = {K}")


def _act_code(t: torch.Tensor):
    if t.dtype in (torch.uint8, torch.float8_e4m3fn):
        return SPENSE_FP8_E4M3FN
    if t.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return SPENSE_BF16
    return None


def _out(out, M, N, out_f32, dev, name="out"):
    """A new output, or the caller's checked: 2-D, rows contiguous, shape (M, N), fp32 or
    bf16 as out_f32 says, on X's device."""
    want = torch.float32 if out_f32 else torch.bfloat16
    if out is None:
        return torch.empty((M, N), dtype=want, device=dev)
    if out.dim() != 2 or out.stride(1) != 1 or (M > 1 and out.stride(0) < N):
        raise ValueError(f"{name} must be a 2-D tensor with contiguous rows")
    if tuple(out.shape) != (M, N):
        raise ValueError(f"{name} has shape {tuple(out.shape)}, expected {(M, N)}")
    if out.dtype != want:
        raise ValueError(f"{name} is {out.dtype}, expected {want}")
    if out.device != dev:
        raise ValueError(f"{name} is on {out.device}, X on {dev}")
    return out


def _check_scale(s, n, dev, name):
    if s is None:
        return
    if s.dtype != torch.float32 or s.dim() != 1 or s.shape[0] != n or not s.is_contiguous() or s.device != dev:
        raise ValueError(f"{name} must be a contiguous fp32 vector of length {n} on {dev}")


def gemm(X: torch.Tensor, pw: PackedWeight, w_scale=None, x_scale=None, out=None, out_f32=False,
         workspace: Workspace | None = None, plan: spense_plan_override_t | None = None) -> torch.Tensor:
    """Y = X W^T for a packed weight (spense_gemm; with ``plan``, spense_gemm_planned:
    parts of the execution plan forced, for tests and tuning)."""
    _check_x(X, pw.dtype, pw.K)
    M = X.shape[0]
    _check_scale(w_scale, pw.N, X.device, "w_scale")
    _check_scale(x_scale, M, X.device, "x_scale")
    out = _out(out, M, pw.N, out_f32, X.device)
    ws = workspace or workspace_for(X.device)
    flags = SPENSE_OUT_F32 if out_f32 else SPENSE_OUT_BF16
    if plan is None:
        wp, wn = ws.get(spense_gemm_workspace_size(M, pw.desc))
        _check(spense_gemm(_ptr(X), M, X.stride(0), pw.desc, _ptr(w_scale), _ptr(x_scale), _ptr(out), out.stride(0),
                           flags, wp, wn, _stream(X.device)))
    else:
        wp, wn = ws.get(spense_gemm_planned_workspace_size(M, pw.desc, plan))
        _check(spense_gemm_planned(_ptr(X), M, X.stride(0), pw.desc, _ptr(w_scale), _ptr(x_scale), _ptr(out),
                                   out.stride(0), flags, wp, wn, plan, _stream(X.device)))
    return out


def gemm_noalloc(X: torch.Tensor, pw: PackedWeight, w_scale=None, x_scale=None, out=None,
                 out_f32=False) -> torch.Tensor:
    """Y = X W^T through spense_gemm_noalloc: spense_gemm with the K-slice partial sums in
    the library's per-device scratch instead of a workspace (for callers that cannot
    allocate; calls that overlap on one device race).  ``out`` should be given by such
    callers, since allocating it here would defeat the purpose."""
    _check_x(X, pw.dtype, pw.K)
    M = X.shape[0]
    _check_scale(w_scale, pw.N, X.device, "w_scale")
    _check_scale(x_scale, M, X.device, "x_scale")
    out = _out(out, M, pw.N, out_f32, X.device)
    _check(spense_gemm_noalloc(_ptr(X), M, X.stride(0), pw.desc, _ptr(w_scale), _ptr(x_scale), _ptr(out),
                               out.stride(0), SPENSE_OUT_F32 if out_f32 else SPENSE_OUT_BF16, _stream(X.device)))
    return out


def gemm_grouped(X: torch.Tensor, pws, w_scales=None, x_scale=None, outs=None, out_f32=False):
    """One launch for several Spense weights sharing X (spense_gemm_grouped): returns
    [X W_i^T].  pws: tiled fp8 output-split PackedWeights with equal K (up to 4)."""
    n = len(pws)
    if n < 1:
        raise ValueError("at least one weight")
    for p in pws:
        _check_x(X, p.dtype, p.K)
    M = X.shape[0]
    if w_scales is not None and len(w_scales) != n:
        raise ValueError("one w_scale per weight")
    if outs is None:
        outs = [None] * n
    if len(outs) != n:
        raise ValueError("one output per weight")
    outs = [_out(o, M, p.N, out_f32, X.device, f"outs[{i}]") for i, (o, p) in enumerate(zip(outs, pws))]
    descs = [p.desc for p in pws]
    for i, p in enumerate(pws):
        _check_scale(w_scales[i] if w_scales is not None else None, p.N, X.device, "w_scale")
    _check_scale(x_scale, M, X.device, "x_scale")
    PP = ctypes.POINTER(spense_packed_t)
    parr = (PP * n)(*[ctypes.pointer(d) for d in descs])
    sarr = (ctypes.c_void_p * n)(*[_ptr(w_scales[i]) if w_scales is not None else None for i in range(n)])
    yarr = (ctypes.c_void_p * n)(*[_ptr(o) for o in outs])
    larr = (ctypes.c_int64 * n)(*[o.stride(0) for o in outs])
    _check(spense_gemm_grouped(_ptr(X), M, X.stride(0), n, parr, sarr if w_scales is not None else None,
                               _ptr(x_scale), yarr, larr, SPENSE_OUT_F32 if out_f32 else SPENSE_OUT_BF16,
                               _stream(X.device)))
    return outs


def gemm_glu(X: torch.Tensor, gate: PackedWeight, up: PackedWeight, gate_scale=None, up_scale=None, x_scale=None,
             out=None) -> torch.Tensor:
    """H = glu(X Wg^T, X Wu^T) in one launch (spense_gemm_glu), fp32 M x N: the gate and
    up GEMMs with the GLU step in their epilogue.  gate, up: tiled fp8 output-split
    PackedWeights with equal N, K and dense_begin."""
    _check_x(X, SPENSE_FP8_E4M3FN, gate.K)
    M = X.shape[0]
    if gate.K != X.shape[1] or up.K != X.shape[1]:
        raise ValueError("X.shape[1] must equal K")
    if gate.N != up.N:
        raise ValueError("gate and up must have the same N")
    if out is None:
        out = torch.empty((M, gate.N), dtype=torch.float32, device=X.device)
    _row_major(out, "out")
    if out.dtype != torch.float32 or out.shape != (M, gate.N):
        raise ValueError(f"out must be fp32 of shape {(M, gate.N)}")
    _check_scale(gate_scale, gate.N, X.device, "gate_scale")
    _check_scale(up_scale, up.N, X.device, "up_scale")
    _check_scale(x_scale, M, X.device, "x_scale")
    _check(spense_gemm_glu(_ptr(X), M, X.stride(0), ctypes.byref(gate.desc), ctypes.byref(up.desc), _ptr(gate_scale),
                           _ptr(up_scale), _ptr(x_scale), _ptr(out), out.stride(0), _stream(X.device)))
    return out


def gemm_glu_fp8(X: torch.Tensor, gate: PackedWeight, up: PackedWeight, gate_scale=None, up_scale=None,
                 x_scale=None, q=None, scales=None, workspace: Workspace | None = None):
    """The producer half of the GLU MLP (spense_gemm_glu_fp8): H = glu(X Wg^T, X Wu^T) in
    the gate / up epilogue, then its per-token fp8 quantisation from the epilogue's row
    maxima.  Returns (codes uint8 M x N, scales fp32 M), the down projection's input."""
    _check_x(X, SPENSE_FP8_E4M3FN, gate.K)
    M = X.shape[0]
    if gate.K != X.shape[1] or up.K != X.shape[1]:
        raise ValueError("X.shape[1] must equal K")
    if gate.N != up.N:
        raise ValueError("gate and up must have the same N")
    N = gate.N
    q = torch.empty((M, N), dtype=torch.uint8, device=X.device) if q is None else q
    scales = torch.empty(M, dtype=torch.float32, device=X.device) if scales is None else scales
    _row_major(q, "q")
    if q.dtype != torch.uint8 or q.shape != (M, N):
        raise ValueError(f"q must be uint8 of shape {(M, N)}")
    _check_scale(scales, M, X.device, "scales")
    _check_scale(gate_scale, N, X.device, "gate_scale")
    _check_scale(up_scale, N, X.device, "up_scale")
    _check_scale(x_scale, M, X.device, "x_scale")
    ws = workspace or workspace_for(X.device)
    wp, wn = ws.get(spense_gemm_glu_fp8_workspace_size(M, N) if M > 0 and N > 0 else 0)
    _check(spense_gemm_glu_fp8(_ptr(X), M, X.stride(0), ctypes.byref(gate.desc), ctypes.byref(up.desc),
                               _ptr(gate_scale), _ptr(up_scale), _ptr(x_scale), _ptr(q), q.stride(0), _ptr(scales),
                               wp, wn, _stream(X.device)))
    return q, scales


def dense_gemm(X: torch.Tensor, W: torch.Tensor, w_scale=None, x_scale=None, out=None, out_f32=False,
               workspace: Workspace | None = None) -> torch.Tensor:
    """The dense baseline Y = X W^T (spense_dense_gemm)."""
    _row_major(W, "W")
    dtype = _dtype_code(W)
    N, K = W.shape
    _check_x(X, dtype, K)
    if W.device != X.device:
        raise ValueError("W and X must be on one device")
    M = X.shape[0]
    _check_scale(w_scale, N, X.device, "w_scale")
    _check_scale(x_scale, M, X.device, "x_scale")
    out = _out(out, M, N, out_f32, X.device)
    ws = workspace or workspace_for(X.device)
    wp, wn = ws.get(spense_dense_gemm_workspace_size(M, N, K, dtype))
    _check(spense_dense_gemm(_ptr(X), M, X.stride(0), _ptr(W), W.stride(0), N, K, dtype, _ptr(w_scale),
                             _ptr(x_scale), _ptr(out), out.stride(0), SPENSE_OUT_F32 if out_f32 else SPENSE_OUT_BF16,
                             wp, wn, _stream(X.device)))
    return out


def _act_type(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SPENSE_BF16
    if t.dtype == torch.float32:
        return SPENSE_F32
    raise TypeError(f"activations must be bfloat16 or float32, got {t.dtype}")


def quantize_fp8(A: torch.Tensor, q=None, scales=None):
    """Per-token fp8 quantisation (spense_quantize_fp8): returns (codes uint8 M x K,
    scales fp32 M) with scales = row absmax / 448 and codes = e4m3fn(A / scale)."""
    _row_major(A, "A")
    M, K = A.shape
    q = torch.empty((M, K), dtype=torch.uint8, device=A.device) if q is None else q
    scales = torch.empty(M, dtype=torch.float32, device=A.device) if scales is None else scales
    _check(spense_quantize_fp8(_ptr(A), _act_type(A), M, K, A.stride(0), _ptr(q), q.stride(0), _ptr(scales),
                               _stream(A.device)))
    return q, scales


def glu_quantize_fp8(G: torch.Tensor, U: torch.Tensor, q=None, scales=None):
    """The GLU step fused with per-token fp8 quantisation (spense_glu_quantize_fp8):
    H = U * silu(G), returned as (codes uint8 M x I, scales fp32 M)."""
    _row_major(G, "G")
    _row_major(U, "U")
    if G.shape != U.shape or G.dtype != U.dtype:
        raise ValueError("G and U must have the same shape and dtype")
    M, I = G.shape
    q = torch.empty((M, I), dtype=torch.uint8, device=G.device) if q is None else q
    scales = torch.empty(M, dtype=torch.float32, device=G.device) if scales is None else scales
    _check(spense_glu_quantize_fp8(_ptr(G), G.stride(0), _ptr(U), U.stride(0), _act_type(G), M, I, _ptr(q),
                                   q.stride(0), _ptr(scales), _stream(G.device)))
    return q, scales


def mlp(X: torch.Tensor, x_scale: torch.Tensor, gate: PackedWeight, up: PackedWeight, down: PackedWeight,
        gate_scale=None, up_scale=None, down_scale=None, out=None, workspace: Workspace | None = None):
    """The GLU MLP of the paper's sec. 3.3.1 Eq. (4) on Spense weights: H = glu(gate(X),
    up(X)) (output-split) and (Hq, sh) its per-token fp8 quantisation (for tiled fp8
    weights of one geometry and up to 64 tokens the GLU in the gate / up epilogue, then
    the quantisation from the epilogue's row maxima; otherwise G and U in fp32 and the GLU
    fused with the quantisation), Y = down(Hq) (input-split, bf16 out).  X: fp8 codes
    with x_scale."""
    # the paired launch runs the row-split kernel, which pays for one block of up to 64
    # tokens; above that the grouped call (one 256 x 256 tile grid over both weights where
    # it fills the GPU, else a plan per weight) gives G and U
    groupable = (gate.kind == up.kind == SPENSE_LAYOUT_TILED and gate.dtype == up.dtype == SPENSE_FP8_E4M3FN
                 and gate.split == up.split == SPENSE_SPLIT_OUTPUT)
    paired = groupable and X.shape[0] <= 64
    if paired and gate.N == up.N and gate.K == up.K and gate.dense_begin == up.dense_begin:
        Hq, sh = gemm_glu_fp8(X, gate, up, gate_scale, up_scale, x_scale, workspace=workspace)
    else:
        if groupable and gate.K == up.K:
            scales = None if gate_scale is None and up_scale is None else [gate_scale, up_scale]
            G, U = gemm_grouped(X, [gate, up], scales, x_scale, out_f32=True)
        else:
            G = gemm(X, gate, gate_scale, x_scale, out_f32=True, workspace=workspace)
            U = gemm(X, up, up_scale, x_scale, out_f32=True, workspace=workspace)
        Hq, sh = glu_quantize_fp8(G, U)
    return gemm(Hq, down, down_scale, sh, out=out, workspace=workspace)



# ------------------------------------------------------------------ dense-index selection
def index_scores(Wg: torch.Tensor, Wu: torch.Tensor, Wd: torch.Tensor, h_in: torch.Tensor, h_mid: torch.Tensor,
                 eps: float = 1e-8) -> dict:
    """SpenseGPT+ priorities of the intermediate indices of a GLU MLP (spense_index_scores,
    sec. 3.3.1).  Wg, Wu: I x D, Wd: D x I (bf16 or fp32, the same dtype); h_in (D) and
    h_mid (I): fp32 diagonals of the input Hessians.  Returns the raw gate / up / down
    score vectors and their mean-normalised sum ``total`` (fp32, on the device)."""
    for t, n in ((Wg, "Wg"), (Wu, "Wu"), (Wd, "Wd")):
        _row_major(t, n)
    if Wg.shape != Wu.shape or Wg.stride(0) != Wu.stride(0) or Wd.shape != (Wg.shape[1], Wg.shape[0]):
        raise ValueError("Wg, Wu must be I x D with one leading dimension and Wd D x I")
    if not (Wg.dtype == Wu.dtype == Wd.dtype):
        raise ValueError("the three weights must have one dtype")
    I, D = Wg.shape
    h_in = h_in.to(torch.float32).contiguous()
    h_mid = h_mid.to(torch.float32).contiguous()
    if h_in.numel() != D or h_mid.numel() != I:
        raise ValueError("h_in must have D entries and h_mid I")
    raw = torch.empty((3, I), dtype=torch.float32, device=Wg.device)
    total = torch.empty(I, dtype=torch.float32, device=Wg.device)
    _check(spense_index_scores(_ptr(Wg), _ptr(Wu), Wg.stride(0), _ptr(Wd), Wd.stride(0), _act_type(Wg), I, D,
                               _ptr(h_in), _ptr(h_mid), eps, _ptr(raw), _ptr(total), _stream(Wg.device)))
    return {"gate": raw[0], "up": raw[1], "down": raw[2], "total": total}


def dense_permutation(total: torch.Tensor, n_dense: int):
    """TopK of the priorities and the permutation moving them to the back
    (spense_dense_permutation): returns (flags uint8 I, perm int32 I, perm[new] = old)."""
    if total.dtype != torch.float32 or total.dim() != 1 or not total.is_contiguous():
        raise ValueError("total must be a contiguous fp32 vector")
    I = total.numel()
    flags = torch.empty(I, dtype=torch.uint8, device=total.device)
    perm = torch.empty(I, dtype=torch.int32, device=total.device)
    _check(spense_dense_permutation(_ptr(total), I, n_dense, _ptr(flags), _ptr(perm), _stream(total.device)))
    return flags, perm


def _perm_arg(perm: torch.Tensor, n: int):
    if perm.dtype != torch.int32 or perm.numel() != n or not perm.is_contiguous():
        raise ValueError(f"perm must be a contiguous int32 vector of {n} entries")


def gather_rows(src: torch.Tensor, perm: torch.Tensor, out=None) -> torch.Tensor:
    """out[r] = src[perm[r]] (spense_gather_rows) for a row-major 2-D tensor."""
    _row_major(src, "src")
    _perm_arg(perm, src.shape[0])
    out = torch.empty_like(src, memory_format=torch.contiguous_format) if out is None else out
    es = src.element_size()
    _check(spense_gather_rows(_ptr(src), src.stride(0) * es, _ptr(out), out.stride(0) * es, src.shape[0],
                              src.shape[1] * es, _ptr(perm), _stream(src.device)))
    return out


def gather_cols(src: torch.Tensor, perm: torch.Tensor, out=None) -> torch.Tensor:
    """out[:, c] = src[:, perm[c]] (spense_gather_cols) for a row-major 2-D tensor."""
    _row_major(src, "src")
    _perm_arg(perm, src.shape[1])
    out = torch.empty_like(src, memory_format=torch.contiguous_format) if out is None else out
    _check(spense_gather_cols(_ptr(src), src.stride(0), _ptr(out), out.stride(0), src.shape[0], src.shape[1],
                              src.element_size(), _ptr(perm), _stream(src.device)))
    return out


def select_dense_indices(Wg: torch.Tensor, Wu: torch.Tensor, Wd: torch.Tensor, h_in: torch.Tensor,
                         h_mid: torch.Tensor, n_dense: int, eps: float = 1e-8) -> dict:
    """The whole SpenseGPT+ index step of sec. 3.3.1 on the device: priorities, TopK, and
    Wg, Wu (rows) and Wd (columns) permuted so the n_dense chosen indices form the
    trailing dense region of all three.  Eq. (4): the MLP computes the same function."""
    sc = index_scores(Wg, Wu, Wd, h_in, h_mid, eps)
    flags, perm = dense_permutation(sc["total"], n_dense)
    return {"scores": sc, "flags": flags, "perm": perm, "Wg": gather_rows(Wg, perm), "Wu": gather_rows(Wu, perm),
            "Wd": gather_cols(Wd, perm)}


# ------------------------------------------------------------------ SparseGPT 2:4 with a protected dense region
def obs_factor(H: torch.Tensor, percdamp: float = 0.01, workspace: Workspace | None = None):
    """The inverse-Hessian factor of the SparseGPT sweep (spense_obs_factor): H (K x K fp32,
    lower triangle read) -> (U upper K x K with (H + lambda I)^{-1} = U^T U, dead uint8 K).
    Synchronous."""
    _row_major(H, "H")
    if H.dtype != torch.float32 or H.shape[0] != H.shape[1]:
        raise ValueError("H must be a square fp32 matrix")
    K = H.shape[0]
    U = torch.empty((K, K), dtype=torch.float32, device=H.device)
    dead = torch.empty(K, dtype=torch.uint8, device=H.device)
    ws = workspace or workspace_for(H.device)
    wp, wn = ws.get(spense_obs_factor_workspace_size(K))
    _check(spense_obs_factor(_ptr(H), H.stride(0), K, percdamp, _ptr(U), U.stride(0), _ptr(dead), wp, wn,
                             _stream(H.device)))
    return U, dead


def obs_prune_24(W: torch.Tensor, U: torch.Tensor, dense_begin: int, dead: torch.Tensor | None = None,
                 workspace: Workspace | None = None):
    """SparseGPT 2:4 on W's columns [0, dense_begin) with the columns after it kept dense
    and compensated (spense_obs_prune_24); W (N x K fp32) is updated in place.  Returns
    the kept flags (uint8 N x K)."""
    _row_major(W, "W")
    _row_major(U, "U")
    if W.dtype != torch.float32 or U.dtype != torch.float32 or U.shape != (W.shape[1], W.shape[1]):
        raise ValueError("W (N x K) and U (K x K) must be fp32")
    N, K = W.shape
    keep = torch.empty((N, K), dtype=torch.uint8, device=W.device)
    ws = workspace or workspace_for(W.device)
    wp, wn = ws.get(spense_obs_prune_workspace_size(N))
    _check(spense_obs_prune_24(_ptr(W), W.stride(0), N, K, _ptr(U), U.stride(0), _ptr(dead), dense_begin, _ptr(keep),
                               keep.stride(0), wp, wn, _stream(W.device)))
    return keep
