"""spense_gemm_noalloc (the no-allocation variant of spense_gemm, K-slice partial sums in
the library's per-device scratch) through the C ABI, against spense_gemm and the oracle.

Two calls in a row on K-sliced plans, the second with fewer tokens (the scratch keeps the
first call's partial sums; the second must not read any of them), a plan without K
slices, and the header's limit.  Exact-integer data, so every output is compared bit for
bit with spense_gemm's (the same plan) and with the oracle's.
"""
import sys

import numpy as np
import pytest
import torch

import gen
import oracle

pytestmark = pytest.mark.gpu

FP8 = 1


@pytest.fixture(scope="module")
def S():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10445_amd as S
    return S


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def tdev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.cpu().numpy()


# (name, N, K, split, first M, second M): down and o slice K into 4 at these token counts,
# k (64 tiles) at every M; down at 66-128 tokens runs as two 64-token halves in 6 slices
CASES = [("down", 5120, 25600, 1, 64, 16), ("k", 1024, 5120, 0, 64, 1), ("seed_o", 5120, 10240, 1, 48, 20),
         ("down_128", 5120, 25600, 1, 128, 66)]  # two 64-token halves, 6 K slices: 15.7 MB of scratch


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name,N,K,split,m1,m2", CASES)
def test_noalloc_equals_spense_gemm_on_two_calls(S, name, N, K, split, m1, m2):
    axis = gen.OUTPUT if split == 0 else gen.INPUT
    db = gen.split_point(N, K, axis, 0.25)
    say(f"[noalloc] {name} {N}x{K} M={m1} then {m2}")
    W, mask, X, sw, sx = gen.make_exact_int(30, N % 83, m1, N, K, axis, db, gen.FP8)
    pw = S.tile(S.compress(tdev(W), tdev(mask), split, db))
    assert S.spense_gemm_workspace_size(m1, pw.desc) > 0 and S.spense_gemm_workspace_size(m2, pw.desc) > 0
    assert S.spense_gemm_workspace_size(m1, pw.desc) <= S.SPENSE_NOALLOC_SCRATCH_BYTES
    v, m, d, _ = oracle.compress(W, mask, FP8, split, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, split, db, sw, sx)
    Xd, swd, sxd = tdev(X), tdev(sw), tdev(sx)
    for M in (m1, m2):
        for out_f32 in (True, False):
            dt = torch.float32 if out_f32 else torch.bfloat16
            a = torch.full((M, N), 5.0, dtype=dt, device="cuda")
            b = torch.full((M, N), -5.0, dtype=dt, device="cuda")
            S.gemm_noalloc(Xd[:M], pw, swd, sxd[:M], out=a, out_f32=out_f32)
            S.gemm(Xd[:M], pw, swd, sxd[:M], out=b, out_f32=out_f32)
            torch.cuda.synchronize()
            assert np.array_equal(bits(a), bits(b)), f"{name} M={M}: noalloc differs from spense_gemm"
            assert np.array_equal(bits(a), ref["y_f32" if out_f32 else "y_bf16"][:M]), f"{name} M={M}: oracle"


def test_noalloc_without_k_slices_and_empty_calls(S):
    """A plan with no K slices (no scratch needed) and M = 0 both go through."""
    N, K, db = 1600, 1024, 1200
    W, mask, X, sw, sx = gen.make_exact_int(31, 0, 64, N, K, gen.OUTPUT, db, gen.FP8)
    pw = S.tile(S.compress(tdev(W), tdev(mask), 0, db))
    v, m, d, _ = oracle.compress(W, mask, FP8, 0, db)
    ref = oracle.spense_gemm(X, v, m, d, N, K, FP8, 0, db, sw, sx)
    y = S.gemm_noalloc(tdev(X), pw, tdev(sw), tdev(sx), out_f32=True)
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy(), ref["y_f32"])
    rc = S.spense_gemm_noalloc(None, 0, K, pw.desc, None, None, None, N, 0, torch.cuda.current_stream().cuda_stream)
    assert rc == S.SPENSE_OK
