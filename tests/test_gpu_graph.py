"""Graph capture: the library's launches recorded into a HIP graph (torch.cuda.graph)
and replayed several times, with eager work and synchronisations between the replays,
give the eager results bit for bit.  Covers a K-sliced GEMM (partials in the workspace,
then the reduction launch), the grouped launch, the paired gate / up launch with the
row-maxima quantisation, and the whole MLP block, on the Qwen3-like shapes at M = 16,
64 and 100 (at 100 down runs as two 64-token halves in K slices and the grouped gate /
up as one two-half launch per weight; random data; the comparison is against the same
calls run eagerly)."""
import sys

import numpy as np
import pytest
import torch

import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10445_amd as S
    return S


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def packed(S, name, i, N, K, axis):
    m = gen.make_matrix(7, i, name, N, K, axis, 0.25, gen.FP8)
    pw = S.tile(S.compress(torch.from_numpy(m.W).cuda(), torch.from_numpy(m.mask).cuda(),
                           0 if axis == gen.OUTPUT else 1, m.dense_begin))
    return pw, torch.from_numpy(m.sw).cuda()


@pytest.mark.parametrize("M", [16, 64, 100])
def test_graph_replays_match_eager(S, M):
    say(f"[graph] M={M}")
    D, I = 5120, 25600
    gate, sg = packed(S, "gate", 0, I, D, gen.OUTPUT)
    up, su = packed(S, "up", 1, I, D, gen.OUTPUT)
    down, sd = packed(S, "down", 2, D, I, gen.INPUT)
    X, sx = gen.make_x(7, 0, M, D, gen.FP8)
    Xd, sxd = torch.from_numpy(X).cuda(), torch.from_numpy(sx).cuda()
    Xh, sxh = gen.make_x(7, 1, M, I, gen.FP8, "student_t4")
    Xhd, sxhd = torch.from_numpy(Xh).cuda(), torch.from_numpy(sxh).cuda()
    ws = S.Workspace("cuda")
    ws.get(S.spense_gemm_workspace_size(M, down.desc) + S.spense_gemm_glu_fp8_workspace_size(M, I) + (1 << 20))
    assert S.spense_gemm_workspace_size(M, down.desc) > 0  # down is K-sliced at this M
    Yd = torch.empty((M, D), dtype=torch.bfloat16, device="cuda")
    G = torch.empty((M, I), dtype=torch.float32, device="cuda")
    U = torch.empty_like(G)
    q = torch.empty((M, I), dtype=torch.uint8, device="cuda")
    s = torch.empty(M, dtype=torch.float32, device="cuda")
    Ym = torch.empty((M, D), dtype=torch.bfloat16, device="cuda")

    def run():
        S.gemm(Xhd, down, sd, sxhd, out=Yd, workspace=ws)
        S.gemm_grouped(Xd, [gate, up], [sg, su], sxd, outs=[G, U], out_f32=True)
        S.gemm_glu_fp8(Xd, gate, up, sg, su, sxd, q=q, scales=s, workspace=ws)
        Ym.copy_(S.mlp(Xd, sxd, gate, up, down, sg, su, sd, workspace=ws))

    outs = (Yd, G, U, q, s, Ym)
    run()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()  # warm-up on the capture stream (allocator, library state)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    for rep in range(3):
        for o in outs:
            o.zero_()
        # eager work between the replays on the same buffers
        S.gemm(Xhd, down, sd, sxhd, out=Yd, workspace=ws)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, o, r in zip(("down", "G", "U", "q", "scales", "mlp"), outs, ref):
            assert torch.equal(o.view(torch.uint8) if o.dtype != torch.uint8 else o,
                               r.view(torch.uint8) if r.dtype != torch.uint8 else r), (rep, name)
