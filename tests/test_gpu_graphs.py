"""The kernels inside a captured HIP graph (as the benchmark runs them).

A grouped decode launch (three matrices sharing the activations), a sparse
prefill call and a sparse int8 call are captured in one graph.  The graph is
replayed three times; between replays the test fills every output with NaN
(or a sentinel) eagerly, runs unrelated eager work and synchronises, and each
replay must reproduce the eager results bit for bit (the same kernels on the
same inputs are deterministic).  The library records no memset or copy nodes:
zero fills are kernels."""
import ctypes

import numpy as np
import pytest

import synth
from tests._helpers import from_dev_bits, to_dev

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager():
    import torch

    import paper_2405_03594_amd as spl

    spl.lib()
    K, M1, M2 = 1056, 4, 300
    mats = []
    for j, N in enumerate((300, 180, 520)):
        W, mask = synth.weight(970 + j, N, K, "bf16", 0.7)
        mats.append(spl.pack_sparse(to_dev(W, "bf16"), torch.from_numpy(mask).cuda()))
    X1 = to_dev(synth.activations(975, M1, K, "bf16"), "bf16")
    X2 = to_dev(synth.activations(976, M2, K, "bf16"), "bf16")
    Wq, maskq, sw = synth.int8_weight(977, 260, K, 0.7)
    Wqc = spl.pack_sparse(torch.from_numpy(Wq).cuda(), torch.from_numpy(maskq).cuda())
    q, sx = synth.int8_activations(978, 16, K)
    Xq, sxd, swd = torch.from_numpy(q).cuda(), torch.from_numpy(sx).cuda(), torch.from_numpy(sw).cuda()

    outs_dec = [torch.empty((M1, m.rows), dtype=torch.bfloat16, device="cuda") for m in mats]
    out_pf = torch.empty((M2, mats[2].rows), dtype=torch.bfloat16, device="cuda")
    out_i8 = torch.empty((16, Wqc.rows), dtype=torch.float16, device="cuda")
    acc_i8 = torch.empty((16, Wqc.rows), dtype=torch.int32, device="cuda")

    def run():
        spl.sparse_linear_group([X1, X1, X1], mats, outs=outs_dec, algo="decode")
        spl.sparse_linear(X2, mats[2], out=out_pf, algo="prefill")
        spl.sparse_linear_int8(Xq, sxd, Wqc, swd, out=out_i8, acc_out=acc_i8)

    def snapshot():
        return [from_dev_bits(o) for o in outs_dec] + [from_dev_bits(out_pf), from_dev_bits(out_i8),
                                                       acc_i8.cpu().numpy().copy()]

    def poison():
        for o in outs_dec + [out_pf, out_i8]:
            o.fill_(float("nan"))
        acc_i8.fill_(-1)

    run()
    torch.cuda.synchronize()
    eager = snapshot()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                      # warm-up on the capture stream, as torch recommends
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run()
    torch.cuda.synchronize()

    scratch = torch.randn(1 << 20, device="cuda")
    for rep in range(3):
        poison()
        scratch.mul_(1.0001).add_(0.5)                 # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = snapshot()
        for i, (a, b) in enumerate(zip(got, eager)):
            assert np.array_equal(a, b), f"replay {rep}, output {i} differs from the eager run"


def test_graph_replays_new_ops_match_eager():
    """The gated silu(gate) * up launch (both kernel families), the magnitude
    mask (zero fill, histogram atomics, tie ranks), the weight gradient
    (transposes, product, gather) and the packed-transpose permutation in one
    captured graph: three replays with poisoned outputs and eager work in
    between reproduce the eager results bit for bit."""
    import torch

    import paper_2405_03594_amd as spl

    spl.lib()
    N, K = 200, 1056
    Wg, mg = synth.weight(980, N, K, "bf16", 0.7)
    Wu, mu = synth.weight(981, N, K, "bf16", 0.5)
    g = spl.pack_sparse(to_dev(Wg, "bf16"), torch.from_numpy(mg).cuda())
    u = spl.pack_sparse(to_dev(Wu, "bf16"), torch.from_numpy(mu).cuda())
    gt = spl.pack_sparse(spl.transpose16(spl.unpack(g)), torch.from_numpy(mg).cuda().t().contiguous())
    perm = spl.transpose_perm(g, gt)
    X1 = to_dev(synth.activations(982, 8, K, "bf16"), "bf16")
    X2 = to_dev(synth.activations(983, 136, K, "bf16"), "bf16")
    dY = to_dev(synth.activations(984, 136, N, "bf16"), "bf16")
    Wp = to_dev(synth.round_to(synth.normal_f32(985, (300, 4096), 0.02), "bf16"), "bf16")
    ws_m = torch.empty((spl.lib().spl_magnitude_mask_workspace_bytes(),), dtype=torch.uint8, device="cuda")
    ws_g = torch.empty((spl.lib().spl_sparse_weight_grad_workspace_bytes(136, N, K),), dtype=torch.uint8,
                       device="cuda")
    y1 = torch.empty((8, N), dtype=torch.bfloat16, device="cuda")
    y2 = torch.empty((136, N), dtype=torch.bfloat16, device="cuda")
    mask = torch.empty((300, 4096), dtype=torch.uint8, device="cuda")
    grad = torch.empty_like(g.values)
    tv = torch.empty_like(gt.values)

    def run():
        spl.sparse_linear_silu_mul(X1, g, u, out=y1)
        spl.sparse_linear_silu_mul(X2, g, u, out=y2)
        spl.magnitude_mask(Wp, 300 * 4096 * 7 // 10, out=mask, workspace=ws_m)
        spl.sparse_weight_grad(dY, X2, g, out=grad, workspace=ws_g)
        spl.permute_values(g.values, perm, g.nnz, tv)

    def snapshot():
        return [from_dev_bits(y1), from_dev_bits(y2), mask.cpu().numpy().copy(), from_dev_bits(grad)[:g.nnz],
                from_dev_bits(tv)[:g.nnz]]

    def poison():
        for o in (y1, y2, grad, tv):
            o.fill_(float("nan"))
        mask.fill_(7)
        ws_m.fill_(0xAB)                               # the histogram must be cleared inside the graph
        ws_g.fill_(0xCD)

    run()
    torch.cuda.synchronize()
    eager = snapshot()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run()
    torch.cuda.synchronize()
    scratch = torch.randn(1 << 20, device="cuda")
    for rep in range(3):
        poison()
        scratch.mul_(1.0001).add_(0.5)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(snapshot(), eager)):
            assert np.array_equal(a, b), f"replay {rep}, output {i} differs from the eager run"


def test_graph_replays_training_kernels_match_eager():
    """The training step's direct kernels in one captured graph - the grouped
    weight gradient read straight from dY and X (two tasks, one launch) and
    the input gradient from W's packed tiles - plus the input gradient's
    decoded fallback: three replays with poisoned outputs and eager work in
    between reproduce the eager results bit for bit."""
    import torch

    import paper_2405_03594_amd as spl

    spl.lib()
    M, N, K = 256, 2048, 8192                          # 64 x 8 and 64 x 8 blocks: each at least one per CU
    Wa, ma = synth.weight(990, N, K, "bf16", 0.7)
    Wb, mb = synth.weight(991, N, K, "bf16", 0.5)
    A = spl.pack_sparse(to_dev(Wa, "bf16"), torch.from_numpy(ma).cuda())
    Bm = spl.pack_sparse(to_dev(Wb, "bf16"), torch.from_numpy(mb).cuda())
    X = to_dev(synth.activations(992, M, K, "bf16"), "bf16")
    dYa = to_dev(synth.activations(993, M, N, "bf16"), "bf16")
    dYb = to_dev(synth.activations(994, M, N, "bf16"), "bf16")
    Ws, ms = synth.weight(995, 96, 200, "bf16", 0.6)   # the input gradient's fallback shape
    S = spl.pack_sparse(to_dev(Ws, "bf16"), torch.from_numpy(ms).cuda())
    dYs = to_dev(synth.activations(996, 40, 96, "bf16"), "bf16")
    dYd = to_dev(synth.activations(997, 1024, N, "bf16"), "bf16")       # the input gradient: 64 x 4 blocks
    assert spl.lib().spl_sparse_input_grad_workspace_bytes(1024, ctypes.byref(A.view())) == 0
    ws_s = torch.empty((spl.lib().spl_sparse_input_grad_workspace_bytes(40, ctypes.byref(S.view())),),
                       dtype=torch.uint8, device="cuda")
    ga, gb = torch.empty_like(A.values), torch.empty_like(Bm.values)
    dx = torch.empty((1024, K), dtype=torch.bfloat16, device="cuda")
    dxs = torch.empty((40, 200), dtype=torch.bfloat16, device="cuda")

    def run():
        spl.sparse_weight_grad_group([dYa, dYb], [X, X], [A, Bm], outs=[ga, gb])
        spl.sparse_input_grad(dYd, A, out=dx)
        spl.sparse_input_grad(dYs, S, out=dxs, workspace=ws_s)

    def snapshot():
        return [from_dev_bits(ga)[:A.nnz], from_dev_bits(gb)[:Bm.nnz], from_dev_bits(dx), from_dev_bits(dxs)]

    def poison():
        for o in (ga, gb, dx, dxs):
            o.fill_(float("nan"))
        ws_s.fill_(0xCD)

    run()
    torch.cuda.synchronize()
    eager = snapshot()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run()
    torch.cuda.synchronize()
    scratch = torch.randn(1 << 20, device="cuda")
    for rep in range(3):
        poison()
        scratch.mul_(1.0001).add_(0.5)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(snapshot(), eager)):
            assert np.array_equal(a, b), f"replay {rep}, output {i} differs from the eager run"
