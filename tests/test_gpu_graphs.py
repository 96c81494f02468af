"""The kernels inside a captured HIP graph (as the benchmark runs them).

A grouped decode launch (three matrices sharing the activations), a sparse
prefill call and a sparse int8 call are captured in one graph.  The graph is
replayed three times; between replays the test fills every output with NaN
(or a sentinel) eagerly, runs unrelated eager work and synchronises, and each
replay must reproduce the eager results bit for bit (the same kernels on the
same inputs are deterministic).  The library records no memset or copy nodes:
zero fills are kernels."""
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
