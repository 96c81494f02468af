"""Sparse-quantized (int8 weights, int8 activations) linear layers on the GPU
vs the oracle: int32 accumulators and fp16 outputs are compared bit for bit."""
import numpy as np
import pytest

import synth
from tests._helpers import to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def spl():
    import paper_2405_03594_amd as spl

    spl.lib()
    return spl


def _run_sparse(spl, Xq, sx, Wq, mask, sw):
    import torch

    Wqc = spl.pack_sparse(to_dev(Wq, "i8"), torch.from_numpy(mask).cuda())
    M, N = Xq.shape[0], Wq.shape[0]
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    Y = spl.sparse_linear_int8(to_dev(Xq, "i8"), torch.from_numpy(sx).cuda(), Wqc, torch.from_numpy(sw).cuda(),
                               acc_out=acc)
    return acc.cpu().numpy(), Y.cpu().view(torch.int16).numpy().view(np.uint16)


def _assert_equal(got, ref, what):
    if not np.array_equal(got, ref):
        bad = np.argwhere(got != ref)
        i = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} of {ref.size} differ; first at {i}: got {got[i]!r}, "
                             f"oracle {ref[i]!r}")


INT8_M = [1, 5, 16, 17, 32, 33, 64, 65, 100, 127]       # 127: the last batch of the streaming kernels


@pytest.mark.parametrize("N,K,s", [(1, 16, 0.5), (16, 48, 0.5), (33, 64, 0.7), (100, 1008, 0.7), (64, 4096, 0.5),
                                   (200, 336, 0.0), (17, 512, 1.0), (48, 2064, 0.9)])
def test_int8_small(orc, spl, N, K, s):
    Wq, mask, sw = synth.int8_weight(600 + N, N, K, s)
    Xq, sx = synth.int8_activations(700 + K, max(INT8_M), K)
    p = orc.pack(Wq, "i8", mask)
    for M in INT8_M:
        acc_ref, y_ref = orc.linear_i8(Xq[:M], sx[:M], p, sw)
        acc, y = _run_sparse(spl, Xq[:M], sx[:M], Wq, mask, sw)
        _assert_equal(acc, acc_ref, f"acc N={N} K={K} s={s} M={M}")
        _assert_equal(y, y_ref, f"Y N={N} K={K} s={s} M={M}")


def test_int8_full_code_range(orc, spl):
    """Codes over the whole int8 range, -128 included, and accumulators near the
    largest magnitude a 4096-column row can reach."""
    rng = np.random.default_rng(41)
    N, K, M = 64, 4096, 20
    Wq = rng.integers(-128, 128, size=(N, K)).astype(np.int8)
    Xq = rng.integers(-128, 128, size=(M, K)).astype(np.int8)
    Wq[0, :] = -128
    Xq[0, :] = -128                                   # acc[0][0] = 4096 * 2^14 = 2^26
    mask = (rng.random((N, K)) < 0.4).astype(np.uint8)
    mask[0, :] = 1
    sx = rng.uniform(1e-4, 1e-2, size=M).astype(np.float32)
    sw = rng.uniform(1e-4, 1e-2, size=N).astype(np.float32)
    acc_ref, y_ref = orc.linear_i8(Xq, sx, orc.pack(Wq, "i8", mask), sw)
    assert acc_ref[0, 0] == 4096 * 128 * 128
    acc, y = _run_sparse(spl, Xq, sx, Wq, mask, sw)
    _assert_equal(acc, acc_ref, "acc")
    _assert_equal(y, y_ref, "Y")


def test_int8_without_acc_out(orc, spl):
    import torch

    Wq, mask, sw = synth.int8_weight(31, 50, 320, 0.7)
    Xq, sx = synth.int8_activations(32, 3, 320)
    _, y_ref = orc.linear_i8(Xq, sx, orc.pack(Wq, "i8", mask), sw)
    Wqc = spl.pack_sparse(to_dev(Wq, "i8"), torch.from_numpy(mask).cuda())
    Y = spl.sparse_linear_int8(to_dev(Xq, "i8"), torch.from_numpy(sx).cuda(), Wqc, torch.from_numpy(sw).cuda())
    _assert_equal(Y.cpu().view(torch.int16).numpy().view(np.uint16), y_ref, "Y")


@pytest.mark.parametrize("name,N,K", synth.LLAMA2_7B_LINEARS[3:])   # o, gate, up, down
def test_int8_llama_shapes_70(orc, spl, name, N, K):
    j = [n for n, _, _ in synth.LLAMA2_7B_LINEARS].index(name)
    Wq, mask, sw = synth.int8_weight(synth.weight_seed(0, j), N, K, 0.7)
    Xq, sx = synth.int8_activations(synth.activation_seed(j), 64, K)
    p = orc.pack(Wq, "i8", mask)
    for M in (1, 16, 64):
        acc_ref, y_ref = orc.linear_i8(Xq[:M], sx[:M], p, sw)
        acc, y = _run_sparse(spl, Xq[:M], sx[:M], Wq, mask, sw)
        _assert_equal(acc, acc_ref, f"{name} acc M={M}")
        _assert_equal(y, y_ref, f"{name} Y M={M}")


@pytest.mark.parametrize("N,K", [(16, 64), (100, 1008), (130, 272), (4096, 4096)])
def test_dense_int8(orc, spl, N, K):
    import torch

    rng = np.random.default_rng(N + K)
    Wq = rng.integers(-128, 128, size=(N, K)).astype(np.int8)
    Xq, sx = synth.int8_activations(55, 65, K)
    sw = rng.uniform(1e-4, 1e-2, size=N).astype(np.float32)
    Wd = to_dev(Wq, "i8")
    for M in (1, 16, 17, 64, 65):
        acc_ref, y_ref = orc.dense_i8(Xq[:M], sx[:M], Wq, sw)
        acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
        Y = spl.dense_linear_int8(to_dev(Xq[:M], "i8"), torch.from_numpy(sx[:M]).cuda(), Wd,
                                  torch.from_numpy(sw).cuda(), acc_out=acc)
        _assert_equal(acc.cpu().numpy(), acc_ref, f"dense acc M={M}")
        _assert_equal(Y.cpu().view(torch.int16).numpy().view(np.uint16), y_ref, f"dense Y M={M}")


def _tie_cases(count, seed=0):
    """(acc, sx, sw) whose binary32 result (float(acc) * sx) * sw lies exactly
    halfway between two binary16 values while the exact product does not: a
    single-rounding multiply-and-convert would round these differently."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        acc = rng.integers(1, 128, size=200000)
        sx = rng.uniform(0.5, 1.0, size=acc.size).astype(np.float32)
        sw = rng.uniform(2.0 ** -6, 2.0 ** -5, size=acc.size).astype(np.float32)
        t = (acc * sx.astype(np.float64)).astype(np.float32)
        y64 = t.astype(np.float64) * sw.astype(np.float64)           # exact: 24 + 24 bits
        y = y64.astype(np.float32)
        bits = y.view(np.uint32)
        tie = ((bits & 0x1FFF) == 0x1000) & (y64 != y.astype(np.float64))
        for i in np.flatnonzero(tie):
            out.append((int(acc[i]), sx[i], sw[i]))
    return out[:count]


@pytest.mark.parametrize("count", [48, 160])          # 160: the batch takes the prefill tiling
def test_int8_epilogue_rounds_each_product(orc, spl, count):
    cases = _tie_cases(count)
    M = N = len(cases)
    K = 32
    Xq = np.zeros((M, K), dtype=np.int8)
    Wq = np.zeros((N, K), dtype=np.int8)
    mask = np.zeros((N, K), dtype=np.uint8)
    Xq[:, 3] = [c[0] for c in cases]
    Wq[:, 3] = 1
    mask[:, 3] = 1
    sx = np.array([c[1] for c in cases], dtype=np.float32)
    sw = np.array([c[2] for c in cases], dtype=np.float32)
    acc_ref, y_ref = orc.linear_i8(Xq, sx, orc.pack(Wq, "i8", mask), sw)
    acc, y = _run_sparse(spl, Xq, sx, Wq, mask, sw)
    _assert_equal(acc, acc_ref, "acc")
    _assert_equal(np.diag(y), np.diag(y_ref), "Y at the ties")
    _assert_equal(y, y_ref, "Y")


@pytest.mark.parametrize("M", [1, 16, 40, 70, 130])
def test_int8_group_matches_oracle_and_single_calls(orc, spl, M):
    """A group of three layers with different N and K (one launch for all):
    every task's int32 sums and fp16 outputs equal the oracle and the single
    calls bit for bit, sparse and dense (M = 1: staged activations; 16, 40,
    70: one, two and four batch fragments, 70 on two batch blocks; 130: the
    prefill tiling, one launch per task)."""
    import torch

    shapes = [(40, 96, 0.7), (100, 528, 0.5), (33, 96, 0.9)]
    Xqs, sxs, Wcs, sws, dense, refs = [], [], [], [], [], []
    for i, (N, K, s) in enumerate(shapes):
        Wq, mask, sw = synth.int8_weight(800 + i, N, K, s)
        Xq, sx = synth.int8_activations(810 + i, M, K)
        refs.append(orc.linear_i8(Xq, sx, orc.pack(Wq, "i8", mask), sw))
        Xqs.append(to_dev(Xq, "i8"))
        sxs.append(torch.from_numpy(sx).cuda())
        Wcs.append(spl.pack_sparse(to_dev(Wq, "i8"), torch.from_numpy(mask).cuda()))
        sws.append(torch.from_numpy(sw).cuda())
        dense.append(to_dev(np.where(mask.astype(bool), Wq, np.int8(0)), "i8"))
    accs = [torch.empty((M, N), dtype=torch.int32, device="cuda") for N, _, _ in shapes]
    outs = spl.sparse_linear_int8_group(Xqs, sxs, Wcs, sws, acc_outs=accs)
    daccs = [torch.empty((M, N), dtype=torch.int32, device="cuda") for N, _, _ in shapes]
    douts = spl.dense_linear_int8_group(Xqs, sxs, dense, sws, acc_outs=daccs)
    for i, (acc_ref, y_ref) in enumerate(refs):
        for what, acc, y in (("sparse", accs[i], outs[i]), ("dense", daccs[i], douts[i])):
            _assert_equal(acc.cpu().numpy(), acc_ref, f"{what} group task {i} acc M={M}")
            _assert_equal(y.cpu().view(torch.int16).numpy().view(np.uint16), y_ref, f"{what} group task {i} Y M={M}")
        single = spl.sparse_linear_int8(Xqs[i], sxs[i], Wcs[i], sws[i])
        assert torch.equal(single.view(torch.int16), outs[i].view(torch.int16))


PREFILL_I8_M = [128, 129, 300]


def _sample_rows(M, seed, count=62):
    rows = np.concatenate([[0, M - 1], np.random.default_rng(seed).choice(np.arange(1, M - 1), count, replace=False)])
    return np.sort(rows)


@pytest.mark.parametrize("N,K,s", [(1, 16, 0.5), (33, 64, 0.7), (130, 1008, 0.7), (64, 4096, 0.5), (200, 336, 0.0),
                                   (17, 512, 1.0), (48, 2064, 0.9), (300, 144, 0.5)])
def test_int8_prefill_small(orc, spl, N, K, s):
    """Batches of 128 rows and more take the MFMA-tiled prefill kernel: ragged
    N, M and K (a partial last 128-byte stage) compared in full, bit for bit."""
    Wq, mask, sw = synth.int8_weight(620 + N, N, K, s)
    Xq, sx = synth.int8_activations(720 + K, max(PREFILL_I8_M), K)
    p = orc.pack(Wq, "i8", mask)
    for M in PREFILL_I8_M:
        acc_ref, y_ref = orc.linear_i8(Xq[:M], sx[:M], p, sw)
        acc, y = _run_sparse(spl, Xq[:M], sx[:M], Wq, mask, sw)
        _assert_equal(acc, acc_ref, f"acc N={N} K={K} s={s} M={M}")
        _assert_equal(y, y_ref, f"Y N={N} K={K} s={s} M={M}")


def _run_dense(spl, Xq, sx, Wd, sw):
    import torch

    M, N = Xq.shape[0], Wd.shape[0]
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    Y = spl.dense_linear_int8(to_dev(Xq, "i8"), torch.from_numpy(sx).cuda(), to_dev(Wd, "i8"),
                              torch.from_numpy(sw).cuda(), acc_out=acc)
    return acc.cpu().numpy(), Y.cpu().view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("N,K,M,s", [(2000, 144, 4100, 0.7), (2048, 128, 8192, 0.7), (256, 256, 256, 0.5)])
def test_int8_prefill_grids(orc, spl, N, K, M, s):
    """A ragged grid of at least one 128 x 256 block per CU, an aligned grid of
    two blocks per CU (branch-free loads) and an aligned grid small enough to
    split the reduction in two: compared in full, sparse and dense."""
    Wq, mask, sw = synth.int8_weight(950 + N, N, K, s)
    Xq, sx = synth.int8_activations(951 + K, M, K)
    acc_ref, y_ref = orc.linear_i8(Xq, sx, orc.pack(Wq, "i8", mask), sw)
    acc, y = _run_sparse(spl, Xq, sx, Wq, mask, sw)
    _assert_equal(acc, acc_ref, f"acc N={N} K={K} M={M}")
    _assert_equal(y, y_ref, f"Y N={N} K={K} M={M}")
    acc, y = _run_dense(spl, Xq, sx, np.where(mask.astype(bool), Wq, np.int8(0)), sw)
    _assert_equal(acc, acc_ref, f"dense acc N={N} K={K} M={M}")
    _assert_equal(y, y_ref, f"dense Y N={N} K={K} M={M}")


@pytest.mark.parametrize("name,M,s", [("q", 512, 0.7), ("gate", 512, 0.7), ("down", 512, 0.7), ("up", 2048, 0.5),
                                      ("o", 2048, 0.7), ("down", 2048, 0.7), ("down", 2048, 0.5)])
def test_int8_prefill_llama_shapes_sampled(orc, spl, name, M, s):
    """Llama-2-7B shapes at the prefill batch sizes: every output of 64 rows
    (the first, the last and 62 seeded ones) equals the oracle bit for bit;
    the rows are independent, so the oracle runs on those rows alone."""
    j = [n for n, _, _ in synth.LLAMA2_7B_LINEARS].index(name)
    _, N, K = synth.LLAMA2_7B_LINEARS[j]
    Wq, mask, sw = synth.int8_weight(synth.weight_seed(0, j), N, K, s)
    Xq, sx = synth.int8_activations(synth.activation_seed(j), M, K)
    rows = _sample_rows(M, N + M)
    acc_ref, y_ref = orc.linear_i8(Xq[rows], sx[rows], orc.pack(Wq, "i8", mask), sw)
    acc, y = _run_sparse(spl, Xq, sx, Wq, mask, sw)
    _assert_equal(acc[rows], acc_ref, f"{name} acc M={M}")
    _assert_equal(y[rows], y_ref, f"{name} Y M={M}")


def test_dense_int8_prefill(orc, spl):
    """The dense int8 comparator at prefill batch sizes: ragged shapes in full,
    the gate shape at M = 512 on 64 sampled rows."""
    rng = np.random.default_rng(77)
    for N, K in ((100, 1008), (130, 272), (16, 64)):
        Wq = rng.integers(-128, 128, size=(N, K)).astype(np.int8)
        sw = rng.uniform(1e-4, 1e-2, size=N).astype(np.float32)
        Xq, sx = synth.int8_activations(78, 300, K)
        for M in (128, 129, 300):
            acc_ref, y_ref = orc.dense_i8(Xq[:M], sx[:M], Wq, sw)
            acc, y = _run_dense(spl, Xq[:M], sx[:M], Wq, sw)
            _assert_equal(acc, acc_ref, f"dense acc N={N} K={K} M={M}")
            _assert_equal(y, y_ref, f"dense Y N={N} K={K} M={M}")
    N, K, M = 11008, 4096, 512
    Wq = rng.integers(-128, 128, size=(N, K)).astype(np.int8)
    sw = rng.uniform(1e-4, 1e-2, size=N).astype(np.float32)
    Xq, sx = synth.int8_activations(79, M, K)
    rows = _sample_rows(M, 80)
    acc_ref, y_ref = orc.dense_i8(Xq[rows], sx[rows], Wq, sw)
    acc, y = _run_dense(spl, Xq, sx, Wq, sw)
    _assert_equal(acc[rows], acc_ref, "dense gate acc M=512")
    _assert_equal(y[rows], y_ref, "dense gate Y M=512")


@pytest.mark.parametrize("N,K,M,s", [(100, 1008, 70, 0.7), (130, 272, 300, 0.5), (2000, 144, 4100, 0.7),
                                     (33, 512, 1, 1.0)])
def test_int8_expanded(orc, spl, N, K, M, s):
    """The decoded-copy int8 path: int32 sums and fp16 outputs bit for bit the
    oracle's in full (ragged shapes, a large ragged grid, one row, an
    all-pruned matrix) and bit for bit spl_sparse_linear_int8's."""
    import torch

    Wq, mask, sw = synth.int8_weight(990 + N, N, K, s)
    Xq, sx = synth.int8_activations(991 + K, M, K)
    acc_ref, y_ref = orc.linear_i8(Xq, sx, orc.pack(Wq, "i8", mask), sw)
    Wqc = spl.pack_sparse(to_dev(Wq, "i8"), torch.from_numpy(mask).cuda())
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    Xd, sxd, swd = to_dev(Xq, "i8"), torch.from_numpy(sx).cuda(), torch.from_numpy(sw).cuda()
    Y = spl.sparse_linear_int8_expanded(Xd, sxd, Wqc, swd, acc_out=acc)
    _assert_equal(acc.cpu().numpy(), acc_ref, f"expanded acc N={N} K={K} M={M}")
    _assert_equal(Y.cpu().view(torch.int16).numpy().view(np.uint16), y_ref, f"expanded Y N={N} K={K} M={M}")
    Y2 = spl.sparse_linear_int8(Xd, sxd, Wqc, swd)
    assert torch.equal(Y.view(torch.int16), Y2.view(torch.int16))


@pytest.mark.parametrize("name", ["gate", "down"])
def test_int8_expanded_and_dense_llama_rows(orc, spl, name):
    """Llama-2-7B gate and down at 70% and M = 2048 (the direct-to-LDS dense
    int8 core on the decoded codes, and on the dense codes for the comparator):
    64 full rows bit for bit."""
    import torch

    j = [n for n, _, _ in synth.LLAMA2_7B_LINEARS].index(name)
    _, N, K = synth.LLAMA2_7B_LINEARS[j]
    M = 2048
    Wq, mask, sw = synth.int8_weight(synth.weight_seed(0, j), N, K, 0.7)
    Xq, sx = synth.int8_activations(synth.activation_seed(j), M, K)
    rows = _sample_rows(M, 31 + j)
    acc_ref, y_ref = orc.linear_i8(Xq[rows], sx[rows], orc.pack(Wq, "i8", mask), sw)
    Wqc = spl.pack_sparse(to_dev(Wq, "i8"), torch.from_numpy(mask).cuda())
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    Y = spl.sparse_linear_int8_expanded(to_dev(Xq, "i8"), torch.from_numpy(sx).cuda(), Wqc,
                                        torch.from_numpy(sw).cuda(), acc_out=acc)
    _assert_equal(acc.cpu().numpy()[rows], acc_ref, f"{name} expanded acc")
    _assert_equal(Y.cpu().view(torch.int16).numpy().view(np.uint16)[rows], y_ref, f"{name} expanded Y")
    Wm = np.where(mask.astype(bool), Wq, np.zeros_like(Wq))
    dacc, dy = _run_dense(spl, Xq, sx, Wm, sw)
    _assert_equal(dacc[rows], acc_ref, f"{name} dense acc")
    _assert_equal(dy[rows], y_ref, f"{name} dense Y")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("M,K", [(1, 8), (3, 520), (5, 6000), (3, 20000), (300, 4096), (17, 11008), (2048, 11008)])
def test_quantize_rows_matches_oracle(orc, spl, dtype, M, K):
    """Per-token activation quantisation on the GPU: codes and scales bit for
    bit equal to the oracle's, with a zero row, rows of exact ties and rows of
    large magnitude mixed in."""
    rng = np.random.default_rng(M + K)
    v = (rng.standard_normal((M, K)) * rng.uniform(0.05, 20.0, (M, 1))).astype(np.float32)
    if M >= 3:
        v[1] = 0.0
        v[2] = np.resize(np.array([127, 2.5, 3.5, -2.5, 126.5, -0.5, 1.5, 0.25], np.float32), K)
    X = synth.round_to(v, dtype)
    ref_q, ref_s = orc.quantize_rows_i8(X, dtype)
    q, s = spl.quantize_rows_i8(to_dev(X, dtype))
    assert np.array_equal(s.cpu().numpy().view(np.uint32), ref_s.view(np.uint32)), "scales differ"
    assert np.array_equal(q.cpu().numpy(), ref_q), "codes differ"
