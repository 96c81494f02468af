"""Sparse training with the mask held fixed (Algorithm 1) on the GPU vs the
oracle: the transposes and the gather into a tile pattern are data movement
(bit for bit); the weight gradient (fp32 sums over M, one rounding) and the
input gradient (the sparse linear layer on the packed transpose) are checked
with |y - y64| <= max(2e-2, 1e-2 |y64|); one SGD step (binary32 product and
difference, one rounding) within 2^-8 |y64| (bf16) / 2^-11 |y64| (fp16), plus
2^-22 (|w| + lr |g|) for the binary32 steps and the smallest normal of the
payload type."""
import ctypes

import numpy as np
import pytest

import synth
from tests._helpers import assert_close, from_dev_bits, from_dev_f64, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def spl():
    import paper_2405_03594_amd as spl

    spl.lib()
    return spl


def _with_values(spl, Wc, values):
    return spl.SparseMatrix(Wc.bitmask, values, None, Wc.tile_offsets, Wc.rows, Wc.cols, Wc.nnz, "tile16")


@pytest.mark.parametrize("R,C", [(1, 1), (3, 70), (65, 129), (16, 12), (8, 8), (72, 520), (136, 24), (1000, 4096),
                                 (4096, 64), (2048, 11008)])
def test_transpose16(spl, R, C):
    """Both kernels: 8 x 8 register blocks when R and C are multiples of 8
    (whole and partial 64 x 256 workgroup tiles), LDS tiles otherwise."""
    A = np.random.default_rng(R * C).integers(0, 1 << 16, size=(R, C), dtype=np.uint16)
    got = from_dev_bits(spl.transpose16(to_dev(A, "bf16")))
    assert np.array_equal(got, A.T)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,s", [(1, 8, 0.5), (17, 72, 0.7), (100, 1000, 0.0), (300, 264, 0.9), (33, 512, 1.0)])
def test_gather_tiled_matches_oracle_encoder(orc, spl, dtype, N, K, s):
    """Gathering a dense matrix at W's pattern gives the oracle's tile-layout
    values of that matrix under W's mask: for W itself and for another dense
    matrix (a gradient's role), whose entries at pruned positions must not
    leak in."""
    import torch

    W, mask = synth.weight(600 + N, N, K, dtype, s)
    D, _ = synth.weight(700 + N, N, K, dtype, 0.0)
    Wc = spl.pack_sparse(to_dev(W, dtype), torch.from_numpy(mask).cuda())
    for name, A in (("W", W), ("D", D)):
        got = from_dev_bits(spl.gather_tiled(to_dev(A, dtype), Wc))[:Wc.nnz]
        assert np.array_equal(got, orc.pack_tiled(A, dtype, mask).values), name


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,M,s", [(24, 64, 16, 0.6), (100, 1000, 64, 0.7), (300, 264, 136, 0.5), (33, 512, 8, 0.9),
                                     (130, 96, 520, 0.7), (2000, 4104, 72, 0.7)])
def test_weight_grad(orc, spl, dtype, N, K, M, s):
    """Small products (64 x 128 workgroups, split over M when they leave CUs
    idle) and a ragged large one (128 x 256 workgroups, bounds-checked loads:
    4104 columns, 2000 rows), compared with the oracle on every kept entry."""
    import torch

    W, mask = synth.weight(610 + N, N, K, dtype, s)
    X = synth.activations(611 + K, M, K, dtype)
    dY = synth.activations(612 + M, M, N, dtype)
    Wc = spl.pack_sparse(to_dev(W, dtype), torch.from_numpy(mask).cuda())
    g = spl.sparse_weight_grad(to_dev(dY, dtype), to_dev(X, dtype), Wc)
    G = from_dev_f64(spl.unpack(_with_values(spl, Wc, g)))
    ref = orc.weight_grad_f64(dY, X, dtype, orc.pack(W, dtype, mask))
    assert_close(G, ref, f"weight grad {dtype} N={N} K={K} M={M}")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,M,s", [(1024, 8192, 64, 0.7), (1024, 8192, 192, 0.5), (2048, 4096, 128, 0.9),
                                     (2048, 4096, 320, 0.7)])
def test_weight_grad_contraction_major(orc, spl, dtype, N, K, M, s):
    """Shapes whose weight gradient is read straight from dY and X (the
    token as the row of both; no transposed copies): N % 256, K % 128 and
    M % 64 zero and one 128 x 256 block per CU, over one, two, three and five
    64-token stages (the three stage buffers used once, and rotated), every
    kept entry compared with the oracle."""
    import torch

    W, mask = synth.weight(620 + N, N, K, dtype, s)
    X = synth.activations(621 + M, M, K, dtype)
    dY = synth.activations(622 + M, M, N, dtype)
    Wc = spl.pack_sparse(to_dev(W, dtype), torch.from_numpy(mask).cuda())
    g = spl.sparse_weight_grad(to_dev(dY, dtype), to_dev(X, dtype), Wc)
    G = from_dev_f64(spl.unpack(_with_values(spl, Wc, g)))
    ref = orc.weight_grad_f64(dY, X, dtype, orc.pack(W, dtype, mask))
    assert_close(G, ref, f"weight grad {dtype} N={N} K={K} M={M}")


def test_weight_grad_direct_path_and_fallback_agree(orc, spl):
    """The same product through both paths: with 16-byte aligned dY and X the
    weight gradient reads them as stored and leaves the workspace untouched;
    with X 8 bytes off that alignment (a view into a larger buffer) it
    transposes both into the workspace first.  Both match the oracle on every
    kept entry, and they agree bit for bit (the same 128 x 256 blocks, the
    same MFMA operands in the same token order)."""
    import torch

    N, K, M = 2048, 4096, 128
    W, mask = synth.weight(630, N, K, "bf16", 0.7)
    X = synth.activations(631, M, K, "bf16")
    dY = synth.activations(632, M, N, "bf16")
    Wc = spl.pack_sparse(to_dev(W, "bf16"), torch.from_numpy(mask).cuda())
    dYd, Xd = to_dev(dY, "bf16"), to_dev(X, "bf16")
    nws = spl.lib().spl_sparse_weight_grad_workspace_bytes(M, N, K)
    ws = torch.full((nws,), 0xA5, dtype=torch.uint8, device="cuda")
    g_direct = spl.sparse_weight_grad(dYd, Xd, Wc, workspace=ws)
    torch.cuda.synchronize()
    assert bool((ws == 0xA5).all()), "the direct path wrote to the workspace"
    flat = torch.empty((M * K + 4,), dtype=Xd.dtype, device="cuda")
    Xu = flat[4:].view(M, K)
    Xu.copy_(Xd)
    assert Xu.data_ptr() % 16 == 8
    g_fallback = spl.sparse_weight_grad(dYd, Xu, Wc, workspace=ws)
    torch.cuda.synchronize()
    assert not bool((ws == 0xA5).all()), "the fallback path did not use the workspace"
    ref = orc.weight_grad_f64(dY, X, "bf16", orc.pack(W, "bf16", mask))
    for g, name in ((g_direct, "direct"), (g_fallback, "fallback")):
        G = from_dev_f64(spl.unpack(_with_values(spl, Wc, g)))
        assert_close(G, ref, f"weight grad ({name} path)")
    n = Wc.nnz                                         # the buffers' tails past nnz are never written
    assert torch.equal(g_direct[:n].view(torch.int16), g_fallback[:n].view(torch.int16))


def test_weight_grad_group_matches_single_calls(orc, spl):
    """q, k, v (one X, three dY) at M = 256 and gate, up at M = 128, each
    group in one call (one launch: every task reads its factors as stored):
    the kept entries equal the single calls' bit for bit, and q's and gate's
    equal the oracle within tolerance.  A group with a task the direct path
    does not take (2000 x 4104) runs task by task and equals the single calls
    too, and so does a group of five (two launches of the grouped core)."""
    import torch

    def task(j, N, K, M, seed):
        W, mask = synth.weight(seed, N, K, "bf16", 0.7)
        Wc = spl.pack_sparse(to_dev(W, "bf16"), torch.from_numpy(mask).cuda())
        dY = synth.activations(seed + 1, M, N, "bf16")
        return W, mask, Wc, dY

    for shapes, M in (([(4096, 4096)] * 3, 256), ([(11008, 4096)] * 2, 128), ([(2048, 4096), (2000, 4104)], 128),
                      ([(2048, 4096)] * 5, 64)):                     # five tasks: two launches (four, then one)
        Ks = {K for _, K in shapes}
        Xh = {K: synth.activations(690 + K, M, K, "bf16") for K in Ks}
        Xd = {K: to_dev(Xh[K], "bf16") for K in Ks}
        ts = [task(j, N, K, M, 700 + 10 * j + N) for j, (N, K) in enumerate(shapes)]
        dYd = [to_dev(t[3], "bf16") for t in ts]
        outs = spl.sparse_weight_grad_group(dYd, [Xd[K] for _, K in shapes], [t[2] for t in ts])
        for i, ((N, K), t) in enumerate(zip(shapes, ts)):
            single = spl.sparse_weight_grad(dYd[i], Xd[K], t[2])
            n = t[2].nnz
            assert torch.equal(outs[i][:n].view(torch.int16), single[:n].view(torch.int16)), (shapes, i)
        W, mask, Wc, dY = ts[0]
        G = from_dev_f64(spl.unpack(_with_values(spl, Wc, outs[0])))
        ref = orc.weight_grad_f64(dY, Xh[shapes[0][1]], "bf16", orc.pack(W, "bf16", mask))
        assert_close(G, ref, f"grouped weight grad {shapes[0]} M={M}")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_sgd_update(orc, spl, dtype):
    import torch

    N, K = 200, 528
    W, mask = synth.weight(620, N, K, dtype, 0.7)
    Wc = spl.pack_sparse(to_dev(W, dtype), torch.from_numpy(mask).cuda())
    w0 = orc.to_f64(from_dev_bits(Wc.values)[:Wc.nnz], dtype)
    G = synth.round_to(synth.normal_f32(621, (Wc.values.numel(),), 1.0), dtype)
    for lr in (0.01, 0.5):
        w = orc.to_f64(from_dev_bits(Wc.values)[:Wc.nnz], dtype)
        spl.sparse_sgd_update(Wc, to_dev(G, dtype), lr)
        got = orc.to_f64(from_dev_bits(Wc.values)[:Wc.nnz], dtype)
        g = orc.to_f64(G[:Wc.nnz], dtype)
        ref = orc.sgd_f64(w, g, lr)
        rel, tiny = (2.0 ** -8, 2.0 ** -126) if dtype == "bf16" else (2.0 ** -11, 2.0 ** -14)
        # + the binary32 rounding of lr * g and of the difference, relative to the operands
        tol = rel * np.abs(ref) + 2.0 ** -22 * (np.abs(w) + lr * np.abs(g)) + tiny
        assert (np.abs(got - ref) <= tol).all(), f"lr={lr}"
    assert not np.array_equal(got, w0)
    dense = from_dev_f64(spl.unpack(Wc))
    assert not dense[mask == 0].any()                  # pruned entries stay zero


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,M,s", [(104, 1000, 64, 0.7), (296, 264, 136, 0.5), (48, 520, 3, 0.9)])
def test_input_grad_via_packed_transpose(orc, spl, dtype, N, K, M, s):
    import torch

    W, mask = synth.weight(630 + N, N, K, dtype, s)
    dY = synth.activations(631 + M, M, N, dtype)
    Wc = spl.pack_sparse(to_dev(W, dtype), torch.from_numpy(mask).cuda())
    Wt = spl.pack_sparse(spl.transpose16(spl.unpack(Wc)))          # [K][N], the non-zero kept entries
    dX = from_dev_f64(spl.sparse_linear(to_dev(dY, dtype), Wt))       # N % 8 == 0: rows of dY in 16-byte pieces
    assert_close(dX, orc.input_grad_f64(dY, dtype, orc.pack(W, dtype, mask)), f"dX {dtype} N={N} K={K} M={M}")


@pytest.mark.parametrize("name,j,M", [("q", 0, 256), ("gate", 4, 128), ("down", 6, 64)])
def test_weight_grad_llama_shapes(orc, spl, name, j, M):
    import torch

    _, N, K = synth.LLAMA2_7B_LINEARS[j]
    W, mask = synth.weight(synth.weight_seed(0, j), N, K, "bf16", 0.7)
    X = synth.activations(synth.activation_seed(j), M, K, "bf16")
    dY = synth.activations(640 + j, M, N, "bf16")
    Wc = spl.pack_sparse(to_dev(W, "bf16"), torch.from_numpy(mask).cuda())
    g = spl.sparse_weight_grad(to_dev(dY, "bf16"), to_dev(X, "bf16"), Wc)
    G = from_dev_f64(spl.unpack(_with_values(spl, Wc, g)))
    ref = orc.to_f64(dY, "bf16").T @ orc.to_f64(X, "bf16") * mask
    assert_close(G, ref, f"{name} weight grad M={M}")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,M,s", [(64, 8192, 1024, 0.7), (192, 16384, 512, 0.5), (320, 4096, 2048, 0.9),
                                     (128, 4096, 2048, 0.0)])
def test_input_grad_from_packed_tiles(orc, spl, dtype, N, K, M, s):
    """dX = dY (W.Mask) straight from W's tiles (no packed transpose, no
    workspace): shapes of one 128 x 256 block per CU over one, three, five
    (an odd count: the two-stage loop's tail) and two 64-row stages of W,
    every output compared with the oracle."""
    import torch

    W, mask = synth.weight(650 + N, N, K, dtype, s)
    dY = synth.activations(651 + M, M, N, dtype)
    Wc = spl.pack_sparse(to_dev(W, dtype), torch.from_numpy(mask).cuda())
    assert spl.lib().spl_sparse_input_grad_workspace_bytes(M, ctypes.byref(Wc.view())) == 0
    dX = from_dev_f64(spl.sparse_input_grad(to_dev(dY, dtype), Wc))
    assert_close(dX, orc.input_grad_f64(dY, dtype, orc.pack(W, dtype, mask)), f"dX {dtype} N={N} K={K} M={M}")


@pytest.mark.parametrize("N,K,M,s", [(104, 1000, 64, 0.7), (296, 264, 136, 0.5), (48, 520, 3, 0.9),
                                     (4096, 4096, 2000, 0.7)])
def test_input_grad_decoded_fallback(orc, spl, N, K, M, s):
    """Shapes the direct kernel does not take: W decoded and transposed into
    the workspace, then the dense product; compared with the oracle (every
    output, or 64 full rows at 4096 x 4096, M = 2000)."""
    import torch

    W, mask = synth.weight(660 + N, N, K, "bf16", s)
    dY = synth.activations(661 + M, M, N, "bf16")
    Wc = spl.pack_sparse(to_dev(W, "bf16"), torch.from_numpy(mask).cuda())
    assert spl.lib().spl_sparse_input_grad_workspace_bytes(M, ctypes.byref(Wc.view())) > 0
    dX = from_dev_f64(spl.sparse_input_grad(to_dev(dY, "bf16"), Wc))
    rows = np.arange(M) if M * K <= 1 << 22 else np.sort(np.concatenate(
        [[0, M - 1], np.random.default_rng(N).choice(np.arange(1, M - 1), 62, replace=False)]))
    ref = orc.input_grad_f64(dY[rows], "bf16", orc.pack(W, "bf16", mask))
    assert_close(dX[rows], ref, f"dX fallback N={N} K={K} M={M}")


def test_input_grad_edge_cases(spl):
    """No kept entry: dX = 0 on both paths; no tokens: nothing to do."""
    import torch

    for N, K, M in ((64, 8192, 1024), (40, 72, 24)):
        Wc = spl.pack_sparse(torch.zeros((N, K), dtype=torch.bfloat16, device="cuda"))
        assert Wc.nnz == 0
        dX = spl.sparse_input_grad(torch.ones((M, N), dtype=torch.bfloat16, device="cuda"), Wc,
                                   out=torch.full((M, K), 7.0, dtype=torch.bfloat16, device="cuda"))
        assert not bool(dX.any())
    W, mask = synth.weight(670, 64, 128, "bf16", 0.5)
    Wc = spl.pack_sparse(to_dev(W, "bf16"), torch.from_numpy(mask).cuda())
    out = spl.sparse_input_grad(torch.empty((0, 64), dtype=torch.bfloat16, device="cuda"), Wc)
    assert out.shape == (0, 128)


@pytest.mark.parametrize("name,j", [("q", 0), ("gate", 4), ("down", 6)])
def test_input_grad_llama_shapes(orc, spl, name, j):
    """The bench's training shapes at M = 2048 (the direct kernel): 64 full
    rows (0, M - 1 and 62 seeded) of dX against the oracle, and the same rows
    through the packed transpose (spl_sparse_linear on Wt) within the same
    tolerance."""
    import torch

    _, N, K = synth.LLAMA2_7B_LINEARS[j]
    M = 2048
    W, mask = synth.weight(synth.weight_seed(0, j), N, K, "bf16", 0.7)
    dY = synth.activations(680 + j, M, N, "bf16")
    md = torch.from_numpy(mask).cuda()
    Wc = spl.pack_sparse(to_dev(W, "bf16"), md)
    dYd = to_dev(dY, "bf16")
    dX = from_dev_f64(spl.sparse_input_grad(dYd, Wc))
    rng = np.random.default_rng(j)
    rows = np.sort(np.concatenate([[0, M - 1], rng.choice(np.arange(1, M - 1), 62, replace=False)]))
    ref = orc.input_grad_f64(dY[rows], "bf16", orc.pack(W, "bf16", mask))
    assert_close(dX[rows], ref, f"{name} dX M={M}")
    Wt = spl.pack_sparse(spl.transpose16(spl.unpack(Wc)), md.t().contiguous())
    dXt = from_dev_f64(spl.sparse_linear(dYd, Wt))
    assert_close(dXt[rows], ref, f"{name} dX via the packed transpose M={M}")


@pytest.mark.parametrize("N,K,s", [(8, 8, 0.5), (104, 1000, 0.7), (296, 264, 0.0), (64, 520, 0.9)])
def test_transpose_perm_keeps_the_transpose_in_step(orc, spl, N, K, s):
    """The packed transpose (transposed mask) refreshed by the permutation
    holds the oracle's tile-layout values of the transposed weights, for the
    packed weights and again after new values are written into them."""
    import torch

    W, mask = synth.weight(650 + N, N, K, "bf16", s)
    md = torch.from_numpy(mask).cuda()
    Wc = spl.pack_sparse(to_dev(W, "bf16"), md)
    mt = md.t().contiguous()
    Wt = spl.pack_sparse(spl.transpose16(spl.unpack(Wc)), mt)
    perm = spl.transpose_perm(Wc, Wt)
    D, _ = synth.weight(660 + N, N, K, "bf16", 0.0)        # the next weights (dense draw; pruned by the mask)
    for step, A in enumerate((W, D)):
        if step:
            Wc.values[:Wc.nnz].copy_(to_dev(orc.pack_tiled(A, "bf16", mask).values, "bf16"))
        out = torch.empty_like(Wt.values)
        spl.permute_values(Wc.values, perm, Wc.nnz, out)
        ref = orc.pack_tiled(np.ascontiguousarray(A.T), "bf16", np.ascontiguousarray(mask.T)).values
        assert np.array_equal(from_dev_bits(out)[:Wc.nnz], ref), step


@pytest.mark.parametrize("name,j", [("gate", 4), ("down", 6)])
def test_train_at_bench_size(orc, spl, name, j):
    """The bench's training configuration (M = 2048 tokens, 70%): the weight
    gradient at 3000 sampled kept positions (each sum over the 2048 tokens
    in binary64) and the input gradient on 64 sampled rows, through the packed
    transpose refreshed by the permutation."""
    import torch

    _, N, K = synth.LLAMA2_7B_LINEARS[j]
    M = 2048
    W, mask = synth.weight(synth.weight_seed(0, j), N, K, "bf16", 0.7)
    X = synth.activations(synth.activation_seed(j), M, K, "bf16")
    dY = synth.activations(700 + j, M, N, "bf16")
    md = torch.from_numpy(mask).cuda()
    Wc = spl.pack_sparse(to_dev(W, "bf16"), md)
    g = spl.sparse_weight_grad(to_dev(dY, "bf16"), to_dev(X, "bf16"), Wc)
    G = from_dev_f64(spl.unpack(_with_values(spl, Wc, g)))
    rng = np.random.default_rng(j)
    kept = np.argwhere(mask == 1)
    pick = kept[rng.choice(len(kept), 3000, replace=False)]
    x64, dy64 = orc.to_f64(X, "bf16"), orc.to_f64(dY, "bf16")
    ref = np.einsum("mi,mi->i", dy64[:, pick[:, 0]], x64[:, pick[:, 1]])
    assert_close(G[pick[:, 0], pick[:, 1]], ref, f"{name} weight grad M={M}")
    assert not G[mask == 0].any()
    Wt = spl.pack_sparse(spl.transpose16(spl.unpack(Wc)), md.t().contiguous())
    perm = spl.transpose_perm(Wc, Wt)
    spl.permute_values(Wc.values, perm, Wc.nnz, Wt.values)
    dX = from_dev_f64(spl.sparse_linear(to_dev(dY, "bf16"), Wt))
    rows = np.sort(np.concatenate([[0, M - 1], rng.choice(np.arange(1, M - 1), 62, replace=False)]))
    ref_dx = orc.input_grad_f64(dY[rows], "bf16", orc.pack(W, "bf16", mask))
    assert_close(dX[rows], ref_dx, f"{name} input grad M={M}")
