"""Prefill-shaped (large batch) sparse and dense fp16/bf16 linear layers on the
GPU vs the oracle.

Tolerance (fp16/bf16 outputs): |y - y64| <= max(2e-2, 1e-2 |y64|) per element.
Small shapes span several output blocks (64 x 128 for launches that would
leave CUs idle, 128 x 256 otherwise) with ragged edges in N, M and K and are
compared in full; every Llama-2-7B matrix at both sparsities and the batch
sizes of the prefill workloads (M = 512, 2048) is compared on 64 full rows,
and the q matrix at M = 512 in full."""
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


def _pack(spl, W, mask, dtype):
    import torch

    return spl.pack_sparse(to_dev(W, dtype), torch.from_numpy(mask).cuda())


PREFILL_M = [1, 16, 33, 64, 127, 128, 129, 300]


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,s", [(1, 8, 0.5), (16, 32, 0.5), (65, 72, 0.7), (130, 1000, 0.7), (64, 4096, 0.5),
                                   (200, 328, 0.0), (33, 512, 1.0), (17, 264, 0.9)])
def test_prefill_small(orc, spl, dtype, N, K, s):
    W, mask = synth.weight(400 + N, N, K, dtype, s)
    X = synth.activations(500 + K, max(PREFILL_M), K, dtype)
    ref_p = orc.pack(W, dtype, mask)
    Wc = _pack(spl, W, mask, dtype)
    Xd = to_dev(X, dtype)
    ref = orc.linear_f64(X, ref_p)
    for M in PREFILL_M:
        Y = spl.sparse_linear(Xd[:M].contiguous(), Wc, algo="prefill")
        assert_close(from_dev_f64(Y), ref[:M], f"prefill {dtype} N={N} K={K} s={s} M={M}")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_prefill_exact_arithmetic(orc, spl, dtype):
    rng = np.random.default_rng(23)
    N, K, M = 150, 1064, 200
    wi = rng.integers(-15, 16, size=(N, K))
    xi = rng.integers(-3, 4, size=(M, K))
    W = synth.round_to((wi / 64.0).astype(np.float32), dtype)
    X = synth.round_to(xi.astype(np.float32), dtype)
    mask = (rng.random((N, K)) < 0.35).astype(np.uint8)
    ref = orc.linear_f64(X, orc.pack(W, dtype, mask))      # exact: all partial sums are multiples of 2^-6
    expect = synth.round_to(ref.astype(np.float32), dtype)
    Y = spl.sparse_linear(to_dev(X, dtype), _pack(spl, W, mask, dtype), algo="prefill")
    norm = lambda a: np.where(a == 0x8000, np.uint16(0), a)   # +0 == -0
    assert np.array_equal(norm(from_dev_bits(Y)), norm(expect))


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_prefill_identity_activations(spl, dtype):
    N, K = 70, 96                                      # X = I_K -> Y = (W . Mask)^T, bit for bit
    W, mask = synth.weight(78, N, K, dtype, 0.6)
    X = synth.round_to(np.eye(K, dtype=np.float32), dtype)
    Y = spl.sparse_linear(to_dev(X, dtype), _pack(spl, W, mask, dtype), algo="prefill")
    norm = lambda a: np.where(a == 0x8000, 0, a)
    assert np.array_equal(norm(from_dev_bits(Y)), norm(np.where(mask.astype(bool), W, np.uint16(0)).T))


def _sample(rng, M, N, count):
    """Sampled output positions: the four corners, the block edges, random interior points."""
    ms = [0, 0, M - 1, M - 1, 127, 128, M // 2]
    ns = [0, N - 1, 0, N - 1, 63, 64, N // 2]
    ms += list(rng.integers(0, M, size=count))
    ns += list(rng.integers(0, N, size=count))
    return np.array(ms, dtype=np.int64), np.array(ns, dtype=np.int64)


def _sample_rows(M, seed, count=62):
    """Row 0, row M - 1 and `count` seeded rows between them."""
    rows = np.concatenate([[0, M - 1], np.random.default_rng(seed).choice(np.arange(1, M - 1), count, replace=False)])
    return np.sort(rows)


@pytest.mark.parametrize("s", [0.5, 0.7])
@pytest.mark.parametrize("name", [n for n, _, _ in synth.LLAMA2_7B_LINEARS])
def test_prefill_llama_shapes_rows(orc, spl, name, s):
    """Every Llama-2-7B matrix at both sparsities and both prefill batches
    (M = 512, 2048; the launch the auto choice takes): every output of 64
    rows (the first, the last and 62 seeded ones) within the tolerance, and
    the q matrix at M = 512 in full.  Rows are independent, so the oracle
    runs on the sampled rows alone."""
    j = [n for n, _, _ in synth.LLAMA2_7B_LINEARS].index(name)
    _, N, K = synth.LLAMA2_7B_LINEARS[j]
    W, mask = synth.weight(synth.weight_seed(0, j), N, K, "bf16", s)
    X = synth.activations(synth.activation_seed(j), 2048, K, "bf16")
    ref_p = orc.pack(W, "bf16", mask)
    Wc = _pack(spl, W, mask, "bf16")
    Xd = to_dev(X, "bf16")
    for M in (512, 2048):
        Y = from_dev_f64(spl.sparse_linear(Xd[:M].contiguous(), Wc))
        assert np.isfinite(Y).all()
        if name == "q" and M == 512:
            assert_close(Y, orc.linear_f64(X[:M], ref_p), f"{name} M={M} s={s} (all rows)")
        else:
            rows = _sample_rows(M, N + K + M)
            assert_close(Y[rows], orc.linear_f64(X[rows], ref_p), f"{name} M={M} s={s} (64 rows)")


def test_prefill_matches_decode_where_both_apply(orc, spl):
    W, mask = synth.weight(61, 300, 1024, "bf16", 0.7)
    X = synth.activations(62, 32, 1024, "bf16")
    Wc = _pack(spl, W, mask, "bf16")
    Xd = to_dev(X, "bf16")
    ref = orc.linear_f64(X, orc.pack(W, "bf16", mask))
    for algo in ("decode", "prefill"):
        assert_close(from_dev_f64(spl.sparse_linear(Xd, Wc, algo=algo)), ref, algo)


def test_prefill_deterministic_and_overwrites(spl):
    import torch

    W, mask = synth.weight(9, 300, 2048, "bf16", 0.7)
    X = synth.activations(10, 130, 2048, "bf16")
    Wc = _pack(spl, W, mask, "bf16")
    Xd = to_dev(X, "bf16")
    buf = torch.full((130 * 300 + 64,), float("nan"), dtype=torch.bfloat16, device="cuda")
    Y1 = buf[: 130 * 300].view(130, 300)
    spl.sparse_linear(Xd, Wc, out=Y1, algo="prefill")
    assert not torch.isnan(Y1).any()
    assert torch.isnan(buf[130 * 300:]).all()
    Y2 = spl.sparse_linear(Xd, Wc, algo="prefill")
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K", [(16, 64), (100, 1000), (130, 264)])
def test_dense_prefill_small(orc, spl, dtype, N, K):
    W, _ = synth.weight(910 + N, N, K, dtype, 0.0)
    X = synth.activations(911, 300, K, dtype)
    ref = orc.dense_f64(X, W, dtype)
    Wd = to_dev(W, dtype)
    Xd = to_dev(X, dtype)
    for M in (1, 64, 129, 300):
        Y = spl.dense_linear(Xd[:M].contiguous(), Wd, algo="prefill")
        assert_close(from_dev_f64(Y), ref[:M], f"dense prefill {dtype} M={M}")


def test_dense_prefill_llama_sampled(orc, spl):
    N, K, M = 11008, 4096, 512
    W, mask = synth.weight(912, N, K, "bf16", 0.0)
    X = synth.activations(913, M, K, "bf16")
    Y = spl.dense_linear(to_dev(X, "bf16"), to_dev(W, "bf16"))
    ms, ns = _sample(np.random.default_rng(5), M, N, 3000)
    ref = orc.linear_f64_pairs(X, orc.pack(W, "bf16", mask), ms, ns)   # all-ones mask: the dense product
    assert_close(from_dev_f64(Y)[ms, ns], ref, "dense prefill gate M=512")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K", [(4096, 4096), (4096, 11008)])
def test_dense_prefill_llama_rows(orc, spl, dtype, N, K):
    """The dense comparator at M = 2048 on Llama-2-7B shapes (the direct-to-LDS
    core: every block and stage inside, 64 or 172 stages through three
    rotating buffers): 64 full rows against the oracle."""
    M = 2048
    W, _ = synth.weight(914 + K, N, K, dtype, 0.0)
    X = synth.activations(915 + K, M, K, dtype)
    Y = from_dev_f64(spl.dense_linear(to_dev(X, dtype), to_dev(W, dtype), algo="prefill"))
    rows = _sample_rows(M, 17 + K)
    assert_close(Y[rows], orc.dense_f64(X[rows], W, dtype), f"dense prefill {dtype} {N}x{K} M={M}")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,M,s", [(100, 1000, 70, 0.7), (300, 264, 300, 0.5), (2000, 72, 4100, 0.7),
                                     (33, 512, 1, 1.0)])
def test_sparse_linear_expanded(orc, spl, dtype, N, K, M, s):
    """The decoded-copy path against the oracle in full (ragged shapes, a
    large grid, one row, an all-pruned matrix), and bit for bit the dense
    prefill kernel on spl_unpack's output."""
    import torch

    W, mask = synth.weight(980 + N, N, K, dtype, s)
    X = synth.activations(981 + K, M, K, dtype)
    Wc = _pack(spl, W, mask, dtype)
    Xd = to_dev(X, dtype)
    Y = spl.sparse_linear_expanded(Xd, Wc)
    assert_close(from_dev_f64(Y), orc.linear_f64(X, orc.pack(W, dtype, mask)), f"expanded {dtype} {N}x{K} M={M}")
    Yd = spl.dense_linear(Xd, spl.unpack(Wc), algo="prefill")
    assert torch.equal(Y.view(torch.int16), Yd.view(torch.int16))


@pytest.mark.parametrize("name,j", [("gate", 4), ("down", 6)])
def test_sparse_linear_expanded_llama_rows(orc, spl, name, j):
    """Llama-2-7B gate and down at 70% and M = 2048 (the direct-to-LDS dense
    core on the decoded copy, one workspace reused): 64 full rows."""
    import torch

    _, N, K = synth.LLAMA2_7B_LINEARS[j]
    M = 2048
    W, mask = synth.weight(synth.weight_seed(0, j), N, K, "bf16", 0.7)
    X = synth.activations(synth.activation_seed(j), M, K, "bf16")
    Wc = _pack(spl, W, mask, "bf16")
    ws = torch.empty((2 * 11008 * 4096,), dtype=torch.uint8, device="cuda")
    Y = from_dev_f64(spl.sparse_linear_expanded(to_dev(X, "bf16"), Wc, workspace=ws))
    rows = _sample_rows(M, 23 + j)
    assert_close(Y[rows], orc.linear_f64(X[rows], orc.pack(W, "bf16", mask)), f"expanded {name} M={M}")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_prefill_large_grid_ragged(orc, spl, dtype):
    """A grid of at least one 128 x 256 block per CU (the large tiling) with
    ragged N, M and an odd number of 32-column steps, compared in full, sparse
    and dense."""
    N, K, M, s = 2000, 72, 4100, 0.7          # 16 x 17 = 272 workgroups of 128 x 256
    W, mask = synth.weight(930, N, K, dtype, s)
    X = synth.activations(931, M, K, dtype)
    ref = orc.linear_f64(X, orc.pack(W, dtype, mask))
    Xd = to_dev(X, dtype)
    Y = spl.sparse_linear(Xd, _pack(spl, W, mask, dtype), algo="prefill")
    assert_close(from_dev_f64(Y), ref, f"prefill {dtype} N={N} K={K} M={M}")
    Wm = np.where(mask.astype(bool), W, np.zeros_like(W))
    Yd = spl.dense_linear(Xd, to_dev(Wm, dtype), algo="prefill")
    assert_close(from_dev_f64(Yd), ref, f"dense prefill {dtype} N={N} K={K} M={M}")


@pytest.mark.parametrize("N,K,M", [(2048, 128, 8192), (256, 192, 256)])
def test_prefill_aligned_grids(orc, spl, N, K, M):
    """Launches whose blocks and stages all lie inside the matrix take the
    unchecked (branch-free) kernels: a 128 x 256 grid with two blocks per CU
    and a 64 x 128 grid, compared in full, sparse and dense."""
    W, mask = synth.weight(940 + N, N, K, "bf16", 0.7)
    X = synth.activations(941 + K, M, K, "bf16")
    ref = orc.linear_f64(X, orc.pack(W, "bf16", mask))
    Xd = to_dev(X, "bf16")
    Y = spl.sparse_linear(Xd, _pack(spl, W, mask, "bf16"), algo="prefill")
    assert_close(from_dev_f64(Y), ref, f"prefill N={N} K={K} M={M}")
    Wm = np.where(mask.astype(bool), W, np.zeros_like(W))
    Yd = spl.dense_linear(Xd, to_dev(Wm, "bf16"), algo="prefill")
    assert_close(from_dev_f64(Yd), ref, f"dense prefill N={N} K={K} M={M}")
