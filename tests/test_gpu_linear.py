"""fp16/bf16 sparse linear layers on the GPU vs the oracle.

Tolerance (fp16/bf16 outputs): |y - y64| <= max(2e-2, 1e-2 |y64|) per element.
Exact-arithmetic inputs and identity activations are compared bit for bit.
Both kernel families are forced for every batch size they accept."""
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


DECODE_M = [1, 2, 3, 4, 5, 8, 15, 16, 17, 31, 32]


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,s", [(1, 8, 0.5), (2, 16, 0.5), (15, 64, 0.7), (17, 264, 0.5), (100, 1000, 0.7),
                                   (48, 2056, 0.0), (33, 512, 1.0)])
def test_decode_small(orc, spl, dtype, N, K, s):
    W, mask = synth.weight(200 + N, N, K, dtype, s)
    X = synth.activations(300 + K, 32, K, dtype)
    ref_p = orc.pack(W, dtype, mask)
    Wc = _pack(spl, W, mask, dtype)
    Xd = to_dev(X, dtype)
    ref = orc.linear_f64(X, ref_p)
    for M in DECODE_M:
        Y = spl.sparse_linear(Xd[:M].contiguous(), Wc, algo="decode")
        assert_close(from_dev_f64(Y), ref[:M], f"decode {dtype} N={N} K={K} s={s} M={M}")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_decode_exact_arithmetic(orc, spl, dtype):
    rng = np.random.default_rng(17)
    N, K = 70, 1064
    wi = rng.integers(-15, 16, size=(N, K))
    xi = rng.integers(-3, 4, size=(32, K))
    W = synth.round_to((wi / 64.0).astype(np.float32), dtype)
    X = synth.round_to(xi.astype(np.float32), dtype)
    mask = (rng.random((N, K)) < 0.35).astype(np.uint8)
    ref_p = orc.pack(W, dtype, mask)
    Wc = _pack(spl, W, mask, dtype)
    ref = orc.linear_f64(X, ref_p)                     # exact: all partial sums are multiples of 2^-6
    expect = synth.round_to(ref.astype(np.float32), dtype)
    Xd = to_dev(X, dtype)
    for M in (1, 4, 16, 17, 32):
        Y = spl.sparse_linear(Xd[:M].contiguous(), Wc, algo="decode")
        got = from_dev_bits(Y)
        norm = lambda a: np.where(a == 0x8000, np.uint16(0), a)   # +0 == -0
        assert np.array_equal(norm(got), norm(expect[:M])), f"M={M}"


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_decode_identity_activations(orc, spl, dtype):
    N, K = 37, 32                                      # X = I_K (M = K = 32) -> Y = (W . Mask)^T
    W, mask = synth.weight(77, N, K, dtype, 0.6)
    X = synth.round_to(np.eye(K, dtype=np.float32), dtype)
    Wc = _pack(spl, W, mask, dtype)
    Y = spl.sparse_linear(to_dev(X, dtype), Wc, algo="decode")
    got = from_dev_bits(Y)
    expect = np.where(mask.astype(bool), W, np.uint16(0)).T
    norm = lambda a: np.where(a == 0x8000, 0, a)
    assert np.array_equal(norm(got), norm(expect))


CFG2 = [(name, N, K) for (name, N, K) in synth.LLAMA2_7B_LINEARS]


@pytest.mark.parametrize("name,N,K", CFG2[3:])      # o (4096x4096), gate, up, down
def test_decode_llama_shapes_bf16_70(orc, spl, name, N, K):
    j = [n for n, _, _ in synth.LLAMA2_7B_LINEARS].index(name)
    W, mask = synth.weight(synth.weight_seed(0, j), N, K, "bf16", 0.7)
    X = synth.activations(synth.activation_seed(j), 16, K, "bf16")
    ref_p = orc.pack(W, "bf16", mask)
    Wc = _pack(spl, W, mask, "bf16")
    ref = orc.linear_f64(X, ref_p)
    Xd = to_dev(X, "bf16")
    for M in (1, 4, 16):
        Y = spl.sparse_linear(Xd[:M].contiguous(), Wc)
        assert_close(from_dev_f64(Y), ref[:M], f"{name} M={M}")


def test_decode_cfg1_fp16_50(orc, spl):
    W, mask = synth.weight(0, 4096, 4096, "f16", 0.5)
    X = synth.activations(1, 1, 4096, "f16")
    ref = orc.linear_f64(X, orc.pack(W, "f16", mask))
    Wc = _pack(spl, W, mask, "f16")
    Y = spl.sparse_linear(to_dev(X, "f16"), Wc)
    assert_close(from_dev_f64(Y), ref, "cfg1")


def test_decode_deterministic_and_overwrites(orc, spl):
    import torch

    W, mask = synth.weight(5, 300, 2048, "bf16", 0.7)
    X = synth.activations(6, 7, 2048, "bf16")
    Wc = _pack(spl, W, mask, "bf16")
    Xd = to_dev(X, "bf16")
    buf = torch.full((7 * 300 + 64,), float("nan"), dtype=torch.bfloat16, device="cuda")
    Y1 = buf[: 7 * 300].view(7, 300)
    spl.sparse_linear(Xd, Wc, out=Y1)
    assert not torch.isnan(Y1).any()                  # every output written
    assert torch.isnan(buf[7 * 300:]).all()           # nothing written past Y
    Y2 = spl.sparse_linear(Xd, Wc)
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K", [(16, 64), (100, 1000), (4096, 4096)])
def test_dense_decode(orc, spl, dtype, N, K):
    W, _ = synth.weight(900 + N, N, K, dtype, 0.0)
    X = synth.activations(901, 32, K, dtype)
    ref = orc.dense_f64(X, W, dtype)
    Wd = to_dev(W, dtype)
    Xd = to_dev(X, dtype)
    for M in (1, 5, 16, 17, 32):
        Y = spl.dense_linear(Xd[:M].contiguous(), Wd, algo="decode")
        assert_close(from_dev_f64(Y), ref[:M], f"dense decode {dtype} M={M}")


def test_zero_batch_is_noop(spl):
    import torch

    W, mask = synth.weight(1, 8, 64, "bf16", 0.5)
    Wc = _pack(spl, W, mask, "bf16")
    Y = spl.sparse_linear(torch.empty((0, 64), dtype=torch.bfloat16, device="cuda"), Wc)
    assert Y.shape == (0, 8)


@pytest.mark.parametrize("M", [1, 4, 16, 17, 32])
def test_decode_group_matches_single_calls(orc, spl, M):
    """One launch over several matrices of different shapes (ragged N and K,
    an all-pruned matrix) gives each matrix the oracle's result, bit for bit
    the same as one call per matrix."""
    import torch

    shapes = [(100, 1000, 0.7), (48, 2056, 0.5), (17, 264, 0.9), (64, 4096, 0.7), (33, 512, 1.0), (16, 11008, 0.7)]
    Ws, refs, Xs = [], [], []
    for i, (N, K, s) in enumerate(shapes):
        W, mask = synth.weight(700 + i, N, K, "bf16", s)
        X = synth.activations(800 + i, M, K, "bf16")
        Ws.append(_pack(spl, W, mask, "bf16"))
        Xs.append(to_dev(X, "bf16"))
        refs.append(orc.linear_f64(X, orc.pack(W, "bf16", mask)))
    Ys = spl.sparse_linear_group(Xs, Ws, algo="decode")
    for i, (Y, ref) in enumerate(zip(Ys, refs)):
        assert_close(from_dev_f64(Y), ref, f"group task {i} M={M}")
        single = spl.sparse_linear(Xs[i], Ws[i], algo="decode")
        assert torch.equal(Y.view(torch.int16), single.view(torch.int16)), f"task {i}"


@pytest.mark.parametrize("M", [1, 4, 17])
def test_dense_decode_group(orc, spl, M):
    shapes = [(100, 1000), (48, 2056), (64, 4096), (16, 11008)]
    Ws, Xs, refs = [], [], []
    for i, (N, K) in enumerate(shapes):
        W, _ = synth.weight(720 + i, N, K, "f16", 0.0)
        X = synth.activations(820 + i, M, K, "f16")
        Ws.append(to_dev(W, "f16"))
        Xs.append(to_dev(X, "f16"))
        refs.append(orc.dense_f64(X, W, "f16"))
    for i, (Y, ref) in enumerate(zip(spl.dense_linear_group(Xs, Ws, algo="decode"), refs)):
        assert_close(from_dev_f64(Y), ref, f"dense group task {i} M={M}")


def test_prefill_group(orc, spl):
    Ws, Xs, refs = [], [], []
    for i, (N, K) in enumerate([(100, 1000), (130, 264)]):
        W, mask = synth.weight(740 + i, N, K, "bf16", 0.7)
        X = synth.activations(840 + i, 70, K, "bf16")
        Ws.append(_pack(spl, W, mask, "bf16"))
        Xs.append(to_dev(X, "bf16"))
        refs.append(orc.linear_f64(X, orc.pack(W, "bf16", mask)))
    for i, (Y, ref) in enumerate(zip(spl.sparse_linear_group(Xs, Ws), refs)):   # auto -> prefill at M = 70
        assert_close(from_dev_f64(Y), ref, f"prefill group task {i}")


@pytest.mark.parametrize("s", [0.7, 0.0])
def test_decode_long_rows(orc, spl, s):
    """K = 40960: each wave's range (80 tiles) outgrows one load of tile offsets."""
    N, K = 40, 40960
    W, mask = synth.weight(950, N, K, "bf16", s)
    X = synth.activations(951, 17, K, "bf16")
    ref = orc.linear_f64(X, orc.pack(W, "bf16", mask))
    Wc = _pack(spl, W, mask, "bf16")
    Xd = to_dev(X, "bf16")
    for M in (1, 5, 17):
        Y = spl.sparse_linear(Xd[:M].contiguous(), Wc, algo="decode")
        assert_close(from_dev_f64(Y), ref[:M], f"long rows s={s} M={M}")


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,M", [(8200, 1056, 16), (8200, 3296, 5), (8192, 2112, 9), (8200, 1056, 17),
                                   (8200, 3296, 32), (8192, 4096, 31)])
def test_decode_row_block_pairs(orc, spl, dtype, N, K, M):
    """Launches of at least 512 row blocks whose activations are loaded directly
    (M x K too large to stage in LDS) run two row blocks per workgroup, with
    one batch tile up to 16 rows and two above: an odd row-block count (8200
    rows = 512 blocks + a ragged 8-row block, the last pair half empty) and an
    even one, compared in full with the oracle, and as one task of a group
    with a smaller matrix."""
    W, mask = synth.weight(950 + M, N, K, dtype, 0.7)
    X = synth.activations(951, M, K, dtype)
    ref = orc.linear_f64(X, orc.pack(W, dtype, mask))
    Xd, Wc = to_dev(X, dtype), _pack(spl, W, mask, dtype)
    Y = spl.sparse_linear(Xd, Wc, algo="decode")
    assert_close(from_dev_f64(Y), ref, f"pairs {dtype} N={N} K={K} M={M}")
    W2, mask2 = synth.weight(952, 40, K, dtype, 0.5)
    ref2 = orc.linear_f64(X, orc.pack(W2, dtype, mask2))
    Y1, Y2 = spl.sparse_linear_group([Xd, Xd], [Wc, _pack(spl, W2, mask2, dtype)], algo="decode")
    assert_close(from_dev_f64(Y1), ref, f"pairs group task 0 {dtype} N={N} K={K} M={M}")
    assert_close(from_dev_f64(Y2), ref2, f"pairs group task 1 {dtype} N=40 K={K} M={M}")


@pytest.mark.parametrize("N,K,M", [(8200, 1056, 2), (8192, 4096, 2), (8200, 3296, 3), (8192, 4096, 4), (8200, 8192, 3),
                                   (8200, 11008, 4)])
def test_decode_large_grid_small_batches(orc, spl, N, K, M):
    """Launches of at least 512 row blocks at batches 2-4: activations staged in
    LDS while the copy fits 32 KB (2 x 1056, 2 x 4096, 3 x 3296, 4 x 4096),
    loaded directly by the single-block kernel otherwise (3 x 8192,
    4 x 11008), compared in full."""
    W, mask = synth.weight(960 + M + K, N, K, "bf16", 0.7)
    X = synth.activations(961, M, K, "bf16")
    ref = orc.linear_f64(X, orc.pack(W, "bf16", mask))
    Y = spl.sparse_linear(to_dev(X, "bf16"), _pack(spl, W, mask, "bf16"), algo="decode")
    assert_close(from_dev_f64(Y), ref, f"large grid N={N} K={K} M={M}")
