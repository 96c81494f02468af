"""One-shot magnitude pruning on the GPU vs the oracle: the keep-masks are
compared bit for bit (index work), at small ragged sizes with many equal
magnitudes, at the edge counts (nothing, everything, one entry), with signed
zeros, and at the full Llama-2-7B shapes."""
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


def _mask(spl, W, dtype, prune, ws=None):
    return spl.magnitude_mask(to_dev(W, dtype), prune, workspace=ws).cpu().numpy()


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K", [(1, 8), (3, 16), (17, 72), (100, 1000), (130, 8192), (257, 520)])
def test_prune_small(orc, spl, dtype, N, K):
    W = synth.round_to(synth.normal_f32(N * 7 + K, (N, K), 0.02), dtype)
    n = N * K
    for prune in sorted({0, 1, n // 2, n * 7 // 10, n * 9 // 10, n - 1, n}):
        got = _mask(spl, W, dtype, prune)
        ref = orc.magnitude_mask(W, dtype, prune)
        assert np.array_equal(got, ref), f"{dtype} N={N} K={K} prune={prune}: {int((got != ref).sum())} differ"


def test_prune_ties_and_signed_zeros(orc, spl):
    """Few distinct magnitudes (long runs of ties across chunk boundaries),
    -0 and +0 mixed, and ties of both signs."""
    rng = np.random.default_rng(5)
    N, K = 300, 4096                                   # 1.2 M entries: 19 chunks of 64 K
    v = rng.choice(np.array([0.0, -0.0, 0.5, -0.5, 1.0, 2.0, -2.0], np.float32), size=(N, K))
    W = synth.round_to(v, "bf16")
    for prune in (1, 200000, 350000, 350001, 600000, N * K - 3):
        got = _mask(spl, W, "bf16", prune)
        assert np.array_equal(got, orc.magnitude_mask(W, "bf16", prune)), prune


def test_prune_workspace_reuse(orc, spl):
    """One workspace for consecutive calls of different sizes: each call
    clears what it needs."""
    import torch

    ws = torch.empty((spl.lib().spl_magnitude_mask_workspace_bytes(),), dtype=torch.uint8, device="cuda")
    for seed, (N, K, s) in enumerate([(200, 4096, 0.7), (40, 80, 0.5), (300, 1024, 0.9)]):
        W = synth.round_to(synth.normal_f32(seed, (N, K), 0.02), "f16")
        prune = N * K * int(s * 10) // 10
        assert np.array_equal(_mask(spl, W, "f16", prune, ws), orc.magnitude_mask(W, "f16", prune))


@pytest.mark.parametrize("name,j", [("q", 0), ("gate", 4), ("down", 6)])
def test_prune_llama_shapes(orc, spl, name, j):
    """Full Llama-2-7B shapes at 70% (and 50% for q), compared in full; the
    mask equals the one the input generator draws for the same weights."""
    _, N, K = synth.LLAMA2_7B_LINEARS[j]
    W = synth.round_to(synth.normal_f32(synth.weight_seed(0, j), (N, K), synth.WEIGHT_STD), "bf16")
    for s in ((0.7, 0.5) if name == "q" else (0.7,)):
        num, den = synth.parse_sparsity(s)
        prune = N * K * num // den
        got = _mask(spl, W, "bf16", prune)
        ref = orc.magnitude_mask(W, "bf16", prune)
        assert np.array_equal(got, ref), f"{name} s={s}: {int((got != ref).sum())} differ"
