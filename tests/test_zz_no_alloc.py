"""The allocation-free pruning entry point (spl_magnitude_mask_noalloc)
against the entry point that takes a workspace, bit for bit (the keep-mask
is index work): two calls in a row on the library's shared scratch, the
second smaller, so whatever the first left there must not leak into the
second.  The small cases are also checked against the oracle."""
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


def _pair(spl, W, dtype, prune):
    import torch

    Wd = to_dev(W, dtype)
    ref = spl.magnitude_mask(Wd, prune)
    got = torch.full(tuple(W.shape), 7, dtype=torch.uint8, device="cuda")
    spl.magnitude_mask_noalloc(Wd, prune, out=got)
    return got.cpu().numpy(), ref.cpu().numpy()


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("first,second", [((4096, 4096, 0.7), (130, 8192, 0.5)),
                                          ((11008, 4096, 0.5), (17, 72, 0.9)),
                                          ((300, 4096, 0.7), (1, 8, 0.5))])
def test_noalloc_matches_workspace_entry_twice(orc, spl, dtype, first, second):
    for seed, (N, K, s) in enumerate((first, second)):
        W = synth.round_to(synth.normal_f32(40 + seed + N, (N, K), 0.02), dtype)
        prune = N * K * int(round(s * 10)) // 10
        got, ref = _pair(spl, W, dtype, prune)
        assert np.array_equal(got, ref), f"{dtype} N={N} K={K}: {int((got != ref).sum())} differ"
        assert int((got == 0).sum()) == prune
        if N * K <= 1 << 20:
            assert np.array_equal(got, orc.magnitude_mask(W, dtype, prune)), f"oracle {dtype} N={N} K={K}"


def test_noalloc_ties_then_smaller(orc, spl):
    """Long runs of equal magnitudes over many chunks, then a small matrix."""
    rng = np.random.default_rng(11)
    v = rng.choice(np.array([0.0, -0.0, 0.5, -0.5, 1.0, 2.0], np.float32), size=(300, 4096))
    W = synth.round_to(v, "bf16")
    got, ref = _pair(spl, W, "bf16", 350001)
    assert np.array_equal(got, ref)
    W2 = synth.round_to(synth.normal_f32(3, (3, 16), 0.02), "bf16")
    for prune in (0, 1, 47, 48):
        got, ref = _pair(spl, W2, "bf16", prune)
        assert np.array_equal(got, ref) and np.array_equal(got, orc.magnitude_mask(W2, "bf16", prune)), prune


def test_noalloc_rejects_bad_arguments(spl):
    import torch

    W = torch.zeros((16, 12), dtype=torch.bfloat16, device="cuda")      # K % 8 != 0
    out = torch.empty((16, 12), dtype=torch.uint8, device="cuda")
    with pytest.raises(RuntimeError, match="spl_magnitude_mask_noalloc"):
        spl.magnitude_mask_noalloc(W, 3, out=out)
    W = torch.zeros((16, 16), dtype=torch.bfloat16, device="cuda")
    out = torch.empty((16, 16), dtype=torch.uint8, device="cuda")
    with pytest.raises(RuntimeError, match="spl_magnitude_mask_noalloc"):
        spl.magnitude_mask_noalloc(W, 16 * 16 + 1, out=out)             # prune > N K


def test_noalloc_largest_size_then_small(spl):
    """N K = 2^31 - 8192, the largest the entry takes (bf16 W drawn on the
    device from a seeded generator), then a small matrix."""
    import torch

    N, K = (1 << 31) // 8192 - 1, 8192
    g = torch.Generator(device="cuda").manual_seed(77)
    W = (torch.randn((N, K), generator=g, device="cuda", dtype=torch.float32) * 0.02).to(torch.bfloat16)
    prune = N * K * 7 // 10
    ref = spl.magnitude_mask(W, prune)
    got = torch.full((N, K), 7, dtype=torch.uint8, device="cuda")
    spl.magnitude_mask_noalloc(W, prune, out=got)
    assert torch.equal(got, ref)
    assert int((got == 0).sum()) == prune
    del W, ref, got
    torch.cuda.empty_cache()
    W2 = to_dev(synth.round_to(synth.normal_f32(5, (17, 72), 0.02), "bf16"), "bf16")
    ref = spl.magnitude_mask(W2, 600)
    got = torch.empty((17, 72), dtype=torch.uint8, device="cuda")
    assert torch.equal(spl.magnitude_mask_noalloc(W2, 600, out=got), ref)
