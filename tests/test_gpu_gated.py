"""The gated half of a Llama MLP, Y = silu(X Wg^T) * (X Wu^T), in one launch on
the GPU vs the oracle (binary64).

Tolerance (fp16/bf16 outputs): |y - y64| <= max(2e-2, 1e-2 |y64|) per element:
g and u are fp32 sums as in the plain linear layers, silu is evaluated in
fp32 and the product is rounded once to the payload type.  Small shapes with
ragged N, M and K are compared in full on both kernel families (the paired
decode kernel for M <= 16 and the prefill tiling for any M); the Llama-2-7B
gate/up shape is compared in full at decode batches and on sampled outputs at
prefill batches."""
import numpy as np
import pytest

import synth
from tests._helpers import assert_close, from_dev_f64, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def spl():
    import paper_2405_03594_amd as spl

    spl.lib()
    return spl


def _pair(spl, orc, seed, N, K, dtype, sg, su):
    import torch

    Wg, mg = synth.weight(seed, N, K, dtype, sg)
    Wu, mu = synth.weight(seed + 1, N, K, dtype, su)
    dev = [spl.pack_sparse(to_dev(W, dtype), torch.from_numpy(m).cuda()) for W, m in ((Wg, mg), (Wu, mu))]
    ref = (orc.pack(Wg, dtype, mg), orc.pack(Wu, dtype, mu))
    return dev, ref


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,sg,su", [(1, 8, 0.5, 0.5), (16, 32, 0.5, 0.7), (40, 72, 0.7, 0.7), (100, 1000, 0.7, 0.5),
                                       (300, 264, 0.0, 0.7), (33, 512, 0.9, 0.0), (64, 4096, 0.7, 0.7)])
def test_gated_small(orc, spl, dtype, N, K, sg, su):
    (g, u), (pg, pu) = _pair(spl, orc, 500 + N + K, N, K, dtype, sg, su)
    X = synth.activations(501 + K, 300, K, dtype)
    ref = orc.silu_mul_f64(X, pg, pu)
    Xd = to_dev(X, dtype)
    for M in (1, 5, 16):
        for algo in ("decode", "prefill"):
            Y = spl.sparse_linear_silu_mul(Xd[:M].contiguous(), g, u, algo=algo)
            assert_close(from_dev_f64(Y), ref[:M], f"{algo} {dtype} N={N} K={K} M={M}")
    for M in (17, 64, 129, 300):
        Y = spl.sparse_linear_silu_mul(Xd[:M].contiguous(), g, u)
        assert_close(from_dev_f64(Y), ref[:M], f"auto {dtype} N={N} K={K} M={M}")


def test_gated_zero_matrices(orc, spl):
    """A gate or an up matrix with no kept entries gives zeros, both families."""
    import torch

    N, K = 48, 96
    (g, u), _ = _pair(spl, orc, 520, N, K, "bf16", 0.7, 0.7)
    z = spl.pack_sparse(torch.zeros((N, K), dtype=torch.bfloat16, device="cuda"),
                        torch.zeros((N, K), dtype=torch.uint8, device="cuda"))
    X = to_dev(synth.activations(521, 40, K, "bf16"), "bf16")
    for M, algo in ((3, "decode"), (40, "prefill")):
        for a, b in ((z, u), (g, z)):
            Y = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
            spl.sparse_linear_silu_mul(X[:M].contiguous(), a, b, out=Y, algo=algo)
            assert not Y.float().abs().max().item()


@pytest.mark.parametrize("N,K,M", [(2048, 128, 2048), (128, 192, 256)])
def test_gated_aligned_grids(orc, spl, N, K, M):
    """Launches whose blocks all lie inside the matrices take the unchecked
    prefill loads: 2N virtual rows on 128 x 256 and 64 x 128 tiles."""
    (g, u), (pg, pu) = _pair(spl, orc, 530 + N, N, K, "bf16", 0.7, 0.5)
    X = synth.activations(531, M, K, "bf16")
    Y = spl.sparse_linear_silu_mul(to_dev(X, "bf16"), g, u)
    assert_close(from_dev_f64(Y), orc.silu_mul_f64(X, pg, pu), f"N={N} K={K} M={M}")


@pytest.mark.parametrize("s", [0.7, 0.5])
def test_gated_llama_gate_up(orc, spl, s):
    """Llama-2-7B gate/up (11008 x 4096), the benchmark's batches: in full at
    1, 4 and 16 (paired decode kernel), on sampled outputs at 512 and 2048
    (prefill tiling)."""
    N, K = 11008, 4096
    (g, u), (pg, pu) = _pair(spl, orc, synth.weight_seed(0, 4), N, K, "bf16", s, s)
    X = synth.activations(synth.activation_seed(4), 2048, K, "bf16")
    Xd = to_dev(X, "bf16")
    for M in (1, 4, 16):
        Y = spl.sparse_linear_silu_mul(Xd[:M].contiguous(), g, u)
        assert_close(from_dev_f64(Y), orc.silu_mul_f64(X[:M], pg, pu), f"gate/up M={M} s={s}")
    rng = np.random.default_rng(54)
    for M in (512, 2048):
        ms = np.concatenate([[0, M - 1, M // 2, 0], rng.integers(0, M, 3000)])
        ns = np.concatenate([[0, N - 1, 5000, 16], rng.integers(0, N, 3000)])
        Y = from_dev_f64(spl.sparse_linear_silu_mul(Xd[:M].contiguous(), g, u))
        assert_close(Y[ms, ns], orc.silu_mul_f64_pairs(X[:M], pg, pu, ms, ns), f"gate/up M={M} s={s}")
        assert np.isfinite(Y).all()
