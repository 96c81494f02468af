"""GPU compressor (bitmask expansion encoder/decoder) vs the oracle, bit-exact."""
import numpy as np
import pytest

import synth
from tests._helpers import assert_pack_equal, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def spl():
    import paper_2405_03594_amd as spl

    spl.lib()
    return spl


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("N,K,s", [
    (1, 1, 0.0), (1, 1, 1.0), (3, 7, 0.5), (17, 100, 0.7), (5, 64, 0.3), (33, 65, 0.5),
    (130, 1000, 0.5), (64, 4096, 0.7), (16, 8, 0.0), (9, 96, 1.0),
])
def test_pack_small(orc, spl, dtype, N, K, s):
    W, mask = synth.weight(100 + N + K, N, K, dtype, s)
    ref = orc.pack(W, dtype, mask)
    Wc = spl.pack_sparse(to_dev(W, dtype), to_dev(mask, "i8").view(dtype=__import__("torch").uint8), layout="rows")
    assert_pack_equal(Wc, ref)
    dense = spl.unpack(Wc)
    from tests._helpers import from_dev_bits
    assert np.array_equal(from_dev_bits(dense), orc.unpack(ref))
    Wt = spl.retile16(Wc)                               # tile layout, bit-exact against the oracle's encoder
    assert_pack_equal(Wt, orc.pack_tiled(W, dtype, mask))
    assert np.array_equal(from_dev_bits(spl.unpack(Wt)), orc.unpack(ref))


@pytest.mark.parametrize("name,N,K,dtype,s", [
    ("cfg1 4096x4096 fp16 50%", 4096, 4096, "f16", 0.5),
    ("q 4096x4096 bf16 70%", 4096, 4096, "bf16", 0.7),
    ("gate 11008x4096 bf16 70%", 11008, 4096, "bf16", 0.7),
    ("down 4096x11008 bf16 70%", 4096, 11008, "bf16", 0.7),
    ("up 11008x4096 bf16 50%", 11008, 4096, "bf16", 0.5),
])
def test_pack_llama_shapes(orc, spl, name, N, K, dtype, s):
    import torch

    W, mask = synth.weight(7, N, K, dtype, s)
    ref = orc.pack(W, dtype, mask)
    Wc = spl.pack_sparse(to_dev(W, dtype), torch.from_numpy(mask).cuda(), layout="rows")
    assert Wc.nnz == N * K - int(s * N * K)
    assert_pack_equal(Wc, ref)
    assert_pack_equal(spl.retile16(Wc), orc.pack_tiled(W, dtype, mask))


def test_pack_without_mask_keeps_nonzero_payloads(orc, spl):
    rng = np.random.default_rng(3)
    W = rng.integers(0, 1 << 16, size=(40, 200), dtype=np.uint16)
    W[:, ::3] = 0
    W[:, 1::7] = 0x8000                 # -0.0: not kept without a mask
    W[:, 2::11] = 0x7FC1                # NaN payloads are kept and copied bit for bit
    ref = orc.pack(W, "bf16", None)
    Wc = spl.pack_sparse(to_dev(W, "bf16"), None, layout="rows")
    assert_pack_equal(Wc, ref)
    assert_pack_equal(spl.pack_sparse(to_dev(W, "bf16"), None), orc.pack_tiled(W, "bf16", None))


def test_pack_keeps_masked_zero_payloads(orc, spl):
    import torch

    W = np.zeros((8, 64), dtype=np.uint16)
    W[:, ::2] = 0x8000
    mask = np.ones((8, 64), dtype=np.uint8)
    mask[:, 5::9] = 0
    ref = orc.pack(W, "f16", mask)
    Wc = spl.pack_sparse(to_dev(W, "f16"), torch.from_numpy(mask).cuda(), layout="rows")
    assert_pack_equal(Wc, ref)


@pytest.mark.parametrize("N,K", [(21, 80), (4096, 4096), (11008, 4096)])
def test_pack_int8(orc, spl, N, K):
    import torch

    Wq, mask, _ = synth.int8_weight(9, N, K, 0.7)
    ref = orc.pack(Wq, "i8", mask)
    Wc = spl.pack_sparse(to_dev(Wq, "i8"), torch.from_numpy(mask).cuda(), layout="rows")
    assert_pack_equal(Wc, ref)
    dense = spl.unpack(Wc).cpu().numpy()
    assert np.array_equal(dense, orc.unpack(ref))
    Wt = spl.retile16(Wc)
    assert_pack_equal(Wt, orc.pack_tiled(Wq, "i8", mask))
    assert np.array_equal(spl.unpack(Wt).cpu().numpy(), orc.unpack(ref))
