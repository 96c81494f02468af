"""4-bit sparse payloads on the GPU vs the oracle: the packed nibbles bit for
bit against the oracle's tile encoder + 4-bit packer, and the int32 sums and
fp16 outputs of the decode kernel bit for bit against the int8 oracle on the
same integer codes (the 4-bit codes are int8 integers in [-7, 7])."""
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


def _assert_equal(got, ref, what):
    if not np.array_equal(got, ref):
        bad = np.argwhere(got != ref)
        i = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} of {ref.size} differ; first at {i}: got {got[i]!r}, "
                             f"oracle {ref[i]!r}")


def _pack4(spl, Wq, mask):
    import torch

    W8 = spl.pack_sparse(to_dev(Wq, "i8"), torch.from_numpy(mask).cuda())
    return spl.pack_int4(W8)


@pytest.mark.parametrize("N,K,s", [(1, 16, 0.5), (16, 48, 0.5), (33, 64, 0.7), (100, 1008, 0.7), (64, 4096, 0.5),
                                   (200, 336, 0.0), (17, 512, 1.0), (48, 2064, 0.9)])
def test_int4_pack_and_linear(orc, spl, N, K, s):
    import torch

    Wq, mask, sw = synth.int4_weight(900 + N, N, K, s)
    W4 = _pack4(spl, Wq, mask)
    ref_bytes = orc.pack_i4(orc.pack_tiled(Wq, "i8", mask).values)
    got_bytes = W4.values.cpu().numpy()[:ref_bytes.size]
    _assert_equal(got_bytes, ref_bytes, f"nibbles N={N} K={K} s={s}")
    Xq, sx = synth.int8_activations(901 + K, 16, K)
    p = orc.pack(Wq, "i8", mask)
    for M in (1, 5, 16):
        acc_ref, y_ref = orc.linear_i8(Xq[:M], sx[:M], p, sw)
        acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
        Y = spl.sparse_linear_int4(to_dev(Xq[:M], "i8"), torch.from_numpy(sx[:M]).cuda(), W4,
                                   torch.from_numpy(sw).cuda(), acc_out=acc)
        _assert_equal(acc.cpu().numpy(), acc_ref, f"acc N={N} K={K} s={s} M={M}")
        _assert_equal(Y.cpu().view(torch.int16).numpy().view(np.uint16), y_ref, f"Y N={N} K={K} s={s} M={M}")


@pytest.mark.parametrize("N,K,s", [(1, 16, 0.5), (33, 64, 0.7), (100, 1008, 0.5), (48, 2064, 0.9)])
def test_int4_full_code_range(orc, spl, N, K, s):
    """Code -8 (rows of all -8 among them) packs, widens and multiplies exactly."""
    import torch

    Wq, mask, sw = synth.int4_weight_full_range(910 + N, N, K, s)
    W4 = _pack4(spl, Wq, mask)
    ref_bytes = orc.pack_i4(orc.pack_tiled(Wq, "i8", mask).values)
    _assert_equal(W4.values.cpu().numpy()[:ref_bytes.size], ref_bytes, f"nibbles N={N} K={K} s={s}")
    Xq, sx = synth.int8_activations(911 + K, 16, K)
    p = orc.pack(Wq, "i8", mask)
    for M in (1, 7, 16):
        acc_ref, y_ref = orc.linear_i8(Xq[:M], sx[:M], p, sw)
        acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
        Y = spl.sparse_linear_int4(to_dev(Xq[:M], "i8"), torch.from_numpy(sx[:M]).cuda(), W4,
                                   torch.from_numpy(sw).cuda(), acc_out=acc)
        _assert_equal(acc.cpu().numpy(), acc_ref, f"acc N={N} K={K} s={s} M={M}")
        _assert_equal(Y.cpu().view(torch.int16).numpy().view(np.uint16), y_ref, f"Y N={N} K={K} s={s} M={M}")


def test_int4_pack_counts_codes_outside_the_range(spl):
    """Codes 8 and -9 are counted and rejected by the binding; in range, 0."""
    import torch

    N, K = 33, 64
    Wq, mask, _ = synth.int4_weight_full_range(920, N, K, 0.5)
    kept = np.argwhere(mask.astype(bool))
    bad = Wq.copy()
    for (r, c), v in zip(kept[[0, 5, 17]], (8, -9, 127)):
        bad[r, c] = v
    W8 = spl.pack_sparse(to_dev(bad, "i8"), torch.from_numpy(mask).cuda())
    with pytest.raises(ValueError, match="3 codes outside"):
        spl.pack_int4(W8)
    spl.pack_int4(W8, check=False)           # stored as their low 4 bits
    W8 = spl.pack_sparse(to_dev(Wq, "i8"), torch.from_numpy(mask).cuda())
    spl.pack_int4(W8)                        # the count was cleared: no error


@pytest.mark.parametrize("name", ["o", "gate", "down"])
def test_int4_llama_shapes(orc, spl, name):
    import torch

    j = [n for n, _, _ in synth.LLAMA2_7B_LINEARS].index(name)
    _, N, K = synth.LLAMA2_7B_LINEARS[j]
    Wq, mask, sw = synth.int4_weight(synth.weight_seed(0, j), N, K, 0.7)
    W4 = _pack4(spl, Wq, mask)
    Xq, sx = synth.int8_activations(synth.activation_seed(j), 16, K)
    p = orc.pack(Wq, "i8", mask)
    for M in (1, 16):
        acc_ref, y_ref = orc.linear_i8(Xq[:M], sx[:M], p, sw)
        acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
        Y = spl.sparse_linear_int4(to_dev(Xq[:M], "i8"), torch.from_numpy(sx[:M]).cuda(), W4,
                                   torch.from_numpy(sw).cuda(), acc_out=acc)
        _assert_equal(acc.cpu().numpy(), acc_ref, f"{name} acc M={M}")
        _assert_equal(Y.cpu().view(torch.int16).numpy().view(np.uint16), y_ref, f"{name} Y M={M}")
