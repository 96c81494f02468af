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


@pytest.mark.parametrize("dtype", ["bf16", "f16", "i8"])
@pytest.mark.parametrize("N,K,s", [(1, 8, 0.5), (3, 7, 0.5), (17, 100, 0.7), (33, 65, 0.0), (16, 96, 1.0),
                                   (130, 1000, 0.5), (40, 4104, 0.7)])
def test_pack_straight_into_tiles(orc, spl, dtype, N, K, s):
    """spl_pack_count / spl_pack_sparse with the tile layout: bit-exact against the
    oracle's tile encoder and against the row pack converted by spl_retile16."""
    import torch

    if dtype == "i8":
        W, mask, _ = synth.int8_weight(400 + N + K, N, K, s)
    else:
        W, mask = synth.weight(400 + N + K, N, K, dtype, s)
    m = torch.from_numpy(mask).cuda()
    Wt = spl.pack_sparse(to_dev(W, dtype), m, layout="tile16")
    ref = orc.pack_tiled(W, dtype, mask)
    assert_pack_equal(Wt, ref)
    assert_pack_equal(spl.retile16(spl.pack_sparse(to_dev(W, dtype), m, layout="rows")), ref)
    assert spl.validate(Wt)


@pytest.mark.parametrize("name,N,K,s", [("q", 4096, 4096, 0.7), ("gate", 11008, 4096, 0.7),
                                        ("down", 4096, 11008, 0.7), ("cfg1 fp16", 4096, 4096, 0.5)])
def test_pack_straight_into_tiles_llama(orc, spl, name, N, K, s):
    import torch

    dtype = "f16" if "fp16" in name else "bf16"
    W, mask = synth.weight(11, N, K, dtype, s)
    Wt = spl.pack_sparse(to_dev(W, dtype), torch.from_numpy(mask).cuda())
    assert_pack_equal(Wt, orc.pack_tiled(W, dtype, mask))


@pytest.mark.parametrize("N,K,s,M", [(17, 264, 0.7, 1), (100, 1000, 0.5, 4), (4096, 4096, 0.7, 1),
                                     (48, 2056, 0.0, 16), (16, 64, 1.0, 2)])
def test_pack_count_pack_sparse_sparse_linear_through_the_c_abi(orc, spl, N, K, s, M):
    """The three boundary calls alone (ctypes, device memory from torch): the
    tile-layout pack is read by spl_sparse_linear with no conversion step."""
    import ctypes

    import torch

    from tests._helpers import assert_close, from_dev_f64

    L = spl.lib()
    W, mask = synth.weight(500 + N, N, K, "bf16", s)
    X = synth.activations(600 + K, M, K, "bf16")
    Wd, md, Xd = to_dev(W, "bf16"), torch.from_numpy(mask).cuda(), to_dev(X, "bf16")
    T = int(L.spl_tile16_count(N, K))
    toff = torch.empty(T + 1, dtype=torch.int32, device="cuda")
    nnz = ctypes.c_int64(-1)
    st = L.spl_pack_count(ctypes.c_void_p(Wd.data_ptr()), 2, ctypes.c_void_p(md.data_ptr()), N, K, 1,
                          ctypes.c_void_p(toff.data_ptr()), ctypes.byref(nnz), None)
    assert st == 0 and nnz.value == N * K - int(s * N * K)
    bm = torch.empty(16 * T, dtype=torch.int32, device="cuda")
    vb = int(L.spl_values_bytes(2, nnz.value))
    vals = torch.empty(vb, dtype=torch.uint8, device="cuda")
    st = L.spl_pack_sparse(ctypes.c_void_p(Wd.data_ptr()), 2, ctypes.c_void_p(md.data_ptr()), N, K, 1,
                           ctypes.c_void_p(toff.data_ptr()), ctypes.c_void_p(bm.data_ptr()),
                           ctypes.c_void_p(vals.data_ptr()), None)
    assert st == 0
    view = spl._Matrix(N, K, 2, 1, nnz.value, bm.data_ptr(), vals.data_ptr(), 0, toff.data_ptr(), vb)
    assert L.spl_validate(ctypes.byref(view), None) == 0
    Y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    st = L.spl_sparse_linear(ctypes.c_void_p(Xd.data_ptr()), M, ctypes.byref(view), ctypes.c_void_p(Y.data_ptr()),
                             None)
    assert st == 0
    torch.cuda.synchronize()
    assert_close(from_dev_f64(Y), orc.linear_f64(X, orc.pack(W, "bf16", mask)), f"N={N} K={K} M={M}")


def _corrupt(Wc, field, index, fn):
    """A copy of Wc with one entry of one array changed (host-side edit)."""
    import copy

    import torch

    c = copy.copy(Wc)
    arr = getattr(Wc, field).clone()
    flat = arr.view(-1)
    v = flat[index].item()
    flat[index] = torch.tensor(fn(v), dtype=flat.dtype)
    setattr(c, field, arr)
    return c


@pytest.mark.parametrize("layout", ["tile16", "rows"])
def test_validate_finds_inconsistent_formats(orc, spl, layout):
    import copy

    import torch

    N, K = 40, 200                                      # ragged: rows past N in the last tile row block,
    W, mask = synth.weight(71, N, K, "bf16", 0.7)       # columns past K in the last 32-column step
    Wc = spl.pack_sparse(to_dev(W, "bf16"), torch.from_numpy(mask).cuda(), layout=layout)
    assert spl.validate(Wc)
    offs = "tile_offsets" if layout == "tile16" else "row_offsets"
    nblocks = getattr(Wc, offs).numel() - 1
    assert not spl.validate(_corrupt(Wc, offs, nblocks // 2, lambda v: v + 1))      # offsets vs popcounts
    assert not spl.validate(_corrupt(Wc, offs, 0, lambda v: v + 1))                 # first offset
    bad = copy.copy(Wc)
    bad.nnz = Wc.nnz - 1                                                           # last offset != nnz
    assert not spl.validate(bad)
    S = -(-K // 32)
    if layout == "tile16":
        last = (nblocks - 1) * 16                     # last tile: column 200 % 32 = 8 -> bit 8 is a pad bit
        assert not spl.validate(_corrupt(Wc, "bitmask", last, lambda v: v | (1 << 8)))
        row_past_n = (nblocks - 1) * 16 + (N % 16)    # a row >= N of the last row block
        assert not spl.validate(_corrupt(Wc, "bitmask", row_past_n, lambda v: v | 1))
    else:
        assert not spl.validate(_corrupt(Wc, "bitmask", S - 1, lambda v: v | (1 << 8)))
    # the same bit moved inside the matrix is a consistent-looking mask with a wrong count
    i = int(np.flatnonzero(Wc.bitmask.cpu().numpy().view(np.uint32) == 0)[0]) if (Wc.bitmask == 0).any() else 0
    assert not spl.validate(_corrupt(Wc, "bitmask", i, lambda v: v ^ 1))
