"""Pins of the CPU oracle to things other than itself (no GPU needed).

Each test checks the oracle against something the paper or the mathematics
fixes: the paper's worked example of bitmask expansion (section 2.4.1), brute
force over every mask of tiny blocks, format invariants, NumPy/BLAS and
NumPy's own fp16 conversion, exact-arithmetic inputs and closed forms.  The
shapes are rectangular (M != N != K) so that a transposed operand, a swapped
index or a dropped term fails at least one of them.
"""
import itertools
import os

import numpy as np
import pytest

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example.txt")


def _read_golden():
    d = {}
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, rest = line.split(":", 1)
            d[key.strip()] = rest.split()
    return d


def _payloads(tokens):
    """Distinct non-zero 16-bit payloads for the symbolic entries; 0 stays 0."""
    names = sorted({t for t in tokens if t != "0"})
    table = {n: 0x1000 + 37 * i for i, n in enumerate(names)}
    table["0"] = 0
    return table


def _bits_lsb_first(word, n):
    return "".join("1" if (int(word) >> j) & 1 else "0" for j in range(n))


# ------------------------------------------------------------ worked example

def test_worked_example_register_is_vnni_interleave():
    g = _read_golden()
    a, b, reg = g["rowA"], g["rowB"], g["register"]
    assert len(a) == len(b) == 8 and len(reg) == 16
    # VNNI pairs the two rows along the reduction dimension: A1 B1 A2 B2 ...
    assert reg == [t for pair in zip(a, b) for t in pair]


def test_worked_example_pack(orc):
    g = _read_golden()
    reg = g["register"]
    table = _payloads(reg)
    W = np.array([[table[t] for t in reg]], dtype=np.uint16)
    mask = (W != 0).astype(np.uint8)
    p = orc.pack(W, "f16", mask)
    assert p.values.tolist() == [table[t] for t in g["values"]]
    assert _bits_lsb_first(p.bitmask[0, 0], 16) == g["bitmask"][0]
    assert p.bitmask.shape == (1, 1) and int(p.bitmask[0, 0]) == 0xE94E
    assert p.row_offsets.tolist() == [0, 9]
    assert np.array_equal(orc.unpack(p), W)


def test_worked_example_row_major(orc):
    g = _read_golden()
    table = _payloads(g["rowA"] + g["rowB"])
    W = np.array([[table[t] for t in g["rowA"]], [table[t] for t in g["rowB"]]], dtype=np.uint16)
    p = orc.pack(W, "f16", (W != 0).astype(np.uint8))
    kept_a = [j for j in range(8) if (int(p.bitmask[0, 0]) >> j) & 1]
    kept_b = [j for j in range(8) if (int(p.bitmask[1, 0]) >> j) & 1]
    assert kept_a == [1, 3, 4, 7] and kept_b == [0, 1, 5, 6, 7]
    assert p.values.tolist() == [table[t] for t in ["A2", "A4", "A5", "A8", "B1", "B2", "B6", "B7", "B8"]]
    assert p.row_offsets.tolist() == [0, 4, 9]


# ------------------------------------------------------------ brute force

def _check_pack_against_numpy(orc, W, mask, dtype):
    p = orc.pack(W, dtype, mask)
    N, K = W.shape
    m = mask.astype(bool)
    # row offsets: exclusive prefix of per-row kept counts
    assert p.row_offsets[0] == 0
    assert np.array_equal(np.diff(p.row_offsets.astype(np.int64)), m.sum(axis=1))
    # bitmask: bit (k % 32) of word k // 32, everything past K zero
    words = (K + 31) // 32
    pad = np.zeros((N, words * 32), dtype=bool)
    pad[:, :K] = m
    expect = np.zeros((N, words), dtype=np.uint64)
    for j in range(32):
        expect |= pad[:, j::32].astype(np.uint64) << np.uint64(j)
    assert np.array_equal(p.bitmask.astype(np.uint64), expect)
    # values: kept payloads in row-major order (NumPy boolean indexing order)
    assert np.array_equal(p.values, W[m])
    # round trip: decode gives W where kept and +0 elsewhere, bit for bit
    zero = np.zeros((), dtype=W.dtype)
    assert np.array_equal(orc.unpack(p), np.where(m, W, zero))
    return p


def test_bruteforce_all_masks_2x8(orc):
    rng = np.random.default_rng(5)
    idx = np.arange(1 << 16, dtype=np.uint32)
    bits = ((idx[:, None] >> np.arange(16, dtype=np.uint32)) & 1).astype(np.uint8)
    mask = bits.reshape(-1, 8)                      # block i -> rows 2i, 2i+1
    W = rng.integers(0, 1 << 16, size=mask.shape, dtype=np.uint16)
    W[::7] = 0                                      # kept zeros and -0.0 payloads stay stored
    W[1::11] = 0x8000
    _check_pack_against_numpy(orc, W, mask, "f16")


def test_bruteforce_all_masks_small_shapes(orc):
    rng = np.random.default_rng(11)
    shapes = [(r, c) for r in range(1, 13) for c in range(1, 13) if r * c <= 12]
    for (r, c) in shapes:
        n = r * c
        W = rng.integers(1, 1 << 16, size=(r, c), dtype=np.uint16)
        for code in range(1 << n):
            mask = ((code >> np.arange(n)) & 1).astype(np.uint8).reshape(r, c)
            p = orc.pack(W, "bf16", mask)
            assert p.nnz == int(mask.sum())
            assert np.array_equal(p.values, W[mask.astype(bool)])
            assert np.array_equal(orc.unpack(p), np.where(mask.astype(bool), W, np.uint16(0)))


def test_int8_payloads_and_null_mask(orc):
    rng = np.random.default_rng(3)
    W8 = rng.integers(-128, 128, size=(9, 77), dtype=np.int8)
    W8[W8 % 3 == 0] = 0
    p = orc.pack(W8, "i8", None)                    # no mask: kept iff non-zero
    assert np.array_equal(p.values, W8[W8 != 0])
    assert np.array_equal(orc.unpack(p), W8)
    W16 = rng.integers(0, 1 << 16, size=(5, 40), dtype=np.uint16)
    W16[:, ::3] = 0x8000                            # -0.0 is not kept without a mask
    W16[:, 1::5] = 0
    p = orc.pack(W16, "bf16", None)
    keep = (W16 & 0x7FFF) != 0
    assert np.array_equal(p.values, W16[keep])


# ------------------------------------------------------------ invariants

@pytest.mark.parametrize("N,K,s,expect_nnz", [
    (4096, 4096, 0.7, 5_033_165),
    (4096, 4096, 0.5, 8_388_608),
    (300, 100, 0.7, 9_000),
])
def test_format_invariants(orc, N, K, s, expect_nnz):
    W, mask = synth.weight(123, N, K, "bf16", s)
    p = orc.pack(W, "bf16", mask)
    numel = N * K
    assert p.nnz == expect_nnz == numel - int(np.floor(s * numel + 1e-9))
    pc = np.unpackbits(p.bitmask.view(np.uint8), bitorder="little").reshape(N, -1).sum(axis=1)
    assert np.array_equal(np.diff(p.row_offsets.astype(np.int64)), pc)
    assert int(pc.sum()) == p.nnz
    words = p.bitmask.shape[1]
    if K % 32:
        tail = p.bitmask[:, words - 1] >> np.uint32(K % 32)
        assert not tail.any()


# ------------------------------------------------------------ fp linear

def _np_dense(bits, dtype):
    return synth.bits_to_f32(bits, dtype).astype(np.float64)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("M,N,K,s", [(5, 37, 101, 0.5), (3, 64, 96, 0.7), (1, 19, 260, 0.3)])
def test_linear_matches_blas(orc, dtype, M, N, K, s):
    W, mask = synth.weight(7 + K, N, K, dtype, s)
    X = synth.activations(8 + K, M, K, dtype)
    p = orc.pack(W, dtype, mask)
    Y = orc.linear_f64(X, p)
    Wd = np.where(mask.astype(bool), _np_dense(W, dtype), 0.0)
    Xd = _np_dense(X, dtype)
    Yref = Xd @ Wd.T
    scale = np.abs(Xd) @ np.abs(Wd).T
    assert Y.shape == (M, N)
    assert np.all(np.abs(Y - Yref) <= 1e-12 * scale + 1e-300)


def test_linear_exact_arithmetic(orc):
    rng = np.random.default_rng(17)
    M, N, K = 7, 23, 333
    wi = rng.integers(-15, 16, size=(N, K))          # W = wi / 64, exact in bf16
    xi = rng.integers(-3, 4, size=(M, K))            # X in {0, +-1, +-2, +-3}
    W = synth.round_bf16((wi / 64.0).astype(np.float32))
    X = synth.round_bf16(xi.astype(np.float32))
    mask = (rng.random((N, K)) < 0.4).astype(np.uint8)
    p = orc.pack(W, "bf16", mask)
    Y = orc.linear_f64(X, p)
    exact = (xi @ (wi * mask).T) / 64.0              # integer arithmetic, one exact scaling
    assert np.array_equal(Y, exact)


def test_identity_activations_give_transpose(orc):
    N, K = 45, 70
    W, mask = synth.weight(31, N, K, "f16", 0.6)
    X = synth.round_f16(np.eye(K, dtype=np.float32))
    p = orc.pack(W, "f16", mask)
    Y = orc.linear_f64(X, p)                         # [K][N]
    expect = np.where(mask.astype(bool), _np_dense(W, "f16"), 0.0).T
    assert np.array_equal(Y, expect)


def test_sparsity_zero_and_one(orc):
    M, N, K = 4, 33, 50
    X = synth.activations(1, M, K, "bf16")
    W, mask0 = synth.weight(2, N, K, "bf16", 0.0)
    assert mask0.all()
    p0 = orc.pack(W, "bf16", mask0)
    assert np.array_equal(orc.linear_f64(X, p0), orc.dense_f64(X, W, "bf16"))
    _, mask1 = synth.weight(2, N, K, "bf16", 1.0)
    assert not mask1.any()
    p1 = orc.pack(W, "bf16", mask1)
    assert p1.nnz == 0
    assert not orc.linear_f64(X, p1).any()


def test_dense_of_masked_weight_equals_sparse(orc):
    M, N, K = 6, 29, 131
    W, mask = synth.weight(41, N, K, "bf16", 0.7)
    X = synth.activations(42, M, K, "bf16")
    p = orc.pack(W, "bf16", mask)
    Wm = np.where(mask.astype(bool), W, np.uint16(0))
    assert np.array_equal(orc.linear_f64(X, p), orc.dense_f64(X, Wm, "bf16"))


def test_pairs_agree_with_full(orc):
    M, N, K = 9, 40, 75
    W, mask = synth.weight(51, N, K, "f16", 0.5)
    X = synth.activations(52, M, K, "f16")
    p = orc.pack(W, "f16", mask)
    Y = orc.linear_f64(X, p)
    rng = np.random.default_rng(0)
    ms = rng.integers(0, M, 100)
    ns = rng.integers(0, N, 100)
    assert np.array_equal(orc.linear_f64_pairs(X, p, ms, ns), Y[ms, ns])


# ------------------------------------------------------------ int8 linear

def _np_dequant(acc, sx, sw):
    y = (acc.astype(np.float32) * sx.astype(np.float32)[:, None]).astype(np.float32)
    y = (y * sw.astype(np.float32)[None, :]).astype(np.float32)
    return y.astype(np.float16).view(np.uint16)


@pytest.mark.parametrize("M,N,K", [(3, 21, 200), (1, 64, 4096)])
def test_int8_matches_numpy(orc, M, N, K):
    Wq, mask, sw = synth.int8_weight(61 + K, N, K, 0.7)
    Xq, sx = synth.int8_activations(62 + K, M, K)
    p = orc.pack(Wq, "i8", mask)
    acc, Y = orc.linear_i8(Xq, sx, p, sw)
    ref = Xq.astype(np.int64) @ (Wq.astype(np.int64) * mask).T
    assert np.array_equal(acc.astype(np.int64), ref)
    assert np.array_equal(Y, _np_dequant(acc, sx, sw))
    acc_d, Y_d = orc.dense_i8(Xq, sx, np.where(mask.astype(bool), Wq, np.int8(0)), sw)
    assert np.array_equal(acc_d, acc) and np.array_equal(Y_d, Y)


def test_int8_extreme_accumulators(orc):
    K = 11008
    Xq = np.full((2, K), 127, dtype=np.int8)
    Xq[1] = -127
    Wq = np.full((3, K), 127, dtype=np.int8)
    Wq[1, ::2] = -127
    Wq[2, :] = -127
    mask = np.ones((3, K), dtype=np.uint8)
    sx = np.array([0.013, 0.0071], dtype=np.float32)
    sw = np.array([3.1e-4, 2.2e-4, 1.7e-4], dtype=np.float32)
    p = orc.pack(Wq, "i8", mask)
    acc, Y = orc.linear_i8(Xq, sx, p, sw)
    assert int(acc[0, 0]) == 127 * 127 * K == 177_548_032
    assert int(acc[1, 2]) == 127 * 127 * K
    assert np.array_equal(Y, _np_dequant(acc, sx, sw))


# ------------------------------------------------------------ number formats

def test_f16_decode_exhaustive(orc):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    mine = orc.f16_to_f64(bits)
    ref = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(mine), nan)
    assert np.array_equal(mine[~nan], ref[~nan])
    assert np.array_equal(np.signbit(mine[~nan]), np.signbit(ref[~nan]))


def test_bf16_decode_exhaustive(orc):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    mine = orc.bf16_to_f64(bits)
    ref = (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(mine), nan)
    assert np.array_equal(mine[~nan], ref[~nan])


def test_f16_encode_against_numpy(orc):
    rng = np.random.default_rng(99)
    parts = [
        (rng.standard_normal(200_000) * np.exp2(rng.uniform(-30, 17, 200_000))).astype(np.float32),
        rng.integers(0, 1 << 32, 200_000, dtype=np.uint64).astype(np.uint32).view(np.float32),
    ]
    # exact midpoints between neighbouring fp16 values (ties go to the even neighbour)
    h = np.arange(0, 0x7C00, dtype=np.uint16)
    lo = h.view(np.float16).astype(np.float64)
    hi = (h + 1).view(np.float16).astype(np.float64)
    mid = ((lo + hi) / 2).astype(np.float32)
    parts += [mid, -mid, np.nextafter(mid, np.float32(np.inf)), np.nextafter(mid, np.float32(0))]
    parts.append(np.array([0.0, -0.0, 65504.0, 65519.996, 65520.0, 1e9, -1e9, np.inf, -np.inf,
                           6.1035156e-05, 5.9604645e-08, 2.9802322e-08, 2.98e-08, 1e-45], dtype=np.float32))
    x = np.concatenate(parts)
    mine = orc.f32_to_f16(x)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    nan = np.isnan(x)
    assert np.array_equal(mine[~nan], ref[~nan])
    assert np.all((mine[nan] & 0x7C00) == 0x7C00) and np.all((mine[nan] & 0x3FF) != 0)


def test_dequant_matches_numpy_chain(orc):
    rng = np.random.default_rng(7)
    acc = rng.integers(-(1 << 28), 1 << 28, 100_000).astype(np.int32)
    acc[:10] = [0, 1, -1, 16777217, -16777217, 177_548_032, 2**31 - 1, -(2**31), 33554435, 100]
    sx = (rng.random(100_000) * 0.05).astype(np.float32)
    sw = (rng.random(100_000) * 1e-3).astype(np.float32)
    mine = orc.dequant_f16(acc, sx, sw)
    t = (acc.astype(np.float32) * sx).astype(np.float32)
    y = (t * sw).astype(np.float32)
    with np.errstate(over="ignore"):
        ref = y.astype(np.float16).view(np.uint16)
    assert np.array_equal(mine, ref)


# ------------------------------------------------------------ generator sanity (inputs, not parity)

def test_magnitude_mask_count_and_ties():
    # all magnitudes equal -> the lowest row-major indices are zeroed
    bits = np.full((10, 13), 0x3C00, dtype=np.uint16)
    bits[::2] |= 0x8000
    m = synth.magnitude_mask(bits, 0.7)
    z = (130 * 7) // 10
    assert int((m == 0).sum()) == z
    assert not m.ravel()[:z].any() and m.ravel()[z:].all()
    # strictly ordered magnitudes -> exactly the z smallest are zeroed
    rng = np.random.default_rng(1)
    vals = rng.permutation(np.arange(1, 1001, dtype=np.uint16)).reshape(20, 50)
    m = synth.magnitude_mask(vals, 0.5)
    assert np.array_equal(m.astype(bool), vals > 500)


@pytest.mark.parametrize("s,cut", [(0.5, 0.6745), (0.7, 1.0364)])
def test_magnitude_cut_matches_normal_quantile(s, cut):
    W, mask = synth.weight(1234, 1024, 1024, "bf16", s)
    mags = np.abs(synth.bits_to_f32(W, "bf16").astype(np.float64))
    kept_min = mags[mask.astype(bool)].min()
    assert abs(kept_min / synth.WEIGHT_STD - cut) < 0.01
    assert int(mask.sum()) == 1024 * 1024 - int(s * 1024 * 1024)


def test_activation_rows_are_prefixes():
    a = synth.activations(5, 16, 64, "bf16")
    b = synth.activations(5, 4, 64, "bf16")
    assert np.array_equal(a[:4], b)


# ------------------------------------------------------------ tiled (GPU submatrix) layout

@pytest.mark.parametrize("N,K,s", [(16, 32, 0.5), (33, 70, 0.6), (5, 300, 0.3), (48, 96, 0.0), (17, 40, 1.0)])
def test_tiled_round_trip_and_invariants(orc, N, K, s):
    W, mask = synth.weight(71 + N + K, N, K, "bf16", s)
    t = orc.pack_tiled(W, "bf16", mask)
    m = mask.astype(bool)
    B, S = -(-N // 16), -(-K // 32)
    assert t.bitmask.shape == (B * S * 16,) and t.tile_offsets.shape == (B * S + 1,)
    assert t.nnz == int(m.sum())
    # round trip: decode gives W where kept, +0 elsewhere, bit for bit
    assert np.array_equal(orc.unpack_tiled(t), np.where(m, W, np.uint16(0)))
    # every tile's word is the mask block read LSB-first; tile offsets step by the tile popcounts
    padded = np.zeros((B * 16, S * 32), dtype=bool)
    padded[:N, :K] = m
    blocks = padded.reshape(B, 16, S, 32).transpose(0, 2, 1, 3)        # [B][S][16][32]
    words = (blocks.astype(np.uint64) << np.arange(32, dtype=np.uint64)).sum(axis=-1)
    assert np.array_equal(t.bitmask.astype(np.uint64), words.reshape(-1))
    counts = blocks.reshape(B * S, -1).sum(axis=1)
    assert np.array_equal(np.diff(t.tile_offsets.astype(np.int64)), counts)
    # values: tile by tile; inside a tile by 8-column group, then row, then column (NumPy boolean
    # indexing of the tile block viewed as [group][row][column in group])
    Wp = np.zeros((B * 16, S * 32), dtype=np.uint16)
    Wp[:N, :K] = W
    wb = Wp.reshape(B, 16, S, 32).transpose(0, 2, 1, 3)
    grouped = lambda x: x.reshape(16, 4, 8).transpose(1, 0, 2)
    expect = np.concatenate([grouped(wb[b, s_])[grouped(blocks[b, s_])] for b in range(B) for s_ in range(S)]
                            + [np.zeros(0, np.uint16)])
    assert np.array_equal(t.values, expect)


def test_tiled_and_row_layouts_hold_the_same_entries(orc):
    W, mask = synth.weight(5, 50, 200, "f16", 0.7)
    a = orc.unpack(orc.pack(W, "f16", mask))
    b = orc.unpack_tiled(orc.pack_tiled(W, "f16", mask))
    assert np.array_equal(a, b)


def test_tiled_int8(orc):
    Wq, mask, _ = synth.int8_weight(6, 40, 96, 0.7)
    t = orc.pack_tiled(Wq, "i8", mask)
    assert np.array_equal(orc.unpack_tiled(t), np.where(mask.astype(bool), Wq, np.int8(0)))
    # int8 column groups are 16 columns wide (16 bytes, like the 8 columns of a 16-bit payload)
    N, K = Wq.shape
    B, S = -(-N // 16), -(-K // 32)
    Wp = np.zeros((B * 16, S * 32), dtype=np.int8)
    Wp[:N, :K] = Wq
    Mp = np.zeros((B * 16, S * 32), dtype=bool)
    Mp[:N, :K] = mask.astype(bool)
    tiles = lambda x: x.reshape(B, 16, S, 32).transpose(0, 2, 1, 3).reshape(B * S, 16, 2, 16).transpose(0, 2, 1, 3)
    wt, mt = tiles(Wp), tiles(Mp)
    expect = np.concatenate([wt[i][mt[i]] for i in range(B * S)])
    assert np.array_equal(t.values, expect)


@pytest.mark.parametrize("dtype,G", [("bf16", 8), ("i8", 16)])
def test_tiled_value_order_worked_example(orc, dtype, G):
    """One 16 x 32 tile: row 0 keeps columns 0, 9 and 17, row 1 keeps 1 and 8,
    the other rows nothing; entry (r, j) holds 100 r + j.  Column groups of G
    columns, rows inside a group, columns inside a row."""
    W = (100 * np.arange(16)[:, None] + np.arange(32)[None, :]).astype(np.uint16 if dtype == "bf16" else np.int16)
    if dtype == "i8":
        W = (W % 128).astype(np.int8)
    mask = np.zeros((16, 32), np.uint8)
    mask[0, [0, 9, 17]] = 1
    mask[1, [1, 8]] = 1
    t = orc.pack_tiled(W, dtype, mask)
    order = [(0, 0), (1, 1), (0, 9), (1, 8), (0, 17)] if G == 8 else [(0, 0), (0, 9), (1, 1), (1, 8), (0, 17)]
    assert [int(v) for v in t.values] == [int(W[r, j]) for r, j in order]
    assert list(t.bitmask[:2]) == [(1 << 0) | (1 << 9) | (1 << 17), (1 << 1) | (1 << 8)]


# ---------------------------------------------------------------- per-token activation quantisation

def _bits(vals, dtype):
    return synth.round_to(np.asarray(vals, dtype=np.float32), dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_quantize_rows_closed_forms(orc, dtype):
    """Rows whose scale is exact (amax 127 -> 1, amax 254 -> 2) give codes that
    are the round-half-to-even of x / scale by hand; a zero row gets scale 1."""
    X = np.stack([
        _bits([127, 2.5, 3.5, -2.5, 126.5, -0.5, 1.5, 0.25], dtype),
        _bits([254, 5, 7, -254, 253, -3, 1, 0], dtype),
        _bits([0] * 8, dtype),
        _bits([-127, 127, -1, 1, 0.5, -1.5, 4.5, -4.5], dtype),
    ])
    Xq, sx = orc.quantize_rows_i8(X, dtype)
    assert sx.tolist() == [1.0, 2.0, 1.0, 1.0]
    assert Xq.tolist() == [[127, 2, 4, -2, 126, 0, 2, 0],
                           [127, 2, 4, -127, 126, -2, 0, 0],
                           [0] * 8,
                           [-127, 127, -1, 1, 0, -2, 4, -4]]


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_quantize_rows_invariants(orc, dtype):
    """Random rows: |code| <= 127, the largest magnitude of a row codes to +-127,
    and code * scale is within half a step (and rounding) of the value."""
    rng = np.random.default_rng(3)
    v = (rng.standard_normal((40, 300)) * rng.uniform(0.01, 50, (40, 1))).astype(np.float32)
    X = synth.round_to(v, dtype)
    x = orc.to_f64(X, dtype)
    Xq, sx = orc.quantize_rows_i8(X, dtype)
    assert np.abs(Xq.astype(np.int64)).max() <= 127
    arg = np.argmax(np.abs(x), axis=1)
    assert (np.abs(Xq[np.arange(40), arg]) == 127).all()
    assert np.allclose(sx.astype(np.float64), np.abs(x).max(axis=1) / 127.0, rtol=1e-6)
    err = np.abs(x - Xq.astype(np.float64) * sx[:, None].astype(np.float64))
    assert (err <= sx[:, None] * (0.5 + 1e-5)).all()


def test_quantize_rows_agrees_with_generator(orc):
    """The oracle's quantiser and the input generator's (NumPy) coding of the
    int8 activations give the same codes and scales bit for bit."""
    x = synth.activations(7, 33, 520, "bf16")
    q1, s1 = orc.quantize_rows_i8(x, "bf16")
    q2, s2 = synth.quantize_rows_int8(synth.bits_to_f32(x, "bf16"))
    assert np.array_equal(q1, q2) and np.array_equal(s1.view(np.uint32), s2.view(np.uint32))


def test_silu_mul_identities(orc):
    """silu(z) - silu(-z) = z and silu(z) + silu(-z) = z tanh(z / 2): with the
    gate negated (the same mask) the two outputs differ by exactly g * u and
    sum to g tanh(g / 2) u, where g and u come from the plain products; a zero
    gate or a zero up matrix gives zeros."""
    N, K, M = 40, 96, 7
    Wg, mask = synth.weight(71, N, K, "bf16", 0.5)
    Wu, masku = synth.weight(72, N, K, "bf16", 0.7)
    X = synth.activations(73, M, K, "bf16")
    neg = Wg ^ np.uint16(0x8000)                          # exact negation of every bf16 payload
    pg, pn, pu = orc.pack(Wg, "bf16", mask), orc.pack(neg, "bf16", mask), orc.pack(Wu, "bf16", masku)
    g, u = orc.linear_f64(X, pg), orc.linear_f64(X, pu)
    assert np.array_equal(orc.linear_f64(X, pn), -g)
    a, b = orc.silu_mul_f64(X, pg, pu), orc.silu_mul_f64(X, pn, pu)
    assert np.allclose(a - b, g * u, rtol=1e-12, atol=1e-15)
    assert np.allclose(a + b, g * np.tanh(g / 2) * u, rtol=1e-12, atol=1e-15)
    zero = orc.pack(np.zeros((N, K), np.uint16), "bf16", mask)
    assert not orc.silu_mul_f64(X, zero, pu).any()
    assert not orc.silu_mul_f64(X, pg, orc.pack(np.zeros((N, K), np.uint16), "bf16", masku)).any()


def test_silu_mul_matches_library_and_limits(orc):
    """Against scipy's logistic function (silu(z) = z expit(z)) on random
    layers, at chosen output pairs too, and the limits silu(z) -> z for large
    z and -> 0 for very negative z (identity activations make g = the stored
    gate weights, chosen here)."""
    from scipy.special import expit

    N, K, M = 33, 64, 5
    Wg, mg = synth.weight(81, N, K, "f16", 0.7)
    Wu, mu = synth.weight(82, N, K, "f16", 0.5)
    X = synth.activations(83, M, K, "f16")
    pg, pu = orc.pack(Wg, "f16", mg), orc.pack(Wu, "f16", mu)
    g, u = orc.linear_f64(X, pg), orc.linear_f64(X, pu)
    y = orc.silu_mul_f64(X, pg, pu)
    assert np.allclose(y, g * expit(g) * u, rtol=1e-13, atol=1e-16)
    ms, ns = np.array([0, 4, 2, 3]), np.array([0, 32, 7, 20])
    assert np.allclose(orc.silu_mul_f64_pairs(X, pg, pu, ms, ns), y[ms, ns], rtol=1e-15, atol=0)
    big = np.array([[40.0, -800.0, 0.0, 1.0]])
    G = synth.round_to(np.diag(big[0]).astype(np.float32), "f16")          # 4 x 4, gate row n = e_n * big[n]
    U = synth.round_to(np.eye(4, dtype=np.float32) * 3.0, "f16")
    I = synth.round_to(np.eye(4, dtype=np.float32), "f16")
    out = orc.silu_mul_f64(I, orc.pack(G, "f16"), orc.pack(U, "f16", np.ones((4, 4), np.uint8)))
    d = np.diag(out)
    assert abs(d[0] - 3 * 40.0) < 1e-12 and d[1] == 0.0 and d[2] == 0.0
    assert abs(d[3] - 3.0 / (1.0 + np.exp(-1.0))) < 1e-15


def _prune_by_selection(mags, prune):
    """Brute force: repeatedly remove the smallest remaining magnitude, the
    lowest index among equals."""
    left = list(range(len(mags)))
    keep = [1] * len(mags)
    for _ in range(prune):
        i = min(left, key=lambda j: (mags[j], j))
        keep[i] = 0
        left.remove(i)
    return keep


def test_magnitude_mask_worked_cases(orc):
    """Hand-derived: |w| = [3, 1, 1, 3, 0, 2] (the -0 and +0 tie, -1 and 1 tie,
    -3 and 3 tie); each extra pruned entry follows magnitude, then index."""
    W = _bits([3, -1, 1, -3, -0.0, 2], "bf16").reshape(2, 3)
    want = {0: [1, 1, 1, 1, 1, 1], 1: [1, 1, 1, 1, 0, 1], 2: [1, 0, 1, 1, 0, 1], 3: [1, 0, 0, 1, 0, 1],
            4: [1, 0, 0, 1, 0, 0], 5: [0, 0, 0, 1, 0, 0], 6: [0, 0, 0, 0, 0, 0]}
    for prune, keep in want.items():
        assert orc.magnitude_mask(W, "bf16", prune).ravel().tolist() == keep, prune
    Z = _bits([0.0, -0.0, 0.0, -0.0], "f16").reshape(1, 4)
    assert orc.magnitude_mask(Z, "f16", 2).ravel().tolist() == [0, 0, 1, 1]


def test_magnitude_mask_brute_force(orc):
    """Every 2 x 3 matrix over {0, +-1, 2} (signs and ties included) at every
    prune count against selection by brute force."""
    vals = [0.0, 1.0, -1.0, 2.0]
    for combo in itertools.product(range(4), repeat=6):
        v = [vals[c] for c in combo]
        W = _bits(v, "f16").reshape(2, 3)
        mags = [abs(x) for x in v]
        for prune in range(7):
            assert orc.magnitude_mask(W, "f16", prune).ravel().tolist() == _prune_by_selection(mags, prune)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("sparsity", [0.5, 0.7, 0.9])
def test_magnitude_mask_invariants_and_generator(orc, dtype, sparsity):
    """Random N(0, 0.02) matrices (bf16 has many equal magnitudes): exactly
    the requested count is zeroed, no kept |w| is below a pruned one, at the
    threshold magnitude every pruned index precedes every kept one, and the
    input generator's own (histogram) formulation gives the same mask."""
    N, K = 96, 200
    W = synth.round_to(synth.normal_f32(11, (N, K), 0.02), dtype)
    num, den = synth.parse_sparsity(sparsity)
    prune = N * K * num // den
    keep = orc.magnitude_mask(W, dtype, prune)
    mag = np.abs(orc.to_f64(W, dtype)).ravel()
    k = keep.ravel().astype(bool)
    assert (~k).sum() == prune
    t = mag[~k].max()
    assert t <= mag[k].min()
    cut, kept = np.flatnonzero(~k & (mag == t)), np.flatnonzero(k & (mag == t))
    assert cut.size and (not kept.size or cut.max() < kept.min())
    assert np.array_equal(keep, synth.magnitude_mask(W, sparsity))


def _loss(orc, X, p, dY, dtype):
    """L = sum_{m,n} dY[m][n] Y[m][n] with Y from the forward oracle."""
    return float((orc.to_f64(dY, dtype) * orc.linear_f64(X, p)).sum())


def test_weight_grad_finite_difference(orc):
    """L is linear in each weight, so replacing a kept weight w by w' changes
    the forward oracle's L by exactly (w' - w) G[n][k] (up to binary64
    rounding); a pruned position has no gradient."""
    N, K, M = 24, 64, 9
    W, mask = synth.weight(91, N, K, "bf16", 0.6)
    X = synth.activations(92, M, K, "bf16")
    dY = synth.activations(93, M, N, "bf16")
    p = orc.pack(W, "bf16", mask)
    G = orc.weight_grad_f64(dY, X, "bf16", p)
    assert not G[mask == 0].any()
    base = _loss(orc, X, p, dY, "bf16")
    rng = np.random.default_rng(0)
    kept = np.argwhere(mask == 1)
    for n, k in kept[rng.choice(len(kept), 12, replace=False)]:
        W2 = W.copy()
        W2[n, k] = synth.round_to(np.array([0.375], np.float32), "bf16")[0]
        delta = orc.to_f64(W2[n:n + 1, k:k + 1], "bf16")[0, 0] - orc.to_f64(W[n:n + 1, k:k + 1], "bf16")[0, 0]
        dl = _loss(orc, X, orc.pack(W2, "bf16", mask), dY, "bf16") - base
        assert abs(dl - delta * G[n, k]) <= 1e-9 * (1 + abs(dl))


def test_input_grad_finite_difference_and_library(orc):
    """dX from the oracle: changing X[m][k] to x' changes L by (x' - x) dX[m][k];
    and dY (W.Mask) by numpy on the unpacked weights."""
    N, K, M = 20, 48, 6
    W, mask = synth.weight(94, N, K, "f16", 0.7)
    X = synth.activations(95, M, K, "f16")
    dY = synth.activations(96, M, N, "f16")
    p = orc.pack(W, "f16", mask)
    D = orc.input_grad_f64(dY, "f16", p)
    dense = orc.to_f64(W, "f16") * mask
    assert np.allclose(D, orc.to_f64(dY, "f16") @ dense, rtol=1e-13, atol=1e-15)
    base = _loss(orc, X, p, dY, "f16")
    for m, k in [(0, 0), (5, 47), (3, 11), (2, 30)]:
        X2 = X.copy()
        X2[m, k] = synth.round_to(np.array([2.5], np.float32), "f16")[0]
        delta = orc.to_f64(X2[m:m + 1, k:k + 1], "f16")[0, 0] - orc.to_f64(X[m:m + 1, k:k + 1], "f16")[0, 0]
        dl = _loss(orc, X2, p, dY, "f16") - base
        assert abs(dl - delta * D[m, k]) <= 1e-9 * (1 + abs(dl))


def test_mask_of_and_sgd(orc):
    """mask_of reproduces the mask given to pack (row layout bits); one SGD
    step is w - lr g exactly on representable inputs."""
    W, mask = synth.weight(97, 9, 70, "bf16", 0.5)
    assert np.array_equal(orc.mask_of(orc.pack(W, "bf16", mask)), mask.astype(np.float64))
    w = np.array([1.0, -2.0, 0.5]); g = np.array([4.0, 0.25, -1.0])
    assert orc.sgd_f64(w, g, 0.5).tolist() == [-1.0, -2.125, 1.0]


def test_pack_i4_worked_and_round_trip(orc):
    """Hand-derived bytes (low nibble first, two's complement), an odd count,
    and unpack(pack(c)) == c over every code in [-8, 7] in both positions."""
    assert orc.pack_i4(np.array([1, -1, 7, -8, 3], np.int8)).tolist() == [0xF1, 0x87, 0x03]
    assert orc.pack_i4(np.array([], np.int8)).size == 0
    codes = np.array([a for a in range(-8, 8) for _ in range(2)] + list(range(7, -9, -1)), np.int8)
    assert np.array_equal(orc.unpack_i4(orc.pack_i4(codes), codes.size), codes)


def test_int4_generator_codes(orc):
    """The generator's 4-bit codes: within [-7, 7], zero off the mask, each
    row's largest kept magnitude coded +-7, scale = absmax / 7."""
    Wq, mask, sw = synth.int4_weight(5, 40, 96, 0.7)
    assert Wq.min() >= -7 and Wq.max() <= 7 and not Wq[mask == 0].any()
    w, _ = synth.weight(5, 40, 96, "bf16", 0.7)
    v = synth.bits_to_f32(w, "bf16") * mask
    amax = np.abs(v).max(axis=1)
    assert np.allclose(sw, np.where(amax == 0, 1, amax / 7), rtol=1e-6)
    assert (np.abs(Wq).max(axis=1)[amax > 0] == 7).all()


def test_int4_full_range_generator(orc):
    """The planted-edge generator: codes in [-8, 7], rows 0 and N - 1 all -8
    where kept, row N // 2 all 7, zero off the mask, and -8 in other rows."""
    N, K = 40, 96
    Wq, mask, _ = synth.int4_weight_full_range(6, N, K, 0.5)
    keep = mask.astype(bool)
    assert Wq.min() == -8 and Wq.max() <= 7 and not Wq[~keep].any()
    assert (Wq[0, keep[0]] == -8).all() and (Wq[N - 1, keep[N - 1]] == -8).all()
    assert (Wq[N // 2, keep[N // 2]] == 7).all()
    assert (Wq[1:N - 1][keep[1:N - 1]] == -8).any()
