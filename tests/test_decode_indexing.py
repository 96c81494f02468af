"""Host-side replay of the decode kernels' indexing (no GPU).

The decode kernels split a 16-row block's k-steps (32-column tiles) into one
contiguous range per wave and walk each range in chunks: as many tiles as
fit a staging buffer (at most C), whose values are fetched with aligned
16-byte loads into LDS.  This test replays that schedule, with the constants
read from the kernel source and the tile offsets of real encodings from the
oracle, and checks that

  * the wave ranges partition [0, S) and the chunks partition each range;
  * every tile offset, bitmask word, 16-byte value piece, LDS window and
    activation element the schedule touches lies inside its buffer
    (values: the encoding rounded up to 16 bytes plus a 16-byte tail);
  * a lane's 8-byte window read from the staging buffer, realigned with
    v_alignbyte_b32 and expanded with the selector table, equals the dense
    masked tile row.

It guards against an earlier fault in which a prefetch ran past a wave's
staging region."""
import os
import re

import numpy as np
import pytest

import synth

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2405_03594_amd", "csrc", "k_decode.hip")


def _constants():
    src = open(SRC).read()
    assert "if (small_grid(blocks)) return sparse_group_w<T, 16>(g, kmax, s);" in src and \
        "return large_grid(blocks) && g.M <= 16 ? sparse_group_w<T, 4>(g, kmax, s) : sparse_group_w<T, 8>(g, kmax, s);" \
        in src, "waves per workgroup changed: update this replay"
    waves = (4, 8, 16)
    chunk = int(re.search(r"constexpr int kChunk = (\d+);", src).group(1))
    assert "constexpr int C = MT == 1 ? kChunk : kChunk / 2;" in src, "chunk size formula changed: update this replay"
    vbuf = int(re.search(r"constexpr int kVBuf = (\d+);", src).group(1))
    alloc = re.search(r"constexpr int kVBufAlloc = kVBuf \+ (\d+);", src)
    assert alloc, "staging buffer size changed: update this replay"
    assert "constexpr int kPieceRounds = kVBuf / 16 / kWave;" in src
    assert "const int t = base + lane < kend ? base + lane : kend;" in src, "offset clamp changed: update this replay"
    assert "const uint32_t lim = (ch.a0 + kVBuf) >> 1;" in src and \
        "const bool fit = lane >= r + 1 && lane <= r + jmax && (uint32_t)o <= lim;" in src, \
        "chunk rule changed: update this replay"
    assert "if (c1 - ob + C > kOffsetLanes) {" in src and "constexpr int kOffsetLanes = kWave - 1;" in src, \
        "offset window changed: update this replay"
    return waves, {1: chunk, 2: chunk // 2}, vbuf, vbuf + int(alloc.group(1))


def _wave_range(S, waves, w):
    L = -(-S // waves)
    b = min(w * L, S)
    return b, min(b + L, S)


def _chunks(tob, kbeg, kend, C, vbuf):
    """The kernel's chunk selection: [(c0, cn, a0, np, offsets)].  Offsets come
    from a window of 64 lanes (lane i: tile ob + i, clamped to the range end)
    that is reloaded at a chunk that would reach past lane 63."""
    out = []
    c0 = kbeg
    ob = kbeg
    while c0 < kend:
        if c0 - ob + C > 63:
            ob = c0
        window = [int(tob[min(ob + i, kend)]) for i in range(64)]
        r = c0 - ob
        assert 0 <= r and r + C <= 63                  # every readlane index of the chunk is a lane
        to = [window[r + j] for j in range(C + 1)]
        a0 = (2 * to[0]) & ~15
        lim = (a0 + vbuf) >> 1                          # a tile fits iff its end offset <= lim
        jmax = min(kend - c0, C)
        cn = sum(1 for j in range(1, C + 1) if j <= jmax and to[j] <= lim)
        assert cn >= 1 and all(to[j] <= lim for j in range(1, cn + 1))   # the fitting lanes form a prefix
        np_ = (2 * to[cn] - a0 + 15) >> 4
        out.append((c0, cn, a0, np_, to))
        c0 += cn
    return out


def _replay(T, N, K, MT, W):
    _, Cs, vbuf, alloc = _constants()
    waves = W
    C = Cs[MT]
    S, B = -(-K // 32), -(-N // 16)
    value_bytes = -(-2 * T.nnz // 16) * 16 + 16           # allocation of the values buffer
    for b in range(B):
        tob = T.tile_offsets[b * S:(b + 1) * S + 1]
        covered = np.zeros(S, dtype=np.int64)
        for w in range(waves):
            kbeg, kend = _wave_range(S, waves, w)
            for c0, cn, a0, np_, to in _chunks(tob, kbeg, kend, C, vbuf):
                assert 1 <= cn <= C and c0 + cn <= kend
                covered[c0:c0 + cn] += 1
                assert np_ <= vbuf // 16, (b, w, c0, np_)       # pieces fit the rounds of loads
                assert a0 + 16 * np_ <= value_bytes             # global value reads
                for j in range(cn):
                    assert 2 * to[j + 1] - a0 + 12 <= alloc     # third dword of any window stays in the buffer
                    for fg in range(4):
                        k = 32 * (c0 + j) + 8 * fg
                        assert k >= K or k + 8 <= K             # activation reads (K % 8 == 0)
        assert (covered == 1).all(), b


@pytest.mark.parametrize("W", [4, 8, 16])
@pytest.mark.parametrize("MT", [1, 2])
@pytest.mark.parametrize("N,K,s", [(16, 8, 0.5), (33, 40, 0.0), (20, 264, 0.7), (17, 520, 1.0), (48, 1064, 0.5),
                                   (16, 4096, 0.0), (32, 4104, 0.7), (16, 11008, 0.5), (16, 16384, 0.0),
                                   (16, 65536, 0.7), (16, 65544, 0.0)])   # ranges longer than the offset window
def test_schedule_stays_in_bounds(orc, N, K, s, MT, W):
    Wt, mask = synth.weight(11 + N + K, N, K, "bf16", s)
    _replay(orc.pack_tiled(Wt, "bf16", mask), N, K, MT, W)


# ---------------------------------------------------------------- expansion

def _popc(x):
    return bin(int(x) & 0xFFFFFFFF).count("1")


def _perm(s0, s1, sel):
    src = int(s1).to_bytes(4, "little") + int(s0).to_bytes(4, "little")
    out = 0
    for j in range(4):
        b = (sel >> (8 * j)) & 0xFF
        assert b < 8 or b == 12
        out |= (src[b] if b < 8 else 0) << (8 * j)
    return out


def _nibble_selector(nib, h):
    sel = 0
    for e in range(2):
        j = 2 * h + e
        s16 = 0x0C0C
        if (nib >> j) & 1:
            r = _popc(nib & ((1 << j) - 1))
            s16 = (2 * r) | ((2 * r + 1) << 8)
        sel |= s16 << (16 * e)
    return sel


@pytest.mark.parametrize("N,K,s", [(1, 8, 0.5), (17, 264, 0.9), (33, 96, 0.0), (20, 520, 0.7)])
def test_lane_expansion_matches_dense_rows(orc, N, K, s):
    _, Cs, vbuf, alloc = _constants()
    waves = 8
    C = Cs[1]
    W, mask = synth.weight(31 + N, N, K, "bf16", s)
    T = orc.pack_tiled(W, "bf16", mask)
    vals = np.concatenate([T.values.view(np.uint8), np.zeros(16 + 16, np.uint8)])
    dense = np.where(mask.astype(bool), W, np.uint16(0))
    S, B = -(-K // 32), -(-N // 16)
    bm = T.bitmask.reshape(-1)

    def alignbyte(hi, lo, sh):
        return ((int(hi) << 32 | int(lo)) >> (8 * (sh & 3))) & 0xFFFFFFFF

    for b in range(B):
        tob = T.tile_offsets[b * S:(b + 1) * S + 1]
        for w in range(waves):
            kbeg, kend = _wave_range(S, waves, w)
            for c0, cn, a0, np_, to in _chunks(tob, kbeg, kend, C, vbuf):
                stage = np.zeros(alloc, np.uint8)
                stage[:16 * np_] = vals[a0:a0 + 16 * np_]
                st32 = stage.view(np.uint32)
                for j in range(cn):
                    t = b * S + c0 + j
                    words = [int(bm[t * 16 + r]) for r in range(16)]
                    for lane in range(64):
                        fr, fg = lane & 15, lane >> 4
                        wd = words[fr]
                        byte = (wd >> (8 * fg)) & 0xFF
                        # values before this lane's: column groups before fg (all rows), then rows above fr in fg
                        before = sum(_popc((words[r] >> (8 * g)) & 0xFF) for g in range(fg) for r in range(16)) + \
                            sum(_popc((words[r] >> (8 * fg)) & 0xFF) for r in range(fr))
                        oa = to[j] + before
                        ob = oa + _popc(byte & 0xF)
                        pa, pb = 2 * oa - a0, 2 * ob - a0
                        qa, qb = pa >> 2, pb >> 2
                        vlo, vhi = alignbyte(st32[qa + 1], st32[qa], pa), alignbyte(st32[qa + 2], st32[qa + 1], pa)
                        ulo, uhi = alignbyte(st32[qb + 1], st32[qb], pb), alignbyte(st32[qb + 2], st32[qb + 1], pb)
                        lo, hi = byte & 15, byte >> 4
                        a = [_perm(vhi, vlo, _nibble_selector(lo, 0)), _perm(vhi, vlo, _nibble_selector(lo, 1)),
                             _perm(uhi, ulo, _nibble_selector(hi, 0)), _perm(uhi, ulo, _nibble_selector(hi, 1))]
                        got = np.array(a, dtype=np.uint32).view(np.uint16)
                        n, k0 = b * 16 + fr, 32 * (c0 + j) + 8 * fg
                        exp = np.zeros(8, np.uint16)
                        if n < N:
                            seg = dense[n, k0:min(k0 + 8, K)]
                            exp[:seg.size] = seg
                        assert np.array_equal(got, exp), (b, c0 + j, lane)


# ---------------------------------------------------------------- two row blocks per workgroup

def _pair_constants():
    src = open(SRC).read()
    vbuf = int(re.search(r"constexpr int kVBuf = (\d+);", src).group(1))
    assert "constexpr int kHalfVBuf = kVBuf / 2;" in src and "constexpr int kHalfVBufAlloc = kHalfVBuf + 16;" in src
    assert "constexpr int kHalfPieceRounds = (kHalfVBuf / 16 + kWave - 1) / kWave;" in src
    assert "const uint32_t lim = (ch.a0[b] + kHalfVBuf) >> 1;" in src and "cn = cb < cn ? cb : cn;" in src, \
        "pair chunk rule changed: update this replay"
    assert "if (v == 1 && g.M > 4 && !small_grid(blocks)) return sparse_pair_launch<T, 8, 1>(g, s);" in src and \
        "if (v == 2 && !small_grid(blocks)) return sparse_pair_launch<T, 8, 2>(g, s);" in src, \
        "pair launch rule changed: update this replay"
    assert "constexpr int C = MT == 1 ? kChunk : kChunk / 2;" in src, "pair chunk length changed: update this replay"
    half = vbuf // 2
    return half, half + 16, -(-(half // 16) // 64)


def _pair_chunks(tobs, kbeg, kend, C, half):
    """Chunks of the pair kernel: per block a 64-lane offsets window (reloaded
    together) and half the buffer; the chunk is the shorter of the two fits."""
    out, c0, ob = [], kbeg, kbeg
    while c0 < kend:
        if c0 - ob + C > 63:
            ob = c0
        r = c0 - ob
        assert r + C <= 63
        tos = [[int(t[min(ob + r + j, kend)]) for j in range(C + 1)] for t in tobs]
        jmax = min(kend - c0, C)
        cn, a0s = C, []
        for to in tos:
            a0 = (2 * to[0]) & ~15
            lim = (a0 + half) >> 1
            cb = sum(1 for j in range(1, C + 1) if j <= jmax and to[j] <= lim)
            assert cb >= 1
            cn, a0s = min(cn, cb), a0s + [a0]
        nps = [(2 * to[cn] - a0 + 15) >> 4 for to, a0 in zip(tos, a0s)]
        out.append((c0, cn, a0s, nps, tos))
        c0 += cn
    return out


@pytest.mark.parametrize("N,K,s", [(16, 1056, 0.5), (48, 1056, 0.7), (40, 3296, 0.0), (17, 11008, 0.5),
                                   (33, 4096, 0.9), (16, 65552, 0.7)])
@pytest.mark.parametrize("MT", [1, 2])
def test_pair_schedule_stays_in_bounds(orc, N, K, s, MT):
    half, alloc, rounds = _pair_constants()
    C = _constants()[1][1] // MT             # kChunk tiles per chunk, half of them with two batch tiles
    W, mask = synth.weight(61 + N, N, K, "bf16", s)
    T = orc.pack_tiled(W, "bf16", mask)
    S, B = -(-K // 32), -(-N // 16)
    value_bytes = -(-2 * T.nnz // 16) * 16 + 16
    for p in range(-(-B // 2)):
        blocks = (2 * p, 2 * p + 1 if 2 * p + 1 < B else 2 * p)           # a missing second block aliases the first
        tobs = [T.tile_offsets[b * S:(b + 1) * S + 1] for b in blocks]
        covered = np.zeros(S, dtype=np.int64)
        for w in range(8):
            kbeg, kend = _wave_range(S, 8, w)
            for c0, cn, a0s, nps, tos in _pair_chunks(tobs, kbeg, kend, C, half):
                covered[c0:c0 + cn] += 1
                for a0, np_, to in zip(a0s, nps, tos):
                    assert np_ <= half // 16 and np_ <= 64 * rounds       # pieces fit the rounds of loads
                    assert a0 + 16 * np_ <= value_bytes                   # global value reads
                    for j in range(cn):
                        assert 2 * to[j + 1] - a0 + 12 <= alloc          # windows stay in the block's half
        assert (covered == 1).all(), p


def _xl_shapes():
    """(M, K) pairs whose activations the kernels stage in LDS: M * 32S * 2 <= 32 KB."""
    out = []
    for K in (8, 24, 64, 520, 1000, 4096, 8200, 11008, 16384):
        S = -(-K // 32)
        for M in (1, 2, 3, 5, 16, 31):
            if M * 32 * S * 2 <= 32 * 1024:
                out.append((M, K))
    return out


@pytest.mark.parametrize("W", [4, 8, 16])
def test_activation_staging_covers_each_piece_once(W):
    """XStager: thread t, round i takes piece p = t + i * threads, i.e. row
    p // per_row and piece p % per_row, from one division and a step per
    round; every piece of the copy is written once, loads stay inside X and
    stores inside the LDS rows."""
    src = open(SRC).read()
    for line in ("dm = kThreads / per_row;", "dq = kThreads - dm * per_row;",
                 "if (q >= per_row) q -= per_row, ++m;",
                 "if ((int)__umul24(m, per_row) > p) --m;", "if ((int)__umul24(m + 1, per_row) <= p) ++m;",
                 "static constexpr int kXRounds = kXLdsMax / 16 / kThreads;",
                 "if (p < total && q < kp)   // 32-bit byte offsets from the uniform base (SGPR-based loads)",
                 "2u * (__umul24(m, (uint32_t)K) + 8u * (uint32_t)q));",
                 "if (p < total) *reinterpret_cast<u32x4*>(xs + __umul24(m, stride) + 8 * q) = r[i];"):
        assert line in src, f"staging changed: update this replay ({line})"
    threads = 64 * W
    rounds = 32 * 1024 // 16 // threads
    for M, K in _xl_shapes():
        S = -(-K // 32)
        per_row, kp, total = 4 * S, K // 8, M * 4 * S
        stride = 32 * S + 8
        assert rounds * threads >= total
        dm, dq = threads // per_row, threads - (threads // per_row) * per_row
        seen = np.zeros(total, dtype=np.int64)
        for t in range(threads):
            m = int(np.float32(t) * (np.float32(1.0) / np.float32(per_row)))
            if m * per_row > t:
                m -= 1
            if (m + 1) * per_row <= t:
                m += 1
            q = t - m * per_row
            for i in range(rounds):
                p = t + i * threads
                if p < total:
                    assert (m, q) == divmod(p, per_row), (M, K, t, i)
                    assert m * K < 1 << 24 and m * stride < 1 << 24
                    if q < kp:
                        assert 2 * (m * K + 8 * q) + 16 <= 2 * M * K
                    assert m * stride + 8 * q + 8 <= M * stride
                    seen[p] += 1
                m, q = m + dm, q + dq
                if q >= per_row:
                    q, m = q - per_row, m + 1
        assert (seen == 1).all(), (M, K)


@pytest.mark.parametrize("MT", [1, 2])
@pytest.mark.parametrize("K", [8, 40, 520, 4096, 4104, 11008])
def test_activation_buffer_offsets(MT, K):
    """XGlobal: lane (fr, fg) of batch tile t loads 16 bytes at byte offset
    2 (m K + 8 fg) + 64 s with m = 16t + fr; a row past M, or on the last
    k-step of a ragged K a column past K, uses an offset beyond X so the
    hardware returns zeros.  Every other load is inside X and brings exactly
    X[m][32s + 8fg .. +8]."""
    src = open(SRC).read()
    for line in ("constexpr uint32_t kXOob = 0x80000000u;",
                 "off[t] = m < M ? 2u * ((uint32_t)m * (uint32_t)K + 8u * (uint32_t)fg) : kXOob;",
                 "if (ragged && (uint32_t)(32 * s + 8 * fg) >= (uint32_t)K) o = kXOob;",
                 "xb[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, o, 64 * s, 0));",
                 "if (j < cur.cn) xop.load(xb[j], c0 + j, c0 + j == S - 1 && (K & 31) != 0, fg, K);",
                 "if (2 * M * kmax > kXBufMax) return hipErrorNotSupported;"):
        assert line in src, f"activation loads changed: update this replay ({line})"
    oob = 0x80000000
    S = -(-K // 32)
    for M in sorted({1, 2, 7, 16 * MT - 1, 16 * MT} - {0}):
        nbytes = 2 * M * K
        assert nbytes <= oob
        X = np.arange(M * K, dtype=np.int64).reshape(M, K)
        for s in range(S):
            ragged = s == S - 1 and K % 32 != 0
            for lane in range(64):
                fr, fg = lane & 15, lane >> 4
                for t in range(MT):
                    m = 16 * t + fr
                    o = 2 * (m * K + 8 * fg) if m < M else oob
                    if ragged and 32 * s + 8 * fg >= K:
                        o = oob
                    live = m < M and 32 * s + 8 * fg < K
                    if o == oob:
                        assert not live, (M, s, lane, t)
                        continue                      # the voffset alone is past X: zeros
                    assert live and o + 64 * s + 16 <= nbytes, (M, s, lane, t)
                    e = (o + 64 * s) // 2
                    got = X.ravel()[e:e + 8]
                    assert (got == X[m, 32 * s + 8 * fg:32 * s + 8 * fg + 8]).all()
