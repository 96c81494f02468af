"""Host-side replay of the sparse int8 kernel's indexing (no GPU).

The int8 kernel multiplies pairs of 16 x 32 tiles (one v_mfma_i32_16x16x64_i8
each), so its wave ranges and chunks keep pairs whole.  This test replays the
schedule with the constants read from the kernel source and the tile offsets
of real encodings from the oracle, and checks that every tile is multiplied
once, that chunks end on a pair boundary unless the range ends there, and
that every value piece, LDS window and staged activation read lies inside
its buffer.  It also replays a lane's four nibble windows (aligned dword pair
+ v_alignbyte_b32 + the selector table + v_perm_b32) and compares the
expanded operand with the dense int8 row."""
import os
import re

import numpy as np
import pytest

import synth

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2405_03594_amd", "csrc", "k_int8.hip")


def _constants():
    src = open(SRC).read()
    chunk = int(re.search(r"constexpr int kI8Chunk = (\d+);", src).group(1))
    vbuf = int(re.search(r"constexpr int kI8VBuf = (\d+);", src).group(1))
    alloc = re.search(r"constexpr int kI8VBufAlloc = kI8VBuf \+ (\d+);", src)
    assert alloc
    for line in ("constexpr int C = MT == 4 ? kI8Chunk / 2 : kI8Chunk;",
                 "const bool fit = lane >= r + 1 && lane <= r + jmax && (uint32_t)o <= lim;",
                 "if (cn < jmax) cn &= ~1;",
                 "const uint32_t lim = ch.a0 + kI8VBuf;",
                 "const int t = base + lane < kend ? base + lane : kend;",
                 "if (c1 - ob + C > kI8OffsetLanes) {",
                 "return 64 * ((tile_steps(K) + 1) / 2) + 16;"):
        assert line in src, f"kernel changed: update this replay ({line})"
    return chunk, vbuf, vbuf + int(alloc.group(1))


def _ranges(S, W):
    P = (S + 1) // 2
    Lp = -(-P // W)
    out = []
    for w in range(W):
        pb = min(w * Lp, P)
        pe = min(pb + Lp, P)
        kbeg, kend = 2 * pb, min(2 * pe, S)
        out.append((min(kbeg, kend), kend))
    return out


def _chunks(tob, kbeg, kend, C, vbuf):
    out, c0, ob = [], kbeg, kbeg
    while c0 < kend:
        if c0 - ob + C > 63:
            ob = c0
        window = [int(tob[min(ob + i, kend)]) for i in range(64)]
        r = c0 - ob
        assert r + C <= 63
        a0 = window[r] & ~15
        lim = a0 + vbuf
        jmax = min(C, kend - c0)
        cn = sum(1 for i in range(64) if r + 1 <= i <= r + jmax and window[i] <= lim)
        if cn < jmax:
            cn &= ~1
        assert cn >= 1
        end = window[r + cn]
        npieces = (end - a0 + 15) >> 4
        out.append((c0, cn, a0, npieces, [window[r + j] for j in range(C + 1)]))
        c0 += cn
    return out


@pytest.mark.parametrize("W", [8, 16])
@pytest.mark.parametrize("MT", [1, 4])
@pytest.mark.parametrize("N,K,s", [(16, 16, 0.5), (33, 48, 0.0), (20, 272, 0.7), (16, 4096, 0.0), (32, 4112, 0.7),
                                   (16, 11008, 0.5), (17, 512, 1.0), (16, 65552, 0.7)])
def test_int8_schedule_stays_in_bounds(orc, N, K, s, MT, W):
    chunk, vbuf, alloc = _constants()
    C = chunk // 2 if MT == 4 else chunk
    Wq, mask, _ = synth.int8_weight(5 + N + K, N, K, s)
    T = orc.pack_tiled(Wq, "i8", mask)
    S, B = -(-K // 32), -(-N // 16)
    value_bytes = -(-T.nnz // 16) * 16 + 16
    stride = 64 * ((S + 1) // 2) + 16
    for b in range(B):
        tob = T.tile_offsets[b * S:(b + 1) * S + 1]
        covered = np.zeros(S, dtype=np.int64)
        for kbeg, kend in _ranges(S, W):
            assert kbeg % 2 == 0 or kbeg == kend          # empty ranges are clamped to the end
            for c0, cn, a0, npieces, to in _chunks(tob, kbeg, kend, C, vbuf):
                assert c0 % 2 == 0 and (cn % 2 == 0 or c0 + cn == kend), (c0, cn, kend)
                covered[c0:c0 + cn] += 1
                assert npieces <= vbuf // 16 and a0 + 16 * npieces <= value_bytes
                for q in range(-(-cn // 2)):
                    for tsel in (0, 1):
                        j = 2 * q + tsel
                        t0 = to[j]                       # j <= cn: at most the chunk's end offset
                        assert t0 - a0 + 8 <= alloc       # a lane whose word is zero reads at its tile offset
                        end_j = to[min(j + 1, cn)]
                        assert end_j - a0 + 8 <= alloc    # the last nibble window of the tile
                    for fg in range(4):                   # staged activation read of this pair
                        kx = 64 * ((c0 >> 1) + q) + 16 * fg
                        assert kx + 16 <= stride - 16
        assert (covered == 1).all()


def _popc(x):
    return bin(int(x) & 0xFFFFFFFF).count("1")


def _sel(nib):
    out = 0
    for j in range(4):
        b = _popc(nib & ((1 << j) - 1)) if (nib >> j) & 1 else 12
        out |= b << (8 * j)
    return out


def _perm(s0, s1, sel):
    src = int(s1).to_bytes(4, "little") + int(s0).to_bytes(4, "little")
    out = 0
    for j in range(4):
        b = (sel >> (8 * j)) & 0xFF
        assert b < 8 or b == 12
        out |= (src[b] if b < 8 else 0) << (8 * j)
    return out


@pytest.mark.parametrize("N,K,s", [(16, 16, 0.5), (20, 272, 0.7), (33, 96, 0.0), (17, 528, 0.9)])
def test_int8_lane_expansion_matches_dense_rows(orc, N, K, s):
    chunk, vbuf, alloc = _constants()
    Wq, mask, _ = synth.int8_weight(41 + N, N, K, s)
    T = orc.pack_tiled(Wq, "i8", mask)
    vals = np.concatenate([T.values.view(np.uint8), np.zeros(32, np.uint8)])
    dense = np.where(mask.astype(bool), Wq, 0).astype(np.int8).view(np.uint8)
    S, B = -(-K // 32), -(-N // 16)
    bm = T.bitmask.reshape(-1)

    def alignbyte(hi, lo, sh):
        return ((int(hi) << 32 | int(lo)) >> (8 * (sh & 3))) & 0xFFFFFFFF

    for b in range(B):
        tob = T.tile_offsets[b * S:(b + 1) * S + 1]
        for kbeg, kend in _ranges(S, 8):
            for c0, cn, a0, npieces, to in _chunks(tob, kbeg, kend, chunk, vbuf):
                stage = np.zeros(alloc + 8, np.uint8)
                stage[:16 * npieces] = vals[a0:a0 + 16 * npieces]
                for q in range(-(-cn // 2)):
                    for lane in range(64):
                        fr, fg = lane & 15, lane >> 4
                        tsel, half = fg >> 1, fg & 1
                        j = 2 * q + tsel
                        t = b * S + c0 + j
                        words = [int(bm[t * 16 + r]) if j < cn else 0 for r in range(16)]
                        w = words[fr]
                        # values before this lane's: the 16-column group before (all rows), then rows above fr
                        o = to[j] + sum(_popc((words[r] >> (16 * g)) & 0xFFFF) for g in range(half) for r in range(16)) + \
                            sum(_popc((words[r] >> (16 * half)) & 0xFFFF) for r in range(fr))
                        got = []
                        for i in range(4):
                            nib = (w >> (16 * half + 4 * i)) & 15
                            p = o - a0
                            d = p & ~3
                            lo = int(stage[d:d + 4].view(np.uint32)[0])
                            hi = int(stage[d + 4:d + 8].view(np.uint32)[0])
                            got.append(_perm(0, alignbyte(hi, lo, p), _sel(nib)))
                            o += _popc(nib)
                        got = np.array(got, dtype=np.uint32).view(np.uint8)
                        n, k0 = b * 16 + fr, 32 * (c0 + j) + 16 * half
                        exp = np.zeros(16, np.uint8)
                        if n < N and j < cn and k0 < K:
                            seg = dense[n, k0:min(k0 + 16, K)]
                            exp[:seg.size] = seg
                        assert np.array_equal(got, exp), (b, c0 + j, lane)
