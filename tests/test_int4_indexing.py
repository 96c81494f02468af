"""CPU replay of the 4-bit decode kernel's schedule (k_int4.hip): for every
workgroup, wave, tile pair and lane, the nibble offset from the tile offset
and the half-wave scan, the three dwords it reads (inside the values buffer
of spl_int4_values_bytes(nnz) bytes, which the kernel is never allowed to
leave), and the 16 sign-extended bytes it builds, which must equal the dense
codes of its row and 16 columns (zeros where pruned).  The packed values come
from the oracle's tile encoder and 4-bit packer, so this also checks that the
kernel reads the layout the oracle defines."""
import os

import numpy as np
import pytest

import synth

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2405_03594_amd", "csrc", "k_int4.hip")


def _widen(w):
    """i4_widen: four nibbles -> four bytes, 0xF0 or'ed into those with bit 3 set (mod 2^32)."""
    y = (w & 0xF) | ((w & 0xF0) << 4) | ((w & 0xF00) << 8) | ((w & 0xF000) << 12)
    m = y & 0x08080808
    return (y | (((m << 5) - (m << 1)) & 0xFFFFFFFF)) & 0xFFFFFFFF


def _selector(nib):
    """nibble_selector8(nib, 0): byte j <- rank of column j among the nibble's set bits, 12 (zero) if clear."""
    return [bin(nib & ((1 << j) - 1)).count("1") if (nib >> j) & 1 else 12 for j in range(4)]


def _perm0(y, sel):
    """v_perm_b32(0, y, sel) for selectors 0-3 (bytes of y) and 12 (zero), as signed bytes."""
    out = []
    for sj in sel:
        v = 0 if sj == 12 else (y >> (8 * sj)) & 0xFF
        out.append(v - 256 if v >= 128 else v)
    return out


def _values_bytes(nnz):
    """spl_values_bytes(SPL_I4, nnz): the nibble bytes rounded up to 16, plus 16."""
    return ((nnz + 1) // 2 + 15) // 16 * 16 + 16


@pytest.mark.parametrize("gen", ["int4_weight", "int4_weight_full_range"])
@pytest.mark.parametrize("waves", [8, 16])
@pytest.mark.parametrize("N,K,s", [(1, 16, 0.5), (17, 48, 0.7), (40, 96, 0.0), (33, 208, 0.9), (16, 64, 1.0)])
def test_int4_schedule_reads_and_operands(orc, N, K, s, waves, gen):
    src = open(SRC).read()
    for line in ("const uint32_t s = (uint32_t)(2 * p + (fg >> 1));",
                 "const bool ok = p < pe;",
                 "const_cast<uint32_t*>(g.bm + b * S * 16), (short)0, 64 * S, 0x00020000);",
                 "const_cast<int32_t*>(g.toff + b * S), (short)0, 4 * S, 0x00020000);",
                 "m.w = __builtin_amdgcn_raw_buffer_load_b32(bm_rsrc, ok ? 4u * (16u * s + (uint32_t)fr) : kOob, 0, 0);",
                 "m.base = __builtin_amdgcn_raw_buffer_load_b32(to_rsrc, ok ? 4u * s : kOob, 0, 0);",
                 "v.hw = (m.w >> (16 * h)) & 0xffffu;",
                 "const uint32_t off = m.base + half_inclusive_scan(cnt) - cnt;   // nibble index of my first value",
                 "const uint32_t* d = reinterpret_cast<const uint32_t*>(g.v4 + (byte0 & ~3u));",
                 "v.sh = (byte0 & 3u) * 8u + (off & 1u) * 4u;",
                 "const bool ok = p < pe && xlive && (int64_t)k0 < g.K;",
                 "x_rsrc, ok ? (uint32_t)fr * (uint32_t)g.K + k0 : kOob, 0, 0));",
                 "Meta m1 = load_meta(pb + 1);",
                 "const Meta m2 = load_meta(p + 2);",
                 "m1 = load_meta(p + 3);",
                 "for (int p = pb; p < pe; p += 2) {",
                 "const int L = (P + W - 1) / W;",
                 "const uint32_t y = i4_widen((uint32_t)(nibs >> (4u * rank)) & 0xFFFFu);   // ranks rank .. rank + 3",
                 "a[q] = __builtin_amdgcn_perm(0u, y, sel4[m4]);",
                 "return y | ((m << 5) - (m << 1));",
                 "int64_t int4_values_bytes(int64_t nnz) { return spl_values_bytes(SPL_I4, nnz); }",
                 "outside += (a < -8 || a > 7) + (b < -8 || b > 7);"):
        assert line in src, f"kernel changed: update this replay ({line})"
    Wq, mask, _ = getattr(synth, gen)(300 + N + K, N, K, s)
    T = orc.pack_tiled(Wq, "i8", mask)
    nnz = int(T.tile_offsets[-1])
    packed = np.zeros(_values_bytes(nnz), dtype=np.uint8)
    packed[:(nnz + 1) // 2] = orc.pack_i4(T.values)
    words = packed.view(np.uint32)
    B, S = (N + 15) // 16, (K + 31) // 32
    P = (S + 1) // 2
    dense = np.where(mask.astype(bool), Wq, np.int8(0))
    for b in range(B):
        L = (P + waves - 1) // waves
        for w in range(waves):
            pb = min(w * L, P)
            pe = min(pb + L, P)
            # every pair whose pattern the pipeline loads: two pairs per
            # iteration, pattern loads up to p + 3; a pair past the range
            # (or a tile past S) reads zeros through the buffer bounds
            last = pb + 2 * ((pe - pb + 1) // 2) + 1 if pe > pb else pb + 1
            for p in range(pb, last + 1):
                ok = p < pe
                hw = np.zeros(64, np.int64)
                base = np.zeros(64, np.int64)
                for lane in range(64):
                    fr, fg = lane & 15, lane >> 4
                    sk, h = 2 * p + (fg >> 1), fg & 1
                    if ok and 4 * (16 * sk + fr) < 64 * S:
                        assert 4 * sk < 4 * S
                        t = b * S + sk
                        hw[lane] = (int(T.bitmask[t * 16 + fr]) >> (16 * h)) & 0xFFFF
                        base[lane] = int(T.tile_offsets[t])
                cnt = np.array([bin(int(x)).count("1") for x in hw])
                for half in range(2):
                    seg = slice(32 * half, 32 * half + 32)
                    excl = np.cumsum(cnt[seg]) - cnt[seg]
                    for i, lane in enumerate(range(32 * half, 32 * half + 32)):
                        # every lane reads its three dwords, kept values or not
                        off = int(base[lane] + excl[i])
                        assert off + cnt[lane] <= nnz
                        byte0 = off >> 1
                        first = (byte0 & ~3) // 4
                        assert 0 <= first and (first + 3) * 4 <= packed.size, (b, w, p, lane)
                        if hw[lane] == 0:
                            continue
                        assert ok
                        d0, d1, d2 = (int(x) for x in words[first:first + 3])
                        sh = (byte0 & 3) * 8 + (off & 1) * 4
                        lo = ((d1 << 32 | d0) >> sh) & 0xFFFFFFFF
                        hi = ((d2 << 32 | d1) >> sh) & 0xFFFFFFFF
                        got, r = [], 0
                        for j in range(16):
                            if (int(hw[lane]) >> j) & 1:
                                nib = ((lo >> (4 * r)) if r < 8 else (hi >> (4 * (r - 8)))) & 0xF
                                got.append(nib - 16 if nib >= 8 else nib)
                                r += 1
                            else:
                                got.append(0)
                        # the kernel's formulation: per 4-column nibble, widen 4 nibbles, select by table
                        nibs, rank, got2 = (hi << 32) | lo, 0, []
                        for q in range(4):
                            m4 = (int(hw[lane]) >> (4 * q)) & 0xF
                            y = _widen((nibs >> (4 * rank)) & 0xFFFF)
                            got2 += _perm0(y, _selector(m4))
                            rank += bin(m4).count("1")
                        assert got2 == got, (b, w, p, lane)
                        fr, fg = lane & 15, lane >> 4
                        n = 16 * b + fr
                        k0 = 64 * p + 16 * fg
                        want = [int(dense[n, k0 + j]) if n < N and k0 + j < K else 0 for j in range(16)]
                        assert got == want, (b, w, p, lane)
