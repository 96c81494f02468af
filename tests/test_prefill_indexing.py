"""Host-side replay of the sparse prefill kernel's indexing (no GPU).

A workgroup of NW waves owns BN output rows (BN/16 row blocks) and walks K
in stages of two 32-column k-steps.  At every stage each wave expands TW
tiles: tile i is row block (TW/2) wave + i/2 of the workgroup, k-step
2 st + i % 2.  Lane (fr, fg) reads the tile's bitmask word of row fr, the
pair of tiles shares one exclusive wave scan of the lanes' kept counts (in
16-bit halves), and the lane loads two 8-byte value windows (unaligned) at
the first value of each of its nibbles.

This test replays that schedule with the constants read from the kernel
source and real encodings from the oracle, and checks that

  * every tile is expanded exactly once per workgroup, and tiles past the
    matrix (row blocks >= B, k-steps >= S) read tile 0's offset and a zero
    word;
  * every window lies inside the values buffer the interface guarantees
    (the payloads plus a 16-byte readable tail);
  * every expanded 16-byte chunk lands inside the workgroup's A buffer, in
    a distinct slot;
  * the expanded chunk (selector table + v_perm_b32) equals the dense
    masked row segment."""
import os
import re

import numpy as np
import pytest

import synth

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2405_03594_amd", "csrc", "k_prefill.hip")


def _constants():
    src = open(SRC).read()
    bk = int(re.search(r"constexpr int kPfBK = (\d+);", src).group(1))
    assert "constexpr int kPfRow = kPfBK * 2;" in src
    for line in ("constexpr int TW = BN / 8 / NW;",
                 "const int64_t wb = kGated ? (int64_t)blockIdx.x * (BN / 32) + (wave >> 1) : n0 / 16 + (TW / 2) * wave;",
                 "const int64_t b = wb + (i >> 1);",
                 "const int s = kI8 ? 4 * st + 2 * (i & 1) + (fg >> 1) : 2 * st + (i & 1);",
                 "const int64_t t = ok ? b * S + s : 0;",
                 "tw.w[i] = ok ? bm_tiles[t * 16 + fr] : 0u;",
                 "const uint32_t pc = __popc(b0) | (__popc(b1) << 16);",
                 "const uint32_t oa = (uint32_t)tw.off[i + h] + (h ? ex >> 16 : ex & 0xffffu);",
                 "const uint32_t ob = oa + __popc(byte & 0xfu);",
                 "__builtin_memcpy(&tv.v0[i + h], vbytes + 2u * oa, 8);",
                 "__builtin_memcpy(&tv.v1[i + h], vbytes + 2u * ob, 8);",
                 "const uint32_t at = buf + pf_chunk(16 * ((TW / 2) * wave + (i >> 1)) + fr, 4 * (i & 1) + fg);",
                 "if (pf_large_tile(a.N, a.M)) return sparse_prefill_tile<T, 128, 256, 8, 1>(a, s);",
                 "return pf_split_k(a.N, a.M) ? sparse_prefill_tile<T, 64, 128, 4, 2>(a, s)",
                 ": sparse_prefill_tile<T, 64, 128, 4, 1>(a, s);",
                 "fetch_words(tw, sb + 1);",
                 "if (st + 3 < nl) fetch_words(tw, sb + st + 3);"):
        assert line in src, f"kernel changed: update this replay ({line})"
    return bk, [(128, 8), (64, 4)]                      # (BN, NW) of the two workgroup shapes


def _popc(x):
    return bin(int(x) & 0xFFFFFFFF).count("1")


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


def _perm(s0, s1, sel):
    src = int(s1).to_bytes(4, "little") + int(s0).to_bytes(4, "little")
    out = 0
    for j in range(4):
        b = (sel >> (8 * j)) & 0xFF
        assert b < 8 or b == 12
        out |= (src[b] if b < 8 else 0) << (8 * j)
    return out


def _chunk(r, c, row_bytes):
    return r * row_bytes + 16 * (c ^ (r & 7))


@pytest.mark.parametrize("N,K,s", [(16, 32, 0.5), (48, 200, 0.7), (300, 96, 0.0), (33, 264, 1.0), (130, 520, 0.9)])
def test_prefill_schedule_and_expansion(orc, N, K, s):
    bk, shapes = _constants()
    row_bytes = 2 * bk
    W, mask = synth.weight(57 + N + K, N, K, "bf16", s)
    T = orc.pack_tiled(W, "bf16", mask)
    vbytes = np.concatenate([T.values.view(np.uint8), np.zeros(16, np.uint8)])   # the readable tail
    limit = 2 * T.nnz + 16
    dense = np.where(mask.astype(bool), W.view(np.uint16), 0).astype(np.uint16)
    S, B = -(-K // 32), -(-N // 16)
    nst = (S + 1) // 2
    bm = T.bitmask.reshape(-1).astype(np.uint64)
    offs = T.tile_offsets.astype(np.int64)
    for BN, NW in shapes:
        TW = BN // 8 // NW
        assert TW % 2 == 0
        for wg in range(-(-N // BN)):
            nb0 = wg * BN // 16
            for st in range(nst):
                seen = {}
                for wave in range(NW):
                    for i in range(0, TW, 2):
                        tiles = []
                        for h in range(2):
                            b = nb0 + (TW // 2) * wave + ((i + h) >> 1)
                            sk = 2 * st + ((i + h) & 1)
                            ok = b < B and sk < S
                            t = b * S + sk if ok else 0
                            words = [int(bm[t * 16 + r]) if ok else 0 for r in range(16)]
                            tiles.append((b, sk, ok, int(offs[t]), words))
                            if ok:
                                assert (b, sk) not in seen, "tile expanded twice"
                                seen[(b, sk)] = True
                        # the pair's scan: counts in lane order (fg-major, fr within), 16-bit halves
                        cnt = np.array([[_popc((tiles[h][4][l & 15] >> (8 * (l >> 4))) & 0xFF) for l in range(64)]
                                        for h in range(2)])
                        packed = cnt[0] | (cnt[1] << 16)
                        ex = np.cumsum(packed) - packed
                        assert (np.cumsum(cnt, axis=1) <= 512).all()
                        for h in range(2):
                            b, sk, ok, off, words = tiles[h]
                            for lane in range(64):
                                fr, fg = lane & 15, lane >> 4
                                byte = (words[fr] >> (8 * fg)) & 0xFF
                                e = int(ex[lane] >> 16) if h else int(ex[lane] & 0xFFFF)
                                oa = off + e
                                ob = oa + _popc(byte & 0xF)
                                for o in (oa, ob):
                                    assert 0 <= 2 * o and 2 * o + 8 <= limit, (wg, st, wave, i + h, lane)
                                at = _chunk(16 * ((TW // 2) * wave + ((i + h) >> 1)) + fr, 4 * ((i + h) & 1) + fg,
                                            row_bytes)
                                assert 0 <= at and at + 16 <= BN * row_bytes
                                v0 = vbytes[2 * oa:2 * oa + 8].view(np.uint32)
                                v1 = vbytes[2 * ob:2 * ob + 8].view(np.uint32)
                                lo, hi = byte & 0xF, byte >> 4
                                got = [_perm(v0[1], v0[0], _nibble_selector(lo, 0)),
                                       _perm(v0[1], v0[0], _nibble_selector(lo, 1)),
                                       _perm(v1[1], v1[0], _nibble_selector(hi, 0)),
                                       _perm(v1[1], v1[0], _nibble_selector(hi, 1))]
                                got = np.array(got, dtype=np.uint32).view(np.uint16)
                                exp = np.zeros(8, np.uint16)
                                n, k0 = 16 * b + fr, 32 * sk + 8 * fg
                                if ok and n < N and k0 < K:
                                    seg = dense[n, k0:min(k0 + 8, K)]
                                    exp[:seg.size] = seg
                                assert np.array_equal(got, exp), (wg, st, wave, i + h, lane)
                # the workgroup's row blocks inside the matrix, both k-steps of the stage, each once
                want = {(b, sk) for b in range(nb0, min(nb0 + BN // 16, B)) for sk in (2 * st, 2 * st + 1) if sk < S}
                assert set(seen) == want


def _inside_rule():
    src = open(SRC).read()
    rule = "return N % BN == 0 && M % BM == 0 && K % kPfBK == 0;"
    assert rule in src, "launch rule for the unchecked kernels changed: update this replay"
    for line in ("return pf_inside(a.N, a.M, pf_units<T>(a.K), BN, BM) ? sparse_prefill_launch<T, BN, BM, NW, KS, false>(a, s)",
                 "return pf_inside(a.N, a.M, pf_units<T>(a.K), BN, BM)\n             ? dense_prefill_launch<T, BN, BM, NW, KS, false, kGather>(a, s)",
                 "const int64_t t = b * S + s;",
                 "for (int i = 0; i < P; ++i) sl.v[i] = *reinterpret_cast<const u32x4*>(row0 + i * stride + k0);"):
        assert line in src, f"kernel changed: update this replay ({line})"
    return lambda N, M, K, BN, BM, bk: N % BN == 0 and M % BM == 0 and K % bk == 0


@pytest.mark.parametrize("N,M,K", [(4096, 512, 4096), (11008, 2048, 4096), (4096, 2048, 11008), (128, 256, 64),
                                   (64, 128, 128), (2000, 4100, 72), (130, 300, 1000)])
def test_unchecked_loads_stay_inside(N, M, K):
    """Launches the host sends to the unchecked kernels (every block and stage
    inside the matrix) touch only valid tiles, rows and columns."""
    bk, shapes = _constants()
    inside = _inside_rule()
    S, B = -(-K // 32), -(-N // 16)
    nst = (S + 1) // 2
    for BN, NW in shapes:
        BM, RR, TW = 32 * NW, 8 * NW, BN // 8 // NW
        if not inside(N, M, K, BN, BM, bk):
            continue
        # tiles: b = nb0 + (TW/2) wave + i/2 over every workgroup and wave, k-step 2 st + i % 2
        bs = {wg * BN // 16 + (TW // 2) * w + i // 2 for wg in range(N // BN) for w in range(NW) for i in range(TW)}
        assert max(bs) < B and 2 * (nst - 1) + 1 < S
        # slabs: rows r0 + t/8 + RR i of BM (X) and BN (W) rows, columns k0 + 8 (t % 8) .. + 8 of every stage
        for rows, R in ((BM, M), (BN, N)):
            last = (R // rows - 1) * rows + (64 * NW - 1) // 8 + RR * (rows // RR - 1)
            assert last < R
        assert bk * (nst - 1) + 8 * 7 + 8 <= K


def _split_rule():
    src = open(SRC).read()
    for line in ("const int nh = (nst + KS - 1) / KS;",
                 "const int sb = kh * nh;",
                 "const int nl = nst - sb < nh ? (nst > sb ? nst - sb : 0) : nh;",
                 "if (st < nl) pf_mfma_stage<T, FN, FM>(acc, abuf[cur], bbuf[cur], wn, wm, fr, fg);",
                 "if (st + 1 < nh) __syncthreads();",
                 "unsigned char* gb = dsm + kh * pf_lds(BN, BM);",
                 "A* part = reinterpret_cast<A*>(dsm);             // [FN * FM][NT]"):
        assert line in src, f"split-K schedule changed: update this replay ({line})"


@pytest.mark.parametrize("nst", [1, 2, 3, 4, 5, 64, 172])
@pytest.mark.parametrize("KS", [1, 2])
def test_split_k_stages_partition(nst, KS):
    """The k-groups' stage ranges [sb, sb + nl) partition [0, nst); every group
    runs the same number of barriers (derived from nh only); the partial sums
    of the two-group kernel fit the LDS it is launched with."""
    _split_rule()
    bk, _ = _constants()
    nh = -(-nst // KS)
    seen = []
    barriers = set()
    for kh in range(KS):
        sb = kh * nh
        nl = (max(nst - sb, 0)) if nst - sb < nh else nh
        seen += list(range(sb, sb + nl))
        # prologue barriers + one per stage transition + the combine's two
        barriers.add(2 + (nh - 1) + (2 if KS == 2 else 0))
    assert seen == list(range(nst)) and len(barriers) == 1
    BN, BM, NW = 64, 128, 4
    lds = 2 * (BN + BM) * 2 * bk
    assert (BN // 32) * 4 * 64 * NW * 16 <= KS * lds



# ---------------------------------------------------------------- int8 payloads

def _i8_lines():
    src = open(SRC).read()
    for line in ("const uint32_t h0 = __builtin_amdgcn_ubfe(tw.w[i], 16 * (fg & 1), 16);",
                 "const uint32_t ex = half_inclusive_scan(pc) - pc;",
                 "const uint32_t ob = oa + __popc(hw & 0xffu);   // nibbles 2 and 3 start after nibbles 0 and 1",
                 "__builtin_memcpy(&tv.v0[i + h], vbytes + oa, 8);",
                 "__builtin_memcpy(&tv.v1[i + h], vbytes + ob, 8);",
                 "const uint32_t s1 = lds_load4(lut_addr + 20u * n1 + 4u * __popc(n0_));",
                 "const uint32_t s3 = lds_load4(lut_addr + 20u * n3 + 4u * __popc(n2));",
                 "if (threadIdx.x < 80) lut[threadIdx.x] = nibble_selector8(threadIdx.x / 5, threadIdx.x % 5);",
                 "const int nst = (int)((Kh + kPfBK - 1) / kPfBK);   // stages of 128 bytes per row: 2 tiles (4 for int8)",
                 "const int64_t Kh = kI8 ? K / 2 : K;                // activation row in 16-bit units"):
        assert line in src, f"int8 expansion changed: update this replay ({line})"


def _i8_selector(nib, p):
    sel = 0
    for j in range(4):
        b = 0x0C
        if (nib >> j) & 1:
            b = p + _popc(nib & ((1 << j) - 1))
        sel |= b << (8 * j)
    return sel


@pytest.mark.parametrize("N,K,s", [(16, 128, 0.5), (48, 400, 0.7), (130, 256, 0.0), (33, 528, 1.0), (70, 1040, 0.9)])
def test_prefill_i8_schedule_and_expansion(orc, N, K, s):
    """int8 payloads: per stage (128 columns) a wave expands two tile pairs of
    its row block; lane (fr, fg) takes tile 4 st + 2 (i % 2) + fg / 2, columns
    16 (fg % 2) .. +16 of row fr; its values start at the tile offset plus the
    exclusive scan over the tile's 32 lanes; two 8-byte windows (nibbles 0-1
    and 2-3) and the offset-aware selectors rebuild the 16 dense bytes."""
    _i8_lines()
    bk, shapes = _constants()
    row_bytes = 2 * bk
    Wq, mask, _ = synth.int8_weight(77 + N + K, N, K, s)
    T = orc.pack_tiled(Wq, "i8", mask)
    vbytes = np.concatenate([T.values.view(np.uint8), np.zeros(16, np.uint8)])
    limit = T.nnz + 16
    dense = np.where(mask.astype(bool), Wq, 0).astype(np.int8).view(np.uint8)
    S, B = -(-K // 32), -(-N // 16)
    nst = -(-(K // 2) // bk)
    bm = T.bitmask.reshape(-1).astype(np.uint64)
    offs = T.tile_offsets.astype(np.int64)
    for BN, NW in shapes:
        TW = BN // 8 // NW
        for wg in range(-(-N // BN)):
            nb0 = wg * BN // 16
            for st in range(nst):
                seen = set()
                for wave in range(NW):
                    for i in range(0, TW, 2):
                        units = []
                        for h in range(2):
                            b = nb0 + (TW // 2) * wave + ((i + h) >> 1)
                            lanes = []
                            for lane in range(64):
                                fr, fg = lane & 15, lane >> 4
                                sk = 4 * st + 2 * ((i + h) & 1) + (fg >> 1)
                                ok = b < B and sk < S
                                t = b * S + sk if ok else 0
                                w = int(bm[t * 16 + fr]) if ok else 0
                                hw = (w >> (16 * (fg & 1))) & 0xFFFF
                                lanes.append((b, sk, ok, int(offs[t]), hw))
                                if ok:
                                    seen.add((b, sk))
                            units.append(lanes)
                        cnt = np.array([[_popc(units[h][l][4]) for l in range(64)] for h in range(2)])
                        ex = np.zeros((2, 64), np.int64)
                        for h in range(2):
                            for half in range(2):
                                seg = cnt[h, 32 * half:32 * half + 32]
                                ex[h, 32 * half:32 * half + 32] = np.cumsum(seg) - seg
                                assert seg.sum() <= 512
                        for h in range(2):
                            for lane in range(64):
                                fr, fg = lane & 15, lane >> 4
                                b, sk, ok, off, hw = units[h][lane]
                                oa = off + int(ex[h, lane])
                                ob = oa + _popc(hw & 0xFF)
                                for o in (oa, ob):
                                    assert 0 <= o and o + 8 <= limit, (wg, st, wave, i + h, lane)
                                at = _chunk(16 * ((TW // 2) * wave + ((i + h) >> 1)) + fr, 4 * ((i + h) & 1) + fg,
                                            row_bytes)
                                assert 0 <= at and at + 16 <= BN * row_bytes
                                v0 = vbytes[oa:oa + 8].view(np.uint32)
                                v1 = vbytes[ob:ob + 8].view(np.uint32)
                                n = [(hw >> (4 * j)) & 15 for j in range(4)]
                                got = [_perm(v0[1], v0[0], _i8_selector(n[0], 0)),
                                       _perm(v0[1], v0[0], _i8_selector(n[1], _popc(n[0]))),
                                       _perm(v1[1], v1[0], _i8_selector(n[2], 0)),
                                       _perm(v1[1], v1[0], _i8_selector(n[3], _popc(n[2])))]
                                got = np.array(got, dtype=np.uint32).view(np.uint8)
                                exp = np.zeros(16, np.uint8)
                                row, k0 = 16 * b + fr, 32 * sk + 16 * (fg & 1)
                                if ok and row < N and k0 < K:
                                    seg = dense[row, k0:min(k0 + 16, K)]
                                    exp[:seg.size] = seg
                                assert np.array_equal(got, exp), (wg, st, wave, i + h, lane)
                want = {(b, sk) for b in range(nb0, min(nb0 + BN // 16, B)) for sk in range(4 * st, 4 * st + 4)
                        if sk < S}
                assert seen == want


@pytest.mark.parametrize("N", [16, 40, 64, 100, 128, 11008])
@pytest.mark.parametrize("BN,NW", [(128, 8), (64, 4)])
def test_gated_block_assignment(N, BN, NW):
    """Gated prefill: wave w of workgroup x expands row block x BN/32 + w/2 of
    matrix w % 2; over the grid of ceil(N / (BN/2)) workgroups every row block
    of both matrices is expanded exactly once, the others are past the last
    block (the checked loads skip them), and when N % (BN/2) == 0 (the
    unchecked instantiation) none is past it.  Fragments 2p, 2p + 1 of wave
    (wn, wm) are virtual blocks wn FN + 2p, + 1: gate and up of one real block."""
    src = open(SRC).read()
    for line in ("const int gm = kGated ? (wave & 1) : 0;",
                 "constexpr int RN = kGated ? BN / 2 : BN;",
                 "return pf_inside(2 * a.N, a.M, a.K, BN, BM) ? sparse_prefill_launch<T, BN, BM, NW, KS, false, true>(a, s)",
                 "const int64_t n = n0 + wn * 8 * FN + 16 * p + 4 * fg;"):
        assert line in src, f"kernel changed: update this replay ({line})"
    B = (N + 15) // 16
    grid = (N + BN // 2 - 1) // (BN // 2)
    seen = []
    for x in range(grid):
        for w in range(NW):
            b = x * (BN // 32) + (w >> 1)
            if b < B:
                seen.append((w & 1, b))
            else:
                assert N % (BN // 2) != 0
    assert sorted(seen) == sorted((m, b) for m in (0, 1) for b in range(B))
    assert len(seen) == len(set(seen))
    FN = BN // 32
    for wn in range(2):
        for p in range(FN // 2):
            g, u = wn * FN + 2 * p, wn * FN + 2 * p + 1      # virtual blocks of the fragments (= expanding waves)
            assert g % 2 == 0 and u % 2 == 1 and g >> 1 == u >> 1
            assert (g >> 1) * 16 == wn * 8 * FN + 16 * p      # the real rows pf_store_gated writes


# ---------------------------------------------------------------- the gather epilogue (weight gradients)

def _gather_lines():
    src = open(SRC).read()
    for line in ("const int64_t b0 = (m0 + wm * 16 * FM) / 16, s0 = (n0 + wn * 16 * FN) / 32;",
                 "constexpr int FM = BM / (8 * NW);",
                 "constexpr int FN = 4, FM = kDmaBM / (8 * NW);",
                 "constexpr int kDmaBN = 128, kDmaBM = 256, kDmaStages = 3, kDmaWaves = 8;",
                 "pf_store_gather<T, FN, FM>(acc, g, n0, m0, wn, wm, lane);",
                 "pf_gather_meta<FN, FM>(gm, g, n0, m0, wn, wm, lane);",
                 "pf_store_gather<T, FN, FM>(acc, gm, g, lane);",
                 "const bool ok = b0 + j < B && s0 + p < S;",
                 "gm.w[j][p] = ok ? g.gbm[((b0 + j) * S + s0 + p) * 16 + fr] : 0u;",
                 "const int jl = lane / (FN / 2), pl = lane % (FN / 2);",
                 "const bool okl = lane < FM * FN / 2 && b0 + jl < B && s0 + pl < S;",
                 "gm.off = okl ? (uint32_t)g.gtoff[(b0 + jl) * S + s0 + pl] : 0u;",
                 "const uint32_t w = gm.w[j][p];",
                 "const uint32_t base = (uint32_t)__builtin_amdgcn_readlane((int)gm.off, j * (FN / 2) + p);",
                 "uint32_t idx = n + __builtin_amdgcn_ubfe(above, 8 * f, 8);   // within the run",
                 "if ((nib >> r) & 1u) run[1024 * j + idx++] = v[r];",
                 "n += (tot & 0xffu) + ((tot >> 8) & 0xffu) + ((tot >> 16) & 0xffu) + (tot >> 24);",
                 "const uint32_t base0 = (uint32_t)__builtin_amdgcn_readlane((int)gm.off, j * (FN / 2));",
                 "for (uint32_t i = (uint32_t)lane; i < len[j]; i += 64) g.gval[base0 + i] = run[1024 * j + i];",
                 "pf_store_gather_lds<T, FN, FM>(acc, gm, g, lane, reinterpret_cast<uint16_t*>(dsm) + 1024 * FM * wave);",
                 "const uint32_t incl = row16_inclusive_scan(c);",
                 "const uint32_t tot = (uint32_t)__builtin_amdgcn_readlane((int)incl, 15);",
                 "const uint32_t above = incl - c;",
                 "const int col = 16 * h + 4 * q;",
                 "uint32_t idx = base + __builtin_amdgcn_ubfe(above, 8 * f, 8);",
                 "if (col & 4) idx += __popc(__builtin_amdgcn_ubfe(w, 8 * f, 4));",
                 "const uint32_t nib = __builtin_amdgcn_ubfe(w, col, 4);",
                 "if ((nib >> r) & 1u) g.gval[idx++] = T::from_f32(acc[2 * p + h][j][r]);",
                 "if (pf_large_tile(a.N, a.M)) return dense_prefill_tile<T, 128, 256, 8, 1, kGather>(a, s);",
                 "return pf_split_k(a.N, a.M) ? dense_prefill_tile<T, 64, 128, 4, 2, kGather>(a, s)"):
        assert line in src, f"gather epilogue changed: update this replay ({line})"
    # (BN, BM, NW): the 8-wave cores (register-staged and direct-to-LDS) and the 4-wave core;
    # (128, 256, 4) checks the epilogue's general m-fragment count (FM = 8)
    return [(128, 256, 8), (64, 128, 4), (128, 256, 4)]


@pytest.mark.parametrize("R,C,s", [(24, 64, 0.6), (100, 1000, 0.7), (300, 264, 0.5), (33, 512, 0.9), (130, 96, 0.0),
                                   (16, 32, 1.0), (257, 136, 0.5)])
def test_gather_epilogue_writes_the_value_order(orc, R, C, s):
    """The product G [R][C] is written only at the kept positions of its tile
    pattern: replaying every workgroup's waves (D layout: lane l holds tile
    row l % 16, columns 16 h + 4 (l / 16) + r of fragment 2p + h) writes each
    value index exactly once, and what lands there is the oracle's tile-layout
    value of G at that index."""
    W, mask = synth.weight(71 + R + C, R, C, "bf16", s)
    T = orc.pack_tiled(W, "bf16", mask)
    rng = np.random.default_rng(R * 1000 + C)
    G = rng.integers(1, 60000, size=(R, C)).astype(np.uint16)        # distinct-enough payloads; position-tagged
    want = orc.pack_tiled(G, "bf16", mask).values
    B, S = -(-R // 16), -(-C // 32)
    bm = T.bitmask.reshape(-1).astype(np.int64)
    offs = T.tile_offsets.astype(np.int64)
    for BN, BM, NW in _gather_lines():
        FN, FM = BN // 32, BM // (8 * NW)
        out = np.zeros(T.nnz, np.uint16)
        hits = np.zeros(T.nnz, np.int64)
        runs, run_info = {}, {}
        for gx in range(-(-C // BN)):                 # product columns = pattern columns
            for gy in range(-(-R // BM)):             # product rows = pattern rows
                n0, m0 = gx * BN, gy * BM
                for wave in range(NW):
                    wn, wm = wave & 1, wave >> 1
                    b0, s0 = (m0 + wm * 16 * FM) // 16, (n0 + wn * 16 * FN) // 32
                    # the pattern loads: words per tile (zero past the pattern), tile i's offset in lane i
                    off = []
                    for lane in range(64):
                        jl, pl = lane // (FN // 2), lane % (FN // 2)
                        okl = lane < FM * FN // 2 and b0 + jl < B and s0 + pl < S
                        off.append(int(offs[(b0 + jl) * S + s0 + pl]) if okl else 0)
                    for j in range(FM):
                        for p in range(FN // 2):
                            b, st = b0 + j, s0 + p
                            ok = b < B and st < S
                            t = b * S + st
                            words = [int(bm[t * 16 + fr]) if ok else 0 for fr in range(16)]
                            assert j * (FN // 2) + p < 64
                            base = off[j * (FN // 2) + p]
                            assert not ok or base == int(offs[t])
                            key = (gx, gy, wave, j)
                            runs.setdefault(key, [])
                            rb0, ln = run_info.get(key, (off[j * (FN // 2)], 0))
                            run_info[key] = (rb0, ln + sum(_popc(wd) for wd in words))
                            c = [sum(_popc((w >> (8 * f)) & 0xFF) << (8 * f) for f in range(4)) for w in words]
                            incl = np.cumsum(c)
                            assert all(((int(x) >> (8 * f)) & 0xFF) <= 128 for x in incl for f in range(4))
                            tot = int(incl[15])
                            for lane in range(64):
                                fr, q = lane & 15, lane >> 4
                                w = words[fr]
                                above = int(incl[fr]) - c[fr]
                                for h in range(2):
                                    col = 16 * h + 4 * q
                                    f = col >> 3
                                    idx = base + ((above >> (8 * f)) & 0xFF)
                                    idx += sum((tot >> (8 * g)) & 0xFF for g in range(f))
                                    if col & 4:
                                        idx += _popc((w >> (8 * f)) & 0xF)
                                    nib = (w >> col) & 0xF
                                    for r in range(4):
                                        if (nib >> r) & 1:
                                            row, k = 16 * b + fr, 32 * st + col + r
                                            assert row < R and k < C
                                            out[idx] = G[row, k]
                                            hits[idx] += 1
                                            runs[key].append(idx)
                                            idx += 1
        assert (hits == 1).all(), (BN, "value index written other than once")
        assert np.array_equal(out, want), BN
        if (BN, BM, NW) == (128, 256, 8):
            # the LDS-staged form (the weight gradient's core): tiles (j, 0) and (j, 1) of a wave are one run
            # of nnz(j, 0) + nnz(j, 1) entries from tile (j, 0)'s offset, each slot < 1024 written once
            for key, idxs in runs.items():
                base0, length = run_info[key]
                assert length <= 1024
                assert sorted(i - base0 for i in idxs) == list(range(length)), key


# ---------------------------------------------------------------- direct-to-LDS staging of the dense core

def _dma_lines():
    src = open(SRC).read()
    for line in ("constexpr int kDmaBN = 128, kDmaBM = 256, kDmaStages = 3, kDmaWaves = 8;",
                 "constexpr int GA = kDmaBN / 8 / NW, GB = kDmaBM / 8 / NW;",
                 "const int lr = lane >> 3, lc = (lane & 7) ^ lr;",
                 "const uint16_t* wsrc = g.W + (n0 + 8 * GA * wave + lr) * Kh + 8 * lc;",
                 "const uint16_t* xsrc = g.X + (m0 + 8 * GB * wave + lr) * Kh + 8 * lc;",
                 "lds_dma16(src + 8 * K * i + kPfBK * st, buf + (8 * kGroups * wave + 8 * i) * kPfRow);",
                 "dma_rows<GA>(wsrc, Kh, st, a, wave);",
                 "dma_rows<GB>(xsrc, Kh, st, a + kDmaBN * kPfRow, wave);",
                 "const int64_t Kh = kI8 ? K / 2 : K;",
                 "if (st + 2 < nst) request(st + 2, cur == 0 ? 2 : cur - 1);",
                 "if (pf_large_tile(a.N, a.M) && pf_inside(a.N, a.M, pf_units<T>(a.K), kDmaBN, kDmaBM))"):
        assert line in src, f"direct-to-LDS staging changed: update this replay ({line})"
    return 128, 256, 8


@pytest.mark.parametrize("N,M,K", [(4096, 2048, 4096), (11008, 512, 4096), (4096, 256, 11008), (128, 256, 64),
                                   (4096, 2048, 5504)])
def test_dma_requests_fill_the_swizzled_stage(N, M, K):
    """One stage's direct-to-LDS requests of a workgroup: lane i of a request
    fills 16-byte slot i of a 1 KB run.  Every (row, chunk) of the W and X
    stage lands exactly once, at the swizzled place the MFMA reads use
    (pf_chunk: chunk c of row r at position c ^ (r % 8)), from inside the
    matrices; the three stage buffers rotate so that a request never hits
    the buffer being multiplied or the one published next.  K counts 16-bit
    units (an int8 row of K codes is K / 2 of them: 5504 for the down shape)."""
    BN, BM, NW = _dma_lines()
    bk, _ = _constants()
    row_bytes = 2 * bk
    GA, GB = BN // 8 // NW, BM // 8 // NW
    assert N % BN == 0 and M % BM == 0 and K % bk == 0
    nst = K // bk
    for n0, m0 in ((0, 0), (N - BN, M - BM)):
        for st in (0, nst - 1):
            for rows0, R, groups, region, nrows in ((n0, N, GA, 0, BN), (m0, M, GB, BN * row_bytes, BM)):
                seen = {}
                for wave in range(NW):
                    for i in range(groups):
                        for lane in range(64):
                            lr, lc = lane >> 3, (lane & 7) ^ (lane >> 3)
                            row = rows0 + 8 * groups * wave + lr + 8 * i        # global row
                            col = bk * st + 8 * lc                             # first element of the chunk
                            assert row < R and col + 8 <= K
                            slot = region + (8 * groups * wave + 8 * i) * row_bytes + 16 * lane
                            r = row - rows0                                    # row within the stage buffer
                            assert slot == region + _chunk(r, lc, row_bytes), (wave, i, lane)
                            assert (r, lc) not in seen
                            seen[(r, lc)] = True
                assert len(seen) == nrows * 8
    # buffer rotation: stage st + 2 goes to (st + 2) % 3, never st % 3 (being read) or (st + 1) % 3
    for st in range(12):
        cur = st % 3
        target = 2 if cur == 0 else cur - 1
        assert target == (st + 2) % 3 and target not in (st % 3, (st + 1) % 3)


# ---------------------------------------------------------------- tile-layout expansion (spl_unpack's fast kernels)

PACK_SRC = os.path.join(os.path.dirname(SRC), "k_pack.hip")


def _expand_lines():
    src = open(PACK_SRC).read()
    for line in ("constexpr int kExpandTiles = 4;",
                 "const int64_t t0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * kExpandTiles;",
                 "byte[i] = live ? (bm_tiles[(t0 + i) * 16 + fr] >> (8 * fg)) & 0xffu : 0u;",
                 "const uint32_t pc = __popc(byte[i]) | (__popc(byte[i + 1]) << 16);",
                 "const uint32_t ex = wave_inclusive_scan(pc) - pc;",
                 "__builtin_memcpy(&v1[i], values + oa[i] + __popc(byte[i] & 0xfu), 8);",
                 "const int64_t k0 = (t % S) * 32 + 8 * fg;",
                 "*reinterpret_cast<u32x4*>(Wd + n * K + k0) = a;",
                 "const int64_t t0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * 2 * kExpandTiles;",
                 "const int64_t t = t0 + 2 * p + (lane >> 5);",
                 "hw[p] = live ? (bm_tiles[t * 16 + r] >> (16 * gq)) & 0xffffu : 0u;",
                 "const uint32_t ex = half_inclusive_scan(pc) - pc;",
                 "const int64_t k0 = (t % S) * 32 + 16 * gq;",
                 "__builtin_memcpy(&v1[p], values + oa[p] + __popc(hw[p] & 0xffu), 8);",
                 "a.y = __builtin_amdgcn_perm(v0[p].y, v0[p].x, lut[5 * q1 + __popc(q0)]);",
                 "a.w = __builtin_amdgcn_perm(v1[p].y, v1[p].x, lut[5 * q3 + __popc(q2)]);",
                 "if (Wc.dtype == SPL_I8 && Wc.cols % 16 == 0) {"):
        assert line in src, f"expansion changed: update this replay ({line})"
    # every tile is one wave's (16-bit) or half-wave's (int8) unit; the scans of a wave's tiles,
    # two per scan in 16-bit halves, are each tile's own (sums <= 512)


@pytest.mark.parametrize("dtype", ["bf16", "i8"])
@pytest.mark.parametrize("N,K,s", [(16, 32, 0.5), (33, 64, 0.7), (100, 1008, 0.0), (17, 96, 1.0), (48, 4096, 0.9)])
def test_expand_tiles_rebuild_the_dense_matrix(orc, dtype, N, K, s):
    """Every lane of the expansion kernels, replayed: its windows stay inside
    the payload + 16 readable bytes, and the 16-byte pieces it stores are the
    oracle's dense masked matrix (16-bit: 8 columns per lane of a 64-lane tile;
    int8: 16 columns per lane of a 32-lane half-wave tile)."""
    _expand_lines()
    if dtype == "i8":
        W, mask, _ = synth.int8_weight(77 + N + K, N, K, s)
        eb, width = 1, 16
    else:
        W, mask = synth.weight(77 + N + K, N, K, dtype, s)
        eb, width = 2, 8
    T = orc.pack_tiled(W, dtype, mask)
    vbytes = np.concatenate([T.values.view(np.uint8), np.zeros(16, np.uint8)])
    dense = np.where(mask.astype(bool), W, np.zeros_like(W)).view(np.uint8).reshape(N, K * eb)
    S, B = -(-K // 32), -(-N // 16)
    bm = T.bitmask.reshape(-1).astype(np.int64)
    offs = T.tile_offsets.astype(np.int64)
    got = np.zeros((N, K * eb), np.uint8)
    lanes = 64 if eb == 2 else 32
    for t in range(B * S):
        cnt = []
        for l in range(lanes):
            r, g = l & 15, l >> 4
            bits = (int(bm[t * 16 + r]) >> (width * g)) & ((1 << width) - 1)
            cnt.append(_popc(bits))
        ex = np.cumsum(cnt) - np.array(cnt)
        for l in range(lanes):
            r, g = l & 15, l >> 4
            n, k0 = (t // S) * 16 + r, (t % S) * 32 + width * g
            bits = (int(bm[t * 16 + r]) >> (width * g)) & ((1 << width) - 1)
            if n >= N or k0 >= K:
                assert bits == 0
                continue
            oa = int(offs[t]) + int(ex[l])
            if eb == 2:
                ob = oa + _popc(bits & 0xF)
                assert 2 * ob + 8 <= 2 * T.nnz + 16
                v0 = vbytes[2 * oa:2 * oa + 8].view(np.uint32)
                v1 = vbytes[2 * ob:2 * ob + 8].view(np.uint32)
                words = [_perm(v0[1], v0[0], _nibble_selector(bits & 0xF, 0)),
                         _perm(v0[1], v0[0], _nibble_selector(bits & 0xF, 1)),
                         _perm(v1[1], v1[0], _nibble_selector(bits >> 4, 0)),
                         _perm(v1[1], v1[0], _nibble_selector(bits >> 4, 1))]
            else:
                q = [(bits >> (4 * i)) & 0xF for i in range(4)]
                ob = oa + _popc(bits & 0xFF)
                assert ob + 8 <= T.nnz + 16
                v0 = vbytes[oa:oa + 8].view(np.uint32)
                v1 = vbytes[ob:ob + 8].view(np.uint32)
                words = [_perm(v0[1], v0[0], _i8_selector(q[0], 0)),
                         _perm(v0[1], v0[0], _i8_selector(q[1], _popc(q[0]))),
                         _perm(v1[1], v1[0], _i8_selector(q[2], 0)),
                         _perm(v1[1], v1[0], _i8_selector(q[3], _popc(q[2])))]
            piece = np.array(words, np.uint32).view(np.uint8)
            assert k0 * eb + 16 <= K * eb
            got[n, k0 * eb:k0 * eb + 16] = piece
    assert np.array_equal(got, dense)


# ---------------------------------------------------------------- contraction-major factors (the weight gradient)

TRAIN_SRC = os.path.join(os.path.dirname(SRC), "k_train.hip")


def _tr_lines():
    src = open(SRC).read()
    for line in ("constexpr int kTrRowA = 2 * kDmaBN, kTrRowB = 2 * kDmaBM;",
                 "constexpr int kTrOffB = kPfBK * kTrRowA;",
                 "constexpr int RA = kPfBK * kTrRowA / 1024 / NW, RB = kPfBK * kTrRowB / 1024 / NW;",
                 "const int hw = (wave & 1) << 2;",
                 "const uint16_t* wsrc = g.W + (int64_t)(8 * wave + (lane >> 4)) * N + n0 + 8 * ((lane & 15) ^ "
                 "(2 * ((lane >> 4) | hw)));",
                 "xsrc[p] = g.X + (int64_t)(8 * wave + 2 * p + (lane >> 5)) * M + m0 + 8 * ((lane & 31) ^ "
                 "(2 * ((2 * p + (lane >> 5)) | hw)));",
                 "for (int u = 0; u < RA; ++u) lds_dma16_opaque(wsrc + (k0 + 4 * u) * N, a + (RA * wave + u) * 1024);",
                 "lds_dma16_opaque(xsrc[u & 1] + (k0 + 4 * (u >> 1)) * M, a + kTrOffB + (RB * wave + u) * 1024);",
                 "const int t = lane & 15, r0 = 8 * (lane >> 4) + (t >> 2);",
                 "const int h = (t >> 2) | (((lane >> 4) & 1) << 2);",
                 "ao[i] = (uint32_t)(r0 * kTrRowA + 16 * ((8 * wn + 2 * i + ((t & 3) >> 1)) ^ (2 * h)) + 8 * (t & 1));",
                 "bo[j] = (uint32_t)(kTrOffB + r0 * kTrRowB + 16 * ((8 * wm + 2 * j + ((t & 3) >> 1)) ^ (2 * h)) + "
                 "8 * (t & 1));",
                 "const uint32_t p = buf + ao[i] + 32 * kTrRowA * ks;",
                 "const u32x2 lo = lds_load_tr8(p), hi = lds_load_tr8(p + 4 * kTrRowA);",
                 "const uint32_t p = buf + bo[j] + 32 * kTrRowB * ks;",
                 "const u32x2 lo = lds_load_tr8(p), hi = lds_load_tr8(p + 4 * kTrRowB);",
                 "a[ks][i] = u32x4{lo.x, lo.y, hi.x, hi.y};",
                 "if (st + 2 < nst) request(st + 2, cur == 0 ? 2 : cur - 1);",
                 "return pf_large_tile(N, M) && pf_inside(N, M, K, kDmaBN, kDmaBM) &&",
                 "const int ti = find_task(ga.first, ga.count);",
                 "const int64_t b = (int64_t)blockIdx.x - ga.first[ti], tn = N / kDmaBN;",
                 "const int64_t n0 = (b % tn) * kDmaBN, m0 = (b / tn) * kDmaBM;",
                 "constexpr int kTrGroupMax = 4;",
                 "ga.count = count - c0 < kTrGroupMax ? count - c0 : kTrGroupMax;",
                 "ga.first[i + 1] = ga.first[i] + (int32_t)((a[c0 + i].N / kDmaBN) * (a[c0 + i].M / kDmaBM));",
                 "hipLaunchKernelGGL(kernel, dim3((unsigned)ga.first[ga.count]), dim3(64 * NW), kDmaStages * "
                 "kDmaStageBytes, s, ga);"):
        assert line in src, f"contraction-major core changed: update this replay ({line})"
    train = open(TRAIN_SRC).read()
    for line in ("if (dense_prefill_tr_applies(N, K, M, dY, X)) {",
                 "const TrTask t{dY, X, N, K, M, &Wc, grad_values};",
                 "if (!dense_prefill_tr_applies(W.rows, W.cols, M, tasks[i].dY, tasks[i].X)) direct = false;",
                 "tr[n++] = TrTask{tasks[i].dY, tasks[i].X, W.rows, W.cols, M, &W, tasks[i].grad_values};"):
        assert line in train, f"weight gradient launch changed: update this replay ({line})"
    # (BN, BM, NW, FN, FM)
    return 128, 256, 8, 4, 4


def _tr_read(addrs, lane):
    """ds_read_b64_tr_b16 (CDNA4 LDS transpose load, 16-bit elements): in each
    16-lane quarter, lane t receives as element e the (t % 4)-th 16-bit
    element of the 8 bytes addressed by lane 4 e + t / 4 of its quarter.
    Returns the 4 byte addresses lane `lane` receives."""
    q, t = lane >> 4, lane & 15
    return [addrs[16 * q + 4 * e + (t >> 2)] + 2 * (t & 3) for e in range(4)]


@pytest.mark.parametrize("M,N,K", [(4096, 4096, 2048), (11008, 4096, 2048), (4096, 11008, 2048), (256, 128, 64),
                                   (1024, 8192, 192)])
def test_contraction_major_stage_and_transposed_reads(M, N, K):
    """The weight gradient's core (Y = Xc^T Wc from Xc [K][M] = dY and
    Wc [K][N] = X, the token as the row of both): one stage of a corner
    workgroup, replayed.  The direct-to-LDS requests fill every (contraction
    row, 16-byte chunk) of the stage exactly once, from inside the matrices,
    at the swizzled place (chunk c of row r at chunk c ^ 2 h(r),
    h(r) = r % 4 + 4 ((r / 8) % 2)); through the instruction's lane mapping,
    each lane's two transpose reads per fragment and k-step return exactly
    its MFMA operand (fragment row lane % 16, contraction rows
    8 (lane / 16) + 0..7); and each read is free of bank conflicts (64 banks
    of 4 bytes over half a wave, 32 over a quarter)."""
    BN, BM, NW, FN, FM = _tr_lines()
    bk, _ = _constants()
    rowA, rowB = 2 * BN, 2 * BM
    offB = bk * rowA
    RA, RB = bk * rowA // 1024 // NW, bk * rowB // 1024 // NW
    assert (RA, RB) == (2, 4) and offB + bk * rowB == (BN + BM) * 2 * bk
    assert M % BM == 0 and N % BN == 0 and K % bk == 0

    def h(r):
        return (r & 3) | (((r >> 3) & 1) << 2)

    for n0, m0 in ((0, 0), (N - BN, M - BM)):
        for st in sorted({0, K // bk - 1}):
            k0 = bk * st
            lds = {}                                   # byte -> (operand, contraction row, column)
            for wave in range(NW):
                hw = (wave & 1) << 2
                for lane in range(64):
                    for u in range(RA):
                        row = 8 * wave + (lane >> 4) + 4 * u          # stage row
                        col = n0 + 8 * ((lane & 15) ^ (2 * ((lane >> 4) | hw)))
                        slot = (RA * wave + u) * 1024 + 16 * lane
                        assert k0 + row < K and n0 <= col and col + 8 <= min(N, n0 + BN)
                        assert slot == row * rowA + 16 * (((col - n0) // 8) ^ (2 * h(row)))
                        for e in range(8):
                            assert slot + 2 * e not in lds
                            lds[slot + 2 * e] = ("W", k0 + row, col + e)
                    for u in range(RB):
                        p = u & 1
                        row = 8 * wave + 2 * p + (lane >> 5) + 4 * (u >> 1)
                        col = m0 + 8 * ((lane & 31) ^ (2 * ((2 * p + (lane >> 5)) | hw)))
                        slot = offB + (RB * wave + u) * 1024 + 16 * lane
                        assert k0 + row < K and m0 <= col and col + 8 <= min(M, m0 + BM)
                        assert slot == offB + row * rowB + 16 * (((col - m0) // 8) ^ (2 * h(row)))
                        for e in range(8):
                            assert slot + 2 * e not in lds
                            lds[slot + 2 * e] = ("X", k0 + row, col + e)
            assert len(lds) == (BN + BM) * bk
            for wave in range(NW):
                wn, wm = wave & 1, wave >> 1
                for op, frags, rowb, base, first, c0 in (("W", FN, rowA, 0, n0, 64 * wn),
                                                        ("X", FM, rowB, offB, m0, 64 * wm)):
                    for f in range(frags):
                        off = []
                        for lane in range(64):
                            t, r0 = lane & 15, 8 * (lane >> 4) + ((lane & 15) >> 2)
                            hh = (t >> 2) | (((lane >> 4) & 1) << 2)
                            assert hh == h(r0)
                            off.append(base + r0 * rowb + 16 * (((c0 // 8) + 2 * f + ((t & 3) >> 1)) ^ (2 * hh))
                                       + 8 * (t & 1))
                        for ks in range(2):
                            for half in range(2):
                                addrs = [o + 32 * rowb * ks + 4 * rowb * half for o in off]
                                for part, nb in ((32, 64), (16, 32)):
                                    for l0 in range(0, 64, part):
                                        banks = {(a // 4 + d) % nb for a in addrs[l0:l0 + part] for d in (0, 1)}
                                        assert len(banks) == 2 * part, (op, f, ks, half, part, l0)
                                for lane in range(64):
                                    got = [lds[b] for b in _tr_read(addrs, lane)]
                                    want = [(op, k0 + 32 * ks + 8 * (lane >> 4) + 4 * half + e,
                                             first + c0 + 16 * f + (lane & 15)) for e in range(4)]
                                    assert got == want, (op, wave, f, ks, half, lane)


# ---------------------------------------------------------------- the input gradient from W's packed tiles

def _input_grad_lines():
    src = open(SRC).read()
    for line in ("constexpr int NW = 8, BN = 128, BM = 256, FN = 4, FM = 4, TW = 2, RR = 8 * NW;",
                 "const int nst = (int)(N / kPfBK);",
                 "const int64_t s0 = k0 / 32 + 2 * (wave & 1);",
                 "const int rbw = wave >> 1;",
                 "const int er = 16 * rbw + fr;",
                 "const int eh = (er & 3) | (((er >> 3) & 1) << 2);",
                 "for (int i = 0; i < TW; ++i) eo[i] = (uint32_t)(er * kTrRowA + 16 * ((4 * (2 * (wave & 1) + i) + "
                 "fg) ^ (2 * eh)));",
                 "ao[i] = (uint32_t)(r0 * kTrRowA + 16 * ((8 * wn + 2 * i + ((t & 3) >> 1)) ^ (2 * h)) + 8 * (t & 1));",
                 "const int64_t tt = (int64_t)(4 * st + rbw) * S + s0 + i;",
                 "tw.w[i] = g.bm[tt * 16 + fr];",
                 "const uint32_t ex = wave_inclusive_scan(pc) - pc;",
                 "const uint32_t oa = (uint32_t)tw.off[i] + (i ? ex >> 16 : ex & 0xffffu);",
                 "__builtin_memcpy(&tv.v1[i], g.values + 2u * ob, 8);",
                 "*reinterpret_cast<__attribute__((address_space(3))) u32x4*>((uintptr_t)(buf + eo[i])) = a;",
                 "const uint32_t p = abuf + ao[i] + 32 * kTrRowA * ks;",
                 "const uint32_t b0 = bbuf + pf_chunk(wm * 16 * FM + fr, 4 * ks + fg);",
                 "if (st + 3 < nst) fetch_words(tw, st + 3);",
                 "pf_store<T, FN, FM>(acc, g.Y, M, K, k0, m0, wn, wm, fr, fg);",
                 "return M % 256 == 0 && W.rows % 64 == 0 && W.cols % 128 == 0 && pf_large_tile(W.cols, M);",
                 "hipLaunchKernelGGL(kernel, dim3((unsigned)(W.cols / 128), (unsigned)(M / 256)), dim3(512), lds, s, a);"):
        assert line in src, f"input-gradient kernel changed: update this replay ({line})"


@pytest.mark.parametrize("N,K,s", [(64, 128, 0.5), (128, 256, 0.7), (192, 384, 0.0), (64, 128, 1.0), (256, 512, 0.9)])
def test_input_grad_expansion_and_transposed_reads(orc, N, K, s):
    """dX = dY (W.Mask) from W's packed tiles: every workgroup column's
    stages, replayed.  Each stage's 16 tiles (four row blocks of W x the
    block's four k-steps) are expanded once, by wave w the pair (row block
    4 st + w / 2, k-steps 2 (w % 2) + {0, 1}), with windows inside the payload
    + 16 readable bytes; the expanded 8 columns of each lane equal the dense
    masked W and land once each in the contraction-major stage buffer (row
    of W r at 256 r, chunk c at c ^ 2 h(r)); and through the transpose read's
    lane mapping every lane of every A fragment receives W[64 st + 32 ks +
    8 (lane / 16) + 4 half + e][k0 + 64 wn + 16 i + lane % 16], its operand."""
    _input_grad_lines()
    bk, _ = _constants()
    BN, NW, FN = 128, 8, 4
    rowA = 2 * BN
    W, mask = synth.weight(83 + N + K, N, K, "bf16", s)
    T = orc.pack_tiled(W, "bf16", mask)
    vbytes = np.concatenate([T.values.view(np.uint8), np.zeros(16, np.uint8)])
    limit = 2 * T.nnz + 16
    dense = np.where(mask.astype(bool), W.view(np.uint16), 0).astype(np.uint16)
    S = K // 32
    bm = T.bitmask.reshape(-1).astype(np.uint64)
    offs = T.tile_offsets.astype(np.int64)
    assert N % bk == 0 and K % BN == 0
    for kb in range(K // BN):
        k0 = kb * BN
        for st in range(N // bk):
            lds = {}                                     # byte -> W element (row, col) it holds
            seen = set()
            for wave in range(NW):
                rbw, s0 = wave >> 1, k0 // 32 + 2 * (wave & 1)
                tiles = []
                for i in range(2):
                    t = (4 * st + rbw) * S + s0 + i
                    assert (4 * st + rbw, s0 + i) not in seen
                    seen.add((4 * st + rbw, s0 + i))
                    tiles.append((t, [int(bm[t * 16 + r]) for r in range(16)]))
                cnt = np.array([[_popc((tiles[i][1][l & 15] >> (8 * (l >> 4))) & 0xFF) for l in range(64)]
                                for i in range(2)])
                packed = cnt[0] | (cnt[1] << 16)
                ex = np.cumsum(packed) - packed
                for i in range(2):
                    t, words = tiles[i]
                    for lane in range(64):
                        fr, fg = lane & 15, lane >> 4
                        byte = (words[fr] >> (8 * fg)) & 0xFF
                        oa = int(offs[t]) + (int(ex[lane] >> 16) if i else int(ex[lane] & 0xFFFF))
                        ob = oa + _popc(byte & 0xF)
                        for o in (oa, ob):
                            assert 2 * o + 8 <= limit
                        v0 = vbytes[2 * oa:2 * oa + 8].view(np.uint32)
                        v1 = vbytes[2 * ob:2 * ob + 8].view(np.uint32)
                        lo, hi = byte & 0xF, byte >> 4
                        got = np.array([_perm(v0[1], v0[0], _nibble_selector(lo, 0)),
                                        _perm(v0[1], v0[0], _nibble_selector(lo, 1)),
                                        _perm(v1[1], v1[0], _nibble_selector(hi, 0)),
                                        _perm(v1[1], v1[0], _nibble_selector(hi, 1))], dtype=np.uint32).view(np.uint16)
                        n, kk = 16 * (4 * st + rbw) + fr, 32 * (s0 + i) + 8 * fg
                        assert np.array_equal(got, dense[n, kk:kk + 8]), (kb, st, wave, i, lane)
                        er = 16 * rbw + fr
                        eh = (er & 3) | (((er >> 3) & 1) << 2)
                        eo = er * rowA + 16 * ((4 * (2 * (wave & 1) + i) + fg) ^ (2 * eh))
                        assert 0 <= eo and eo + 16 <= bk * rowA
                        for e in range(8):
                            assert eo + 2 * e not in lds
                            lds[eo + 2 * e] = (n, kk + e)
            assert len(lds) == bk * BN
            for wave in range(NW):
                wn = wave & 1
                for i in range(FN):
                    off = []
                    for lane in range(64):
                        t, r0 = lane & 15, 8 * (lane >> 4) + ((lane & 15) >> 2)
                        h = (t >> 2) | (((lane >> 4) & 1) << 2)
                        off.append(r0 * rowA + 16 * ((8 * wn + 2 * i + ((t & 3) >> 1)) ^ (2 * h)) + 8 * (t & 1))
                    for ks in range(2):
                        for half in range(2):
                            addrs = [o + 32 * rowA * ks + 4 * rowA * half for o in off]
                            for lane in range(64):
                                got = [lds[b] for b in _tr_read(addrs, lane)]
                                want = [(bk * st + 32 * ks + 8 * (lane >> 4) + 4 * half + e,
                                         k0 + 64 * wn + 16 * i + (lane & 15)) for e in range(4)]
                                assert got == want, (kb, st, wave, i, ks, half, lane)


@pytest.mark.parametrize("shapes", [[(4096, 4096)] * 3, [(11008, 4096)] * 2, [(4096, 11008)], [(4096, 4096)] * 7,
                                    [(256, 128), (512, 256), (2048, 384)]])
def test_contraction_major_group_covers_every_block(shapes):
    """A grouped launch of the weight gradient's core (task i: M_i x N_i
    output in 256 x 128 blocks): launches of at most four tasks, workgroup x
    finds its task as the last i with first[i] <= x (find_task) and its block
    b = x - first[i] at n-block b % (N_i / 128), m-block b / (N_i / 128); every
    block of every task is computed exactly once."""
    _tr_lines()
    seen = set()
    for c0 in range(0, len(shapes), 4):
        grp = shapes[c0:c0 + 4]
        first = [0]
        for (M, N) in grp:
            first.append(first[-1] + (N // 128) * (M // 256))
        for x in range(first[-1]):
            ti = 0
            for i in range(1, len(grp)):
                ti = i if x >= first[i] else ti
            M, N = grp[ti]
            b, tn = x - first[ti], N // 128
            n0, m0 = (b % tn) * 128, (b // tn) * 256
            assert n0 + 128 <= N and m0 + 256 <= M
            key = (c0 + ti, n0, m0)
            assert key not in seen
            seen.add(key)
    assert len(seen) == sum((N // 128) * (M // 256) for (M, N) in shapes)
