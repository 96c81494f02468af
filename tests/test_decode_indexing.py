"""Host-side replay of the decode kernel's wave-local LDS slot indexing.

The sparse decode kernel stages each wave's tiles in a zero-padded LDS region
and prefetches one group of k-steps ahead; this test replays the kernel's
loop (with the constants read from its source) for many shapes and checks
that every slot it reads lies inside the region.  Regression test for a
fault where the prefetch ran past a region padded by one group only."""
import os
import re

import pytest

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2405_03594_amd", "csrc", "k_decode.hip")


def _constants():
    src = open(SRC).read()
    waves = int(re.search(r"constexpr int kDecWaves = (\d+);", src).group(1))
    group = int(re.search(r"constexpr int kGroup = (\d+);", src).group(1))
    pad = re.search(r"const int Lp = \(S \+ kDecWaves - 1\) / kDecWaves \+ (\d+) \* kGroup;", src)
    assert pad, "padding formula changed: update this replay"
    return waves, group, int(pad.group(1)) * group


def _slots_read(L, G):
    reads = []

    def issue(j0):
        reads.extend(j0 + i for i in range(G))

    issue(0)
    j0 = 0
    while j0 < L:
        issue(j0 + G)
        if j0 + G >= L:
            break
        issue(j0 + 2 * G)
        j0 += 2 * G
    return reads


@pytest.mark.parametrize("K", [8, 16, 24, 32, 64, 96, 264, 1000, 2056, 4096, 11008, 16384, 49152])
def test_prefetch_stays_inside_the_wave_region(K):
    waves, G, pad = _constants()
    S = -(-K // 32)
    Lp = -(-S // waves) + pad
    for w in range(waves):
        L = S * (w + 1) // waves - S * w // waves
        if L > 0:
            assert max(_slots_read(L, G)) <= Lp - 1, (K, w, L, Lp)
