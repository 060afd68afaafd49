"""The LDS exchange layouts of the transforms (csrc/ntt.hpp), checked on the CPU:
for every supported ring (the shape ntt_le / ntt_first of csrc/internal.hpp pick)
and every pass layout, the word addresses that the 32 lanes of a half wave (and
the 16 of a quarter wave) write or read for one element fall in distinct banks of
8-byte words; the swizzle is a bijection of each wave's block (it flips only
address bits below 5), which the shared exchange buffer of N = 4096 relies on;
and every index of the transform is held by exactly one (thread, element) in
every pass.  The masks are read from the header, the layout formula restated."""
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = open(os.path.join(ROOT, "paper_2609_16915_amd", "csrc", "ntt.hpp")).read()
MASK = [int(x, 16) for x in re.search(r"SWZ_MASK\[5\] = \{([^}]*)\}", HDR).group(1).split(",")]


def shape(logn):
    """(LE, F) as in csrc/internal.hpp."""
    le = 2 if logn == 8 else 3
    return le, (2 if logn == 11 else le)


def swz(j):
    a = j
    for b, m in enumerate(MASK):
        a ^= (bin(j & m).count("1") & 1) << b
    return a


class Layout:
    def __init__(self, logn):
        self.logn = logn
        self.le, self.f = shape(logn)
        self.E = 1 << self.le
        self.T = (1 << logn) // self.E
        self.passes = 1 + (logn - self.f + self.le - 1) // self.le

    def stage_end(self, q):
        e = self.f + q * self.le
        return e if e < self.logn else self.logn

    def lo(self, q):
        if q == 0:
            return self.logn - self.le
        return max(0, self.logn - self.stage_end(q))

    def idx(self, q, tid, k):
        lo = self.lo(q)
        return (tid & ((1 << lo) - 1)) + (k << lo) + ((tid >> lo) << (lo + self.le))


@pytest.mark.parametrize("logn", [8, 9, 10, 11, 12])
def test_every_pass_layout_is_conflict_free_and_complete(logn):
    L = Layout(logn)
    N = 1 << logn
    for q in range(L.passes):
        held = sorted(L.idx(q, t, k) for t in range(L.T) for k in range(L.E))
        assert held == list(range(N)), (logn, q)
        for k in range(L.E):
            for width in (32, 16):
                for base in range(0, min(L.T, 64 * ((L.T + 63) // 64)), width):
                    lanes = range(base, min(base + width, L.T))
                    banks = {swz(L.idx(q, t, k)) % 32 for t in lanes}
                    assert len(banks) == len(lanes), (logn, q, k, width, base)


@pytest.mark.parametrize("logn", [8, 9, 10, 11, 12])
def test_swizzle_keeps_every_32_word_block(logn):
    N = 1 << logn
    image = [swz(j) for j in range(N)]
    assert sorted(image) == list(range(N))
    assert all(a >> 5 == j >> 5 for j, a in enumerate(image))


def test_addresses_are_linear_in_the_element():
    """The exchange computes the address of element k as the thread's base XOR
    swz(k << lo): the element's bits are disjoint from the thread's."""
    for logn in (8, 11, 12):
        L = Layout(logn)
        for q in range(L.passes):
            lo = L.lo(q)
            for t in range(0, L.T, max(1, L.T // 64)):
                for k in range(L.E):
                    assert swz(L.idx(q, t, k)) == swz(L.idx(q, t, 0)) ^ swz(k << lo)
