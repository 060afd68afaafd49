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


# ------------------------------------------------- barrier placement model ---

def _wave_block(L, q):
    return L.T <= 64 or L.lo(q) <= 6


def _sequence(logn, kernel, levels=3, spread_barrier=True):
    """The LDS accesses of one CMux step of the blind rotation (or one round of
    the trace) and of the start of the next, as the kernel issues them, split
    into segments by workgroup barriers: a list of {wave: (reads, writes)}.
    Cross-wave exchanges take a barrier before the writes and one before the
    reads; exchanges inside each wave take none, except the first one after
    a read that may leave a wave's block when the two share a buffer (the
    rule the kernel's LDS buffer object applies)."""
    L = Layout(logn)
    N, T = 1 << logn, L.T
    shared = logn >= 12
    local_base = 0 if shared else N
    waves = range((T + 63) // 64)
    segs = [{}]
    state = {"spread": False}

    def barrier():
        segs.append({})

    def access(w, reads=(), writes=()):
        r, wr = segs[-1].setdefault(w, (set(), set()))
        r.update(reads)
        wr.update(writes)

    def own(q, w, base):
        return {base + swz(L.idx(q, t, k)) for t in range(64 * w, min(64 * w + 64, T))
                for k in range(L.E)}

    def natural(w):
        return {t + T * k for t in range(64 * w, min(64 * w + 64, T)) for k in range(L.E)}

    def cross_gather():
        # write the natural layout, barrier, then read anywhere (rotation or
        # automorphism: the source index depends on the data)
        state["spread"] = True
        barrier()
        for w in waves:
            access(w, writes=natural(w))
        barrier()
        for w in waves:
            access(w, reads=set(range(N)))

    def exchange(qa, qb):
        if _wave_block(L, qa) and _wave_block(L, qb):
            if shared and state["spread"] and spread_barrier:
                barrier()
                state["spread"] = False
            for w in waves:
                access(w, writes=own(qa, w, local_base), reads=own(qb, w, local_base))
        else:
            state["spread"] = True
            barrier()
            for w in waves:
                access(w, writes=own(qa, w, 0))
            barrier()
            for w in waves:
                access(w, reads=own(qb, w, 0))
            if _wave_block(L, qb):
                state["spread"] = False

    def forward():
        for q in range(L.passes - 1):
            exchange(q, q + 1)

    def inverse():
        for q in range(L.passes - 1, 0, -1):
            exchange(q, q - 1)

    if kernel == "blind_rotate_td":
        # accumulator in the transform domain: two forward transforms first,
        # then per step the two inverse transforms of the rotated
        # differences before the digit transforms (no rotation exchange),
        # and two inverse transforms at the end
        forward()
        forward()
        for step in range(2):
            inverse()
            inverse()
            for _u in range(2):
                for _t in range(levels):
                    forward()
        inverse()
        inverse()
        return segs
    for step in range(2):
        if kernel == "blind_rotate":
            for _u in range(2):
                cross_gather()
                for _t in range(levels):
                    forward()
        else:
            cross_gather()
            cross_gather()
            for _t in range(levels):
                forward()
        inverse()
        inverse()
    return segs


def _hazards(segs):
    found = []
    for i, seg in enumerate(segs):
        for a, (ra, wa) in seg.items():
            for b, (rb, wb) in seg.items():
                if a != b and wa & (rb | wb):
                    found.append((i, a, b))
    return found


@pytest.mark.parametrize("logn", [8, 11, 12])
@pytest.mark.parametrize("kernel", ["blind_rotate", "blind_rotate_td", "trace"])
def test_no_two_waves_touch_a_word_without_a_barrier(logn, kernel):
    """Every pair of accesses by two waves to one LDS word, one of them a
    write, is separated by a workgroup barrier (the tiny ring is one wave)."""
    assert _hazards(_sequence(logn, kernel)) == []


@pytest.mark.parametrize("kernel", ["blind_rotate", "blind_rotate_td", "trace"])
def test_the_model_sees_the_race_the_spread_barrier_removes(kernel):
    """Without the barrier that follows a read outside the waves' blocks,
    the shared buffer of N = 4096 has hazards (the second inverse transform
    of a step writing while the first one's last exchange is still read;
    in the transform-domain loop the same pair opens every step)."""
    assert _hazards(_sequence(12, kernel, spread_barrier=False))
