"""GPU: the device field routines every kernel is built from, against exact
integer arithmetic mod p = 2^64 - 2^32 + 1 (Python integers), on edge values
(0, 1, p - 1, the limb boundaries 2^32 - 1, 2^32, 2^63 and their
neighbours, values whose shifted limbs vanish) crossed with each other, and on
seeded random values.  Bit-exact."""
import itertools

import numpy as np
import pytest

from gpu_helpers import require_gpu, say
from paper_2609_16915_amd import rosetta as R

pytestmark = pytest.mark.gpu
P = 0xFFFFFFFF00000001


def edge_values():
    v = {0, 1, 2, 3, P - 1, P - 2, P - 3, (P - 1) // 2, (P + 1) // 2}
    for b in (16, 31, 32, 33, 48, 63):
        for d in (-2, -1, 0, 1, 2):
            x = (1 << b) + d
            if 0 <= x < P:
                v.add(x)
    for x in (0xFFFFFFFF, 0xFFFFFFFF00000000, 0xFFFFFFFEFFFFFFFF, 0xFFFFFFFF00000000 - 1,
              0x8000000000000000, 0x8000000080000000, 0x00000000FFFF0000, 0xFFFF0000FFFF0000,
              0x0000FFFF0000FFFF, 0x7FFFFFFF80000000):
        if x < P:
            v.add(x)
    # x with x * 2^e landing on the 2^96 or 2^128 limb only, for the shifts
    for e in (12, 24, 36, 48, 60, 72, 84):
        for s in (96 - e, 128 - e, 64 - e):
            if 0 <= s < 64:
                v.add(1 << s)
                v.add(((1 << s) * 3) % P)
    return sorted(v)


def pairs():
    ev = edge_values()
    rng = np.random.default_rng(7)
    rnd = [int(x) for x in rng.integers(0, P, size=4000, dtype=np.uint64)]
    a = [x for x, _ in itertools.product(ev, ev)] + rnd
    b = [y for _, y in itertools.product(ev, ev)] + rnd[::-1]
    c = [int(x) for x in rng.integers(0, P, size=len(a), dtype=np.uint64)]
    c[: len(ev)] = ev
    c[len(ev): 2 * len(ev)] = [P - 1] * len(ev)
    return a, b, c


@pytest.fixture(scope="module")
def operands():
    require_gpu()
    a, b, c = pairs()
    to = lambda xs: R.to_device(np.array(xs, dtype=np.uint64))
    return a, b, c, to(a), to(b), to(c)


@pytest.mark.parametrize("op,name,ref", [
    (R.FIELD_ADD, "add", lambda a, b, c: (a + b) % P),
    (R.FIELD_SUB, "sub", lambda a, b, c: (a - b) % P),
    (R.FIELD_MUL, "mul", lambda a, b, c: a * b % P),
    (R.FIELD_MUL_ADD, "mul_add", lambda a, b, c: (a * b + c) % P),
])
def test_field_binary_ops_exact(operands, op, name, ref):
    a, b, c, da, db, dc = operands
    say(f"[field] {name} on {len(a)} operand pairs")
    got = R.to_host(R.field_op(op, da, db, dc))
    want = np.array([ref(x, y, z) for x, y, z in zip(a, b, c)], dtype=np.uint64)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(hex(a[i]), hex(b[i]), hex(int(got[i])), hex(int(want[i])))
                           for i in bad[:5]]


def test_field_add_weak_contract(operands):
    # first operand anywhere below 2^64 (the values at and above p included),
    # second canonical: the result must be congruent to a + b mod p
    _, b, _, _, _, _ = operands
    high = [P, P + 1, P + 2, (1 << 64) - 1, (1 << 64) - 2, (1 << 64) - (1 << 32),
            P + (1 << 31), (1 << 64) - 3]
    rng = np.random.default_rng(11)
    a = [high[i % len(high)] if i % 3 == 0 else int(x)
         for i, x in enumerate(rng.integers(0, 1 << 64, size=len(b), dtype=np.uint64))]
    bb = list(b)
    bb[: len(high)] = [P - 1] * len(high)
    say(f"[field] add_weak on {len(a)} pairs")
    got = R.to_host(R.field_op(R.FIELD_ADD_WEAK, R.to_device(np.array(a, dtype=np.uint64)),
                               R.to_device(np.array(bb, dtype=np.uint64))))
    bad = [i for i in range(len(a)) if int(got[i]) % P != (a[i] + bb[i]) % P]
    assert not bad, [(hex(a[i]), hex(bb[i]), hex(int(got[i]))) for i in bad[:5]]


def test_field_mul_add_weak_contract(operands):
    # first factor and addend anywhere below 2^64, second factor canonical:
    # the result must be congruent to a * b + c mod p
    _, b, _, _, _, _ = operands
    high = [P, P + 1, (1 << 64) - 1, (1 << 64) - (1 << 32), P + (1 << 31)]
    rng = np.random.default_rng(13)
    n = len(b)
    a = [high[i % len(high)] if i % 4 == 0 else int(x)
         for i, x in enumerate(rng.integers(0, 1 << 64, size=n, dtype=np.uint64))]
    c = [high[i % len(high)] if i % 3 == 0 else int(x)
         for i, x in enumerate(rng.integers(0, 1 << 64, size=n, dtype=np.uint64))]
    bb = list(b)
    bb[: len(high)] = [P - 1] * len(high)
    say(f"[field] mul_add_weak on {n} triples")
    to = lambda xs: R.to_device(np.array(xs, dtype=np.uint64))
    got = R.to_host(R.field_op(R.FIELD_MUL_ADD_WEAK, to(a), to(bb), to(c)))
    bad = [i for i in range(n) if int(got[i]) % P != (a[i] * bb[i] + c[i]) % P]
    assert not bad, [(hex(a[i]), hex(bb[i]), hex(c[i]), hex(int(got[i]))) for i in bad[:5]]


def test_field_pow2_every_exponent(operands):
    a, _, _, da, _, _ = operands
    say(f"[field] mul_pow2 e = 0..95 on {len(a)} values")
    for e in range(96):
        got = R.to_host(R.field_op(R.FIELD_MUL_POW2 + e, da))
        t = pow(2, e, P)
        want = np.array([x * t % P for x in a], dtype=np.uint64)
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, (e, [(hex(a[i]), hex(int(got[i])), hex(int(want[i])))
                                   for i in bad[:5]])


def test_field_round_top_every_shift(operands):
    # the rounding that opens the gadget decomposition, in both device forms
    # (64-bit below s = 34, high word from s = 34 up), on the edge values,
    # p itself (the minuend form of -0 in the blind rotation), values just
    # around the centring boundary and whole multiples of 2^32 above it
    a, _, _, _, _, _ = operands
    h = (P - 1) // 2
    extra = [P, h - 1, h, h + 1, h + 2, P - (1 << 32), P - (1 << 32) - 1,
             0xFFFFFFFE00000000, 0x8000000100000000, 0x8000000000000001,
             0x7FFFFFFF80000000, 0x7FFFFFFFFFFFFFFF, 0x7FFFFFFF00000000]
    vals = list(a) + extra
    dv = R.to_device(np.array(vals, dtype=np.uint64))
    say(f"[field] round_top s = 1..63 on {len(vals)} values")
    for s in range(1, 64):
        got = R.to_host(R.field_op(R.FIELD_ROUND_TOP + s, dv)).view(np.int64)
        want = np.array([((x - P if x > h else x) + (1 << (s - 1))) >> s for x in vals],
                        dtype=np.int64)
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, (s, [(hex(vals[i]), int(got[i]), int(want[i]))
                                   for i in bad[:5]])


def test_field_ops_in_place(operands):
    a, b, _, _, _, _ = operands
    x = R.to_device(np.array(a, dtype=np.uint64))
    y = R.to_device(np.array(b, dtype=np.uint64))
    R.field_op(R.FIELD_MUL, x, y, out=x)
    want = np.array([u * v % P for u, v in zip(a, b)], dtype=np.uint64)
    assert np.array_equal(R.to_host(x), want)


def test_modmul_chain_probe_computes_the_powers():
    require_gpu()
    seed, threads, iters = 12345, 300, 37
    got = R.to_host(R.modmul_chain(seed, threads, iters))
    for t in (0, 1, 255, 256, 299):
        w = (seed ^ ((t * 0x9E3779B97F4A7C15) % 2 ** 64)) % P
        w = 3 if w < 2 else w
        want = 0
        for j in range(8):
            want ^= (seed + 8 * t + j + 1) % P * pow(w, iters, P) % P
        assert int(got[t]) == want, t
