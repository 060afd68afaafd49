"""Pins of the oracle's field, ring, transform, rounding and decomposition
against closed forms, invariants and brute force (CPU only)."""
import random
from fractions import Fraction

import numpy as np
import pytest

P = 0xFFFFFFFF00000001
EDGE = [0, 1, 2, P - 1, P - 2, 2 ** 32, 2 ** 32 - 1, 2 ** 32 + 1, 2 ** 63, (P - 1) // 2,
        (P + 1) // 2, 2 ** 64 - 2 ** 32, 0xFFFFFFFF]


def rnd(rng, n):
    return [rng.randrange(P) for _ in range(n)]


# ---------------------------------------------------------------- field ---

def test_goldilocks_closed_forms(O):
    # 2^64 = 2^32 - 1 and 2^96 = -1 (mod p); hence 2 has order 192.
    assert O.mul(2 ** 32, 2 ** 32) == 2 ** 32 - 1
    assert O.mul(2 ** 48, 2 ** 48) == P - 1
    assert O.pow_(2, 96) == P - 1
    assert O.pow_(2, 192) == 1
    assert O.pow_(2, 64) == 2 ** 32 - 1


def test_field_against_integers(O):
    rng = random.Random(1)
    vals = EDGE + rnd(rng, 300)
    for a in vals:
        assert O.neg(a) == (-a) % P
        for b in vals[:20]:
            assert O.add(a, b) == (a + b) % P
            assert O.sub(a, b) == (a - b) % P
            assert O.mul(a, b) == (a * b) % P


def test_field_axioms(O):
    rng = random.Random(2)
    for _ in range(300):
        a, b, c = rnd(rng, 3)
        assert O.mul(a, O.add(b, c)) == O.add(O.mul(a, b), O.mul(a, c))
        assert O.mul(O.mul(a, b), c) == O.mul(a, O.mul(b, c))
        assert O.add(a, O.neg(a)) == 0
        assert O.sub(a, b) == O.add(a, O.neg(b))
        if a:
            assert O.mul(a, O.inv(a)) == 1
            assert O.pow_(a, P - 1) == 1  # Fermat


def test_seven_generates_and_roots(O):
    # p - 1 = 2^32 * 3 * 5 * 17 * 257 * 65537
    assert 2 ** 32 * 3 * 5 * 17 * 257 * 65537 == P - 1
    for q in (2, 3, 5, 17, 257, 65537):
        assert O.pow_(7, (P - 1) // q) != 1
    for logn in range(1, 13):
        N = 1 << logn
        psi = O.root_2n(N)
        assert O.pow_(psi, N) == P - 1          # psi^N = -1
        assert O.pow_(psi, 2 * N) == 1
    # every primitive 64th root of unity is a power of 8 = 2^3
    w64 = O.root_2n(32)
    assert O.pow_(w64, 32) == P - 1
    assert w64 in {pow(8, e, P) for e in range(1, 64, 2)}


def _rev(x, bits):
    return int(format(x, f"0{bits}b")[::-1], 2)


@pytest.mark.parametrize("logn", [8, 10, 11, 12])
def test_small_twiddles_are_powers_of_two(O, logn):
    # The transforms replace their first twiddles by shifts: zeta[m] =
    # psi^rev(m) equals 2^(156 rev3(m) mod 192) for m < 8 and 2^(39 rev5(m)
    # mod 192) for m < 32, at every N (7^((p-1)/16) = 2^156, 7^((p-1)/64) =
    # 2^39), with psi the oracle's primitive 2N-th root.
    psi = O.root_2n(1 << logn)
    for m in range(32):
        z = O.pow_(psi, _rev(m, logn))
        assert z == pow(2, (39 * _rev(m, 5)) % 192, P), m
        if m < 8:
            assert z == pow(2, (156 * _rev(m, 3)) % 192, P), m


# ----------------------------------------------------------------- ring ---

def horner(coeffs, z):
    acc = 0
    for c in reversed([int(x) for x in coeffs]):
        acc = (acc * z + c) % P
    return acc


def test_monomial_closed_forms(O):
    rng = np.random.default_rng(3)
    N = 16
    a = rng.integers(0, 2 ** 63, size=N, dtype=np.uint64)
    assert np.array_equal(O.monomial_mul(a, 0), a)
    neg = np.array([(-int(x)) % P for x in a], dtype=np.uint64)
    assert np.array_equal(O.monomial_mul(a, N), neg)
    for r in range(2 * N):
        for s in (1, 5, 2 * N - 1):
            lhs = O.monomial_mul(O.monomial_mul(a, r), s)
            assert np.array_equal(lhs, O.monomial_mul(a, (r + s) % (2 * N)))
    # X^1 * (a_0 + ... + a_{N-1} X^{N-1}): top coefficient wraps with a sign
    sh = O.monomial_mul(a, 1)
    assert int(sh[0]) == (-int(a[N - 1])) % P
    assert np.array_equal(sh[1:], a[:-1])


@pytest.mark.parametrize("kind", [0, 1])
def test_product_closed_forms(O, kind):
    N = 256
    x = np.zeros(N, dtype=np.uint64)
    x[1] = 1
    xn1 = np.zeros(N, dtype=np.uint64)
    xn1[N - 1] = 1
    prod = O.polymul(x, xn1, kind)
    expect = np.zeros(N, dtype=np.uint64)
    expect[0] = P - 1                       # X * X^(N-1) = X^N = -1
    assert np.array_equal(prod, expect)
    rng = np.random.default_rng(4)
    a = rng.integers(0, 2 ** 63, size=N, dtype=np.uint64)
    for r in (0, 1, 7, N - 1):
        mono = np.zeros(N, dtype=np.uint64)
        mono[r] = 5
        got = O.polymul(a, mono, kind)
        want = O.monomial_mul(a, r)
        want = np.array([(5 * int(w)) % P for w in want], dtype=np.uint64)
        assert np.array_equal(got, want)


@pytest.mark.parametrize("N", [8, 16])
def test_schoolbook_by_evaluation_at_every_root(O, N):
    """a*b mod (X^N+1) is the unique polynomial of degree < N with
    (a*b)(z) = a(z) b(z) at the N distinct roots z of X^N + 1."""
    rng = random.Random(N)
    psi = O.root_2n(N)
    roots = [pow(psi, 2 * k + 1, P) for k in range(N)]
    for z in roots:
        assert (pow(z, N, P) + 1) % P == 0
    assert len(set(roots)) == N
    for _ in range(5):
        a = np.array(rnd(rng, N), dtype=np.uint64)
        b = np.array(rnd(rng, N), dtype=np.uint64)
        c = O.polymul(a, b, 0)
        for z in roots:
            assert horner(c, z) == horner(a, z) * horner(b, z) % P


def test_schoolbook_evaluation_large(O):
    N = 256
    rng = random.Random(5)
    psi = O.root_2n(N)
    a = np.array(rnd(rng, N), dtype=np.uint64)
    b = np.array(rnd(rng, N), dtype=np.uint64)
    c = O.polymul(a, b, 0)
    for k in (0, 1, 77, 255):
        z = pow(psi, 2 * k + 1, P)
        assert horner(c, z) == horner(a, z) * horner(b, z) % P


@pytest.mark.parametrize("N", [4, 16, 256])
def test_ntt_definition(O, N):
    """Forward transform is evaluation at psi^(2k+1), natural order."""
    rng = random.Random(10 + N)
    a = np.array(rnd(rng, N), dtype=np.uint64)
    A = O.ntt_forward(a)
    psi = O.root_2n(N)
    ks = range(N) if N <= 16 else (0, 1, 2, 100, N - 1)
    for k in ks:
        assert int(A[k]) == horner(a, pow(psi, 2 * k + 1, P))
    assert np.array_equal(O.ntt_inverse(A), a)


@pytest.mark.parametrize("N", [2, 4, 256, 512, 2048])
def test_ntt_product_equals_schoolbook(O, N):
    rng = random.Random(20 + N)
    for _ in range(2 if N < 2048 else 1):
        a = np.array(rnd(rng, N), dtype=np.uint64)
        b = np.array(rnd(rng, N), dtype=np.uint64)
        assert np.array_equal(O.polymul(a, b, 0), O.polymul(a, b, 1))
    # small signed digits times a full-size key row (the shape used in PBS)
    d = np.array([(x % 257 - 128) % P for x in rnd(rng, N)], dtype=np.uint64)
    k = np.array(rnd(rng, N), dtype=np.uint64)
    assert np.array_equal(O.polymul(d, k, 0), O.polymul(d, k, 1))


# ------------------------------------------------------- modulus switch ---

def exact_round_modswitch(a, N):
    q = Fraction(2 * N * a, P)
    r = int(q + Fraction(1, 2))        # floor(q + 1/2); q is never a half-integer
    return r % (2 * N)


@pytest.mark.parametrize("N", [4, 256, 2048, 4096])
def test_modswitch_exact_rounding(O, N):
    rng = random.Random(N)
    vals = EDGE + rnd(rng, 500)
    # values on both sides of the rounding boundaries (2j+1) p / (4N)
    for j in list(range(0, 8)) + [2 * N - 1, N, N - 1]:
        c = (2 * j + 1) * P // (4 * N)
        vals += [c - 1, c, c + 1, c + 2]
    for a in vals:
        a %= P
        assert O.modswitch(a, N) == exact_round_modswitch(a, N)
        # never exactly half-way: 4N a is never an odd multiple of p
        assert (4 * N * a) % P != 0 or a == 0


# -------------------------------------------------------- decomposition ---

def centred(a):
    return a if a <= (P - 1) // 2 else a - P


PAIRS = [(2, 8), (2, 10), (3, 8), (3, 4), (5, 3), (6, 3), (2, 3), (3, 2), (1, 20)]


@pytest.mark.parametrize("levels,beta", PAIRS)
def test_decomposition_reconstruction(O, levels, beta):
    rng = random.Random(levels * 100 + beta)
    s = 64 - levels * beta
    B = 1 << beta
    vals = EDGE + rnd(rng, 400)
    # values around every multiple of 2^s near the extremes
    for r in (-(1 << (63 - s)), -3, -1, 0, 1, 3, (1 << (63 - s)) - 1):
        for off in (-(1 << (s - 1)) - 1, -(1 << (s - 1)), 0, (1 << (s - 1)) - 1, 1 << (s - 1)):
            vals.append((r * (1 << s) + off) % P)
    for a in vals:
        d = O.decompose(a, levels, beta)
        recon = sum(d[t] * (1 << (64 - (t + 1) * beta)) for t in range(levels))
        err = centred(a) - recon
        assert -(1 << (s - 1)) <= err < (1 << (s - 1)), (a, d)
        for t in range(1, levels):
            assert -B // 2 <= d[t] < B // 2
        assert -B // 2 <= d[0] <= B // 2


@pytest.mark.parametrize("levels,beta", [(2, 3), (3, 2), (2, 2)])
def test_decomposition_brute_force(O, levels, beta):
    """For every rounded value r reachable, the digits are the unique tuple
    with lower digits in [-B/2, B/2) that spells r in base B."""
    s = 64 - levels * beta
    B = 1 << beta
    import itertools
    spell = {}
    ranges = [range(-B // 2, B // 2 + 1)] + [range(-B // 2, B // 2)] * (levels - 1)
    for tup in itertools.product(*ranges):
        r = sum(tup[t] * B ** (levels - 1 - t) for t in range(levels))
        spell.setdefault(r, []).append(list(tup))
    rmax = 1 << (63 - s)
    rng = random.Random(7)
    for r in range(-rmax, rmax + 1):
        off = rng.randrange(-(1 << (s - 1)), 1 << (s - 1))
        a_c = r * (1 << s) + off
        if not (-(P - 1) // 2 <= a_c <= (P - 1) // 2):
            continue
        d = O.decompose(a_c % P, levels, beta)
        assert len(spell[r]) >= 1
        assert d in spell[r]
        # lower digits balanced in [-B/2, B/2): unique such spelling
        balanced = [t for t in spell[r] if all(-B // 2 <= x < B // 2 for x in t[1:])]
        assert balanced == [d]


# ------------------------------------------------------------ randomness ---

def test_splitmix64_published_vector(O):
    """SplitMix64 seeded with 0: the first outputs of the published
    generator (the same vector seeds the xoshiro family's reference code)."""
    assert O.splitmix_word(0, 0) == 0xE220A8397B1DCDAF
    assert O.splitmix_word(0, 1) == 0x6E789E6AA1B965F4
    assert O.splitmix_word(0, 2) == 0x06C45D188009454F


def test_box_muller_is_standard_normal(O):
    key = O.splitmix_word(123, 4)
    z = np.array([O.gauss(key, i) for i in range(100000)])
    assert abs(z.mean()) < 0.015
    assert abs(z.var() - 1.0) < 0.02
    assert abs(np.mean(np.abs(z) < 1.0) - 0.6827) < 0.01
    assert abs(np.mean(np.abs(z) < 2.0) - 0.9545) < 0.005
