"""The rotation of the transform-domain accumulator, pinned in exact integers.

The four-wave blind rotation at N = 4096 keeps its accumulator as
H = N^-1 NTT(ACC) and forms the rotated difference X^a ACC - ACC as the
inverse transform of (W^a - 1) H, where slot j of the transform holds the
evaluation at psi^(2 rev(j) + 1).  For the eight slots j = 8 t + k of a
thread t in the last pass it computes W_j^a as g 2^(120 m) with
g = psi^(c0 a), c0 = 2 rev(t) + 1 and m = (rev3(k) a) mod 8.  These tests
check that factorisation against the definition for every slot and many
rotations, and the rotation identity itself on small rings, with Python
integers only (no kernel code)."""
import numpy as np
import pytest

P = 2**64 - 2**32 + 1


def rev(x, bits):
    return int(format(x, f"0{bits}b")[::-1], 2) if bits else 0


def psi_of(N):
    return pow(7, (P - 1) // (2 * N), P)


def test_the_eighth_root_is_a_shift():
    """psi^(N/4) = 7^((p-1)/8) = 2^120 for every N (the shared 8th root)."""
    assert pow(7, (P - 1) // 8, P) == pow(2, 120, P)
    for N in (256, 2048, 4096):
        assert pow(psi_of(N), N // 4, P) == pow(2, 120, P)


@pytest.mark.parametrize("logn", [11, 12])
def test_slot_factor_matches_its_definition(logn):
    N = 1 << logn
    T = N // 8
    psi = psi_of(N)
    rng = np.random.default_rng(logn)
    rots = [0, 1, 2, 7, 8, N - 1, N, N + 1, 2 * N - 1] + [int(a) for a in rng.integers(0, 2 * N, 24)]
    for t in range(T):
        c0 = 2 * rev(t, logn - 3) + 1
        for a in rots:
            g = pow(psi, (c0 * a) % (2 * N), P)
            for k in range(8):
                j = 8 * t + k
                want = pow(psi, (2 * rev(j, logn) + 1) * a, P)
                m = (rev(k, 3) * a) % 8
                assert g * pow(2, 120 * m, P) % P == want, (t, k, a)


def _ntt(a, psi):
    """The transform's definition: slot j is a(psi^(2 rev(j) + 1))."""
    N = len(a)
    bits = N.bit_length() - 1
    return [sum(int(a[i]) * pow(psi, (2 * rev(j, bits) + 1) * i, P) for i in range(N)) % P
            for j in range(N)]


def _rotate(a, r):
    """X^r a in Z_p[X]/(X^N + 1), 0 <= r < 2N."""
    N = len(a)
    out = [0] * N
    for i, v in enumerate(a):
        e = i + r
        s = -1 if (e // N) % 2 else 1
        out[e % N] = (s * int(v)) % P
    return out


@pytest.mark.parametrize("N", [16, 32])
def test_rotated_difference_in_the_transform_domain(N):
    """NTT(X^a A - A) = (W^a - 1) NTT(A) slot by slot, for every a."""
    psi = psi_of(N)
    bits = N.bit_length() - 1
    rng = np.random.default_rng(N)
    A = [int(x) for x in rng.integers(0, P, N, dtype=np.uint64)]
    FA = _ntt(A, psi)
    for a in range(2 * N):
        D = [(x - y) % P for x, y in zip(_rotate(A, a), A)]
        FD = _ntt(D, psi)
        for j in range(N):
            w = pow(psi, (2 * rev(j, bits) + 1) * a, P)
            assert FD[j] == (w - 1) * FA[j] % P, (a, j)
