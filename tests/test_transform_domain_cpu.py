"""The rotation of the transform-domain accumulator, pinned in exact integers.

The four-wave blind rotation at N = 4096 keeps its accumulator as
H = N^-1 NTT(ACC) and forms the rotated difference X^a ACC - ACC as the
inverse transform of (W^a - 1) H, where slot j of the transform holds the
evaluation at psi^(2 rev(j) + 1).  For the eight slots j = 8 t + k of a
thread t in the last pass it computes W_j^a as g 2^(120 m) with
g = psi^(c0 a), c0 = 2 rev(t) + 1 and m = (rev3(k) a) mod 8.  These tests
check that factorisation against the definition for every slot and many
rotations, the rotation identity itself on small rings, and a model of the
whole transform-domain loop against the oracle's blind rotation, with Python
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


# ------------------------------- the whole loop against the oracle ---------

def _td_blind_rotate(O, prm, lwe, bsk, acc0):
    """The blind rotation as the kernels at N >= 2048 run it, in exact
    integers on a small ring: H_c = N^-1 F(ACC_c) with F the transform's
    definition (slot j holds the evaluation at psi^(2 rev(j) + 1)); per step
    the rotated difference is the N-scaled inverse of (W^a - 1) H_u for both
    components, its digits are transformed and multiplied into H with the
    key rows scaled by N^-1; at the end ACC_c is the N-scaled inverse of H_c.
    Modulus switch and digits come from the oracle's own definitions."""
    N, n, l, beta = prm.N, prm.n, prm.pbs_level, prm.pbs_base_log
    bits = N.bit_length() - 1
    psi = psi_of(N)
    ninv = pow(N, P - 2, P)
    pts = [pow(psi, 2 * rev(j, bits) + 1, P) for j in range(N)]
    fwd = [[pow(x, i, P) for i in range(N)] for x in pts]
    inv = [[pow(x, (2 * N - i) % (2 * N), P) for x in pts] for i in range(N)]  # N-scaled inverse

    def F(a):
        return [sum(r[i] * a[i] for i in range(N)) % P for r in fwd]

    def Finv_N(X):
        return [sum(r[j] * X[j] for j in range(N)) % P for r in inv]

    key = np.asarray(bsk, dtype=np.uint64).reshape(n, 2, l, 2, N)
    K = [[[[[ninv * x % P for x in F([int(v) for v in key[i, u, t, c]])] for c in range(2)]
           for t in range(l)] for u in range(2)] for i in range(n)]
    H = [[ninv * x % P for x in F([int(v) for v in acc0[c * N:(c + 1) * N]])] for c in range(2)]
    for i in range(n):
        a = O.modswitch(int(lwe[i]), N)
        w = [(pow(x, a, P) - 1) % P for x in pts]
        D = [Finv_N([w[j] * H[u][j] % P for j in range(N)]) for u in range(2)]
        for u in range(2):
            digits = [O.decompose(d, l, beta) for d in D[u]]
            for t in range(l):
                Fd = F([digits[x][t] % P for x in range(N)])
                for c in range(2):
                    H[c] = [(H[c][j] + Fd[j] * K[i][u][t][c][j]) % P for j in range(N)]
    return np.array(Finv_N(H[0]) + Finv_N(H[1]), dtype=np.uint64)


@pytest.mark.parametrize("prm", [
    dict(n=4, N=16, pbs_level=2, pbs_base_log=8, ks_level=2, ks_base_log=4, msg_bits=2),
    dict(n=6, N=32, pbs_level=3, pbs_base_log=14, ks_level=3, ks_base_log=4, msg_bits=3),
])
def test_transform_domain_loop_equals_the_oracle(O, prm):
    """Trivial test polynomial (0, X^-b~ v) and a GLWE test polynomial
    rotated by X^-b~: the transform-domain loop gives the oracle's
    accumulator word for word, on noisy keys."""
    p = O.Params.make(**prm)
    ks = O.KeySet(p, 7 + prm["N"], 2.0 ** -20, 2.0 ** -40)
    rng = np.random.default_rng(prm["N"])
    for case in range(2):
        lwe = rng.integers(0, P, p.n + 1, dtype=np.uint64)
        btil = O.modswitch(int(lwe[p.n]), p.N)
        r = (2 * p.N - btil) % (2 * p.N)
        if case == 0:
            v = rng.integers(0, P, p.N, dtype=np.uint64)
            ref = O.blind_rotate(p, lwe, ks.bsk, v)
            acc0 = [0] * p.N + [int(x) for x in _rotate([int(y) for y in v], r)]
        else:
            tp = rng.integers(0, P, 2 * p.N, dtype=np.uint64)
            ref = O.blind_rotate_glwe(p, lwe, ks.bsk, tp)
            acc0 = (_rotate([int(y) for y in tp[:p.N]], r) +
                    _rotate([int(y) for y in tp[p.N:]], r))
        got = _td_blind_rotate(O, p, lwe, ks.bsk, acc0)
        assert np.array_equal(got, ref), case
