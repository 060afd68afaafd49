"""Pins of the oracle's lookup-protocol primitives (CPU only): Galois
automorphisms, GLWE key switching, the RLWE trace (Sec. 2.2.3), blind
rotation of a ciphertext test polynomial, plaintext-ciphertext products and
recombination (Sec. 3.2), each against closed forms, exact identities,
deterministic noise bounds, and the paper's running example end to end."""
import json
import math
import os

import numpy as np
import pytest

from oracle import seglut as G

P = 0xFFFFFFFF00000001
HERE = os.path.dirname(os.path.abspath(__file__))
EX = json.load(open(os.path.join(HERE, "golden", "paper_lookup_example.json")))
TR_L, TR_B = 4, 12                     # trace decomposition used by these pins


def centred(x):
    x = int(x) % P
    return x if x <= (P - 1) // 2 else x - P


def horner(a, z):
    acc = 0
    for c in reversed([int(v) for v in a]):
        acc = (acc * z + c) % P
    return acc


def roots(N):
    """All roots of X^N + 1 in Z_p: psi^(2k+1), psi a primitive 2N-th root."""
    psi = pow(7, (P - 1) // (2 * N), P)
    assert pow(psi, N, P) == P - 1
    return [pow(psi, 2 * k + 1, P) for k in range(N)]


def rand_poly(rng, N):
    return rng.integers(0, P, N, dtype=np.uint64)


def small_params(O, n=8, N=32, sigma=0.0, seed=3, l=2, beta=10):
    prm = O.Params.make(n=n, N=N, pbs_level=l, pbs_base_log=beta, ks_level=3, ks_base_log=4,
                        msg_bits=2)
    return prm, O.KeySet(prm, seed, sigma, sigma)


# ------------------------------------------------------------ automorphisms ---

def test_automorphism_is_evaluation_at_powers(O):
    """(tau_d a)(z) = a(z^d) at every root z of X^N + 1 (big-integer Horner)."""
    rng = np.random.default_rng(1)
    for N in (8, 16):
        a = rand_poly(rng, N)
        for d in range(1, 2 * N, 2):
            t = O.automorphism(a, d)
            for z in roots(N):
                assert horner(t, z) == horner(a, pow(z, d, P))


def test_automorphism_group_and_ring_map(O):
    rng = np.random.default_rng(2)
    N = 16
    a, b = rand_poly(rng, N), rand_poly(rng, N)
    assert np.array_equal(O.automorphism(a, 1), a)
    assert np.array_equal(O.automorphism(a, 2 * N + 1), a)
    for d in (3, 5, 17, 31):
        for e in (3, 9, 2 * N - 1):
            lhs = O.automorphism(O.automorphism(a, e), d)
            assert np.array_equal(lhs, O.automorphism(a, (d * e) % (2 * N)))
        ab = O.polymul(a, b, O.SCHOOLBOOK)
        assert np.array_equal(O.automorphism(ab, d),
                              O.polymul(O.automorphism(a, d), O.automorphism(b, d)))


def test_sum_over_galois_group_is_n_times_constant(O):
    """Sum of tau_d(a) over all odd d < 2N equals N a_0 (constant term)."""
    rng = np.random.default_rng(3)
    for N in (4, 8, 16):
        a = rand_poly(rng, N)
        tot = [0] * N
        for d in range(1, 2 * N, 2):
            tot = [(x + int(y)) % P for x, y in zip(tot, O.automorphism(a, d))]
        assert tot[0] == N * int(a[0]) % P and all(x == 0 for x in tot[1:])


# ------------------------------------------------------ keys, key switching ---

def test_autk_rows_have_the_stated_phase(O):
    """Noise-free automorphism keys: phase(autk[k-1][t]) = tau_(2^k+1)(S) g_t."""
    N = 32
    prm, ks = small_params(O, N=N)
    S = ks.glwe_key
    autk = O.autk_keygen(11, N, TR_L, TR_B, 0.0, S)
    rows = autk.reshape(int(math.log2(N)), TR_L, 2 * N)
    for k in range(1, int(math.log2(N)) + 1):
        tS = O.automorphism(S, 2 ** k + 1)
        for t in range(TR_L):
            g = pow(2, 64 - (t + 1) * TR_B, P)
            ph = O.glwe_phase(S, rows[k - 1, t], O.SCHOOLBOOK)
            assert [int(x) for x in ph] == [int(x) * g % P for x in tS]


def test_glwe_keyswitch(O):
    """Switching tau_d(c) from tau_d(S) back to S keeps the phase within
    N 2^(s-1) with a noise-free key; a mask-free input comes out unchanged."""
    N = 64
    prm, ks = small_params(O, N=N)
    S = ks.glwe_key
    autk = O.autk_keygen(12, N, TR_L, TR_B, 0.0, S).reshape(int(math.log2(N)), TR_L * 2 * N)
    s = 64 - TR_L * TR_B
    rng = np.random.default_rng(4)
    for k in (1, 3, int(math.log2(N))):
        d = 2 ** k + 1
        tS = O.automorphism(S, d)
        for _ in range(3):
            c = rand_poly(rng, 2 * N)
            ph_in = O.glwe_phase(tS, c, O.SCHOOLBOOK)
            for kind in (O.SCHOOLBOOK, O.NTT):
                out = O.glwe_keyswitch(N, TR_L, TR_B, c, autk[k - 1], kind)
                ph = O.glwe_phase(S, out, O.SCHOOLBOOK)
                err = max(abs(centred(int(x) - int(y))) for x, y in zip(ph, ph_in))
                assert err <= N * 2 ** (s - 1)
        triv = np.concatenate([np.zeros(N, np.uint64), rand_poly(rng, N)])
        out = O.glwe_keyswitch(N, TR_L, TR_B, triv, autk[k - 1])
        assert np.array_equal(out, triv)


# -------------------------------------------------------------------- trace ---

def test_trace_of_trivial_ciphertext_is_exact(O):
    """Trace((0, m)) = (0, m_0): the digits of a zero mask are zero, so only
    the automorphisms and N^-1 act, and their sum is exact."""
    rng = np.random.default_rng(5)
    for N in (4, 32):
        S = np.asarray(rng.integers(0, 2, N), dtype=np.uint64)
        autk = O.autk_keygen(13, N, TR_L, TR_B, 2.0 ** -40, S)
        m = rand_poly(rng, N)
        c = np.concatenate([np.zeros(N, np.uint64), m])
        for kind in (O.SCHOOLBOOK, O.NTT):
            out = O.trace(N, TR_L, TR_B, c, autk, kind)
            assert np.all(out[:N] == 0)
            assert int(out[N]) == int(m[0]) and np.all(out[N + 1:] == 0)


def test_trace_phase_noise_free_bound(O):
    """Noise-free keys: phase(Trace(c)) = (phase(c)_0, 0, .., 0) + E with
    |E_j| <= (N - 1) N 2^(s-1): each of the log2 N rounds adds a key-switch
    rounding error of at most N 2^(s-1) per coefficient, and every later
    round at most doubles what is there."""
    rng = np.random.default_rng(6)
    s = 64 - TR_L * TR_B
    for N in (16, 64):
        S = np.asarray(rng.integers(0, 2, N), dtype=np.uint64)
        autk = O.autk_keygen(14, N, TR_L, TR_B, 0.0, S)
        bound = (N - 1) * N * 2 ** (s - 1)
        for _ in range(2):
            c = rand_poly(rng, 2 * N)
            ph = O.glwe_phase(S, c, O.SCHOOLBOOK)
            out = O.trace(N, TR_L, TR_B, c, autk, O.SCHOOLBOOK)
            assert np.array_equal(out, O.trace(N, TR_L, TR_B, c, autk, O.NTT))
            ph_out = O.glwe_phase(S, out, O.SCHOOLBOOK)
            want = [int(ph[0])] + [0] * (N - 1)
            err = max(abs(centred(int(x) - y)) for x, y in zip(ph_out, want))
            assert err <= bound < 2 ** 40


def test_trace_with_noise_keeps_constant(O):
    """With Gaussian keys (sigma = 2^-51, the GLWE noise of the workloads)
    the trace error stays far below a 2^-20 fraction of p."""
    rng = np.random.default_rng(7)
    N = 256
    S = np.asarray(rng.integers(0, 2, N), dtype=np.uint64)
    autk = O.autk_keygen(15, N, TR_L, TR_B, 2.0 ** -51, S)
    m = rand_poly(rng, N)
    c = O.glwe_encrypt(16, 2.0 ** -51, S, m)[0]
    ph = O.glwe_phase(S, c)
    out = O.trace(N, TR_L, TR_B, c, autk, O.NTT)
    ph_out = O.glwe_phase(S, out)
    err = max(abs(centred(int(x) - y)) for x, y in zip(ph_out, [int(ph[0])] + [0] * (N - 1)))
    assert err < 2 ** 44


# ----------------------------------------------- blind rotation of a ciphertext ---

def test_blind_rotate_glwe_trivial_selector(O):
    """A trivial LWE selector (a = 0) leaves ACC = X^(-b~) TP exactly."""
    prm, ks = small_params(O)
    N = prm.N
    rng = np.random.default_rng(8)
    tp = rand_poly(rng, 2 * N)
    for b in (0, 1, P // 3, P - 1):
        lwe = np.zeros(prm.n + 1, np.uint64)
        lwe[prm.n] = b
        r = (2 * N - O.modswitch(b, N)) % (2 * N)
        for kind in (O.SCHOOLBOOK, O.NTT):
            acc = O.blind_rotate_glwe(prm, lwe, ks.bsk, tp, kind)
            assert np.array_equal(acc[:N], O.monomial_mul(tp[:N], r))
            assert np.array_equal(acc[N:], O.monomial_mul(tp[N:], r))


def test_blind_rotate_glwe_reduces_to_pbs_rotation(O):
    """A trivial test-polynomial ciphertext (0, v) gives the PBS accumulator."""
    prm, ks = small_params(O, sigma=2.0 ** -40)
    rng = np.random.default_rng(9)
    v = rand_poly(rng, prm.N)
    tp = np.concatenate([np.zeros(prm.N, np.uint64), v])
    lwe = rand_poly(rng, prm.n + 1)
    assert np.array_equal(O.blind_rotate_glwe(prm, lwe, ks.bsk, tp, O.SCHOOLBOOK),
                          O.blind_rotate(prm, lwe, ks.bsk, v, O.SCHOOLBOOK))


def test_blind_rotate_glwe_phase(O):
    """Noise-free bootstrapping key: phase(ACC) = X^(-rot) phase(TP) + err,
    rot = b~ - sum a~_i s_i mod 2N, |err| <= n (1 + N) 2^(s-1) (one external
    product bound per CMux step)."""
    prm, ks = small_params(O, n=8, N=32)
    N, n = prm.N, prm.n
    s = 64 - prm.pbs_level * prm.pbs_base_log
    rng = np.random.default_rng(10)
    for _ in range(3):
        m = rand_poly(rng, N)
        tp = O.glwe_encrypt(int(rng.integers(1, 1 << 30)), 2.0 ** -40, ks.glwe_key, m)[0]
        lwe = rand_poly(rng, n + 1)
        rot = (O.modswitch(int(lwe[n]), N)
               - sum(O.modswitch(int(lwe[i]), N) * int(ks.lwe_key[i]) for i in range(n))) % (2 * N)
        want = O.monomial_mul(O.glwe_phase(ks.glwe_key, tp), (2 * N - rot) % (2 * N))
        acc = O.blind_rotate_glwe(prm, lwe, ks.bsk, tp, O.SCHOOLBOOK)
        got = O.glwe_phase(ks.glwe_key, acc)
        err = max(abs(centred(int(x) - int(y))) for x, y in zip(got, want))
        assert err <= n * (1 + N) * 2 ** (s - 1)


def test_batched_forms_match(O):
    prm, ks = small_params(O, sigma=2.0 ** -40)
    N = prm.N
    rng = np.random.default_rng(11)
    lwe = rng.integers(0, P, (5, prm.n + 1), dtype=np.uint64)
    tp = rng.integers(0, P, (5, 2 * N), dtype=np.uint64)
    acc = O.blind_rotate_glwe_batch(prm, lwe, ks.bsk, tp, O.NTT, 2)
    for q in range(5):
        assert np.array_equal(acc[q], O.blind_rotate_glwe(prm, lwe[q], ks.bsk, tp[q]))
    autk = O.autk_keygen(3, N, TR_L, TR_B, 2.0 ** -40, ks.glwe_key)
    tr = O.trace_batch(N, TR_L, TR_B, acc, autk, O.NTT, 2)
    for q in range(5):
        assert np.array_equal(tr[q], O.trace(N, TR_L, TR_B, acc[q], autk))


# ------------------------------------------------------------ construct/recombine ---

def test_mul_plain_and_recombine_phases(O):
    """phase(pa * c + pb) = pa * phase(c) + pb and
    phase(sum_s X^s r_s) = sum_s X^s phase(r_s), exactly."""
    rng = np.random.default_rng(12)
    N = 32
    S = np.asarray(rng.integers(0, 2, N), dtype=np.uint64)
    c = rand_poly(rng, 2 * N)
    pa, pb = rand_poly(rng, N), rand_poly(rng, N)
    out = O.glwe_mul_plain(c, pa, pb)
    assert np.array_equal(O.glwe_mul_plain(c, pa, pb, O.NTT), out)
    want = (O.polymul(pa, O.glwe_phase(S, c, O.SCHOOLBOOK)).astype(object) + pb.astype(object)) % P
    assert [int(x) for x in O.glwe_phase(S, out, O.SCHOOLBOOK)] == [int(x) for x in want]
    rs = rng.integers(0, P, (3, 2 * N), dtype=np.uint64)
    R = O.glwe_recombine(rs)
    want = np.zeros(N, dtype=object)
    for s in range(3):
        want = (want + O.monomial_mul(O.glwe_phase(S, rs[s], O.SCHOOLBOOK), s).astype(object)) % P
    assert [int(x) for x in O.glwe_phase(S, R, O.SCHOOLBOOK)] == [int(x) for x in want]


# ---------------------------------------------------------- the paper's example ---

def test_paper_lookup_example_end_to_end(O):
    """Sec. 3.2 on the running example (N_br = N = 4, two segments, x = 0.22):
    Step 2 builds t = p x + q = (1.200, -0.747); Step 3 builds r_0, r_1, keeps
    coefficient I = 1 of each by blind rotation and trace (4.571 and 1.714),
    recombines them and keeps coefficient S = 0: 4.571.  Values are fixed
    point: x at scale 2^36, polynomial coefficients at 2^20, products and
    offsets at 2^56; keys and encryptions carry 2^-51 noise (the GLWE noise
    of the workloads), which the plaintext product scales by at most
    N max|coefficient| 2^20."""
    pr = EX["protocol"]
    N = EX["n_br"]
    sigma = 2.0 ** -51
    prm, ks = small_params(O, n=4, N=N, sigma=sigma, l=2, beta=12)
    S_key = ks.glwe_key
    autk = O.autk_keygen(21, N, TR_L, TR_B, sigma, S_key)
    sx, sp = 36, 20

    def enc_fixed(v, scale):
        return int(round(v * 2 ** scale)) % P

    def dec_phase(ct, scale):
        return [centred(v) / 2 ** scale for v in O.glwe_phase(S_key, ct, O.SCHOOLBOOK)]

    def poly(coefs, scale):
        out = np.zeros(N, np.uint64)
        out[:len(coefs)] = [enc_fixed(c, scale) for c in coefs]
        return out

    x = EX["x"]
    cx = O.glwe_encrypt(31, sigma, S_key, poly([x], sx))[0]
    taus = EX["segments"]
    A, B = G.build(G.FUNCTIONS["inv"], taus, N)
    p, q, a, b = G.protocol_polys(taus, A, B)

    t = O.glwe_mul_plain(cx, poly(p, sp), poly(q, sx + sp))
    got = dec_phase(t, sx + sp)
    assert all(abs(u - v) <= 5e-4 for u, v in zip(got[:2], pr["t"]))

    def select(ct, index):
        """Trace(BlindRot(ct, trivial LWE of `index` at scale p / 2N))."""
        lwe = np.zeros(prm.n + 1, np.uint64)
        lwe[prm.n] = (P // (2 * N)) * index
        assert O.modswitch(int(lwe[prm.n]), N) == index
        return O.trace(N, TR_L, TR_B, O.blind_rotate_glwe(prm, lwe, ks.bsk, ct), autk)

    rs = []
    for s, want in ((0, pr["r_0"]), (1, pr["r_1"])):
        r = O.glwe_mul_plain(cx, poly(a[s], sp), poly(b[s], sx + sp))
        assert all(abs(u - v) <= 5e-4 for u, v in zip(dec_phase(r, sx + sp), want))
        r1 = select(r, 1)                                   # I = 1
        ph = dec_phase(r1, sx + sp)
        assert abs(ph[0] - want[1]) <= 5e-4 and all(abs(v) < 1e-6 for v in ph[1:])
        rs.append(r1)
    R = O.glwe_recombine(np.stack(rs))
    ph = dec_phase(R, sx + sp)
    assert abs(ph[0] - pr["r_0"][1]) <= 5e-4 and abs(ph[1] - pr["r_1"][1]) <= 5e-4
    out = dec_phase(select(R, 0), sx + sp)                  # S = 0
    assert abs(out[0] - pr["result"]) <= 5e-4 and all(abs(v) < 1e-6 for v in out[1:])


@pytest.mark.parametrize("spacing,lo,hi", [("uniform", -20.0, 20.0), ("log", 0.01, 10.0)])
def test_encoding_selects_the_segmented_lut_interval(spacing, lo, hi):
    """The plaintext polynomials of Steps 2-3 in the clear (no encryption):
    for each segment s and each rotation r of its window (the rotations that
    round to s N/nseg, those below zero for s = 0 read through X^N = -1),
    the constant term of X^(-r) (p x + q) is (x - tau_s) nbr / width_s -
    1/2 + margin, which rounds to the interval index of the segmented LUT
    (oracle/seglut.py, the cleartext lookup of Sec. 3.1) plus the margin, at
    several positions inside every probed interval; coefficient i + margin
    of (a_s, b_s) holds that interval's line, and W keeps the window."""
    from oracle import lookup as OL
    N, nseg, margin, sx, sv, sc = 256, 4, 8, 40, 16, 50
    sp = 63 - int(math.log2(N)) - sx
    nbr = N - 2 * margin
    tau = G.boundaries(lo, hi, nseg, spacing)
    A, B = G.build(G.FUNCTIONS["silu" if spacing == "uniform" else "inv"], tau, nbr)
    parts = OL.encode(N, nseg, nbr, margin, sx, sp, sv, sc, tau, A, B)
    box, h = N // nseg, N // nseg // 2

    def const_after(poly, r):                   # constant term of X^(-r) poly
        return int(poly[r]) if r >= 0 else (P - int(poly[N + r])) % P

    for s in range(nseg):
        width = tau[s + 1] - tau[s]
        rots = [s * box + d for d in range(-h, box - h)]
        for r in rots[::7] + [rots[0], rots[-1]]:
            pr, qr = const_after(parts["p_hat"], r), const_after(parts["q_hat"], r)
            for i in (0, 1, nbr // 3, nbr - 2, nbr - 1):
                for frac in (0.1, 0.45, 0.55, 0.9):
                    x = tau[s] + (i + frac) * width / nbr
                    v = centred(pr * OL.enc(x, sx) + qr) / 2.0 ** (sx + sp)
                    assert abs(v - ((x - tau[s]) * nbr / width - 0.5 + margin)) < 1e-3, (s, r)
                    I = int(G.interval_index(np.array([x]), tau, np.array([s]), nbr)[0])
                    assert round(v) == I + margin, (s, r, i, frac, v)
        for i in (0, nbr // 2, nbr - 1):
            assert centred(parts["a_hat"][s, i + margin]) == centred(OL.enc(A[s][i], sv))
            assert centred(parts["b_hat"][s, i + margin]) == centred(OL.enc(B[s][i], sx + sv))
    # W = sum over the window of rotations of segment 0: X^d for 0 <= d < box - h,
    # and X^d = -X^(N+d) for -h <= d < 0
    w = [centred(c) for c in parts["window"]]
    assert w[:box - h] == [1] * (box - h) and w[N - h:] == [-1] * h
    assert all(c == 0 for c in w[box - h:N - h])


# ---------------------------------------------------------- multi-value batching ---

def test_multi_value_batching_trivial_exact(O):
    """Sec. 3.3.2: element j of a packed ciphertext is moved to the constant
    term by X^(-c_j) and isolated by the trace; shifting each result back by
    X^(c_j) and summing restores the packed values.  On a mask-free
    ciphertext every step is exact."""
    rng = np.random.default_rng(20)
    N = 64
    S = np.asarray(rng.integers(0, 2, N), dtype=np.uint64)
    autk = O.autk_keygen(22, N, TR_L, TR_B, 2.0 ** -40, S)
    m = rand_poly(rng, N)
    c = np.concatenate([np.zeros(N, np.uint64), m])
    pos = [0, 3, 17, 40, 63]
    singles = []
    for cj in pos:
        moved = np.concatenate([O.monomial_mul(c[:N], (2 * N - cj) % (2 * N)),
                                O.monomial_mul(c[N:], (2 * N - cj) % (2 * N))])
        t = O.trace(N, TR_L, TR_B, moved, autk)
        assert np.all(t[:N] == 0) and int(t[N]) == int(m[cj]) and np.all(t[N + 1:] == 0)
        singles.append(t)
    back = O.glwe_recombine(np.stack(singles), np.array(pos, np.uint32))
    want = np.zeros(N, np.uint64)
    want[pos] = m[pos]
    assert np.all(back[:N] == 0) and np.array_equal(back[N:], want)


def test_multi_value_batching_noise_free_bound(O):
    """With noise-free keys each extracted element's phase is the packed
    value within the trace bound (N-1) N 2^(s-1), and the recombined phase
    holds every value at its position within K times that."""
    rng = np.random.default_rng(21)
    N = 32
    s_bits = 64 - TR_L * TR_B
    S = np.asarray(rng.integers(0, 2, N), dtype=np.uint64)
    autk = O.autk_keygen(23, N, TR_L, TR_B, 0.0, S)
    c = rand_poly(rng, 2 * N)
    ph = O.glwe_phase(S, c, O.SCHOOLBOOK)
    pos = [1, 5, 30]
    bound = (N - 1) * N * 2 ** (s_bits - 1)
    singles = []
    for cj in pos:
        moved = np.concatenate([O.monomial_mul(c[:N], 2 * N - cj), O.monomial_mul(c[N:], 2 * N - cj)])
        t = O.trace(N, TR_L, TR_B, moved, autk)
        pt = O.glwe_phase(S, t, O.SCHOOLBOOK)
        assert abs(centred(int(pt[0]) - int(ph[cj]))) <= bound
        assert all(abs(centred(v)) <= bound for v in pt[1:])
        singles.append(t)
    back = O.glwe_phase(S, O.glwe_recombine(np.stack(singles), np.array(pos, np.uint32)),
                        O.SCHOOLBOOK)
    for j in range(N):
        want = int(ph[j]) if j in pos else 0
        assert abs(centred(int(back[j]) - want)) <= len(pos) * bound
