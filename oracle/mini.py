"""Independent pure-Python PBS (the oracle's tier 0).

TEST INFRASTRUCTURE ONLY: imported by tests/ alone, never by the product
package, the benchmark or the C oracle.  It imports nothing from
oracle/oracle.c or oracle/oracle.py and shares no helper with them: every
step of the bootstrap is written out again here, in Python integers, from
the definitions, so that a slip in one coding of the shared conventions
(loop order, which word is modulus-switched, the CMux form, the extraction
index, the key-switch sign, the decomposition) shows up as a disagreement
with the other.

What is computed (ROSETTA, Sec. 2.2 "TFHE Scheme", PBS paragraph and
Fig. rlwe_primitives(a); Sec. 2.2.3 for the extraction): the test polynomial
v holding the table is rotated by the negated, modulus-switched message of
an LWE ciphertext, one CMux per mask coefficient, so that f(m) reaches the
constant term; that term is extracted as an LWE ciphertext under the GLWE
key and switched back to the n-dimensional key.  The conventions the paper
leaves open are the library's and the C oracle's (they decide the output
bits):

  * q = p = 2^64 - 2^32 + 1, ring Z_p[X]/(X^N + 1), k = 1;
  * modulus switch: the integer nearest to 2N a / p, reduced mod 2N (p is
    odd, so no value lies half-way);
  * accumulator start (0, X^(-b~) v); CMux for i = 0, 1, .., n-1:
    ACC <- ACC + GGSW_i (x) (X^(a~_i) ACC - ACC);
  * decomposition of a word a into l signed base-2^beta digits: centred
    representative, rounded half up at s = 64 - l beta bits, balanced digits
    taken from the least significant level, the top level keeps the rest;
    level t weighs 2^(64 - (t+1) beta); digits enter products as d mod p;
  * bootstrapping key [i][u][t][c][x]: row (u, t) of GGSW(s_i) is a GLWE
    encryption of zero with s_i 2^(64-(t+1) beta) added to component u;
  * extraction a'_0 = A_0, a'_j = -A_{N-j}, b' = B_0 (phase B - A S);
  * key switching out = (0, .., 0, b') - sum_j sum_t d_{j,t} KSK[j][t],
    KSK [N][l_ks][n+1].

Ring products use Kronecker substitution, a method neither C tier uses
(those are schoolbook and a radix-2 transform): both operands' coefficients
(as residues in [0, p)) are packed into one integer each at a slot width
that no sum of products can overflow, the two integers are multiplied with
Python's exact big-integer product, and the slots of the result are the
coefficients of the plain product in Z[X]; folding X^N = -1 and reducing mod
p gives the negacyclic product.
"""
from __future__ import annotations

from fractions import Fraction

P = 2 ** 64 - 2 ** 32 + 1

# Slot width (bytes) of the Kronecker packing.  A slot of the product holds a
# sum of at most 2 l N products of residues below p, each below 2^128; with
# l <= 8 and N <= 4096 that is below 2^144, so 20 bytes (160 bits) leave
# room to spare and slots never carry into each other.
_SLOT = 20


def _pack(coeffs) -> int:
    """The integer sum_j c_j 2^(160 j) of residues c_j in [0, p)."""
    return int.from_bytes(b"".join(int(c).to_bytes(_SLOT, "little") for c in coeffs), "little")


def _unpack_fold(x: int, N: int):
    """Slots 0 .. 2N-1 of a packed product, folded by X^N = -1, mod p."""
    raw = x.to_bytes(2 * N * _SLOT, "little")
    slot = [int.from_bytes(raw[j * _SLOT:(j + 1) * _SLOT], "little") for j in range(2 * N)]
    return [(slot[j] - slot[j + N]) % P for j in range(N)]


def ring_mul(a, b, N: int):
    """Negacyclic product a b in Z_p[X]/(X^N + 1) by Kronecker substitution."""
    return _unpack_fold(_pack(a) * _pack(b), N)


def monomial(a, r: int, N: int):
    """X^r a in Z_p[X]/(X^N + 1) for any integer r: coefficient a_i moves to
    position i + r taken mod 2N, and a position N + e stands for -X^e."""
    out = [0] * N
    for i, c in enumerate(a):
        e = (i + r) % (2 * N)
        if e < N:
            out[e] = c % P
        else:
            out[e - N] = (-c) % P
    return out


def modswitch(a: int, N: int) -> int:
    """Nearest integer to 2N a / p, mod 2N (exact rational rounding)."""
    return round(Fraction(2 * N * int(a), P)) % (2 * N)


def decompose(a: int, levels: int, beta: int):
    """Signed digits [d_0 .. d_(l-1)] of the word a (d_0 the most significant):
    sum_t d_t 2^(64-(t+1) beta) is the centred value of a rounded half up at
    s = 64 - l beta bits; every digit but d_0 lies in [-B/2, B/2), d_0 in
    [-B/2, B/2]."""
    B = 1 << beta
    s = 64 - levels * beta
    ac = int(a) if a <= (P - 1) // 2 else int(a) - P
    r = (ac + (1 << (s - 1))) >> s          # floor division by 2^s (arbitrary precision)
    digits = [0] * levels
    for t in range(levels - 1, 0, -1):
        d = (r + B // 2) % B - B // 2
        digits[t] = d
        r = (r - d) // B
    digits[0] = r
    return digits


def test_poly(table, N: int, msg_bits: int):
    """Test polynomial of a table of M = 2^msg_bits entries: with a padding
    bit the messages occupy M of 2M rotation slots, each a box of N/M
    coefficients centred on its rotation (half a box before it, half after),
    and the half box that wraps below 0 is stored negated at the top."""
    M = 1 << msg_bits
    delta = P // (2 * M)
    box = N // M
    h = box // 2
    v = []
    for j in range(N):
        if j < N - h:
            v.append(delta * int(table[(j + h) // box]) % P)
        else:
            v.append((-delta * int(table[0])) % P)
    return v


def blind_rotate(lwe, bsk, v, n: int, N: int, levels: int, beta: int, acc0=None):
    """Blind rotation of v (or of the GLWE ciphertext acc0 = (A, B)) by the LWE
    ciphertext lwe = (a_0 .. a_(n-1), b), bsk indexed [i][u][t][c][x] as a flat
    sequence of words.  Returns the accumulator (A, B)."""
    bt = modswitch(lwe[n], N)
    if acc0 is None:
        A = [0] * N
        B = monomial(v, -bt, N)
    else:
        A = monomial(acc0[0], -bt, N)
        B = monomial(acc0[1], -bt, N)
    row = lambda i, u, t, c: bsk[(((i * 2 + u) * levels + t) * 2 + c) * N:
                                 (((i * 2 + u) * levels + t) * 2 + c + 1) * N]
    for i in range(n):
        ai = modswitch(lwe[i], N)
        acc = (A, B)
        diff = [[(x - y) % P for x, y in zip(monomial(acc[u], ai, N), acc[u])] for u in (0, 1)]
        # digit polynomials delta[u][t] (as residues), from each coefficient's digits
        digs = [[decompose(x, levels, beta) for x in diff[u]] for u in (0, 1)]
        packed = {}
        for u in (0, 1):
            for t in range(levels):
                packed[u, t] = _pack([d[t] % P for d in digs[u]])
        new = []
        for c in (0, 1):
            total = 0
            for u in (0, 1):
                for t in range(levels):
                    total += packed[u, t] * _pack(row(i, u, t, c))
            prod = _unpack_fold(total, N)
            new.append([(x + y) % P for x, y in zip(acc[c], prod)])
        A, B = new
    return A, B


def sample_extract(A, B, N: int):
    """LWE ciphertext (a'_0 .. a'_(N-1), b') of the constant coefficient of the
    GLWE phase B - A S: a'_0 = A_0, a'_j = -A_(N-j), b' = B_0."""
    return [A[0]] + [(-A[N - j]) % P for j in range(1, N)] + [B[0]]


def keyswitch(big, ksk, n: int, N: int, levels: int, beta: int):
    """(0, .., 0, b') - sum_j sum_t d_(j,t) KSK[j][t], KSK flat [N][l][n+1]."""
    out = [0] * n + [big[N]]
    for j in range(N):
        for t, d in enumerate(decompose(big[j], levels, beta)):
            if d == 0:
                continue
            base = (j * levels + t) * (n + 1)
            for c in range(n + 1):
                out[c] = (out[c] - d * ksk[base + c]) % P
    return out


def pbs(lwe, bsk, ksk, v, prm: dict):
    """Whole bootstrap of one ciphertext; returns (accumulator A + B as one
    list of 2N words, extracted [N+1], key-switched [n+1])."""
    n, N = prm["n"], prm["N"]
    A, B = blind_rotate([int(x) for x in lwe], bsk, v, n, N, prm["pbs_level"],
                        prm["pbs_base_log"])
    big = sample_extract(A, B, N)
    out = keyswitch(big, ksk, n, N, prm["ks_level"], prm["ks_base_log"])
    return A + B, big, out


def lwe_phase(ct, key):
    """b - <a, s> mod p."""
    return (int(ct[-1]) - sum(int(a) * int(s) for a, s in zip(ct[:-1], key))) % P


def lwe_decrypt(ct, key, msg_bits: int) -> int:
    """Nearest multiple of p / 2M to the phase, as an element of Z_(2M)."""
    M2 = 2 << msg_bits
    return round(Fraction(M2 * lwe_phase(ct, key), P)) % M2
