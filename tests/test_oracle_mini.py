"""The independent tier-0 oracle (oracle/mini.py) against the C oracle's
schoolbook tier, and against the facts that pin it on its own: the paper's
N = 4 rotation example (Sec. 2.2, PBS paragraph), decryption of every
message of the tiny workload to its table entry, ring products against
evaluation at every root of X^N + 1, and the decomposition's reconstruction
bound.

The two codings share only their inputs (keys, ciphertexts and tables,
which are data); agreement bit for bit on whole bootstraps pins the parts
of the C oracle that its two product tiers share (modulus switch,
accumulator start, CMux loop order, extraction and key switching)."""
import json
import os
import random

import numpy as np
import pytest

from oracle import mini
from paper_2609_16915_amd import workloads as W

P = mini.P
HERE = os.path.dirname(os.path.abspath(__file__))


def params_of(O, d):
    return O.Params.make(**{k: v for k, v in d.items() if k != "k"})


def run_both(O, prm_d, ks, cts, v):
    """Tier 1 (C, schoolbook) and tier 0 (Python) on every ciphertext;
    returns the two sets of (accumulators, extracted, key-switched)."""
    prm = params_of(O, prm_d)
    out1, big1, acc1 = O.pbs(prm, cts, ks.bsk, ks.ksk, v, O.SCHOOLBOOK, 0, want_big=True,
                             want_acc=True)
    bsk = [int(x) for x in ks.bsk]
    ksk = [int(x) for x in ks.ksk]
    vv = [int(x) for x in v]
    acc0, big0, out0 = [], [], []
    for ct in cts:
        a, b, o = mini.pbs(ct, bsk, ksk, vv, prm_d)
        acc0.append(a)
        big0.append(b)
        out0.append(o)
    to = lambda rows: np.array(rows, dtype=np.uint64)
    return (acc1, big1, out1), (to(acc0), to(big0), to(out0))


# ----------------------------------------------------------------- tiny ---

@pytest.fixture(scope="module")
def tiny(O):
    w = W.get("tiny")
    prm = params_of(O, w.params())
    ks = O.KeySet(prm, w.key_seed, w.sigma_lwe, w.sigma_glwe)
    msgs = w.messages()
    cts = O.lwe_encrypt(prm, w.enc_seed, w.sigma_lwe, ks.lwe_key, msgs)
    return w, prm, ks, msgs, cts


@pytest.mark.parametrize("table", ["identity", "square_mod"])
def test_tiny_workload_tier0_equals_tier1(O, tiny, table):
    """The whole tiny batch (8 ciphertexts, n = 64, N = 256), both tables:
    accumulators, extracted and key-switched ciphertexts equal bit for bit,
    and the tier-0 outputs decrypt to T[m]."""
    w, prm, ks, msgs, cts = tiny
    T = w.table(table)
    v = O.test_poly(prm, T)
    assert [int(x) for x in v] == mini.test_poly(T, w.N, w.msg_bits)
    one, zero = run_both(O, w.params(), ks, cts, v)
    for name, a, b in zip(("accumulator", "extracted", "key-switched"), one, zero):
        assert np.array_equal(a, b), f"{name} ciphertexts differ"
    lwe_key = [int(x) for x in ks.lwe_key]
    glwe_key = [int(x) for x in ks.glwe_key]
    for m, big, out in zip(msgs, zero[1], zero[2]):
        assert mini.lwe_decrypt(big, glwe_key, w.msg_bits) == T[m]
        assert mini.lwe_decrypt(out, lwe_key, w.msg_bits) == T[m]


def test_tiny_every_message_decrypts(O, tiny):
    """Every message of the 3-bit space through tier 0 alone (fresh
    encryptions of 0..7) decrypts to m^2 mod 8."""
    w, prm, ks, _, _ = tiny
    T = w.table("square_mod")
    msgs = np.arange(w.M, dtype=np.uint32)
    cts = O.lwe_encrypt(prm, 4242, w.sigma_lwe, ks.lwe_key, msgs)
    bsk = [int(x) for x in ks.bsk]
    ksk = [int(x) for x in ks.ksk]
    v = mini.test_poly(T, w.N, w.msg_bits)
    key = [int(x) for x in ks.lwe_key]
    for m, ct in zip(msgs, cts):
        _, _, out = mini.pbs(ct, bsk, ksk, v, w.params())
        assert mini.lwe_decrypt(out, key, w.msg_bits) == T[m]


# ------------------------------------------------------ paper example ---

def test_paper_example_tier0(O):
    """Sec. 2.2 PBS example: LUT (6, 7, 3, 5) on N = 4; trivial encryptions of
    m with a noise-free key rotate f(m) into the constant term (m = 2 -> 3),
    and tier 0 equals tier 1 on every accumulator."""
    g = json.load(open(os.path.join(HERE, "golden", "paper_pbs_example.json")))
    N, table = g["N"], g["table"]
    d = dict(n=4, k=1, N=N, pbs_level=2, pbs_base_log=8, ks_level=3, ks_base_log=4, msg_bits=2)
    prm = params_of(O, d)
    ks = O.KeySet(prm, 77, 0.0, 0.0)
    v = mini.test_poly(table, N, 2)
    delta = P // 8
    assert v == [delta * t % P for t in table]
    checks = [(e["m"], e["f_m"]) for e in g["examples"]] + [(0, 6), (1, 7), (3, 5)]
    cts = np.zeros((len(checks), d["n"] + 1), dtype=np.uint64)
    for q, (m, _) in enumerate(checks):
        cts[q, d["n"]] = delta * m
    one, zero = run_both(O, d, ks, cts, np.array(v, dtype=np.uint64))
    for a, b in zip(one, zero):
        assert np.array_equal(a, b)
    glwe_key = [int(x) for x in ks.glwe_key]
    lwe_key = [int(x) for x in ks.lwe_key]
    for (m, fm), acc, big, out in zip(checks, *zero):
        assert all(int(x) == 0 for x in acc[:N])
        assert int(acc[N]) == delta * fm % P
        assert mini.lwe_decrypt(big, glwe_key, 2) == fm
        assert mini.lwe_decrypt(out, lwe_key, 2) == fm


# ------------------------------------------------- small noisy sets ---

SMALL = [
    dict(n=8, k=1, N=32, pbs_level=2, pbs_base_log=8, ks_level=3, ks_base_log=4, msg_bits=2),
    dict(n=8, k=1, N=32, pbs_level=3, pbs_base_log=10, ks_level=5, ks_base_log=3, msg_bits=3),
    dict(n=5, k=1, N=64, pbs_level=1, pbs_base_log=20, ks_level=2, ks_base_log=12, msg_bits=2),
    dict(n=6, k=1, N=16, pbs_level=4, pbs_base_log=14, ks_level=8, ks_base_log=7, msg_bits=1),
]


@pytest.mark.parametrize("d", SMALL, ids=lambda d: f"n{d['n']}N{d['N']}l{d['pbs_level']}")
def test_small_noisy_sets_tier0_equals_tier1(O, d):
    """Noisy keys (sigma 2^-20 p, so that digits and rounding see every bit
    pattern) and ciphertexts with uniform masks and bodies, plus the edge
    words 0, 1, (p-1)/2, (p+1)/2 and p-1 in every position: both codings
    agree on every output word."""
    prm = params_of(O, d)
    ks = O.KeySet(prm, 9000 + d["N"] + d["pbs_level"], 2.0 ** -20, 2.0 ** -20)
    rng = np.random.default_rng(d["N"] * 7 + d["pbs_level"])
    cts = rng.integers(0, P, size=(6, d["n"] + 1), dtype=np.uint64)
    edges = np.array([0, 1, (P - 1) // 2, (P + 1) // 2, P - 1], dtype=np.uint64)
    cts[0, :] = edges[np.arange(d["n"] + 1) % 5]
    cts[1, :] = edges[(np.arange(d["n"] + 1) + 2) % 5]
    v = rng.integers(0, P, size=d["N"], dtype=np.uint64)
    one, zero = run_both(O, d, ks, cts, v)
    for name, a, b in zip(("accumulator", "extracted", "key-switched"), one, zero):
        assert np.array_equal(a, b), f"{name} ciphertexts differ"


# ----------------------------------------------------- tier-0 pieces ---

def _eval(poly, z):
    acc = 0
    for c in reversed(poly):
        acc = (acc * z + c) % P
    return acc


@pytest.mark.parametrize("N", [4, 32, 256])
def test_ring_product_at_every_root(N):
    """(a b)(z) = a(z) b(z) at all N roots z of X^N + 1 (the odd powers of a
    primitive 2N-th root of unity, 7 generating Z_p^*)."""
    rnd = random.Random(N)
    psi = pow(7, (P - 1) // (2 * N), P)
    assert pow(psi, N, P) == P - 1
    a = [rnd.randrange(P) for _ in range(N)]
    b = [rnd.randrange(P) for _ in range(N)]
    c = mini.ring_mul(a, b, N)
    for k in range(N):
        z = pow(psi, 2 * k + 1, P)
        assert _eval(c, z) == _eval(a, z) * _eval(b, z) % P
    # X * X^(N-1) = -1
    x1 = [0] * N
    x1[1] = 1
    xl = [0] * N
    xl[N - 1] = 1
    assert mini.ring_mul(x1, xl, N) == [P - 1] + [0] * (N - 1)
    assert mini.monomial(x1, N - 1, N) == [P - 1] + [0] * (N - 1)


@pytest.mark.parametrize("levels,beta", [(2, 8), (3, 8), (1, 30), (4, 14), (6, 3), (5, 3)])
def test_decompose_reconstruction(levels, beta):
    """sum_t d_t 2^(64-(t+1) beta) is within 2^(s-1) of the centred value,
    digits in range, on edge and random words."""
    s = 64 - levels * beta
    B = 1 << beta
    rnd = random.Random(levels * 100 + beta)
    words = [0, 1, (P - 1) // 2, (P + 1) // 2, P - 1, P - 2, 1 << 63, (1 << s) - 1,
             1 << (s - 1), (1 << (s - 1)) - 1] + [rnd.randrange(P) for _ in range(300)]
    for a in words:
        d = mini.decompose(a, levels, beta)
        ac = a if a <= (P - 1) // 2 else a - P
        val = sum(dt << (64 - (t + 1) * beta) for t, dt in enumerate(d))
        assert -(1 << (s - 1)) <= ac - val < (1 << (s - 1))
        assert all(-B // 2 <= dt < B // 2 for dt in d[1:])
        assert -B // 2 <= d[0] <= B // 2


def test_modswitch_boundaries():
    """Nearest integer to 2N a / p: just below and above each half-way point,
    and the ends of Z_p."""
    for N in (4, 256, 2048, 4096):
        assert mini.modswitch(0, N) == 0
        assert mini.modswitch(P - 1, N) == 0
        for k in (0, 1, N - 1, 2 * N - 1):
            # a with 2N a / p closest to k + 1/2 from below and above
            lo = ((2 * k + 1) * P) // (4 * N)
            assert mini.modswitch(lo, N) == k % (2 * N)
            assert mini.modswitch(lo + 1, N) == (k + 1) % (2 * N)
