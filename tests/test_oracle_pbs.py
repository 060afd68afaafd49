"""Pins of the oracle's PBS pipeline (CPU only): the paper's worked example,
closed forms on trivial ciphertexts, exact phase identities, deterministic
noise bounds, and decrypt(PBS(Enc m)) = T[m] on small parameter sets."""
import json
import os

import numpy as np
import pytest

from paper_2609_16915_amd import workloads as W

P = 0xFFFFFFFF00000001
HERE = os.path.dirname(os.path.abspath(__file__))


def centred(x):
    x = int(x)
    return x if x <= (P - 1) // 2 else x - P


def params_of(O, w):
    return O.Params.make(**{k: v for k, v in w.params().items() if k != "k"})


@pytest.fixture(scope="module")
def tiny(O):
    w = W.get("tiny")
    prm = params_of(O, w)
    ks = O.KeySet(prm, w.key_seed, w.sigma_lwe, w.sigma_glwe)
    return w, prm, ks


# ------------------------------------------------------- paper example ---

def test_paper_rotation_example(O):
    """Sec. 2.2 PBS example: LUT (6, 7, 3, 5) as the coefficients of the test
    polynomial; an encryption of m = 2 rotates f(2) = 3 into the constant
    term.  Noise-free keys and a trivial input ciphertext make every step
    exact."""
    g = json.load(open(os.path.join(HERE, "golden", "paper_pbs_example.json")))
    N = g["N"]
    table = np.array(g["table"], dtype=np.uint32)
    prm = O.Params.make(n=4, N=N, pbs_level=2, pbs_base_log=8, ks_level=3, ks_base_log=4,
                        msg_bits=2)
    ks = O.KeySet(prm, 77, 0.0, 0.0)
    v = O.test_poly(prm, table)
    delta = P // (2 * 4)
    assert [int(x) for x in v] == [delta * int(t) % P for t in table]
    checks = [(e["m"], e["f_m"]) for e in g["examples"]] + [(0, 6), (1, 7), (3, 5)]
    for m, fm in checks:
        lwe = np.zeros(prm.n + 1, dtype=np.uint64)
        lwe[prm.n] = delta * m                           # trivial encryption of m
        for kind in (O.SCHOOLBOOK, O.NTT):
            acc = O.blind_rotate(prm, lwe, ks.bsk, v, kind)
            assert np.all(acc[:N] == 0)
            assert np.array_equal(acc[N:], O.monomial_mul(v, (2 * N - m) % (2 * N)))
            assert int(acc[N]) == delta * fm % P        # f(m) in the constant term
        out, big = O.pbs(prm, lwe[None, :], ks.bsk, ks.ksk, v, O.SCHOOLBOOK, 1, want_big=True)
        assert int(O.lwe_decrypt(prm, ks.glwe_key, big)[0]) == fm
        assert int(O.lwe_decrypt(prm, ks.lwe_key, out)[0]) == fm


# -------------------------------------------------------- closed forms ---

def test_trivial_input_closed_form(O, tiny):
    """With a = 0 every CMux difference is zero, so blind rotation returns
    exactly (0, X^(-b~) v) whatever the (noisy) key."""
    w, prm, ks = tiny
    N = prm.N
    rng = np.random.default_rng(9)
    v = O.test_poly(prm, w.table("square_mod"))
    for b in [0, 1, P - 1, P // 2] + [int(x) for x in rng.integers(0, P, 4, dtype=np.uint64)]:
        lwe = np.zeros(prm.n + 1, dtype=np.uint64)
        lwe[prm.n] = b
        bt = O.modswitch(b, N)
        acc = O.blind_rotate(prm, lwe, ks.bsk, v, O.NTT)
        assert np.all(acc[:N] == 0)
        assert np.array_equal(acc[N:], O.monomial_mul(v, (2 * N - bt) % (2 * N)))


def test_sample_extract_phase_identity(O):
    """decrypt_S(extract(C)) equals the constant coefficient of phase(C)."""
    N = 64
    rng = np.random.default_rng(11)
    S = rng.integers(0, 2, N, dtype=np.uint64)
    for _ in range(5):
        C = rng.integers(0, P, 2 * N, dtype=np.uint64)
        big = O.sample_extract(N, C)
        assert int(O.lwe_phase(S, big)[0]) == int(O.glwe_phase(S, C, O.SCHOOLBOOK)[0])


def test_external_product_noise_free(O):
    """Noise-free GGSW: GGSW(0) (x) C has phase exactly 0; GGSW(1) (x) C has
    phase(C) + err with |err| <= (1 + N) 2^(s-1) coefficient-wise (rounding of
    the decomposition, the mask part multiplied by the binary key)."""
    prm = O.Params.make(n=16, N=64, pbs_level=2, pbs_base_log=8, ks_level=3, ks_base_log=4,
                        msg_bits=3)
    ks = O.KeySet(prm, 5, 0.0, 0.0)
    N = prm.N
    s = 64 - prm.pbs_level * prm.pbs_base_log
    bound = (1 + N) * 2 ** (s - 1)
    rng = np.random.default_rng(12)
    ones = [i for i in range(prm.n) if ks.lwe_key[i] == 1]
    zeros = [i for i in range(prm.n) if ks.lwe_key[i] == 0]
    assert ones and zeros
    for _ in range(3):
        C = rng.integers(0, P, 2 * N, dtype=np.uint64)
        ph = O.glwe_phase(ks.glwe_key, C, O.SCHOOLBOOK)
        for kind in (O.SCHOOLBOOK, O.NTT):
            r0 = O.external_product(prm, ks.ggsw(zeros[0]), C, kind)
            assert np.all(O.glwe_phase(ks.glwe_key, r0, O.SCHOOLBOOK) == 0)
            r1 = O.external_product(prm, ks.ggsw(ones[0]), C, kind)
            ph1 = O.glwe_phase(ks.glwe_key, r1, O.SCHOOLBOOK)
            err = [centred((int(a) - int(b)) % P) for a, b in zip(ph1, ph)]
            assert max(abs(e) for e in err) <= bound
            # the bound is not vacuous: the error is far below the modulus
            assert bound < 2 ** 60


def test_keyswitch_phase_bound(O):
    """Key switching preserves the phase up to the decomposition rounding,
    |err| <= N 2^(s_ks - 1) (binary extracted key), when the key-switching
    key is noise-free; with noise a probabilistic term of at most
    8 sigma 2^64 sqrt(N l_ks (B^2/12 + 1/6)) is added."""
    rng = np.random.default_rng(13)
    for sigma in (0.0, 2.0 ** -40):
        prm = O.Params.make(n=32, N=256, pbs_level=2, pbs_base_log=8, ks_level=3,
                            ks_base_log=4, msg_bits=3)
        ks = O.KeySet(prm, 6, sigma, 0.0)
        s_ks = 64 - prm.ks_level * prm.ks_base_log
        B = 1 << prm.ks_base_log
        bound = prm.N * 2 ** (s_ks - 1)
        if sigma:
            bound += 8 * sigma * 2 ** 64 * np.sqrt(prm.N * prm.ks_level * (B * B / 12 + 1 / 6))
        for _ in range(4):
            big = rng.integers(0, P, prm.N + 1, dtype=np.uint64)
            ph_big = int(O.lwe_phase(ks.glwe_key, big)[0])
            out = O.keyswitch(prm, big, ks.ksk)
            ph_out = int(O.lwe_phase(ks.lwe_key, out)[0])
            assert abs(centred((ph_out - ph_big) % P)) <= bound


def test_keygen_rows_decrypt(O, tiny):
    """Each bootstrapping-key row decrypts to s_i g_t on its component, and
    each key-switching-key row to S_j g^ks_t, within the noise."""
    w, prm, ks = tiny
    N, l, beta = prm.N, prm.pbs_level, prm.pbs_base_log
    noise = 10 * w.sigma_glwe * 2 ** 64
    S = [int(x) for x in ks.glwe_key]
    for i in (0, 1, prm.n - 1):
        si = int(ks.lwe_key[i])
        G = ks.ggsw(i)
        for u in range(2):
            for t in range(l):
                row = G[(u * l + t) * 2 * N:(u * l + t + 1) * 2 * N]
                ph = O.glwe_phase(ks.glwe_key, row, O.SCHOOLBOOK)
                g = 2 ** (64 - (t + 1) * beta) % P
                if u == 1:   # body row: phase = s_i g_t + E
                    want = [si * g if x == 0 else 0 for x in range(N)]
                else:        # mask row: phase = -s_i g_t S + E
                    want = [(-si * g * S[x]) % P for x in range(N)]
                err = [abs(centred((int(a) - b) % P)) for a, b in zip(ph, want)]
                assert max(err) <= noise
    s_ks = prm.ks_base_log
    kn = 10 * w.sigma_lwe * 2 ** 64
    ksk = ks.ksk.reshape(N, prm.ks_level, prm.n + 1)
    for j in (0, 5, N - 1):
        for t in range(prm.ks_level):
            ph = int(O.lwe_phase(ks.lwe_key, ksk[j, t])[0])
            want = S[j] * 2 ** (64 - (t + 1) * s_ks) % P
            assert abs(centred((ph - want) % P)) <= kn


# ------------------------------------------------------- full PBS: tiny ---

@pytest.mark.parametrize("fn", ["identity", "square_mod"])
def test_pbs_decrypts_to_table_every_message(O, tiny, fn):
    """decrypt(PBS(Enc m)) = T[m] for every m of the 3-bit message space,
    and tier 1 (schoolbook) equals tier 2 (transform) bit for bit on the
    accumulators, the extracted and the key-switched ciphertexts."""
    w, prm, ks = tiny
    table = w.table(fn)
    v = O.test_poly(prm, table)
    msgs = np.array(list(range(w.M)) * 2, dtype=np.uint32)
    cts = O.lwe_encrypt(prm, w.enc_seed, w.sigma_lwe, ks.lwe_key, msgs)
    assert np.array_equal(O.lwe_decrypt(prm, ks.lwe_key, cts), msgs)
    o1, b1, a1 = O.pbs(prm, cts, ks.bsk, ks.ksk, v, O.SCHOOLBOOK, 0, True, True)
    o2, b2, a2 = O.pbs(prm, cts, ks.bsk, ks.ksk, v, O.NTT, 0, True, True)
    assert np.array_equal(a1, a2) and np.array_equal(b1, b2) and np.array_equal(o1, o2)
    assert np.array_equal(O.lwe_decrypt(prm, ks.glwe_key, b1), table[msgs])
    assert np.array_equal(O.lwe_decrypt(prm, ks.lwe_key, o1), table[msgs])


def test_pbs_output_chains(O, tiny):
    """The output is again a ciphertext under the input key, so PBS chains:
    T2[T1[m]] after two bootstraps."""
    w, prm, ks = tiny
    t1, t2 = w.table("square_mod"), w.table("identity")[::-1].copy()
    msgs = np.arange(w.M, dtype=np.uint32)
    cts = O.lwe_encrypt(prm, 3, w.sigma_lwe, ks.lwe_key, msgs)
    o1 = O.pbs(prm, cts, ks.bsk, ks.ksk, O.test_poly(prm, t1), O.NTT)
    o2 = O.pbs(prm, o1, ks.bsk, ks.ksk, O.test_poly(prm, t2), O.NTT)
    assert np.array_equal(O.lwe_decrypt(prm, ks.lwe_key, o2), t2[t1[msgs]])


def test_test_poly_layout(O):
    """v_j = Delta T[floor((j + h)/box)] for j < N - h, and -Delta T[0] in the
    last half-box (negacyclic wrap of entry 0)."""
    prm = O.Params.make(n=4, N=32, pbs_level=2, pbs_base_log=8, ks_level=3, ks_base_log=4,
                        msg_bits=2)
    table = np.array([1, 2, 3, 0], dtype=np.uint32)
    v = [int(x) for x in O.test_poly(prm, table)]
    delta = P // 8
    box, h = 8, 4
    assert v[:4] == [delta * 1] * 4                      # first half-box: entry 0
    assert v[4:12] == [delta * 2] * 8                    # entry 1 centred on j = 8
    assert v[12:20] == [delta * 3] * 8
    assert v[20:28] == [0] * 8
    assert v[28:] == [(-delta) % P] * 4                  # wrap of entry 0
    assert box * 4 == 32 and h == 4


# -------------------------------------------------- full PBS: GPT-2 GELU ---

def test_pbs_gpt2_gelu_semantics(O):
    """At the GPT-2 GELU parameters (n = 742, N = 2048, l = 2, beta = 10)
    decrypt(PBS(Enc m)) = T[m] for every m of the 4-bit space."""
    w = W.get("gpt2_gelu")
    prm = params_of(O, w)
    ks = O.KeySet(prm, w.key_seed, w.sigma_lwe, w.sigma_glwe)
    table = w.table()
    v = O.test_poly(prm, table)
    msgs = np.arange(w.M, dtype=np.uint32)
    cts = O.lwe_encrypt(prm, w.enc_seed, w.sigma_lwe, ks.lwe_key, msgs)
    out, big = O.pbs(prm, cts, ks.bsk, ks.ksk, v, O.NTT, 0, want_big=True)
    assert np.array_equal(O.lwe_decrypt(prm, ks.glwe_key, big), table[msgs])
    assert np.array_equal(O.lwe_decrypt(prm, ks.lwe_key, out), table[msgs])
