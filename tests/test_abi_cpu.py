"""CPU-side checks of librosetta: it loads, exports every symbol the header
declares, validates arguments before touching a device, and its host helpers
(key generation, encryption, decryption, test polynomial) agree bit for bit
with the oracle's independent implementations of the same definitions."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2609_16915_amd import rosetta as R
from paper_2609_16915_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rosetta.h")


@pytest.fixture(scope="module")
def L():
    return R.lib()


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rosetta_\w+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    names = header_functions()
    assert len(names) >= 20
    for name in names:
        assert hasattr(L, name), name
    # and the binding covers exactly the declared set
    assert sorted(R.SIGNATURES) == names


def test_status_strings(L):
    for code, name in R.STATUS.items():
        assert L.rosetta_status_string(code).decode() == name
    assert L.rosetta_version().decode().startswith("rosetta-pbs")


def test_version_names_the_built_sources(L):
    """rosetta_version() carries the digest of the sources the library was
    compiled from; it must equal the digest of the sources in the tree (a
    stale library, built before a source change, fails here)."""
    from paper_2609_16915_amd import build as B
    v = L.rosetta_version().decode()
    assert v.endswith("src:" + B.source_digest()), (v, B.source_digest())


def test_bsk_device_words_is_the_standard_size(L):
    for kw in (dict(), dict(n=1024, N=2048, pbs_level=3), dict(n=7, N=4096, pbs_level=4)):
        p = P(**kw)
        assert L.rosetta_bsk_device_words(C.byref(p)) == L.rosetta_bsk_words(C.byref(p)) == \
            p.n * 2 * p.pbs_level * 2 * p.N


def P(**kw):
    base = dict(n=64, k=1, N=256, pbs_level=2, pbs_base_log=8, ks_level=3, ks_base_log=4,
                msg_bits=3)
    base.update(kw)
    return R.Params.from_dict(base)


@pytest.mark.parametrize("kw,matrix", [
    ({}, True),                                                   # 3 x 4 bits, N = 256
    ({"n": 1024, "N": 2048, "ks_level": 6, "ks_base_log": 3}, True),   # headline shape
    ({"n": 1024, "N": 4096, "ks_level": 6, "ks_base_log": 3}, True),
    ({"ks_level": 2, "ks_base_log": 7}, True),                    # digits up to 64
    ({"ks_level": 2, "ks_base_log": 8}, False),                   # a digit of 128
    ({"ks_level": 5, "ks_base_log": 6}, True),                    # 30-bit rounded value
    ({"ks_level": 4, "ks_base_log": 8}, False),                   # 32-bit rounded value
    # the largest digit sums a valid set allows (N = 4096, 4 x 7 bits) stay
    # at 2^27, inside the int32 bound the dispatch also checks
    ({"N": 4096, "ks_level": 4, "ks_base_log": 7}, True),
    ({"n": 2048, "N": 2048, "ks_level": 2, "ks_base_log": 8}, False),
])
def test_ksk_device_words_follow_the_documented_layouts(L, kw, matrix):
    # the prepared key-switching key is the byte-plane layout exactly when
    # the header's matrix-core condition holds, else key words + column sums
    p = P(**kw)
    n, N, lks, b = p.n, p.N, p.ks_level, p.ks_base_log
    cond = (1 <= b <= 7 and lks * b <= 30 and N % 32 == 0
            and N * lks * (1 << (b - 1)) * 128 < (1 << 31))
    assert cond == matrix
    plane_words = -(-(n + 1) // 32) * (N * lks // 32) * 1024
    std_words = N * lks * (n + 1)
    assert L.rosetta_ksk_words(C.byref(p)) == std_words
    assert L.rosetta_ksk_device_words(C.byref(p)) == (plane_words if matrix
                                                      else std_words + n + 1)


def test_byte_plane_identity_of_the_key_switch():
    # the arithmetic the matrix-core key switch rests on, checked in exact
    # integers: for every word K in [0, p), V = K or K - p lies in the range
    # of 8 balanced base-256 digits [-128 S, 127 S] (S = (2^64 - 1) / 255),
    # X = V + 128 S = K + 128 S (+ 2^32 - 1 when V = K - p) mod 2^64, and the
    # bytes of X with the top bit flipped, read as signed, are those digits
    p = 0xFFFFFFFF00000001
    S = (2 ** 64 - 1) // 255
    rng = np.random.default_rng(11)
    words = [0, 1, 2, p - 1, p - 2, 127 * S - 1, 127 * S, 127 * S + 1, 2 ** 63 - 1, 2 ** 63,
             p - 2 ** 63 - 1, p - 2 ** 63, 2 ** 32 - 1, 2 ** 32]
    words += [int(x) for x in rng.integers(0, p, 20000, dtype=np.uint64)]
    for K in words:
        V = K if K <= 127 * S else K - p
        assert -128 * S <= V <= 127 * S
        X = (K + 128 * S + (0 if K <= 127 * S else 2 ** 32 - 1)) % 2 ** 64
        assert X == V + 128 * S
        digits = [((X >> (8 * m)) & 0xFF) ^ 0x80 for m in range(8)]
        digits = [d - 256 if d >= 128 else d for d in digits]
        assert all(-128 <= d <= 127 for d in digits)
        assert sum(d * 256 ** m for m, d in enumerate(digits)) == V
        assert V % p == K


@pytest.mark.parametrize("kw,status", [
    ({}, 0),
    ({"k": 2}, 3),
    ({"N": 128}, 3), ({"N": 8192}, 3), ({"N": 1000}, 3),
    ({"n": 0}, 2), ({"n": 4096}, 3),
    ({"pbs_level": 0}, 2), ({"pbs_level": 5}, 3), ({"pbs_base_log": 31}, 3),
    ({"pbs_level": 4, "pbs_base_log": 16}, 3),
    ({"ks_level": 9}, 3), ({"ks_level": 0}, 2),
    ({"ks_level": 8, "ks_base_log": 20, "N": 4096}, 3),
    ({"msg_bits": 0}, 2), ({"msg_bits": 9}, 2),
])
def test_param_validation(L, kw, status):
    assert L.rosetta_check_params(C.byref(P(**kw))) == status
    if status:
        assert L.rosetta_last_error().decode()


def test_null_and_empty_batches_touch_no_device(L):
    p = P()
    fake = 0x10000
    assert L.rosetta_pbs_batch(None, fake, fake, fake, fake, 4, C.byref(p), None) == 1
    assert L.rosetta_pbs_batch(fake, fake, fake, fake, fake + 10 ** 6, 0, C.byref(p), None) == 0
    assert L.rosetta_pbs_batch(None, None, None, None, None, 0, C.byref(p), None) == 0
    assert L.rosetta_keyswitch(None, fake, fake, 3, C.byref(p), None) == 1
    assert L.rosetta_ntt_forward(None, None, 0, 256, None) == 0
    assert L.rosetta_ntt_forward(None, fake, 2, 256, None) == 1
    assert L.rosetta_ntt_forward(fake, fake, 2, 100, None) == 3
    assert L.rosetta_check_params(None) == 1
    # field ops: unknown op, missing operands, empty
    assert L.rosetta_field_op(6, fake, fake, fake, fake, 2, None) == 2
    assert L.rosetta_field_op(4, fake, None, None, fake, 2, None) == 1
    assert L.rosetta_field_op(5, fake, fake, None, fake, 2, None) == 1
    assert L.rosetta_field_op(256 + 96, fake, None, None, fake, 2, None) == 2
    assert L.rosetta_field_op(-1, fake, fake, fake, fake, 2, None) == 2
    assert L.rosetta_field_op(2, fake, None, None, fake, 2, None) == 1
    assert L.rosetta_field_op(3, fake, fake, None, fake, 2, None) == 1
    assert L.rosetta_field_op(256 + 48, None, None, None, fake, 2, None) == 1
    assert L.rosetta_field_op(512, fake, None, None, fake, 2, None) == 2  # s = 0
    assert L.rosetta_field_op(512 + 64, fake, None, None, fake, 2, None) == 2
    assert L.rosetta_field_op(512 + 34, None, None, None, fake, 2, None) == 1
    assert L.rosetta_field_op(512 + 34, fake, None, None, fake, 0, None) == 0
    assert L.rosetta_field_op(2, None, None, None, None, 0, None) == 0
    assert L.rosetta_modmul_chain(1, 0, 10, None, None) == 0
    assert L.rosetta_modmul_chain(1, 5, 10, None, None) == 1


def test_alias_and_size_detection(L):
    p = P()
    base = 1 << 40
    io = 4 * (p.n + 1) * 8
    bsk, ksk, lut = base + 10 ** 9, base + 2 * 10 ** 9, base + 3 * 10 ** 9
    ws = base + 4 * 10 ** 9
    need = L.rosetta_pbs_workspace_bytes(C.byref(p), 4)
    assert need == 4 * (p.N + 1) * 8
    # partial overlap of input and output
    st = L.rosetta_pbs_batch_ws(base, bsk, ksk, lut, base + 8, 4, C.byref(p), ws, need, None)
    assert st == 4
    # workspace too small
    st = L.rosetta_pbs_batch_ws(base, bsk, ksk, lut, base + io, 4, C.byref(p), ws, need - 8,
                                None)
    assert st == 7
    # workspace overlapping the output
    st = L.rosetta_pbs_batch_ws(base, bsk, ksk, lut, ws + 16, 4, C.byref(p), ws, need, None)
    assert st == 4
    # blind rotation output overlapping the key
    st = L.rosetta_blind_rotate(base, bsk, lut, bsk + 64, 4, C.byref(p), None)
    assert st == 4


# ------------------------------------------------------ host helpers ---

@pytest.mark.parametrize("name", ["tiny", "gpt2_gelu"])
def test_keygen_matches_oracle(O, name):
    w = W.get(name)
    lib_keys = R.keygen(w.key_seed, w.params(), w.sigma_lwe, w.sigma_glwe)
    op = O.Params.make(**{k: v for k, v in w.params().items() if k != "k"})
    ks = O.KeySet(op, w.key_seed, w.sigma_lwe, w.sigma_glwe)
    assert np.array_equal(lib_keys["lwe_key"], ks.lwe_key)
    assert np.array_equal(lib_keys["glwe_key"], ks.glwe_key)
    assert np.array_equal(lib_keys["bsk"], ks.bsk)
    assert np.array_equal(lib_keys["ksk"], ks.ksk)


def test_encrypt_decrypt_lut_match_oracle(O):
    w = W.get("tiny")
    op = O.Params.make(**{k: v for k, v in w.params().items() if k != "k"})
    ks = O.KeySet(op, w.key_seed, w.sigma_lwe, w.sigma_glwe)
    msgs = np.arange(16, dtype=np.uint32) % (2 * w.M)
    a = R.lwe_encrypt(w.enc_seed, w.params(), w.sigma_lwe, ks.lwe_key, msgs)
    b = O.lwe_encrypt(op, w.enc_seed, w.sigma_lwe, ks.lwe_key, msgs)
    assert np.array_equal(a, b)
    assert np.array_equal(R.lwe_decrypt(w.params(), ks.lwe_key, a), msgs)
    plain = np.random.default_rng(3).integers(0, 2 ** 64 - 2 ** 32, 9, dtype=np.uint64)
    assert np.array_equal(R.lwe_encrypt_plain(w.enc_seed, w.params(), w.sigma_lwe, ks.lwe_key,
                                              plain),
                          O.lwe_encrypt_plain(w.enc_seed, w.sigma_lwe, ks.lwe_key, plain))
    assert np.array_equal(R.lwe_decrypt(w.params(), ks.lwe_key, a), O.lwe_decrypt(op, ks.lwe_key, a))
    for fn in ("identity", "square_mod"):
        t = w.table(fn)
        assert np.array_equal(R.lut_build(w.params(), t), O.test_poly(op, t))
    for name in ("gpt2_gelu", "llama3_8b_silu", "llama3_8b_softmax_exp"):
        w2 = W.get(name)
        op2 = O.Params.make(**{k: v for k, v in w2.params().items() if k != "k"})
        assert np.array_equal(R.lut_build(w2.params(), w2.table()), O.test_poly(op2, w2.table()))


# ------------------------------------------------ lookup-protocol entry points ---

def test_lookup_validation_touches_no_device(L):
    p = P()
    fake = 1 << 40
    assert L.rosetta_autk_words(C.byref(p), 4) == 8 * 4 * 2 * 256
    # trace parameters
    for lv, bl, st in [(0, 12, 2), (5, 12, 3), (4, 31, 3), (4, 16, 3), (4, 12, 0)]:
        got = L.rosetta_trace(fake, fake + 10 ** 9, fake + 2 * 10 ** 9, 2, C.byref(p), lv, bl, None)
        if st == 0:
            continue                 # valid arguments would launch; not on a CPU machine
        assert got == st, (lv, bl)
    # empty batches are no-ops, NULL pointers are rejected
    assert L.rosetta_trace(None, None, None, 0, C.byref(p), 4, 12, None) == 0
    assert L.rosetta_trace(None, fake, fake, 1, C.byref(p), 4, 12, None) == 1
    assert L.rosetta_blind_rotate_glwe(None, None, None, None, 0, 1, C.byref(p), 0, None) == 0
    assert L.rosetta_blind_rotate_glwe(fake, fake, fake, fake, 1, 0, C.byref(p), 0, None) == 2
    assert L.rosetta_blind_rotate_glwe(fake, fake, None, fake, 1, 1, C.byref(p), 0, None) == 1
    assert L.rosetta_glwe_mul_plain(None, None, None, None, 0, 2, 256, None) == 0
    assert L.rosetta_glwe_mul_plain(fake, fake, None, fake, 1, 0, 256, None) == 2
    assert L.rosetta_glwe_mul_plain(fake, fake, None, fake, 1, 2, 100, None) == 3
    assert L.rosetta_glwe_recombine(None, None, None, 0, 2, 256, None) == 0
    assert L.rosetta_glwe_recombine(fake, None, fake, 1, 0, 256, None) == 2
    assert L.rosetta_glwe_recombine(fake, None, fake, 1, 257, 256, None) == 2
    bad = (C.c_uint32 * 2)(0, 512)                     # exponent not below 2N
    assert L.rosetta_glwe_recombine(fake, C.addressof(bad), fake, 1, 2, 256, None) == 2
    assert L.rosetta_glwe_monomial_mul(fake, None, fake, 1, 2, 256, None) == 1
    assert L.rosetta_glwe_monomial_mul(fake, C.addressof(bad), fake, 1, 2, 256, None) == 2
    assert L.rosetta_sample_extract(None, None, 0, 256, None) == 0
    assert L.rosetta_sample_extract(fake, fake + 8, 1, 256, None) == 4
    # aliasing
    two_n = 2 * p.N * 8
    assert L.rosetta_trace(fake, fake + 10 ** 9, fake + 8, 2, C.byref(p), 4, 12, None) == 4
    assert L.rosetta_blind_rotate_glwe(fake, fake + 10 ** 9, fake + 2 * 10 ** 9,
                                       fake + 2 * 10 ** 9 + 8, 1, 1, C.byref(p), 0, None) == 4
    assert L.rosetta_glwe_recombine(fake, None, fake + two_n, 1, 2, 256, None) == 4
    assert L.rosetta_glwe_mul_plain(fake, fake + 10 ** 9, None, fake + two_n // 2, 1, 1, 256,
                                    None) == 4


def test_glwe_helpers_match_oracle(O):
    w = W.get("tiny")
    prm = w.params()
    op = O.Params.make(**{k: v for k, v in prm.items() if k != "k"})
    ks = O.KeySet(op, w.key_seed, w.sigma_lwe, w.sigma_glwe)
    rng = np.random.default_rng(5)
    msgs = rng.integers(0, 2 ** 63, (3, w.N), dtype=np.uint64)
    a = R.glwe_encrypt(77, prm, 2.0 ** -40, ks.glwe_key, msgs)
    assert np.array_equal(a, O.glwe_encrypt(77, 2.0 ** -40, ks.glwe_key, msgs))
    ph = R.glwe_phase(prm, ks.glwe_key, a)
    for q in range(3):
        assert np.array_equal(ph[q], O.glwe_phase(ks.glwe_key, a[q]))
    for lv, bl in ((4, 12), (2, 20)):
        k1 = R.autk_keygen(78, prm, lv, bl, 2.0 ** -51, ks.glwe_key)
        k2 = O.autk_keygen(78, w.N, lv, bl, 2.0 ** -51, ks.glwe_key)
        assert k1.shape == k2.shape and np.array_equal(k1, k2)
