"""ctypes binding of the plain CPU oracle (oracle/oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg, never by the product package.  It marshals
numpy arrays into the C oracle and holds no arithmetic of its own.

Conventions (all fixed in oracle.c, next to each function):
  * field Z_p, p = 2^64 - 2^32 + 1; ring Z_p[X]/(X^N + 1);
  * LWE ciphertexts (a_0..a_{d-1}, b), phase b - <a, s>;
  * GLWE (k = 1) ciphertexts (A[0..N), B[0..N)), phase B - A*S;
  * bootstrapping key [n][u][t][c][N], key-switching key [N][l_ks][n+1].
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# ROSETTA_ORACLE_LIB names another build of oracle.c (the mutation tests load
# copies with one planted mistake each through it)
LIB_PATH = os.environ.get("ROSETTA_ORACLE_LIB") or os.path.join(HERE, "liboracle.so")

P = 0xFFFFFFFF00000001
SCHOOLBOOK = 0
NTT = 1


class Params(C.Structure):
    """Parameter set (independent mirror of the C struct in oracle.c)."""

    _fields_ = [(name, C.c_uint32) for name in
                ("n", "k", "N", "pbs_level", "pbs_base_log", "ks_level",
                 "ks_base_log", "msg_bits")]

    @classmethod
    def make(cls, n, N, pbs_level, pbs_base_log, ks_level, ks_base_log, msg_bits, k=1):
        return cls(n=n, k=k, N=N, pbs_level=pbs_level, pbs_base_log=pbs_base_log,
                   ks_level=ks_level, ks_base_log=ks_base_log, msg_bits=msg_bits)

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            import importlib.util
            spec = importlib.util.spec_from_file_location("_oracle_build",
                                                          os.path.join(HERE, "build.py"))
            mod = importlib.util.module_from_spec(spec)
            spec.loader.exec_module(mod)
            mod.build()
        _lib = C.CDLL(LIB_PATH)
        _declare(_lib)
    return _lib


_u64p = C.POINTER(C.c_uint64)
_i64p = C.POINTER(C.c_int64)
_u32p = C.POINTER(C.c_uint32)
_pp = C.POINTER(Params)


def _declare(L):
    sig = {
        "or_add": (C.c_uint64, [C.c_uint64, C.c_uint64]),
        "or_sub": (C.c_uint64, [C.c_uint64, C.c_uint64]),
        "or_neg": (C.c_uint64, [C.c_uint64]),
        "or_mul": (C.c_uint64, [C.c_uint64, C.c_uint64]),
        "or_pow": (C.c_uint64, [C.c_uint64, C.c_uint64]),
        "or_inv": (C.c_uint64, [C.c_uint64]),
        "or_root_2n": (C.c_uint64, [C.c_int]),
        "or_polymul_schoolbook": (None, [_u64p, _u64p, _u64p, C.c_int]),
        "or_polymul_ntt": (None, [_u64p, _u64p, _u64p, C.c_int]),
        "or_ntt_forward": (None, [_u64p, C.c_int]),
        "or_ntt_inverse": (None, [_u64p, C.c_int]),
        "or_poly_monomial_mul": (None, [_u64p, C.c_int, _u64p, C.c_int]),
        "or_modswitch": (C.c_uint32, [C.c_uint64, C.c_int]),
        "or_decompose": (None, [C.c_uint64, C.c_int, C.c_int, _i64p]),
        "or_splitmix_word": (C.c_uint64, [C.c_uint64, C.c_uint64]),
        "or_gauss": (C.c_double, [C.c_uint64, C.c_uint64]),
        "or_lwe_phase": (None, [_u64p, C.c_int, _u64p, C.c_size_t, _u64p]),
        "or_lwe_decrypt": (None, [_pp, _u64p, C.c_int, _u64p, C.c_size_t, _u32p]),
        "or_lwe_encrypt_plain": (None, [C.c_uint64, C.c_double, _u64p, C.c_int, _u64p,
                                        C.c_size_t, _u64p]),
        "or_lwe_encrypt": (None, [C.c_uint64, _pp, C.c_double, _u64p, C.c_int, _u32p,
                                  C.c_size_t, _u64p]),
        "or_glwe_phase": (None, [C.c_int, _u64p, _u64p, _u64p, C.c_int]),
        "or_test_poly": (None, [_pp, _u32p, _u64p]),
        "or_bsk_words": (C.c_size_t, [_pp]),
        "or_ksk_words": (C.c_size_t, [_pp]),
        "or_keygen": (None, [C.c_uint64, _pp, C.c_double, C.c_double, _u64p, _u64p, _u64p,
                             _u64p]),
        "or_external_product": (None, [_pp, _u64p, _u64p, _u64p, C.c_int]),
        "or_bsk_transform": (None, [_pp, _u64p, _u64p, C.c_int]),
        "or_blind_rotate": (None, [_pp, _u64p, _u64p, _u64p, _u64p, _u64p, C.c_int]),
        "or_sample_extract": (None, [C.c_int, _u64p, _u64p]),
        "or_keyswitch": (None, [_pp, _u64p, _u64p, _u64p]),
        "or_pbs": (None, [_pp, _u64p, _u64p, _u64p, _u64p, _u64p, _u64p, _u64p, C.c_size_t,
                          C.c_int, C.c_int]),
        "or_pbs_prepared": (None, [_pp, _u64p, _u64p, _u64p, _u64p, _u64p, _u64p, _u64p, _u64p,
                                   C.c_size_t, C.c_int, C.c_int]),
        "or_blind_rotate_glwe": (None, [_pp, _u64p, _u64p, _u64p, _u64p, _u64p, C.c_int]),
        "or_automorphism": (None, [_u64p, C.c_int, _u64p, C.c_int]),
        "or_glwe_keyswitch": (None, [C.c_int, C.c_int, C.c_int, _u64p, _u64p, _u64p, C.c_int]),
        "or_autk_words": (C.c_size_t, [C.c_int, C.c_int]),
        "or_autk_keygen": (None, [C.c_uint64, C.c_int, C.c_int, C.c_int, C.c_double, _u64p,
                                  _u64p]),
        "or_trace": (None, [C.c_int, C.c_int, C.c_int, _u64p, _u64p, _u64p, C.c_int]),
        "or_glwe_encrypt": (None, [C.c_uint64, C.c_int, C.c_double, _u64p, _u64p, C.c_size_t,
                                   _u64p]),
        "or_glwe_mul_plain": (None, [C.c_int, _u64p, _u64p, _u64p, _u64p, C.c_int]),
        "or_glwe_recombine": (None, [C.c_int, _u64p, C.c_int, _u32p, _u64p]),
        "or_blind_rotate_glwe_batch": (None, [_pp, _u64p, _u64p, _u64p, _u64p, C.c_size_t,
                                              C.c_int, C.c_int]),
        "or_trace_batch": (None, [C.c_int, C.c_int, C.c_int, _u64p, _u64p, _u64p, C.c_size_t,
                                  C.c_int, C.c_int]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args


def _u64(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.uint64)
    return a


def _ptr(a: np.ndarray | None, typ=_u64p):
    if a is None:
        return None
    return a.ctypes.data_as(typ)


# --------------------------------------------------------------------------
# scalar field operations
# --------------------------------------------------------------------------

def add(a, b): return lib().or_add(a, b)
def sub(a, b): return lib().or_sub(a, b)
def neg(a): return lib().or_neg(a)
def mul(a, b): return lib().or_mul(a, b)
def pow_(a, e): return lib().or_pow(a, e)
def inv(a): return lib().or_inv(a)
def root_2n(N): return lib().or_root_2n(N)
def modswitch(a, N): return lib().or_modswitch(a, N)
def splitmix_word(key, idx): return lib().or_splitmix_word(key, idx)
def gauss(key, idx): return lib().or_gauss(key, idx)


def decompose(a: int, levels: int, beta: int) -> list[int]:
    d = np.zeros(levels, dtype=np.int64)
    lib().or_decompose(a, levels, beta, _ptr(d, _i64p))
    return [int(x) for x in d]


# --------------------------------------------------------------------------
# polynomials
# --------------------------------------------------------------------------

def polymul(a, b, kind=SCHOOLBOOK) -> np.ndarray:
    a, b = _u64(a), _u64(b)
    N = a.shape[0]
    c = np.zeros(N, dtype=np.uint64)
    f = lib().or_polymul_schoolbook if kind == SCHOOLBOOK else lib().or_polymul_ntt
    f(_ptr(a), _ptr(b), _ptr(c), N)
    return c


def ntt_forward(a) -> np.ndarray:
    a = _u64(a).copy()
    lib().or_ntt_forward(_ptr(a), a.shape[0])
    return a


def ntt_inverse(a) -> np.ndarray:
    a = _u64(a).copy()
    lib().or_ntt_inverse(_ptr(a), a.shape[0])
    return a


def monomial_mul(a, r: int) -> np.ndarray:
    a = _u64(a)
    c = np.zeros_like(a)
    lib().or_poly_monomial_mul(_ptr(a), r, _ptr(c), a.shape[0])
    return c


# --------------------------------------------------------------------------
# keys, encryption, encodings
# --------------------------------------------------------------------------

class KeySet:
    """Oracle key material for one parameter set and seed."""

    def __init__(self, params: Params, seed: int, sigma_lwe: float, sigma_glwe: float):
        self.params = params
        self.seed = seed
        self.sigma_lwe = sigma_lwe
        self.sigma_glwe = sigma_glwe
        L = lib()
        pp = C.byref(params)
        self.lwe_key = np.zeros(params.n, dtype=np.uint64)
        self.glwe_key = np.zeros(params.N, dtype=np.uint64)
        self.bsk = np.zeros(L.or_bsk_words(pp), dtype=np.uint64)
        self.ksk = np.zeros(L.or_ksk_words(pp), dtype=np.uint64)
        L.or_keygen(seed, pp, sigma_lwe, sigma_glwe, _ptr(self.lwe_key), _ptr(self.glwe_key),
                    _ptr(self.bsk), _ptr(self.ksk))

    def ggsw(self, i: int) -> np.ndarray:
        p = self.params
        w = 2 * p.pbs_level * 2 * p.N
        return self.bsk[i * w:(i + 1) * w]


def lwe_encrypt(params: Params, seed: int, sigma: float, key, msgs) -> np.ndarray:
    key = _u64(key)
    msgs = np.ascontiguousarray(msgs, dtype=np.uint32)
    dim = key.shape[0]
    out = np.zeros((msgs.shape[0], dim + 1), dtype=np.uint64)
    lib().or_lwe_encrypt(seed, C.byref(params), sigma, _ptr(key), dim, _ptr(msgs, _u32p),
                         msgs.shape[0], _ptr(out))
    return out


def lwe_encrypt_plain(seed: int, sigma: float, key, plain) -> np.ndarray:
    key, plain = _u64(key), _u64(plain)
    dim = key.shape[0]
    out = np.zeros((plain.shape[0], dim + 1), dtype=np.uint64)
    lib().or_lwe_encrypt_plain(seed, sigma, _ptr(key), dim, _ptr(plain), plain.shape[0],
                               _ptr(out))
    return out


def lwe_decrypt(params: Params, key, cts) -> np.ndarray:
    key = _u64(key)
    cts = _u64(cts)
    dim = key.shape[0]
    cts = cts.reshape(-1, dim + 1)
    out = np.zeros(cts.shape[0], dtype=np.uint32)
    lib().or_lwe_decrypt(C.byref(params), _ptr(key), dim, _ptr(cts), cts.shape[0],
                         _ptr(out, _u32p))
    return out


def lwe_phase(key, cts) -> np.ndarray:
    key = _u64(key)
    dim = key.shape[0]
    cts = _u64(cts).reshape(-1, dim + 1)
    out = np.zeros(cts.shape[0], dtype=np.uint64)
    lib().or_lwe_phase(_ptr(key), dim, _ptr(cts), cts.shape[0], _ptr(out))
    return out


def glwe_phase(glwe_key, ct, kind=NTT) -> np.ndarray:
    S, ct = _u64(glwe_key), _u64(ct)
    N = S.shape[0]
    out = np.zeros(N, dtype=np.uint64)
    lib().or_glwe_phase(N, _ptr(S), _ptr(ct), _ptr(out), kind)
    return out


def test_poly(params: Params, table) -> np.ndarray:
    table = np.ascontiguousarray(table, dtype=np.uint32)
    assert table.shape[0] == (1 << params.msg_bits)
    v = np.zeros(params.N, dtype=np.uint64)
    lib().or_test_poly(C.byref(params), _ptr(table, _u32p), _ptr(v))
    return v


# --------------------------------------------------------------------------
# the PBS pipeline
# --------------------------------------------------------------------------

def external_product(params: Params, ggsw, glwe, kind=SCHOOLBOOK) -> np.ndarray:
    ggsw, glwe = _u64(ggsw), _u64(glwe)
    out = np.zeros(2 * params.N, dtype=np.uint64)
    lib().or_external_product(C.byref(params), _ptr(ggsw), _ptr(glwe), _ptr(out), kind)
    return out


def blind_rotate(params: Params, lwe, bsk, v, kind=SCHOOLBOOK) -> np.ndarray:
    lwe, bsk, v = _u64(lwe), _u64(bsk), _u64(v)
    acc = np.zeros(2 * params.N, dtype=np.uint64)
    lib().or_blind_rotate(C.byref(params), _ptr(lwe), _ptr(bsk), None, _ptr(v), _ptr(acc), kind)
    return acc


def sample_extract(N: int, acc) -> np.ndarray:
    acc = _u64(acc)
    big = np.zeros(N + 1, dtype=np.uint64)
    lib().or_sample_extract(N, _ptr(acc), _ptr(big))
    return big


def keyswitch(params: Params, big, ksk) -> np.ndarray:
    big, ksk = _u64(big), _u64(ksk)
    out = np.zeros(params.n + 1, dtype=np.uint64)
    lib().or_keyswitch(C.byref(params), _ptr(big), _ptr(ksk), _ptr(out))
    return out


def pbs(params: Params, lwe_in, bsk, ksk, v, kind=NTT, nthreads=0,
        want_big=False, want_acc=False):
    """Full PBS of a batch [count][n+1].  Returns lwe_out (and optionally the
    extracted [count][N+1] and the accumulators [count][2N])."""
    lwe_in = _u64(lwe_in).reshape(-1, params.n + 1)
    bsk, ksk, v = _u64(bsk), _u64(ksk), _u64(v)
    count = lwe_in.shape[0]
    out = np.zeros((count, params.n + 1), dtype=np.uint64)
    big = np.zeros((count, params.N + 1), dtype=np.uint64) if want_big else None
    acc = np.zeros((count, 2 * params.N), dtype=np.uint64) if want_acc else None
    lib().or_pbs(C.byref(params), _ptr(lwe_in), _ptr(bsk), _ptr(ksk), _ptr(v), _ptr(out),
                 _ptr(big), _ptr(acc), count, kind, nthreads)
    res = [out]
    if want_big:
        res.append(big)
    if want_acc:
        res.append(acc)
    return res[0] if len(res) == 1 else tuple(res)


def bsk_transform(params: Params, bsk, nthreads=0) -> np.ndarray:
    """Forward transform of every bootstrapping-key row (the tier-2 PBS's
    once-per-key work)."""
    bsk = _u64(bsk)
    out = np.zeros_like(bsk)
    lib().or_bsk_transform(C.byref(params), _ptr(bsk), _ptr(out), nthreads)
    return out


def pbs_prepared(params: Params, lwe_in, fbsk, ksk, v, nthreads=0, want_big=False):
    """Tier-2 PBS of a batch with the key transform already done
    (bsk_transform): returns lwe_out (and the extracted [count][N+1])."""
    lwe_in = _u64(lwe_in).reshape(-1, params.n + 1)
    fbsk, ksk, v = _u64(fbsk), _u64(ksk), _u64(v)
    out = np.zeros((lwe_in.shape[0], params.n + 1), dtype=np.uint64)
    big = np.zeros((lwe_in.shape[0], params.N + 1), dtype=np.uint64) if want_big else None
    lib().or_pbs_prepared(C.byref(params), _ptr(lwe_in), None, _ptr(fbsk), _ptr(ksk), _ptr(v),
                          _ptr(out), _ptr(big), None, lwe_in.shape[0], NTT, nthreads)
    return (out, big) if want_big else out


# --------------------------------------------------------------------------
# lookup-protocol primitives (Sec. 3.2, Sec. 2.2.3)
# --------------------------------------------------------------------------

def blind_rotate_glwe(params: Params, lwe, bsk, tp, kind=SCHOOLBOOK) -> np.ndarray:
    """Blind rotation of one GLWE test-polynomial ciphertext tp [2N]."""
    lwe, bsk, tp = _u64(lwe), _u64(bsk), _u64(tp)
    acc = np.zeros(2 * params.N, dtype=np.uint64)
    lib().or_blind_rotate_glwe(C.byref(params), _ptr(lwe), _ptr(bsk), None, _ptr(tp), _ptr(acc),
                               kind)
    return acc


def blind_rotate_glwe_batch(params: Params, lwe, bsk, tp, kind=NTT, nthreads=0) -> np.ndarray:
    lwe = _u64(lwe).reshape(-1, params.n + 1)
    count = lwe.shape[0]
    tp = _u64(tp).reshape(count, 2 * params.N)
    acc = np.zeros((count, 2 * params.N), dtype=np.uint64)
    lib().or_blind_rotate_glwe_batch(C.byref(params), _ptr(lwe), _ptr(_u64(bsk)), _ptr(tp),
                                     _ptr(acc), count, kind, nthreads)
    return acc


def automorphism(a, d: int) -> np.ndarray:
    a = _u64(a)
    out = np.zeros_like(a)
    lib().or_automorphism(_ptr(a), d, _ptr(out), a.shape[0])
    return out


def glwe_keyswitch(N: int, levels: int, beta: int, ct, ksk, kind=SCHOOLBOOK) -> np.ndarray:
    ct, ksk = _u64(ct), _u64(ksk)
    out = np.zeros(2 * N, dtype=np.uint64)
    lib().or_glwe_keyswitch(N, levels, beta, _ptr(ct), _ptr(ksk), _ptr(out), kind)
    return out


def autk_words(N: int, levels: int) -> int:
    return lib().or_autk_words(N, levels)


def autk_keygen(seed: int, N: int, levels: int, beta: int, sigma: float, glwe_key) -> np.ndarray:
    S = _u64(glwe_key)
    out = np.zeros(autk_words(N, levels), dtype=np.uint64)
    lib().or_autk_keygen(seed, N, levels, beta, sigma, _ptr(S), _ptr(out))
    return out


def trace(N: int, levels: int, beta: int, ct, autk, kind=SCHOOLBOOK) -> np.ndarray:
    ct, autk = _u64(ct), _u64(autk)
    out = np.zeros(2 * N, dtype=np.uint64)
    lib().or_trace(N, levels, beta, _ptr(ct), _ptr(autk), _ptr(out), kind)
    return out


def trace_batch(N: int, levels: int, beta: int, cts, autk, kind=NTT, nthreads=0) -> np.ndarray:
    cts = _u64(cts).reshape(-1, 2 * N)
    out = np.zeros_like(cts)
    lib().or_trace_batch(N, levels, beta, _ptr(cts), _ptr(_u64(autk)), _ptr(out), cts.shape[0],
                         kind, nthreads)
    return out


def glwe_encrypt(seed: int, sigma: float, glwe_key, msgs) -> np.ndarray:
    """GLWE encryptions of plaintext polynomials msgs [count][N] (scaled into Z_p)."""
    S = _u64(glwe_key)
    N = S.shape[0]
    msgs = _u64(msgs).reshape(-1, N)
    out = np.zeros((msgs.shape[0], 2 * N), dtype=np.uint64)
    lib().or_glwe_encrypt(seed, N, sigma, _ptr(S), _ptr(msgs), msgs.shape[0], _ptr(out))
    return out


def glwe_mul_plain(ct, pa, pb=None, kind=SCHOOLBOOK) -> np.ndarray:
    ct, pa = _u64(ct), _u64(pa)
    N = pa.shape[0]
    out = np.zeros(2 * N, dtype=np.uint64)
    pbp = None if pb is None else _u64(pb)
    lib().or_glwe_mul_plain(N, _ptr(ct), _ptr(pa), _ptr(pbp), _ptr(out), kind)
    return out


def glwe_recombine(cts, exps=None) -> np.ndarray:
    """sum_s X^(exps[s]) cts[s] (exps None: X^s)."""
    cts = _u64(cts)
    count, twoN = cts.shape
    out = np.zeros(twoN, dtype=np.uint64)
    e = None if exps is None else np.ascontiguousarray(exps, dtype=np.uint32)
    lib().or_glwe_recombine(twoN // 2, _ptr(cts), count, _ptr(e, _u32p), _ptr(out))
    return out
