"""Python binding of librosetta (batched TFHE PBS on MI355X).

Argument marshalling only: every step of the PBS runs in the library's HIP
kernels.  Device buffers are torch tensors on a ROCm device (dtype uint64, or
int64 read as raw 64-bit words), passed by data_ptr() together with the
current HIP stream; host helpers take and return numpy arrays.  There is no
fallback: if the library is not built, or a call fails, an exception is
raised.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librosetta.so")
P = 0xFFFFFFFF00000001

STATUS = {0: "ROSETTA_OK", 1: "ROSETTA_ERR_NULL", 2: "ROSETTA_ERR_PARAMS",
          3: "ROSETTA_ERR_UNSUPPORTED", 4: "ROSETTA_ERR_ALIAS", 5: "ROSETTA_ERR_NOMEM",
          6: "ROSETTA_ERR_DEVICE", 7: "ROSETTA_ERR_SIZE"}


class RosettaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class Params(C.Structure):
    """rosetta_params (include/rosetta.h)."""

    _fields_ = [(name, C.c_uint32) for name in
                ("n", "k", "N", "pbs_level", "pbs_base_log", "ks_level", "ks_base_log",
                 "msg_bits")]

    @classmethod
    def from_dict(cls, d: dict) -> "Params":
        d = dict(d)
        d.setdefault("k", 1)
        return cls(**d)

    @property
    def M(self) -> int:
        return 1 << self.msg_bits


# Every symbol the header declares, with its ctypes signature.
_u64p = C.c_void_p
_pp = C.POINTER(Params)
_ST = C.c_int
SIGNATURES = {
    "rosetta_version": (C.c_char_p, []),
    "rosetta_status_string": (C.c_char_p, [C.c_int]),
    "rosetta_last_error": (C.c_char_p, []),
    "rosetta_check_params": (_ST, [_pp]),
    "rosetta_bsk_words": (C.c_size_t, [_pp]),
    "rosetta_bsk_device_words": (C.c_size_t, [_pp]),
    "rosetta_ksk_words": (C.c_size_t, [_pp]),
    "rosetta_ksk_device_words": (C.c_size_t, [_pp]),
    "rosetta_bsk_prepare": (_ST, [_u64p, _u64p, _pp, C.c_void_p]),
    "rosetta_ksk_prepare": (_ST, [_u64p, _u64p, _pp, C.c_void_p]),
    "rosetta_pbs_batch": (_ST, [_u64p, _u64p, _u64p, _u64p, _u64p, C.c_size_t, _pp,
                                C.c_void_p]),
    "rosetta_pbs_workspace_bytes": (C.c_size_t, [_pp, C.c_size_t]),
    "rosetta_pbs_batch_ws": (_ST, [_u64p, _u64p, _u64p, _u64p, _u64p, C.c_size_t, _pp,
                                   C.c_void_p, C.c_size_t, C.c_void_p]),
    "rosetta_pbs_batch_noalloc": (_ST, [_u64p, _u64p, _u64p, _u64p, _u64p, C.c_size_t, _pp,
                                        C.c_void_p]),
    "rosetta_blind_rotate": (_ST, [_u64p, _u64p, _u64p, _u64p, C.c_size_t, _pp, C.c_void_p]),
    "rosetta_blind_rotate_extract": (_ST, [_u64p, _u64p, _u64p, _u64p, C.c_size_t, _pp,
                                           C.c_void_p]),
    "rosetta_keyswitch": (_ST, [_u64p, _u64p, _u64p, C.c_size_t, _pp, C.c_void_p]),
    "rosetta_ntt_forward": (_ST, [_u64p, _u64p, C.c_size_t, C.c_uint32, C.c_void_p]),
    "rosetta_ntt_inverse": (_ST, [_u64p, _u64p, C.c_size_t, C.c_uint32, C.c_void_p]),
    "rosetta_poly_mul": (_ST, [_u64p, _u64p, _u64p, C.c_size_t, C.c_uint32, C.c_void_p]),
    "rosetta_field_op": (_ST, [C.c_int, _u64p, _u64p, _u64p, _u64p, C.c_size_t, C.c_void_p]),
    "rosetta_modmul_chain": (_ST, [C.c_uint64, C.c_uint32, C.c_uint32, _u64p, C.c_void_p]),
    "rosetta_keygen": (_ST, [C.c_uint64, _pp, C.c_double, C.c_double, _u64p, _u64p, _u64p,
                             _u64p]),
    "rosetta_lwe_encrypt": (_ST, [C.c_uint64, _pp, C.c_double, _u64p, C.c_uint32, _u64p,
                                  C.c_size_t, _u64p]),
    "rosetta_lwe_decrypt": (_ST, [_pp, _u64p, C.c_uint32, _u64p, C.c_size_t, _u64p]),
    "rosetta_lwe_encrypt_plain": (_ST, [C.c_uint64, C.c_double, _u64p, C.c_uint32, _u64p,
                                        C.c_size_t, _u64p]),
    "rosetta_lut_build": (_ST, [_pp, _u64p, _u64p]),
    "rosetta_shutdown": (_ST, []),
    "rosetta_blind_rotate_glwe": (_ST, [_u64p, _u64p, _u64p, _u64p, C.c_size_t, C.c_uint32,
                                        _pp, C.c_int, C.c_void_p]),
    "rosetta_lwe_add_consts": (_ST, [_u64p, _u64p, _u64p, C.c_size_t, C.c_uint32, C.c_uint32,
                                     C.c_void_p]),
    "rosetta_lwe_sum_groups": (_ST, [_u64p, C.c_uint64, _u64p, C.c_size_t, C.c_uint32,
                                     C.c_uint32, C.c_void_p]),
    "rosetta_lwe_combine": (_ST, [_u64p, C.c_uint64, _u64p, C.c_uint64, _u64p, C.c_uint64, _u64p,
                                  C.c_size_t, C.c_void_p]),
    "rosetta_autk_words": (C.c_size_t, [_pp, C.c_uint32]),
    "rosetta_autk_prepare": (_ST, [_u64p, _u64p, _pp, C.c_uint32, C.c_void_p]),
    "rosetta_trace": (_ST, [_u64p, _u64p, _u64p, C.c_size_t, _pp, C.c_uint32, C.c_uint32,
                            C.c_void_p]),
    "rosetta_plain_prepare": (_ST, [_u64p, _u64p, C.c_size_t, C.c_uint32, C.c_void_p]),
    "rosetta_glwe_mul_plain": (_ST, [_u64p, _u64p, _u64p, _u64p, C.c_size_t, C.c_uint32,
                                     C.c_uint32, C.c_void_p]),
    "rosetta_glwe_recombine": (_ST, [_u64p, _u64p, _u64p, C.c_size_t, C.c_uint32, C.c_uint32,
                                     C.c_void_p]),
    "rosetta_glwe_monomial_mul": (_ST, [_u64p, _u64p, _u64p, C.c_size_t, C.c_uint32,
                                        C.c_uint32, C.c_void_p]),
    "rosetta_sample_extract": (_ST, [_u64p, _u64p, C.c_size_t, C.c_uint32, C.c_void_p]),
    "rosetta_glwe_encrypt": (_ST, [C.c_uint64, _pp, C.c_double, _u64p, _u64p, C.c_size_t,
                                   _u64p]),
    "rosetta_glwe_phase": (_ST, [_pp, _u64p, _u64p, C.c_size_t, _u64p]),
    "rosetta_autk_keygen": (_ST, [C.c_uint64, _pp, C.c_uint32, C.c_uint32, C.c_double, _u64p,
                                  _u64p]),
    "rosetta_seglut_boundaries": (_ST, [C.c_double, C.c_double, C.c_uint32, C.c_int, _u64p]),
    "rosetta_seglut_build": (_ST, [C.c_int, _u64p, C.c_uint32, C.c_uint32, C.c_int, _u64p,
                                   _u64p]),
    "rosetta_seglut_protocol_polys": (_ST, [_u64p, C.c_uint32, C.c_uint32, _u64p, _u64p]),
    "rosetta_seglut_eval": (_ST, [_u64p, C.c_uint32, C.c_uint32, _u64p, _u64p, _u64p, _u64p,
                                  C.c_size_t, _u64p]),
    "rosetta_seglut_precision": (_ST, [C.c_int, _u64p, C.c_uint32, C.c_uint32, _u64p, _u64p,
                                       _u64p, _u64p, C.c_size_t, _u64p]),
    "rosetta_encode_fixed": (_ST, [_u64p, C.c_size_t, C.c_int, _u64p]),
}



class LookupParams(C.Structure):
    """rosetta_lookup_params (include/rosetta.h)."""

    _fields_ = [(name, C.c_uint32) for name in
                ("nseg", "nbr", "margin", "x_scale_log", "coef_scale_log", "val_scale_log",
                 "cmp_scale_log", "trace_level", "trace_base_log", "cmp_refine_log")]


_lpp = C.POINTER(LookupParams)
SIGNATURES.update({
    "rosetta_lookup_plain_words": (C.c_size_t, [_pp, _lpp]),
    "rosetta_lookup_encode": (_ST, [_pp, _lpp, _u64p, _u64p, _u64p, _u64p, _u64p]),
    "rosetta_lookup_prepare": (_ST, [_u64p, _u64p, _pp, _lpp, C.c_void_p]),
    "rosetta_lookup_workspace_bytes": (C.c_size_t, [_pp, _lpp, C.c_size_t]),
    "rosetta_lookup_workspace_offset": (C.c_size_t, [_pp, _lpp, C.c_size_t, C.c_uint32]),
    "rosetta_lookup_eval": (_ST, [_u64p, _u64p, _u64p, _u64p, _u64p, _u64p, _u64p, _u64p,
                                  C.c_size_t, _pp, _lpp, _u64p, C.c_size_t, C.c_void_p]),
})

FUNCTIONS = {"inv": 0, "inv_sqrt": 1, "silu": 2, "gelu": 3, "exp": 4}
SPACINGS = {"uniform": 0, "log": 1}
FITS = {"linear": 0, "constant": 1}

_lib = None


def lib():
    """Load librosetta.so (built in-tree by paper_2609_16915_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run "
                               "`python -m paper_2609_16915_amd.build` first")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise RosettaError(status, lib().rosetta_last_error().decode())


def _params(p) -> Params:
    return p if isinstance(p, Params) else Params.from_dict(p)


# --------------------------------------------------------------------------
# device buffers (torch)
# --------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _dev(t, name: str) -> int:
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a torch tensor on a ROCm device")
    if t.element_size() != 8 or not t.is_contiguous():
        raise TypeError(f"{name} must be contiguous with 64-bit elements")
    return t.data_ptr()


def _stream(stream) -> int:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _words(t) -> int:
    """Element count of a tensor (or numpy array)."""
    return int(t.numel()) if hasattr(t, "numel") else int(t.size)


def _expect(t, name: str, words: int):
    """Raise ValueError unless `t` holds exactly `words` elements.  Runs before
    any library call, so that a buffer of the wrong size never reaches a
    kernel (which would read or write out of its bounds)."""
    got = _words(t)
    if got != words:
        raise ValueError(f"{name} holds {got} words, the call needs {words}")


def _batch_of(t, name: str, row: int, allow_empty: bool = True) -> int:
    """Rows of `row` words in `t`; ValueError if the size is not a multiple."""
    got = _words(t)
    if got % row or (got == 0 and not allow_empty):
        raise ValueError(f"{name} holds {got} words, not a whole number of {row}-word rows")
    return got // row


def empty(words, device="cuda"):
    torch = _torch()
    return torch.empty(words, dtype=torch.uint64, device=device)


def to_device(a: np.ndarray, device="cuda"):
    torch = _torch()
    a = np.ascontiguousarray(a, dtype=np.uint64)
    return torch.from_numpy(a).to(device)


def to_host(t) -> np.ndarray:
    return t.cpu().numpy().view(np.uint64)


def bsk_words(params) -> int:
    return lib().rosetta_bsk_words(C.byref(_params(params)))


def version() -> str:
    """rosetta_version(): the version and the digest of the sources built."""
    return lib().rosetta_version().decode()


def ksk_words(params) -> int:
    return lib().rosetta_ksk_words(C.byref(_params(params)))


def ksk_device_words(params) -> int:
    return lib().rosetta_ksk_device_words(C.byref(_params(params)))


def check_params(params):
    _check(lib().rosetta_check_params(C.byref(_params(params))))


def bsk_prepare(bsk_std, params, out=None, stream=None):
    p = _params(params)
    _expect(bsk_std, "bsk_std", bsk_words(p))
    if out is None:
        out = empty(bsk_words(p), bsk_std.device)
    _expect(out, "bsk_dev", bsk_words(p))
    _check(lib().rosetta_bsk_prepare(_dev(bsk_std, "bsk_std"), _dev(out, "bsk_dev"), C.byref(p),
                                     _stream(stream)))
    return out


def ksk_prepare(ksk_std, params, out=None, stream=None):
    p = _params(params)
    _expect(ksk_std, "ksk_std", ksk_words(p))
    if out is None:
        out = empty(ksk_device_words(p), ksk_std.device)
    _expect(out, "ksk_dev", ksk_device_words(p))
    _check(lib().rosetta_ksk_prepare(_dev(ksk_std, "ksk_std"), _dev(out, "ksk_dev"), C.byref(p),
                                     _stream(stream)))
    return out


def _check_pbs_args(p, lwe_in, bsk_dev, ksk_dev, lut) -> int:
    """Sizes of the PBS inputs against the parameters; returns the batch."""
    batch = _batch_of(lwe_in, "lwe_in", p.n + 1)
    _expect(bsk_dev, "bsk_dev", bsk_words(p))
    _expect(ksk_dev, "ksk_dev", ksk_device_words(p))
    _expect(lut, "lut", p.N)
    return batch


def pbs_batch(lwe_in, bsk_dev, ksk_dev, lut, params, out=None, stream=None):
    p = _params(params)
    batch = _check_pbs_args(p, lwe_in, bsk_dev, ksk_dev, lut)
    if out is None:
        out = empty((batch, p.n + 1), lwe_in.device)
    _expect(out, "lwe_out", batch * (p.n + 1))
    _check(lib().rosetta_pbs_batch(_dev(lwe_in, "lwe_in"), _dev(bsk_dev, "bsk_dev"),
                                   _dev(ksk_dev, "ksk_dev"), _dev(lut, "lut"),
                                   _dev(out, "lwe_out"), batch, C.byref(p), _stream(stream)))
    return out


def pbs_workspace_bytes(params, batch: int) -> int:
    return lib().rosetta_pbs_workspace_bytes(C.byref(_params(params)), batch)


def pbs_batch_ws(lwe_in, bsk_dev, ksk_dev, lut, params, workspace, out=None, stream=None):
    p = _params(params)
    batch = _check_pbs_args(p, lwe_in, bsk_dev, ksk_dev, lut)
    if out is None:
        out = empty((batch, p.n + 1), lwe_in.device)
    _expect(out, "lwe_out", batch * (p.n + 1))
    if _words(workspace) * 8 < pbs_workspace_bytes(p, batch):
        raise ValueError(f"workspace holds {_words(workspace) * 8} bytes, the call needs "
                         f"{pbs_workspace_bytes(p, batch)}")
    _check(lib().rosetta_pbs_batch_ws(_dev(lwe_in, "lwe_in"), _dev(bsk_dev, "bsk_dev"),
                                      _dev(ksk_dev, "ksk_dev"), _dev(lut, "lut"),
                                      _dev(out, "lwe_out"), batch, C.byref(p),
                                      _dev(workspace, "workspace"),
                                      workspace.numel() * workspace.element_size(),
                                      _stream(stream)))
    return out


NOALLOC_SCRATCH_BYTES = 64 << 20


def pbs_batch_noalloc(lwe_in, bsk_dev, ksk_dev, lut, params, out, stream=None):
    """rosetta_pbs_batch_noalloc: the PBS with the library's static scratch
    (the caller passes the output buffer; nothing is allocated)."""
    p = _params(params)
    batch = _check_pbs_args(p, lwe_in, bsk_dev, ksk_dev, lut)
    _expect(out, "lwe_out", batch * (p.n + 1))
    _check(lib().rosetta_pbs_batch_noalloc(_dev(lwe_in, "lwe_in"), _dev(bsk_dev, "bsk_dev"),
                                           _dev(ksk_dev, "ksk_dev"), _dev(lut, "lut"),
                                           _dev(out, "lwe_out"), batch, C.byref(p),
                                           _stream(stream)))
    return out


def blind_rotate(lwe_in, bsk_dev, lut, params, out=None, stream=None):
    p = _params(params)
    batch = _batch_of(lwe_in, "lwe_in", p.n + 1)
    _expect(bsk_dev, "bsk_dev", bsk_words(p))
    _expect(lut, "lut", p.N)
    if out is None:
        out = empty((batch, 2 * p.N), lwe_in.device)
    _expect(out, "glwe_out", batch * 2 * p.N)
    _check(lib().rosetta_blind_rotate(_dev(lwe_in, "lwe_in"), _dev(bsk_dev, "bsk_dev"),
                                      _dev(lut, "lut"), _dev(out, "glwe_out"), batch, C.byref(p),
                                      _stream(stream)))
    return out


def blind_rotate_extract(lwe_in, bsk_dev, lut, params, out=None, stream=None):
    p = _params(params)
    batch = _batch_of(lwe_in, "lwe_in", p.n + 1)
    _expect(bsk_dev, "bsk_dev", bsk_words(p))
    _expect(lut, "lut", p.N)
    if out is None:
        out = empty((batch, p.N + 1), lwe_in.device)
    _expect(out, "big_out", batch * (p.N + 1))
    _check(lib().rosetta_blind_rotate_extract(_dev(lwe_in, "lwe_in"), _dev(bsk_dev, "bsk_dev"),
                                              _dev(lut, "lut"), _dev(out, "big_out"), batch,
                                              C.byref(p), _stream(stream)))
    return out


def keyswitch(big_in, ksk_dev, params, out=None, stream=None):
    p = _params(params)
    batch = _batch_of(big_in, "big_in", p.N + 1)
    _expect(ksk_dev, "ksk_dev", ksk_device_words(p))
    if out is None:
        out = empty((batch, p.n + 1), big_in.device)
    _expect(out, "lwe_out", batch * (p.n + 1))
    _check(lib().rosetta_keyswitch(_dev(big_in, "big_in"), _dev(ksk_dev, "ksk_dev"),
                                   _dev(out, "lwe_out"), batch, C.byref(p), _stream(stream)))
    return out


def ntt_forward(x, N: int, out=None, stream=None):
    count = _batch_of(x, "in", N)
    out = empty(x.shape, x.device) if out is None else out
    _expect(out, "out", count * N)
    _check(lib().rosetta_ntt_forward(_dev(x, "in"), _dev(out, "out"), count, N, _stream(stream)))
    return out


def ntt_inverse(x, N: int, out=None, stream=None):
    count = _batch_of(x, "in", N)
    out = empty(x.shape, x.device) if out is None else out
    _expect(out, "out", count * N)
    _check(lib().rosetta_ntt_inverse(_dev(x, "in"), _dev(out, "out"), count, N, _stream(stream)))
    return out


def poly_mul(a, b, N: int, out=None, stream=None):
    count = _batch_of(a, "a", N)
    _expect(b, "b", count * N)
    out = empty(a.shape, a.device) if out is None else out
    _expect(out, "c", count * N)
    _check(lib().rosetta_poly_mul(_dev(a, "a"), _dev(b, "b"), _dev(out, "c"), count, N,
                                  _stream(stream)))
    return out


FIELD_ADD, FIELD_SUB, FIELD_MUL, FIELD_MUL_ADD, FIELD_ADD_WEAK = 0, 1, 2, 3, 4
FIELD_MUL_ADD_WEAK, FIELD_MUL_POW2, FIELD_ROUND_TOP = 5, 256, 512


def field_op(op: int, a, b=None, c=None, out=None, stream=None):
    """Elementwise Goldilocks arithmetic with the kernels' device routines
    (op: FIELD_ADD, FIELD_SUB, FIELD_MUL, FIELD_MUL_ADD, FIELD_ADD_WEAK,
    FIELD_MUL_ADD_WEAK, FIELD_MUL_POW2 + e, FIELD_ROUND_TOP + s; the last
    returns int64 values as uint64)."""
    count = _words(a)
    for t, name in ((b, "b"), (c, "c")):
        if t is not None:
            _expect(t, name, count)
    out = empty(a.shape, a.device) if out is None else out
    _expect(out, "out", count)
    _check(lib().rosetta_field_op(op, _dev(a, "a"), None if b is None else _dev(b, "b"),
                                  None if c is None else _dev(c, "c"), _dev(out, "out"), count,
                                  _stream(stream)))
    return out


def modmul_chain(seed: int, threads: int, iters: int, out=None, stream=None):
    """Throughput probe: 8 register-resident product chains per thread
    (see rosetta_modmul_chain); returns out[threads]."""
    out = empty(threads) if out is None else out
    if _words(out) < threads:
        raise ValueError(f"out holds {_words(out)} words, the call needs {threads}")
    _check(lib().rosetta_modmul_chain(seed, threads, iters, _dev(out, "out"), _stream(stream)))
    return out


def shutdown():
    _check(lib().rosetta_shutdown())


# lookup-protocol primitives ------------------------------------------------

def blind_rotate_glwe(lwe_in, bsk_dev, glwe_tp, params, extract=False, group=1, out=None,
                      stream=None):
    """Blind rotation of GLWE test polynomials glwe_tp [batch*group][2N], each
    LWE selector of lwe_in [batch][n+1] serving `group` consecutive ones."""
    p = _params(params)
    batch = _batch_of(lwe_in, "lwe_in", p.n + 1)
    _expect(bsk_dev, "bsk_dev", bsk_words(p))
    _expect(glwe_tp, "glwe_tp", batch * group * 2 * p.N)
    shape = (batch * group, p.N + 1) if extract else (batch * group, 2 * p.N)
    if out is None:
        out = empty(shape, lwe_in.device)
    _expect(out, "out", shape[0] * shape[1])
    _check(lib().rosetta_blind_rotate_glwe(_dev(lwe_in, "lwe_in"), _dev(bsk_dev, "bsk_dev"),
                                           _dev(glwe_tp, "glwe_tp"), _dev(out, "out"), batch,
                                           group, C.byref(p), 1 if extract else 0,
                                           _stream(stream)))
    return out


def lwe_add_consts(lwe_in, consts, dim: int, out=None, stream=None):
    """out[q][j] = lwe_in[q] + (0, .., 0, consts[j])."""
    batch = _batch_of(lwe_in, "lwe_in", dim + 1)
    c = np.ascontiguousarray(consts, dtype=np.uint64)
    if out is None:
        out = empty((batch, c.size, dim + 1), lwe_in.device)
    _expect(out, "lwe_out", batch * c.size * (dim + 1))
    _check(lib().rosetta_lwe_add_consts(_dev(lwe_in, "lwe_in"), _np_ptr(c), _dev(out, "lwe_out"),
                                        batch, c.size, dim, _stream(stream)))
    return out


def lwe_sum_groups(lwe_in, count: int, dim: int, c0: int = 0, out=None, stream=None):
    """out[q] = sum_j lwe_in[q][j] + (0, .., 0, c0)."""
    batch = _batch_of(lwe_in, "lwe_in", (dim + 1) * count)
    if out is None:
        out = empty((batch, dim + 1), lwe_in.device)
    _expect(out, "lwe_out", batch * (dim + 1))
    _check(lib().rosetta_lwe_sum_groups(_dev(lwe_in, "lwe_in"), c0, _dev(out, "lwe_out"), batch,
                                        count, dim, _stream(stream)))
    return out


def lwe_combine(a, alpha: int, b=None, beta: int = 0, c=None, gamma: int = 0, out=None,
                stream=None):
    """out = alpha a + beta b + gamma c mod p, word by word (b, c optional)."""
    words = _words(a)
    for t, name in ((b, "b"), (c, "c")):
        if t is not None:
            _expect(t, name, words)
    out = empty(a.shape, a.device) if out is None else out
    _expect(out, "out", words)
    _check(lib().rosetta_lwe_combine(_dev(a, "a"), alpha, None if b is None else _dev(b, "b"),
                                     beta, None if c is None else _dev(c, "c"), gamma,
                                     _dev(out, "out"), words, _stream(stream)))
    return out


def autk_words(params, level: int) -> int:
    return lib().rosetta_autk_words(C.byref(_params(params)), level)


def autk_prepare(autk_std, params, level: int, out=None, stream=None):
    p = _params(params)
    _expect(autk_std, "autk_std", autk_words(p, level))
    if out is None:
        out = empty(autk_words(p, level), autk_std.device)
    _expect(out, "autk_dev", autk_words(p, level))
    _check(lib().rosetta_autk_prepare(_dev(autk_std, "autk_std"), _dev(out, "autk_dev"),
                                      C.byref(p), level, _stream(stream)))
    return out


def trace(glwe_in, autk_dev, params, level: int, base_log: int, out=None, stream=None):
    p = _params(params)
    batch = _batch_of(glwe_in, "glwe_in", 2 * p.N)
    _expect(autk_dev, "autk_dev", autk_words(p, level))
    if out is None:
        out = empty((batch, 2 * p.N), glwe_in.device)
    _expect(out, "glwe_out", batch * 2 * p.N)
    _check(lib().rosetta_trace(_dev(glwe_in, "glwe_in"), _dev(autk_dev, "autk_dev"),
                               _dev(out, "glwe_out"), batch, C.byref(p), level, base_log,
                               _stream(stream)))
    return out


def plain_prepare(plain, N: int, out=None, stream=None):
    count = _batch_of(plain, "plain", N)
    out = empty(plain.shape, plain.device) if out is None else out
    _expect(out, "plain_prep", count * N)
    _check(lib().rosetta_plain_prepare(_dev(plain, "plain"), _dev(out, "plain_prep"), count, N,
                                       _stream(stream)))
    return out


def glwe_mul_plain(glwe_in, pa_prep, pb, N: int, out=None, stream=None):
    """out[q][s] = pa_s * glwe_in[q] + (0, pb_s); pb may be None."""
    batch = _batch_of(glwe_in, "glwe_in", 2 * N)
    npoly = _batch_of(pa_prep, "pa_prep", N)
    if pb is not None:
        _expect(pb, "pb", npoly * N)
    if out is None:
        out = empty((batch, npoly, 2 * N), glwe_in.device)
    _expect(out, "glwe_out", batch * npoly * 2 * N)
    _check(lib().rosetta_glwe_mul_plain(_dev(glwe_in, "glwe_in"), _dev(pa_prep, "pa_prep"),
                                        None if pb is None else _dev(pb, "pb"),
                                        _dev(out, "glwe_out"), batch, npoly, N, _stream(stream)))
    return out


def _exps(exps, count):
    if exps is None:
        return None, None
    e = np.ascontiguousarray(exps, dtype=np.uint32)
    if e.size != count:
        raise ValueError("need one exponent per ciphertext")
    return e, _np_ptr(e)


def glwe_recombine(glwe_in, count: int, N: int, exps=None, out=None, stream=None):
    """out[q] = sum_s X^(exps[s]) glwe_in[q][s] (exps None: X^s)."""
    batch = _batch_of(glwe_in, "glwe_in", 2 * N * count)
    if out is None:
        out = empty((batch, 2 * N), glwe_in.device)
    _expect(out, "glwe_out", batch * 2 * N)
    e, ep = _exps(exps, count)
    _check(lib().rosetta_glwe_recombine(_dev(glwe_in, "glwe_in"), ep, _dev(out, "glwe_out"),
                                        batch, count, N, _stream(stream)))
    return out


def glwe_monomial_mul(glwe_in, exps, N: int, out=None, stream=None):
    """out[q][s] = X^(exps[s]) glwe_in[q]."""
    batch = _batch_of(glwe_in, "glwe_in", 2 * N)
    e, ep = _exps(exps, len(exps))
    if out is None:
        out = empty((batch, e.size, 2 * N), glwe_in.device)
    _expect(out, "glwe_out", batch * e.size * 2 * N)
    _check(lib().rosetta_glwe_monomial_mul(_dev(glwe_in, "glwe_in"), ep, _dev(out, "glwe_out"),
                                           batch, e.size, N, _stream(stream)))
    return out


def sample_extract(glwe_in, N: int, out=None, stream=None):
    batch = _batch_of(glwe_in, "glwe_in", 2 * N)
    if out is None:
        out = empty((batch, N + 1), glwe_in.device)
    _expect(out, "big_out", batch * (N + 1))
    _check(lib().rosetta_sample_extract(_dev(glwe_in, "glwe_in"), _dev(out, "big_out"), batch, N,
                                        _stream(stream)))
    return out


# --------------------------------------------------------------------------
# host helpers (numpy)
# --------------------------------------------------------------------------

def _np_ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def keygen(seed: int, params, sigma_lwe: float, sigma_glwe: float) -> dict:
    p = _params(params)
    keys = dict(lwe_key=np.zeros(p.n, np.uint64), glwe_key=np.zeros(p.N, np.uint64),
                bsk=np.zeros(bsk_words(p), np.uint64), ksk=np.zeros(ksk_words(p), np.uint64))
    _check(lib().rosetta_keygen(seed, C.byref(p), sigma_lwe, sigma_glwe,
                                _np_ptr(keys["lwe_key"]), _np_ptr(keys["glwe_key"]),
                                _np_ptr(keys["bsk"]), _np_ptr(keys["ksk"])))
    return keys


def lwe_encrypt(seed: int, params, sigma: float, key: np.ndarray, msgs) -> np.ndarray:
    p = _params(params)
    key = np.ascontiguousarray(key, np.uint64)
    msgs = np.ascontiguousarray(msgs, np.uint32)
    dim = key.shape[0]
    out = np.zeros((msgs.shape[0], dim + 1), np.uint64)
    _check(lib().rosetta_lwe_encrypt(seed, C.byref(p), sigma, _np_ptr(key), dim, _np_ptr(msgs),
                                     msgs.shape[0], _np_ptr(out)))
    return out


def lwe_encrypt_plain(seed: int, params, sigma: float, key: np.ndarray, plain) -> np.ndarray:
    """LWE encryptions of plaintexts already in Z_p (params unused beyond
    symmetry with lwe_encrypt)."""
    key = np.ascontiguousarray(key, np.uint64)
    plain = np.ascontiguousarray(plain, np.uint64)
    dim = key.shape[0]
    out = np.zeros((plain.shape[0], dim + 1), np.uint64)
    _check(lib().rosetta_lwe_encrypt_plain(seed, sigma, _np_ptr(key), dim, _np_ptr(plain),
                                           plain.shape[0], _np_ptr(out)))
    return out


def lwe_decrypt(params, key: np.ndarray, cts: np.ndarray) -> np.ndarray:
    p = _params(params)
    key = np.ascontiguousarray(key, np.uint64)
    dim = key.shape[0]
    cts = np.ascontiguousarray(cts, np.uint64).reshape(-1, dim + 1)
    out = np.zeros(cts.shape[0], np.uint32)
    _check(lib().rosetta_lwe_decrypt(C.byref(p), _np_ptr(key), dim, _np_ptr(cts), cts.shape[0],
                                     _np_ptr(out)))
    return out


def lut_build(params, table) -> np.ndarray:
    p = _params(params)
    table = np.ascontiguousarray(table, np.uint32)
    if table.shape[0] != p.M:
        raise ValueError(f"table must have {p.M} entries")
    v = np.zeros(p.N, np.uint64)
    _check(lib().rosetta_lut_build(C.byref(p), _np_ptr(table), _np_ptr(v)))
    return v


def glwe_encrypt(seed: int, params, sigma: float, glwe_key: np.ndarray, msgs) -> np.ndarray:
    p = _params(params)
    key = np.ascontiguousarray(glwe_key, np.uint64)
    msgs = np.ascontiguousarray(msgs, np.uint64).reshape(-1, p.N)
    out = np.zeros((msgs.shape[0], 2 * p.N), np.uint64)
    _check(lib().rosetta_glwe_encrypt(seed, C.byref(p), sigma, _np_ptr(key), _np_ptr(msgs),
                                      msgs.shape[0], _np_ptr(out)))
    return out


def glwe_phase(params, glwe_key: np.ndarray, cts) -> np.ndarray:
    p = _params(params)
    key = np.ascontiguousarray(glwe_key, np.uint64)
    cts = np.ascontiguousarray(cts, np.uint64).reshape(-1, 2 * p.N)
    out = np.zeros((cts.shape[0], p.N), np.uint64)
    _check(lib().rosetta_glwe_phase(C.byref(p), _np_ptr(key), _np_ptr(cts), cts.shape[0],
                                    _np_ptr(out)))
    return out


def autk_keygen(seed: int, params, level: int, base_log: int, sigma: float,
                glwe_key: np.ndarray) -> np.ndarray:
    p = _params(params)
    key = np.ascontiguousarray(glwe_key, np.uint64)
    out = np.zeros(autk_words(p, level), np.uint64)
    _check(lib().rosetta_autk_keygen(seed, C.byref(p), level, base_log, sigma, _np_ptr(key),
                                     _np_ptr(out)))
    return out


# segmented LUT (host) --------------------------------------------------------

def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def seglut_boundaries(lo: float, hi: float, nseg: int, spacing: str) -> np.ndarray:
    tau = np.zeros(nseg + 1, np.float64)
    _check(lib().rosetta_seglut_boundaries(lo, hi, nseg, SPACINGS[spacing], _np_ptr(tau)))
    return tau


def seglut_build(function: str, tau, nbr: int, fit: str = "linear"):
    tau = _f64(tau)
    nseg = tau.shape[0] - 1
    a = np.zeros((nseg, nbr), np.float64)
    b = np.zeros((nseg, nbr), np.float64)
    _check(lib().rosetta_seglut_build(FUNCTIONS[function], _np_ptr(tau), nseg, nbr, FITS[fit],
                                      _np_ptr(a), _np_ptr(b)))
    return a, b


def seglut_protocol_polys(tau, nbr: int):
    tau = _f64(tau)
    nseg = tau.shape[0] - 1
    p = np.zeros(nseg, np.float64)
    q = np.zeros(nseg, np.float64)
    _check(lib().rosetta_seglut_protocol_polys(_np_ptr(tau), nseg, nbr, _np_ptr(p), _np_ptr(q)))
    return p, q


def _offsets(index_offset, count):
    if index_offset is None:
        return None, None
    off = np.ascontiguousarray(index_offset, dtype=np.int32)
    if off.size != count:
        raise ValueError("index_offset must have one entry per input")
    return off, _np_ptr(off)


def seglut_eval(tau, a, b, x, index_offset=None) -> np.ndarray:
    tau, a, b, x = _f64(tau), _f64(a), _f64(b), _f64(x)
    y = np.zeros_like(x)
    off, off_p = _offsets(index_offset, x.size)
    _check(lib().rosetta_seglut_eval(_np_ptr(tau), tau.shape[0] - 1, a.shape[1], _np_ptr(a),
                                     _np_ptr(b), _np_ptr(x), off_p, x.size, _np_ptr(y)))
    return y


def seglut_precision(function: str, tau, a, b, x, index_offset=None) -> float:
    tau, a, b, x = _f64(tau), _f64(a), _f64(b), _f64(x)
    bits = np.zeros(1, np.float64)
    off, off_p = _offsets(index_offset, x.size)
    _check(lib().rosetta_seglut_precision(FUNCTIONS[function], _np_ptr(tau), tau.shape[0] - 1,
                                          a.shape[1], _np_ptr(a), _np_ptr(b), _np_ptr(x), off_p,
                                          x.size, _np_ptr(bits)))
    return float(bits[0])


def encode_fixed(v, scale_log: int) -> np.ndarray:
    v = _f64(v)
    out = np.zeros(v.shape, np.uint64)
    _check(lib().rosetta_encode_fixed(_np_ptr(v), v.size, scale_log, _np_ptr(out)))
    return out


# lookup protocol (Algorithm 1, Steps 1-3) ----------------------------------

def lookup_encode(params, lp: LookupParams, tau, a, b):
    """Host plaintext block [(4 + 2 nseg) N] and constants [nseg]."""
    p = _params(params)
    tau, a, b = _f64(tau), _f64(a), _f64(b)
    plain = np.zeros(lib().rosetta_lookup_plain_words(C.byref(p), C.byref(lp)), np.uint64)
    consts = np.zeros(lp.nseg, np.uint64)
    _check(lib().rosetta_lookup_encode(C.byref(p), C.byref(lp), _np_ptr(tau), _np_ptr(a),
                                       _np_ptr(b), _np_ptr(plain), _np_ptr(consts)))
    return plain, consts


def lookup_prepare(plain_dev, params, lp: LookupParams, out=None, stream=None):
    p = _params(params)
    _expect(plain_dev, "plain", lib().rosetta_lookup_plain_words(C.byref(p), C.byref(lp)))
    out = empty(plain_dev.shape, plain_dev.device) if out is None else out
    _expect(out, "plain_prep", _words(plain_dev))
    _check(lib().rosetta_lookup_prepare(_dev(plain_dev, "plain"), _dev(out, "plain_prep"),
                                        C.byref(p), C.byref(lp), _stream(stream)))
    return out


def lookup_workspace_bytes(params, lp: LookupParams, batch: int) -> int:
    return lib().rosetta_lookup_workspace_bytes(C.byref(_params(params)), C.byref(lp), batch)


LOOKUP_PART_CMP, LOOKUP_PART_S, LOOKUP_PART_I = 2, 3, 6


def lookup_workspace_offset(params, lp: LookupParams, batch: int, part: int) -> int:
    """Word offset of an intermediate of rosetta_lookup_eval in its workspace
    (LOOKUP_PART_CMP, LOOKUP_PART_S or LOOKUP_PART_I)."""
    off = lib().rosetta_lookup_workspace_offset(C.byref(_params(params)), C.byref(lp), batch,
                                                part)
    if off == (1 << 64) - 1:
        raise ValueError(f"unknown lookup workspace part {part}")
    return off


def lookup_eval(x_rlwe, x_cmp, bsk_dev, ksk_dev, autk_dev, plain_prep, consts, params,
                lp: LookupParams, workspace=None, out=None, stream=None):
    p = _params(params)
    batch = _batch_of(x_cmp, "x_cmp", p.n + 1)
    _expect(x_rlwe, "x_rlwe", batch * 2 * p.N)
    _expect(bsk_dev, "bsk_dev", bsk_words(p))
    _expect(ksk_dev, "ksk_dev", ksk_device_words(p))
    _expect(autk_dev, "autk_dev", autk_words(p, lp.trace_level))
    _expect(plain_prep, "plain_prep", lib().rosetta_lookup_plain_words(C.byref(p), C.byref(lp)))
    if out is None:
        out = empty((batch, 2 * p.N), x_cmp.device)
    _expect(out, "out", batch * 2 * p.N)
    if workspace is None:
        workspace = empty(lookup_workspace_bytes(p, lp, batch) // 8, x_cmp.device)
    if _words(workspace) * 8 < lookup_workspace_bytes(p, lp, batch):
        raise ValueError(f"workspace holds {_words(workspace) * 8} bytes, the call needs "
                         f"{lookup_workspace_bytes(p, lp, batch)}")
    c = np.ascontiguousarray(consts, np.uint64)
    _expect(c, "consts", lp.nseg)
    _check(lib().rosetta_lookup_eval(_dev(x_rlwe, "x_rlwe"), _dev(x_cmp, "x_cmp"),
                                     _dev(bsk_dev, "bsk"), _dev(ksk_dev, "ksk"),
                                     _dev(autk_dev, "autk"), _dev(plain_prep, "plain_prep"),
                                     _np_ptr(c), _dev(out, "out"), batch, C.byref(p),
                                     C.byref(lp), _dev(workspace, "workspace"),
                                     workspace.numel() * 8, _stream(stream)))
    return out
