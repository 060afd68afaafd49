"""The lookup pipeline's host side (library encoder against the oracle's
independent encoder) and the oracle pipeline's semantics: decrypting its
output gives the segmented LUT's value f~(x) (Sec. 3.1-3.2) up to the
noise and selection error of the parameters."""
import math

import numpy as np
import pytest

from oracle import lookup as OL
from oracle import oracle as O
from oracle import seglut as G
from paper_2609_16915_amd import rosetta as R

P = O.P
# A small ring with a precise key switch, for semantic checks on the CPU.
SMALL = dict(n=64, k=1, N=256, pbs_level=3, pbs_base_log=8, ks_level=4, ks_base_log=5,
             msg_bits=2)
SIG = 2.0 ** -40


def lookup_params(N, nseg=4, margin=16, sc=58, tl=4, tb=12, sx=44, sv=16, refine=0):
    """sx + sp = 63 - log2 N (one unit of t per rotation step); values at
    2^(sx+sv)."""
    sp = 63 - int(math.log2(N)) - sx
    return R.LookupParams(nseg=nseg, nbr=N - 2 * margin, margin=margin, x_scale_log=sx,
                          coef_scale_log=sp, val_scale_log=sv, cmp_scale_log=sc,
                          trace_level=tl, trace_base_log=tb, cmp_refine_log=refine)


@pytest.mark.parametrize("N,fn,lo,hi,spacing,refine", [
    (256, "inv", 1.0, 16.0, "log", 0), (2048, "silu", -20.0, 20.0, "uniform", 0),
    (2048, "inv", 0.01, 10.0, "log", 0), (512, "gelu", -8.0, 8.0, "uniform", 0),
    (256, "inv", 1.0, 16.0, "log", 2), (2048, "silu", -20.0, 20.0, "uniform", 5),
    (4096, "inv_sqrt", 0.01, 100.0, "log", 6), (1024, "gelu", -8.0, 8.0, "uniform", 1)])
def test_encoder_matches_oracle(N, fn, lo, hi, spacing, refine):
    lp = lookup_params(N, sc=56 if N >= 2048 else 58, sx=40 if N >= 2048 else 44,
                       sv=18 if N >= 2048 else 16, refine=refine)
    prm = dict(SMALL, N=N)
    tau = R.seglut_boundaries(lo, hi, lp.nseg, spacing)
    a, b = R.seglut_build(fn, tau, lp.nbr)
    plain, consts = R.lookup_encode(prm, lp, tau, a, b)
    parts = OL.encode(N, lp.nseg, lp.nbr, lp.margin, lp.x_scale_log, lp.coef_scale_log,
                      lp.val_scale_log, lp.cmp_scale_log, tau, a, b, refine=refine)
    assert plain.size == (4 + 2 * lp.nseg + (2 if refine else 0)) * N
    assert np.array_equal(plain, OL.block(parts))
    assert np.array_equal(consts, parts["consts"])


def test_encoder_validation():
    prm = dict(SMALL)
    lp = lookup_params(256)
    tau = R.seglut_boundaries(1.0, 16.0, 4, "log")
    a, b = R.seglut_build("inv", tau, lp.nbr)
    for field, bad in (("nseg", 3), ("nbr", 250), ("x_scale_log", 41), ("trace_level", 5),
                       ("val_scale_log", 19), ("cmp_refine_log", 7)):
        lp2 = lookup_params(256)
        setattr(lp2, field, bad)
        with pytest.raises(R.RosettaError):
            R.lookup_encode(prm, lp2, tau, a, b)


def small_setup(O, fn="inv", lo=1.0, hi=16.0, spacing="log", seed=5):
    op = O.Params.make(**{k: v for k, v in SMALL.items() if k != "k"})
    ks = O.KeySet(op, seed, SIG, SIG)
    lp = lookup_params(256, margin=64)
    autk = O.autk_keygen(seed + 1, 256, lp.trace_level, lp.trace_base_log, SIG, ks.glwe_key)
    tau = G.boundaries(lo, hi, lp.nseg, spacing)
    A, B = G.build(G.FUNCTIONS[fn], tau, lp.nbr)
    parts = OL.encode(256, lp.nseg, lp.nbr, lp.margin, lp.x_scale_log, lp.coef_scale_log,
                      lp.val_scale_log, lp.cmp_scale_log, tau, A, B)
    return op, ks, lp, autk, tau, A, B, parts


def encrypt_inputs(O, op, ks, lp, xs, seed):
    N = op.N
    m = np.zeros((len(xs), N), np.uint64)
    m[:, 0] = [OL.enc(x, lp.x_scale_log) for x in xs]
    x_rlwe = O.glwe_encrypt(seed, SIG, ks.glwe_key, m)
    x_cmp = O.lwe_encrypt_plain(seed + 1, SIG, ks.lwe_key,
                                np.array([OL.enc(x, lp.cmp_scale_log) for x in xs], np.uint64))
    return x_rlwe, x_cmp


def decode(O, key, ct, scale):
    ph = O.glwe_phase(key, ct)
    c = int(ph[0])
    c = c if c <= P // 2 else c - P
    rest = [int(v) if int(v) <= P // 2 else int(v) - P for v in ph[1:]]
    return c / 2.0 ** scale, max(abs(v) for v in rest) / 2.0 ** scale


def test_oracle_pipeline_decrypts_to_the_segmented_lut(O):
    """Steps 1-3 on encryptions of 12 inputs (1/x on [1, 16], 4 log-spaced
    segments, 128 intervals each, margins of 64): the output decrypts to f~(x) within
    2e-3 and every other coefficient to 0 within 1e-4; the intermediate
    segment index decrypts to the true segment away from the boundaries."""
    op, ks, lp, autk, tau, A, B, parts = small_setup(O)
    xs = np.array([1.05, 1.5, 2.5, 3.3, 4.4, 5.0, 6.9, 8.5, 10.0, 12.3, 14.0, 15.5])
    x_rlwe, x_cmp = encrypt_inputs(O, op, ks, lp, xs, 40)
    out, st = OL.evaluate(op, ks, autk, lp.trace_level, lp.trace_base_log, parts, lp.nseg,
                          x_rlwe, x_cmp, want_steps=True)
    scale = lp.x_scale_log + lp.val_scale_log
    want = G.evaluate(xs, tau, A, B)
    for q, x in enumerate(xs):
        v, rest = decode(O, ks.glwe_key, out[q], scale)
        assert abs(v - want[q]) < 5e-4, (x, v, want[q])
        assert rest < 1e-4
        s_phase = int(O.lwe_phase(ks.lwe_key, st["S"][q:q + 1])[0])
        s_phase = s_phase if s_phase <= P // 2 else s_phase - P
        assert round(s_phase / (P / (2 * lp.nseg))) == int(G.segment_index(x, tau))


def test_lookup_eval_validation_touches_no_device():
    """Argument checks of the pipeline entry point run on the host before
    anything is enqueued."""
    import ctypes as C
    L = R.lib()
    p = R.Params.from_dict(SMALL)
    lp = lookup_params(256, margin=64)
    fake = 1 << 40
    consts = (C.c_uint64 * 4)()
    ws = L.rosetta_lookup_workspace_bytes(C.byref(p), C.byref(lp), 3)
    assert ws > 0
    args = [fake, fake + 10 ** 8, fake + 2 * 10 ** 8, fake + 3 * 10 ** 8, fake + 4 * 10 ** 8,
            fake + 5 * 10 ** 8, C.addressof(consts), fake + 6 * 10 ** 8, 3, C.byref(p), C.byref(lp),
            fake + 7 * 10 ** 8, ws, None]
    # empty batch: no-op
    a = list(args); a[8] = 0
    assert L.rosetta_lookup_eval(*a) == 0
    # NULL input, too small a workspace, output overlapping the workspace
    a = list(args); a[0] = None
    assert L.rosetta_lookup_eval(*a) == 1
    a = list(args); a[12] = ws - 8
    assert L.rosetta_lookup_eval(*a) == 7
    a = list(args); a[7] = a[11] + 64
    assert L.rosetta_lookup_eval(*a) == 4
    # invalid lookup parameters
    bad = lookup_params(256, margin=64)
    bad.nseg = 3
    a = list(args); a[10] = C.byref(bad)
    assert L.rosetta_lookup_eval(*a) == 2
