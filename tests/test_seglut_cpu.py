"""The library's segmented-LUT builder and cleartext simulator (host code,
through the C ABI) against the cleartext oracle (oracle/seglut.py) and the
paper's running example (Sec. 3.1, tests/golden/paper_lookup_example.json).
Floating point on both sides in double precision: the same formulas in a
different order of evaluation, compared to 1e-12 relative."""
import json
import os

import numpy as np
import pytest

from oracle import seglut as G
from paper_2609_16915_amd import rosetta as R

HERE = os.path.dirname(os.path.abspath(__file__))
EX = json.load(open(os.path.join(HERE, "golden", "paper_lookup_example.json")))
P = 0xFFFFFFFF00000001
CASES = [("inv", 0.01, 10.0, "log"), ("inv", 0.01, 100.0, "log"),
         ("inv_sqrt", 0.01, 10.0, "log"), ("inv_sqrt", 0.01, 100.0, "log"),
         ("silu", -20.0, 20.0, "uniform"), ("gelu", -20.0, 20.0, "uniform"),
         ("exp", -16.0, 0.0, "uniform")]


def close(a, b, rel=1e-12):
    a, b = np.asarray(a), np.asarray(b)
    return np.all(np.abs(a - b) <= rel * np.maximum(1.0, np.abs(b)))


@pytest.mark.parametrize("name,lo,hi,spacing", CASES)
@pytest.mark.parametrize("nbr", [4, 64])
def test_builder_matches_oracle(name, lo, hi, spacing, nbr):
    tau = R.seglut_boundaries(lo, hi, 4, spacing)
    assert close(tau, G.boundaries(lo, hi, 4, spacing))
    for fit in ("linear", "constant"):
        a, b = R.seglut_build(name, tau, nbr, fit)
        ea, eb = G.build(G.FUNCTIONS[name], tau, nbr, fit)
        assert close(a, ea, 1e-9) and close(b, eb, 1e-9)
    a, b = R.seglut_build(name, tau, nbr)
    p, q = R.seglut_protocol_polys(tau, nbr)
    ep, eq, _, _ = G.protocol_polys(tau, a, b)
    assert close(p, ep) and close(q, eq)
    xs = np.random.default_rng(1).uniform(lo, hi, 5000)
    xs[:3] = [lo, hi, tau[2]]
    assert close(R.seglut_eval(tau, a, b, xs), G.evaluate(xs, tau, a, b), 1e-9)
    bits = R.seglut_precision(name, tau, a, b, xs)
    assert abs(bits - G.precision_bits(G.FUNCTIONS[name], tau, a, b, xs)) < 1e-6


def test_running_example_through_the_library():
    t = EX["two_segment_linear"]
    a, b = R.seglut_build("inv", EX["segments"], EX["n_br"])
    assert abs(a[0, 1] - t["a_01"]) <= 5e-4 and abs(b[0, 1] - t["b_01"]) <= 5e-4
    y = R.seglut_eval(EX["segments"], a, b, [EX["x"]])[0]
    assert abs(y - t["value_at_x"]) <= 5e-4
    p, q = R.seglut_protocol_polys(EX["segments"], EX["n_br"])
    assert np.allclose(p, EX["protocol"]["p_hat"], atol=5e-4)
    assert np.allclose(q, EX["protocol"]["q_hat"], atol=5e-4)
    _, b1 = R.seglut_build("inv", EX["domain"], EX["n_br"], "constant")
    assert abs(b1[0, 0] - EX["single_lut"]["first_entry"]) <= 5e-4


def test_encode_fixed():
    v = np.array([0.0, 1.0, -1.0, 2.5, -0.75, 4.571428])
    got = R.encode_fixed(v, 20)
    want = [int(round(x * 2 ** 20)) % P for x in v]
    assert [int(x) for x in got] == want
    with pytest.raises(R.RosettaError):
        R.encode_fixed([2.0 ** 10], 60)


def test_validation():
    with pytest.raises(R.RosettaError):
        R.seglut_boundaries(0.0, 1.0, 4, "log")
    with pytest.raises(R.RosettaError):
        R.seglut_build("inv", [0.5, 0.4, 1.0], 4)
    with pytest.raises(R.RosettaError):
        R.seglut_boundaries(1.0, 1.0, 2, "uniform")


PAPER_PRECISION = {   # Sec. 5, primitive tables ("Ours", precision in bits)
    ("inv", 0.01, 10.0): 12.7, ("inv", 0.01, 100.0): 12.5,
    ("inv_sqrt", 0.01, 10.0): 16.7, ("inv_sqrt", 0.01, 100.0): 12.7,
    ("silu", -20.0, 20.0): 16.8, ("gelu", -20.0, 20.0): 15.5}


@pytest.mark.parametrize("name,lo,hi,spacing", CASES[:6])
def test_precision_with_index_offsets_matches_oracle(name, lo, hi, spacing):
    """Offsets drawn once (Gaussian, rounded) and given to both sides; the
    noise-free cleartext precision at N_br = 2048 is an upper bound of the
    paper's encrypted figure, and index errors of a few intervals bring the
    simulator down to it."""
    tau = R.seglut_boundaries(lo, hi, 4, spacing)
    a, b = R.seglut_build(name, tau, 2048)
    rng = np.random.default_rng(2)
    xs = rng.uniform(lo, hi, 20000)
    clean = R.seglut_precision(name, tau, a, b, xs)
    assert abs(clean - G.precision_bits(G.FUNCTIONS[name], tau, a, b, xs)) < 1e-6
    assert clean > PAPER_PRECISION[(name, lo, hi)]
    off = np.rint(rng.normal(0.0, 3.0, xs.size)).astype(np.int32)
    noisy = R.seglut_precision(name, tau, a, b, xs, off)
    assert abs(noisy - G.precision_bits(G.FUNCTIONS[name], tau, a, b, xs, off)) < 1e-6
    assert np.allclose(R.seglut_eval(tau, a, b, xs, off), G.evaluate(xs, tau, a, b, off),
                       rtol=1e-9, atol=1e-12)
    assert noisy < clean
