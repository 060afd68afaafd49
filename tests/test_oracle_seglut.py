"""Pins of the cleartext segmented-LUT oracle (oracle/seglut.py) against the
numbers the paper prints for its running example (Sec. 3.1 and Sec. 3.2;
tests/golden/paper_lookup_example.json), plus closed forms."""
import json
import math
import os

import numpy as np
import pytest

from oracle import seglut as G

HERE = os.path.dirname(os.path.abspath(__file__))
EX = json.load(open(os.path.join(HERE, "golden", "paper_lookup_example.json")))
F = G.FUNCTIONS["inv"]


def printed(value, ref):
    """value agrees with a printed decimal `ref` to its last printed digit."""
    s = repr(float(ref))
    decimals = len(s.split(".")[1]) if "." in s else 0
    return abs(value - ref) <= 0.5 * 10 ** (-decimals) + 1e-12


def test_single_lut_baseline():
    s = EX["single_lut"]
    taus = EX["domain"]
    A, B = G.build(F, taus, EX["n_br"], "constant")
    lo, hi = s["first_interval"]
    assert printed(taus[0] + (taus[1] - taus[0]) / EX["n_br"], hi)
    assert printed((lo + hi) / 2, s["first_midpoint"])
    assert printed(B[0, 0], s["first_entry"])
    S = G.segment_index(EX["x"], taus)
    assert int(G.interval_index(EX["x"], taus, S, EX["n_br"])) == s["index_of_x"]
    assert printed(F(EX["x"]), s["exact_at_x"])
    y = float(G.evaluate(EX["x"], taus, A, B))
    assert printed(abs(y - F(EX["x"])) / F(EX["x"]), s["relative_error_at_x"])
    assert printed(G.max_relative_error(F, taus, A, B), s["max_relative_error"])


def test_two_segments():
    taus = EX["segments"]
    Ac, Bc = G.build(F, taus, EX["n_br"], "constant")
    assert printed(G.max_relative_error(F, taus, Ac, Bc),
                   EX["two_segment_constant_max_relative_error"])
    t = EX["two_segment_linear"]
    A, B = G.build(F, taus, EX["n_br"], "linear")
    S = int(G.segment_index(EX["x"], taus))
    I = int(G.interval_index(EX["x"], taus, S, EX["n_br"]))
    assert (S, I) == (t["segment_of_x"], t["interval_of_x"])
    assert printed(A[0, 1], t["a_01"]) and printed(B[0, 1], t["b_01"])
    y = float(G.evaluate(EX["x"], taus, A, B))
    assert printed(y, t["value_at_x"])
    assert printed(abs(y - F(EX["x"])) / F(EX["x"]), t["relative_error_at_x"])
    assert printed(G.max_relative_error(F, taus, A, B), t["max_relative_error"])


def test_protocol_polynomials_and_candidates():
    pr = EX["protocol"]
    taus = EX["segments"]
    A, B = G.build(F, taus, EX["n_br"], "linear")
    p, q, a, b = G.protocol_polys(taus, A, B)
    x = EX["x"]
    assert all(printed(u, v) for u, v in zip(p, pr["p_hat"]))
    assert all(printed(u, v) for u, v in zip(q, pr["q_hat"]))
    assert all(printed(u, v) for u, v in zip(p * x + q, pr["t"]))
    assert all(printed(u, v) for u, v in zip(a[0], pr["a_hat_0"]))
    assert all(printed(u, v) for u, v in zip(b[0], pr["b_hat_0"]))
    assert all(printed(u, v) for u, v in zip(a[0] * x + b[0], pr["r_0"]))
    assert all(printed(u, v) for u, v in zip(a[1] * x + b[1], pr["r_1"]))
    S = int(G.segment_index(x, taus))
    I = int(math.floor((p * x + q)[S]))            # Step 2: select t[S], round down
    assert printed((a[S] * x + b[S])[I], pr["result"])


def test_chebyshev_fit_is_exact_on_lines_and_interpolates():
    """A line is reproduced exactly; for any f the fit agrees with f at both
    nodes; the error of linear interpolation at Chebyshev nodes is at most
    max|f''| r^2 / 4 on an interval of half-width r (r^2 (1/2 + cos^2) / 2 bound)."""
    a, b = G.chebyshev_linear(lambda x: 3.0 * x - 2.0, 0.3, 0.9)
    assert abs(a - 3.0) < 1e-12 and abs(b + 2.0) < 1e-12
    lo, hi = 1.0, 1.5
    a, b = G.chebyshev_linear(F, lo, hi)
    c, r = (lo + hi) / 2, (hi - lo) / 2
    for x in (c - r / math.sqrt(2), c + r / math.sqrt(2)):
        assert abs(a * x + b - F(x)) < 1e-12
    xs = np.linspace(lo, hi, 1001)
    fpp = 2.0 / lo ** 3
    assert np.max(np.abs(a * xs + b - F(xs))) <= fpp * r * r / 4 + 1e-12


def test_boundaries():
    t = G.boundaries(0.01, 100.0, 4, "log")
    assert np.allclose(t, [0.01, 0.1, 1.0, 10.0, 100.0])
    t = G.boundaries(-20.0, 20.0, 4, "uniform")
    assert np.allclose(t, [-20, -10, 0, 10, 20])
    with pytest.raises(ValueError):
        G.boundaries(0, 1, 2, "cubic")


def test_index_edges():
    taus = np.array([0.1, 0.5, 2.0])
    x = np.array([0.1, 0.4999999, 0.5, 2.0])
    S = G.segment_index(x, taus)
    assert list(S) == [0, 0, 1, 1]
    I = G.interval_index(x, taus, S, 4)
    assert list(I) == [0, 3, 0, 3]          # x = tau_end clamps into the last interval


@pytest.mark.parametrize("name,lo,hi,spacing", [
    ("inv", 0.01, 10.0, "log"), ("inv_sqrt", 0.01, 100.0, "log"),
    ("silu", -20.0, 20.0, "uniform"), ("gelu", -20.0, 20.0, "uniform")])
def test_precision_grows_with_entries(name, lo, hi, spacing):
    """Precision bits rise by about 2 per doubling of N_br (linear pieces:
    error ~ h^2) once the intervals resolve the function."""
    f = G.FUNCTIONS[name]
    taus = G.boundaries(lo, hi, 4, spacing)
    xs = np.random.default_rng(0).uniform(lo, hi, 20000)
    bits = []
    for nbr in (256, 512, 1024):
        A, B = G.build(f, taus, nbr)
        bits.append(G.precision_bits(f, taus, A, B, xs))
    assert 1.5 < bits[1] - bits[0] < 2.5 and 1.5 < bits[2] - bits[1] < 2.5
