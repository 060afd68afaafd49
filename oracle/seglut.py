"""Cleartext oracle of the adaptive segmented LUT (ROSETTA Sec. 3.1).

TEST INFRASTRUCTURE ONLY: used by tests/ (and nothing in the product path).
Plain float64 numpy, written from the definitions:

  * the domain [tau_start, tau_end] is cut into N_seg segments by boundaries
    tau_0 < tau_1 < ... < tau_Nseg (Sec. 3.1, "Adaptive LUT Construction");
    the evaluation setup spaces them logarithmically for 1/x and 1/sqrt(x)
    and uniformly for SiLU and GELU (Sec. 5.1, "Experimental Setup");
  * each segment holds N_br equal intervals; interval i of segment s carries
    a linear function a_si x + b_si (or a constant, the function's value at
    the interval midpoint, for the baseline LUT);
  * the linear coefficients interpolate f at the two Chebyshev nodes of the
    interval, c -+ r cos(pi/4) (c the midpoint, r the half-width).  The paper
    prints the coefficients but not the rule; this rule reproduces every
    printed coefficient of the running example, which the tests check;
  * online lookup (Sec. 3.1, "Online Lookup Evaluation"): segment index
    S = sum_{j=1}^{N_seg-1} [x >= tau_j]; local interval index
    I = floor((x - tau_S) / (tau_{S+1} - tau_S) * N_br), clamped to
    [0, N_br) so that x = tau_end falls in the last interval; result
    a_SI x + b_SI;
  * protocol polynomials (Sec. 3.2): slope and offset polynomials of Step 2,
    p_s = N_br / (tau_{s+1} - tau_s), q_s = -tau_s N_br / (tau_{s+1} - tau_s),
    and the per-segment coefficient polynomials a_s(X) = sum_i a_si X^i,
    b_s(X) = sum_i b_si X^i of Step 3;
  * precision in bits = -log2 of the root-mean-square error against the
    exact function (Sec. 5.1).
"""
from __future__ import annotations

import math

import numpy as np

FUNCTIONS = {
    "inv": lambda x: 1.0 / x,
    "inv_sqrt": lambda x: 1.0 / np.sqrt(x),
    "silu": lambda x: x / (1.0 + np.exp(-x)),
    "gelu": lambda x: 0.5 * x * (1.0 + np.vectorize(math.erf)(x / math.sqrt(2.0))),
    "exp": lambda x: np.exp(x),
}


def boundaries(lo: float, hi: float, nseg: int, spacing: str) -> np.ndarray:
    j = np.arange(nseg + 1, dtype=np.float64)
    if spacing == "uniform":
        t = lo + (hi - lo) * j / nseg
    elif spacing == "log":
        t = lo * (hi / lo) ** (j / nseg)
    else:
        raise ValueError(spacing)
    t[0], t[-1] = lo, hi
    return t


def chebyshev_linear(f, a: float, b: float) -> tuple[float, float]:
    """Line through f at the two Chebyshev nodes of [a, b]."""
    c, r = (a + b) / 2.0, (b - a) / 2.0
    x1, x2 = c - r * math.cos(math.pi / 4), c + r * math.cos(math.pi / 4)
    y1, y2 = float(f(np.float64(x1))), float(f(np.float64(x2)))
    slope = (y2 - y1) / (x2 - x1)
    return slope, y1 - slope * x1


def build(f, taus, nbr: int, fit: str = "linear") -> tuple[np.ndarray, np.ndarray]:
    """Coefficients a[s][i], b[s][i] of every interval of every segment."""
    taus = np.asarray(taus, dtype=np.float64)
    nseg = len(taus) - 1
    A = np.zeros((nseg, nbr))
    B = np.zeros((nseg, nbr))
    for s in range(nseg):
        w = (taus[s + 1] - taus[s]) / nbr
        for i in range(nbr):
            lo, hi = taus[s] + i * w, taus[s] + (i + 1) * w
            if fit == "linear":
                A[s, i], B[s, i] = chebyshev_linear(f, lo, hi)
            elif fit == "constant":
                A[s, i], B[s, i] = 0.0, float(f(np.float64((lo + hi) / 2)))
            else:
                raise ValueError(fit)
    return A, B


def segment_index(x, taus) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    S = np.zeros(x.shape, dtype=np.int64)
    for j in range(1, len(taus) - 1):
        S += (x >= taus[j]).astype(np.int64)
    return S


def interval_index(x, taus, S, nbr: int) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    taus = np.asarray(taus, dtype=np.float64)
    lo, hi = taus[S], taus[S + 1]
    I = np.floor((x - lo) / (hi - lo) * nbr).astype(np.int64)
    return np.clip(I, 0, nbr - 1)


def evaluate(x, taus, A, B, index_offset=None) -> np.ndarray:
    """The three-step cleartext lookup of Sec. 3.1; index_offset (one integer
    per input, or None) shifts the interval index before the coefficients
    are read, clamped to the segment."""
    x = np.asarray(x, dtype=np.float64)
    nbr = A.shape[1]
    S = segment_index(x, taus)
    I = interval_index(x, taus, S, nbr)
    if index_offset is not None:
        I = np.clip(I + np.asarray(index_offset, dtype=np.int64), 0, nbr - 1)
    return A[S, I] * x + B[S, I]


def protocol_polys(taus, A, B):
    """(p, q, a_s, b_s) of Sec. 3.2 as coefficient lists."""
    taus = np.asarray(taus, dtype=np.float64)
    nbr = A.shape[1]
    width = taus[1:] - taus[:-1]
    p = nbr / width
    q = -taus[:-1] * nbr / width
    return p, q, A.copy(), B.copy()


def max_relative_error(f, taus, A, B, samples: int = 200001) -> float:
    xs = np.linspace(taus[0], taus[-1], samples)
    y = f(xs)
    return float(np.max(np.abs(evaluate(xs, taus, A, B) - y) / np.abs(y)))


def precision_bits(f, taus, A, B, xs, index_offset=None) -> float:
    err = evaluate(xs, taus, A, B, index_offset) - f(np.asarray(xs, dtype=np.float64))
    return float(-math.log2(math.sqrt(float(np.mean(err * err)))))
