"""Oracle of the TFHE core of the cryptographic lookup (ROSETTA Sec. 3.2,
Algorithm 1, Steps 1-3), composed from the C oracle's primitives.

TEST INFRASTRUCTURE ONLY (tests/ and nothing in the product path).  The
encodings follow the conventions stated in the library header for
rosetta_lookup_params, written out here independently:

  Step 1  y_j = [[x]]_cmp - round(tau_j 2^sc); c_j = PBS(y_j, v = mu) + mu,
          mu = floor(p / 4 nseg); S = sum_j c_j.
          With a refinement of k bits (refine = k > 0) the comparison
          chains three blind rotations instead (the paper's HomComp chains
          several PBS, Sec. 3.2 Step 1), so that its resolution is 2^k times
          finer:
            y'  = y_j + h,  h = floor(p / 2^(k+1))      (half a digit D = p/2^k)
            z   = 2^k y'                                 (fine phase phi)
            e   = SE(BlindRot(z, c1)),  c1 = floor(p / 2^(k+2))
            s1  = KS(e),  s1' = KS(2^k e)                (signs of z at the coarse
                                                          and, within 2^k, the
                                                          fine scale p/4)
            s2  = PBS(z - s1', f),  f(phi) = -phi / 2^k on [-p/4, p/4)
            c_j = PBS(y_j - s1 + s2, mu) + mu
          One blind rotation gives both signs: the extracted ciphertext is
          scaled before the key switch, so that its small blind-rotation
          noise, not the key switch's, is what 2^k multiplies.
          y' - s1 + s2 is about D round(y'/D), a whole number of digits,
          and it is at least D exactly when y_j >= 0, so the last sign
          bootstrap decides half a digit away from zero; only y_j within the
          fine PBS's resolution (the drift of z's modulus switch, divided by
          2^k) can land on either side.
  Step 2  t = p(X) [[x]] + q(X) (segment s over the window of rotations
          rounding to s N/nseg, the wrapped part negated); I = KS(SE(
          BlindRot(t, S))).
  Step 3  r_s = a_s(X) [[x]] + b_s(X) (interval i at coefficient i + margin,
          slopes at 2^sv, offsets and the result at 2^(sx+sv));
          r_s <- Trace(BlindRot(r_s, I)); R = sum_s X^(s N/nseg) r_s;
          out = Trace(BlindRot(W R, S)).
"""
from __future__ import annotations

import numpy as np

from oracle import oracle as O

P = O.P


def enc(v: float, k: int) -> int:
    """round(v 2^k) (half to even, of the double v 2^k) as an element of Z_p."""
    return round(float(v) * 2.0 ** k) % P


def refine_polys(N, k):
    """Test polynomials of the refined comparison: the constant
    floor(p / 2^(k+2)) (the sign at the coarse scale; 2^k times it, the fine
    one) and f with coefficient j = -round(w_j p / (2^(k+1) N)), w_j = min(j, N - j)
    (rounded half up): a rotation r < N/2 selects f_r, the value at phase
    r p / 2N, and a rotation r >= 3N/2 selects -f_(r-N), the value at phase
    (r - 2N) p / 2N, so that on phases in [-p/4, p/4) the bootstrap returns
    -phase / 2^k."""
    c1 = np.full(N, P // 2 ** (k + 2), np.uint64)
    f = np.zeros(N, np.uint64)
    for j in range(N):
        w = min(j, N - j)
        g = (2 * w * P + 2 ** (k + 1) * N) // (2 ** (k + 2) * N)   # round half up
        f[j] = (P - g) % P
    return c1, f


def encode(N, nseg, nbr, margin, sx, sp, sv, sc, tau, a, b, refine=0):
    """Plaintext polynomials and constants of the lookup (host side)."""
    box = N // nseg
    h = box // 2
    p_hat = np.zeros(N, np.uint64)
    q_hat = np.zeros(N, np.uint64)
    for j in range(N):
        wrapped = j >= N - h
        s = 0 if wrapped else (j + h) // box
        width = tau[s + 1] - tau[s]
        pv = enc(nbr / width, sp)
        qv = enc(-tau[s] * nbr / width - 0.5 + margin, sx + sp)
        p_hat[j] = (P - pv) % P if wrapped else pv
        q_hat[j] = (P - qv) % P if wrapped else qv
    a_hat = np.zeros((nseg, N), np.uint64)
    b_hat = np.zeros((nseg, N), np.uint64)
    for s in range(nseg):
        for j in range(N):
            i = min(max(j - margin, 0), nbr - 1)
            a_hat[s, j] = enc(a[s][i], sv)
            b_hat[s, j] = enc(b[s][i], sx + sv)
    window = np.zeros(N, np.uint64)
    for k in range(-h, box - h):
        if k >= 0:
            window[k] = 1
        else:
            window[N + k] = P - 1          # X^k = -X^(N+k)
    mu = P // (4 * nseg)
    sign_lut = np.full(N, mu, np.uint64)
    consts = np.array([enc(-tau[j], sc) for j in range(1, nseg)] + [(nseg - 1) * mu % P],
                      dtype=np.uint64)
    out = dict(p_hat=p_hat, q_hat=q_hat, a_hat=a_hat, b_hat=b_hat, window=window,
               sign_lut=sign_lut, consts=consts, refine=refine)
    if refine:
        out["c1"], out["f"] = refine_polys(N, refine)
    return out


def block(parts) -> np.ndarray:
    """The library's plaintext block order: p, q, a_s, b_s, W, sign LUT, then
    with a refined comparison its two test polynomials."""
    extra = [parts["c1"], parts["f"]] if parts.get("refine") else []
    return np.concatenate([parts["p_hat"], parts["q_hat"], parts["a_hat"].reshape(-1),
                           parts["b_hat"].reshape(-1), parts["window"], parts["sign_lut"],
                           *extra])


def lwe_add(a, b):
    return ((a.astype(object) + b.astype(object)) % P).astype(np.uint64)


def lwe_sub(a, b):
    return ((a.astype(object) - b.astype(object)) % P).astype(np.uint64)


def lwe_scale(a, m: int):
    return ((a.astype(object) * m) % P).astype(np.uint64)


def compare(prm, ks, parts, ys, kind=O.NTT, nthreads=0, want_steps=False):
    """HomComp of Step 1 on the comparison inputs ys [count][n+1] (phase
    (x - tau) 2^sc): c = 0 or 2 mu, mu = the sign test polynomial's value."""
    n = prm.n
    k = parts.get("refine", 0)
    mu_poly = parts["sign_lut"]
    mu = int(mu_poly[0])

    def pbs(cts, v, want_big=False):
        return O.pbs(prm, cts, ks.bsk, ks.ksk, v, kind, nthreads, want_big=want_big)

    steps = {}
    if k == 0:
        y2 = ys
    else:
        h = P // 2 ** (k + 1)
        yp = ys.copy()
        yp[:, n] = (yp[:, n].astype(object) + h) % P
        z = lwe_scale(yp, 2 ** k)
        s1, e = pbs(z, parts["c1"], want_big=True)
        s1p = np.stack([O.keyswitch(prm, row, ks.ksk) for row in lwe_scale(e, 2 ** k)])
        s2 = pbs(lwe_sub(z, s1p), parts["f"])
        y2 = lwe_add(lwe_sub(ys, s1), s2)
        steps = dict(z=z, s1p=s1p, s1=s1, s2=s2, y2=y2)
    c = pbs(y2, mu_poly)
    c[:, n] = (c[:, n].astype(object) + mu) % P
    return (c, steps) if want_steps else c


def evaluate(prm, ks, autk, trace_level, trace_base_log, parts, nseg, x_rlwe, x_cmp,
             kind=O.NTT, nthreads=0, want_steps=False):
    n, N = prm.n, prm.N
    batch = x_cmp.shape[0]
    consts = parts["consts"]
    # Step 1
    ys = np.zeros((batch, nseg - 1, n + 1), np.uint64)
    for q in range(batch):
        for j in range(nseg - 1):
            ys[q, j] = x_cmp[q]
            ys[q, j, n] = (int(x_cmp[q, n]) + int(consts[j])) % P
    cmp = compare(prm, ks, parts, ys.reshape(-1, n + 1), kind, nthreads)
    # c_j = PBS + mu, summed: S = sum_j PBS_j + (nseg - 1) mu
    mu = int(parts["sign_lut"][0])
    cmp[:, n] = (cmp[:, n].astype(object) - mu) % P
    cmp = cmp.reshape(batch, nseg - 1, n + 1)
    S = np.zeros((batch, n + 1), np.uint64)
    for q in range(batch):
        acc = np.zeros(n + 1, np.uint64)
        acc[n] = consts[nseg - 1]
        for j in range(nseg - 1):
            acc = lwe_add(acc, cmp[q, j])
        S[q] = acc
    # Step 2
    T = np.stack([O.glwe_mul_plain(x_rlwe[q], parts["p_hat"], parts["q_hat"], kind)
                  for q in range(batch)])
    acc = O.blind_rotate_glwe_batch(prm, S, ks.bsk, T, kind, nthreads)
    I = np.stack([O.keyswitch(prm, O.sample_extract(N, acc[q]), ks.ksk) for q in range(batch)])
    # Step 3
    rs = np.stack([O.glwe_mul_plain(x_rlwe[q], parts["a_hat"][s], parts["b_hat"][s], kind)
                   for q in range(batch) for s in range(nseg)])
    sel = O.blind_rotate_glwe_batch(prm, np.repeat(I, nseg, axis=0), ks.bsk, rs, kind, nthreads)
    sel = O.trace_batch(N, trace_level, trace_base_log, sel, autk, kind, nthreads)
    exps = np.array([s * (N // nseg) for s in range(nseg)], np.uint32)
    R = np.stack([O.glwe_recombine(sel[q * nseg:(q + 1) * nseg], exps) for q in range(batch)])
    RB = np.stack([O.glwe_mul_plain(R[q], parts["window"], None, kind) for q in range(batch)])
    fin = O.blind_rotate_glwe_batch(prm, S, ks.bsk, RB, kind, nthreads)
    out = O.trace_batch(N, trace_level, trace_base_log, fin, autk, kind, nthreads)
    if want_steps:
        return out, dict(cmp=cmp, S=S, T=T, I=I, r=rs, sel=sel, R=R, RB=RB)
    return out
