"""The oracle's pins against planted mistakes (CPU only).

Each mutant is a copy of one oracle source with one plausible slip (a
dropped term, a wrong sign, index, root or scale, a transposed operand):
oracle/oracle.c compiled the way oracle/build.py compiles it and loaded
through ROSETTA_ORACLE_LIB, or a Python oracle module (oracle/lookup.py,
oracle/mini.py, oracle/seglut.py) executed in place of the real one, each in
a fresh pytest process.  The pins of that part of the oracle (closed forms, the paper's
worked examples, phase identities and noise bounds, decryption of every
message, agreement of the independent codings) must fail on every mutant: a
mutant that passes them names a convention that no pin fixes.  The
unmodified sources, run through the same harness, must pass them.
"""
import concurrent.futures
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
PINS = ["tests/test_oracle_field.py", "tests/test_oracle_pbs.py", "tests/test_oracle_lookup.py",
        "tests/test_oracle_mini.py"]
LOOKUP_PINS = ["tests/test_oracle_lookup.py", "tests/test_oracle_homcomp.py"]
MINI_PINS = ["tests/test_oracle_mini.py"]

# name -> (what the slip breaks, text in oracle.c, its replacement)
MUTANTS = {
    "ntt_root": (
        "cyclic transform with psi instead of psi^2 (negacyclic evaluation points)",
        "or_dft_cyclic(a, N, or_mul(psi, psi));", "or_dft_cyclic(a, N, psi);"),
    "ntt_inverse_scale": (
        "inverse transform without the factor 1/N",
        "u64 ninv = or_inv((u64)N), t = ninv;", "u64 ninv = 1, t = ninv;"),
    "schoolbook_cyclic": (
        "schoolbook product with X^N = +1 (cyclic instead of negacyclic)",
        "acc[e - N] = or_sub(acc[e - N], prod);", "acc[e - N] = or_add(acc[e - N], prod);"),
    "monomial_sign": (
        "X^r a without the sign of the wrapped coefficients",
        "c[e] = sign ? or_neg(a[j]) : a[j];", "c[e] = a[j];"),
    "modswitch_floor": (
        "modulus switch rounding down instead of to nearest",
        "u128 num = (u128)(2 * (u64)N) * a + (OR_P - 1) / 2;",
        "u128 num = (u128)(2 * (u64)N) * a;"),
    "decompose_no_round": (
        "decomposition truncating the discarded bits instead of rounding",
        "i128 r = or_floor_div(ac + ((i128)1 << (s - 1)), (i128)1 << s);",
        "i128 r = or_floor_div(ac, (i128)1 << s);"),
    "decompose_uncentred": (
        "decomposition of the residue instead of the centred representative",
        "i128 ac = (a <= (OR_P - 1) / 2) ? (i128)a : (i128)a - (i128)OR_P;",
        "i128 ac = (i128)a;"),
    "digit_unbalanced": (
        "digits in [0, B) instead of [-B/2, B/2)",
        "i128 d = m - B / 2;", "i128 d = m;"),
    "gadget_exponent": (
        "gadget factor 2^(64 - t beta) instead of 2^(64 - (t+1) beta)",
        "int e = 64 - (t + 1) * beta;", "int e = 64 - t * beta;"),
    "acc_init_sign": (
        "accumulator started at X^(+b~) v instead of X^(-b~) v",
        "or_poly_monomial_mul(v, (int)((2 * (uint32_t)N - bt) % (2 * (uint32_t)N)), acc + N, N);",
        "or_poly_monomial_mul(v, (int)(bt % (2 * (uint32_t)N)), acc + N, N);"),
    "loop_descending": (
        "CMux steps taken from i = n-1 down (same phase, other noise bits)",
        "for (int i = 0; i < n; ++i) {\n    uint32_t ai = or_modswitch(lwe[i], N);",
        "for (int i = n - 1; i >= 0; --i) {\n    uint32_t ai = or_modswitch(lwe[i], N);"),
    "cmux_no_subtract": (
        "CMux on X^(a~) ACC instead of X^(a~) ACC - ACC",
        "diff[(size_t)u * N + j] = or_sub(rot[(size_t)u * N + j], acc[(size_t)u * N + j]);",
        "diff[(size_t)u * N + j] = rot[(size_t)u * N + j];"),
    "extract_sign": (
        "extraction a'_j = A_(N-j) without the negation",
        "for (int j = 1; j < N; ++j) big[j] = or_neg(acc[N - j]);",
        "for (int j = 1; j < N; ++j) big[j] = acc[N - j];"),
    "extract_index": (
        "extraction reading A_j instead of A_(N-j)",
        "for (int j = 1; j < N; ++j) big[j] = or_neg(acc[N - j]);",
        "for (int j = 1; j < N; ++j) big[j] = or_neg(acc[j]);"),
    "ks_sign": (
        "key switching adding the digit-weighted key rows",
        "for (int c = 0; c <= n; ++c) out[c] = or_sub(out[c], or_mul(d, row[c]));",
        "for (int c = 0; c <= n; ++c) out[c] = or_add(out[c], or_mul(d, row[c]));"),
    "ks_body_dropped": (
        "key switching dropping the body column of the key rows",
        "for (int c = 0; c <= n; ++c) out[c] = or_sub(out[c], or_mul(d, row[c]));",
        "for (int c = 0; c < n; ++c) out[c] = or_sub(out[c], or_mul(d, row[c]));"),
    "test_poly_offset": (
        "test polynomial boxes not centred on their rotation",
        "v[j] = or_mul(delta, table[(j + h) / box]);", "v[j] = or_mul(delta, table[j / box]);"),
    "test_poly_tail_sign": (
        "wrapped half box of T[0] stored without its negacyclic sign",
        "v[j] = or_neg(or_mul(delta, table[0]));", "v[j] = or_mul(delta, table[0]);"),
    "ext_product_u_t_transposed": (
        "external product indexing the key [t][u] instead of [u][t]",
        "const u64 *row = ggsw + (((size_t)u * l + t) * 2 + c) * N;",
        "const u64 *row = ggsw + (((size_t)t * 2 + u) * 2 + c) * N;"),
    "ext_product_c_swapped": (
        "external product with the two output components swapped",
        "const u64 *row = ggsw + (((size_t)u * l + t) * 2 + c) * N;",
        "const u64 *row = ggsw + (((size_t)u * l + t) * 2 + (1 - c)) * N;"),
    "ntt_tier_c_swapped": (
        "transform-domain CMux with the two output components swapped",
        "size_t off = (((size_t)u * l + t) * 2 + c) * N;",
        "size_t off = (((size_t)u * l + t) * 2 + (1 - c)) * N;"),
    "ntt_tier_level_reversed": (
        "transform-domain CMux pairing digit l-1-t with key level t",
        "fd[x] = or_from_i64(dg[t]);", "fd[x] = or_from_i64(dg[l - 1 - t]);"),
    "keygen_component": (
        "GGSW rows adding s_i g_t to the wrong component",
        "if (u == 0)\n          A[0] = or_add(A[0], g);", "if (u == 1)\n          A[0] = or_add(A[0], g);"),
    "field_sub": (
        "subtraction without the added p (wraps modulo 2^128 instead)",
        "u64 or_sub(u64 a, u64 b) { return (u64)(((u128)a + OR_P - b) % OR_P); }",
        "u64 or_sub(u64 a, u64 b) { return (u64)(((u128)a - b) % OR_P); }"),
    "automorphism_sign": (
        "automorphism without the sign of exponents past N",
        "      out[e - N] = or_sub(out[e - N], a[j]);", "      out[e - N] = or_add(out[e - N], a[j]);"),
    "automorphism_power": (
        "automorphism X^j -> X^(j (d+2)) instead of X^(j d)",
        "u64 e = ((u64)j * (u64)d) % (2 * (u64)N);", "u64 e = ((u64)j * (u64)(d + 2)) % (2 * (u64)N);"),
    "glwe_ks_sign": (
        "GLWE key switching adding the digit-weighted rows",
        "res[(size_t)c * N + x] = or_sub(res[(size_t)c * N + x], prod[x]);",
        "res[(size_t)c * N + x] = or_add(res[(size_t)c * N + x], prod[x]);"),
    "glwe_ks_body_dropped": (
        "GLWE key switching starting from a zero body",
        "    res[N + x] = ct[N + x];", "    res[N + x] = 0;"),
    "autk_key_power": (
        "automorphism key of tau_(2^k - 1) instead of tau_(2^k + 1)",
        "      int d = (1 << k) + 1;\n      u64 *A = autk", "      int d = (1 << k) - 1;\n      u64 *A = autk"),
    "trace_scale_last": (
        "trace without the factor N^-1",
        "for (int j = 0; j < 2 * N; ++j) c[j] = or_mul(ct[j], ninv);",
        "for (int j = 0; j < 2 * N; ++j) c[j] = ct[j];"),
    "trace_round_key": (
        "trace round k keyed with the automorphism key of round k+1",
        "autk + (size_t)(k - 1) * levels * 2 * N, ks, kind);",
        "autk + (size_t)(k % rounds) * levels * 2 * N, ks, kind);"),
    "mul_plain_offset_dropped": (
        "plaintext product without the offset polynomial",
        "tmp[N + x] = or_add(prod[x], pb ? pb[x] : 0);", "tmp[N + x] = prod[x];"),
    "recombine_exponent": (
        "recombination placing r_s at X^(e_s + 1)",
        "exps ? (int)exps[s] : s, tmp, N);", "exps ? (int)exps[s] + 1 : s + 1, tmp, N);"),
    "br_glwe_init_one_side": (
        "encrypted test polynomial with only its body rotated by X^(-b~)",
        "  or_poly_monomial_mul(tp, r0, acc, N);", "  memcpy(acc, tp, (size_t)N * sizeof(u64));"),
    "delta_no_padding": (
        "plaintext scale p/M instead of p/2M (no padding bit)",
        "static u64 or_delta(const or_params *P) { return OR_P / (2ULL << P->msg_bits); }",
        "static u64 or_delta(const or_params *P) { return OR_P / (1ULL << P->msg_bits); }"),
}


# Mutants of the Python oracle modules: module -> name -> (slip, text, replacement)
PY_MUTANTS = {
    "lookup": {
        "refine_f_sign": (
            "fine test polynomial +phase/2^k instead of -phase/2^k",
            "f[j] = (P - g) % P", "f[j] = g % P"),
        "refine_no_half_digit": (
            "comparison input not moved by half a digit",
            "h = P // 2 ** (k + 1)\n", "h = 0\n"),
        "refine_scale": (
            "fine phase scaled by 2^(k-1) instead of 2^k",
            "z = lwe_scale(yp, 2 ** k)", "z = lwe_scale(yp, 2 ** (k - 1))"),
        "refine_recombine_sign": (
            "y - s1 + s2 formed as y + s1 + s2",
            "y2 = lwe_add(lwe_sub(ys, s1), s2)", "y2 = lwe_add(lwe_add(ys, s1), s2)"),
        "refine_coarse_const": (
            "coarse sign of p / 2^(k+1) instead of p / 2^(k+2)",
            "c1 = np.full(N, P // 2 ** (k + 2), np.uint64)",
            "c1 = np.full(N, P // 2 ** (k + 1), np.uint64)"),
        "refine_fine_sign_unscaled": (
            "fine sign taken from the extracted ciphertext without the 2^k scale",
            "lwe_scale(e, 2 ** k)", "lwe_scale(e, 1)"),
        "refine_fine_input": (
            "fine bootstrap on z instead of z - s1' (a quarter-phase off)",
            "s2 = pbs(lwe_sub(z, s1p), parts[\"f\"])", "s2 = pbs(z, parts[\"f\"])"),
        "compare_no_mu": (
            "comparison output without the + mu offset",
            "c[:, n] = (c[:, n].astype(object) + mu) % P", "c[:, n] = c[:, n]"),
        "encode_margin": (
            "interval lines stored without the margin offset",
            "i = min(max(j - margin, 0), nbr - 1)", "i = min(max(j, 0), nbr - 1)"),
        "encode_window_sign": (
            "window terms below zero stored without the sign of X^N = -1",
            "window[N + k] = P - 1", "window[N + k] = 1"),
        "encode_p_wrap": (
            "slope polynomial's wrapped half box not negated",
            "p_hat[j] = (P - pv) % P if wrapped else pv", "p_hat[j] = pv"),
        "encode_q_half": (
            "interval index rounded instead of floored (no -1/2)",
            "qv = enc(-tau[s] * nbr / width - 0.5 + margin, sx + sp)",
            "qv = enc(-tau[s] * nbr / width + margin, sx + sp)"),
        "encode_b_scale": (
            "offsets at scale 2^sv instead of 2^(sx+sv)",
            "b_hat[s, j] = enc(b[s][i], sx + sv)", "b_hat[s, j] = enc(b[s][i], sv)"),
        "encode_boundary_sign": (
            "comparison constants +tau instead of -tau",
            "consts = np.array([enc(-tau[j], sc) for j in range(1, nseg)]",
            "consts = np.array([enc(tau[j], sc) for j in range(1, nseg)]"),
        "step1_S_offset": (
            "segment sum without its (nseg - 1) mu offset",
            "acc[n] = consts[nseg - 1]", "acc[n] = 0"),
        "step3_exponents_reversed": (
            "recombination placing segment s at (nseg-1-s) N/nseg",
            "exps = np.array([s * (N // nseg) for s in range(nseg)], np.uint32)",
            "exps = np.array([(nseg - 1 - s) * (N // nseg) for s in range(nseg)], np.uint32)"),
        "step3_window_dropped": (
            "final selection without the window polynomial",
            "RB = np.stack([O.glwe_mul_plain(R[q], parts[\"window\"], None, kind) for q in range(batch)])",
            "RB = R"),
        "mu_value": (
            "sign value p / 2 nseg instead of p / 4 nseg",
            "mu = P // (4 * nseg)", "mu = P // (2 * nseg)"),
    },
    "mini": {
        "loop_descending": (
            "CMux steps from i = n-1 down",
            "for i in range(n):\n        ai", "for i in reversed(range(n)):\n        ai"),
        "extract_sign": (
            "extraction without the negation",
            "[(-A[N - j]) % P for j", "[(A[N - j]) % P for j"),
        "ks_sign": (
            "key switching adding the rows",
            "(out[c] - d * ksk[base + c])", "(out[c] + d * ksk[base + c])"),
        "init_sign": (
            "accumulator started at X^(+b~) v",
            "B = monomial(v, -bt, N)", "B = monomial(v, bt, N)"),
        "decompose_no_round": (
            "decomposition truncating instead of rounding",
            "(ac + (1 << (s - 1))) >> s", "(ac) >> s"),
        "cmux_no_subtract": (
            "CMux on X^(a~) ACC instead of X^(a~) ACC - ACC",
            "[(x - y) % P for x, y in zip(monomial(acc[u], ai, N), acc[u])]",
            "[x % P for x in monomial(acc[u], ai, N)]"),
        "ring_cyclic_fold": (
            "product folded with X^N = +1",
            "[(slot[j] - slot[j + N]) % P for j in range(N)]",
            "[(slot[j] + slot[j + N]) % P for j in range(N)]"),
        "modswitch_floor": (
            "modulus switch rounding down",
            "round(Fraction(2 * N * int(a), P)) % (2 * N)", "(2 * N * int(a) // P) % (2 * N)"),
        "monomial_sign": (
            "X^r a without the sign of the wrapped coefficients",
            "out[e - N] = (-c) % P", "out[e - N] = c % P"),
        "test_poly_offset": (
            "test polynomial boxes not centred",
            "v.append(delta * int(table[(j + h) // box]) % P)",
            "v.append(delta * int(table[j // box]) % P)"),
    },
}
PY_MUTANTS["seglut"] = {
    "log_spacing_linear": (
        "logarithmic boundaries spaced linearly",
        "t = lo * (hi / lo) ** (j / nseg)", "t = lo + (hi - lo) * j / nseg"),
    "chebyshev_nodes_at_ends": (
        "lines through the interval's end points instead of its Chebyshev nodes",
        "x1, x2 = c - r * math.cos(math.pi / 4), c + r * math.cos(math.pi / 4)",
        "x1, x2 = c - r, c + r"),
    "intercept_at_x2": (
        "intercept taken at the wrong node",
        "return slope, y1 - slope * x1", "return slope, y1 - slope * x2"),
    "segment_includes_first": (
        "segment index counting tau_0 too",
        "for j in range(1, len(taus) - 1):", "for j in range(0, len(taus) - 1):"),
    "segment_strict": (
        "x = tau_j counted in the lower segment",
        "S += (x >= taus[j]).astype(np.int64)", "S += (x > taus[j]).astype(np.int64)"),
    "interval_round": (
        "interval index rounded instead of floored",
        "I = np.floor((x - lo) / (hi - lo) * nbr).astype(np.int64)",
        "I = np.round((x - lo) / (hi - lo) * nbr).astype(np.int64)"),
    "protocol_q_sign": (
        "Step 2 offset +tau_s N_br / width",
        "q = -taus[:-1] * nbr / width", "q = taus[:-1] * nbr / width"),
    "protocol_q_upper": (
        "Step 2 offset from the segment's upper boundary",
        "q = -taus[:-1] * nbr / width", "q = -taus[1:] * nbr / width"),
}
SEGLUT_PINS = ["tests/test_oracle_seglut.py"]
PY_PINS = {"lookup": LOOKUP_PINS, "mini": MINI_PINS, "seglut": SEGLUT_PINS}

# Runs the pins with one module of the oracle package replaced by the source
# file given: argv = repository root, module name, source file, pin files.
_DRIVER = """
import sys, types
sys.path.insert(0, sys.argv[1])
import oracle
name, path = "oracle." + sys.argv[2], sys.argv[3]
m = types.ModuleType(name)
m.__file__ = path
sys.modules[name] = m
exec(compile(open(path).read(), path, "exec"), m.__dict__)
setattr(oracle, sys.argv[2], m)
import pytest
sys.exit(pytest.main(["-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu", *sys.argv[4:]]))
"""


def _compile_to():
    import importlib.util
    spec = importlib.util.spec_from_file_location("_oracle_build",
                                                  os.path.join(ROOT, "oracle", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod.compile_to


def _outcome(r):
    lines = r.stdout.splitlines()
    failed = next((l for l in lines if l.startswith("FAILED tests/test_oracle_")), None)
    errored = any(l.startswith("ERROR") for l in lines) or r.returncode not in (0, 1)
    return r.returncode, failed, errored


def _run_c(name, text, pins, workdir, compile_to):
    """Build `text` as the C oracle and run `pins` against it in a new
    process; returns (exit status, first FAILED line, whether anything
    errored)."""
    d = os.path.join(workdir, "c_" + name)
    os.makedirs(d)
    src = os.path.join(d, "oracle.c")
    with open(src, "w") as f:
        f.write(text)
    so = compile_to(src, os.path.join(d, "liboracle.so"))
    env = dict(os.environ, ROSETTA_ORACLE_LIB=so, OMP_NUM_THREADS="1")
    return _outcome(subprocess.run(
        [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
         *pins], cwd=ROOT, env=env, capture_output=True, text=True))


def _run_py(module, name, text, pins, workdir):
    """Run `pins` with oracle.<module> executed from `text` instead."""
    d = os.path.join(workdir, f"{module}_{name}")
    os.makedirs(d)
    src = os.path.join(d, module + ".py")
    with open(src, "w") as f:
        f.write(text)
    driver = os.path.join(d, "driver.py")
    with open(driver, "w") as f:
        f.write(_DRIVER)
    env = dict(os.environ, OMP_NUM_THREADS="1")
    return _outcome(subprocess.run([sys.executable, driver, ROOT, module, src, *pins], cwd=ROOT,
                                   env=env, capture_output=True, text=True))


@pytest.fixture(scope="module")
def outcomes():
    with open(SRC) as f:
        src = f.read()
    for name, (_, old, _new) in MUTANTS.items():
        assert src.count(old) == 1, f"mutant {name}: its text is not found once in oracle.c"
    py_src = {}
    for module, muts in PY_MUTANTS.items():
        with open(os.path.join(ROOT, "oracle", module + ".py")) as f:
            py_src[module] = f.read()
        for name, (_, old, _new) in muts.items():
            assert py_src[module].count(old) == 1, f"mutant {module}.{name}: text not found once"
    compile_to = _compile_to()
    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    with tempfile.TemporaryDirectory(prefix="oracle_mutants_") as work:
        with concurrent.futures.ThreadPoolExecutor(workers) as ex:
            futs = {"c.control": ex.submit(_run_c, "control", src, PINS[:1], work, compile_to)}
            for name, (_, old, new) in MUTANTS.items():
                futs["c." + name] = ex.submit(_run_c, name, src.replace(old, new), PINS, work,
                                              compile_to)
            for module, muts in PY_MUTANTS.items():
                futs[module + ".control"] = ex.submit(_run_py, module, "control", py_src[module],
                                                      PY_PINS[module], work)
                for name, (_, old, new) in muts.items():
                    futs[f"{module}.{name}"] = ex.submit(
                        _run_py, module, name, py_src[module].replace(old, new),
                        PY_PINS[module], work)
            return {name: f.result() for name, f in futs.items()}


@pytest.mark.parametrize("which", ["c", "lookup", "mini", "seglut"])
def test_unmodified_oracle_passes_through_the_same_harness(outcomes, which):
    rc, failed, errored = outcomes[which + ".control"]
    assert rc == 0 and failed is None and not errored


ALL = [("c", name, slip) for name, (slip, _, _) in sorted(MUTANTS.items())] + \
      [(module, name, slip) for module, muts in PY_MUTANTS.items()
       for name, (slip, _, _) in sorted(muts.items())]


@pytest.mark.parametrize("which,name,slip", ALL, ids=[f"{w}.{n}" for w, n, _ in ALL])
def test_planted_mistake_fails_a_pin(outcomes, which, name, slip):
    rc, failed, errored = outcomes[f"{which}.{name}"]
    assert not errored, f"{which}.{name}: the pin run errored instead of failing"
    assert rc == 1 and failed, f"{which}.{name} ({slip}) passes every pin"
