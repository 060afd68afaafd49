"""GPU parity of the lookup-protocol primitives (blind rotation of ciphertext
test polynomials, RLWE trace, plaintext products, recombination) against the
CPU oracle, through the C ABI.  Integer work: bit-exact everywhere.

Small cases run whole batches with ragged sizes; the full-size cases run the
headline shape (n = 1024, N = 2048, batch 14336) and N = 4096 in the launch
configuration the benchmark times and compare seeded samples one by one."""
import numpy as np
import pytest

from gpu_helpers import keyset, require_gpu, say
from paper_2609_16915_amd import rosetta as R
from paper_2609_16915_amd import workloads as W

pytestmark = pytest.mark.gpu
P = 0xFFFFFFFF00000001
SIGMA = 2.0 ** -51


@pytest.fixture(scope="session")
def torch_dev():
    return require_gpu()


def ring_params(N, n=16):
    return dict(n=n, k=1, N=N, pbs_level=2, pbs_base_log=8, ks_level=3, ks_base_log=4,
                msg_bits=2)


def sample_rows(count, k=4, seed=0):
    rng = np.random.default_rng(seed)
    picks = {0, count - 1} | set(int(x) for x in rng.integers(0, count, k))
    return sorted(picks)


# ------------------------------------------------------------------- trace ---

@pytest.mark.parametrize("N,level,base_log,batch", [
    (256, 4, 12, 7), (256, 2, 20, 5), (256, 3, 10, 9), (256, 1, 30, 3),
    (512, 4, 12, 3), (1024, 4, 12, 3), (2048, 4, 12, 5), (4096, 4, 12, 3),
    (2048, 2, 16, 3)])
def test_trace_vs_oracle(O, torch_dev, N, level, base_log, batch):
    rng = np.random.default_rng(N + level)
    S = np.asarray(rng.integers(0, 2, N), dtype=np.uint64)
    autk = O.autk_keygen(N + 1, N, level, base_log, SIGMA, S)
    prm = ring_params(N)
    autk_dev = R.autk_prepare(R.to_device(autk), prm, level)
    cts = rng.integers(0, P, (batch, 2 * N), dtype=np.uint64)
    say(f"[trace] N={N} level={level} base_log={base_log} batch={batch}")
    got = R.to_host(R.trace(R.to_device(cts), autk_dev, prm, level, base_log))
    ref = O.trace_batch(N, level, base_log, cts, autk, O.NTT)
    assert np.array_equal(got, ref)
    # in place
    t = R.to_device(cts)
    R.trace(t, autk_dev, prm, level, base_log, out=t)
    assert np.array_equal(R.to_host(t), ref)


def test_trace_semantics(O, torch_dev):
    """Trace of an encryption keeps the constant coefficient of the phase
    and cancels the rest (phase checked with the oracle's key)."""
    N = 2048
    rng = np.random.default_rng(3)
    S = np.asarray(rng.integers(0, 2, N), dtype=np.uint64)
    autk = O.autk_keygen(9, N, 4, 12, SIGMA, S)
    m = rng.integers(0, P, (4, N), dtype=np.uint64)
    cts = O.glwe_encrypt(10, SIGMA, S, m)
    out = R.to_host(R.trace(R.to_device(cts), R.autk_prepare(R.to_device(autk), ring_params(N), 4),
                            ring_params(N), 4, 12))
    for q in range(4):
        ph_in, ph = O.glwe_phase(S, cts[q]), O.glwe_phase(S, out[q])
        err = [(int(a) - int(b)) % P for a, b in zip(ph, [int(ph_in[0])] + [0] * (N - 1))]
        err = [e if e <= P // 2 else e - P for e in err]
        assert max(abs(e) for e in err) < 2 ** 44


# --------------------------------------------- blind rotation of a ciphertext ---

def test_blind_rotate_glwe_tiny_whole_batch(O, torch_dev):
    w, op, ks, bsk, ksk = keyset(O, "tiny")
    rng = np.random.default_rng(4)
    for batch in (1, 5, 33):
        lwe = rng.integers(0, P, (batch, w.n + 1), dtype=np.uint64)
        tp = O.glwe_encrypt(int(batch), SIGMA, ks.glwe_key,
                            rng.integers(0, P, (batch, w.N), dtype=np.uint64))
        say(f"[br_glwe] tiny batch={batch}")
        ref = O.blind_rotate_glwe_batch(op, lwe, ks.bsk, tp, O.NTT)
        got = R.to_host(R.blind_rotate_glwe(R.to_device(lwe), bsk, R.to_device(tp), w.params()))
        assert np.array_equal(got, ref)
        ext = R.to_host(R.blind_rotate_glwe(R.to_device(lwe), bsk, R.to_device(tp), w.params(),
                                            extract=True))
        for q in range(batch):
            assert np.array_equal(ext[q], O.sample_extract(w.N, ref[q]))


def test_blind_rotate_glwe_trivial_tp_equals_pbs_rotation(O, torch_dev):
    """tp = (0, v) for every ciphertext gives the shared-LUT blind rotation."""
    w, op, ks, bsk, ksk = keyset(O, "tiny")
    rng = np.random.default_rng(5)
    lwe = R.to_device(rng.integers(0, P, (6, w.n + 1), dtype=np.uint64))
    v = rng.integers(0, P, w.N, dtype=np.uint64)
    tp = np.zeros((6, 2 * w.N), np.uint64)
    tp[:, w.N:] = v
    a = R.to_host(R.blind_rotate_glwe(lwe, bsk, R.to_device(tp), w.params()))
    b = R.to_host(R.blind_rotate(lwe, bsk, R.to_device(v), w.params()))
    assert np.array_equal(a, b)


@pytest.mark.parametrize("name", ["llama3_8b_silu", "llama3_8b_softmax_exp"])
def test_blind_rotate_glwe_full_size_sampled(O, torch_dev, name):
    w, op, ks, bsk, ksk = keyset(O, name)
    batch = w.batch if name == "llama3_8b_silu" else 4096
    rng = np.random.default_rng(6)
    lwe = rng.integers(0, P, (batch, w.n + 1), dtype=np.uint64)
    tp = rng.integers(0, P, (batch, 2 * w.N), dtype=np.uint64)
    say(f"[br_glwe] {name} batch={batch}")
    got = R.to_host(R.blind_rotate_glwe(R.to_device(lwe), bsk, R.to_device(tp), w.params()))
    rows = sample_rows(batch, 2, seed=7)
    ref = O.blind_rotate_glwe_batch(op, lwe[rows], ks.bsk, tp[rows], O.NTT)
    for i, q in enumerate(rows):
        assert np.array_equal(got[q], ref[i]), q


# ------------------------------------------------------ construct, recombine ---

@pytest.mark.parametrize("N,npoly,batch,with_pb", [
    (256, 1, 5, True), (256, 3, 4, False), (2048, 4, 6, True), (4096, 2, 3, True)])
def test_glwe_mul_plain_vs_oracle(O, torch_dev, N, npoly, batch, with_pb):
    rng = np.random.default_rng(N + npoly)
    cts = rng.integers(0, P, (batch, 2 * N), dtype=np.uint64)
    pa = rng.integers(0, P, (npoly, N), dtype=np.uint64)
    pb = rng.integers(0, P, (npoly, N), dtype=np.uint64) if with_pb else None
    pa_prep = R.plain_prepare(R.to_device(pa), N)
    got = R.to_host(R.glwe_mul_plain(R.to_device(cts), pa_prep,
                                     None if pb is None else R.to_device(pb), N))
    got = got.reshape(batch, npoly, 2 * N)
    for q in range(batch):
        for s in range(npoly):
            ref = O.glwe_mul_plain(cts[q], pa[s], None if pb is None else pb[s], O.NTT)
            assert np.array_equal(got[q, s], ref), (q, s)


@pytest.mark.parametrize("N,nseg,batch", [(256, 4, 5), (2048, 4, 3), (4096, 7, 2)])
def test_glwe_recombine_vs_oracle(O, torch_dev, N, nseg, batch):
    rng = np.random.default_rng(N + nseg)
    cts = rng.integers(0, P, (batch, nseg, 2 * N), dtype=np.uint64)
    got = R.to_host(R.glwe_recombine(R.to_device(cts), nseg, N))
    for q in range(batch):
        assert np.array_equal(got[q], O.glwe_recombine(cts[q]))
    exps = rng.integers(0, 2 * N, nseg).astype(np.uint32)
    exps[0] = 2 * N - 1
    got = R.to_host(R.glwe_recombine(R.to_device(cts), nseg, N, exps=exps))
    for q in range(batch):
        assert np.array_equal(got[q], O.glwe_recombine(cts[q], exps))


@pytest.mark.parametrize("N,count,batch", [(256, 3, 4), (2048, 16, 3), (4096, 5, 2)])
def test_monomial_copies_and_extract_vs_oracle(O, torch_dev, N, count, batch):
    rng = np.random.default_rng(N + count + 1)
    cts = rng.integers(0, P, (batch, 2 * N), dtype=np.uint64)
    exps = rng.integers(0, 2 * N, count).astype(np.uint32)
    exps[0], exps[-1] = 0, 2 * N - 1
    got = R.to_host(R.glwe_monomial_mul(R.to_device(cts), exps, N)).reshape(batch, count, 2 * N)
    for q in range(batch):
        for s in range(count):
            want = np.concatenate([O.monomial_mul(cts[q, :N], int(exps[s])),
                                   O.monomial_mul(cts[q, N:], int(exps[s]))])
            assert np.array_equal(got[q, s], want)
    big = R.to_host(R.sample_extract(R.to_device(cts), N))
    for q in range(batch):
        assert np.array_equal(big[q], O.sample_extract(N, cts[q]))


# ------------------------------------------------- Step 3 of the lookup, chained ---

def test_select_chain_bit_exact(O, torch_dev):
    """Construct (N_seg products), select by I (blind rotation + trace),
    recombine, select by S: the GPU chain equals the oracle chain on every
    intermediate, at the headline ring (n = 1024, N = 2048) on a small
    batch."""
    w, op, ks, bsk, ksk = keyset(O, "llama3_8b_silu")
    N, nseg, batch = w.N, 4, 2
    rng = np.random.default_rng(8)
    autk = O.autk_keygen(11, N, 4, 12, SIGMA, ks.glwe_key)
    autk_dev = R.autk_prepare(R.to_device(autk), w.params(), 4)
    x = O.glwe_encrypt(12, SIGMA, ks.glwe_key, rng.integers(0, P, (batch, N), dtype=np.uint64))
    pa = rng.integers(0, P, (nseg, N), dtype=np.uint64)
    pb = rng.integers(0, P, (nseg, N), dtype=np.uint64)
    lwe_I = rng.integers(0, P, (batch, w.n + 1), dtype=np.uint64)
    lwe_S = rng.integers(0, P, (batch, w.n + 1), dtype=np.uint64)

    r = R.glwe_mul_plain(R.to_device(x), R.plain_prepare(R.to_device(pa), N), R.to_device(pb), N)
    lwe_rep = R.to_device(np.repeat(lwe_I, nseg, axis=0))
    sel = R.blind_rotate_glwe(lwe_rep, bsk, r.reshape(batch * nseg, 2 * N), w.params())
    sel = R.trace(sel, autk_dev, w.params(), 4, 12, out=sel)
    Rc = R.glwe_recombine(sel, nseg, N)
    out = R.trace(R.blind_rotate_glwe(R.to_device(lwe_S), bsk, Rc, w.params()), autk_dev,
                  w.params(), 4, 12)
    got_r, got_sel, got_R, got = (R.to_host(t) for t in (r, sel, Rc, out))

    for q in range(batch):
        rs = np.stack([O.glwe_mul_plain(x[q], pa[s], pb[s], O.NTT) for s in range(nseg)])
        assert np.array_equal(got_r.reshape(batch, nseg, 2 * N)[q], rs)
        say(f"[chain] ciphertext {q}: oracle blind rotations")
        br = O.blind_rotate_glwe_batch(op, np.repeat(lwe_I[q:q + 1], nseg, axis=0), ks.bsk, rs,
                                       O.NTT)
        tr = O.trace_batch(N, 4, 12, br, autk, O.NTT)
        assert np.array_equal(got_sel.reshape(batch, nseg, 2 * N)[q], tr)
        Rq = O.glwe_recombine(tr)
        assert np.array_equal(got_R[q], Rq)
        fin = O.trace(N, 4, 12, O.blind_rotate_glwe_batch(op, lwe_S[q:q + 1], ks.bsk,
                                                          Rq[None, :], O.NTT)[0], autk, O.NTT)
        assert np.array_equal(got[q], fin)


def test_multi_value_batching_chain_bit_exact(O, torch_dev):
    """Sec. 3.3.2 on the GPU: K = 16 values packed in one ciphertext per
    batch item, moved to the constant term (monomial copies), isolated by
    the trace, extracted and key-switched to LWE inputs, then shifted back
    and recombined; every intermediate equals the oracle's."""
    w, op, ks, bsk, ksk = keyset(O, "llama3_8b_silu")
    N, K, batch = w.N, 16, 2
    rng = np.random.default_rng(30)
    autk = O.autk_keygen(31, N, 4, 12, SIGMA, ks.glwe_key)
    autk_dev = R.autk_prepare(R.to_device(autk), w.params(), 4)
    packed = O.glwe_encrypt(32, SIGMA, ks.glwe_key, rng.integers(0, P, (batch, N), dtype=np.uint64))
    pos = np.sort(rng.choice(N, K, replace=False)).astype(np.uint32)
    moved = R.glwe_monomial_mul(R.to_device(packed), (2 * N - pos) % (2 * N), N)
    singles = R.trace(moved.reshape(batch * K, 2 * N), autk_dev, w.params(), 4, 12)
    lwe = R.keyswitch(R.sample_extract(singles, N), ksk, w.params())
    back = R.glwe_recombine(singles, K, N, exps=pos)
    got_s, got_l, got_b = R.to_host(singles), R.to_host(lwe), R.to_host(back)
    for q in range(batch):
        mv = np.stack([np.concatenate([O.monomial_mul(packed[q, :N], int(2 * N - c)),
                                       O.monomial_mul(packed[q, N:], int(2 * N - c))])
                       for c in pos])
        tr = O.trace_batch(N, 4, 12, mv, autk, O.NTT)
        assert np.array_equal(got_s.reshape(batch, K, 2 * N)[q], tr)
        for j in range(K):
            big = O.sample_extract(N, tr[j])
            assert np.array_equal(got_l.reshape(batch, K, w.n + 1)[q, j],
                                  O.keyswitch(op, big, ks.ksk))
        assert np.array_equal(got_b[q], O.glwe_recombine(tr, pos))
