"""GPU parity: the HIP path (through the C ABI) against the CPU oracle,
element by element, on the same seeded inputs.  Integer work, so the bar is
bit-exact everywhere.

Small cases cover several tiles and ragged tails; the full-size cases run the
whole batch of each workload in the launch configuration the benchmark times
and compare a seeded sample of ciphertexts (first, last and random picks)
against the oracle computed one by one, plus decryption properties that hold
at any size."""
import numpy as np
import pytest

from gpu_helpers import bitrev, keyset, oparams, require_gpu, say
from paper_2609_16915_amd import rosetta as R
from paper_2609_16915_amd import workloads as W

pytestmark = pytest.mark.gpu
P = 0xFFFFFFFF00000001


@pytest.fixture(scope="session")
def torch_dev():
    return require_gpu()


# ------------------------------------------------------------ transforms ---

@pytest.mark.parametrize("N", [256, 512, 1024, 2048, 4096])
def test_ntt_forward_inverse_vs_oracle(O, torch_dev, N):
    rng = np.random.default_rng(N)
    count = 5
    a = rng.integers(0, P, size=(count, N), dtype=np.uint64)
    fwd = R.to_host(R.ntt_forward(R.to_device(a), N))
    L = N.bit_length() - 1
    perm = np.array([bitrev(j, L) for j in range(N)])
    for c in range(count):
        ref = O.ntt_forward(a[c])                 # natural order, A_k = a(psi^(2k+1))
        assert np.array_equal(fwd[c], ref[perm])  # library order: A_rev(j)
    back = R.to_host(R.ntt_inverse(R.to_device(fwd), N))
    assert np.array_equal(back, a)
    # in place
    t = R.to_device(a)
    R.ntt_forward(t, N, out=t)
    assert np.array_equal(R.to_host(t), fwd)


@pytest.mark.parametrize("N", [256, 1024, 2048, 4096])
def test_ntt_edge_inputs_vs_oracle(O, torch_dev, N):
    # structured inputs whose butterflies meet 0, p - 1 and equal operands:
    # constants, single spikes at the block boundaries of each pass, and
    # alternating extremes
    rows = [[0] * N, [P - 1] * N, [1] * N]
    for j in (0, 1, N // 8, N // 2 - 1, N // 2, N - 1):
        r = [0] * N
        r[j] = P - 1
        rows.append(r)
    rows.append([P - 1 if j % 2 else 0 for j in range(N)])
    rows.append([(P - 1) // 2 + (j % 3) for j in range(N)])
    a = np.array(rows, dtype=np.uint64)
    assert int(a[1, 0]) == P - 1
    say(f"[ntt edges] N={N} rows={len(rows)}")
    fwd = R.to_host(R.ntt_forward(R.to_device(a), N))
    L = N.bit_length() - 1
    perm = np.array([bitrev(j, L) for j in range(N)])
    for c in range(a.shape[0]):
        assert np.array_equal(fwd[c], O.ntt_forward(a[c])[perm]), c
    assert np.array_equal(R.to_host(R.ntt_inverse(R.to_device(fwd), N)), a)


@pytest.mark.parametrize("N", [256, 512, 2048, 4096])
def test_poly_mul_vs_oracle(O, torch_dev, N):
    rng = np.random.default_rng(100 + N)
    count = 3
    a = rng.integers(0, P, size=(count, N), dtype=np.uint64)
    b = rng.integers(0, P, size=(count, N), dtype=np.uint64)
    c = R.to_host(R.poly_mul(R.to_device(a), R.to_device(b), N))
    kind = O.SCHOOLBOOK if N <= 512 else O.NTT
    for i in range(count):
        assert np.array_equal(c[i], O.polymul(a[i], b[i], kind))


# ------------------------------------------------------- tiny, all stages ---

@pytest.mark.parametrize("fn", ["identity", "square_mod"])
def test_tiny_every_stage_bit_exact(O, torch_dev, fn):
    w, op, ks, bsk, ksk = keyset(O, "tiny")
    table = w.table(fn)
    v = O.test_poly(op, table)
    msgs = np.array(list(range(w.M)) * 3, dtype=np.uint32)[: 19]   # 19: ragged vs tiles of 16
    cts = O.lwe_encrypt(op, w.enc_seed, w.sigma_lwe, ks.lwe_key, msgs)
    o_out, o_big, o_acc = O.pbs(op, cts, ks.bsk, ks.ksk, v, O.SCHOOLBOOK, 0, True, True)
    d_in, d_v = R.to_device(cts), R.to_device(v)
    acc = R.to_host(R.blind_rotate(d_in, bsk, d_v, w.params()))
    assert np.array_equal(acc, o_acc)                                    # a1-a6
    big = R.blind_rotate_extract(d_in, bsk, d_v, w.params())
    assert np.array_equal(R.to_host(big), o_big)                         # a7
    assert np.array_equal(R.to_host(R.keyswitch(big, ksk, w.params())), o_out)   # a8
    out = R.to_host(R.pbs_batch(d_in, bsk, ksk, d_v, w.params()))
    assert np.array_equal(out, o_out)                                    # a1-a8
    assert np.array_equal(O.lwe_decrypt(op, ks.lwe_key, out), table[msgs])


def test_trivial_ciphertext_closed_form(O, torch_dev):
    w, op, ks, bsk, ksk = keyset(O, "tiny")
    N = w.N
    v = O.test_poly(op, w.table("square_mod"))
    bs = [0, 1, P - 1, P // 2, 12345678901234567]
    cts = np.zeros((len(bs), w.n + 1), dtype=np.uint64)
    cts[:, w.n] = bs
    acc = R.to_host(R.blind_rotate(R.to_device(cts), bsk, R.to_device(v), w.params()))
    for q, b in enumerate(bs):
        bt = O.modswitch(b, N)
        assert np.all(acc[q, :N] == 0)
        assert np.array_equal(acc[q, N:], O.monomial_mul(v, (2 * N - bt) % (2 * N)))


@pytest.mark.parametrize("batch", [1, 2, 15, 16, 17, 33])
def test_ragged_batches_and_in_place(O, torch_dev, batch):
    w, op, ks, bsk, ksk = keyset(O, "tiny")
    v = O.test_poly(op, w.table("identity"))
    msgs = (np.arange(batch) * 5 % w.M).astype(np.uint32)
    cts = O.lwe_encrypt(op, 7 + batch, w.sigma_lwe, ks.lwe_key, msgs)
    ref = O.pbs(op, cts, ks.bsk, ks.ksk, v, O.NTT)
    t = R.to_device(cts)
    R.pbs_batch(t, bsk, ksk, R.to_device(v), w.params(), out=t)         # in place
    assert np.array_equal(R.to_host(t), ref)


def test_caller_workspace_and_empty_batch(O, torch_dev):
    w, op, ks, bsk, ksk = keyset(O, "tiny")
    v = R.to_device(O.test_poly(op, w.table("identity")))
    cts = O.lwe_encrypt(op, 3, w.sigma_lwe, ks.lwe_key, np.arange(8, dtype=np.uint32))
    ref = O.pbs(op, cts, ks.bsk, ks.ksk, O.test_poly(op, w.table("identity")), O.NTT)
    ws = R.empty(R.pbs_workspace_bytes(w.params(), 8) // 8)
    out = R.pbs_batch_ws(R.to_device(cts), bsk, ksk, v, w.params(), ws)
    assert np.array_equal(R.to_host(out), ref)
    empty_in = R.empty((0, w.n + 1))
    assert R.pbs_batch(empty_in, bsk, ksk, v, w.params()).shape[0] == 0


def test_library_keys_give_same_result(O, torch_dev):
    """Keys from the library's own generator are bit-identical to the
    oracle's, so the PBS on them is too."""
    w, op, ks, bsk, ksk = keyset(O, "tiny")
    lk = R.keygen(w.key_seed, w.params(), w.sigma_lwe, w.sigma_glwe)
    bsk2 = R.bsk_prepare(R.to_device(lk["bsk"]), w.params())
    assert np.array_equal(R.to_host(bsk2), R.to_host(bsk))


# ----------------------------------------------------------- key switch ---

# (n, N, l_ks, beta_ks): the headline shape and its largest LWE dimension
# (2049 columns: a last column block of one column) on the int8 matrix
# cores, the largest digits they take (7 bits: |d| up to 64) at the
# largest ring, and two shapes the VALU kernel takes (beta_ks = 8 digits
# do not fit a signed byte; l_ks beta_ks = 32 does not fit the 31-bit
# rounding)
KS_SHAPES = {"mfma_n1024": (1024, 2048, 6, 3), "mfma_n2048": (2048, 2048, 6, 3),
             "mfma_l8_b3_n742": (742, 2048, 8, 3), "mfma_l4_b7_N4096": (1024, 4096, 4, 7),
             "valu_b8": (1024, 2048, 2, 8),
             "valu_l4_b8_n63": (63, 1024, 4, 8)}
S127 = 0x7F7F7F7F7F7F7F7F    # largest word whose 8 balanced base-256 digits fit


@pytest.mark.parametrize("name", list(KS_SHAPES))
def test_keyswitch_vs_oracle(O, torch_dev, name):
    # any key words (the key switch is linear): uniform ones with planted
    # extremes of the byte-plane encoding; inputs with rounding boundaries
    # and a batch ragged against 16-, 32- and 128-ciphertext tiles
    n, N, lks, beta = KS_SHAPES[name]
    prm = dict(n=n, k=1, N=N, pbs_level=2, pbs_base_log=8, ks_level=lks, ks_base_log=beta,
               msg_bits=2)
    op = O.Params.make(**prm)
    rng = np.random.default_rng(n + N + lks)
    ksk = rng.integers(0, P, (N * lks, n + 1), dtype=np.uint64)
    edges = [0, 1, P - 1, P - 2, S127 - 1, S127, S127 + 1, 1 << 63, P - (1 << 63) - 1,
             P - (1 << 63), (1 << 32) - 1, 1 << 32]
    flat = ksk.reshape(-1)
    pos = rng.choice(flat.size, size=4000, replace=False)
    flat[pos] = np.array(edges, dtype=np.uint64)[np.arange(pos.size) % len(edges)]
    ksk[0, :] = P - 1
    ksk[:, n] = P - 1
    batch = 131
    big = rng.integers(0, P, (batch, N + 1), dtype=np.uint64)
    s = 64 - lks * beta
    half = [(P - 1) // 2, (P + 1) // 2, 0, P - 1, 1 << (s - 1), (1 << (s - 1)) - 1,
            P - (1 << (s - 1)), 3 << (s - 1)]
    big[0, :] = P - 1
    big[1, : len(half)] = half
    big[2, :] = (P - 1) // 2
    say(f"[keyswitch {name}] GPU")
    out = R.to_host(R.keyswitch(R.to_device(big), R.ksk_prepare(R.to_device(ksk), prm), prm))
    picks = [0, 1, 2, 15, 16, 17, 31, 32, 63, 127, 128, 130]   # edge rows, tile boundaries
    say(f"[keyswitch {name}] oracle on {len(picks)} of {batch}")
    assert np.all(out < np.uint64(P))
    for q in picks:
        assert np.array_equal(out[q], O.keyswitch(op, big[q], ksk)), q


def test_keyswitch_rows_independent_of_batch_tiling(O, torch_dev):
    # the headline key-switch shape: each output row depends on its own input
    # row only, so a batch of 257 (two full 128-ciphertext workgroups and one
    # with a single live row) must equal the same rows switched in pieces of
    # 1, 31, 33, 64 and 128 (every position within a 16-, 32- and 128-row
    # tile, and workgroups with idle waves); batches of 1 and 32 and a
    # sample of the rest against the oracle
    n, N, lks, beta = 1024, 2048, 6, 3
    prm = dict(n=n, k=1, N=N, pbs_level=3, pbs_base_log=8, ks_level=lks, ks_base_log=beta,
               msg_bits=2)
    op = O.Params.make(**prm)
    rng = np.random.default_rng(257)
    ksk = rng.integers(0, P, (N * lks, n + 1), dtype=np.uint64)
    big = rng.integers(0, P, (257, N + 1), dtype=np.uint64)
    d_ksk = R.ksk_prepare(R.to_device(ksk), prm)
    say("[keyswitch tiling] GPU batch 257 and its pieces")
    whole = R.to_host(R.keyswitch(R.to_device(big), d_ksk, prm))
    parts, at = [], 0
    for size in (1, 31, 33, 64, 128):
        parts.append(R.to_host(R.keyswitch(R.to_device(big[at:at + size]), d_ksk, prm)))
        at += size
    assert at == 257
    assert np.array_equal(np.concatenate(parts), whole)
    say("[keyswitch tiling] oracle")
    for q in [0, 1, 2, 31, 32, 100, 127, 128, 255, 256]:
        assert np.array_equal(whole[q], O.keyswitch(op, big[q], ksk)), q


# ------------------------------------------------- workloads, full size ---

FULL = ["gpt2_gelu", "tinyllama_silu", "llama3_8b_silu", "llama3_8b_softmax_exp",
        "llama3_8b_softmax_recip"]
# Decryption of the key-switched output recovers T[m] except for the misses
# the noise of these parameter sets implies (binary keys, uniform modulus-
# switch rounding: the drift is about sqrt(n/24) rotation steps against half
# a box of N/2M, and the key switch adds about 2^-9 p): about 1e-30 and 2e-5
# misses for the two n = 742 sets, about 5 % at n = 1024, N = 2048, 6-bit
# messages and about 49 % at N = 4096, 7-bit messages.  The extracted
# ciphertexts (before the key switch, noise about 2^-16 p) miss only by the
# drift: about 1.4 % at n = 1024.
MIN_DECRYPT_RATE = {"gpt2_gelu": 0.9999, "tinyllama_silu": 0.999, "llama3_8b_silu": 0.94,
                    "llama3_8b_softmax_exp": 0.50, "llama3_8b_softmax_recip": 0.40}
MIN_EXTRACTED_RATE = {"gpt2_gelu": 0.9999, "tinyllama_silu": 0.999, "llama3_8b_silu": 0.98,
                      "llama3_8b_softmax_exp": 0.98, "llama3_8b_softmax_recip": 0.90}


def resident_workgroups(N: int) -> int:
    """Blind-rotation workgroups the chip holds at once (256 CUs x 3
    workgroups up to N = 2048, 2 at N = 4096): a batch runs in rounds of
    this many ciphertexts."""
    return 256 * (3 if N <= 2048 else 2)


def dense_picks(batch: int, N: int, seed: int):
    """At least 64 ciphertexts (the whole batch when it is smaller): both
    ends of the first, the second and the last residency round (the last
    one partial unless the batch is a multiple of the round), 48 evenly
    spaced across the batch, and one at random in each of up to 16 rounds
    drawn at random."""
    R = resident_workgroups(N)
    rounds = (batch + R - 1) // R
    last = (rounds - 1) * R
    picks = {0, 1, min(R - 1, batch - 1), min(R, batch - 1), min(2 * R - 1, batch - 1),
             last, min(last + 1, batch - 1), batch - 2 if batch > 1 else 0, batch - 1}
    picks |= {int(x) for x in np.linspace(0, batch - 1, 48)}
    rng = np.random.default_rng(seed)
    for r in rng.choice(rounds, size=min(16, rounds), replace=False):
        lo, hi = r * R, min(batch, (r + 1) * R)
        picks.add(int(rng.integers(lo, hi)))
    extra = iter(rng.permutation(batch))
    while len(picks) < min(64, batch):
        picks.add(int(next(extra)))
    return sorted(picks)


@pytest.mark.parametrize("name", FULL)
def test_full_workload_dense_parity(O, torch_dev, name):
    """The whole batch in the benchmark's launch configuration (blind
    rotation + extraction into one buffer, then the key switch, the two
    kernels rosetta_pbs_batch runs), compared with the oracle on at least 64
    ciphertexts spread over every residency round the batch runs in (first,
    second, last and partial last included), both the extracted and the
    key-switched ciphertexts of that one launch; then the single entry point
    on the same inputs: bit-identical to the pair (determinism across
    launches); then decryption rates over the whole batch."""
    torch = torch_dev
    w, op, ks, bsk, ksk = keyset(O, name)
    msgs = w.messages()
    say(f"[{name}] encrypt batch {w.batch}")
    cts = O.lwe_encrypt(op, w.enc_seed, w.sigma_lwe, ks.lwe_key, msgs)
    table = w.table()
    v = O.test_poly(op, table)
    d_in, d_v = R.to_device(cts), R.to_device(v)
    say(f"[{name}] GPU: blind rotation + extraction, key switch of {w.batch}")
    big_dev = R.blind_rotate_extract(d_in, bsk, d_v, w.params())
    out_dev = R.keyswitch(big_dev, ksk, w.params())
    torch.cuda.synchronize()
    big, out = R.to_host(big_dev), R.to_host(out_dev)
    del big_dev
    picks = dense_picks(w.batch, w.N, w.data_seed)
    assert len(picks) >= min(64, w.batch)
    say(f"[{name}] oracle on {len(picks)} ciphertexts over "
        f"{-(-w.batch // resident_workgroups(w.N))} residency rounds")
    ref_out, ref_big = O.pbs(op, cts[picks], ks.bsk, ks.ksk, v, O.NTT, 0, want_big=True)
    for i, q in enumerate(picks):
        assert np.array_equal(big[q], ref_big[i]), f"extracted ciphertext {q}"
        assert np.array_equal(out[q], ref_out[i]), f"key-switched ciphertext {q}"
    say(f"[{name}] GPU: rosetta_pbs_batch on the same inputs")
    again = R.to_host(R.pbs_batch(d_in, bsk, ksk, d_v, w.params()))
    assert np.array_equal(again, out), "a second launch gave other bits"
    # properties over the whole batch
    assert np.all(out < np.uint64(P)) and np.all(big < np.uint64(P))
    rate = np.mean(O.lwe_decrypt(op, ks.lwe_key, out) == table[msgs])
    rate_big = np.mean(O.lwe_decrypt(op, ks.glwe_key, big) == table[msgs])
    say(f"[{name}] decrypt = T[m]: key-switched {rate:.4%}, extracted {rate_big:.4%} "
        f"of {w.batch}")
    assert rate >= MIN_DECRYPT_RATE[name]
    assert rate_big >= MIN_EXTRACTED_RATE[name]


def test_determinism(O, torch_dev):
    w, op, ks, bsk, ksk = keyset(O, "gpt2_gelu")
    cts = O.lwe_encrypt(op, 5, w.sigma_lwe, ks.lwe_key, w.messages(512, seed=9))
    d_in, d_v = R.to_device(cts), R.to_device(O.test_poly(op, w.table()))
    a = R.to_host(R.pbs_batch(d_in, bsk, ksk, d_v, w.params()))
    b = R.to_host(R.pbs_batch(d_in, bsk, ksk, d_v, w.params()))
    assert np.array_equal(a, b)


# --------------------------------------------------- parameter corners ---

CORNERS = {
    # l*beta > 30 (64-bit rounded value) and beta > 14 (general first stage)
    "l2_b16_N1024": dict(n=32, N=1024, pbs_level=2, pbs_base_log=16, ks_level=4,
                         ks_base_log=4, msg_bits=2),
    # l*beta = 60, the most key-switching levels
    "l4_b15_N512": dict(n=16, N=512, pbs_level=4, pbs_base_log=15, ks_level=8, ks_base_log=3,
                        msg_bits=2),
    # one level of 30 bits, the smallest LWE dimension
    "l1_b30_N256_n1": dict(n=1, N=256, pbs_level=1, pbs_base_log=30, ks_level=2,
                           ks_base_log=10, msg_bits=1),
    # the largest LWE dimension
    "n2048_N2048": dict(n=2048, N=2048, pbs_level=3, pbs_base_log=8, ks_level=2, ks_base_log=8,
                        msg_bits=3),
    # the largest ring, general first stage (a batch of 3: the two-wave instance)
    "l4_b15_N4096": dict(n=24, N=4096, pbs_level=4, pbs_base_log=15, ks_level=3, ks_base_log=6,
                         msg_bits=3),
    # small-digit first stages (integer stages 0-1) at the rings no workload uses
    "l3_b8_N512": dict(n=20, N=512, pbs_level=3, pbs_base_log=8, ks_level=4, ks_base_log=4,
                       msg_bits=2),
    "l2_b14_N1024": dict(n=20, N=1024, pbs_level=2, pbs_base_log=14, ks_level=4, ks_base_log=4,
                         msg_bits=2),
    # the largest small digits (beta = 14) with a 64-bit rounded value, both rings
    # whose first pass differs (N = 256: two stages; N = 4096: three)
    "l4_b14_N4096": dict(n=8, N=4096, pbs_level=4, pbs_base_log=14, ks_level=3, ks_base_log=6,
                         msg_bits=3),
    "l3_b14_N256": dict(n=12, N=256, pbs_level=3, pbs_base_log=14, ks_level=3, ks_base_log=4,
                        msg_bits=2),
    # the headline ring (two-stage first pass, shift-twisted second pass) with
    # the general first stages (beta > 14) and a 64-bit rounded value
    "l2_b16_N2048": dict(n=16, N=2048, pbs_level=2, pbs_base_log=16, ks_level=3, ks_base_log=6,
                         msg_bits=2),
    # the headline ring with the largest small digits and a 64-bit rounded value
    "l3_b14_N2048": dict(n=12, N=2048, pbs_level=3, pbs_base_log=14, ks_level=3, ks_base_log=6,
                         msg_bits=2),
    # the largest LWE dimension on the largest ring (the most LDS a blind
    # rotation takes: 132 KiB), with the headline key switch
    "n2048_N4096": dict(n=2048, N=4096, pbs_level=3, pbs_base_log=8, ks_level=6,
                        ks_base_log=3, msg_bits=2),
}


@pytest.mark.parametrize("name", list(CORNERS))
def test_parameter_corners_bit_exact(O, torch_dev, name):
    prm = CORNERS[name]
    op = O.Params.make(**prm)
    say(f"[corner {name}] oracle keygen")
    ks = O.KeySet(op, 17, 2.0 ** -40, 2.0 ** -40)
    bsk = R.bsk_prepare(R.to_device(ks.bsk), prm | {"k": 1})
    ksk = R.ksk_prepare(R.to_device(ks.ksk), prm | {"k": 1})
    rng = np.random.default_rng(len(name))
    cts = rng.integers(0, P, (3, prm["n"] + 1), dtype=np.uint64)
    v = rng.integers(0, P, prm["N"], dtype=np.uint64)
    say(f"[corner {name}] GPU")
    out = R.to_host(R.pbs_batch(R.to_device(cts), bsk, ksk, R.to_device(v), prm | {"k": 1}))
    big = R.to_host(R.blind_rotate_extract(R.to_device(cts), bsk, R.to_device(v), prm | {"k": 1}))
    say(f"[corner {name}] oracle")
    ref_out, ref_big = O.pbs(op, cts, ks.bsk, ks.ksk, v, O.NTT, 0, want_big=True)
    assert np.array_equal(big, ref_big)
    assert np.array_equal(out, ref_out)


@pytest.mark.parametrize("level,beta", [(3, 8), (3, 15), (1, 20), (2, 16), (4, 7)])
def test_n4096_two_instances_agree(O, torch_dev, level, beta):
    """N = 4096 runs a batch that the CUs hold one workgroup each on the
    blind-rotation instance compiled for two waves per SIMD, a larger one on
    the four-wave instance (both with the accumulator in the transform
    domain, at different register budgets): the first CU-count ciphertexts
    of a batch one larger equal the same ciphertexts run alone, bit for bit
    (both kernels, extracted and key-switched), and both ends equal the
    oracle, for every level count (32- and 64-bit rounded values, digits
    through the small and the general forward transform)."""
    torch = torch_dev
    prm = dict(n=32, N=4096, pbs_level=level, pbs_base_log=beta, ks_level=3, ks_base_log=6,
               msg_bits=3, k=1)
    op = O.Params.make(**{k: v for k, v in prm.items() if k != "k"})
    ks = O.KeySet(op, 23 + beta + 100 * level, 2.0 ** -40, 2.0 ** -40)
    bsk = R.bsk_prepare(R.to_device(ks.bsk), prm)
    ksk = R.ksk_prepare(R.to_device(ks.ksk), prm)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    rng = np.random.default_rng(beta)
    cts = rng.integers(0, P, (cus + 1, prm["n"] + 1), dtype=np.uint64)
    v = rng.integers(0, P, prm["N"], dtype=np.uint64)
    d_v = R.to_device(v)
    say(f"[two instances level={level} beta={beta}] {cus + 1} and {cus} ciphertexts")
    big_all = R.to_host(R.blind_rotate_extract(R.to_device(cts), bsk, d_v, prm))
    out_all = R.to_host(R.pbs_batch(R.to_device(cts), bsk, ksk, d_v, prm))
    big_cu = R.to_host(R.blind_rotate_extract(R.to_device(cts[:cus]), bsk, d_v, prm))
    out_cu = R.to_host(R.pbs_batch(R.to_device(cts[:cus]), bsk, ksk, d_v, prm))
    assert np.array_equal(big_all[:cus], big_cu)
    assert np.array_equal(out_all[:cus], out_cu)
    pick = [0, cus - 1, cus]
    ref_out, ref_big = O.pbs(op, cts[pick], ks.bsk, ks.ksk, v, O.NTT, 0, want_big=True)
    assert np.array_equal(big_all[pick], ref_big)
    assert np.array_equal(out_all[pick], ref_out)


def test_streams(O, torch_dev):
    """Work is enqueued on the stream given: two batches on two non-default
    streams, each with its own workspace, run concurrently and each equals
    the oracle; the default-stream result is the same bits."""
    torch = torch_dev
    w, op, ks, bsk, ksk = keyset(O, "gpt2_gelu")
    v = O.test_poly(op, w.table())
    d_v = R.to_device(v)
    batches = []
    for seed, count in ((21, 300), (22, 517)):
        cts = O.lwe_encrypt(op, seed, w.sigma_lwe, ks.lwe_key, w.messages(count, seed=seed))
        batches.append(cts)
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs, ins = [], []
    for cts, st in zip(batches, streams):
        d_in = R.to_device(cts)
        ws = R.empty(R.pbs_workspace_bytes(w.params(), cts.shape[0]) // 8)
        out = R.empty((cts.shape[0], w.n + 1))
        torch.cuda.synchronize()
        R.pbs_batch_ws(d_in, bsk, ksk, d_v, w.params(), ws, out=out, stream=st)
        outs.append((out, ws))
        ins.append(d_in)
    for st in streams:
        st.synchronize()
    for (out, _), cts, d_in in zip(outs, batches, ins):
        got = R.to_host(out)
        picks = [0, cts.shape[0] // 2, cts.shape[0] - 1]
        assert np.array_equal(got[picks], O.pbs(op, cts[picks], ks.bsk, ks.ksk, v, O.NTT))
        assert np.array_equal(got, R.to_host(R.pbs_batch(d_in, bsk, ksk, d_v, w.params())))
