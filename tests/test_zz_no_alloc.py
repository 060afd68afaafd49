"""rosetta_pbs_batch_noalloc (the allocation-free PBS entry point) against
rosetta_pbs_batch, through the C ABI: two calls in a row, the second on a
smaller batch, bit for bit; the tiny workload also against the oracle; and
the host-side rejection of a batch whose scratch exceeds the static array."""
import ctypes as C

import numpy as np
import pytest

from paper_2609_16915_amd import rosetta as R
from paper_2609_16915_amd import workloads as W

from gpu_helpers import keyset, oparams, require_gpu, say

pytestmark = pytest.mark.gpu
P = R.P


def _random_keys(torch, w, seed):
    """Uniform words in [0, p) as standard-layout keys, prepared on the device
    (both entry points run the same kernels on them; any canonical words are
    valid input)."""
    rng = np.random.default_rng(seed)
    bsk_std = R.to_device(rng.integers(0, P, size=w.bsk_words(), dtype=np.uint64))
    ksk_std = R.to_device(rng.integers(0, P, size=w.ksk_words(), dtype=np.uint64))
    bsk = R.bsk_prepare(bsk_std, w.params())
    ksk = R.ksk_prepare(ksk_std, w.params())
    del bsk_std, ksk_std
    return bsk, ksk


@pytest.mark.parametrize("name,batches", [("llama3_8b_silu", (1500, 333)),
                                          ("llama3_8b_softmax_exp", (700, 129)),
                                          ("gpt2_gelu", (4094, 1))])
def test_noalloc_equals_pbs_batch(name, batches):
    torch = require_gpu()
    w = W.get(name)
    say(f"[noalloc] {name} batches {batches}")
    bsk, ksk = _random_keys(torch, w, 31 + w.N)
    rng = np.random.default_rng(7 + w.n)
    lut = R.to_device(rng.integers(0, P, size=w.N, dtype=np.uint64))
    for batch in batches:
        lwe = R.to_device(rng.integers(0, P, size=(batch, w.n + 1), dtype=np.uint64))
        out_na = R.empty((batch, w.n + 1))
        out_na.fill_(0)
        R.pbs_batch_noalloc(lwe, bsk, ksk, lut, w.params(), out_na)
        ref = R.pbs_batch(lwe, bsk, ksk, lut, w.params())
        torch.cuda.synchronize()
        a, b = R.to_host(out_na), R.to_host(ref)
        assert np.array_equal(a, b), f"{name} batch {batch}: noalloc differs from pbs_batch"
        say(f"[noalloc] {name} batch {batch}: equal")


def test_noalloc_tiny_against_oracle(O):
    torch = require_gpu()
    w, op, ks, bsk, ksk = keyset(O, "tiny")
    v = O.test_poly(op, w.table("square_mod"))
    lut = R.to_device(v)
    for count, seed in ((33, 5), (5, 6)):
        msgs = w.messages(count, seed=seed)
        cts = O.lwe_encrypt(op, 1000 + seed, w.sigma_lwe, ks.lwe_key, msgs)
        ref = O.pbs(op, cts, ks.bsk, ks.ksk, v, O.SCHOOLBOOK)
        out = R.empty((count, w.n + 1))
        R.pbs_batch_noalloc(R.to_device(cts), bsk, ksk, lut, w.params(), out)
        torch.cuda.synchronize()
        assert np.array_equal(R.to_host(out), ref)


def test_noalloc_rejects_batch_beyond_scratch():
    torch = require_gpu()
    w = W.get("llama3_8b_silu")
    p = R.Params.from_dict(w.params())
    max_batch = R.NOALLOC_SCRATCH_BYTES // ((w.N + 1) * 8)
    assert max_batch == 4094
    dummy = R.empty(16)
    ptr = dummy.data_ptr()
    # validated on the host before anything is enqueued: no kernel reads the
    # (too small) buffers
    st = R.lib().rosetta_pbs_batch_noalloc(ptr, ptr + 8, ptr + 16, ptr + 24, ptr + 32,
                                           max_batch + 1, C.byref(p), None)
    assert R.STATUS[st] == "ROSETTA_ERR_SIZE"
    assert b"4094" in R.lib().rosetta_last_error()
    assert R.lib().rosetta_pbs_batch_noalloc(ptr, ptr, ptr, ptr, ptr, 0, C.byref(p), None) == 0
