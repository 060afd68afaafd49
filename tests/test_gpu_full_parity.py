"""Whole-batch parity, opt in: every ciphertext of a workload's batch (or of a
range of it), in the benchmark's launch configuration (blind rotation +
extraction into one buffer, then the key switch), against the oracle, both
the extracted and the key-switched ciphertexts.

The oracle costs about 1.3 s per PBS per host thread at the headline shape, so
this runs only when asked for, with ROSETTA_FULL_PARITY=<workload>,
<workload>:<start>:<stop> (ciphertexts start..stop-1) or
<workload>:<start>:<stop>:<step> (every step-th of them, a sample that reaches
every residency round of a batch too large to recompute whole); the GPU still
runs the whole batch, so that every ciphertext is checked in the launch the
benchmark times.  The oracle works through the range in chunks and reports
each one, so that a long range shows progress."""
import os
import time

import numpy as np
import pytest

from gpu_helpers import keyset, require_gpu, say
from paper_2609_16915_amd import rosetta as R

pytestmark = pytest.mark.gpu
SPEC = os.environ.get("ROSETTA_FULL_PARITY", "")
CHUNK = 128


def _threads():
    env = os.environ.get("OMP_NUM_THREADS")
    return int(env) if env and env.isdigit() else len(os.sched_getaffinity(0))


@pytest.mark.skipif(not SPEC, reason="opt-in: ROSETTA_FULL_PARITY=<workload>[:<start>:<stop>[:<step>]]")
def test_whole_batch_bit_exact(O):
    torch = require_gpu()
    name, *rng = SPEC.split(":")
    w, op, ks, bsk, ksk = keyset(O, name)
    start, stop = (int(rng[0]), int(rng[1])) if rng else (0, w.batch)
    step = int(rng[2]) if len(rng) > 2 else 1
    stop = min(stop, w.batch)
    assert 0 <= start < stop and step >= 1
    idx = np.arange(start, stop, step)
    cts = O.lwe_encrypt(op, w.enc_seed, w.sigma_lwe, ks.lwe_key, w.messages())
    v = O.test_poly(op, w.table())
    say(f"[{name}] GPU: blind rotation + extraction, key switch of {w.batch}")
    big_dev = R.blind_rotate_extract(R.to_device(cts), bsk, R.to_device(v), w.params())
    out_dev = R.keyswitch(big_dev, ksk, w.params())
    torch.cuda.synchronize()
    big, out = R.to_host(big_dev), R.to_host(out_dev)
    nt = _threads()
    t0 = time.perf_counter()
    fbsk = O.bsk_transform(op, ks.bsk, nt)
    say(f"[{name}] oracle key transform {time.perf_counter() - t0:.1f} s; {len(idx)} ciphertexts "
        f"{start}..{stop - 1} step {step} on {nt} threads")
    for c0 in range(0, len(idx), CHUNK):
        part = idx[c0:c0 + CHUNK]
        ref_out, ref_big = O.pbs_prepared(op, cts[part], fbsk, ks.ksk, v, nt, want_big=True)
        bad_big = [int(q) for i, q in enumerate(part) if not np.array_equal(big[q], ref_big[i])]
        bad_out = [int(q) for i, q in enumerate(part) if not np.array_equal(out[q], ref_out[i])]
        say(f"[{name}] {c0 + len(part)}/{len(idx)} compared, {time.perf_counter() - t0:.0f} s")
        assert not bad_big, f"extracted ciphertexts differ: {bad_big[:8]}"
        assert not bad_out, f"key-switched ciphertexts differ: {bad_out[:8]}"
