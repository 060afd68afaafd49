"""Shared pieces of the GPU test modules: progress output, the torch
fixture's check, oracle parameters and a per-process cache of oracle key
material with the matching prepared device keys."""
import sys

from paper_2609_16915_amd import rosetta as R
from paper_2609_16915_amd import workloads as W

P = 0xFFFFFFFF00000001


def say(*a):
    print(*a, flush=True, file=sys.stderr)


def require_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    R.lib()
    return torch


def bitrev(x, bits):
    return int(format(x, f"0{bits}b")[::-1], 2)


def oparams(O, w):
    return O.Params.make(**{k: v for k, v in w.params().items() if k != "k"})


_keys = {}


def keyset(O, name):
    """Oracle key material and prepared device keys for a workload."""
    if name not in _keys:
        w = W.get(name)
        op = oparams(O, w)
        say(f"[keys] oracle keygen {name} n={w.n} N={w.N}")
        ks = O.KeySet(op, w.key_seed, w.sigma_lwe, w.sigma_glwe)
        bsk_std = R.to_device(ks.bsk)
        ksk_std = R.to_device(ks.ksk)
        bsk = R.bsk_prepare(bsk_std, w.params())
        ksk = R.ksk_prepare(ksk_std, w.params())
        del bsk_std, ksk_std
        _keys[name] = (w, op, ks, bsk, ksk)
    return _keys[name]
