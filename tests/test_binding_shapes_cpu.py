"""The binding's size checks, on the CPU: every device wrapper compares the
element counts of its buffers with what the parameters imply and raises
ValueError before any library call, so that a wrongly sized buffer never
reaches a kernel.  CPU tensors stand in for device buffers: a wrapper whose
sizes are right goes on to its device check and raises TypeError there,
which shows that the size check let it through and that nothing ran."""
import numpy as np
import pytest
import torch

from paper_2609_16915_amd import rosetta as R
from paper_2609_16915_amd import workloads as W

W_TINY = W.get("tiny")
PRM = W_TINY.params()
p = R.Params.from_dict(PRM)
N, n = p.N, p.n


def z(words):
    return torch.zeros(int(words), dtype=torch.uint64)


@pytest.fixture(scope="module")
def sizes():
    R.lib()
    return dict(bsk=R.bsk_words(p), ksk=R.ksk_words(p), kskd=R.ksk_device_words(p))


def test_pbs_family(sizes):
    b = 5
    good = (z(b * (n + 1)), z(sizes["bsk"]), z(sizes["kskd"]), z(N))
    with pytest.raises(TypeError):  # sizes fine: stops at the device check
        R.pbs_batch(*good, PRM)
    for i, name in enumerate(("lwe_in", "bsk_dev", "ksk_dev", "lut")):
        bad = list(good)
        bad[i] = z(_words_off(good[i], n + 1 if i == 0 else 1))
        with pytest.raises(ValueError, match=name):
            R.pbs_batch(*bad, PRM)
        with pytest.raises(ValueError, match=name):
            R.pbs_batch_noalloc(*bad, PRM, z(b * (n + 1)))
        with pytest.raises(ValueError, match=name):
            R.pbs_batch_ws(*bad, PRM, z(b * (N + 1)))
    with pytest.raises(ValueError, match="lwe_out"):
        R.pbs_batch(*good, PRM, out=z(b * (n + 1) - 1))
    with pytest.raises(ValueError, match="lwe_out"):
        R.pbs_batch_noalloc(*good, PRM, z(b * (n + 1) + 1))
    with pytest.raises(ValueError, match="workspace"):
        R.pbs_batch_ws(*good, PRM, z(b * (N + 1) - 1))
    with pytest.raises(TypeError):
        R.pbs_batch_ws(*good, PRM, z(b * (N + 1)))


def _words_off(t, row):
    """A size that is wrong for `t`: one row short when rows are longer than
    a word, else one word short."""
    return max(0, t.numel() - 1) if row == 1 else t.numel() + 1


def test_blind_rotation_and_keyswitch(sizes):
    b = 3
    lwe, bsk, lut = z(b * (n + 1)), z(sizes["bsk"]), z(N)
    with pytest.raises(ValueError, match="glwe_out"):
        R.blind_rotate(lwe, bsk, lut, PRM, out=z(b * 2 * N - 1))
    with pytest.raises(ValueError, match="big_out"):
        R.blind_rotate_extract(lwe, bsk, lut, PRM, out=z(b * (N + 1) + 1))
    with pytest.raises(ValueError, match="bsk_dev"):
        R.blind_rotate_extract(lwe, z(sizes["bsk"] - N), lut, PRM)
    with pytest.raises(ValueError, match="lwe_in"):
        R.blind_rotate(z(b * (n + 1) + 2), bsk, lut, PRM)
    with pytest.raises(TypeError):
        R.blind_rotate(lwe, bsk, lut, PRM, out=z(b * 2 * N))
    with pytest.raises(ValueError, match="big_in"):
        R.keyswitch(z(b * (N + 1) - 1), z(sizes["kskd"]), PRM)
    with pytest.raises(ValueError, match="ksk_dev"):
        R.keyswitch(z(b * (N + 1)), z(sizes["ksk"]), PRM)   # standard, not prepared, size
    with pytest.raises(ValueError, match="lwe_out"):
        R.keyswitch(z(b * (N + 1)), z(sizes["kskd"]), PRM, out=z(b * (n + 1) - 1))
    with pytest.raises(TypeError):
        R.keyswitch(z(b * (N + 1)), z(sizes["kskd"]), PRM)


def test_key_preparation(sizes):
    with pytest.raises(ValueError, match="bsk_std"):
        R.bsk_prepare(z(sizes["bsk"] - 1), PRM)
    with pytest.raises(ValueError, match="bsk_dev"):
        R.bsk_prepare(z(sizes["bsk"]), PRM, out=z(sizes["bsk"] + 8))
    with pytest.raises(ValueError, match="ksk_std"):
        R.ksk_prepare(z(sizes["kskd"]), PRM)
    with pytest.raises(ValueError, match="ksk_dev"):
        R.ksk_prepare(z(sizes["ksk"]), PRM, out=z(sizes["ksk"]))
    with pytest.raises(TypeError):
        R.bsk_prepare(z(sizes["bsk"]), PRM, out=z(sizes["bsk"]))


def test_transforms_and_field_ops():
    with pytest.raises(ValueError, match="in"):
        R.ntt_forward(z(N + 1), N)
    with pytest.raises(ValueError, match="out"):
        R.ntt_inverse(z(2 * N), N, out=z(N))
    with pytest.raises(ValueError, match="b"):
        R.poly_mul(z(2 * N), z(N), N)
    with pytest.raises(ValueError, match="c"):
        R.poly_mul(z(N), z(N), N, out=z(2 * N))
    with pytest.raises(ValueError, match="b"):
        R.field_op(R.FIELD_ADD, z(10), z(9))
    with pytest.raises(ValueError, match="c"):
        R.field_op(R.FIELD_MUL_ADD, z(10), z(10), z(11))
    with pytest.raises(ValueError, match="out"):
        R.field_op(R.FIELD_MUL, z(10), z(10), out=z(8))
    with pytest.raises(ValueError, match="out"):
        R.modmul_chain(1, 300, 4, out=z(299))
    with pytest.raises(TypeError):
        R.ntt_forward(z(2 * N), N)


def test_lookup_primitives(sizes):
    b, g = 2, 3
    lwe, bsk = z(b * (n + 1)), z(sizes["bsk"])
    with pytest.raises(ValueError, match="glwe_tp"):
        R.blind_rotate_glwe(lwe, bsk, z(b * 2 * N), PRM, group=g)
    with pytest.raises(ValueError, match="out"):
        R.blind_rotate_glwe(lwe, bsk, z(b * g * 2 * N), PRM, group=g, extract=True,
                            out=z(b * g * 2 * N))
    with pytest.raises(TypeError):
        R.blind_rotate_glwe(lwe, bsk, z(b * g * 2 * N), PRM, group=g)
    with pytest.raises(ValueError, match="lwe_out"):
        R.lwe_add_consts(z(b * (n + 1)), np.arange(4), n, out=z(b * 3 * (n + 1)))
    with pytest.raises(ValueError, match="lwe_in"):
        R.lwe_sum_groups(z(b * 4 * (n + 1) + 1), 4, n)
    aw = R.autk_words(p, 2)
    with pytest.raises(ValueError, match="autk_std"):
        R.autk_prepare(z(aw - 1), PRM, 2)
    with pytest.raises(ValueError, match="autk_dev"):
        R.trace(z(b * 2 * N), z(aw), PRM, 3, 10)        # key built for 2 levels
    with pytest.raises(ValueError, match="glwe_out"):
        R.trace(z(b * 2 * N), z(aw), PRM, 2, 10, out=z(2 * N))
    with pytest.raises(ValueError, match="plain_prep"):
        R.plain_prepare(z(3 * N), N, out=z(2 * N))
    with pytest.raises(ValueError, match="pb"):
        R.glwe_mul_plain(z(b * 2 * N), z(2 * N), z(N), N)
    with pytest.raises(ValueError, match="glwe_out"):
        R.glwe_mul_plain(z(b * 2 * N), z(2 * N), None, N, out=z(b * 2 * N))
    with pytest.raises(ValueError, match="glwe_in"):
        R.glwe_recombine(z(b * 2 * N * 3 + N), 3, N)
    with pytest.raises(ValueError, match="glwe_out"):
        R.glwe_monomial_mul(z(b * 2 * N), [1, 2], N, out=z(b * 2 * N))
    with pytest.raises(ValueError, match="big_out"):
        R.sample_extract(z(b * 2 * N), N, out=z(b * N))
