"""Seeded synthetic workloads for batched PBS.

This module is the shared input generator: parameter sets, seeded activation
samples, their quantisation to LUT indices, and the LUT tables themselves
(function values rounded to the message grid).  It holds none of the PBS
arithmetic (no encryption, no encoding into a test polynomial, nothing mod p)
and imports nothing from the rest of the package, so the oracle tests and the
GPU path can both take their inputs from it.

Workloads (one decode step of the models in the paper's model table; the
parameter sets follow the paper's TFHE setting of n_LWE = 1024, N_br = 2048 in
Sec. 5 "Cryptographic Configuration", with the ciphertext modulus replaced by
the Goldilocks prime):

  tiny                  n=64,   N=256,  l=2 beta=8,  KS 3x4, 3-bit messages,
                        identity and m^2 mod 8 tables, batch 8
  gpt2_gelu             n=742,  N=2048, l=2 beta=10, KS 5x3, 4-bit, GELU on
                        [-4,4), batch 3072 = GPT-2 FFN width 4*768
  tinyllama_silu        as gpt2_gelu, 5-bit, SiLU on [-8,8), batch 5632
  llama3_8b_silu        n=1024, N=2048, l=3 beta=8,  KS 6x3, 6-bit, SiLU on
                        [-8,8), batch 14336 = LLaMA-3-8B FFN width
  llama3_8b_softmax_exp n=1024, N=4096, l=3 beta=8,  KS 6x3, 7-bit, exp on
                        [-16,0] of scores minus the row max, batch 65536 =
                        32 heads x 2048 context; plus a 32-element reciprocal
                        batch over the row sums.
  llama3_8b_lookup      keys of the lookup protocol (Algorithm 1): n=1024,
                        N=2048, l=3 beta=14, KS 8x2, batch 14336.

LUT semantics (Sec. 3.1, single uniform LUT): the input range is cut into M
equal intervals; index m = clamp(floor((x - lo) / dx), 0, M-1) and the entry
stores f at the interval midpoint c_m = lo + (m + 1/2) dx, rounded to the same
grid (or, for exp and 1/x, scaled to 7-bit integers).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n: int
    N: int
    pbs_level: int
    pbs_base_log: int
    ks_level: int
    ks_base_log: int
    msg_bits: int
    batch: int
    sigma_lwe: float      # noise standard deviation as a fraction of p
    sigma_glwe: float
    key_seed: int
    enc_seed: int
    data_seed: int
    function: str         # LUT function name
    lo: float = 0.0       # input interval [lo, lo + M*dx)
    dx: float = 1.0
    act_sigma: float = 1.0

    @property
    def M(self) -> int:
        return 1 << self.msg_bits

    def params(self) -> dict:
        return dict(n=self.n, k=1, N=self.N, pbs_level=self.pbs_level,
                    pbs_base_log=self.pbs_base_log, ks_level=self.ks_level,
                    ks_base_log=self.ks_base_log, msg_bits=self.msg_bits)

    # ---- sizes (64-bit words) ------------------------------------------
    def bsk_words(self) -> int:
        return self.n * 2 * self.pbs_level * 2 * self.N

    def ksk_words(self) -> int:
        return self.N * self.ks_level * (self.n + 1)

    # ---- algorithmic work (radix-2 transform counts) --------------------
    def br_modmul_per_pbs(self) -> int:
        """Modular multiplications of one blind rotation with radix-2 NTTs:
        n steps x [(2l forward + 2 inverse) x (N/2) log2 N butterflies
        + 4 l N pointwise products]."""
        L = int(math.log2(self.N))
        return self.n * ((2 * self.pbs_level + 2) * (self.N // 2) * L
                         + 4 * self.pbs_level * self.N)

    def ks_mac_per_pbs(self) -> int:
        return self.N * self.ks_level * (self.n + 1)

    def trace_modmul(self, level: int) -> int:
        """Modular multiplications of one RLWE trace: 2N for the N^-1
        scaling, then log2 N rounds of [(level forward + 2 inverse) x
        (N/2) log2 N butterflies + 2 level N pointwise products]."""
        L = int(math.log2(self.N))
        return 2 * self.N + L * ((level + 2) * (self.N // 2) * L + 2 * level * self.N)

    def autk_words(self, level: int) -> int:
        return int(math.log2(self.N)) * level * 2 * self.N

    # ---- seeded inputs ---------------------------------------------------
    def messages(self, count: int | None = None, seed: int | None = None) -> np.ndarray:
        """Quantised activations (LUT indices in [0, M)) for `count` inputs."""
        count = self.batch if count is None else count
        rng = np.random.default_rng(self.data_seed if seed is None else seed)
        if self.function in ("identity", "square_mod"):
            return rng.integers(0, self.M, size=count, dtype=np.int64).astype(np.uint32)
        if self.function == "exp":
            # scores z ~ N(0, act_sigma^2) per row of 2048, minus the row max
            rows = max(1, count // 2048) if count >= 2048 else 1
            per = count // rows if count >= 2048 else count
            z = rng.normal(0.0, self.act_sigma, size=(rows, per))
            x = (z - z.max(axis=1, keepdims=True)).reshape(-1)[:count]
            x = np.clip(x, self.lo, 0.0)
        elif self.function == "recip":
            x = rng.uniform(1.0, 64.0, size=count)
        else:
            x = np.clip(rng.normal(0.0, self.act_sigma, size=count), -8.0, 8.0)
        return self.quantize(x)

    def quantize(self, x: np.ndarray) -> np.ndarray:
        m = np.floor((np.asarray(x, dtype=np.float64) - self.lo) / self.dx)
        return np.clip(m, 0, self.M - 1).astype(np.uint32)

    def midpoints(self) -> np.ndarray:
        return self.lo + (np.arange(self.M) + 0.5) * self.dx

    def table(self, function: str | None = None) -> np.ndarray:
        """LUT entries T[0..M) (integers in [0, M))."""
        f = self.function if function is None else function
        M = self.M
        m = np.arange(M)
        if f == "identity":
            return m.astype(np.uint32)
        if f == "square_mod":
            return ((m * m) % M).astype(np.uint32)
        c = self.midpoints()
        if f == "gelu":
            y = 0.5 * c * (1.0 + np.array([math.erf(v / math.sqrt(2.0)) for v in c]))
            return self.quantize(y)
        if f == "silu":
            y = c / (1.0 + np.exp(-c))
            return self.quantize(y)
        if f == "exp":
            return np.clip(np.rint(127.0 * np.exp(c)), 0, M - 1).astype(np.uint32)
        if f == "recip":
            return np.clip(np.rint(127.0 / np.maximum(c, 1.0)), 0, M - 1).astype(np.uint32)
        raise ValueError(f"unknown LUT function {f!r}")


_S17 = 2.0 ** -17
_S51 = 2.0 ** -51

WORKLOADS: dict[str, Workload] = {
    "tiny": Workload("tiny", n=64, N=256, pbs_level=2, pbs_base_log=8, ks_level=3,
                     ks_base_log=4, msg_bits=3, batch=8, sigma_lwe=2.0 ** -40,
                     sigma_glwe=2.0 ** -40, key_seed=1, enc_seed=101, data_seed=201,
                     function="identity"),
    "gpt2_gelu": Workload("gpt2_gelu", n=742, N=2048, pbs_level=2, pbs_base_log=10, ks_level=5,
                          ks_base_log=3, msg_bits=4, batch=3072, sigma_lwe=_S17,
                          sigma_glwe=_S51, key_seed=2, enc_seed=102, data_seed=202,
                          function="gelu", lo=-4.0, dx=0.5, act_sigma=1.0),
    "tinyllama_silu": Workload("tinyllama_silu", n=742, N=2048, pbs_level=2, pbs_base_log=10,
                               ks_level=5, ks_base_log=3, msg_bits=5, batch=5632,
                               sigma_lwe=_S17, sigma_glwe=_S51, key_seed=3, enc_seed=103,
                               data_seed=203, function="silu", lo=-8.0, dx=0.5,
                               act_sigma=1.5),
    "llama3_8b_silu": Workload("llama3_8b_silu", n=1024, N=2048, pbs_level=3, pbs_base_log=8,
                               ks_level=6, ks_base_log=3, msg_bits=6, batch=14336,
                               sigma_lwe=_S17, sigma_glwe=_S51, key_seed=4, enc_seed=104,
                               data_seed=204, function="silu", lo=-8.0, dx=0.25,
                               act_sigma=1.0),
    "llama3_8b_softmax_exp": Workload("llama3_8b_softmax_exp", n=1024, N=4096, pbs_level=3,
                                      pbs_base_log=8, ks_level=6, ks_base_log=3, msg_bits=7,
                                      batch=65536, sigma_lwe=_S17, sigma_glwe=_S51, key_seed=5,
                                      enc_seed=105, data_seed=205, function="exp", lo=-16.0,
                                      dx=0.125, act_sigma=3.0),
    # reciprocal of the 32 softmax row sums, at the exp workload's parameters
    "llama3_8b_softmax_recip": Workload("llama3_8b_softmax_recip", n=1024, N=4096,
                                        pbs_level=3, pbs_base_log=8, ks_level=6, ks_base_log=3,
                                        msg_bits=7, batch=32, sigma_lwe=_S17, sigma_glwe=_S51,
                                        key_seed=5, enc_seed=106, data_seed=206,
                                        function="recip", lo=0.0, dx=0.5),
    # the lookup protocol of Algorithm 1 at the LLaMA-3-8B FFN width: the
    # headline ring and LWE dimension with 14-bit gadget digits (the blind
    # rotation's noise on a selected value drops from about 2^48 to 2^37
    # absolute at the same cost) and an 8 x 2-bit key switch (smaller
    # noise on the selectors S and I)
    "llama3_8b_lookup": Workload("llama3_8b_lookup", n=1024, N=2048, pbs_level=3,
                                 pbs_base_log=14, ks_level=8, ks_base_log=2, msg_bits=6,
                                 batch=14336, sigma_lwe=_S17, sigma_glwe=_S51, key_seed=7,
                                 enc_seed=107, data_seed=207, function="silu", lo=-8.0,
                                 dx=0.25, act_sigma=1.0),
}

# The headline workload (LLaMA-3-8B FFN SiLU, N = 2048, batch 14336).
HEADLINE = "llama3_8b_silu"


def get(name: str) -> Workload:
    return WORKLOADS[name]
