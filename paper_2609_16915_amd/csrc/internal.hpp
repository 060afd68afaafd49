// Internal interface between the C ABI (abi.cpp) and the kernels
// (kernels.hip).  Not installed; the public surface is include/rosetta.h.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "rosetta.h"

namespace rosetta {

// Largest LWE dimension the blind-rotation kernel accepts (its rounded
// rotation amounts are staged in LDS).
constexpr uint32_t MAX_LWE_N = 2048;

// Shape of the transform the kernels use at N = 2^logn: E = 2^ntt_le(logn)
// elements per thread, pass 0 spanning ntt_first(logn) stages and every
// later pass ntt_le(logn) (Ntt in ntt.hpp).  The twiddle table (abi.cpp)
// is laid out for exactly this shape.
constexpr int ntt_le(int logn) { return logn == 8 ? 2 : 3; }
constexpr int ntt_first(int logn) { return logn == 11 ? 2 : ntt_le(logn); }

// Per-device, per-N transform tables (device pointers) and N^-1.
struct Tables {
  // N words: zeta[m] = psi^rev(m) (zeta[0] = 1), with the regions of the
  // twisted passes holding their block powers and the stages of a last
  // pass that is not twisted stored slot-major (see ntt.hpp)
  const uint64_t *zeta;
  // N words: psi^e for e = 0 .. N-1 (psi^N = -1 gives the rest), read by the
  // blind rotation that keeps its accumulator in the transform domain
  const uint64_t *psi;
  uint64_t ninv;
};

enum BrMode { BR_GLWE = 0, BR_EXTRACT = 1 };

// Record the calling thread's error message (read by rosetta_last_error).
void set_last_error(const char *msg);

hipError_t launch_bsk_prepare(const uint64_t *bsk_std, uint64_t *bsk_dev,
                              const rosetta_params &p, const Tables &tb, hipStream_t st);
hipError_t launch_ksk_prepare(const uint64_t *ksk_std, uint64_t *ksk_dev,
                              const rosetta_params &p, hipStream_t st);
hipError_t launch_blind_rotate(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                               const uint64_t *lut, uint64_t *out, size_t batch,
                               const rosetta_params &p, const Tables &tb, BrMode mode,
                               int tp_glwe, hipStream_t st);
hipError_t launch_rows_prepare(const uint64_t *rows_std, uint64_t *rows_dev, size_t rows,
                               uint32_t N, const Tables &tb, hipStream_t st);
hipError_t launch_trace(const uint64_t *in, const uint64_t *autk_dev, uint64_t *out,
                        size_t batch, uint32_t N, int level, int base_log, const Tables &tb,
                        hipStream_t st);
hipError_t launch_glwe_mul_plain(const uint64_t *in, const uint64_t *pa_dev, const uint64_t *pb,
                                 uint64_t *out, size_t batch, int npoly, uint32_t N,
                                 const Tables &tb, hipStream_t st);
// Monomial exponents (each in [0, 2N)) passed by value to the kernels.
constexpr int MAX_MONOMIALS = 256;
struct Exponents {
  uint16_t e[MAX_MONOMIALS];
};

hipError_t launch_glwe_recombine(const uint64_t *in, uint64_t *out, size_t batch, int count,
                                 const Exponents &ex, uint32_t N, hipStream_t st);
hipError_t launch_glwe_monomial_mul(const uint64_t *in, uint64_t *out, size_t batch, int count,
                                    const Exponents &ex, uint32_t N, hipStream_t st);
hipError_t launch_sample_extract(const uint64_t *in, uint64_t *out, size_t batch, uint32_t N,
                                 hipStream_t st);

// Per-copy constants passed by value (at most MAX_MONOMIALS).
struct Consts {
  uint64_t c[MAX_MONOMIALS / 4];
};
hipError_t launch_lwe_add_consts(const uint64_t *in, uint64_t *out, size_t batch, int count,
                                int dim, const Consts &cs, hipStream_t st);
hipError_t launch_lwe_combine(const uint64_t *a, uint64_t alpha, const uint64_t *b, uint64_t beta,
                              const uint64_t *c, uint64_t gamma, uint64_t *out, size_t words,
                              hipStream_t st);
hipError_t launch_lwe_sum_groups(const uint64_t *in, uint64_t *out, size_t batch, int count,
                                 int dim, uint64_t c0, hipStream_t st);
// op as in rosetta_field_op (validated by the caller)
hipError_t launch_field_op(int op, const uint64_t *a, const uint64_t *b, const uint64_t *c,
                           uint64_t *out, size_t count, hipStream_t st);
hipError_t launch_modmul_chain(uint64_t seed, uint32_t threads, uint32_t iters, uint64_t *out,
                               hipStream_t st);
hipError_t launch_keyswitch(const uint64_t *big, const uint64_t *ksk_dev, uint64_t *out,
                            size_t batch, const rosetta_params &p, hipStream_t st);

// The key switch is one integer matrix product over the batch (digits x
// key), run on the int8 matrix cores when the signed digits fit a byte
// (|d| <= 2^(beta_ks-1) <= 64), the rounded value 31 bits (l_ks beta_ks
// <= 30), N is a multiple of 32 (whole 32-deep k blocks), and no int32 sum
// of N l_ks digit x key-byte products can overflow (N l_ks 2^(beta_ks-1)
// 128 < 2^31).  Otherwise the VALU kernel runs.  The prepared key's layout
// follows the choice (launch_ksk_prepare).
inline bool ks_on_matrix_cores(const rosetta_params &p) {
  if (p.ks_base_log < 1 || p.ks_base_log > 7 || p.ks_level < 1) return false;
  if (p.ks_level * p.ks_base_log > 30 || p.N % 32 != 0) return false;
  const uint64_t bound = (uint64_t)p.N * p.ks_level * (1ull << (p.ks_base_log - 1)) * 128;
  return bound < (1ull << 31);
}
// Words of the byte-plane key: ceil((n+1)/32) column blocks x N l_ks / 32
// k blocks x 1024 words (16 operand fragments of 64 lanes x 8 bytes).
inline size_t ks_matrix_key_words(const rosetta_params &p) {
  return (size_t)((p.n + 1 + 31) / 32) * ((size_t)p.N * p.ks_level / 32) * 1024;
}
hipError_t launch_ntt(const uint64_t *in, uint64_t *out, size_t count, uint32_t N,
                      const Tables &tb, bool inverse, hipStream_t st);
hipError_t launch_poly_mul(const uint64_t *a, const uint64_t *b, uint64_t *c, size_t count,
                           uint32_t N, const Tables &tb, hipStream_t st);

}  // namespace rosetta
