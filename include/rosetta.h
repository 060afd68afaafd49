/*
 * rosetta.h - batched TFHE programmable bootstrapping on AMD Instinct MI355X
 * (gfx950), over the Goldilocks prime p = 2^64 - 2^32 + 1.
 *
 * The operation is the one the ROSETTA paper (arXiv 2609.16915) builds its
 * nonlinear layers on, Sec. 2.2 "TFHE Scheme", PBS paragraph and
 * Fig. rlwe_primitives(a): a lookup table f is written into the coefficients
 * of a test polynomial v(X) in Z_p[X]/(X^N + 1); blind rotation turns an LWE
 * encryption of m into a GLWE encryption of X^(-m) v(X), whose constant
 * term f(m) is extracted (Sec. 2.2.3, LWE Extract) into a fresh LWE
 * ciphertext.  A final key switch brings it back under the input key, so
 * outputs can be bootstrapped again.
 *
 * CONVENTIONS (they decide every output bit; the paper leaves them open):
 *  - Modulus q = Q = p for LWE and GLWE.  Values are canonical, in [0, p).
 *  - LWE ciphertext of dimension d: (a_0, ..., a_{d-1}, b), phase b - <a, s>.
 *  - GLWE ciphertext (k = 1): (A[0..N), B[0..N)), phase B - A*S.
 *  - Messages m in Z_M, M = 2^msg_bits, with one padding bit: plaintext
 *    Delta*m, Delta = floor(p / 2M).  Decryption rounds 2M*phase/p.
 *  - Modulus switch: a~ = floor((2N a + (p-1)/2) / p) mod 2N.
 *  - Blind rotation: ACC = (0, X^(-b~) v); for i = 0..n-1 ascending,
 *    ACC += GGSW_i (x) (X^(a~_i) ACC - ACC)   (CMux form).
 *  - Gadget decomposition of a in Z_p, l levels of base B = 2^beta: centred
 *    representative a_c, r = floor((a_c + 2^(s-1)) / 2^s) with s = 64 - l beta,
 *    balanced digits d_t in [-B/2, B/2) for t = l-1..1, top digit d_0 = the
 *    remaining carry; digit t pairs with g_t = 2^(64 - (t+1) beta).
 *  - Bootstrapping key (standard layout) [i < n][u < 2][t < l][c < 2][x < N]:
 *    row (u, t) of GGSW_i is a GLWE encryption of 0 with s_i g_t added to the
 *    constant coefficient of component u (0 = mask, 1 = body).
 *  - Sample extraction: a'_0 = A_0, a'_j = -A_{N-j}, b' = B_0.
 *  - Key switching: out = (0, .., 0, b') - sum_{j<N, t<l_ks} d_{j,t} KSK[j][t]
 *    with d = Dec(a'_j; l_ks, beta_ks); key-switching key (standard layout)
 *    [j < N][t < l_ks][0..n], row (j, t) an LWE encryption of S_j g^ks_t.
 *  - Test polynomial for a table T[0..M) (entries in Z_2M), box = N/M,
 *    h = floor(box/2): v_j = Delta T[floor((j+h)/box)] for j < N - h and
 *    v_j = -Delta T[0] for j >= N - h.
 *
 * MEMORY AND STREAMS.  Device pointers are plain HIP device addresses; the
 * caller owns every buffer.  `stream` is a hipStream_t passed as void*
 * (NULL: the default stream).  Calls that take device pointers only enqueue
 * work and return; results are ready once the stream is synchronised.  A
 * device-side fault surfaces at that synchronisation, not in the status.
 * Inputs not in [0, p) are a precondition violation: the output is then
 * unspecified, but every memory access stays in bounds.
 *
 * ERRORS.  Every call returns a rosetta_status; nothing throws across the
 * ABI.  Arguments are validated on the host before anything is enqueued; on
 * error nothing is enqueued and rosetta_last_error() (thread-local) holds a
 * message.  batch == 0 (count == 0) is a successful no-op once the
 * parameters are valid; pointers are then not inspected.
 *
 * Supported parameters: k = 1; N in {256, 512, 1024, 2048, 4096};
 * 1 <= n <= 2048; 1 <= l <= 4, beta <= 30, l*beta <= 62; 1 <= l_ks <= 8,
 * beta_ks <= 30, l_ks*beta_ks <= 62, N * l_ks * 2^beta_ks < 2^32;
 * 1 <= msg_bits <= 20, 2^msg_bits <= N.
 */
#ifndef ROSETTA_H
#define ROSETTA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rosetta_params {
  uint32_t n;            /* LWE dimension */
  uint32_t k;            /* GLWE dimension; must be 1 */
  uint32_t N;            /* ring degree (power of two, 256..4096) */
  uint32_t pbs_level;    /* l */
  uint32_t pbs_base_log; /* beta */
  uint32_t ks_level;     /* l_ks */
  uint32_t ks_base_log;  /* beta_ks */
  uint32_t msg_bits;     /* log2 M */
} rosetta_params;

typedef enum rosetta_status {
  ROSETTA_OK = 0,
  ROSETTA_ERR_NULL = 1,        /* a required pointer is NULL */
  ROSETTA_ERR_PARAMS = 2,      /* inconsistent parameters */
  ROSETTA_ERR_UNSUPPORTED = 3, /* valid but outside what the kernels support */
  ROSETTA_ERR_ALIAS = 4,       /* partially overlapping input and output */
  ROSETTA_ERR_NOMEM = 5,       /* device allocation failed */
  ROSETTA_ERR_DEVICE = 6,      /* a HIP call failed */
  ROSETTA_ERR_SIZE = 7         /* a caller-provided buffer is too small */
} rosetta_status;

/* Library version string, ending in "src:" and the first 16 hex digits of
 * the SHA-256 of the sources the library was compiled from (every file of
 * csrc/ and this header, each as its path then its bytes, in path order),
 * so that a loaded library names the sources behind it. */
const char *rosetta_version(void);

/* Name of a status code. */
const char *rosetta_status_string(int status);

/* Message for the last error returned on the calling thread ("" if none). */
const char *rosetta_last_error(void);

/* Validate a parameter set (ROSETTA_OK, _PARAMS or _UNSUPPORTED). */
rosetta_status rosetta_check_params(const rosetta_params *params);

/* Sizes in 64-bit words.  The standard and the device (prepared) layouts of
 * the bootstrapping key have the same size, n*2*l*2*N.  The standard
 * key-switching key is N*l_ks*(n+1) words.  Its prepared layout depends on
 * the parameters: where the key switch runs on the int8 matrix cores
 * (beta_ks <= 7, l_ks*beta_ks <= 30, N a multiple of 32 and
 * N*l_ks*2^(beta_ks-1)*128 < 2^31) it is the key's 8 signed byte planes,
 * ceil((n+1)/32) * (N*l_ks/32) * 1024 words; otherwise the key words plus
 * n+1 column sums. */
size_t rosetta_bsk_words(const rosetta_params *params);
size_t rosetta_bsk_device_words(const rosetta_params *params); /* = rosetta_bsk_words */
size_t rosetta_ksk_words(const rosetta_params *params);
size_t rosetta_ksk_device_words(const rosetta_params *params);

/* a0: bootstrapping-key preparation (once per key, not part of a PBS).
 * The bootstrapping key is what blind rotation multiplies by (Sec. 2.2.2
 * "TFHE Scheme", PBS item: the encrypted message drives the rotation, one
 * GGSW encryption of each key bit s_i selecting X^(a~_i) or 1).
 * Transforms every GGSW row of `bsk_std_dev` (standard layout, device) into
 * the library's transform-domain layout in `bsk_dev` (device, same size,
 * must not overlap).  Rows are pre-scaled by N^-1 so that the inverse
 * transforms in the blind-rotation loop need no scaling. */
rosetta_status rosetta_bsk_prepare(const uint64_t *bsk_std_dev, uint64_t *bsk_dev,
                                   const rosetta_params *params, void *stream);

/* Key-switching-key preparation (once per key, not part of a PBS; the key
 * switch is the last step of the PBS, Sec. 2.2.2 "TFHE Scheme", PBS item,
 * whose output is a fresh TFHE ciphertext under the input's key): writes
 * the prepared layout of the standard key `ksk_std_dev` into `ksk_dev`
 * (rosetta_ksk_device_words words, device, must not overlap):
 * the signed byte planes of every key word (each word w replaced by w or
 * w - p, whichever 8 balanced base-256 digits represent) in the operand
 * order of the matrix-core kernel, or the key copied with its column sums
 * appended for the VALU kernel. */
rosetta_status rosetta_ksk_prepare(const uint64_t *ksk_std_dev, uint64_t *ksk_dev,
                                   const rosetta_params *params, void *stream);

/* THE HOT PATH: programmable bootstrapping of `batch` LWE ciphertexts
 * (Sec. 2.2.2 "TFHE Scheme", PBS item, and Fig. rlwe_primitives(a): the
 * table f in the coefficients of the test polynomial v, blind rotation by
 * the encrypted message so that f(m) reaches the constant term, extraction
 * of that term, Sec. 2.2.3 "LWE Extract", as a fresh ciphertext, then key
 * switching back to the n-dimensional key).
 *   lwe_in   [batch][n+1]  device, canonical
 *   bsk_dev  prepared bootstrapping key (rosetta_bsk_prepare)
 *   ksk_dev  prepared key-switching key (rosetta_ksk_prepare)
 *   lut      [N]           device, the test polynomial (rosetta_lut_build)
 *   lwe_out  [batch][n+1]  device; may be exactly lwe_in (in place) but must
 *                          not partially overlap it (ROSETTA_ERR_ALIAS)
 * Steps a1-a8: modulus switch and accumulator set-up, n CMux steps
 * (rotate-subtract, decompose, forward transforms, transform-domain
 * multiply-accumulate with GGSW_i, inverse transforms, accumulate), sample
 * extraction, key switching.  Uses a library-owned device workspace of
 * rosetta_pbs_workspace_bytes(params, batch) bytes, grown on demand and kept
 * per device until rosetta_shutdown(); calls sharing that workspace on one
 * device must therefore be serialised (one stream at a time), or use
 * rosetta_pbs_batch_ws with distinct workspaces. */
rosetta_status rosetta_pbs_batch(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                 const uint64_t *ksk_dev, const uint64_t *lut, uint64_t *lwe_out,
                                 size_t batch, const rosetta_params *params, void *stream);

/* Workspace size (bytes) for a PBS of `batch` ciphertexts. */
size_t rosetta_pbs_workspace_bytes(const rosetta_params *params, size_t batch);

/* rosetta_pbs_batch with a caller-provided device workspace of at least
 * rosetta_pbs_workspace_bytes bytes (else ROSETTA_ERR_SIZE). */
rosetta_status rosetta_pbs_batch_ws(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                    const uint64_t *ksk_dev, const uint64_t *lut,
                                    uint64_t *lwe_out, size_t batch,
                                    const rosetta_params *params, void *workspace,
                                    size_t workspace_bytes, void *stream);

/* Allocation-free rosetta_pbs_batch, for callers that cannot allocate device
 * memory while they run: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments, layouts, validation and
 * output bits as rosetta_pbs_batch (the same two kernels run); the scratch
 * between them (the extracted ciphertexts, rosetta_pbs_workspace_bytes
 * bytes) is a static device array of ROSETTA_NOALLOC_SCRATCH_BYTES that
 * each GPU the library runs on holds until the process ends, and the
 * transform tables (the twiddles and the powers of psi) are static device
 * memory too.  Nothing is allocated: not on the first call on a device
 * (which looks up that device's addresses of the arrays and uploads the
 * tables of N with hipMemcpy if no earlier call did: a caller that captures
 * a graph makes one call at that N before it starts capturing), not later.  A batch whose scratch exceeds the array,
 * batch * (N+1) * 8 > ROSETTA_NOALLOC_SCRATCH_BYTES (at most 4094
 * ciphertexts at N = 2048, 2047 at N = 4096), is rejected with
 * ROSETTA_ERR_SIZE before anything is enqueued.  All calls on one device
 * share its array: calls on one stream run in order, but calls that overlap
 * in time on one device (several streams or threads) race on it and give
 * unspecified results.  The array needs no clearing between calls. */
#define ROSETTA_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
rosetta_status rosetta_pbs_batch_noalloc(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                         const uint64_t *ksk_dev, const uint64_t *lut,
                                         uint64_t *lwe_out, size_t batch,
                                         const rosetta_params *params, void *stream);

/* Steps a1-a6 alone: blind rotation (Sec. 2.2.2, PBS item: the RLWE
 * encryption of the rotated test polynomial), returning the GLWE accumulators
 * glwe_out [batch][2N] (device; must not overlap the inputs). */
rosetta_status rosetta_blind_rotate(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                    const uint64_t *lut, uint64_t *glwe_out, size_t batch,
                                    const rosetta_params *params, void *stream);

/* Steps a1-a7: blind rotation and sample extraction (Sec. 2.2.3 "Scheme
 * Conversion and Other Primitives", LWE Extract item), returning LWE
 * ciphertexts of dimension N under the GLWE key, big_out [batch][N+1]
 * (device; must not overlap the inputs). */
rosetta_status rosetta_blind_rotate_extract(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                            const uint64_t *lut, uint64_t *big_out,
                                            size_t batch, const rosetta_params *params,
                                            void *stream);

/* Step a8: key switching (the PBS's return to the input key, Sec. 2.2.2,
 * PBS item) of big_in [batch][N+1] to lwe_out [batch][n+1]
 * (device; must not overlap). */
rosetta_status rosetta_keyswitch(const uint64_t *big_in, const uint64_t *ksk_dev,
                                 uint64_t *lwe_out, size_t batch, const rosetta_params *params,
                                 void *stream);

/* Negacyclic number-theoretic transform of `count` polynomials of degree N
 * (device, [count][N], in and out may be the same buffer).  Forward output
 * order: out[j] = a(psi^(2 rev(j) + 1)) with psi = 7^((p-1)/2N) and rev the
 * log2(N)-bit reversal.  The inverse takes that order back to coefficients
 * and includes the 1/N scaling. */
rosetta_status rosetta_ntt_forward(const uint64_t *in, uint64_t *out, size_t count, uint32_t N,
                                   void *stream);
rosetta_status rosetta_ntt_inverse(const uint64_t *in, uint64_t *out, size_t count, uint32_t N,
                                   void *stream);

/* Negacyclic products c = a * b mod (X^N + 1) of `count` pairs through the
 * transform (device, [count][N] each; c may alias a or b exactly). */
rosetta_status rosetta_poly_mul(const uint64_t *a, const uint64_t *b, uint64_t *c, size_t count,
                                uint32_t N, void *stream);

/* Elementwise Goldilocks arithmetic with the device routines that every
 * kernel above is built from (Sec. 2.2 works over Z_p; here p = 2^64 -
 * 2^32 + 1), so that they can be checked on their own, edge values
 * included.  out[i] = f(a[i], b[i], c[i]) mod p for op:
 *   ROSETTA_FIELD_ADD      a + b
 *   ROSETTA_FIELD_SUB      a - b
 *   ROSETTA_FIELD_MUL      a * b
 *   ROSETTA_FIELD_MUL_ADD  a * b + c
 *   ROSETTA_FIELD_ADD_WEAK a + b for any a < 2^64 and canonical b, as the
 *       digit transforms of the blind rotation add: a result below 2^64 and
 *       congruent to a + b mod p, not necessarily canonical
 *   ROSETTA_FIELD_MUL_ADD_WEAK  a * b + c for any a, c < 2^64 and canonical
 *       b, as the blind rotation's key multiply-accumulate runs: below 2^64
 *       and congruent, not necessarily canonical
 *   ROSETTA_FIELD_MUL_POW2 + e   a * 2^e   (0 <= e < 96; 2^96 = -1 mod p)
 *   ROSETTA_FIELD_ROUND_TOP + s  (1 <= s <= 63) the rounding that opens the
 *       gadget decomposition of the blind rotation (Sec. 2.2, PBS
 *       paragraph): floor((a_c + 2^(s-1)) / 2^s) for the centred
 *       representative a_c of a in (-p/2, p/2], as a two's-complement int64;
 *       a = p is also accepted (as 0)
 * a, b, c, out: device [count] u64.  Every input must be canonical (< p)
 * unless stated; the result is canonical.  b and c are not read (and may be
 * NULL) when the op does not use them; out may alias an input exactly.  Errors:
 * ROSETTA_ERR_PARAMS for an unknown op, ROSETTA_ERR_NULL for a missing
 * pointer the op reads or writes. */
enum {
  ROSETTA_FIELD_ADD = 0,
  ROSETTA_FIELD_SUB = 1,
  ROSETTA_FIELD_MUL = 2,
  ROSETTA_FIELD_MUL_ADD = 3,
  ROSETTA_FIELD_ADD_WEAK = 4,
  ROSETTA_FIELD_MUL_ADD_WEAK = 5,
  ROSETTA_FIELD_MUL_POW2 = 256,
  ROSETTA_FIELD_ROUND_TOP = 512
};
rosetta_status rosetta_field_op(int op, const uint64_t *a, const uint64_t *b, const uint64_t *c,
                                uint64_t *out, size_t count, void *stream);

/* Throughput probe of the device modular multiplication (the roofline
 * reference for the transform kernels): `threads` threads (256 per
 * workgroup) each run 8 independent chains x <- x * w mod p for `iters`
 * steps in registers, with x_j = (seed + 8 t + j + 1) mod p and
 * w = (seed ^ (t * 0x9E3779B97F4A7C15)) mod p, or 3 where that is below 2;
 * out[t] (device, [threads] u64) receives the XOR of the eight final values,
 * x_j w^iters mod p, so that the work is checkable.  Errors: ROSETTA_ERR_NULL
 * for a NULL out with threads > 0. */
rosetta_status rosetta_modmul_chain(uint64_t seed, uint32_t threads, uint32_t iters,
                                    uint64_t *out, void *stream);

/* ---- lookup-protocol primitives (Sec. 3.2 "Cryptographic Lookup Protocol",
 * Steps 2-3 and Algorithm 1; Sec. 2.2.3 "RLWE Trace Computation") ---------
 *
 * CONVENTIONS (beyond those above):
 *  - Galois automorphism tau_d (d odd): a(X) -> a(X^d); X^j goes to
 *    X^(j d mod 2N), an exponent e >= N standing for -X^(e-N).
 *  - GLWE key switching with a key K for S' -> S, rows K[t] = GLWE_S(S' g_t):
 *    (A', B') -> (0, B') - sum_t Dec_t(A') * K[t]  (Dec as for the
 *    bootstrapping key, with the trace's own level and base_log).
 *  - Trace: c <- N^-1 c (mod p) first; then for k = log2 N down to 1,
 *    d = 2^k + 1: c <- c + KS_d(tau_d(c)).  The phase of the result is the
 *    constant coefficient of the phase of c (plus key-switching noise), all
 *    other coefficients cancel.
 *  - Automorphism key (standard layout) [k-1 < log2 N][t < level][c < 2][x < N]:
 *    row (k-1, t) is a GLWE encryption under S of tau_(2^k+1)(S) g_t. */

/* Blind rotation of ciphertext test polynomials (Sec. 3.2, Step 3
 * "BlindRot" and the selection of Step 2): LWE selector q of lwe_in
 * [batch][n+1] is paired with the `group` consecutive GLWE ciphertexts
 * glwe_tp[q*group .. q*group+group) (device, [batch*group][2N], under the
 * GLWE key); for each, ACC = X^(-b~) tp (both components), then the CMux
 * loop of rosetta_blind_rotate.  extract = 0: out [batch*group][2N] holds
 * the accumulators; extract != 0: out [batch*group][N+1] holds their
 * sample extractions (rosetta_keyswitch then completes a PBS whose table is
 * encrypted).  1 <= group <= 4096; out must not overlap the inputs. */
rosetta_status rosetta_blind_rotate_glwe(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                         const uint64_t *glwe_tp, uint64_t *out, size_t batch,
                                         uint32_t group, const rosetta_params *params,
                                         int extract, void *stream);

/* LWE copies with shifted bodies (comparison inputs x - tau_j of Step 1):
 * lwe_out[q][j] = lwe_in[q] + (0, .., 0, consts[j]) for j < count, with
 * lwe_in [batch][dim+1], lwe_out [batch][count][dim+1] (device, not
 * overlapping); consts: host array, values below p; 1 <= count <= 64. */
rosetta_status rosetta_lwe_add_consts(const uint64_t *lwe_in, const uint64_t *consts,
                                      uint64_t *lwe_out, size_t batch, uint32_t count,
                                      uint32_t dim, void *stream);

/* Linear combination of LWE arrays, word by word (an LWE ciphertext is
 * linear in its phase, so this is the ciphertext of the same combination of
 * phases; the refined comparison of Step 1 scales and subtracts with it):
 * out[i] = alpha a[i] + beta b[i] + gamma c[i] mod p for i < words.  b and c
 * may be NULL (their term is then left out); alpha, beta, gamma below p
 * (else ROSETTA_ERR_PARAMS); out may be exactly a, b or c but must not
 * partially overlap them (device). */
rosetta_status rosetta_lwe_combine(const uint64_t *a, uint64_t alpha, const uint64_t *b,
                                   uint64_t beta, const uint64_t *c, uint64_t gamma,
                                   uint64_t *out, size_t words, void *stream);

/* Group sums (the segment index S = sum_j [x >= tau_j] of Step 1):
 * lwe_out[q] = sum_{j < count} lwe_in[q][j] + (0, .., 0, c0), lwe_in
 * [batch][count][dim+1], lwe_out [batch][dim+1] (device, not overlapping). */
rosetta_status rosetta_lwe_sum_groups(const uint64_t *lwe_in, uint64_t c0, uint64_t *lwe_out,
                                      size_t batch, uint32_t count, uint32_t dim, void *stream);

/* Words of an automorphism key with `level` gadget levels: log2(N) level 2 N. */
size_t rosetta_autk_words(const rosetta_params *params, uint32_t level);

/* Automorphism key, standard layout -> library layout (device buffers of
 * rosetta_autk_words words each, not overlapping): every row to the
 * transform domain, scaled by N^-1.  Only params->N is used beyond the
 * usual validation. */
rosetta_status rosetta_autk_prepare(const uint64_t *autk_std_dev, uint64_t *autk_dev,
                                    const rosetta_params *params, uint32_t level, void *stream);

/* RLWE trace (Sec. 2.2.3) of glwe_in [batch][2N] into glwe_out [batch][2N]
 * (device; the two may be the same buffer, not partially overlapping), with
 * a prepared automorphism key.  Supported: 1 <= level <= 4,
 * base_log <= 30, level*base_log <= 62. */
rosetta_status rosetta_trace(const uint64_t *glwe_in, const uint64_t *autk_dev,
                             uint64_t *glwe_out, size_t batch, const rosetta_params *params,
                             uint32_t level, uint32_t base_log, void *stream);

/* Plaintext polynomials [count][N] (coefficients, device) -> the prepared
 * form that rosetta_glwe_mul_plain multiplies by (transform domain, N^-1,
 * library order), into a separate buffer of the same size. */
rosetta_status rosetta_plain_prepare(const uint64_t *plain_dev, uint64_t *plain_prep_dev,
                                     size_t count, uint32_t N, void *stream);

/* Plaintext-ciphertext products (Sec. 3.2, "Construct": the linear mapping
 * p(X) [[x]] + q(X)): for ciphertext q of glwe_in [batch][2N] and plaintext
 * s < npoly, glwe_out[q][s] = (pa_s * A_q, pa_s * B_q + pb_s), so that
 * phase(out) = pa_s * phase(in) + pb_s.  pa_prep_dev [npoly][N] from
 * rosetta_plain_prepare; pb_dev [npoly][N] coefficients, or NULL for none.
 * glwe_out [batch][npoly][2N] must not overlap the inputs. */
rosetta_status rosetta_glwe_mul_plain(const uint64_t *glwe_in, const uint64_t *pa_prep_dev,
                                      const uint64_t *pb_dev, uint64_t *glwe_out, size_t batch,
                                      uint32_t npoly, uint32_t N, void *stream);

/* Recombination (Sec. 3.2, Step 3 Phase 2, and the recombination of
 * Sec. 3.3.2): glwe_out[q] = sum_{s < count} X^(e_s) glwe_in[q][s],
 * glwe_in [batch][count][2N], glwe_out [batch][2N] (device, not
 * overlapping).  exps: host array of `count` exponents in [0, 2N), or NULL
 * for e_s = s; 1 <= count <= 256. */
rosetta_status rosetta_glwe_recombine(const uint64_t *glwe_in, const uint32_t *exps,
                                      uint64_t *glwe_out, size_t batch, uint32_t count,
                                      uint32_t N, void *stream);

/* Monomial copies (Sec. 3.3.2, multi-value batching: X^(-c) moves the value
 * at coefficient c to the constant term): glwe_out[q][s] = X^(e_s)
 * glwe_in[q], glwe_in [batch][2N], glwe_out [batch][count][2N] (device, not
 * overlapping); exps: host array of `count` exponents in [0, 2N)
 * (X^(-c) = X^(2N-c)); 1 <= count <= 256. */
rosetta_status rosetta_glwe_monomial_mul(const uint64_t *glwe_in, const uint32_t *exps,
                                         uint64_t *glwe_out, size_t batch, uint32_t count,
                                         uint32_t N, void *stream);

/* Sample extraction alone (LWE Extract, Sec. 2.2.3): big_out[q] = (A_0,
 * -A_{N-1}, .., -A_1, B_0) from glwe_in [batch][2N]; big_out [batch][N+1]
 * (device, not overlapping). */
rosetta_status rosetta_sample_extract(const uint64_t *glwe_in, uint64_t *big_out, size_t batch,
                                      uint32_t N, void *stream);

/* ---- the TFHE core of the cryptographic lookup (Sec. 3.2, Algorithm 1,
 * Steps 1-3) ---------------------------------------------------------------
 *
 * For a batch of inputs x, each given as a GLWE ciphertext [[x]]_RLWE of
 * round(x 2^sx) in the constant coefficient and an LWE ciphertext
 * [[x]]_cmp of round(x 2^sc) under the LWE key, the pipeline returns GLWE
 * ciphertexts of round(f~(x) 2^(sx+sp)) in the constant coefficient (other
 * coefficients zero up to noise) at scale 2^(sx+sv), f~ the segmented LUT
 * (a, b, tau) of rosetta_seglut_build.
 *
 * ENCODINGS (the paper names the steps but not their encodings):
 *  - Step 1, HomComp(x, tau_j) for j = 1..nseg-1: a PBS of
 *    y_j = [[x]]_cmp - round(tau_j 2^sc) with the constant test polynomial
 *    mu = floor(p / 4 nseg) (a sign bootstrap), plus mu: 2 mu if x >= tau_j,
 *    else 0 (up to noise; inputs within the bootstrap's resolution of tau_j
 *    may fall on either side).  S = sum_j of them: the segment index at scale
 *    2 mu ~ p / 2 nseg, i.e. a rotation by S N / nseg.
 *    With cmp_refine_log = k > 0 each comparison chains three blind
 *    rotations (the paper's HomComp chains several PBS for precision), which
 *    divides the resolution by 2^k: with h = floor(p / 2^(k+1)),
 *      z   = 2^k (y_j + (0, h)),
 *      e   = SE(BlindRot(z, floor(p / 2^(k+2)))),  s1 = KS(e),
 *      s1' = KS(2^k e) (the sign at the fine scale, within 2^k of p/4; e
 *            is scaled before the key switch so that 2^k multiplies only
 *            the blind rotation's noise),
 *      s2  = PBS(z - s1', f),  f_i = -round(min(i, N-i) p / (2^(k+1) N))
 *            (half up; the bootstrap then returns -phase / 2^k on phases
 *            in [-p/4, p/4), where z - s1' lies),
 *      c_j = PBS(y_j - s1 + s2, mu) + mu;
 *    y_j - s1 + s2 is a whole number of digits p / 2^k less half a digit,
 *    positive exactly when x >= tau_j (up to the fine resolution).
 *  - Step 2, construct: t = p(X) [[x]]_RLWE + q(X), where coefficient j of
 *    p and q holds segment s = floor((j + h) / box)'s slope
 *    nbr / (tau_{s+1} - tau_s) at scale 2^sp and offset
 *    -tau_s nbr / (tau_{s+1} - tau_s) - 1/2 + margin at 2^(sx+sp)
 *    (box = N / nseg, h = box / 2; coefficients j >= N - h hold segment 0's
 *    values negated, the negacyclic image).  Select: I = PBS(t, S) (blind
 *    rotation of t by S, extraction, key switching); with
 *    sx + sp = 63 - log2 N one unit of t is one rotation step, so I rotates
 *    by floor(t_S) + margin.
 *  - Step 3, construct: r_s = a_s(X) [[x]]_RLWE + b_s(X), coefficient j
 *    holding interval clamp(j - margin, 0, nbr-1) of segment s (slope at
 *    2^sv, offset at 2^(sx+sv): the values get their own scale, larger than
 *    the rotation unit of the selectors, since the trace's key-switching
 *    noise grows with N).  Select by I: Trace(BlindRot(r_s, I)) for
 *    every s (one selector, nseg test polynomials).  Recombine:
 *    R = sum_s X^(s box) r_s, spread over each segment's window by the
 *    product with W(X) = sum_{k=-h}^{box-h-1} X^k.  Select by S:
 *    Trace(BlindRot(R W, S)).
 *  - Requirements: nseg a power of two in [2, 16]; nbr + 2 margin <= N;
 *    sx + sp = 63 - log2 N; sx + sv <= 62; cmp_refine_log <= 6;
 *    |x - tau_j| 2^sc < p / 4.  Coefficients are
 *    round(v 2^k) (half to even, as doubles) reduced exactly mod p, so
 *    offsets larger than the scale allows (q_s) wrap harmlessly: only
 *    p_s x + q_s, in [0, nbr) for the selected segment, must fit.
 *
 * The plaintext block [(4 + 2 nseg) N] words: p, q, a_0..a_{nseg-1},
 * b_0..b_{nseg-1}, W, the sign test polynomial, then with a refined
 * comparison floor(p / 2^(k+2)) and f (2 N more); constants [nseg]:
 * -round(tau_j 2^sc) mod p for j = 1..nseg-1, then (nseg-1) mu. */
typedef struct rosetta_lookup_params {
  uint32_t nseg;           /* N_seg, a power of two in [2, 16] */
  uint32_t nbr;            /* intervals per segment */
  uint32_t margin;         /* guard coefficients before and after the intervals */
  uint32_t x_scale_log;    /* sx: scale of [[x]]_RLWE */
  uint32_t coef_scale_log; /* sp: scale of Step 2 slopes (sx + sp = 63 - log2 N) */
  uint32_t val_scale_log;  /* sv: scale of Step 3 slopes; output at 2^(sx+sv) */
  uint32_t cmp_scale_log;  /* sc: scale of [[x]]_cmp */
  uint32_t trace_level;    /* automorphism key levels */
  uint32_t trace_base_log; /* automorphism key base log */
  uint32_t cmp_refine_log; /* k: bits of refinement of the comparison (0: one sign
                              bootstrap per boundary; 1..6: three blind
                              rotations and four key switches, see Step 1) */
} rosetta_lookup_params;

/* Words of the plaintext block: (4 + 2 nseg) N, plus 2 N with a refined
 * comparison. */
size_t rosetta_lookup_plain_words(const rosetta_params *params,
                                  const rosetta_lookup_params *lp);

/* Host encoder of the plaintext block and constants (layouts above) from
 * boundaries tau[nseg+1] and coefficients a, b [nseg][nbr] (host arrays). */
rosetta_status rosetta_lookup_encode(const rosetta_params *params,
                                     const rosetta_lookup_params *lp, const double *tau,
                                     const double *a, const double *b, uint64_t *plain,
                                     uint64_t *consts);

/* Plaintext block (device) -> prepared block (device, same size, not
 * overlapping): p, the a_s and W to the multiplier form of
 * rosetta_plain_prepare, the rest copied. */
rosetta_status rosetta_lookup_prepare(const uint64_t *plain_dev, uint64_t *plain_prep_dev,
                                      const rosetta_params *params,
                                      const rosetta_lookup_params *lp, void *stream);

/* Device workspace of rosetta_lookup_eval for `batch` inputs. */
size_t rosetta_lookup_workspace_bytes(const rosetta_params *params,
                                      const rosetta_lookup_params *lp, size_t batch);

/* Where rosetta_lookup_eval leaves its intermediates in the workspace, so
 * that a caller holding the keys can inspect them after the call: the word
 * offset of part `part` for `batch` inputs, or (size_t)-1 for an unknown
 * part.  Parts: ROSETTA_LOOKUP_PART_CMP, the comparison results
 * [batch][nseg-1][n+1] (LWE); ROSETTA_LOOKUP_PART_S, the segment index S
 * [batch][n+1] (LWE, S at scale 2 floor(p / 4 nseg)); ROSETTA_LOOKUP_PART_I,
 * the interval selector I [batch][n+1] (LWE, one rotation step p / 2N per
 * unit). */
enum { ROSETTA_LOOKUP_PART_CMP = 2, ROSETTA_LOOKUP_PART_S = 3, ROSETTA_LOOKUP_PART_I = 6 };
size_t rosetta_lookup_workspace_offset(const rosetta_params *params,
                                       const rosetta_lookup_params *lp, size_t batch,
                                       uint32_t part);

/* Steps 1-3 for a batch: x_rlwe [batch][2N], x_cmp [batch][n+1], prepared
 * keys (bootstrapping, key switching, automorphism), the prepared plaintext
 * block and the host constants; out [batch][2N] (device, not overlapping the
 * workspace).  Per input: nseg-1 PBS (Step 1; with a refined comparison
 * 3 (nseg-1) blind rotations and 4 (nseg-1) key switches), one blind
 * rotation of an
 * encrypted test polynomial + extraction + key switch (Step 2), nseg + 1
 * blind rotations of encrypted test polynomials and traces (Step 3), and
 * nseg + 2 plaintext products. */
rosetta_status rosetta_lookup_eval(const uint64_t *x_rlwe, const uint64_t *x_cmp,
                                   const uint64_t *bsk_dev, const uint64_t *ksk_dev,
                                   const uint64_t *autk_dev, const uint64_t *plain_prep_dev,
                                   const uint64_t *consts, uint64_t *out, size_t batch,
                                   const rosetta_params *params, const rosetta_lookup_params *lp,
                                   void *workspace, size_t workspace_bytes, void *stream);

/* ---- adaptive segmented LUT (Sec. 3.1), host ---------------------------
 *
 * The domain [tau_0, tau_nseg] is cut into nseg segments; segment s holds
 * nbr equal intervals; interval i of segment s carries a_si x + b_si.
 * Coefficient arrays are [nseg][nbr] doubles.  Linear fits interpolate f at
 * the interval's two Chebyshev nodes c -+ r cos(pi/4) (c midpoint, r
 * half-width); constant fits store f(c) (the single-LUT baseline).  Lookup:
 * S = #{j in 1..nseg-1 : x >= tau_j}, I = floor((x - tau_S) nbr /
 * (tau_{S+1} - tau_S)) clamped to [0, nbr), y = a_SI x + b_SI. */
typedef enum {
  ROSETTA_FN_INV = 0,      /* 1/x */
  ROSETTA_FN_INV_SQRT = 1, /* 1/sqrt(x) */
  ROSETTA_FN_SILU = 2,     /* x / (1 + e^-x) */
  ROSETTA_FN_GELU = 3,     /* x (1 + erf(x / sqrt 2)) / 2 */
  ROSETTA_FN_EXP = 4       /* e^x */
} rosetta_function;
typedef enum { ROSETTA_SPACING_UNIFORM = 0, ROSETTA_SPACING_LOG = 1 } rosetta_spacing;
typedef enum { ROSETTA_FIT_LINEAR = 0, ROSETTA_FIT_CONSTANT = 1 } rosetta_fit;

/* Boundaries tau[nseg+1] on [lo, hi]: uniform, or geometric (lo > 0; the
 * evaluation setup of Sec. 5.1 spaces them logarithmically for 1/x and
 * 1/sqrt(x) and uniformly for SiLU and GELU). */
rosetta_status rosetta_seglut_boundaries(double lo, double hi, uint32_t nseg, int spacing,
                                         double *tau);

/* Coefficients a, b [nseg][nbr] of `function` (rosetta_function) with the
 * given fit (rosetta_fit) over strictly increasing boundaries tau[nseg+1]. */
rosetta_status rosetta_seglut_build(int function, const double *tau, uint32_t nseg, uint32_t nbr,
                                    int fit, double *a, double *b);

/* Step 2 polynomials of Sec. 3.2: p[s] = nbr / (tau_{s+1} - tau_s),
 * q[s] = -tau_s nbr / (tau_{s+1} - tau_s), so that p[s] x + q[s] is the
 * (real) local interval index of x in segment s. */
rosetta_status rosetta_seglut_protocol_polys(const double *tau, uint32_t nseg, uint32_t nbr,
                                             double *p, double *q);

/* Cleartext three-step lookup of x[count] into y[count].  index_offset
 * (NULL for none) adds offset[k] to input k's interval index before the
 * coefficients are read (clamped to [0, nbr)): a model of the selection
 * error of the encrypted lookup, drawn by the caller. */
rosetta_status rosetta_seglut_eval(const double *tau, uint32_t nseg, uint32_t nbr,
                                   const double *a, const double *b, const double *x,
                                   const int32_t *index_offset, size_t count, double *y);

/* Precision in bits, -log2 of the RMS error of the cleartext lookup (with
 * the optional index offsets) against `function` over x[count] (count >= 1). */
rosetta_status rosetta_seglut_precision(int function, const double *tau, uint32_t nseg,
                                        uint32_t nbr, const double *a, const double *b,
                                        const double *x, const int32_t *index_offset,
                                        size_t count, double *bits);

/* Fixed-point encoding into Z_p: out[k] = round(v[k] 2^scale_log) mod p
 * (round half to even); |v 2^scale_log| must stay below 2^62. */
rosetta_status rosetta_encode_fixed(const double *v, size_t count, int scale_log,
                                    uint64_t *out);

/* ---- test helpers: host memory, deterministic from the seed ------------ */

/* Key generation for the PBS (Sec. 2.2.2 "TFHE Scheme": LWE encryption of
 * scalars, the GGSW bootstrapping key of blind rotation, and the
 * key-switching key that returns its output to the LWE key).
 * Binary keys and the two switching keys in standard layout (host arrays of
 * n, N, rosetta_bsk_words and rosetta_ksk_words words).  Randomness is
 * SplitMix64 used as a counter-based generator (Steele, Lea and Flood 2014):
 * word(key, i) = mix(key + (i+1) * 0x9E3779B97F4A7C15); sub-stream keys
 * word(seed, stream) with streams 1 (LWE key bits, top bit of word i),
 * 2 (GLWE key bits), 3/4 (key mask words r*N+x / noise of row r, coefficient
 * x, r = (2i+u)l+t), 5/6 (key-switching mask words r*n+c / noise r,
 * r = j l_ks + t).  Uniform elements: w - p if w >= p.  Gaussian number g:
 * Box-Muller on words 2g, 2g+1, rounded after scaling by sigma * 2^64
 * (sigma is a fraction of the modulus).  The products A*S run on the host. */
rosetta_status rosetta_keygen(uint64_t seed, const rosetta_params *params, double sigma_lwe,
                              double sigma_glwe, uint64_t *lwe_key, uint64_t *glwe_key,
                              uint64_t *bsk_std, uint64_t *ksk_std);

/* TFHE-Enc of Sec. 2.2.2 "TFHE Scheme" (Encryption and Decryption item):
 * encryption of msgs[count] (values in Z_2M) under a binary key of length
 * `dim` (host): masks from stream 7 word q*dim+c, noise from stream 8
 * Gaussian q, of sub-stream keys of `seed`. */
rosetta_status rosetta_lwe_encrypt(uint64_t seed, const rosetta_params *params, double sigma,
                                   const uint64_t *key, uint32_t dim, const uint32_t *msgs,
                                   size_t count, uint64_t *lwe_out);

/* Encryption of plaintexts already in Z_p (host; same randomness as
 * rosetta_lwe_encrypt: masks stream 7, noise stream 8). */
rosetta_status rosetta_lwe_encrypt_plain(uint64_t seed, double sigma, const uint64_t *key,
                                         uint32_t dim, const uint64_t *plain, size_t count,
                                         uint64_t *lwe_out);

/* TFHE-Dec of Sec. 2.2.2 "TFHE Scheme" (Encryption and Decryption item):
 * decryption of `count` ciphertexts of dimension `dim` to Z_2M (host):
 * m = floor((2M (b - <a, s>) + (p-1)/2) / p) mod 2M. */
rosetta_status rosetta_lwe_decrypt(const rosetta_params *params, const uint64_t *key,
                                   uint32_t dim, const uint64_t *lwe, size_t count,
                                   uint32_t *msgs_out);

/* Test polynomial v [N] for a table of M entries in Z_2M (host): the LUT
 * entries laid out as coefficients (Sec. 2.2.2 "TFHE Scheme", PBS item, and
 * Fig. rlwe_primitives(a)), with the padding-bit, half-box layout of the
 * CONVENTIONS above. */
rosetta_status rosetta_lut_build(const rosetta_params *params, const uint32_t *table,
                                 uint64_t *test_poly);

/* GLWE encryption (host) of `count` plaintext polynomials msgs [count][N],
 * already scaled into Z_p, under the GLWE key: mask coefficient x of
 * ciphertext q from stream 11 word q*N+x, noise from stream 12 Gaussian
 * q*N+x; B = A*S + M + E.  out [count][2N]. */
rosetta_status rosetta_glwe_encrypt(uint64_t seed, const rosetta_params *params, double sigma,
                                    const uint64_t *glwe_key, const uint64_t *msgs, size_t count,
                                    uint64_t *glwe_out);

/* Phases B - A*S of `count` GLWE ciphertexts [count][2N] (host). */
rosetta_status rosetta_glwe_phase(const rosetta_params *params, const uint64_t *glwe_key,
                                  const uint64_t *glwe, size_t count, uint64_t *phase_out);

/* Automorphism key in standard layout (host, rosetta_autk_words words):
 * row r = (k-1) level + t encrypts tau_(2^k+1)(S) g_t, g_t = 2^(64-(t+1)
 * base_log), mask coefficient x from stream 9 word r*N+x, noise from
 * stream 10 Gaussian r*N+x. */
rosetta_status rosetta_autk_keygen(uint64_t seed, const rosetta_params *params, uint32_t level,
                                   uint32_t base_log, double sigma, const uint64_t *glwe_key,
                                   uint64_t *autk_std);

/* Release the library's device state on every device it touched (the
 * workspaces; the transform tables live in static device memory and stay).
 * The library re-initialises lazily afterwards. */
rosetta_status rosetta_shutdown(void);

#ifdef __cplusplus
}
#endif

#endif /* ROSETTA_H */
