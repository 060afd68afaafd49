// The TFHE core of ROSETTA's cryptographic lookup (Sec. 3.2, Algorithm 1,
// Steps 1-3) as one batched device pipeline, and the host encoder of its
// plaintexts.  Every step runs in the library's kernels; this file only
// sequences launches on the caller's stream.
//
// Encodings (the paper gives the operations, not their encodings; each
// choice is stated in rosetta.h next to rosetta_lookup_params):
//   * Step 1: HomComp(x, tau_j) is a sign bootstrap of the comparison input
//     [[x]]_cmp - tau_j 2^sc with the constant test polynomial mu =
//     floor(p / 4 nseg); mu is added back so that [x >= tau_j] is 0 or 2 mu,
//     and S = sum_j of them is the segment index at scale p / 2 nseg, i.e. a
//     rotation by S N / nseg.
//   * Step 2: t = p(X) [[x]] + q(X) with segment s's slope and offset
//     repeated over the window of rotations that round to s (N/nseg wide,
//     centred; the wrapped part negated), the offset also carrying -1/2 and
//     the margin, so that the selected coefficient, extracted and key
//     switched, rotates by floor(t_S) + margin in Step 3.
//   * Step 3: r_s = a_s(X) [[x]] + b_s(X) with interval i at coefficient
//     i + margin (the margins repeat the end intervals), at the value scale; selection by I
//     (blind rotation + trace), recombination at X^(s N / nseg), spread over
//     the segment's window by a product with the window polynomial W, then
//     selection by S (blind rotation + trace).
#include <cmath>
#include <cstdint>
#include <vector>

#include "gl.hpp"
#include "internal.hpp"
#include "rosetta.h"

using namespace rosetta;

namespace {

rosetta_status err(rosetta_status st, const char *msg) {
  set_last_error(msg);
  return st;
}

int ilog2(uint32_t N) {
  int l = 0;
  while ((1u << l) < N) ++l;
  return l;
}

rosetta_status check_lookup(const rosetta_params *p, const rosetta_lookup_params *lp) {
  rosetta_status st = rosetta_check_params(p);
  if (st) return st;
  if (!lp) return err(ROSETTA_ERR_NULL, "lookup params is NULL");
  const uint32_t N = p->N;
  if (lp->nseg < 2 || lp->nseg > 16 || (lp->nseg & (lp->nseg - 1)))
    return err(ROSETTA_ERR_PARAMS, "nseg must be a power of two in [2, 16]");
  if (lp->nbr < 1 || (uint64_t)lp->nbr + 2ull * lp->margin > N)
    return err(ROSETTA_ERR_PARAMS, "need nbr >= 1 and nbr + 2 margin <= N");
  if (lp->x_scale_log + lp->coef_scale_log != (uint32_t)(63 - ilog2(N)))
    return err(ROSETTA_ERR_PARAMS, "need x_scale_log + coef_scale_log = 63 - log2 N");
  if (lp->cmp_scale_log > 62) return err(ROSETTA_ERR_PARAMS, "cmp_scale_log must be <= 62");
  if (lp->x_scale_log + lp->val_scale_log > 62)
    return err(ROSETTA_ERR_PARAMS, "need x_scale_log + val_scale_log <= 62");
  if (lp->trace_level < 1 || lp->trace_level > 4 || lp->trace_base_log < 1 ||
      lp->trace_base_log > 30 || lp->trace_level * lp->trace_base_log > 62)
    return err(ROSETTA_ERR_UNSUPPORTED, "trace level/base_log out of range");
  if (lp->cmp_refine_log > 6) return err(ROSETTA_ERR_PARAMS, "cmp_refine_log must be <= 6");
  return ROSETTA_OK;
}

// round(v 2^k) (half to even) as an element of Z_p, exactly: beyond 2^53
// a double is an integer m 2^e with m < 2^53, reduced as m 2^e mod p.
bool enc(double v, int k, u64 *out) {
  const double r = std::nearbyint(std::ldexp(v, k));
  const double ar = std::fabs(r);
  if (!std::isfinite(r) || ar >= 0x1p120) return false;
  u64 val;
  if (ar < 0x1p64) {
    val = (u64)ar;
    if (val >= GL_P) val -= GL_P;
  } else {
    int e;
    const double m = std::frexp(ar, &e);  // ar = m 2^e, m in [1/2, 1)
    val = gl_mul((u64)std::ldexp(m, 53), gl_pow(2, (u64)(e - 53)));
  }
  *out = r < 0 ? gl_neg(val) : val;
  return true;
}

// Words of each part of the plaintext block.
struct Block {
  size_t N, nseg, refine;
  size_t p_hat() const { return 0; }
  size_t q_hat() const { return N; }
  size_t a_hat(size_t s) const { return (2 + s) * N; }
  size_t b_hat(size_t s) const { return (2 + nseg + s) * N; }
  size_t window() const { return (2 + 2 * nseg) * N; }
  size_t sign_lut() const { return (3 + 2 * nseg) * N; }
  // the refined comparison's test polynomials (present when refine > 0)
  size_t coarse_sign() const { return (4 + 2 * nseg) * N; }
  size_t fine_part() const { return (5 + 2 * nseg) * N; }
  size_t words() const { return (4 + 2 * nseg + (refine ? 2 : 0)) * N; }
};

struct Scratch {
  size_t off = 0;
  uint64_t *base;
  explicit Scratch(void *b) : base((uint64_t *)b) {}
  uint64_t *take(size_t words) {
    uint64_t *r = base + off;
    off += (words + 31) & ~(size_t)31;  // 256-byte alignment
    return r;
  }
};

// Workspace layout of rosetta_lookup_eval (words), in call order.
constexpr int LOOKUP_WS_PARTS = 17;

size_t lookup_ws_words(const rosetta_params *p, const rosetta_lookup_params *lp, size_t batch,
                       uint64_t **parts, void *base, size_t *offsets = nullptr) {
  const size_t N = p->N, w = p->n + 1, ns = lp->nseg, nc = ns - 1;
  const size_t rf = lp->cmp_refine_log ? 1 : 0;  // refined comparison parts
  Scratch sc(base);
  const size_t sizes[] = {
      batch * nc * w,        // 0 comparison inputs
      batch * nc * (N + 1),  // 1 PBS workspace (extracted LWEs)
      batch * nc * w,        // 2 comparison results
      batch * w,             // 3 S
      batch * 2 * N,         // 4 t
      batch * (N + 1),       // 5 extracted selection of Step 2
      batch * w,             // 6 I
      batch * ns * 2 * N,    // 7 r_s
      batch * ns * 2 * N,    // 8 selected r_s
      batch * 2 * N,         // 9 R
      batch * 2 * N,         // 10 R spread over the windows
      rf * batch * nc * w,   // 11 z = 2^k (y + h)
      rf * batch * nc * w,   // 12 s1' (sign of z at the fine scale, 2^k s1 before the KS)
      rf * batch * nc * w,   // 13 s1 (sign of z at the coarse scale)
      rf * batch * nc * w,   // 14 z - s1'
      rf * batch * nc * w,   // 15 s2 (-phase / 2^k)
      rf * batch * nc * w,   // 16 y - s1 + s2
  };
  for (int i = 0; i < LOOKUP_WS_PARTS; ++i) {
    if (offsets) offsets[i] = sc.off;
    uint64_t *q = sc.take(sizes[i]);
    if (parts) parts[i] = q;
  }
  return sc.off;
}

}  // namespace

extern "C" {

size_t rosetta_lookup_plain_words(const rosetta_params *p, const rosetta_lookup_params *lp) {
  if (!p || !lp) return 0;
  return Block{p->N, lp->nseg, lp->cmp_refine_log}.words();
}

rosetta_status rosetta_lookup_encode(const rosetta_params *p, const rosetta_lookup_params *lp,
                                     const double *tau, const double *a, const double *b,
                                     uint64_t *plain, uint64_t *consts) {
  rosetta_status st = check_lookup(p, lp);
  if (st) return st;
  if (!tau || !a || !b || !plain || !consts) return err(ROSETTA_ERR_NULL, "NULL pointer");
  const int N = (int)p->N, ns = (int)lp->nseg, nbr = (int)lp->nbr, m = (int)lp->margin;
  const int sx = (int)lp->x_scale_log, sp = (int)lp->coef_scale_log;
  const int sv = (int)lp->val_scale_log;
  for (int s = 0; s < ns; ++s)
    if (!(tau[s] < tau[s + 1])) return err(ROSETTA_ERR_PARAMS, "boundaries must increase");
  const Block B{(size_t)N, (size_t)ns, lp->cmp_refine_log};
  const int box = N / ns, h = box / 2;
  // Step 2: slope and offset repeated over each segment's rotation window
  for (int j = 0; j < N; ++j) {
    const bool tail = j >= N - h;
    const int s = tail ? 0 : (j + h) / box;
    const double w = tau[s + 1] - tau[s];
    u64 pv, qv;
    if (!enc(nbr / w, sp, &pv) || !enc(-tau[s] * nbr / w - 0.5 + m, sx + sp, &qv))
      return err(ROSETTA_ERR_PARAMS, "Step 2 coefficient out of range for the scales");
    plain[B.p_hat() + j] = tail ? gl_neg(pv) : pv;
    plain[B.q_hat() + j] = tail ? gl_neg(qv) : qv;
  }
  // Step 3: interval i at coefficient i + margin, ends repeated
  for (int s = 0; s < ns; ++s)
    for (int j = 0; j < N; ++j) {
      int i = j - m;
      i = i < 0 ? 0 : (i > nbr - 1 ? nbr - 1 : i);
      u64 av, bv;
      if (!enc(a[(size_t)s * nbr + i], sv, &av) || !enc(b[(size_t)s * nbr + i], sx + sv, &bv))
        return err(ROSETTA_ERR_PARAMS, "Step 3 coefficient out of range for the scales");
      plain[B.a_hat(s) + j] = av;
      plain[B.b_hat(s) + j] = bv;
    }
  // window: X^k for k in [-h, box - h), negative powers wrapped with a sign
  for (int j = 0; j < N; ++j)
    plain[B.window() + j] = j < box - h ? 1 : (j >= N - h ? GL_P - 1 : 0);
  // sign test polynomial and constants
  const u64 mu = GL_P / (4 * (u64)ns);
  for (int j = 0; j < N; ++j) plain[B.sign_lut() + j] = mu;
  for (int j = 1; j < ns; ++j) {
    u64 t;
    if (!enc(-tau[j], (int)lp->cmp_scale_log, &t))
      return err(ROSETTA_ERR_PARAMS, "boundary out of range for the comparison scale");
    consts[j - 1] = t;
  }
  consts[ns - 1] = gl_mul(mu, (u64)(ns - 1));
  // the refined comparison: floor(p / 2^(k+2)) and
  // f_i = -round(min(i, N-i) p / (2^(k+1) N)) (half up)
  if (const int k = (int)lp->cmp_refine_log) {
    const u64 c1 = GL_P >> (k + 2);
    const unsigned __int128 den = (unsigned __int128)N << (k + 2);
    for (int j = 0; j < N; ++j) {
      const u64 w = (u64)(j < N - j ? j : N - j);
      const u64 g = (u64)(((unsigned __int128)2 * w * GL_P + (den >> 1)) / den);
      plain[B.coarse_sign() + j] = c1;
      plain[B.fine_part() + j] = g ? GL_P - g : 0;
    }
  }
  return ROSETTA_OK;
}

rosetta_status rosetta_lookup_prepare(const uint64_t *plain_dev, uint64_t *plain_prep_dev,
                                      const rosetta_params *p, const rosetta_lookup_params *lp,
                                      void *stream) {
  rosetta_status st = check_lookup(p, lp);
  if (st) return st;
  if (!plain_dev || !plain_prep_dev) return err(ROSETTA_ERR_NULL, "NULL pointer argument");
  const Block B{p->N, lp->nseg, lp->cmp_refine_log};
  const size_t bytes = B.words() * 8;
  {
    const char *x = (const char *)plain_dev, *y = (const char *)plain_prep_dev;
    if (x < y + bytes && y < x + bytes)
      return err(ROSETTA_ERR_ALIAS, "plain_dev and plain_prep_dev overlap");
  }
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipMemcpyAsync(plain_prep_dev, plain_dev, bytes, hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return err(ROSETTA_ERR_DEVICE, "copy of the plaintext block failed");
  // transform the multiplier rows in place: p, the a_s, the window
  if ((st = rosetta_plain_prepare(plain_dev + B.p_hat(), plain_prep_dev + B.p_hat(), 1, p->N, s)))
    return st;
  if ((st = rosetta_plain_prepare(plain_dev + B.a_hat(0), plain_prep_dev + B.a_hat(0), lp->nseg,
                                  p->N, s)))
    return st;
  return rosetta_plain_prepare(plain_dev + B.window(), plain_prep_dev + B.window(), 1, p->N, s);
}

size_t rosetta_lookup_workspace_bytes(const rosetta_params *p, const rosetta_lookup_params *lp,
                                      size_t batch) {
  if (!p || !lp || lp->nseg < 2) return 0;
  return lookup_ws_words(p, lp, batch, nullptr, nullptr) * 8;
}

size_t rosetta_lookup_workspace_offset(const rosetta_params *p, const rosetta_lookup_params *lp,
                                       size_t batch, uint32_t part) {
  if (!p || !lp || lp->nseg < 2) return (size_t)-1;
  if (part != ROSETTA_LOOKUP_PART_CMP && part != ROSETTA_LOOKUP_PART_S &&
      part != ROSETTA_LOOKUP_PART_I)
    return (size_t)-1;
  size_t offsets[LOOKUP_WS_PARTS];
  lookup_ws_words(p, lp, batch, nullptr, nullptr, offsets);
  return offsets[part];
}

rosetta_status rosetta_lookup_eval(const uint64_t *x_rlwe, const uint64_t *x_cmp,
                                   const uint64_t *bsk_dev, const uint64_t *ksk_dev,
                                   const uint64_t *autk_dev, const uint64_t *plain_prep_dev,
                                   const uint64_t *consts, uint64_t *out, size_t batch,
                                   const rosetta_params *p, const rosetta_lookup_params *lp,
                                   void *workspace, size_t workspace_bytes, void *stream) {
  rosetta_status st = check_lookup(p, lp);
  if (st) return st;
  if (batch == 0) return ROSETTA_OK;
  if (!x_rlwe || !x_cmp || !bsk_dev || !ksk_dev || !autk_dev || !plain_prep_dev || !consts ||
      !out || !workspace)
    return err(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t need = rosetta_lookup_workspace_bytes(p, lp, batch);
  if (workspace_bytes < need) return err(ROSETTA_ERR_SIZE, "workspace too small");
  {
    const char *o = (const char *)out, *w = (const char *)workspace;
    const size_t ob = batch * 2 * (size_t)p->N * 8;
    if (o < w + need && w < o + ob) return err(ROSETTA_ERR_ALIAS, "out overlaps the workspace");
  }
  const uint32_t N = p->N, n = p->n, ns = lp->nseg, nc = ns - 1;
  const Block B{N, ns, lp->cmp_refine_log};
  uint64_t *ws[LOOKUP_WS_PARTS];
  lookup_ws_words(p, lp, batch, ws, workspace);
  void *s = stream;
  const uint32_t tl = lp->trace_level, tb = lp->trace_base_log;

  // Step 1: segment index S = sum_j HomComp(x, tau_j)
  const size_t cmp_cts = batch * nc, cmp_words = cmp_cts * (n + 1);
  const size_t pbs_ws = cmp_cts * (N + 1) * 8;
  if ((st = rosetta_lwe_add_consts(x_cmp, consts, ws[0], batch, nc, n, s))) return st;
  const uint64_t *cmp_in = ws[0];
  if (const int k = (int)lp->cmp_refine_log) {
    // z = 2^k (y + h); s1, s1' its signs at the coarse and the fine scale
    // from one blind rotation (the extracted ciphertexts key-switched, then
    // scaled by 2^k and key-switched again); s2 = -(z - s1') / 2^k; the
    // sign bootstrap then takes y - s1 + s2
    uint64_t shifted[MAX_MONOMIALS / 4];
    const u64 h = GL_P >> (k + 1);
    for (uint32_t j = 0; j < nc; ++j) shifted[j] = gl_add(consts[j], h);
    if ((st = rosetta_lwe_add_consts(x_cmp, shifted, ws[11], batch, nc, n, s))) return st;
    if ((st = rosetta_lwe_combine(ws[11], (u64)1 << k, nullptr, 0, nullptr, 0, ws[11], cmp_words,
                                  s)))
      return st;
    if ((st = rosetta_blind_rotate_extract(ws[11], bsk_dev, plain_prep_dev + B.coarse_sign(),
                                           ws[1], cmp_cts, p, s)))
      return st;
    if ((st = rosetta_keyswitch(ws[1], ksk_dev, ws[13], cmp_cts, p, s))) return st;
    if ((st = rosetta_lwe_combine(ws[1], (u64)1 << k, nullptr, 0, nullptr, 0, ws[1],
                                  cmp_cts * (N + 1), s)))
      return st;
    if ((st = rosetta_keyswitch(ws[1], ksk_dev, ws[12], cmp_cts, p, s))) return st;
    if ((st = rosetta_lwe_combine(ws[11], 1, ws[12], GL_P - 1, nullptr, 0, ws[14], cmp_words, s)))
      return st;
    if ((st = rosetta_pbs_batch_ws(ws[14], bsk_dev, ksk_dev, plain_prep_dev + B.fine_part(),
                                   ws[15], cmp_cts, p, ws[1], pbs_ws, s)))
      return st;
    if ((st = rosetta_lwe_combine(ws[0], 1, ws[13], GL_P - 1, ws[15], 1, ws[16], cmp_words, s)))
      return st;
    cmp_in = ws[16];
  }
  if ((st = rosetta_pbs_batch_ws(cmp_in, bsk_dev, ksk_dev, plain_prep_dev + B.sign_lut(), ws[2],
                                 cmp_cts, p, ws[1], pbs_ws, s)))
    return st;
  if ((st = rosetta_lwe_sum_groups(ws[2], consts[nc], ws[3], batch, nc, n, s))) return st;
  // Step 2: t = p [[x]] + q; I = PBS(t, S)
  if ((st = rosetta_glwe_mul_plain(x_rlwe, plain_prep_dev + B.p_hat(),
                                   plain_prep_dev + B.q_hat(), ws[4], batch, 1, N, s)))
    return st;
  if ((st = rosetta_blind_rotate_glwe(ws[3], bsk_dev, ws[4], ws[5], batch, 1, p, 1, s))) return st;
  if ((st = rosetta_keyswitch(ws[5], ksk_dev, ws[6], batch, p, s))) return st;
  // Step 3: r_s = a_s [[x]] + b_s; select by I; recombine; select by S
  if ((st = rosetta_glwe_mul_plain(x_rlwe, plain_prep_dev + B.a_hat(0),
                                   plain_prep_dev + B.b_hat(0), ws[7], batch, ns, N, s)))
    return st;
  if ((st = rosetta_blind_rotate_glwe(ws[6], bsk_dev, ws[7], ws[8], batch, ns, p, 0, s)))
    return st;
  if ((st = rosetta_trace(ws[8], autk_dev, ws[8], batch * ns, p, tl, tb, s))) return st;
  std::vector<uint32_t> ex(ns);
  for (uint32_t j = 0; j < ns; ++j) ex[j] = j * (N / ns);
  if ((st = rosetta_glwe_recombine(ws[8], ex.data(), ws[9], batch, ns, N, s))) return st;
  if ((st = rosetta_glwe_mul_plain(ws[9], plain_prep_dev + B.window(), nullptr, ws[10], batch, 1,
                                   N, s)))
    return st;
  if ((st = rosetta_blind_rotate_glwe(ws[3], bsk_dev, ws[10], out, batch, 1, p, 0, s))) return st;
  return rosetta_trace(out, autk_dev, out, batch, p, tl, tb, s);
}

}  // extern "C"
