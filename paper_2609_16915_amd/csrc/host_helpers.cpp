// Host-side helpers of librosetta: key generation (bootstrapping,
// key-switching and automorphism keys), LWE and GLWE encryption, decryption
// and phases, and the test polynomial of a lookup table.  They produce test
// and benchmark inputs; none of them is on the PBS path.  The GLWE products
// A*S of key generation use a host transform over the same field (merged
// Cooley-Tukey forward, Gentleman-Sande inverse) and run over all host
// threads; every random draw is a pure function of (seed, stream, index),
// so the result does not depend on the thread count.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

#include "gl.hpp"
#include "internal.hpp"
#include "rosetta.h"

using namespace rosetta;

namespace {

// SplitMix64 output number idx (0-based) from state `key`
// (Steele, Lea and Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014).
inline u64 sm64(u64 key, u64 idx) {
  u64 z = key + (idx + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

enum Stream : u64 {
  LWE_KEY = 1, GLWE_KEY = 2, BSK_MASK = 3, BSK_NOISE = 4,
  KSK_MASK = 5, KSK_NOISE = 6, ENC_MASK = 7, ENC_NOISE = 8,
  AUTK_MASK = 9, AUTK_NOISE = 10, GLWE_ENC_MASK = 11, GLWE_ENC_NOISE = 12
};

inline u64 substream(u64 seed, Stream s) { return sm64(seed, (u64)s); }

inline u64 uniform_zp(u64 key, u64 idx) {
  const u64 w = sm64(key, idx);
  return w >= GL_P ? w - GL_P : w;
}

// Box-Muller transform of words 2g and 2g+1.
inline double std_normal(u64 key, u64 g) {
  const u64 w1 = sm64(key, 2 * g), w2 = sm64(key, 2 * g + 1);
  const double u1 = (double)((w1 >> 11) + 1) * 0x1.0p-53;  // (0, 1]
  const double u2 = (double)(w2 >> 11) * 0x1.0p-53;        // [0, 1)
  return std::sqrt(-2.0 * std::log(u1)) * std::cos(6.283185307179586 * u2);
}

// Rounded Gaussian with standard deviation sigma * 2^64, into Z_p.
inline u64 noise_zp(u64 key, u64 g, double sigma) {
  const double sd = std::ldexp(sigma, 64);
  const double x = std::floor(sd * std_normal(key, g) + 0.5);
  return gl_from_i64((i64)x);
}

// Host negacyclic transform for the key-generation products.
struct HostNtt {
  int N = 0, logn = 0;
  std::vector<u64> z, zi;
  u64 ninv = 0;
  explicit HostNtt(int n_) : N(n_) {
    while ((1 << logn) < N) ++logn;
    const u64 psi = gl_pow(7, (GL_P - 1) / (2 * (u64)N));
    z.resize(N);
    zi.resize(N);
    for (int m = 0; m < N; ++m) {
      int r = 0;
      for (int b = 0; b < logn; ++b)
        if (m & (1 << b)) r |= 1 << (logn - 1 - b);
      z[m] = gl_pow(psi, (u64)r);
      zi[m] = gl_pow(psi, (2 * (u64)N - (u64)r) % (2 * (u64)N));
    }
    ninv = gl_inv((u64)N);
  }
  void forward(u64 *a) const {
    for (int s = 0, len = N / 2; len >= 1; len >>= 1, ++s)
      for (int b = 0; b < (1 << s); ++b) {
        const u64 w = z[(1 << s) + b];
        for (int j = b * 2 * len; j < b * 2 * len + len; ++j) {
          const u64 t = gl_mul(a[j + len], w);
          a[j + len] = gl_sub(a[j], t);
          a[j] = gl_add(a[j], t);
        }
      }
  }
  void inverse(u64 *a) const {
    for (int s = logn - 1, len = 1; len < N; len <<= 1, --s)
      for (int b = 0; b < (1 << s); ++b) {
        const u64 w = zi[(1 << s) + b];
        for (int j = b * 2 * len; j < b * 2 * len + len; ++j) {
          const u64 u = a[j], v = a[j + len];
          a[j] = gl_add(u, v);
          a[j + len] = gl_mul(gl_sub(u, v), w);
        }
      }
    for (int j = 0; j < N; ++j) a[j] = gl_mul(a[j], ninv);
  }
};

template <class F>
void parallel_rows(size_t rows, F &&f) {
  unsigned nt = std::max(1u, std::min(32u, std::thread::hardware_concurrency()));
  if (rows < 64) nt = 1;
  std::vector<std::thread> th;
  for (unsigned w = 0; w < nt; ++w)
    th.emplace_back([&, w] {
      for (size_t r = w; r < rows; r += nt) f(r);
    });
  for (auto &t : th) t.join();
}

// a(X) -> a(X^d) modulo X^N + 1 (d odd).
void automorphism(const u64 *a, u64 *out, int N, u64 d) {
  for (int j = 0; j < N; ++j) {
    const u64 e = ((u64)j * d) & (2 * (u64)N - 1);
    if (e < (u64)N)
      out[e] = a[j];
    else
      out[e - N] = gl_neg(a[j]);
  }
}

// A * S for a GLWE key S already transformed (fS).
void mul_by_key(const HostNtt &ntt, const u64 *A, const std::vector<u64> &fS, u64 *out) {
  std::vector<u64> f(A, A + ntt.N);
  ntt.forward(f.data());
  for (int x = 0; x < ntt.N; ++x) f[x] = gl_mul(f[x], fS[x]);
  ntt.inverse(f.data());
  std::copy(f.begin(), f.end(), out);
}

bool ring_ok(const rosetta_params *p) {
  return p && p->N >= 4 && p->N <= 65536 && (p->N & (p->N - 1)) == 0;
}

rosetta_status herr(rosetta_status st, const char *msg) {
  set_last_error(msg);
  return st;
}

}  // namespace

extern "C" {

rosetta_status rosetta_keygen(uint64_t seed, const rosetta_params *p, double sigma_lwe,
                              double sigma_glwe, uint64_t *lwe_key, uint64_t *glwe_key,
                              uint64_t *bsk_std, uint64_t *ksk_std) {
  rosetta_status st = rosetta_check_params(p);
  if (st) return st;
  if (!lwe_key || !glwe_key || !bsk_std || !ksk_std)
    return herr(ROSETTA_ERR_NULL, "NULL pointer argument");
  const int n = (int)p->n, N = (int)p->N, l = (int)p->pbs_level, lk = (int)p->ks_level;
  const u64 k1 = substream(seed, LWE_KEY), k2 = substream(seed, GLWE_KEY);
  for (int i = 0; i < n; ++i) lwe_key[i] = sm64(k1, (u64)i) >> 63;
  for (int x = 0; x < N; ++x) glwe_key[x] = sm64(k2, (u64)x) >> 63;

  HostNtt ntt(N);
  std::vector<u64> fS(glwe_key, glwe_key + N);
  ntt.forward(fS.data());

  const u64 kbm = substream(seed, BSK_MASK), kbn = substream(seed, BSK_NOISE);
  parallel_rows((size_t)n * 2 * l, [&](size_t r) {
    const int i = (int)(r / (2 * l)), u = (int)((r / l) % 2), t = (int)(r % l);
    u64 *A = bsk_std + r * 2 * N, *B = A + N;
    std::vector<u64> f(N);
    for (int x = 0; x < N; ++x) f[x] = A[x] = uniform_zp(kbm, (u64)r * N + x);
    ntt.forward(f.data());
    for (int x = 0; x < N; ++x) f[x] = gl_mul(f[x], fS[x]);
    ntt.inverse(f.data());
    for (int x = 0; x < N; ++x) B[x] = gl_add(f[x], noise_zp(kbn, (u64)r * N + x, sigma_glwe));
    if (lwe_key[i]) {
      const u64 g = gl_pow(2, (u64)(64 - (t + 1) * (int)p->pbs_base_log));
      if (u == 0)
        A[0] = gl_add(A[0], g);
      else
        B[0] = gl_add(B[0], g);
    }
  });

  const u64 kkm = substream(seed, KSK_MASK), kkn = substream(seed, KSK_NOISE);
  parallel_rows((size_t)N * lk, [&](size_t r) {
    const int j = (int)(r / lk), t = (int)(r % lk);
    u64 *row = ksk_std + r * (n + 1);
    u64 b = 0;
    for (int c = 0; c < n; ++c) {
      row[c] = uniform_zp(kkm, (u64)r * n + c);
      if (lwe_key[c]) b = gl_add(b, row[c]);
    }
    if (glwe_key[j]) b = gl_add(b, gl_pow(2, (u64)(64 - (t + 1) * (int)p->ks_base_log)));
    row[n] = gl_add(b, noise_zp(kkn, (u64)r, sigma_lwe));
  });
  return ROSETTA_OK;
}

rosetta_status rosetta_lwe_encrypt(uint64_t seed, const rosetta_params *p, double sigma,
                                   const uint64_t *key, uint32_t dim, const uint32_t *msgs,
                                   size_t count, uint64_t *out) {
  if (!p) return herr(ROSETTA_ERR_NULL, "params is NULL");
  if (!key || !msgs || !out) return herr(ROSETTA_ERR_NULL, "NULL pointer argument");
  if (p->msg_bits < 1 || p->msg_bits > 30) return herr(ROSETTA_ERR_PARAMS, "bad msg_bits");
  const u64 delta = GL_P / (2ull << p->msg_bits);
  const u64 km = substream(seed, ENC_MASK), kn = substream(seed, ENC_NOISE);
  parallel_rows(count, [&](size_t q) {
    u64 *ct = out + q * (dim + 1);
    u64 b = 0;
    for (uint32_t c = 0; c < dim; ++c) {
      ct[c] = uniform_zp(km, (u64)q * dim + c);
      b = gl_add(b, gl_mul(ct[c], key[c]));
    }
    b = gl_add(b, gl_mul(delta, (u64)msgs[q]));
    ct[dim] = gl_add(b, noise_zp(kn, (u64)q, sigma));
  });
  return ROSETTA_OK;
}

rosetta_status rosetta_lwe_encrypt_plain(uint64_t seed, double sigma, const uint64_t *key,
                                         uint32_t dim, const uint64_t *plain, size_t count,
                                         uint64_t *out) {
  if (!key || !plain || !out) return herr(ROSETTA_ERR_NULL, "NULL pointer argument");
  const u64 km = substream(seed, ENC_MASK), kn = substream(seed, ENC_NOISE);
  parallel_rows(count, [&](size_t q) {
    u64 *ct = out + q * (dim + 1);
    u64 b = 0;
    for (uint32_t c = 0; c < dim; ++c) {
      ct[c] = uniform_zp(km, (u64)q * dim + c);
      b = gl_add(b, gl_mul(ct[c], key[c]));
    }
    b = gl_add(b, plain[q] >= GL_P ? plain[q] - GL_P : plain[q]);
    ct[dim] = gl_add(b, noise_zp(kn, (u64)q, sigma));
  });
  return ROSETTA_OK;
}

rosetta_status rosetta_lwe_decrypt(const rosetta_params *p, const uint64_t *key, uint32_t dim,
                                   const uint64_t *lwe, size_t count, uint32_t *msgs_out) {
  if (!p) return herr(ROSETTA_ERR_NULL, "params is NULL");
  if (!key || !lwe || !msgs_out) return herr(ROSETTA_ERR_NULL, "NULL pointer argument");
  if (p->msg_bits < 1 || p->msg_bits > 30) return herr(ROSETTA_ERR_PARAMS, "bad msg_bits");
  const u64 twoM = 2ull << p->msg_bits;
  for (size_t q = 0; q < count; ++q) {
    const u64 *ct = lwe + q * (dim + 1);
    u64 ph = ct[dim];
    for (uint32_t c = 0; c < dim; ++c) ph = gl_sub(ph, gl_mul(ct[c], key[c]));
    const unsigned __int128 num = (unsigned __int128)twoM * ph + (GL_P - 1) / 2;
    msgs_out[q] = (uint32_t)((u64)(num / GL_P) % twoM);
  }
  return ROSETTA_OK;
}

rosetta_status rosetta_lut_build(const rosetta_params *p, const uint32_t *table,
                                 uint64_t *test_poly) {
  if (!p) return herr(ROSETTA_ERR_NULL, "params is NULL");
  if (!table || !test_poly) return herr(ROSETTA_ERR_NULL, "NULL pointer argument");
  if (p->msg_bits < 1 || p->N == 0 || (p->N & (p->N - 1)) || (1u << p->msg_bits) > p->N)
    return herr(ROSETTA_ERR_PARAMS, "need N a power of two and 2^msg_bits <= N");
  const int N = (int)p->N, M = 1 << p->msg_bits, box = N / M, h = box / 2;
  const u64 delta = GL_P / (2ull * M);
  for (int j = 0; j < N - h; ++j) test_poly[j] = gl_mul(delta, table[(j + h) / box]);
  for (int j = N - h; j < N; ++j) test_poly[j] = gl_neg(gl_mul(delta, table[0]));
  return ROSETTA_OK;
}

rosetta_status rosetta_glwe_encrypt(uint64_t seed, const rosetta_params *p, double sigma,
                                    const uint64_t *glwe_key, const uint64_t *msgs, size_t count,
                                    uint64_t *out) {
  if (!ring_ok(p)) return herr(p ? ROSETTA_ERR_PARAMS : ROSETTA_ERR_NULL, "need N a power of two");
  if (!glwe_key || !msgs || !out) return herr(ROSETTA_ERR_NULL, "NULL pointer argument");
  const int N = (int)p->N;
  HostNtt ntt(N);
  std::vector<u64> fS(glwe_key, glwe_key + N);
  ntt.forward(fS.data());
  const u64 km = substream(seed, GLWE_ENC_MASK), kn = substream(seed, GLWE_ENC_NOISE);
  parallel_rows(count, [&](size_t q) {
    u64 *A = out + q * 2 * N, *B = A + N;
    for (int x = 0; x < N; ++x) A[x] = uniform_zp(km, (u64)q * N + x);
    mul_by_key(ntt, A, fS, B);
    for (int x = 0; x < N; ++x)
      B[x] = gl_add(gl_add(B[x], msgs[q * N + x]), noise_zp(kn, (u64)q * N + x, sigma));
  });
  return ROSETTA_OK;
}

rosetta_status rosetta_glwe_phase(const rosetta_params *p, const uint64_t *glwe_key,
                                  const uint64_t *glwe, size_t count, uint64_t *phase_out) {
  if (!ring_ok(p)) return herr(p ? ROSETTA_ERR_PARAMS : ROSETTA_ERR_NULL, "need N a power of two");
  if (!glwe_key || !glwe || !phase_out) return herr(ROSETTA_ERR_NULL, "NULL pointer argument");
  const int N = (int)p->N;
  HostNtt ntt(N);
  std::vector<u64> fS(glwe_key, glwe_key + N);
  ntt.forward(fS.data());
  parallel_rows(count, [&](size_t q) {
    const u64 *A = glwe + q * 2 * N, *B = A + N;
    u64 *o = phase_out + q * N;
    mul_by_key(ntt, A, fS, o);
    for (int x = 0; x < N; ++x) o[x] = gl_sub(B[x], o[x]);
  });
  return ROSETTA_OK;
}

rosetta_status rosetta_autk_keygen(uint64_t seed, const rosetta_params *p, uint32_t level,
                                   uint32_t base_log, double sigma, const uint64_t *glwe_key,
                                   uint64_t *autk) {
  if (!ring_ok(p)) return herr(p ? ROSETTA_ERR_PARAMS : ROSETTA_ERR_NULL, "need N a power of two");
  if (!glwe_key || !autk) return herr(ROSETTA_ERR_NULL, "NULL pointer argument");
  if (level < 1 || base_log < 1 || level * base_log > 62)
    return herr(ROSETTA_ERR_PARAMS, "need level, base_log >= 1 and level*base_log <= 62");
  const int N = (int)p->N;
  int logn = 0;
  while ((1 << logn) < N) ++logn;
  HostNtt ntt(N);
  std::vector<u64> fS(glwe_key, glwe_key + N);
  ntt.forward(fS.data());
  const u64 km = substream(seed, AUTK_MASK), kn = substream(seed, AUTK_NOISE);
  parallel_rows((size_t)logn * level, [&](size_t r) {
    const int k = (int)(r / level) + 1, t = (int)(r % level);
    u64 *A = autk + r * 2 * N, *B = A + N;
    std::vector<u64> ts(N);
    automorphism(glwe_key, ts.data(), N, (1ull << k) + 1);
    const u64 g = gl_pow(2, (u64)(64 - (t + 1) * (int)base_log));
    for (int x = 0; x < N; ++x) A[x] = uniform_zp(km, (u64)r * N + x);
    mul_by_key(ntt, A, fS, B);
    for (int x = 0; x < N; ++x)
      B[x] = gl_add(gl_add(B[x], noise_zp(kn, (u64)r * N + x, sigma)), gl_mul(ts[x], g));
  });
  return ROSETTA_OK;
}

}  // extern "C"
