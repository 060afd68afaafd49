// C ABI of librosetta: host-side validation, per-device state (transform
// tables, PBS workspace) and dispatch to the HIP kernels.  Nothing here
// computes on the host except the twiddle tables; every step of the PBS runs
// in kernels.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "gl.hpp"
#include "internal.hpp"
#include "rosetta.h"

using namespace rosetta;

static __device__ __align__(256) uint64_t twiddle_store[256 + 512 + 1024 + 2048 + 4096];
static __device__ __align__(256) uint64_t psi_store[256 + 512 + 1024 + 2048 + 4096];

namespace {

thread_local std::string g_last_error;

rosetta_status fail(rosetta_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

rosetta_status ok() {
  g_last_error.clear();
  return ROSETTA_OK;
}

rosetta_status hip_fail(hipError_t e, const char *what) {
  if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation)
    return fail(ROSETTA_ERR_NOMEM, "%s: %s", what, hipGetErrorString(e));
  return fail(ROSETTA_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

bool is_pow2_in(uint32_t N, uint32_t lo, uint32_t hi) {
  return N >= lo && N <= hi && (N & (N - 1)) == 0;
}

int ilog2u(uint32_t N) {
  int l = 0;
  while ((1u << l) < N) ++l;
  return l;
}

rosetta_status check_params(const rosetta_params *p) {
  if (!p) return fail(ROSETTA_ERR_NULL, "params is NULL");
  if (p->k != 1) return fail(ROSETTA_ERR_UNSUPPORTED, "only k = 1 is supported (got %u)", p->k);
  if (!is_pow2_in(p->N, 256, 4096))
    return fail(ROSETTA_ERR_UNSUPPORTED, "N must be a power of two in [256, 4096] (got %u)",
                p->N);
  if (p->n < 1) return fail(ROSETTA_ERR_PARAMS, "n must be >= 1");
  if (p->n > MAX_LWE_N)
    return fail(ROSETTA_ERR_UNSUPPORTED, "n must be <= %u (got %u)", MAX_LWE_N, p->n);
  if (p->pbs_level < 1 || p->pbs_base_log < 1)
    return fail(ROSETTA_ERR_PARAMS, "pbs_level and pbs_base_log must be >= 1");
  if (p->pbs_level > 4 || p->pbs_base_log > 30 || p->pbs_level * p->pbs_base_log > 62)
    return fail(ROSETTA_ERR_UNSUPPORTED,
                "need pbs_level <= 4, pbs_base_log <= 30 and l*beta <= 62");
  if (p->ks_level < 1 || p->ks_base_log < 1)
    return fail(ROSETTA_ERR_PARAMS, "ks_level and ks_base_log must be >= 1");
  if (p->ks_level > 8 || p->ks_base_log > 30 || p->ks_level * p->ks_base_log > 62)
    return fail(ROSETTA_ERR_UNSUPPORTED, "need ks_level <= 8, ks_base_log <= 30, l*beta <= 62");
  const unsigned long long acc_bound =
      (unsigned long long)p->N * p->ks_level << p->ks_base_log;
  if (acc_bound >= (1ull << 32))
    return fail(ROSETTA_ERR_UNSUPPORTED, "N * ks_level * 2^ks_base_log must be < 2^32");
  if (p->msg_bits < 1 || p->msg_bits > 20 || (1u << p->msg_bits) > p->N)
    return fail(ROSETTA_ERR_PARAMS, "need 1 <= msg_bits and 2^msg_bits <= N");
  return ROSETTA_OK;
}

// [a, a + na) and [b, b + nb) overlap without being the same range start
bool partial_overlap(const void *a, size_t na, const void *b, size_t nb) {
  const char *x = (const char *)a, *y = (const char *)b;
  if (x == y) return false;
  return x < y + nb && y < x + na;
}

bool any_overlap(const void *a, size_t na, const void *b, size_t nb) {
  const char *x = (const char *)a, *y = (const char *)b;
  return x < y + nb && y < x + na;
}

// ---- per-device state ------------------------------------------------------

// Twiddle tables of every supported N live in one static device array (N
// words each, at offset N - 256: 256 -> 0, 512 -> 256, .., 4096 -> 3840),
// and the powers psi^0 .. psi^(N-1) in a second one laid out alike, both
// uploaded per device on first use of an N, so that no entry point ever
// allocates memory for them.  Host code reaches the array only through the
// address hipGetSymbolAddress returns on each device.
constexpr size_t TWIDDLE_STORE_WORDS = 256 + 512 + 1024 + 2048 + 4096;

struct DeviceState {
  uint64_t *twiddle_base = nullptr;  // this device's copy of twiddle_store
  uint64_t *psi_base = nullptr;      // this device's copy of psi_store
  std::map<uint32_t, uint64_t> ninv;  // N -> N^-1, present once uploaded
  void *workspace = nullptr;
  size_t workspace_bytes = 0;
};

std::mutex g_mu;
std::map<int, DeviceState> g_dev;

uint32_t bitrev(uint32_t x, int bits) {
  uint32_t r = 0;
  for (int b = 0; b < bits; ++b)
    if (x & (1u << b)) r |= 1u << (bits - 1 - b);
  return r;
}

rosetta_status get_tables(uint32_t N, Tables &out) {
  if (!is_pow2_in(N, 256, 4096))
    return fail(ROSETTA_ERR_UNSUPPORTED, "no twiddle table for N = %u", N);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceState &ds = g_dev[dev];
  if (!ds.twiddle_base) {
    e = hipGetSymbolAddress((void **)&ds.twiddle_base, HIP_SYMBOL(twiddle_store));
    if (e != hipSuccess) {
      ds.twiddle_base = nullptr;
      return hip_fail(e, "hipGetSymbolAddress(twiddle_store)");
    }
  }
  if (!ds.psi_base) {
    e = hipGetSymbolAddress((void **)&ds.psi_base, HIP_SYMBOL(psi_store));
    if (e != hipSuccess) {
      ds.psi_base = nullptr;
      return hip_fail(e, "hipGetSymbolAddress(psi_store)");
    }
  }
  uint64_t *dst = ds.twiddle_base + (N - 256);
  auto it = ds.ninv.find(N);
  if (it == ds.ninv.end()) {
    const int logn = ilog2u(N);
    const u64 psi = gl_pow(7, (GL_P - 1) / (2 * (u64)N));
    std::vector<u64> z(N);
    for (uint32_t m = 0; m < N; ++m) z[m] = gl_pow(psi, bitrev(m, logn));
    // The pass structure of the kernels' transform (E = 2^le elements per
    // thread, pass 0 spanning f stages, every later pass le: ntt_le and
    // ntt_first).  Passes after the first that span le = 3 stages run in
    // twisted radix-8 form: their table region [2^s0, 2^(s0+3)) (the
    // twiddles of stages s0..s0+2, read by no other pass) becomes the powers
    // q^1..q^7 of q = zeta[4 (2^s0 + b)], 7 words per block b.  The last pass (threads own E consecutive
    // indices), when it is not twisted: each of its stages s stores block
    // t nc + c (nc = E / 2^(logn - s) blocks per thread, T = N / E threads)
    // at 2^s + c T + t.
    {
      const int le = ntt_le(logn), f = ntt_first(logn);
      std::vector<int> begin;  // first stage of each pass
      for (int s = 0; s < logn; s += begin.size() == 1 ? f : le) begin.push_back(s);
      const std::vector<u64> z0 = z;
      const int s_last = begin.back();
      const bool last_twisted = begin.size() > 1 && le == 3 && logn - s_last == le;
      if (!last_twisted) {
        const uint32_t T = N >> le;
        for (int s = s_last; s < logn; ++s) {
          const uint32_t nc = (1u << le) >> (logn - s);
          for (uint32_t t = 0; t < T; ++t)
            for (uint32_t c = 0; c < nc; ++c) z[(1u << s) + c * T + t] = z0[(1u << s) + t * nc + c];
        }
      }
      for (size_t q = 1; q < begin.size(); ++q) {
        const int s0 = begin[q];
        if (le != 3 || std::min(logn, s0 + le) - s0 != le) continue;
        const uint32_t nb = 1u << s0, np = (1u << le) - 1;
        for (uint32_t b = 0; b < nb; ++b) {
          const u64 qq = z0[(1u << (le - 1)) * (nb + b)];
          u64 pw = qq;
          for (uint32_t i = 0; i < np; ++i) {
            z[nb + np * b + i] = pw;
            pw = gl_mul(pw, qq);
          }
        }
      }
    }
    static_assert(256 + 512 + 1024 + 2048 + 4096 == TWIDDLE_STORE_WORDS, "table offsets");
    e = hipMemcpy(dst, z.data(), z.size() * sizeof(u64), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy(twiddles)");
    // psi^e, e < N, for the transform-domain rotation (Tables::psi)
    std::vector<u64> pw(N);
    pw[0] = 1;
    for (uint32_t i = 1; i < N; ++i) pw[i] = gl_mul(pw[i - 1], psi);
    e = hipMemcpy(ds.psi_base + (N - 256), pw.data(), pw.size() * sizeof(u64),
                  hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy(psi powers)");
    it = ds.ninv.emplace(N, gl_inv(N)).first;
  }
  out.zeta = dst;
  out.psi = ds.psi_base + (N - 256);
  out.ninv = it->second;
  return ROSETTA_OK;
}

rosetta_status get_workspace(size_t bytes, void **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceState &ds = g_dev[dev];
  if (ds.workspace_bytes < bytes) {
    if (ds.workspace) {
      // earlier calls may still read the old buffer
      e = hipDeviceSynchronize();
      if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
      (void)hipFree(ds.workspace);
      ds.workspace = nullptr;
      ds.workspace_bytes = 0;
    }
    e = hipMalloc(&ds.workspace, bytes);
    if (e != hipSuccess) {
      ds.workspace = nullptr;
      return hip_fail(e, "hipMalloc(workspace)");
    }
    ds.workspace_bytes = bytes;
  }
  *ptr = ds.workspace;
  return ROSETTA_OK;
}

size_t lwe_words(const rosetta_params *p, size_t batch) { return batch * (size_t)(p->n + 1); }

}  // namespace

void rosetta::set_last_error(const char *msg) { g_last_error = msg; }

extern "C" {

#ifndef ROSETTA_SOURCE_DIGEST
#define ROSETTA_SOURCE_DIGEST "unknown"
#endif
const char *rosetta_version(void) {
  return "rosetta-pbs 0.2.0 (gfx950) src:" ROSETTA_SOURCE_DIGEST;
}

const char *rosetta_status_string(int st) {
  switch (st) {
    case ROSETTA_OK: return "ROSETTA_OK";
    case ROSETTA_ERR_NULL: return "ROSETTA_ERR_NULL";
    case ROSETTA_ERR_PARAMS: return "ROSETTA_ERR_PARAMS";
    case ROSETTA_ERR_UNSUPPORTED: return "ROSETTA_ERR_UNSUPPORTED";
    case ROSETTA_ERR_ALIAS: return "ROSETTA_ERR_ALIAS";
    case ROSETTA_ERR_NOMEM: return "ROSETTA_ERR_NOMEM";
    case ROSETTA_ERR_DEVICE: return "ROSETTA_ERR_DEVICE";
    case ROSETTA_ERR_SIZE: return "ROSETTA_ERR_SIZE";
    default: return "ROSETTA_ERR_UNKNOWN";
  }
}

const char *rosetta_last_error(void) { return g_last_error.c_str(); }

rosetta_status rosetta_check_params(const rosetta_params *params) {
  rosetta_status st = check_params(params);
  return st == ROSETTA_OK ? ok() : st;
}

size_t rosetta_bsk_words(const rosetta_params *p) {
  return p ? (size_t)p->n * 2 * p->pbs_level * 2 * p->N : 0;
}

size_t rosetta_bsk_device_words(const rosetta_params *p) { return rosetta_bsk_words(p); }

size_t rosetta_ksk_words(const rosetta_params *p) {
  return p ? (size_t)p->N * p->ks_level * (p->n + 1) : 0;
}

size_t rosetta_ksk_device_words(const rosetta_params *p) {
  if (!p) return 0;
  return ks_on_matrix_cores(*p) ? ks_matrix_key_words(*p) : rosetta_ksk_words(p) + (p->n + 1);
}

rosetta_status rosetta_bsk_prepare(const uint64_t *bsk_std_dev, uint64_t *bsk_dev,
                                   const rosetta_params *params, void *stream) {
  rosetta_status st = check_params(params);
  if (st) return st;
  if (!bsk_std_dev || !bsk_dev) return fail(ROSETTA_ERR_NULL, "bsk pointer is NULL");
  const size_t bytes = rosetta_bsk_words(params) * 8;
  if (any_overlap(bsk_std_dev, bytes, bsk_dev, bytes))
    return fail(ROSETTA_ERR_ALIAS, "bsk_std_dev and bsk_dev overlap");
  Tables tb;
  if ((st = get_tables(params->N, tb))) return st;
  hipError_t e = launch_bsk_prepare(bsk_std_dev, bsk_dev, *params, tb, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "bsk_prepare launch");
}

rosetta_status rosetta_ksk_prepare(const uint64_t *ksk_std_dev, uint64_t *ksk_dev,
                                   const rosetta_params *params, void *stream) {
  rosetta_status st = check_params(params);
  if (st) return st;
  if (!ksk_std_dev || !ksk_dev) return fail(ROSETTA_ERR_NULL, "ksk pointer is NULL");
  if (any_overlap(ksk_std_dev, rosetta_ksk_words(params) * 8, ksk_dev,
                  rosetta_ksk_device_words(params) * 8))
    return fail(ROSETTA_ERR_ALIAS, "ksk_std_dev and ksk_dev overlap");
  hipError_t e = launch_ksk_prepare(ksk_std_dev, ksk_dev, *params, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "ksk_prepare launch");
}

size_t rosetta_pbs_workspace_bytes(const rosetta_params *p, size_t batch) {
  return p ? batch * (size_t)(p->N + 1) * sizeof(uint64_t) : 0;
}

static rosetta_status check_br_args(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                    const uint64_t *lut, const void *out, size_t out_bytes,
                                    size_t batch, const rosetta_params *p) {
  if (!lwe_in || !bsk_dev || !lut || !out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t in_bytes = lwe_words(p, batch) * 8;
  if (any_overlap(out, out_bytes, lwe_in, in_bytes) ||
      any_overlap(out, out_bytes, lut, (size_t)p->N * 8) ||
      any_overlap(out, out_bytes, bsk_dev, rosetta_bsk_words(p) * 8))
    return fail(ROSETTA_ERR_ALIAS, "output overlaps an input");
  return ROSETTA_OK;
}

rosetta_status rosetta_pbs_batch_ws(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                    const uint64_t *ksk_dev, const uint64_t *lut,
                                    uint64_t *lwe_out, size_t batch,
                                    const rosetta_params *params, void *workspace,
                                    size_t workspace_bytes, void *stream) {
  rosetta_status st = check_params(params);
  if (st) return st;
  if (batch == 0) return ok();
  if (!lwe_in || !bsk_dev || !ksk_dev || !lut || !lwe_out)
    return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  if (!workspace) return fail(ROSETTA_ERR_NULL, "workspace is NULL");
  const size_t need = rosetta_pbs_workspace_bytes(params, batch);
  if (workspace_bytes < need)
    return fail(ROSETTA_ERR_SIZE, "workspace of %zu bytes, need %zu", workspace_bytes, need);
  const size_t io = lwe_words(params, batch) * 8;
  if (partial_overlap(lwe_in, io, lwe_out, io))
    return fail(ROSETTA_ERR_ALIAS, "lwe_in and lwe_out partially overlap");
  if (any_overlap(workspace, need, lwe_in, io) || any_overlap(workspace, need, lwe_out, io) ||
      any_overlap(workspace, need, lut, (size_t)params->N * 8) ||
      any_overlap(lwe_out, io, lut, (size_t)params->N * 8) ||
      any_overlap(lwe_out, io, bsk_dev, rosetta_bsk_words(params) * 8) ||
      any_overlap(lwe_out, io, ksk_dev, rosetta_ksk_device_words(params) * 8))
    return fail(ROSETTA_ERR_ALIAS, "workspace or output overlaps another buffer");
  Tables tb;
  if ((st = get_tables(params->N, tb))) return st;
  uint64_t *big = (uint64_t *)workspace;
  hipError_t e = launch_blind_rotate(lwe_in, bsk_dev, lut, big, batch, *params, tb, BR_EXTRACT,
                                     0, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "blind_rotate launch");
  e = launch_keyswitch(big, ksk_dev, lwe_out, batch, *params, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "keyswitch launch");
  return ok();
}

rosetta_status rosetta_pbs_batch(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                 const uint64_t *ksk_dev, const uint64_t *lut, uint64_t *lwe_out,
                                 size_t batch, const rosetta_params *params, void *stream) {
  rosetta_status st = check_params(params);
  if (st) return st;
  if (batch == 0) return ok();
  if (!lwe_in || !bsk_dev || !ksk_dev || !lut || !lwe_out)
    return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  void *ws = nullptr;
  const size_t need = rosetta_pbs_workspace_bytes(params, batch);
  if ((st = get_workspace(need, &ws))) return st;
  return rosetta_pbs_batch_ws(lwe_in, bsk_dev, ksk_dev, lut, lwe_out, batch, params, ws, need,
                              stream);
}

rosetta_status rosetta_blind_rotate(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                    const uint64_t *lut, uint64_t *glwe_out, size_t batch,
                                    const rosetta_params *params, void *stream) {
  rosetta_status st = check_params(params);
  if (st) return st;
  if (batch == 0) return ok();
  if ((st = check_br_args(lwe_in, bsk_dev, lut, glwe_out, batch * 2 * (size_t)params->N * 8,
                          batch, params)))
    return st;
  Tables tb;
  if ((st = get_tables(params->N, tb))) return st;
  hipError_t e = launch_blind_rotate(lwe_in, bsk_dev, lut, glwe_out, batch, *params, tb, BR_GLWE,
                                     0, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "blind_rotate launch");
}

rosetta_status rosetta_blind_rotate_extract(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                            const uint64_t *lut, uint64_t *big_out,
                                            size_t batch, const rosetta_params *params,
                                            void *stream) {
  rosetta_status st = check_params(params);
  if (st) return st;
  if (batch == 0) return ok();
  if ((st = check_br_args(lwe_in, bsk_dev, lut, big_out, batch * ((size_t)params->N + 1) * 8,
                          batch, params)))
    return st;
  Tables tb;
  if ((st = get_tables(params->N, tb))) return st;
  hipError_t e = launch_blind_rotate(lwe_in, bsk_dev, lut, big_out, batch, *params, tb,
                                     BR_EXTRACT, 0, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "blind_rotate launch");
}

rosetta_status rosetta_keyswitch(const uint64_t *big_in, const uint64_t *ksk_dev,
                                 uint64_t *lwe_out, size_t batch, const rosetta_params *params,
                                 void *stream) {
  rosetta_status st = check_params(params);
  if (st) return st;
  if (batch == 0) return ok();
  if (!big_in || !ksk_dev || !lwe_out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t out_bytes = lwe_words(params, batch) * 8;
  if (any_overlap(lwe_out, out_bytes, big_in, batch * ((size_t)params->N + 1) * 8) ||
      any_overlap(lwe_out, out_bytes, ksk_dev, rosetta_ksk_device_words(params) * 8))
    return fail(ROSETTA_ERR_ALIAS, "output overlaps an input");
  hipError_t e = launch_keyswitch(big_in, ksk_dev, lwe_out, batch, *params, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "keyswitch launch");
}

static rosetta_status check_ntt_args(const void *in, const void *out, size_t count, uint32_t N) {
  if (!is_pow2_in(N, 256, 4096))
    return fail(ROSETTA_ERR_UNSUPPORTED, "N must be a power of two in [256, 4096]");
  if (count == 0) return ROSETTA_OK;
  if (!in || !out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t bytes = count * (size_t)N * 8;
  if (partial_overlap(in, bytes, out, bytes))
    return fail(ROSETTA_ERR_ALIAS, "in and out partially overlap");
  return ROSETTA_OK;
}

rosetta_status rosetta_ntt_forward(const uint64_t *in, uint64_t *out, size_t count, uint32_t N,
                                   void *stream) {
  rosetta_status st = check_ntt_args(in, out, count, N);
  if (st) return st;
  if (count == 0) return ok();
  Tables tb;
  if ((st = get_tables(N, tb))) return st;
  hipError_t e = launch_ntt(in, out, count, N, tb, false, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "ntt launch");
}

rosetta_status rosetta_ntt_inverse(const uint64_t *in, uint64_t *out, size_t count, uint32_t N,
                                   void *stream) {
  rosetta_status st = check_ntt_args(in, out, count, N);
  if (st) return st;
  if (count == 0) return ok();
  Tables tb;
  if ((st = get_tables(N, tb))) return st;
  hipError_t e = launch_ntt(in, out, count, N, tb, true, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "ntt launch");
}

rosetta_status rosetta_poly_mul(const uint64_t *a, const uint64_t *b, uint64_t *c, size_t count,
                                uint32_t N, void *stream) {
  rosetta_status st = check_ntt_args(a, c, count, N);
  if (st) return st;
  if ((st = check_ntt_args(b, c, count, N))) return st;
  if (count == 0) return ok();
  Tables tb;
  if ((st = get_tables(N, tb))) return st;
  hipError_t e = launch_poly_mul(a, b, c, count, N, tb, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "poly_mul launch");
}

rosetta_status rosetta_field_op(int op, const uint64_t *a, const uint64_t *b, const uint64_t *c,
                                uint64_t *out, size_t count, void *stream) {
  const bool pow2 = op >= ROSETTA_FIELD_MUL_POW2 && op < ROSETTA_FIELD_MUL_POW2 + 96;
  const bool round = op > ROSETTA_FIELD_ROUND_TOP && op < ROSETTA_FIELD_ROUND_TOP + 64;
  const bool unary = pow2 || round;
  if (!unary && (op < ROSETTA_FIELD_ADD || op > ROSETTA_FIELD_MUL_ADD_WEAK))
    return fail(ROSETTA_ERR_PARAMS, "unknown field op %d", op);
  if (count == 0) return ok();
  const bool reads_c = op == ROSETTA_FIELD_MUL_ADD || op == ROSETTA_FIELD_MUL_ADD_WEAK;
  if (!a || !out || (!unary && !b) || (reads_c && !c))
    return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  hipError_t e = launch_field_op(op, a, b, c, out, count, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "field_op launch");
}

rosetta_status rosetta_modmul_chain(uint64_t seed, uint32_t threads, uint32_t iters,
                                    uint64_t *out, void *stream) {
  if (threads == 0) return ok();
  if (!out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  hipError_t e = launch_modmul_chain(seed, threads, iters, out, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "modmul_chain launch");
}

// ---- lookup-protocol primitives -----------------------------------------

rosetta_status rosetta_blind_rotate_glwe(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                         const uint64_t *glwe_tp, uint64_t *out, size_t batch,
                                         uint32_t group, const rosetta_params *params,
                                         int extract, void *stream) {
  rosetta_status st = check_params(params);
  if (st) return st;
  if (group < 1 || group > 4096) return fail(ROSETTA_ERR_PARAMS, "need 1 <= group <= 4096");
  if (batch == 0) return ok();
  if (!lwe_in || !bsk_dev || !glwe_tp || !out)
    return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t N = params->N, tps = batch * group;
  const size_t out_bytes = tps * (extract ? N + 1 : 2 * N) * 8;
  if (any_overlap(out, out_bytes, lwe_in, lwe_words(params, batch) * 8) ||
      any_overlap(out, out_bytes, glwe_tp, tps * 2 * N * 8) ||
      any_overlap(out, out_bytes, bsk_dev, rosetta_bsk_words(params) * 8))
    return fail(ROSETTA_ERR_ALIAS, "output overlaps an input");
  Tables tb;
  if ((st = get_tables(params->N, tb))) return st;
  hipError_t e = launch_blind_rotate(lwe_in, bsk_dev, glwe_tp, out, tps, *params, tb,
                                     extract ? BR_EXTRACT : BR_GLWE, (int)group,
                                     (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "blind_rotate_glwe launch");
}

rosetta_status rosetta_lwe_add_consts(const uint64_t *lwe_in, const uint64_t *consts,
                                      uint64_t *lwe_out, size_t batch, uint32_t count,
                                      uint32_t dim, void *stream) {
  if (count < 1 || count > (uint32_t)(MAX_MONOMIALS / 4))
    return fail(ROSETTA_ERR_PARAMS, "need 1 <= count <= %d", MAX_MONOMIALS / 4);
  if (dim < 1) return fail(ROSETTA_ERR_PARAMS, "need dim >= 1");
  if (!consts) return fail(ROSETTA_ERR_NULL, "consts is NULL");
  Consts cs;
  for (uint32_t j = 0; j < count; ++j) {
    if (consts[j] >= GL_P) return fail(ROSETTA_ERR_PARAMS, "constant %u is not below p", j);
    cs.c[j] = consts[j];
  }
  if (batch == 0) return ok();
  if (!lwe_in || !lwe_out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t w = (size_t)dim + 1;
  if (any_overlap(lwe_out, batch * count * w * 8, lwe_in, batch * w * 8))
    return fail(ROSETTA_ERR_ALIAS, "output overlaps the input");
  hipError_t e = launch_lwe_add_consts(lwe_in, lwe_out, batch, (int)count, (int)dim, cs,
                                       (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "lwe_add_consts launch");
}

rosetta_status rosetta_lwe_combine(const uint64_t *a, uint64_t alpha, const uint64_t *b,
                                   uint64_t beta, const uint64_t *c, uint64_t gamma,
                                   uint64_t *out, size_t words, void *stream) {
  if (alpha >= GL_P || beta >= GL_P || gamma >= GL_P)
    return fail(ROSETTA_ERR_PARAMS, "coefficients must be below p");
  if (words == 0) return ok();
  if (!a || !out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t bytes = words * 8;
  if (partial_overlap(a, bytes, out, bytes) || (b && partial_overlap(b, bytes, out, bytes)) ||
      (c && partial_overlap(c, bytes, out, bytes)))
    return fail(ROSETTA_ERR_ALIAS, "out partially overlaps an input");
  hipError_t e = launch_lwe_combine(a, alpha, b, beta, c, gamma, out, words, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "lwe_combine launch");
}

rosetta_status rosetta_lwe_sum_groups(const uint64_t *lwe_in, uint64_t c0, uint64_t *lwe_out,
                                      size_t batch, uint32_t count, uint32_t dim,
                                      void *stream) {
  if (count < 1 || dim < 1) return fail(ROSETTA_ERR_PARAMS, "need count, dim >= 1");
  if (c0 >= GL_P) return fail(ROSETTA_ERR_PARAMS, "constant is not below p");
  if (batch == 0) return ok();
  if (!lwe_in || !lwe_out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t w = (size_t)dim + 1;
  if (any_overlap(lwe_out, batch * w * 8, lwe_in, batch * count * w * 8))
    return fail(ROSETTA_ERR_ALIAS, "output overlaps the input");
  hipError_t e = launch_lwe_sum_groups(lwe_in, lwe_out, batch, (int)count, (int)dim, c0,
                                       (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "lwe_sum_groups launch");
}

static rosetta_status check_trace_params(const rosetta_params *p, uint32_t level,
                                         uint32_t base_log) {
  rosetta_status st = check_params(p);
  if (st) return st;
  if (level < 1 || base_log < 1)
    return fail(ROSETTA_ERR_PARAMS, "trace level and base_log must be >= 1");
  if (level > 4 || base_log > 30 || level * base_log > 62)
    return fail(ROSETTA_ERR_UNSUPPORTED,
                "need trace level <= 4, base_log <= 30 and level*base_log <= 62");
  return ROSETTA_OK;
}

size_t rosetta_autk_words(const rosetta_params *p, uint32_t level) {
  return p ? (size_t)ilog2u(p->N) * level * 2 * p->N : 0;
}

rosetta_status rosetta_autk_prepare(const uint64_t *autk_std_dev, uint64_t *autk_dev,
                                    const rosetta_params *params, uint32_t level,
                                    void *stream) {
  rosetta_status st = check_trace_params(params, level, 1);
  if (st) return st;
  if (!autk_std_dev || !autk_dev) return fail(ROSETTA_ERR_NULL, "autk pointer is NULL");
  const size_t words = rosetta_autk_words(params, level);
  if (any_overlap(autk_std_dev, words * 8, autk_dev, words * 8))
    return fail(ROSETTA_ERR_ALIAS, "autk_std_dev and autk_dev overlap");
  Tables tb;
  if ((st = get_tables(params->N, tb))) return st;
  hipError_t e = launch_rows_prepare(autk_std_dev, autk_dev, words / params->N, params->N, tb,
                                     (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "autk_prepare launch");
}

rosetta_status rosetta_trace(const uint64_t *glwe_in, const uint64_t *autk_dev,
                             uint64_t *glwe_out, size_t batch, const rosetta_params *params,
                             uint32_t level, uint32_t base_log, void *stream) {
  rosetta_status st = check_trace_params(params, level, base_log);
  if (st) return st;
  if (batch == 0) return ok();
  if (!glwe_in || !autk_dev || !glwe_out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t bytes = batch * 2 * (size_t)params->N * 8;
  if (partial_overlap(glwe_in, bytes, glwe_out, bytes))
    return fail(ROSETTA_ERR_ALIAS, "glwe_in and glwe_out partially overlap");
  if (any_overlap(glwe_out, bytes, autk_dev, rosetta_autk_words(params, level) * 8))
    return fail(ROSETTA_ERR_ALIAS, "output overlaps the automorphism key");
  Tables tb;
  if ((st = get_tables(params->N, tb))) return st;
  hipError_t e = launch_trace(glwe_in, autk_dev, glwe_out, batch, params->N, (int)level,
                              (int)base_log, tb, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "trace launch");
}

rosetta_status rosetta_plain_prepare(const uint64_t *plain_dev, uint64_t *plain_prep_dev,
                                     size_t count, uint32_t N, void *stream) {
  rosetta_status st = check_ntt_args(plain_dev, plain_prep_dev, count, N);
  if (st) return st;
  if (count == 0) return ok();
  if (any_overlap(plain_dev, count * (size_t)N * 8, plain_prep_dev, count * (size_t)N * 8))
    return fail(ROSETTA_ERR_ALIAS, "plain_dev and plain_prep_dev overlap");
  Tables tb;
  if ((st = get_tables(N, tb))) return st;
  hipError_t e = launch_rows_prepare(plain_dev, plain_prep_dev, count, N, tb,
                                     (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "plain_prepare launch");
}

rosetta_status rosetta_glwe_mul_plain(const uint64_t *glwe_in, const uint64_t *pa_prep_dev,
                                      const uint64_t *pb_dev, uint64_t *glwe_out, size_t batch,
                                      uint32_t npoly, uint32_t N, void *stream) {
  if (!is_pow2_in(N, 256, 4096))
    return fail(ROSETTA_ERR_UNSUPPORTED, "N must be a power of two in [256, 4096]");
  if (npoly < 1 || npoly > 4096) return fail(ROSETTA_ERR_PARAMS, "need 1 <= npoly <= 4096");
  if (batch == 0) return ok();
  if (!glwe_in || !pa_prep_dev || !glwe_out)
    return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t in_bytes = batch * 2 * (size_t)N * 8, out_bytes = in_bytes * npoly;
  const size_t pbytes = (size_t)npoly * N * 8;
  if (any_overlap(glwe_out, out_bytes, glwe_in, in_bytes) ||
      any_overlap(glwe_out, out_bytes, pa_prep_dev, pbytes) ||
      (pb_dev && any_overlap(glwe_out, out_bytes, pb_dev, pbytes)))
    return fail(ROSETTA_ERR_ALIAS, "output overlaps an input");
  Tables tb;
  rosetta_status st = get_tables(N, tb);
  if (st) return st;
  hipError_t e = launch_glwe_mul_plain(glwe_in, pa_prep_dev, pb_dev, glwe_out, batch, (int)npoly,
                                       N, tb, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "glwe_mul_plain launch");
}

static rosetta_status load_exponents(const uint32_t *exps, uint32_t count, uint32_t N,
                                     Exponents &ex) {
  if (count < 1 || count > (uint32_t)MAX_MONOMIALS)
    return fail(ROSETTA_ERR_PARAMS, "need 1 <= count <= %d", MAX_MONOMIALS);
  for (uint32_t s = 0; s < count; ++s) {
    const uint32_t e = exps ? exps[s] : s;
    if (e >= 2 * N) return fail(ROSETTA_ERR_PARAMS, "exponent %u is not below 2N", e);
    ex.e[s] = (uint16_t)e;
  }
  return ROSETTA_OK;
}

rosetta_status rosetta_glwe_recombine(const uint64_t *glwe_in, const uint32_t *exps,
                                      uint64_t *glwe_out, size_t batch, uint32_t count,
                                      uint32_t N, void *stream) {
  if (!is_pow2_in(N, 256, 4096))
    return fail(ROSETTA_ERR_UNSUPPORTED, "N must be a power of two in [256, 4096]");
  Exponents ex;
  rosetta_status st = load_exponents(exps, count, N, ex);
  if (st) return st;
  if (batch == 0) return ok();
  if (!glwe_in || !glwe_out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t out_bytes = batch * 2 * (size_t)N * 8;
  if (any_overlap(glwe_out, out_bytes, glwe_in, out_bytes * count))
    return fail(ROSETTA_ERR_ALIAS, "output overlaps the input");
  hipError_t e = launch_glwe_recombine(glwe_in, glwe_out, batch, (int)count, ex, N,
                                       (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "glwe_recombine launch");
}

rosetta_status rosetta_glwe_monomial_mul(const uint64_t *glwe_in, const uint32_t *exps,
                                         uint64_t *glwe_out, size_t batch, uint32_t count,
                                         uint32_t N, void *stream) {
  if (!is_pow2_in(N, 256, 4096))
    return fail(ROSETTA_ERR_UNSUPPORTED, "N must be a power of two in [256, 4096]");
  if (!exps) return fail(ROSETTA_ERR_NULL, "exps is NULL");
  Exponents ex;
  rosetta_status st = load_exponents(exps, count, N, ex);
  if (st) return st;
  if (batch == 0) return ok();
  if (!glwe_in || !glwe_out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  const size_t in_bytes = batch * 2 * (size_t)N * 8;
  if (any_overlap(glwe_out, in_bytes * count, glwe_in, in_bytes))
    return fail(ROSETTA_ERR_ALIAS, "output overlaps the input");
  hipError_t e = launch_glwe_monomial_mul(glwe_in, glwe_out, batch, (int)count, ex, N,
                                          (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "glwe_monomial_mul launch");
}

rosetta_status rosetta_sample_extract(const uint64_t *glwe_in, uint64_t *big_out, size_t batch,
                                      uint32_t N, void *stream) {
  if (!is_pow2_in(N, 256, 4096))
    return fail(ROSETTA_ERR_UNSUPPORTED, "N must be a power of two in [256, 4096]");
  if (batch == 0) return ok();
  if (!glwe_in || !big_out) return fail(ROSETTA_ERR_NULL, "NULL pointer argument");
  if (any_overlap(big_out, batch * (size_t)(N + 1) * 8, glwe_in, batch * 2 * (size_t)N * 8))
    return fail(ROSETTA_ERR_ALIAS, "output overlaps the input");
  hipError_t e = launch_sample_extract(glwe_in, big_out, batch, N, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "sample_extract launch");
}

rosetta_status rosetta_shutdown(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  int cur = 0;
  (void)hipGetDevice(&cur);
  for (auto &kv : g_dev) {
    (void)hipSetDevice(kv.first);
    (void)hipDeviceSynchronize();
    // the transform tables stay: they live in static device memory
    if (kv.second.workspace) (void)hipFree(kv.second.workspace);
    kv.second.workspace = nullptr;
    kv.second.workspace_bytes = 0;
  }
  (void)hipSetDevice(cur);
  return ok();
}

}  // extern "C"
