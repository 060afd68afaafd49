// Negacyclic NTT of one polynomial per workgroup, held in registers.
//
// N = 2^LOGN coefficients are spread over T = N / E threads, E = 2^LE per
// thread.  The forward transform is the merged-twist Cooley-Tukey form: stage
// s (s = 0 .. LOGN-1) pairs indices j and j + N/2^(s+1) inside block
// b = j >> (LOGN - s) and multiplies the upper element by
// zeta[2^s + b] = psi^rev(2^s + b)  (psi a primitive 2N-th root of unity,
// rev the LOGN-bit reversal), so the result at in-place index j is
// a(psi^(2 rev(j) + 1)).  The inverse runs the Gentleman-Sande mirror with
// the inverse twiddles and leaves the factor N for the caller.
//
// Stages are grouped into passes of LE stages.  During pass q a thread holds
// the E elements whose index bits [lo_q, lo_q + LE) vary, lo_q =
// max(0, LOGN - (q+1) LE); the thread id fills the remaining bits in order:
//   j = (tid mod 2^lo) + (k << lo) + ((tid >> lo) << (lo + LE)).
// Butterflies inside a pass are register-only; between passes the workgroup
// transposes through LDS (one write, one barrier, one read), alternating
// between two buffers so that one barrier per transpose suffices.  Pass 0
// is the natural layout j = tid + T*k.
//
// Addresses are written as a per-thread base plus a compile-time offset per
// element, so that LDS accesses use the instructions' immediate offsets and
// twiddle loads need one address register per stage.
#pragma once

#include "gl.hpp"

namespace rosetta {

typedef const u64 __attribute__((address_space(1))) gconst_u64;

template <int LOGN_, int LE_>
struct Ntt {
  static constexpr int LOGN = LOGN_;
  static constexpr int LE = LE_;
  static constexpr int N = 1 << LOGN;
  static constexpr int E = 1 << LE;
  static constexpr int T = N / E;
  static constexpr int PASSES = (LOGN + LE - 1) / LE;
  // one padding word every 32 elements breaks power-of-two strides
  static constexpr int PAD_SHIFT = 5;
  static constexpr int LDS_WORDS = N + (N >> PAD_SHIFT);

  __host__ __device__ static constexpr int lo(int q) {
    return (LOGN - (q + 1) * LE) > 0 ? (LOGN - (q + 1) * LE) : 0;
  }
  __host__ __device__ static constexpr int stage_begin(int q) { return q * LE; }
  __host__ __device__ static constexpr int stage_end(int q) {
    return (q + 1) * LE < LOGN ? (q + 1) * LE : LOGN;
  }
  __host__ __device__ static constexpr int pad(int j) { return j + (j >> PAD_SHIFT); }
  // index held by element k of thread tid during pass q
  __host__ __device__ static constexpr int idx(int q, int tid, int k) {
    return (tid & ((1 << lo(q)) - 1)) + (k << lo(q)) + ((tid >> lo(q)) << (lo(q) + LE));
  }
  // padded LDS word of element k = per-thread base + constant offset.  The
  // thread part and the k part of the index occupy disjoint bits, so the
  // padding (j >> 5) splits the same way.
  __host__ __device__ static constexpr int lds_base(int q, int tid) {
    return pad(idx(q, tid, 0));
  }
  __host__ __device__ static constexpr int lds_off(int q, int k) { return pad(k << lo(q)); }
};

// Forward stages of pass Q.  For stage s (shift sh = LOGN - s) the twiddle
// of the pair led by element k is
//   zeta[2^s + ((tid >> lo) << (lo + LE - sh)) + ((k >> (sh - lo)) ...)],
// i.e. a per-thread base for the stage plus a compile-time offset.
template <class S, int Q>
__device__ __forceinline__ void ntt_fwd_pass(u64 (&x)[S::E], int tid, gconst_u64 *zeta) {
  constexpr int lo = S::lo(Q);
  const int hb = tid >> lo;
#pragma unroll
  for (int s = S::stage_begin(Q); s < S::stage_end(Q); ++s) {
    const int sh = S::LOGN - s;
    const int b = sh - 1 - lo;  // k-bit split by this stage
    gconst_u64 *zs = zeta + (1 << s) + (hb << (lo + S::LE - sh));
#pragma unroll
    for (int k = 0; k < S::E; ++k) {
      if (k & (1 << b)) continue;
      const int k2 = k | (1 << b);
      const u64 w = zs[k >> (sh - lo)];
      const u64 t = gl_mul(x[k2], w);
      x[k2] = gl_sub(x[k], t);
      x[k] = gl_add(x[k], t);
    }
  }
}

// Inverse (Gentleman-Sande) stages of pass Q, in reverse stage order.
template <class S, int Q>
__device__ __forceinline__ void ntt_inv_pass(u64 (&x)[S::E], int tid, gconst_u64 *zeta_inv) {
  constexpr int lo = S::lo(Q);
  const int hb = tid >> lo;
#pragma unroll
  for (int s = S::stage_end(Q) - 1; s >= S::stage_begin(Q); --s) {
    const int sh = S::LOGN - s;
    const int b = sh - 1 - lo;
    gconst_u64 *zs = zeta_inv + (1 << s) + (hb << (lo + S::LE - sh));
#pragma unroll
    for (int k = 0; k < S::E; ++k) {
      if (k & (1 << b)) continue;
      const int k2 = k | (1 << b);
      const u64 w = zs[k >> (sh - lo)];
      const u64 u = x[k], v = x[k2];
      x[k] = gl_add(u, v);
      x[k2] = gl_mul(gl_sub(u, v), w);
    }
  }
}

// Move from the layout of pass QW to that of pass QR through one LDS buffer.
template <class S, int QW, int QR>
__device__ __forceinline__ void ntt_exchange(u64 (&x)[S::E], u64 *lds, int tid) {
  u64 *w = lds + S::lds_base(QW, tid);
#pragma unroll
  for (int k = 0; k < S::E; ++k) w[S::lds_off(QW, k)] = x[k];
  __syncthreads();
  const u64 *r = lds + S::lds_base(QR, tid);
#pragma unroll
  for (int k = 0; k < S::E; ++k) x[k] = r[S::lds_off(QR, k)];
}

// Two LDS buffers of `words` words each, used alternately.
struct LdsPair {
  u64 *base;
  int words;
  int par;
  __device__ __forceinline__ LdsPair(u64 *b, int w) : base(b), words(w), par(0) {}
  __device__ __forceinline__ u64 *next() {
    u64 *p = base + par * words;
    par ^= 1;
    return p;
  }
};

template <class S, int Q>
__device__ __forceinline__ void ntt_fwd_from(u64 (&x)[S::E], LdsPair &lds, int tid,
                                             gconst_u64 *zeta) {
  ntt_fwd_pass<S, Q>(x, tid, zeta);
  if constexpr (Q + 1 < S::PASSES) {
    ntt_exchange<S, Q, Q + 1>(x, lds.next(), tid);
    ntt_fwd_from<S, Q + 1>(x, lds, tid, zeta);
  }
}

template <class S, int Q>
__device__ __forceinline__ void ntt_inv_from(u64 (&x)[S::E], LdsPair &lds, int tid,
                                             gconst_u64 *zeta_inv) {
  ntt_inv_pass<S, Q>(x, tid, zeta_inv);
  if constexpr (Q > 0) {
    ntt_exchange<S, Q, Q - 1>(x, lds.next(), tid);
    ntt_inv_from<S, Q - 1>(x, lds, tid, zeta_inv);
  }
}

// Natural layout in, in-place (bit-reversed evaluation) layout of the last
// pass out.
template <class S>
__device__ __forceinline__ void ntt_forward(u64 (&x)[S::E], LdsPair &lds, int tid,
                                            gconst_u64 *zeta) {
  ntt_fwd_from<S, 0>(x, lds, tid, zeta);
}

// Last-pass layout in, natural layout out, result scaled by N.
template <class S>
__device__ __forceinline__ void ntt_inverse(u64 (&x)[S::E], LdsPair &lds, int tid,
                                            gconst_u64 *zeta_inv) {
  ntt_inv_from<S, S::PASSES - 1>(x, lds, tid, zeta_inv);
}

// Global-address-space view of a device pointer.
__device__ __forceinline__ gconst_u64 *as_global(const u64 *p) { return (gconst_u64 *)p; }

}  // namespace rosetta
