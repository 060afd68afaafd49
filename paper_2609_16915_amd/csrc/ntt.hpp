// Negacyclic NTT of one polynomial per workgroup, held in registers.
//
// N = 2^LOGN coefficients are spread over T = N / E threads, E = 2^LE per
// thread.  The forward transform is the merged-twist Cooley-Tukey form: stage
// s (s = 0 .. LOGN-1) pairs indices j and j + N/2^(s+1) inside block
// b = j >> (LOGN - s) and multiplies the upper element by
// zeta[2^s + b] = psi^rev(2^s + b)  (psi a primitive 2N-th root of unity,
// rev the LOGN-bit reversal), so the result at in-place index j is
// a(psi^(2 rev(j) + 1)).  The inverse runs the Gentleman-Sande mirror and
// leaves the factor N for the caller.  It needs psi^-rev(m); within stage s
// that equals -zeta[3*2^s - 1 - m], so a single table serves both
// directions and the sign is absorbed by computing (v - u) * zeta instead of
// (u - v) * zeta^-1.
//
// Stages are grouped into passes: pass 0 takes the first F <= LE stages, every
// later pass the next LE (the last one what remains).  During pass q >= 1 a
// thread holds the E elements whose index bits [lo_q, lo_q + LE) vary, lo_q =
// max(0, LOGN - (end of the pass's stages)); the thread id fills the
// remaining bits in order:
//   j = (tid mod 2^lo) + (k << lo) + ((tid >> lo) << (lo + LE)).
// Pass 0 is the natural layout j = tid + T*k (lo_0 = LOGN - LE).
// Butterflies inside a pass are register-only; between passes the workgroup
// transposes through LDS: between waves a barrier, the writes, a barrier and
// the reads; within each wave (both layouts keep the wave's block) a
// wave-level fence between writes and reads (ntt_exchange).
//
// LDS word addresses of the transposes go through a linear XOR swizzle
// (bit b < 5 of the address is flipped by the parity of j & SWZ_MASK[b],
// masks holding only bits above b).  It was chosen so that in every pass
// layout of every supported (N, E) the 32 lanes of each half wave touch 32
// distinct banks of 8-byte words, and the 16 lanes of each quarter wave 16
// distinct ones.  Being linear over GF(2), the address of element k is the
// thread's swizzled base XOR a compile-time constant.  The twiddle table
// itself lives in LDS: the key streams through the vector memory path, so
// keeping twiddle reads off it keeps their latency off the in-order
// vector-memory counter.
#pragma once

#include <type_traits>

#include "gl.hpp"

namespace rosetta {

typedef const u64 __attribute__((address_space(1))) gconst_u64;

constexpr unsigned SWZ_MASK[5] = {0x7b0, 0x574, 0x538, 0xa60, 0x3e0};

__host__ __device__ constexpr int swz_masks(int j, const unsigned *m) {
  int a = j;
  for (int b = 0; b < 5; ++b) a ^= (__builtin_popcount((unsigned)j & m[b]) & 1) << b;
  return a;
}
__host__ __device__ constexpr int swz(int j) { return swz_masks(j, SWZ_MASK); }

template <int LOGN_, int LE_, int F_ = LE_>
struct Ntt {
  static_assert(F_ >= 1 && F_ <= LE_, "the first pass spans 1..LE stages");
  static constexpr int LOGN = LOGN_;
  static constexpr int LE = LE_;
  static constexpr int F = F_;  // stages of pass 0
  static constexpr int N = 1 << LOGN;
  static constexpr int E = 1 << LE;
  static constexpr int T = N / E;
  static constexpr int PASSES = 1 + (LOGN - F + LE - 1) / LE;

  __host__ __device__ static constexpr int stage_begin(int q) { return q == 0 ? 0 : F + (q - 1) * LE; }
  __host__ __device__ static constexpr int stage_end(int q) {
    return F + q * LE < LOGN ? F + q * LE : LOGN;
  }
  __host__ __device__ static constexpr int lo(int q) {
    return q == 0 ? LOGN - LE : (LOGN - stage_end(q) > 0 ? LOGN - stage_end(q) : 0);
  }
  // index held by element k of thread tid during pass q
  __host__ __device__ static constexpr int idx(int q, int tid, int k) {
    return (tid & ((1 << lo(q)) - 1)) + (k << lo(q)) + ((tid >> lo(q)) << (lo(q) + LE));
  }
  // Passes after the first that span three stages run in twisted radix-8
  // form and need, per block b of their first stage s0, the powers q^1..q^7
  // of q = zeta[4 (2^s0 + b)].  The table region [2^s0, 2^(s0+3)) holds the
  // twiddles of exactly those three stages and no other pass reads it, so
  // for such a pass it stores q^1..q^7 of block b at 2^s0 + 7 b instead:
  // 7 words per block fill it exactly, and the odd stride puts the blocks
  // of a half wave on distinct LDS banks.
  __host__ __device__ static constexpr bool twisted(int q) {
    return q >= 1 && LE == 3 && stage_end(q) - stage_begin(q) == 3;
  }
  // word address of index j in an exchange buffer
  __host__ __device__ static constexpr int swz(int j) { return swz_masks(j, SWZ_MASK); }
  // A twisted pass whose first stage is s0 <= 2 has q = zeta[4 (2^s0 + b)]
  // among the 64th roots of unity, which are powers of two; when, in
  // addition, lo >= 6, the block b = tid >> lo is the wave's index, so the
  // wave can branch (uniformly) to a copy of the pass in which the powers
  // q^k are compile-time shifts instead of products.
  __host__ __device__ static constexpr bool shift_twist(int q) {
    return twisted(q) && stage_begin(q) <= 2 && lo(q) >= 6;
  }
  // words of the LDS twiddle area (the table above, with the regions of the
  // twisted passes as described there and the stages of a last pass that is
  // not twisted stored slot-major, see ntt_fwd_pass; the shift-twisted
  // passes read none of it)
  static constexpr int TW_WORDS = N;
  // In pass q each wave (64 threads) holds one contiguous block of
  // 2^(6+LE) indices when lo(q) <= 6 (the wave id then sets the top index
  // bits), or the whole transform when the workgroup is one wave.  An
  // exchange between two such passes moves data only within each wave.
  __host__ __device__ static constexpr bool wave_block(int q) { return T <= 64 || lo(q) <= 6; }
  __host__ __device__ static constexpr bool local_exchange(int qa, int qb) {
    return wave_block(qa) && wave_block(qb);
  }
  // At N = 4096 the exchanges within a wave share the one cross-wave buffer
  // (SHARED): after a cross exchange into a layout that keeps each wave's
  // block, each wave reads only its own block, so writing that block again
  // needs no barrier; after one into a layout that spreads a wave over the
  // buffer (pass 0: the second inverse transform of a step starts right
  // after the first one's last exchange), and after the rotation and
  // automorphism reads, the next local exchange starts with a barrier
  // (LdsBufs::spread); every cross exchange starts with one.  That keeps the
  // LDS of a workgroup at 2N words plus the rotation amounts, so that two
  // 512-thread workgroups fit a CU.
  static constexpr bool SHARED = LOGN >= 12;
  // words after the twiddle area: the cross-wave buffer, then (unless
  // SHARED) one N-word buffer in which every wave exchanges within its own
  // block
  static constexpr int XCHG_WORDS = (SHARED ? 1 : 2) * N;
};

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// zeta[m] for m < 8 is a 16th root of unity, and with psi = 7^((p-1)/2N)
// it equals 2^((156 * rev3(m)) mod 192) for every N, 7^((p-1)/16) being
// 2^156.  Pass 0 (stages 0..F-1, F <= 4) uses only zeta[m] with m < 16
// (powers of two too, below), so its twiddle products are shifts
// (gl_mul_pow2) and need no table.
__host__ __device__ constexpr int rev3(int m) {
  return ((m & 1) << 2) | (m & 2) | ((m >> 2) & 1);
}
__host__ __device__ constexpr int zeta_log2(int m) { return (156 * rev3(m)) % 192; }

// zeta[m] for m < 32 is a 64th root of unity: with 7^((p-1)/64) = 2^39 it
// equals 2^(39 rev5(m) mod 192) for every N >= 32 (rev5 the 5-bit reversal;
// below 8 this is zeta_log2).
__host__ __device__ constexpr int rev5(int m) {
  return ((m & 1) << 4) | ((m & 2) << 2) | (m & 4) | ((m >> 2) & 2) | ((m >> 4) & 1);
}
__host__ __device__ constexpr int zeta_log2_64(int m) { return (39 * rev5(m)) % 192; }
__host__ __device__ constexpr bool zeta_logs_agree() {
  for (int m = 0; m < 8; ++m)
    if (zeta_log2_64(m) != zeta_log2(m)) return false;
  return true;
}
static_assert(zeta_logs_agree(), "the two closed forms of the small roots disagree");

// |zeta[M]| * x for M < 32 (64th roots, powers of two); zeta[M] is
// negative when its exponent is >= 96.
template <int M>
__device__ __forceinline__ u64 mul_small_root(u64 x) {
  static_assert(M < 32, "a power of two only below 32");
  constexpr int e = zeta_log2_64(M);
  return gl_mul_pow2<(e >= 96 ? e - 96 : e)>(x);
}
template <int M>
__host__ __device__ constexpr bool small_root_negative() {
  return zeta_log2_64(M) >= 96;
}



// x * (+-2^E) for a compile-time E mod 192 (2^96 = -1): the magnitude as a
// shift; the sign is the caller's (sign_pow2).
template <int E>
__device__ __forceinline__ u64 mul_pow2_mag(u64 x) {
  return gl_mul_pow2<(E % 192 >= 96 ? E % 192 - 96 : E % 192)>(x);
}
__host__ __device__ constexpr int sign_pow2(int e) { return e % 192 >= 96 ? -1 : 1; }


// Sums of the forward butterflies.  A weak forward transform (W) feeds only
// products (the key multiply-accumulate), so its values need only stay below
// 2^64 and congruent: a sum whose second operand is canonical (a product, a
// shift, or a value kept canonical for that purpose) takes gl_add_weak, and
// every difference has a canonical subtrahend, which gl_sub accepts with any
// minuend.  Products and shifts accept any input and return canonical values.
template <bool W>
__device__ __forceinline__ u64 fwd_sum(u64 a, u64 b) {
  if constexpr (W)
    return gl_add_weak(a, b);
  else
    return gl_add(a, b);
}

// Butterfly on signed operands A = SA a, B = SB b (signs known at compile
// time, a and b the stored values): a <- A + B, b <- A - B, both returned
// with the sign SA, which costs nothing: for SA != SB the sum and the
// difference of the stored values trade places.  The subtrahend is always
// b.  CF: the first result must be canonical (a and b canonical); a sum in
// any other place may be weak (W, see fwd_sum).
template <int SA, int SB, bool W, bool CF>
__device__ __forceinline__ void signed_bfly(u64 &a, u64 &b) {
  const u64 u = a, v = b;
  if constexpr (SA == SB) {
    a = CF ? gl_add(u, v) : fwd_sum<W>(u, v);
    b = gl_sub(u, v);
  } else {
    a = gl_sub(u, v);
    b = fwd_sum<W>(u, v);
  }
}

// Pass 0 of the forward transform (all twiddles compile-time powers of
// two), starting at stage FIRST.
template <class S, int FIRST, bool W = false>
__device__ __forceinline__ void ntt_fwd_pass0(u64 (&x)[S::E]) {
  constexpr int lo = S::lo(0);
  static_for<FIRST, S::stage_end(0)>([&](auto sc) {
    constexpr int s = decltype(sc)::value;
    constexpr int sh = S::LOGN - s;
    constexpr int b = sh - 1 - lo;
    static_for<0, S::E>([&](auto kc) {
      constexpr int k = decltype(kc)::value;
      if constexpr (!(k & (1 << b))) {
        constexpr int k2 = k | (1 << b);
        constexpr int m = (1 << s) + (k >> (sh - lo));
        const u64 t = mul_small_root<m>(x[k2]);
        const u64 u = x[k];
        if constexpr (small_root_negative<m>()) {  // w = -|w|
          x[k] = gl_sub(u, t);
          x[k2] = fwd_sum<W>(u, t);
        } else {
          x[k] = fwd_sum<W>(u, t);
          x[k2] = gl_sub(u, t);
        }
      }
    });
  });
}

// Pass 0 of the inverse transform: (u, v) -> (u + v, (v - u) zeta[2^(s+1)-1-b]).
template <class S>
__device__ __forceinline__ void ntt_inv_pass0(u64 (&x)[S::E]) {
  constexpr int lo = S::lo(0);
  static_for<0, S::stage_end(0)>([&](auto rc) {
    constexpr int s = S::stage_end(0) - 1 - decltype(rc)::value;
    constexpr int sh = S::LOGN - s;
    constexpr int b = sh - 1 - lo;
    static_for<0, S::E>([&](auto kc) {
      constexpr int k = decltype(kc)::value;
      if constexpr (!(k & (1 << b))) {
        constexpr int k2 = k | (1 << b);
        constexpr int m = (2 << s) - 1 - (k >> (sh - lo));
        const u64 u = x[k], v = x[k2];
        x[k] = gl_add(u, v);
        if constexpr (small_root_negative<m>())  // (v - u)(-|w|) = (u - v)|w|
          x[k2] = mul_small_root<m>(gl_sub(u, v));
        else
          x[k2] = mul_small_root<m>(gl_sub(v, u));
      }
    });
  });
}

// Stages 0 and 1 of the forward transform on small signed inputs
// (|d| <= 2^13), in exact integer arithmetic.  Their twiddles are 16th roots
// that are signed powers of two: zeta[1] = 2^48, zeta[2] = -2^24 and
// zeta[3] = -2^72.  After the two stages every element is a signed sum of
// four inputs, one at each weight 2^0, 2^24, 2^48, 2^72 (a pure sign and
// index bookkeeping, computed at compile time by first_terms), and with
// 2^72 = 2^40 - 2^8 (mod p) its value is
//   L + 2^32 H,  L = s0 a + s24 2^24 b - s72 2^8 d,  H = s48 2^16 c + s72 2^8 d,
// an exact integer of magnitude below 2^62; one sign fix makes it a field
// element.
struct FirstTerm {
  int idx, sgn;  // input index and sign of the term at one weight
};
struct FirstElem {
  FirstTerm w[4];  // weights 2^0, 2^24, 2^48, 2^72
};
template <int E>
struct FirstTerms {
  FirstElem el[E];
  bool complete;  // every element has exactly one term at each weight
};

template <class S>
constexpr FirstTerms<S::E> first_terms() {
  static_assert(S::stage_end(0) >= 2, "the first pass must span two stages");
  constexpr int E = S::E, lo = S::lo(0);
  // terms as (input, weight exponent in units of 24 bits, sign)
  int idx[E][4] = {}, ex[E][4] = {}, sg[E][4] = {}, n[E] = {};
  for (int k = 0; k < E; ++k) {
    idx[k][0] = k;
    ex[k][0] = 0;
    sg[k][0] = 1;
    n[k] = 1;
  }
  for (int s = 0; s < 2; ++s) {
    const int sh = S::LOGN - s, b = sh - 1 - lo;
    for (int k = 0; k < E; ++k) {
      if (k & (1 << b)) continue;
      const int k2 = k | (1 << b);
      const int m = (1 << s) + (k >> (sh - lo));
      const int em = zeta_log2(m) / 24;  // zeta[m] = 2^(24 em), em < 8
      const int nu = n[k], nv = n[k2];
      int ti[4], te[4], ts[4];
      for (int i = 0; i < nv; ++i) {  // t = zeta[m] x[k2]; 2^96 = -1
        int e = ex[k2][i] + em, g = sg[k2][i];
        if (e >= 8) e -= 8;
        if (e >= 4) {
          e -= 4;
          g = -g;
        }
        ti[i] = idx[k2][i];
        te[i] = e;
        ts[i] = g;
      }
      for (int i = 0; i < nv; ++i) {  // x[k2] = x[k] - t, x[k] = x[k] + t
        idx[k2][i] = idx[k][i];
        ex[k2][i] = ex[k][i];
        sg[k2][i] = sg[k][i];
      }
      for (int i = 0; i < nv; ++i) {
        idx[k][nu + i] = ti[i];
        ex[k][nu + i] = te[i];
        sg[k][nu + i] = ts[i];
        idx[k2][nu + i] = ti[i];
        ex[k2][nu + i] = te[i];
        sg[k2][nu + i] = -ts[i];
      }
      n[k] = n[k2] = nu + nv;
    }
  }
  FirstTerms<E> r{};
  r.complete = true;
  for (int k = 0; k < E; ++k) {
    int seen = 0;
    for (int i = 0; i < n[k]; ++i) {
      seen |= 1 << ex[k][i];
      r.el[k].w[ex[k][i]] = FirstTerm{idx[k][i], sg[k][i]};
    }
    r.complete = r.complete && n[k] == 4 && seen == 15;
  }
  return r;
}

template <class S, typename RT>
__device__ __forceinline__ void ntt_fwd_stages01_small(const RT (&d)[S::E], u64 (&x)[S::E]) {
  constexpr FirstTerms<S::E> T = first_terms<S>();
  static_assert(T.complete, "two stages must give one term per weight");
  static_for<0, S::E>([&](auto kc) {
    constexpr FirstElem f = T.el[decltype(kc)::value];
    const int32_t a = (int32_t)d[f.w[0].idx], b = (int32_t)d[f.w[1].idx];
    const int32_t c = (int32_t)d[f.w[2].idx], e = (int32_t)d[f.w[3].idx];
    const int32_t t = f.w[0].sgn * a - f.w[3].sgn * (e * 256);
#if defined(__HIP_DEVICE_COMPILE__)
    const int64_t L = isa::mad_i64(b, f.w[1].sgn * (1 << 24), (int64_t)t);
#else
    const int64_t L = (int64_t)b * (f.w[1].sgn * (1 << 24)) + t;
#endif
    const int32_t H = f.w[2].sgn * (c * 65536) + f.w[3].sgn * (e * 256);
    const uint64_t X = (uint64_t)L + ((uint64_t)(uint32_t)H << 32);
    // negative X: add p, i.e. subtract 2^32 - 1 modulo 2^64
    const uint32_t neg = (uint32_t)((int32_t)(X >> 32) >> 31);
    x[decltype(kc)::value] = X - (uint64_t)neg;
  });
}

// Twisted radix-8 form of a three-stage pass (Q >= 1).  The thread's eight
// elements are the coefficients x_k of one block polynomial sum x_k Z^k
// taken modulo Z^8 - zeta[m]^2 (m the block at the pass's first stage).  The
// three merged-twist stages evaluate it at q w^e, q = zeta[4m] (q^4 =
// zeta[m]) and w = psi^(N/4) a primitive 8th root, i.e. they equal
//   y_k = q^k x_k   followed by an 8-point transform of y
// whose twiddles are the 8th roots i = w^2 = 2^48, w = -2^24 and
// w^3 = -2^72: shifts, not multiplications.  7 products + 5 shifts replace
// 12 products.  The inverse undoes it: psi^-rev(4m) = w^-1 zeta[4 m_r] with
// m_r = 3*2^s - 1 - m (the block reflected within its stage), and the
// factor w^-k is absorbed by feeding the inverse 8-point transform its
// inputs rotated by one frequency (slots 7,6,4,5,0,1,2,3), after which the
// untwist multiplies by powers of zeta[4 m_r].
//
// Weak form (W, see fwd_sum): only x[0] may arrive non-canonical; the sums
// that later serve as the second operand of a twiddle-1 butterfly (x[1],
// x[2], x[3] after the first stage, x[1] after the second) stay canonical.
template <class S, int Q, bool W = false>
__device__ __forceinline__ void ntt_fwd_pass_twisted(u64 (&x)[S::E], int tid, const u64 *tw) {
  constexpr int lo = S::lo(Q), s0 = S::stage_begin(Q);
  const int b = tid >> lo;  // block at stage s0
  const u64 *qp = tw + (1 << s0) + 7 * b;  // q^1 .. q^7
#pragma unroll
  for (int k = 1; k < 8; ++k) x[k] = gl_mul(x[k], qp[k - 1]);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const u64 u = x[k], v = x[k + 4];
    x[k] = k == 0 ? fwd_sum<W>(u, v) : gl_add(u, v);
    x[k + 4] = gl_sub(u, v);
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    u64 u = x[k], v = x[k + 2];
    x[k] = k == 0 ? fwd_sum<W>(u, v) : gl_add(u, v);
    x[k + 2] = gl_sub(u, v);
    u = x[k + 4];
    v = gl_mul_pow2<48>(x[k + 6]);  // i
    x[k + 4] = fwd_sum<W>(u, v);
    x[k + 6] = gl_sub(u, v);
  }
  {
    u64 u = x[0], v = x[1];
    x[0] = fwd_sum<W>(u, v);
    x[1] = gl_sub(u, v);
    u = x[2];
    v = gl_mul_pow2<48>(x[3]);  // i
    x[2] = fwd_sum<W>(u, v);
    x[3] = gl_sub(u, v);
    u = x[4];
    v = gl_mul_pow2<24>(x[5]);  // w = -2^24
    x[4] = gl_sub(u, v);
    x[5] = fwd_sum<W>(u, v);
    u = x[6];
    v = gl_mul_pow2<72>(x[7]);  // w^3 = -2^72
    x[6] = gl_sub(u, v);
    x[7] = fwd_sum<W>(u, v);
  }
}

// The 8-point inverse transform of a twisted inverse pass, on the inputs
// rotated by one frequency (see ntt_fwd_pass_twisted), into z.
__device__ __forceinline__ void ntt_inv_dft8(const u64 (&x)[8], u64 (&z)[8]) {
  z[0] = x[7];
  z[1] = x[6];
  z[2] = x[4];
  z[3] = x[5];
  z[4] = x[0];
  z[5] = x[1];
  z[6] = x[2];
  z[7] = x[3];
  {
    u64 u = z[0], v = z[1];
    z[0] = gl_add(u, v);
    z[1] = gl_sub(u, v);
    u = z[2];
    v = z[3];
    z[2] = gl_add(u, v);
    z[3] = gl_mul_pow2<48>(gl_sub(v, u));  // i^-1 = -2^48
    u = z[4];
    v = z[5];
    z[4] = gl_add(u, v);
    z[5] = gl_mul_pow2<72>(gl_sub(u, v));  // w^-1 = 2^72
    u = z[6];
    v = z[7];
    z[6] = gl_add(u, v);
    z[7] = gl_mul_pow2<24>(gl_sub(u, v));  // w^-3 = 2^24
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    u64 u = z[k], v = z[k + 2];
    z[k] = gl_add(u, v);
    z[k + 2] = gl_sub(u, v);
    u = z[k + 4];
    v = z[k + 6];
    z[k + 4] = gl_add(u, v);
    z[k + 6] = gl_mul_pow2<48>(gl_sub(v, u));  // i^-1
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const u64 u = z[k], v = z[k + 4];
    z[k] = gl_add(u, v);
    z[k + 4] = gl_sub(u, v);
  }
}

template <class S, int Q>
__device__ __forceinline__ void ntt_inv_pass_twisted(u64 (&x)[S::E], int tid, const u64 *tw) {
  constexpr int lo = S::lo(Q), s0 = S::stage_begin(Q);
  const int br = (1 << s0) - 1 - (tid >> lo);  // reflected block
  const u64 *qp = tw + (1 << s0) + 7 * br;  // powers of q_r = zeta[4 (2^s0 + br)]
  u64 z[8];
  ntt_inv_dft8(x, z);
  x[0] = z[0];
#pragma unroll
  for (int k = 1; k < 8; ++k) x[k] = gl_mul(z[k], qp[k - 1]);
}

// Twisted pass Q for the block B at its first stage when q = zeta[4 (2^s0 +
// B)] is a power of two (Ntt::shift_twist): the twist y_k = q^k x_k is a
// shift by |q^k|, and the signs of the q^k ride through the 8-point
// transform in signed_bfly, so that every output leaves with the sign of
// y_0 = x_0, positive, at no cost.  Weak and canonical sums sit where
// ntt_fwd_pass_twisted has them (CF marks the canonical ones).
template <class S, int Q, bool W, int B>
__device__ __forceinline__ void ntt_fwd_pass_shift_twist(u64 (&x)[S::E]) {
  constexpr int eq = zeta_log2_64(4 * ((1 << S::stage_begin(Q)) + B));
  constexpr int s1 = sign_pow2(eq), s2 = sign_pow2(2 * eq), s3 = sign_pow2(3 * eq),
                s4 = sign_pow2(4 * eq), s5 = sign_pow2(5 * eq), s6 = sign_pow2(6 * eq),
                s7 = sign_pow2(7 * eq);
  x[1] = mul_pow2_mag<eq>(x[1]);
  x[2] = mul_pow2_mag<2 * eq>(x[2]);
  x[3] = mul_pow2_mag<3 * eq>(x[3]);
  x[4] = mul_pow2_mag<4 * eq>(x[4]);
  x[5] = mul_pow2_mag<5 * eq>(x[5]);
  x[6] = mul_pow2_mag<6 * eq>(x[6]);
  x[7] = mul_pow2_mag<7 * eq>(x[7]);
  // stage A; afterwards x[j] and x[j + 4] carry the sign of y_j
  signed_bfly<1, s4, W, false>(x[0], x[4]);
  signed_bfly<s1, s5, W, true>(x[1], x[5]);
  signed_bfly<s2, s6, W, true>(x[2], x[6]);
  signed_bfly<s3, s7, W, true>(x[3], x[7]);
  // stage B (i = 2^48); afterwards x[0], x[2], x[4], x[6] are positive and
  // x[1], x[3], x[5], x[7] carry s1
  signed_bfly<1, s2, W, false>(x[0], x[2]);
  signed_bfly<s1, s3, W, true>(x[1], x[3]);
  x[6] = gl_mul_pow2<48>(x[6]);
  signed_bfly<1, s2, W, false>(x[4], x[6]);
  x[7] = gl_mul_pow2<48>(x[7]);
  signed_bfly<s1, s3, W, false>(x[5], x[7]);
  // stage C (i, w = -2^24, w^3 = -2^72)
  signed_bfly<1, s1, W, false>(x[0], x[1]);
  x[3] = gl_mul_pow2<48>(x[3]);
  signed_bfly<1, s1, W, false>(x[2], x[3]);
  x[5] = gl_mul_pow2<24>(x[5]);
  signed_bfly<1, -s1, W, false>(x[4], x[5]);
  x[7] = gl_mul_pow2<72>(x[7]);
  signed_bfly<1, -s1, W, false>(x[6], x[7]);
}

// The inverse of ntt_fwd_pass_shift_twist for block B: the 8-point inverse
// of ntt_inv_pass_twisted, then the untwist by the powers of q_r =
// zeta[4 (2^s0 + 2^s0 - 1 - B)] as shifts, negated (gl_neg) where q_r^k is.
template <class S, int Q, int B>
__device__ __forceinline__ void ntt_inv_pass_shift_twist(u64 (&x)[S::E]) {
  constexpr int s0 = S::stage_begin(Q);
  constexpr int er = zeta_log2_64(4 * ((1 << s0) + (1 << s0) - 1 - B));
  u64 z[8];
  ntt_inv_dft8(x, z);
  x[0] = z[0];
  static_for<1, 8>([&](auto kc) {
    constexpr int k = decltype(kc)::value;
    const u64 r = mul_pow2_mag<k * er>(z[k]);
    x[k] = sign_pow2(k * er) < 0 ? gl_neg(r) : r;
  });
}

// Dispatch of a shift-twisted pass to the copy of the wave's block b
// (wave-uniform, so the branches are scalar).
template <class S, int Q, bool W, int B = 0>
__device__ __forceinline__ void ntt_fwd_shift_twist_block(u64 (&x)[S::E], int b) {
  if constexpr (B + 1 < (1 << S::stage_begin(Q))) {
    if (b == B)
      ntt_fwd_pass_shift_twist<S, Q, W, B>(x);
    else
      ntt_fwd_shift_twist_block<S, Q, W, B + 1>(x, b);
  } else {
    ntt_fwd_pass_shift_twist<S, Q, W, B>(x);
  }
}
template <class S, int Q, int B = 0>
__device__ __forceinline__ void ntt_inv_shift_twist_block(u64 (&x)[S::E], int b) {
  if constexpr (B + 1 < (1 << S::stage_begin(Q))) {
    if (b == B)
      ntt_inv_pass_shift_twist<S, Q, B>(x);
    else
      ntt_inv_shift_twist_block<S, Q, B + 1>(x, b);
  } else {
    ntt_inv_pass_shift_twist<S, Q, B>(x);
  }
}

// Forward stages of pass Q; `tw` is the LDS twiddle table.  In the last
// pass (lo = 0) thread t holds indices E t .. E t + E - 1, so at stage s it
// needs the nc = E / 2^(LOGN - s) consecutive blocks t nc .. t nc + nc - 1;
// that stage's table region is stored slot-major there (block t nc + c at
// 2^s + c T + t), so that a wave's reads of one slot are consecutive words.
template <class S, int Q, bool W = false>
__device__ __forceinline__ void ntt_fwd_pass(u64 (&x)[S::E], int tid, const u64 *tw) {
  constexpr int lo = S::lo(Q);
  const int jt = S::idx(Q, tid, 0);
#pragma unroll
  for (int s = S::stage_begin(Q); s < S::stage_end(Q); ++s) {
    const int sh = S::LOGN - s;
    const int b = sh - 1 - lo;  // k-bit split by this stage
    const u64 *zs = lo == 0 ? tw + (1 << s) + tid : tw + (1 << s) + (jt >> sh);
#pragma unroll
    for (int k = 0; k < S::E; ++k) {
      if (k & (1 << b)) continue;
      const int k2 = k | (1 << b);
      const u64 w = lo == 0 ? zs[(k >> sh) * S::T] : zs[k >> (sh - lo)];
      const u64 t = gl_mul(x[k2], w);
      x[k2] = gl_sub(x[k], t);
      x[k] = fwd_sum<W>(x[k], t);
    }
  }
}

// Inverse (Gentleman-Sande) stages of pass Q, in reverse stage order:
// (u, v) -> (u + v, (v - u) * zeta[2^(s+1) - 1 - b]).  In the last pass the
// reflected block 2^s - 1 - (t nc + c) = (T - 1 - t) nc + (nc - 1 - c) is
// read from the slot-major layout of ntt_fwd_pass.
template <class S, int Q>
__device__ __forceinline__ void ntt_inv_pass(u64 (&x)[S::E], int tid, const u64 *tw) {
  constexpr int lo = S::lo(Q);
  const int jt = S::idx(Q, tid, 0);
#pragma unroll
  for (int s = S::stage_end(Q) - 1; s >= S::stage_begin(Q); --s) {
    const int sh = S::LOGN - s;
    const int b = sh - 1 - lo;
    const int nc = S::E >> sh;
    const u64 *zs = lo == 0 ? tw + (1 << s) + (S::T - 1 - tid) : tw + (2 << s) - 1 - (jt >> sh);
#pragma unroll
    for (int k = 0; k < S::E; ++k) {
      if (k & (1 << b)) continue;
      const int k2 = k | (1 << b);
      const u64 w = lo == 0 ? zs[(nc - 1 - (k >> sh)) * S::T] : zs[-(k >> (sh - lo))];
      const u64 u = x[k], v = x[k2];
      x[k] = gl_add(u, v);
      x[k2] = gl_mul(gl_sub(v, u), w);
    }
  }
}

// Order this wave's LDS accesses (compiler and hardware) without waiting
// for the other waves of the workgroup.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// LDS exchange buffers after the twiddle area (layout in Ntt::XCHG_WORDS).
// cross(): a buffer for an exchange between waves, free of the previous
// contents every wave may still read (alternation with one buffer in
// between, or a barrier).  local(): the buffer of exchanges inside each
// wave's own block; no other wave touches that block of it.  When the two
// are one buffer (SHARED), `spread` records that some wave may still be
// reading outside its own block (any use of cross() except an exchange
// whose reading layout keeps each wave's block): the next local() then
// starts with a barrier.  In the unrolled transforms the flag is known at
// compile time; across the non-unrolled loops it is uniform.
template <class S>
struct LdsBufs {
  u64 *base;
  bool spread;
  __device__ __forceinline__ explicit LdsBufs(u64 *b) : base(b), spread(false) {}
  __device__ __forceinline__ u64 *cross() {
    spread = true;
    __syncthreads();
    return base;
  }
  __device__ __forceinline__ u64 *local() {
    if constexpr (S::SHARED) {
      if (spread) {
        __syncthreads();
        spread = false;
      }
    }
    return S::SHARED ? base : base + S::N;
  }
};

// Move from the layout of pass QW to that of pass QR through an LDS buffer
// (swizzled word addresses); within each wave when both layouts keep the
// wave's block, else through a cross-wave buffer and a barrier.
template <class S, int QW, int QR>
__device__ __forceinline__ void ntt_exchange(u64 (&x)[S::E], LdsBufs<S> &lds, int tid) {
  const int wb = S::swz(S::idx(QW, tid, 0));
  const int rb = S::swz(S::idx(QR, tid, 0));
  if constexpr (S::local_exchange(QW, QR)) {
    u64 *buf = lds.local();
    wave_sync();
#pragma unroll
    for (int k = 0; k < S::E; ++k) buf[wb ^ S::swz(k << S::lo(QW))] = x[k];
    wave_sync();
#pragma unroll
    for (int k = 0; k < S::E; ++k) x[k] = buf[rb ^ S::swz(k << S::lo(QR))];
  } else {
    u64 *buf = lds.cross();
#pragma unroll
    for (int k = 0; k < S::E; ++k) buf[wb ^ S::swz(k << S::lo(QW))] = x[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < S::E; ++k) x[k] = buf[rb ^ S::swz(k << S::lo(QR))];
    // each wave read its own block only: a local exchange may follow
    // without a barrier
    if constexpr (S::wave_block(QR)) lds.spread = false;
  }
}

template <class S, int Q, bool W = false>
__device__ __forceinline__ void ntt_fwd_from(u64 (&x)[S::E], LdsBufs<S> &lds, int tid,
                                             const u64 *tw) {
  if constexpr (Q == 0)
    ntt_fwd_pass0<S, 0, W>(x);
  else if constexpr (S::shift_twist(Q))
    ntt_fwd_shift_twist_block<S, Q, W>(x, __builtin_amdgcn_readfirstlane(tid >> S::lo(Q)));
  else if constexpr (S::twisted(Q))
    ntt_fwd_pass_twisted<S, Q, W>(x, tid, tw);
  else
    ntt_fwd_pass<S, Q, W>(x, tid, tw);
  if constexpr (Q + 1 < S::PASSES) {
    ntt_exchange<S, Q, Q + 1>(x, lds, tid);
    ntt_fwd_from<S, Q + 1, W>(x, lds, tid, tw);
  }
}

template <class S, int Q>
__device__ __forceinline__ void ntt_inv_from(u64 (&x)[S::E], LdsBufs<S> &lds, int tid,
                                             const u64 *tw) {
  if constexpr (Q == 0)
    ntt_inv_pass0<S>(x);
  else if constexpr (S::shift_twist(Q))
    ntt_inv_shift_twist_block<S, Q>(x, __builtin_amdgcn_readfirstlane(tid >> S::lo(Q)));
  else if constexpr (S::twisted(Q))
    ntt_inv_pass_twisted<S, Q>(x, tid, tw);
  else
    ntt_inv_pass<S, Q>(x, tid, tw);
  if constexpr (Q > 0) {
    ntt_exchange<S, Q, Q - 1>(x, lds, tid);
    ntt_inv_from<S, Q - 1>(x, lds, tid, tw);
  }
}

// Natural layout in, in-place (bit-reversed evaluation) layout of the last
// pass out.
template <class S>
__device__ __forceinline__ void ntt_forward(u64 (&x)[S::E], LdsBufs<S> &lds, int tid,
                                            const u64 *tw) {
  ntt_fwd_from<S, 0>(x, lds, tid, tw);
}

// Forward transform of a polynomial with small signed coefficients d
// (|d| <= 2^13): stages 0 and 1 in integer arithmetic, then as ntt_forward
// in the weak form (fwd_sum): each output is below 2^64 and congruent to
// the transform, for callers that only multiply it (gl_mul_add).
template <class S, typename RT>
__device__ __forceinline__ void ntt_forward_small(const RT (&d)[S::E], u64 (&x)[S::E],
                                                  LdsBufs<S> &lds, int tid, const u64 *tw) {
  ntt_fwd_stages01_small<S, RT>(d, x);
  ntt_fwd_pass0<S, 2, true>(x);
  if constexpr (S::PASSES > 1) {
    ntt_exchange<S, 0, 1>(x, lds, tid);
    ntt_fwd_from<S, 1, true>(x, lds, tid, tw);
  }
}

// Last-pass layout in, natural layout out, result scaled by N.
template <class S>
__device__ __forceinline__ void ntt_inverse(u64 (&x)[S::E], LdsBufs<S> &lds, int tid,
                                            const u64 *tw) {
  ntt_inv_from<S, S::PASSES - 1>(x, lds, tid, tw);
}

// Copy the twiddle area (TW_WORDS words: zeta with the twisted passes'
// regions holding their block powers)
// into LDS (all threads of the workgroup).
template <class S>
__device__ __forceinline__ void load_twiddles(u64 *tw_lds, const u64 *__restrict__ zeta,
                                              int tid) {
  for (int i = tid; i < S::TW_WORDS; i += S::T) tw_lds[i] = zeta[i];
}

// Global-address-space view of a device pointer.
__device__ __forceinline__ gconst_u64 *as_global(const u64 *p) { return (gconst_u64 *)p; }

}  // namespace rosetta
