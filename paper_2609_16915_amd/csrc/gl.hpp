// Goldilocks field arithmetic, p = 2^64 - 2^32 + 1, for gfx950 VALU and host.
//
// 2^64 = 2^32 - 1 (mod p), so a 128-bit value hi*2^64 + lo with
// hi = h1*2^32 + h0 reduces to lo - h1 + h0*(2^32 - 1)  (since 2^96 = -1).
// Functions take and return canonical values in [0, p) unless stated: the
// products and power-of-two products accept any 64-bit input, and the
// "weak" forms (gl_add_weak, gl_mul_add_weak) return a value below 2^64
// that is only congruent, for chains that end in a product or in gl_canon.
// The 64x64 product is built from four 32x32+64-bit multiply-adds.  On the
// device the products, the multiply-accumulate, the power-of-two products
// and the subtraction use the carry-out of v_mad_u64_u32 and explicit
// carry chains (see the gfx950 section below); the host compiles the
// portable forms.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace rosetta {

typedef uint64_t u64;
typedef uint32_t u32;
typedef int64_t i64;

constexpr u64 GL_P = 0xFFFFFFFF00000001ull;
constexpr u64 GL_EPS = 0xFFFFFFFFull;  // 2^64 mod p

__host__ __device__ __forceinline__ u64 gl_mk(u32 lo, u32 hi) { return ((u64)hi << 32) | lo; }

// All arithmetic below is written on 32-bit limbs with explicit carry
// chains (v_add_co / v_addc / v_sub_co / v_subb on CDNA) and branch-free
// selects.  Two facts keep the corrections cheap:
//   s - p == s + EPS (mod 2^64), so "wrapped past 2^64" and "s >= p" are
//   both fixed by adding EPS;  and  d + p == d - EPS (mod 2^64).

// (a + b) mod p for canonical a, b: s = a + b wraps past 2^64 or reaches p
// exactly when the result is s + EPS (mod 2^64); the condition selects the
// 32-bit addend, one 64-bit add applies it.
__host__ __device__ __forceinline__ u64 gl_add(u64 a, u64 b) {
  u32 c1;
  const u32 s0 = __builtin_addc((u32)a, (u32)b, 0u, &c1);
  const u32 s1 = __builtin_addc((u32)(a >> 32), (u32)(b >> 32), c1, &c1);
  const u64 s = gl_mk(s0, s1);
  const u32 adj = (c1 | (s >= GL_P)) ? 0xFFFFFFFFu : 0u;
  return s + adj;
}

// (a - b) mod p for canonical a, b: on a borrow add p, i.e. subtract EPS
// mod 2^64, spelled as +borrow on the low word and -borrow on the high word
// with the low word's carry.  (The device uses gl_sub_dev.)  Any a < 2^64
// with canonical b also works: a borrow means a < b < p, and without one
// a - b is below 2^64 and congruent (canonical when a is).
__host__ __device__ __forceinline__ u64 gl_sub_portable(u64 a, u64 b) {
  u32 b1, k;
  const u32 d0 = __builtin_subc((u32)a, (u32)b, 0u, &b1);
  const u32 d1 = __builtin_subc((u32)(a >> 32), (u32)(b >> 32), b1, &b1);
  const u32 r0 = __builtin_addc(d0, 0u, b1, &k);
  u32 kk;
  const u32 r1 = __builtin_subc(__builtin_addc(d1, 0u, k, &kk), 0u, b1, &kk);
  return gl_mk(r0, r1);
}

__host__ __device__ __forceinline__ u64 gl_neg(u64 a) { return a ? GL_P - a : 0; }

// 128-bit product a*b as 32-bit limbs c0..c3 (c0 least significant), from
// four 32x32+64-bit multiply-adds (v_mad_u64_u32, which gfx950 issues at
// full rate): with p00 = a0 b0, p01 = a0 b1 + hi(p00), p10 = a1 b0 + lo(p01)
// and p11 = a1 b1 + hi(p01) + hi(p10), a b = lo(p00) + 2^32 lo(p10) +
// 2^64 p11, and no partial sum exceeds (2^32-1)^2 + 2 (2^32-1) = 2^64 - 1.
__host__ __device__ __forceinline__ void gl_mul_limbs(u64 a, u64 b, u32 &c0, u32 &c1, u32 &c2,
                                                      u32 &c3) {
  const u32 a0 = (u32)a, a1 = (u32)(a >> 32), b0 = (u32)b, b1 = (u32)(b >> 32);
  const u64 p00 = (u64)a0 * b0;
  const u64 p01 = (u64)a0 * b1 + (p00 >> 32);
  const u64 p10 = (u64)a1 * b0 + (u32)p01;
  const u64 p11 = (u64)a1 * b1 + ((p01 >> 32) + (p10 >> 32));
  c0 = (u32)p00;
  c1 = (u32)p10;
  c2 = (u32)p11;
  c3 = (u32)(p11 >> 32);
}

// c0 + c1 2^32 + c2 2^64 + c3 2^96  mod p
//   = (c1:c0) - c3 + c2 (2^32 - 1)          (2^64 = 2^32 - 1, 2^96 = -1)
// t = (c1:c0) - c3 (+ p on a borrow, as in gl_sub) is below 2^64, v = c2 EPS
// is below 2^64 - 2^33 + 2, so t + v wraps past 2^64 at most once and the
// wrapped sum plus EPS stays below p; as in gl_add, one conditional EPS
// then canonicalises.
__host__ __device__ __forceinline__ u64 gl_reduce_limbs(u32 c0, u32 c1, u32 c2, u32 c3) {
  u32 e1, k, kk;
  const u32 d0 = __builtin_subc(c0, c3, 0u, &e1);
  const u32 d1 = __builtin_subc(c1, 0u, e1, &e1);
  const u32 t0 = __builtin_addc(d0, 0u, e1, &k);
  const u32 t1 = __builtin_subc(__builtin_addc(d1, 0u, k, &kk), 0u, e1, &kk);
  u32 bb;
  const u32 v0 = __builtin_subc(0u, c2, 0u, &bb);  // v = c2 EPS = (c2 << 32) - c2
  const u32 v1 = c2 - bb;
  u32 ca;
  const u32 r0 = __builtin_addc(t0, v0, 0u, &ca);
  const u32 r1 = __builtin_addc(t1, v1, ca, &ca);
  const u64 r = gl_mk(r0, r1);
  const u32 adj = (ca | (r >= GL_P)) ? 0xFFFFFFFFu : 0u;
  return r + adj;
}

// (hi*2^64 + lo) mod p for any 128-bit value.
__host__ __device__ __forceinline__ u64 gl_reduce128(u64 lo, u64 hi) {
  return gl_reduce_limbs((u32)lo, (u32)(lo >> 32), (u32)hi, (u32)(hi >> 32));
}

#if defined(__HIP_DEVICE_COMPILE__)
// ---- gfx950 device forms ---------------------------------------------------
// The compiler does not expose the carry-out of v_mad_u64_u32 (a wave64 lane
// mask in an SGPR pair), and without it a 64-bit addend must be
// zero-extended into an aligned register pair (moves) and an overflow
// recovered by a compare.  The wrappers below are single instructions; the
// mask logic between them compiles to scalar instructions.
namespace isa {

// a * b + c and its carry-out (bit 64 per lane)
__device__ __forceinline__ u64 mad_c(u32 a, u32 b, u64 c, u64 &cy) {
  u64 r;
  asm("v_mad_u64_u32 %0, %1, %2, %3, %4" : "=v"(r), "=s"(cy) : "v"(a), "v"(b), "v"(c));
  return r;
}
// a * b + c with signed 32-bit a, b and signed 64-bit c (exact when the
// result fits in 64 bits)
__device__ __forceinline__ int64_t mad_i64(int32_t a, int32_t b, int64_t c) {
  int64_t r;
  u64 cy;
  asm("v_mad_i64_i32 %0, %1, %2, %3, %4" : "=v"(r), "=s"(cy) : "v"(a), "s"(b), "v"(c));
  return r;
}
// a * (2^32 - 1) + c and its carry-out
__device__ __forceinline__ u64 mad_eps_c(u32 a, u64 c, u64 &cy) {
  u64 r;
  asm("v_mad_u64_u32 %0, %1, %2, -1, %3" : "=v"(r), "=s"(cy) : "v"(a), "v"(c));
  return r;
}
// a + b + carry-in, with carry-out
__device__ __forceinline__ u32 addc_c(u32 a, u32 b, u64 ci, u64 &co) {
  u32 r;
  asm("v_addc_co_u32_e64 %0, %1, %2, %3, %4" : "=v"(r), "=s"(co) : "v"(a), "v"(b), "s"(ci));
  return r;
}
// a + b with carry-out
__device__ __forceinline__ u32 add_c(u32 a, u32 b, u64 &co) {
  u32 r;
  asm("v_add_co_u32_e64 %0, %1, %2, %3" : "=v"(r), "=s"(co) : "v"(a), "v"(b));
  return r;
}
// a + carry-in, carry-out discarded
__device__ __forceinline__ u32 inc_ci(u32 a, u64 ci) {
  u32 r;
  u64 co;
  asm("v_addc_co_u32_e64 %0, %1, %2, 0, %3" : "=v"(r), "=s"(co) : "v"(a), "s"(ci));
  return r;
}
// a - b with borrow-out
__device__ __forceinline__ u32 sub_c(u32 a, u32 b, u64 &bo) {
  u32 r;
  asm("v_sub_co_u32_e64 %0, %1, %2, %3" : "=v"(r), "=s"(bo) : "v"(a), "v"(b));
  return r;
}
// a - borrow-in with borrow-out
__device__ __forceinline__ u32 dec_bc(u32 a, u64 bi, u64 &bo) {
  u32 r;
  asm("v_subb_co_u32_e64 %0, %1, %2, 0, %3" : "=v"(r), "=s"(bo) : "v"(a), "s"(bi));
  return r;
}
// lanes with r >= p
__device__ __forceinline__ u64 ge_p(u64 r) {
  u64 m;
  asm("v_cmp_lt_u64_e64 %0, %1, %2" : "=s"(m) : "s"(GL_P - 1), "v"(r));
  return m;
}
// m ? 2^32 - 1 : 0
__device__ __forceinline__ u32 sel_eps(u64 m) {
  u32 e;
  asm("v_cndmask_b32_e64 %0, 0, -1, %1" : "=v"(e) : "s"(m));
  return e;
}
// r + (m ? 2^32 - 1 : 0), i.e. r - p (mod 2^64) on the lanes of m
__device__ __forceinline__ u64 add_eps_if(u64 r, u64 m) { return r + (u64)sel_eps(m); }
// a - b - borrow-in, with borrow-out
__device__ __forceinline__ u32 subb_c(u32 a, u32 b, u64 bi, u64 &bo) {
  u32 r;
  asm("v_subb_co_u32_e64 %0, %1, %2, %3, %4" : "=v"(r), "=s"(bo) : "v"(a), "v"(b), "s"(bi));
  return r;
}
// a + carry-in, with carry-out
__device__ __forceinline__ u32 inc_c(u32 a, u64 ci, u64 &co) {
  u32 r;
  asm("v_addc_co_u32_e64 %0, %1, %2, 0, %3" : "=v"(r), "=s"(co) : "v"(a), "s"(ci));
  return r;
}
// a - borrow-in, borrow-out discarded
__device__ __forceinline__ u32 dec_bi(u32 a, u64 bi) {
  u32 r;
  u64 bo;
  asm("v_subb_co_u32_e64 %0, %1, %2, 0, %3" : "=v"(r), "=s"(bo) : "v"(a), "s"(bi));
  return r;
}
// d - (2^32 - 1), i.e. d + p (mod 2^64), on the lanes of m, in two carry
// instructions: the low word rises by one (carrying out where it was
// 2^32 - 1) and the high word drops by one except where the low word
// carried; the scalar unit forms that lane mask.
__device__ __forceinline__ u64 sub_eps_if(u64 d, u64 m) {
  u64 k;
  const u32 lo = inc_c((u32)d, m, k);
  const u32 hi = dec_bi((u32)(d >> 32), m & ~k);
  return gl_mk(lo, hi);
}

}  // namespace isa

// (c1:c0) + c2 (2^32 - 1) - c3 mod p, canonical.  t = (c1:c0) - c3, minus
// EPS (plus p mod 2^64) on a borrow, which leaves t in [p - 2^32, p); then
// R = c2 EPS + t with its carry: a carry leaves R + EPS below p (R is below
// 2^64 - 2^33 + 1 after the wrap), no carry leaves R in [0, 2^64), so one
// conditional EPS covers "carry or R >= p".  (The borrow correction keeps
// the select form: sub_eps_if is one instruction shorter but puts a scalar
// step on the product's dependent chain, which cost more than it saved.)
// With CANON false only the carry is corrected: the result is below 2^64
// and congruent, not necessarily below p.
template <bool CANON = true>
__device__ __forceinline__ u64 gl_reduce_dev(u32 c0, u32 c1, u32 c2, u32 c3) {
  u64 b0, b1, b2, b3;
  const u32 d0 = isa::sub_c(c0, c3, b0);
  const u32 d1 = isa::dec_bc(c1, b0, b1);
  const u32 e = isa::sel_eps(b1);
  const u32 t0 = isa::sub_c(d0, e, b2);
  const u32 t1 = isa::dec_bc(d1, b2, b3);
  u64 ca;
  const u64 R = isa::mad_eps_c(c2, gl_mk(t0, t1), ca);
  if constexpr (CANON)
    return isa::add_eps_if(R, ca | isa::ge_p(R));
  else
    return isa::add_eps_if(R, ca);
}

// a b as limbs: M = a1 b0, S = a0 b1 + M (65 bits: carry cs),
// P0 = a0 b0, P1 = a1 b1;  a b = P0 + 2^32 S + 2^64 P1, so
// c1 = hi(P0) + lo(S), c2 = lo(P1) + hi(S) + carry, c3 = hi(P1) + carries.
// c3 never overflows (a b < 2^128).
__device__ __forceinline__ u64 gl_mul_dev(u64 a, u64 b) {
  const u32 a0 = (u32)a, a1 = (u32)(a >> 32), b0 = (u32)b, b1 = (u32)(b >> 32);
  u64 cs;
  const u64 S = isa::mad_c(a0, b1, (u64)a1 * b0, cs);
  const u64 P0 = (u64)a0 * b0;
  const u64 P1 = (u64)a1 * b1;
  u64 kc, kd;
  const u32 c1 = isa::add_c((u32)(P0 >> 32), (u32)S, kc);
  const u32 c2 = isa::addc_c((u32)P1, (u32)(S >> 32), kc, kd);
  const u32 c3 = isa::inc_ci(isa::inc_ci((u32)(P1 >> 32), kd), cs);
  return gl_reduce_dev((u32)P0, c1, c2, c3);
}

// a b + c: c enters the multiply-add of P0 (carry cc at weight 2^64, added
// to c2 with its own carry into c3).  Any a, c < 2^64 with canonical b keep
// a b + c below 2^128; CANON false leaves the result weak (gl_reduce_dev).
template <bool CANON = true>
__device__ __forceinline__ u64 gl_mul_add_dev(u64 a, u64 b, u64 c) {
  const u32 a0 = (u32)a, a1 = (u32)(a >> 32), b0 = (u32)b, b1 = (u32)(b >> 32);
  u64 cs, cc;
  const u64 S = isa::mad_c(a0, b1, (u64)a1 * b0, cs);
  const u64 P0 = isa::mad_c(a0, b0, c, cc);
  const u64 P1 = (u64)a1 * b1;
  u64 kc, kd, ke;
  const u32 c1 = isa::add_c((u32)(P0 >> 32), (u32)S, kc);
  const u32 c2a = isa::addc_c((u32)P1, (u32)(S >> 32), kc, kd);
  const u32 c2 = isa::addc_c(c2a, 0u, cc, ke);
  const u32 c3 = isa::inc_ci(isa::inc_ci(isa::inc_ci((u32)(P1 >> 32), kd), cs), ke);
  return gl_reduce_dev<CANON>((u32)P0, c1, c2, c3);
}

// x 2^E for 0 < E <= 32 as lo64 + c2 2^64 = lo64 + c2 EPS, c2 < 2^E; with
// CANON false the result is only reduced below 2^64 (a wrap adds EPS, which
// cannot wrap again since the wrapped sum is below 2^(32+E) <= 2^64 - EPS
// for E < 32).
template <int E, bool CANON>
__device__ __forceinline__ u64 gl_shl_small_dev(u64 x) {
  static_assert(E > 0 && E <= 32, "shift out of range");
  const u32 c2 = (E == 32) ? (u32)(x >> 32) : (u32)(x >> (64 - E));
  u64 ca;
  const u64 R = isa::mad_eps_c(c2, x << E, ca);
  if constexpr (CANON)
    return isa::add_eps_if(R, ca | isa::ge_p(R));
  else
    return isa::add_eps_if(R, ca);
}

template <int E>
__device__ __forceinline__ u64 gl_mul_pow2_dev(u64 x) {
  static_assert(E >= 0 && E < 96, "exponent out of range");
  if constexpr (E == 0) {
    return x;
  } else if constexpr (E <= 32) {
    return gl_shl_small_dev<E, true>(x);
  } else if constexpr (E < 64) {
    // x 2^(E-32) below 2^64, then times 2^32 (whose product step accepts
    // any 64-bit input: c2 = hi word, a wrap leaves the sum below p - EPS)
    return gl_shl_small_dev<32, true>(gl_shl_small_dev<E - 32, false>(x));
  } else {
    // limbs c2 = lo(x) << f at 2^64 and h = x >> (32 - f) at 2^96 (the part
    // above 2^128 = -2^32 included): x 2^E = c2 EPS - h, with c2 EPS < p
    // and h < 2^63, so one conditional p after the subtraction is canonical
    constexpr int f = E - 64;
    const u32 c2 = (u32)x << f;
    const u64 h = f ? (x >> (32 - f)) : (x >> 32);
    const u64 R = (u64)c2 * 0xFFFFFFFFull;
    u64 b0, b1;
    const u32 d0 = isa::sub_c((u32)R, (u32)h, b0);
    const u32 d1 = isa::subb_c((u32)(R >> 32), (u32)(h >> 32), b0, b1);
    return isa::sub_eps_if(gl_mk(d0, d1), b1);
  }
}

// (a - b) mod p for canonical a, b: as gl_sub_portable, with the
// correction applied through carry-ins (4 instructions instead of 5).
__device__ __forceinline__ u64 gl_sub_dev(u64 a, u64 b) {
  u64 b0, b1;
  const u32 d0 = isa::sub_c((u32)a, (u32)b, b0);
  const u32 d1 = isa::subb_c((u32)(a >> 32), (u32)(b >> 32), b0, b1);
  return isa::sub_eps_if(gl_mk(d0, d1), b1);
}
#endif  // __HIP_DEVICE_COMPILE__

__host__ __device__ __forceinline__ u64 gl_sub(u64 a, u64 b) {
#if defined(__HIP_DEVICE_COMPILE__)
  return gl_sub_dev(a, b);
#else
  return gl_sub_portable(a, b);
#endif
}

// a + b up to a multiple of p, for any a < 2^64 and canonical b: the result
// is below 2^64 and congruent to a + b, not necessarily below p.  A wrap
// past 2^64 adds EPS, and cannot wrap again: a + b - 2^64 < p, so the sum
// stays below p + EPS = 2^64.  One compare fewer than gl_add; gl_sub (any
// minuend, canonical subtrahend), gl_mul, gl_mul_add and gl_mul_pow2 all
// accept such values.
__host__ __device__ __forceinline__ u64 gl_add_weak(u64 a, u64 b) {
#if defined(__HIP_DEVICE_COMPILE__)
  // the wrap's EPS through a multiply-add of the 0/1 carry (the sum is
  // already a register pair, so no zero-extended addend is needed)
  u64 c0, c1, cy;
  const u32 s0 = isa::add_c((u32)a, (u32)b, c0);
  const u32 s1 = isa::addc_c((u32)(a >> 32), (u32)(b >> 32), c0, c1);
  u32 w;
  asm("v_cndmask_b32_e64 %0, 0, 1, %1" : "=v"(w) : "s"(c1));
  return isa::mad_eps_c(w, gl_mk(s0, s1), cy);
#else
  const u64 s = a + b;
  return s < a ? s + GL_EPS : s;
#endif
}

__host__ __device__ __forceinline__ u64 gl_mul(u64 a, u64 b) {
#if defined(__HIP_DEVICE_COMPILE__)
  return gl_mul_dev(a, b);
#else
  u32 c0, c1, c2, c3;
  gl_mul_limbs(a, b, c0, c1, c2, c3);
  return gl_reduce_limbs(c0, c1, c2, c3);
#endif
}

// x * 2^E mod p for a compile-time 0 <= E < 96 (2^96 = -1 covers the rest):
// the product is a shifted copy of x's limbs, reduced like any product.
template <int E>
__host__ __device__ __forceinline__ u64 gl_mul_pow2(u64 x) {
  static_assert(E >= 0 && E < 96, "exponent out of range");
#if defined(__HIP_DEVICE_COMPILE__)
  return gl_mul_pow2_dev<E>(x);
#endif
  const u32 x0 = (u32)x, x1 = (u32)(x >> 32);
  if constexpr (E == 0) {
    return x;
  } else if constexpr (E < 32) {
    return gl_reduce_limbs(x0 << E, (x1 << E) | (x0 >> (32 - E)), x1 >> (32 - E), 0u);
  } else if constexpr (E == 32) {
    return gl_reduce_limbs(0u, x0, x1, 0u);
  } else if constexpr (E < 64) {
    constexpr int f = E - 32;
    return gl_reduce_limbs(0u, x0 << f, (x1 << f) | (x0 >> (32 - f)), x1 >> (32 - f));
  } else if constexpr (E == 64) {
    return gl_reduce_limbs(0u, 0u, x0, x1);
  } else {
    constexpr int f = E - 64;
    const u32 c4 = x1 >> (32 - f);  // weight 2^128 = -2^32 (mod p)
    return gl_sub(gl_reduce_limbs(0u, 0u, x0 << f, (x1 << f) | (x0 >> (32 - f))),
                  (u64)c4 << 32);
  }
}

// (a * b + c) mod p with one reduction: c enters the multiply-adds of
// gl_mul_limbs (its low half with a0 b0, its high half with a0 b1), which
// keeps every partial sum below 2^64; a b + c < p^2 + p < 2^128.
__host__ __device__ __forceinline__ u64 gl_mul_add(u64 a, u64 b, u64 c) {
#if defined(__HIP_DEVICE_COMPILE__)
  return gl_mul_add_dev(a, b, c);
#endif
  const u32 a0 = (u32)a, a1 = (u32)(a >> 32), b0 = (u32)b, b1 = (u32)(b >> 32);
  const u64 p00 = (u64)a0 * b0 + (u32)c;
  const u64 p01 = (u64)a0 * b1 + ((p00 >> 32) + (c >> 32));
  const u64 p10 = (u64)a1 * b0 + (u32)p01;
  const u64 p11 = (u64)a1 * b1 + ((p01 >> 32) + (p10 >> 32));
  return gl_reduce_limbs((u32)p00, (u32)p10, (u32)p11, (u32)(p11 >> 32));
}

// a b + c up to a multiple of p, for any a, c < 2^64 and canonical b: below
// 2^64 and congruent (the running sums of the key multiply-accumulate,
// which only feed further such sums until gl_canon).
__host__ __device__ __forceinline__ u64 gl_mul_add_weak(u64 a, u64 b, u64 c) {
#if defined(__HIP_DEVICE_COMPILE__)
  return gl_mul_add_dev<false>(a, b, c);
#else
  return gl_mul_add(a, b, c);
#endif
}

// The canonical representative of any x < 2^64 (x - p = x + EPS mod 2^64
// when x >= p).
__host__ __device__ __forceinline__ u64 gl_canon(u64 x) {
#if defined(__HIP_DEVICE_COMPILE__)
  return isa::add_eps_if(x, isa::ge_p(x));
#else
  return x >= GL_P ? x - GL_P : x;
#endif
}

__host__ __device__ inline u64 gl_pow(u64 a, u64 e) {
  u64 r = 1;
  while (e) {
    if (e & 1) r = gl_mul(r, a);
    a = gl_mul(a, a);
    e >>= 1;
  }
  return r;
}

__host__ __device__ inline u64 gl_inv(u64 a) { return gl_pow(a, GL_P - 2); }

// Small signed integer as a field element.
__host__ __device__ __forceinline__ u64 gl_from_i64(i64 d) {
  return d >= 0 ? (u64)d : (u64)d + GL_P;  // wraps to p - |d|
}

// Modulus switch Z_p -> Z_2N with rounding to nearest:
//   floor((2N a + (p-1)/2) / p) mod 2N,  2N = 2^(logn+1).
// With X = 2N a + (p-1)/2 = hi*2^64 + lo (hi < 2^13), X - hi*p = lo + hi*eps
// lies in [0, 2p), so the quotient is hi or hi + 1.
__host__ __device__ __forceinline__ u32 gl_modswitch(u64 a, int logn) {
  const int sh = logn + 1;
  u64 hi = a >> (64 - sh);
  u64 lo = a << sh;
  const u64 half = (GL_P - 1) / 2;
  lo += half;
  if (lo < half) ++hi;
  const u64 r = lo + hi * GL_EPS;
  u64 q = hi;
  if (r < lo || r >= GL_P) ++q;
  return (u32)(q & ((2ull << logn) - 1));
}

// Gadget decomposition digit t (0 = most significant) of a in Z_p with
// `levels` digits of beta bits: centred representative, rounding of the
// discarded s = 64 - levels*beta low bits to nearest (half up), balanced
// digits in [-B/2, B/2) from the bottom, the top digit absorbing the carry.
// floor((a_c + 2^(s-1)) / 2^s) = (a_c >> s) + bit_(s-1)(a_c) in two's
// complement, which avoids the 64-bit overflow of a_c + 2^(s-1).
__host__ __device__ __forceinline__ i64 gl_round_top(u64 a, int s) {
  const i64 ac = (a > (GL_P - 1) / 2) ? (i64)(a - GL_P) : (i64)a;
  return (ac >> s) + ((ac >> (s - 1)) & 1);
}

// gl_round_top for 34 <= s <= 63 from the high word alone, a 32-bit result.
// The centred value's high word is hi(a), or hi(a - p) = hi(a + EPS) =
// hi(a) + (lo(a) != 0) above (p - 1) / 2; with y = a_c >> (s - 1) =
// hi(a_c) >> (s - 33), floor((a_c + 2^(s-1)) / 2^s) = (y + 1) >> 1, and
// |y| < 2^30 keeps y + 1 from overflowing (at s = 33 it could).  Also exact
// for a = p (the centred value 0).
__host__ __device__ __forceinline__ int32_t gl_round_top32(u64 a, int s) {
  const u32 lo = (u32)a, hi = (u32)(a >> 32);
  const bool upper = a > (GL_P - 1) / 2;
  const int32_t h = (int32_t)(hi + (u32)(upper && lo != 0));
  return ((h >> (s - 33)) + 1) >> 1;
}

__host__ __device__ __forceinline__ i64 gl_digit(i64 r, int levels, int beta, int t) {
  const i64 half = (i64)1 << (beta - 1);
  const i64 mask = ((i64)1 << beta) - 1;
  i64 d = 0;
  for (int u = levels - 1; u >= t; --u) {
    if (u == 0) return r;
    d = ((r + half) & mask) - half;
    r = (r - d) >> beta;
  }
  return d;
}

}  // namespace rosetta
