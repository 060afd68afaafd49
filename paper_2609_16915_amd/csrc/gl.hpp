// Goldilocks field arithmetic, p = 2^64 - 2^32 + 1, for gfx950 VALU and host.
//
// 2^64 = 2^32 - 1 (mod p), so a 128-bit value hi*2^64 + lo with
// hi = h1*2^32 + h0 reduces to lo - h1 + h0*(2^32 - 1)  (since 2^96 = -1).
// All functions take and return canonical values in [0, p).  The 64x64
// product is built from four 32x32->64 multiply-adds (v_mad_u64_u32 on
// CDNA), arranged so that no intermediate overflows 64 bits.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace rosetta {

typedef uint64_t u64;
typedef uint32_t u32;
typedef int64_t i64;

constexpr u64 GL_P = 0xFFFFFFFF00000001ull;
constexpr u64 GL_EPS = 0xFFFFFFFFull;  // 2^64 mod p

__host__ __device__ __forceinline__ u64 gl_add(u64 a, u64 b) {
  u64 s = a + b;
  if (s < a) return s + GL_EPS;  // wrapped: a + b - 2^64 + (2^64 mod p), < p
  return s >= GL_P ? s - GL_P : s;
}

__host__ __device__ __forceinline__ u64 gl_sub(u64 a, u64 b) {
  u64 d = a - b;
  if (a < b) d -= GL_EPS;  // a - b + 2^64 - (2^64 - p)
  return d;
}

__host__ __device__ __forceinline__ u64 gl_neg(u64 a) { return a ? GL_P - a : 0; }

// Full 128-bit product a*b = hi*2^64 + lo.
__host__ __device__ __forceinline__ void mul_wide(u64 a, u64 b, u64 &lo, u64 &hi) {
  const u32 a0 = (u32)a, a1 = (u32)(a >> 32), b0 = (u32)b, b1 = (u32)(b >> 32);
  const u64 p00 = (u64)a0 * b0;
  const u64 t = (u64)a0 * b1 + (p00 >> 32);  // <= (2^32-1)^2 + 2^32-1 < 2^64
  const u64 u = (u64)a1 * b0 + (u32)t;
  u64 w = (u64)a1 * b1 + (t >> 32);
  w += (u >> 32);  // a1 b1 + 2 (2^32-1) <= 2^64 - 1
  lo = (p00 & 0xFFFFFFFFull) | (u << 32);
  hi = w;
}

// (hi*2^64 + lo) mod p for any 128-bit value.
__host__ __device__ __forceinline__ u64 gl_reduce128(u64 lo, u64 hi) {
  const u32 h0 = (u32)hi, h1 = (u32)(hi >> 32);
  u64 t0 = lo - h1;
  if (lo < h1) t0 -= GL_EPS;                      // borrow: add p
  const u64 t1 = ((u64)h0 << 32) - (u64)h0;       // h0 * (2^32 - 1) < p
  u64 r = t0 + t1;
  if (r < t1) r += GL_EPS;                        // wrapped
  return r >= GL_P ? r - GL_P : r;
}

__host__ __device__ __forceinline__ u64 gl_mul(u64 a, u64 b) {
  u64 lo, hi;
  mul_wide(a, b, lo, hi);
  return gl_reduce128(lo, hi);
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
