// HIP kernels for batched programmable bootstrapping on gfx950.
//
// One workgroup owns one ciphertext for the whole blind rotation: the GLWE
// accumulator stays in registers (E coefficients of each component per
// thread, or E transform slots where it is kept in the transform domain) for
// all n CMux steps, and every transform is done by the workgroup in
// registers with LDS transposes (ntt.hpp).  Only the
// bootstrapping key is streamed from memory; all workgroups walk the key in
// the same order i = 0..n-1, so a GGSW row fetched by one workgroup is
// served from L2 / the Infinity Cache to the others.
#include <atomic>
#include <hip/hip_runtime.h>

#include <type_traits>

#include "gl.hpp"
#include "internal.hpp"
#include "ntt.hpp"

namespace rosetta {

// ---------------------------------------------------------------------------
// Key preparation
// ---------------------------------------------------------------------------

// Dynamic LDS of the transform kernels: the twiddle area (TW_WORDS words:
// the zeta table with the twisted passes' block powers, see Ntt), then the
// exchange buffers (XCHG_WORDS, see LdsBufs).
extern __shared__ __align__(16) u64 lds_dyn[];

template <class S>
constexpr size_t ntt_lds_bytes() {
  return (size_t)(S::TW_WORDS + S::XCHG_WORDS) * sizeof(u64);
}

// Row r of the standard key (N coefficients) -> transform domain, scaled by
// N^-1, stored as [r][k][tid] so that thread tid of the blind rotation
// reads its E words of the row with unit stride across the workgroup.
template <class S>
__global__ void __launch_bounds__(S::T)
k_bsk_prepare(const u64 *__restrict__ std_key, u64 *__restrict__ dev_key,
              const u64 *__restrict__ zeta, u64 ninv) {
  u64 *tw = lds_dyn;
  LdsBufs<S> lds(lds_dyn + S::TW_WORDS);
  const int tid = threadIdx.x;
  const size_t row = blockIdx.x;
  load_twiddles<S>(tw, zeta, tid);
  u64 x[S::E];
#pragma unroll
  for (int k = 0; k < S::E; ++k) x[k] = std_key[row * S::N + tid + S::T * k];
  __syncthreads();
  ntt_forward<S>(x, lds, tid, tw);
#pragma unroll
  for (int k = 0; k < S::E; ++k) dev_key[row * S::N + k * S::T + tid] = gl_mul(x[k], ninv);
}

// ---------------------------------------------------------------------------
// Stand-alone transforms
// ---------------------------------------------------------------------------

template <class S>
__global__ void __launch_bounds__(S::T)
k_ntt_forward(const u64 *in, u64 *out, const u64 *__restrict__ zeta) {
  u64 *tw = lds_dyn;
  LdsBufs<S> lds(lds_dyn + S::TW_WORDS);
  const int tid = threadIdx.x;
  const size_t base = (size_t)blockIdx.x * S::N;
  load_twiddles<S>(tw, zeta, tid);
  u64 x[S::E];
#pragma unroll
  for (int k = 0; k < S::E; ++k) x[k] = in[base + tid + S::T * k];
  __syncthreads();
  ntt_forward<S>(x, lds, tid, tw);
#pragma unroll
  for (int k = 0; k < S::E; ++k) out[base + S::idx(S::PASSES - 1, tid, k)] = x[k];
}

template <class S>
__global__ void __launch_bounds__(S::T)
k_ntt_inverse(const u64 *in, u64 *out, const u64 *__restrict__ zeta, u64 ninv) {
  u64 *tw = lds_dyn;
  LdsBufs<S> lds(lds_dyn + S::TW_WORDS);
  const int tid = threadIdx.x;
  const size_t base = (size_t)blockIdx.x * S::N;
  load_twiddles<S>(tw, zeta, tid);
  u64 x[S::E];
#pragma unroll
  for (int k = 0; k < S::E; ++k) x[k] = in[base + S::idx(S::PASSES - 1, tid, k)];
  __syncthreads();
  ntt_inverse<S>(x, lds, tid, tw);
#pragma unroll
  for (int k = 0; k < S::E; ++k) out[base + tid + S::T * k] = gl_mul(x[k], ninv);
}

template <class S>
__global__ void __launch_bounds__(S::T)
k_poly_mul(const u64 *a, const u64 *b, u64 *c, const u64 *__restrict__ zeta, u64 ninv) {
  u64 *tw = lds_dyn;
  LdsBufs<S> lds(lds_dyn + S::TW_WORDS);
  const int tid = threadIdx.x;
  const size_t base = (size_t)blockIdx.x * S::N;
  load_twiddles<S>(tw, zeta, tid);
  u64 x[S::E], y[S::E];
#pragma unroll
  for (int k = 0; k < S::E; ++k) {
    x[k] = a[base + tid + S::T * k];
    y[k] = b[base + tid + S::T * k];
  }
  __syncthreads();
  ntt_forward<S>(x, lds, tid, tw);
  ntt_forward<S>(y, lds, tid, tw);
#pragma unroll
  for (int k = 0; k < S::E; ++k) x[k] = gl_mul(x[k], y[k]);
  ntt_inverse<S>(x, lds, tid, tw);
#pragma unroll
  for (int k = 0; k < S::E; ++k) c[base + tid + S::T * k] = gl_mul(x[k], ninv);
}

// ---------------------------------------------------------------------------
// Blind rotation (+ sample extraction)
// ---------------------------------------------------------------------------

// Waves per SIMD the blind-rotation kernel is compiled for.  Up to N = 2048
// three workgroups fit a CU's LDS, so the kernel targets 3 waves per SIMD
// (<= 168 registers, a few of them spilled; 4 waves at 128 registers, with
// the LDS of the N = 4096 layout below, spilled 107 and ran 1010 instead of
// 902 ms per headline launch with the coefficient-domain loop).
// At N = 4096 a workgroup is 512 threads of 8 elements whose exchanges
// share one LDS buffer (66 KiB): two workgroups share a CU, two waves of
// each per SIMD, with 128 registers each.  With the accumulator in the
// transform domain (no separate running sums, see br_transform_domain) the
// spill traffic of that budget stays in the L2: 1159 ms per 8192
// ciphertexts, against 1301 ms for the coefficient-domain loop at four
// waves and 1426 ms for 16 elements per thread in 256-thread workgroups at
// 2 waves (radix-16 passes, 5 % fewer instructions).
#ifndef BR_WAVES_PER_EU
#define BR_WAVES_PER_EU 3
#endif
template <class S>
constexpr int br_waves_per_eu() {
  return S::LOGN >= 12 ? 4 : BR_WAVES_PER_EU;
}

// Rows of one GGSW read through a raw buffer descriptor: a wave-uniform
// base, the lane's byte offset in a vector register and the row's byte
// offset in a scalar register, so that the address arithmetic of the key
// stream runs on the scalar unit.  Word 3 of the descriptor is the gfx9
// raw-buffer setting (32-bit data format); num_records only bounds the
// lane offset, which stays far below it.
struct KeyRows {
  __amdgpu_buffer_rsrc_t r;
  __device__ __forceinline__ explicit KeyRows(const u64 *base)
      : r(__builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, 0x7FFFFFFF, 0x00020000)) {}
  __device__ __forceinline__ u64 load(int lane_byte, int row_byte) const {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, lane_byte, row_byte, 0);
    return ((u64)v[1] << 32) | v[0];
  }
};

// Coefficient j of X^r * v (negacyclic), 0 <= r < 2N.
template <int N>
__device__ __forceinline__ u64 rotated_coef(const u64 *v, int j, int r) {
  const int rr = r & (N - 1);
  const bool neg = (j < rr) != (r >= N);
  const u64 x = v[(j - rr) & (N - 1)];
  return neg ? gl_neg(x) : x;
}

// Key rows per chunk at the four-wave budget, and the scheduling fence
// between chunks (see br_levels).
#ifndef BR_KEY_CHUNK
#define BR_KEY_CHUNK 1
#endif
#ifndef BR_CHUNK_FENCE
#define BR_CHUNK_FENCE() __builtin_amdgcn_sched_barrier(0)
#endif

// a3-a5 for one component u of the rotated difference, whose rounded
// coefficients R it consumes: levels from the least significant (t = L-1)
// up, each pass taking the balanced low digit of R and shifting it out, the
// last level what remains (the sums over t are exact, so their order is
// free).  Each digit polynomial is transformed and multiplied into the
// running sums Y0, Y1 (the transform-domain accumulator itself, where the
// kernel keeps one) with the two rows of GGSW_i[u][t] (sums weak, below
// 2^64 and congruent).
template <class S, int L, typename RT, bool CHUNKED>
__device__ __forceinline__ void br_levels(RT (&R)[S::E], u64 (&Y0)[S::E], u64 (&Y1)[S::E],
                                          const KeyRows &G, int u, int beta, LdsBufs<S> &lds,
                                          int tid, const u64 *tw) {
  constexpr int N = S::N, E = S::E, T = S::T;
  const RT half = (RT)1 << (beta - 1);
#pragma unroll 1
  for (int t = L - 1; t >= 0; --t) {
    const int row = (u * L + t) * 2 * N * 8;  // byte offset of GGSW_i[u][t][0]
    u64 g0[CHUNKED ? 1 : E], g1[CHUNKED ? 1 : E];
    // chunked: the first chunk of the two key rows is requested before
    // the digit transform, so that the transform hides its latency (the
    // later chunks overlap the chunk before them)
    u64 h0[BR_KEY_CHUNK], h1[BR_KEY_CHUNK];
    if constexpr (CHUNKED) {
#pragma unroll
      for (int k = 0; k < BR_KEY_CHUNK; ++k) {
        h0[k] = G.load(tid * 8, row + k * T * 8);
        h1[k] = G.load(tid * 8, row + (N + k * T) * 8);
      }
    }
    // a3: digit polynomial of level t;  a4: forward transform (its first
    // two stages in integer arithmetic while the digits are small)
    RT d[E];
    if (t == 0) {
#pragma unroll
      for (int k = 0; k < E; ++k) d[k] = R[k];
    } else {
      // the low beta bits sign-extended, the rest carried up
      const int dsh = (int)(8 * sizeof(RT)) - beta;
#pragma unroll
      for (int k = 0; k < E; ++k) {
        d[k] = (RT)((std::make_unsigned_t<RT>)R[k] << dsh) >> dsh;
        R[k] = (R[k] + half) >> beta;
      }
    }
    u64 x[E];
    if (beta <= 14) {
      ntt_forward_small<S, RT>(d, x, lds, tid, tw);
    } else {
#pragma unroll
      for (int k = 0; k < E; ++k) x[k] = gl_from_i64((i64)d[k]);
      ntt_forward<S>(x, lds, tid, tw);
    }
    // a5: multiply-accumulate with the two rows of GGSW_i[u][t]
    // (running sums weak until the inverse transform takes them)
    if constexpr (!CHUNKED) {
      // (requested here, after the transform: loading them before it,
      // with 8 elements per thread and 3 waves, cost more in spills of
      // its 32 registers than the early loads saved)
#pragma unroll
      for (int k = 0; k < E; ++k) {
        g0[k] = G.load(tid * 8, row + k * T * 8);
        g1[k] = G.load(tid * 8, row + (N + k * T) * 8);
      }
#pragma unroll
      for (int k = 0; k < E; ++k) {
        Y0[k] = gl_mul_add_weak(x[k], g0[k], Y0[k]);
        Y1[k] = gl_mul_add_weak(x[k], g1[k], Y1[k]);
      }
    } else {
      // the key rows a chunk at a time (BR_KEY_CHUNK elements, 4
      // registers each), the next chunk requested before the products
      // of the current one, so that 2 chunks rather than 32 registers
      // hold them (N = 4096, ms per 8192 ciphertexts on one box: chunks
      // of 1 1322 and 1329 against 1346 and 1349 for chunks of 2; on
      // another, chunks of 2 with a scheduling fence between chunks
      // 1297, without it 1327, chunks of 4 1489, all rows after the
      // transform 1321; at N = 2048, 3 waves, chunks of 2 ran 908
      // against 902 ms unchunked)
#pragma unroll
      for (int k0 = 0; k0 < E; k0 += BR_KEY_CHUNK) {
        u64 n0[BR_KEY_CHUNK], n1[BR_KEY_CHUNK];
        if (k0 + BR_KEY_CHUNK < E) {
#pragma unroll
          for (int k = 0; k < BR_KEY_CHUNK; ++k) {
            n0[k] = G.load(tid * 8, row + (k0 + BR_KEY_CHUNK + k) * T * 8);
            n1[k] = G.load(tid * 8, row + (N + (k0 + BR_KEY_CHUNK + k) * T) * 8);
          }
        }
#pragma unroll
        for (int k = 0; k < BR_KEY_CHUNK; ++k) {
          Y0[k0 + k] = gl_mul_add_weak(x[k0 + k], h0[k], Y0[k0 + k]);
          Y1[k0 + k] = gl_mul_add_weak(x[k0 + k], h1[k], Y1[k0 + k]);
        }
        if (k0 + BR_KEY_CHUNK < E) {
#pragma unroll
          for (int k = 0; k < BR_KEY_CHUNK; ++k) {
            h0[k] = n0[k];
            h1[k] = n1[k];
          }
        }
        BR_CHUNK_FENCE();
      }
    }
  }
}

// The accumulator in the transform domain (br_transform_domain):
// H_c = N^-1 NTT(ACC_c).  The key rows are scaled by N^-1 as well, so the
// step's products add into H directly and no separate running sums are
// live across the digit transforms; the rotate-subtract becomes a product
// by the transform of X^a - 1, and the inverse transform of (W^a - 1) H_c
// is exactly X^a ACC_c - ACC_c (the inverse transform leaves the factor N
// that cancels N^-1).  Every step is the same arithmetic mod p as the
// coefficient-domain loop, so the outputs are the same bits.
//
// The transform's slot of in-place index j holds the evaluation at
// psi^(2 rev(j) + 1), so the slot's factor is psi^((2 rev(j) + 1) a) - 1.
// In the last pass (lo = 0, E = 8) thread tid holds j = 8 tid + k, and
// 2 rev(j) + 1 = c0 + rev3(k) N/4 with c0 = 2 rev(tid) + 1 (the (LOGN-3)-bit
// reversal), so the factor is g w8^(rev3(k) a) - 1 with g = psi^(c0 a) and
// w8 = psi^(N/4) = 7^((p-1)/8) = 2^120: one table read of g per step and
// shifts for the rest.
template <class S>
constexpr bool td_layout_ok() {
  return S::E == 8 && S::lo(S::PASSES - 1) == 0;
}

// The table read of g = psi^e (e < 2N) from psi^0 .. psi^(N-1): the raw
// word and whether it is negated (psi^N = -1), applied where g is used so
// that the read can be issued a step ahead.
struct PsiPow {
  u64 v;
  bool neg;
};
template <int N>
__device__ __forceinline__ PsiPow psi_read(const u64 *__restrict__ tab, int e) {
  return PsiPow{tab[e & (N - 1)], (e & N) != 0};
}

// w[k] = g 2^(120 ((rev3(k) R) mod 8)) - 1 for the eight slots of a thread.
template <int R>
__device__ __forceinline__ void spectrum_minus_one_r(u64 g, u64 (&w)[8]) {
  static_for<0, 8>([&](auto kc) {
    constexpr int k = decltype(kc)::value;
    constexpr int e = (120 * ((rev3(k) * R) & 7)) % 192;
    const u64 m = mul_pow2_mag<e>(g);
    // -m - 1 = (p - 1) - m
    w[k] = sign_pow2(e) > 0 ? gl_sub(m, 1) : gl_sub(GL_P - 1, m);
  });
}
__device__ __forceinline__ void spectrum_minus_one(PsiPow gp, int a, u64 (&w)[8]) {
  const u64 g = gp.neg ? GL_P - gp.v : gp.v;  // a root of unity: never 0
  switch (__builtin_amdgcn_readfirstlane(a) & 7) {
    case 0: spectrum_minus_one_r<0>(g, w); break;
    case 1: spectrum_minus_one_r<1>(g, w); break;
    case 2: spectrum_minus_one_r<2>(g, w); break;
    case 3: spectrum_minus_one_r<3>(g, w); break;
    case 4: spectrum_minus_one_r<4>(g, w); break;
    case 5: spectrum_minus_one_r<5>(g, w); break;
    case 6: spectrum_minus_one_r<6>(g, w); break;
    default: spectrum_minus_one_r<7>(g, w); break;
  }
}

// One component's rotated difference X^a ACC - ACC = inverse((W^a - 1) H),
// rounded to its top l beta bits (natural layout, as the digits need it).
template <class S, typename RT>
__device__ __forceinline__ void td_difference(const u64 (&H)[S::E], const u64 (&w)[S::E],
                                              RT (&R)[S::E], int s, LdsBufs<S> &lds, int tid,
                                              const u64 *tw) {
  u64 y[S::E];
#pragma unroll
  for (int k = 0; k < S::E; ++k) y[k] = gl_mul(w[k], H[k]);
  ntt_inverse<S>(y, lds, tid, tw);
#pragma unroll
  for (int k = 0; k < S::E; ++k) {
    if constexpr (sizeof(RT) == 4)
      R[k] = gl_round_top32(y[k], s);
    else
      R[k] = gl_round_top(y[k], s);
  }
}

// Whether an instance keeps its accumulator in the transform domain: every
// instance at N >= 2048 (the rings of the workloads).  Measured against the
// coefficient-domain loop on one box: N = 4096 at four waves 1301 -> 1159 ms
// per 8192 ciphertexts (its spill traffic had gone beyond the L2), the 32
// reciprocals at two waves 47.5 -> 46.9 ms, at N = 2048 the 64-bit-rounding
// lookup key set 923 -> 911 ms and the headline and GPT-2 shapes 0.4 and
// 0.8 % faster.  Smaller rings keep the coefficient-domain loop.
template <class S>
constexpr bool br_transform_domain() {
  return S::LOGN >= 11 && td_layout_ok<S>();
}

// One workgroup per ciphertext.  Per CMux step i:
//   a2  D_u = X^(a~_i) ACC_u - ACC_u           (rotation through LDS)
//   a3  digits of D_u, level t                 (registers)
//   a4  forward transform of each digit poly   (registers + LDS)
//   a5  Y_c += digits^ . GGSW_i[u][t][c]^      (key streamed, pre-transformed)
//   a6  ACC_c += inverse transform of Y_c
// or, with the accumulator in the transform domain (H_c = N^-1 NTT(ACC_c)):
//   a2  D_u = inverse transform of (W^a - 1) H_u, both u first
//   a3-a5 as above, the products added into H_c directly (a6 folded in)
// The transform-domain key rows are pre-scaled by N^-1 (k_bsk_prepare).
// RT holds the rounded value before digit extraction: 32 bits suffice when
// l * beta <= 30.  WAVES is the register budget (waves per SIMD): with 4
// the key rows stream a chunk at a time, the first chunk requested before
// the digit's forward transform so that the transform hides its latency.
//
// Dynamic LDS: twiddle area [TW_WORDS], exchange buffers [XCHG_WORDS],
// then the n+1 rounded rotation amounts (u16).
template <class S>
size_t br_lds_bytes(int n) {
  return ntt_lds_bytes<S>() + (((size_t)(n + 1) * 2 + 15) & ~(size_t)15);
}

//
// With tp_glwe = 0, `lut` is one test polynomial v shared by the batch and
// the accumulator starts as the trivial ciphertext (0, X^(-b~) v).  With
// tp_glwe = 1, `lut` holds one GLWE ciphertext [2][N] per ciphertext of the
// batch (a test polynomial that is itself encrypted, as in the lookup
// protocol's construct-then-select) and both of its components are rotated
// by X^(-b~).
//
// tp_glwe = g > 1 pairs each LWE selector with g consecutive test-polynomial
// ciphertexts (workgroup b uses selector b / g), so that one encrypted
// index selects in several ciphertexts at once.
template <class S, int L, typename RT, int WAVES>
__global__ void __launch_bounds__(S::T) __attribute__((amdgpu_waves_per_eu(WAVES)))
k_blind_rotate(const u64 *__restrict__ lwe_in, const u64 *__restrict__ bsk,
               const u64 *__restrict__ lut, u64 *__restrict__ out, int n, int beta, int mode,
               int tp_glwe, const u64 *__restrict__ zeta, const u64 *__restrict__ psi_pow,
               u64 ninv) {
  constexpr int N = S::N, E = S::E, T = S::T;
  static_assert(E <= 8, "at most 8 elements per thread");
  // key rows a chunk at a time at the 128-register budget of four waves
  constexpr bool CHUNKED = WAVES >= 4;
  constexpr bool TD = br_transform_domain<S>();
  u64 *tw = lds_dyn;
  LdsBufs<S> lds(lds_dyn + S::TW_WORDS);
  uint16_t *rot = (uint16_t *)(lds_dyn + S::TW_WORDS + S::XCHG_WORDS);
  const int tid = threadIdx.x;
  const size_t ct = blockIdx.x;

  // a1: rounded rotation amounts of the whole ciphertext; twiddles
  const u64 *lwe = lwe_in + (ct / (size_t)(tp_glwe > 1 ? tp_glwe : 1)) * (size_t)(n + 1);
  for (int i = tid; i <= n; i += T) rot[i] = (uint16_t)gl_modswitch(lwe[i], S::LOGN);
  load_twiddles<S>(tw, zeta, tid);
  __syncthreads();

  u64 accA[E], accB[E];
  {
    const int r = (2 * N - (int)rot[n]) & (2 * N - 1);  // X^(-b~)
    const u64 *tpA = lut + (tp_glwe ? ct * (size_t)(2 * N) : 0);
    const u64 *tpB = tp_glwe ? tpA + N : lut;
#pragma unroll
    for (int k = 0; k < E; ++k) {
      accA[k] = tp_glwe ? rotated_coef<N>(tpA, tid + T * k, r) : 0;
      accB[k] = rotated_coef<N>(tpB, tid + T * k, r);
    }
  }

  const int s = 64 - L * beta;
  constexpr size_t ggsw_words = (size_t)2 * L * 2 * N;
  if constexpr (TD) {
    // H_c = N^-1 NTT(ACC_c)
    const int c0 = 2 * (int)(__builtin_bitreverse32((unsigned)tid) >> (32 - (S::LOGN - 3))) + 1;
    // (once per ciphertext, so the two components share one copy of the
    // transform's code; a zero mask needs no transform)
    u64 HA[E], HB[E];
#pragma unroll
    for (int k = 0; k < E; ++k) HA[k] = 0;
#pragma unroll 1
    for (int c = tp_glwe ? 0 : 1; c < 2; ++c) {
      u64 x[E];
#pragma unroll
      for (int k = 0; k < E; ++k) x[k] = c ? accB[k] : accA[k];
      ntt_forward<S>(x, lds, tid, tw);
#pragma unroll
      for (int k = 0; k < E; ++k) {
        const u64 h = gl_mul(x[k], ninv);
        if (c)
          HB[k] = h;
        else
          HA[k] = h;
      }
    }
    PsiPow g = psi_read<N>(psi_pow, c0 * (int)rot[0]);
    for (int i = 0; i < n; ++i) {
      const int a = rot[i];
      u64 w[E];
      spectrum_minus_one(g, a, w);
      if (i + 1 < n) g = psi_read<N>(psi_pow, c0 * (int)rot[i + 1]);
      // a2 (both components before the products change H), then a3-a5
      RT RA[E], RB[E];
      td_difference<S, RT>(HA, w, RA, s, lds, tid, tw);
      td_difference<S, RT>(HB, w, RB, s, lds, tid, tw);
      const KeyRows G(bsk + (size_t)i * ggsw_words);
      RT R[E];
#pragma unroll
      for (int k = 0; k < E; ++k) R[k] = RA[k];
#pragma unroll 1
      for (int u = 0; u < 2; ++u) {
        br_levels<S, L, RT, CHUNKED>(R, HA, HB, G, u, beta, lds, tid, tw);
#pragma unroll
        for (int k = 0; k < E; ++k) R[k] = RB[k];
      }
    }
    // back to coefficients: the inverse transform of H_c is N N^-1 ACC_c
#pragma unroll 1
    for (int c = 0; c < 2; ++c) {
      u64 y[E];
#pragma unroll
      for (int k = 0; k < E; ++k) y[k] = gl_canon(c ? HB[k] : HA[k]);
      ntt_inverse<S>(y, lds, tid, tw);
#pragma unroll
      for (int k = 0; k < E; ++k) {
        if (c)
          accB[k] = y[k];
        else
          accA[k] = y[k];
      }
    }
  } else {
    for (int i = 0; i < n; ++i) {
      const int a = rot[i];
      const int ar = a & (N - 1);
      const bool flip = a >= N;
      u64 Y0[E], Y1[E];
#pragma unroll
      for (int k = 0; k < E; ++k) Y0[k] = Y1[k] = 0;
      const KeyRows G(bsk + (size_t)i * ggsw_words);

#pragma unroll 1
      for (int u = 0; u < 2; ++u) {
        // a2: rotate-subtract (natural layout), then round away the s low bits
        RT R[E];
        {
          u64 cur[E];
#pragma unroll
          for (int k = 0; k < E; ++k) cur[k] = u ? accB[k] : accA[k];
          u64 *buf = lds.cross();
#pragma unroll
          for (int k = 0; k < E; ++k) buf[tid + T * k] = cur[k];
          __syncthreads();
#pragma unroll
          for (int k = 0; k < E; ++k) {
            const int j = tid + T * k;
            const bool neg = (j < ar) != flip;
            const u64 v = buf[(j - ar) & (N - 1)];
            // -v as p - v: p itself for v = 0 is a valid minuend of gl_sub,
            // and the rounding maps it to 0 as it does 0
            const u64 d = gl_sub(neg ? GL_P - v : v, cur[k]);
            if constexpr (sizeof(RT) == 4)
              R[k] = gl_round_top32(d, s);  // s = 64 - l beta >= 34 here
            else
              R[k] = gl_round_top(d, s);
          }
        }
        br_levels<S, L, RT, CHUNKED>(R, Y0, Y1, G, u, beta, lds, tid, tw);
      }
      // a6: back to coefficients, accumulate (unrolled: with c a compile-time
      // index the accumulator updates need no per-element selection)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        u64 y[E];
#pragma unroll
        for (int k = 0; k < E; ++k) y[k] = gl_canon(c ? Y1[k] : Y0[k]);
        ntt_inverse<S>(y, lds, tid, tw);
#pragma unroll
        for (int k = 0; k < E; ++k) {
          if (c)
            accB[k] = gl_add(accB[k], y[k]);
          else
            accA[k] = gl_add(accA[k], y[k]);
        }
      }
    }
  }

  if (mode == BR_GLWE) {
    u64 *o = out + ct * (size_t)(2 * N);
#pragma unroll
    for (int k = 0; k < E; ++k) {
      o[tid + T * k] = accA[k];
      o[N + tid + T * k] = accB[k];
    }
  } else {
    // a7: sample extraction  a'_0 = A_0, a'_j = -A_{N-j}, b' = B_0
    u64 *o = out + ct * (size_t)(N + 1);
#pragma unroll
    for (int k = 0; k < E; ++k) {
      const int j = tid + T * k;
      o[(N - j) & (N - 1)] = j ? gl_neg(accA[k]) : accA[k];
      if (j == 0) o[N] = accB[k];
    }
  }
}

// ---------------------------------------------------------------------------
// RLWE trace, plaintext products, recombination (lookup protocol)
// ---------------------------------------------------------------------------

// d^-1 modulo 2N for odd d: Newton's iteration x <- x (2 - d x) doubles the
// number of correct low bits, starting from x = d (d^2 = 1 mod 8).
__device__ __forceinline__ u32 odd_inverse_mod(u32 d, u32 two_n) {
  u32 x = d;
#pragma unroll
  for (int it = 0; it < 4; ++it) x *= 2u - d * x;
  return x & (two_n - 1);
}

// Coefficient j of tau_d(a) = a(X^d): with e = j d^-1 mod 2N, the source
// is a_e (e < N) or -a_(e-N) (X^N = -1).  `a` is in natural layout in LDS.
template <int N>
__device__ __forceinline__ u64 automorphism_coef(const u64 *a, int j, u32 dinv) {
  const u32 e = ((u32)j * dinv) & (2 * N - 1);
  const u64 v = a[e & (N - 1)];
  return e < (u32)N ? v : gl_neg(v);
}

// Trace of one GLWE ciphertext per workgroup (the RLWE trace of the lookup
// protocol): c <- N^-1 c, then for k = log2 N down to 1 with d = 2^k + 1,
//   c <- c + KS_d(tau_d(c)),
//   KS_d(A', B') = (0, B') - sum_t Dec_t(A') . autk[k-1][t],
// autk rows prepared like bootstrapping-key rows (transform domain, N^-1).
// Per round: two automorphisms through LDS, L forward transforms of the
// digit polynomials, 2L multiply-accumulates with the streamed key rows and
// two inverse transforms; the ciphertext stays in registers throughout.
#ifndef TRACE_WAVES_PER_EU
#define TRACE_WAVES_PER_EU 3
#endif
// At N = 4096 a workgroup is 512 threads (8 waves): two waves per SIMD,
// one workgroup per CU (its 64-bit digits keep about 190 registers live).
template <class S>
constexpr int trace_waves_per_eu() {
  return S::LOGN >= 12 ? 2 : TRACE_WAVES_PER_EU;
}

template <class S, int L>
__global__ void __launch_bounds__(S::T) __attribute__((amdgpu_waves_per_eu(trace_waves_per_eu<S>())))
k_trace(const u64 *__restrict__ in, const u64 *__restrict__ autk, u64 *__restrict__ out,
        int beta, const u64 *__restrict__ zeta, u64 ninv) {
  constexpr int N = S::N, E = S::E, T = S::T;
  u64 *tw = lds_dyn;
  LdsBufs<S> lds(lds_dyn + S::TW_WORDS);
  const int tid = threadIdx.x;
  const size_t ct = blockIdx.x;
  load_twiddles<S>(tw, zeta, tid);

  u64 A[E], B[E];
  {
    const u64 *c = in + ct * (size_t)(2 * N);
#pragma unroll
    for (int k = 0; k < E; ++k) {
      A[k] = gl_mul(c[tid + T * k], ninv);
      B[k] = gl_mul(c[N + tid + T * k], ninv);
    }
  }
  __syncthreads();

  const int s = 64 - L * beta;
  constexpr size_t round_words = (size_t)L * 2 * N;
#pragma unroll 1
  for (int kr = S::LOGN; kr >= 1; --kr) {
    const u32 dinv = odd_inverse_mod((1u << kr) + 1, 2 * N);
    // B <- B + tau_d(B)
    {
      u64 *buf = lds.cross();
#pragma unroll
      for (int k = 0; k < E; ++k) buf[tid + T * k] = B[k];
      __syncthreads();
#pragma unroll
      for (int k = 0; k < E; ++k) B[k] = gl_add(B[k], automorphism_coef<N>(buf, tid + T * k, dinv));
    }
    // rounded tau_d(A), the input of the decomposition
    i64 R[E];
    {
      u64 *buf = lds.cross();
#pragma unroll
      for (int k = 0; k < E; ++k) buf[tid + T * k] = A[k];
      __syncthreads();
#pragma unroll
      for (int k = 0; k < E; ++k) R[k] = gl_round_top(automorphism_coef<N>(buf, tid + T * k, dinv), s);
    }
    u64 Y0[E], Y1[E];
#pragma unroll
    for (int k = 0; k < E; ++k) Y0[k] = Y1[k] = 0;
    gconst_u64 *G = as_global(autk) + (size_t)(kr - 1) * round_words + tid;
    // levels from the least significant up, as in the blind rotation
    const i64 half = (i64)1 << (beta - 1);
#pragma unroll 1
    for (int t = L - 1; t >= 0; --t) {
      i64 d[E];
      if (t == 0) {
#pragma unroll
        for (int k = 0; k < E; ++k) d[k] = R[k];
      } else {
        const int dsh = 64 - beta;
#pragma unroll
        for (int k = 0; k < E; ++k) {
          d[k] = (i64)((u64)R[k] << dsh) >> dsh;
          R[k] = (R[k] + half) >> beta;
        }
      }
      u64 x[E];
      if (beta <= 14) {
        ntt_forward_small<S, i64>(d, x, lds, tid, tw);
      } else {
#pragma unroll
        for (int k = 0; k < E; ++k) x[k] = gl_from_i64(d[k]);
        ntt_forward<S>(x, lds, tid, tw);
      }
      gconst_u64 *g = G + (size_t)(t * 2) * N;
#pragma unroll
      for (int k = 0; k < E; ++k) {
        Y0[k] = gl_mul_add_weak(x[k], g[k * T], Y0[k]);
        Y1[k] = gl_mul_add_weak(x[k], g[N + k * T], Y1[k]);
      }
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      u64 y[E];
#pragma unroll
      for (int k = 0; k < E; ++k) y[k] = gl_canon(c ? Y1[k] : Y0[k]);
      ntt_inverse<S>(y, lds, tid, tw);
#pragma unroll
      for (int k = 0; k < E; ++k) {
        if (c)
          B[k] = gl_sub(B[k], y[k]);
        else
          A[k] = gl_sub(A[k], y[k]);
      }
    }
  }
  u64 *o = out + ct * (size_t)(2 * N);
#pragma unroll
  for (int k = 0; k < E; ++k) {
    o[tid + T * k] = A[k];
    o[N + tid + T * k] = B[k];
  }
}

// Plaintext-ciphertext products (the "construct" of the lookup protocol):
// for ciphertext q and plaintext s < npoly,
//   out[q][s] = (pa_s * A_q, pa_s * B_q + pb_s),
// pa_s prepared like a key row (transform domain, N^-1), pb_s in
// coefficients (pb may be NULL).  One workgroup per ciphertext: both
// components are transformed once and reused for every s.
template <class S>
__global__ void __launch_bounds__(S::T)
k_glwe_mul_plain(const u64 *__restrict__ in, const u64 *__restrict__ pa,
                 const u64 *__restrict__ pb, u64 *__restrict__ out, int npoly,
                 const u64 *__restrict__ zeta) {
  constexpr int N = S::N, E = S::E, T = S::T;
  u64 *tw = lds_dyn;
  LdsBufs<S> lds(lds_dyn + S::TW_WORDS);
  const int tid = threadIdx.x;
  const size_t ct = blockIdx.x;
  load_twiddles<S>(tw, zeta, tid);
  u64 fa[E], fb[E];
  {
    const u64 *c = in + ct * (size_t)(2 * N);
#pragma unroll
    for (int k = 0; k < E; ++k) {
      fa[k] = c[tid + T * k];
      fb[k] = c[N + tid + T * k];
    }
  }
  __syncthreads();
  ntt_forward<S>(fa, lds, tid, tw);
  ntt_forward<S>(fb, lds, tid, tw);
#pragma unroll 1
  for (int sp = 0; sp < npoly; ++sp) {
    const u64 *w = pa + (size_t)sp * N + tid;
    u64 *o = out + (ct * (size_t)npoly + sp) * (size_t)(2 * N);
#pragma unroll 1
    for (int c = 0; c < 2; ++c) {
      u64 y[E];
#pragma unroll
      for (int k = 0; k < E; ++k) y[k] = gl_mul(c ? fb[k] : fa[k], w[k * T]);
      ntt_inverse<S>(y, lds, tid, tw);
#pragma unroll
      for (int k = 0; k < E; ++k) {
        const int j = tid + T * k;
        o[c * N + j] = (c && pb) ? gl_add(y[k], pb[(size_t)sp * N + j]) : y[k];
      }
    }
  }
}

// Coefficient j of X^e a (0 <= e < 2N; X^N = -1).
__device__ __forceinline__ u64 monomial_coef(const u64 *a, int j, int e, int N) {
  const int r = e & (N - 1);
  const bool neg = (j < r) != (e >= N);
  const u64 v = a[(j - r) & (N - 1)];
  return neg ? gl_neg(v) : v;
}

// Recombination: out[q] = sum_{s < count} X^(e_s) in[q][s] (both
// components).  One thread per output coefficient.
__global__ void k_glwe_recombine(const u64 *__restrict__ in, u64 *__restrict__ out, size_t batch,
                                 int count, Exponents ex, int N) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= batch * 2 * (size_t)N) return;
  const int j = (int)(i % N);
  const size_t qc = i / N;  // q * 2 + c
  const size_t q = qc / 2, c = qc % 2;
  u64 acc = 0;
  for (int s = 0; s < count; ++s)
    acc = gl_add(acc, monomial_coef(in + ((q * count + s) * 2 + c) * N, j, ex.e[s], N));
  out[i] = acc;
}

// Monomial copies: out[q][s] = X^(e_s) in[q] (both components).
__global__ void k_glwe_monomial_mul(const u64 *__restrict__ in, u64 *__restrict__ out,
                                    size_t batch, int count, Exponents ex, int N) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= batch * count * 2 * (size_t)N) return;
  const int j = (int)(i % N);
  const size_t c = (i / N) % 2;
  const size_t s = (i / (2 * (size_t)N)) % count;
  const size_t q = i / (2 * (size_t)N * count);
  out[i] = monomial_coef(in + (q * 2 + c) * N, j, ex.e[s], N);
}

// Sample extraction of the constant coefficient of GLWE ciphertexts:
// a'_0 = A_0, a'_j = -A_{N-j}, b' = B_0 (the BR_EXTRACT epilogue, alone).
__global__ void k_sample_extract(const u64 *__restrict__ in, u64 *__restrict__ out, size_t batch,
                                 int N) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= batch * (size_t)(N + 1)) return;
  const size_t q = i / (N + 1);
  const int j = (int)(i % (N + 1));
  const u64 *g = in + q * 2 * (size_t)N;
  out[i] = j == N ? g[N] : (j == 0 ? g[0] : gl_neg(g[N - j]));
}

// ---------------------------------------------------------------------------
// LWE linear maps (comparison inputs and index sums of the lookup)
// ---------------------------------------------------------------------------

// out[q][j] = in[q] + (0, .., 0, c_j): `count` shifted copies per ciphertext.
__global__ void k_lwe_add_consts(const u64 *__restrict__ in, u64 *__restrict__ out,
                                 size_t batch, int count, int dim, Consts cs) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t w = (size_t)dim + 1;
  if (i >= batch * count * w) return;
  const size_t c = i % w, j = (i / w) % count, q = i / (w * count);
  const u64 v = in[q * w + c];
  out[i] = c == (size_t)dim ? gl_add(v, cs.c[j]) : v;
}

// out[q] = sum_{j < count} in[q][j] + (0, .., 0, c): sums of groups.
__global__ void k_lwe_sum_groups(const u64 *__restrict__ in, u64 *__restrict__ out,
                                 size_t batch, int count, int dim, u64 c0) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t w = (size_t)dim + 1;
  if (i >= batch * w) return;
  const size_t c = i % w, q = i / w;
  u64 acc = c == (size_t)dim ? c0 : 0;
  for (int j = 0; j < count; ++j) acc = gl_add(acc, in[(q * count + j) * w + c]);
  out[i] = acc;
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

#define ROSETTA_DISPATCH_N(LOGN_VAR, ...)                                             \
  switch (LOGN_VAR) {                                                                 \
    case 8: { using S = Ntt<8, ntt_le(8), ntt_first(8)>; __VA_ARGS__; } break;        \
    case 9: { using S = Ntt<9, ntt_le(9), ntt_first(9)>; __VA_ARGS__; } break;        \
    case 10: { using S = Ntt<10, ntt_le(10), ntt_first(10)>; __VA_ARGS__; } break;    \
    case 11: { using S = Ntt<11, ntt_le(11), ntt_first(11)>; __VA_ARGS__; } break;    \
    case 12: { using S = Ntt<12, ntt_le(12), ntt_first(12)>; __VA_ARGS__; } break;    \
    default: return hipErrorInvalidValue;                                             \
  }

static int ilog2(uint32_t N) {
  int l = 0;
  while ((1u << l) < N) ++l;
  return l;
}

// Allow a kernel more than the default 64 KiB of dynamic LDS (gfx950 has
// 160 KiB per workgroup).
template <typename K>
static hipError_t allow_lds(K kernel, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute((const void *)kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

#define ROSETTA_LAUNCH(KERNEL, GRID, BLOCK, LDS, ST, ...)                         \
  do {                                                                           \
    hipError_t e_ = allow_lds(KERNEL, LDS);                                      \
    if (e_ != hipSuccess) return e_;                                             \
    hipLaunchKernelGGL(KERNEL, GRID, BLOCK, LDS, ST, __VA_ARGS__);               \
  } while (0)

hipError_t launch_bsk_prepare(const uint64_t *bsk_std, uint64_t *bsk_dev,
                              const rosetta_params &p, const Tables &tb, hipStream_t st) {
  const size_t rows = (size_t)p.n * 2 * p.pbs_level * 2;
  ROSETTA_DISPATCH_N(ilog2(p.N), ROSETTA_LAUNCH(k_bsk_prepare<S>, dim3(rows), dim3(S::T),
                                                ntt_lds_bytes<S>(), st, bsk_std, bsk_dev,
                                                tb.zeta, tb.ninv));
  return hipGetLastError();
}

// Compute units of the current device (cached per device; 0 if unknown,
// which keeps every batch on the throughput instance).
static int device_cus() {
  static std::atomic<int> cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int c = cus[dev].load(std::memory_order_relaxed);
  if (!c) {
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) c = 0;
    cus[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

template <class S, int L>
static hipError_t launch_br_levels(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                                   const uint64_t *lut, uint64_t *out, size_t batch,
                                   const rosetta_params &p, const Tables &tb, int mode,
                                   int tp_glwe, hipStream_t st) {
  const int n = (int)p.n, beta = (int)p.pbs_base_log;
  const size_t lds = br_lds_bytes<S>(n);
#define ROSETTA_BR_INST(WV)                                                                    \
  do {                                                                                         \
    if (L * beta <= 30)                                                                        \
      ROSETTA_LAUNCH((k_blind_rotate<S, L, int32_t, WV>), dim3(batch), dim3(S::T), lds, st,    \
                     lwe_in, bsk_dev, lut, out, n, beta, mode, tp_glwe, tb.zeta,  \
                     tb.psi, tb.ninv);              \
    else                                                                                       \
      ROSETTA_LAUNCH((k_blind_rotate<S, L, int64_t, WV>), dim3(batch), dim3(S::T), lds, st,    \
                     lwe_in, bsk_dev, lut, out, n, beta, mode, tp_glwe, tb.zeta,  \
                     tb.psi, tb.ninv);              \
  } while (0)
  // At N = 4096 a batch that the CUs hold one workgroup each is latency,
  // not throughput: the instance compiled for two waves per SIMD (256
  // registers, no spills; same LDS and key layout) runs it
  if constexpr (S::LOGN >= 12) {
    if (batch <= (size_t)device_cus()) {
      ROSETTA_BR_INST(2);
      return hipSuccess;
    }
  }
  ROSETTA_BR_INST(br_waves_per_eu<S>());
#undef ROSETTA_BR_INST
  return hipSuccess;
}

hipError_t launch_blind_rotate(const uint64_t *lwe_in, const uint64_t *bsk_dev,
                               const uint64_t *lut, uint64_t *out, size_t batch,
                               const rosetta_params &p, const Tables &tb, BrMode mode,
                               int tp_glwe, hipStream_t st) {
  hipError_t e = hipSuccess;
  const int tpg = tp_glwe;
#define ROSETTA_BR_L(LV)                                                                       \
  case LV:                                                                                     \
    e = launch_br_levels<S, LV>(lwe_in, bsk_dev, lut, out, batch, p, tb, (int)mode, tpg, st); \
    break;
  ROSETTA_DISPATCH_N(ilog2(p.N), switch (p.pbs_level) {
    ROSETTA_BR_L(1) ROSETTA_BR_L(2) ROSETTA_BR_L(3) ROSETTA_BR_L(4)
    default: return hipErrorInvalidValue;
  });
#undef ROSETTA_BR_L
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

hipError_t launch_rows_prepare(const uint64_t *rows_std, uint64_t *rows_dev, size_t rows,
                               uint32_t N, const Tables &tb, hipStream_t st) {
  ROSETTA_DISPATCH_N(ilog2(N), ROSETTA_LAUNCH(k_bsk_prepare<S>, dim3(rows), dim3(S::T),
                                              ntt_lds_bytes<S>(), st, rows_std, rows_dev,
                                              tb.zeta, tb.ninv));
  return hipGetLastError();
}

hipError_t launch_trace(const uint64_t *in, const uint64_t *autk_dev, uint64_t *out,
                        size_t batch, uint32_t N, int level, int base_log, const Tables &tb,
                        hipStream_t st) {
#define ROSETTA_TR_L(LV)                                                                 \
  case LV:                                                                               \
    ROSETTA_LAUNCH((k_trace<S, LV>), dim3(batch), dim3(S::T), ntt_lds_bytes<S>(), st, in, \
                   autk_dev, out, base_log, tb.zeta, tb.ninv);                           \
    break;
  ROSETTA_DISPATCH_N(ilog2(N), switch (level) {
    ROSETTA_TR_L(1) ROSETTA_TR_L(2) ROSETTA_TR_L(3) ROSETTA_TR_L(4)
    default: return hipErrorInvalidValue;
  });
#undef ROSETTA_TR_L
  return hipGetLastError();
}

hipError_t launch_glwe_mul_plain(const uint64_t *in, const uint64_t *pa_dev, const uint64_t *pb,
                                 uint64_t *out, size_t batch, int npoly, uint32_t N,
                                 const Tables &tb, hipStream_t st) {
  ROSETTA_DISPATCH_N(ilog2(N), ROSETTA_LAUNCH(k_glwe_mul_plain<S>, dim3(batch), dim3(S::T),
                                              ntt_lds_bytes<S>(), st, in, pa_dev, pb, out,
                                              npoly, tb.zeta));
  return hipGetLastError();
}

static unsigned grid_of(size_t total) { return (unsigned)((total + 255) / 256); }

hipError_t launch_glwe_recombine(const uint64_t *in, uint64_t *out, size_t batch, int count,
                                 const Exponents &ex, uint32_t N, hipStream_t st) {
  hipLaunchKernelGGL(k_glwe_recombine, dim3(grid_of(batch * 2 * (size_t)N)), dim3(256), 0, st,
                     in, out, batch, count, ex, (int)N);
  return hipGetLastError();
}

hipError_t launch_glwe_monomial_mul(const uint64_t *in, uint64_t *out, size_t batch, int count,
                                    const Exponents &ex, uint32_t N, hipStream_t st) {
  hipLaunchKernelGGL(k_glwe_monomial_mul, dim3(grid_of(batch * count * 2 * (size_t)N)),
                     dim3(256), 0, st, in, out, batch, count, ex, (int)N);
  return hipGetLastError();
}

hipError_t launch_lwe_add_consts(const uint64_t *in, uint64_t *out, size_t batch, int count,
                                int dim, const Consts &cs, hipStream_t st) {
  hipLaunchKernelGGL(k_lwe_add_consts, dim3(grid_of(batch * count * (size_t)(dim + 1))),
                     dim3(256), 0, st, in, out, batch, count, dim, cs);
  return hipGetLastError();
}

hipError_t launch_lwe_sum_groups(const uint64_t *in, uint64_t *out, size_t batch, int count,
                                 int dim, uint64_t c0, hipStream_t st) {
  hipLaunchKernelGGL(k_lwe_sum_groups, dim3(grid_of(batch * (size_t)(dim + 1))), dim3(256), 0,
                     st, in, out, batch, count, dim, (u64)c0);
  return hipGetLastError();
}

hipError_t launch_sample_extract(const uint64_t *in, uint64_t *out, size_t batch, uint32_t N,
                                 hipStream_t st) {
  hipLaunchKernelGGL(k_sample_extract, dim3(grid_of(batch * (size_t)(N + 1))), dim3(256), 0, st,
                     in, out, batch, (int)N);
  return hipGetLastError();
}

hipError_t launch_ntt(const uint64_t *in, uint64_t *out, size_t count, uint32_t N,
                      const Tables &tb, bool inverse, hipStream_t st) {
  if (inverse) {
    ROSETTA_DISPATCH_N(ilog2(N), ROSETTA_LAUNCH(k_ntt_inverse<S>, dim3(count), dim3(S::T),
                                                ntt_lds_bytes<S>(), st, in, out, tb.zeta,
                                                tb.ninv));
  } else {
    ROSETTA_DISPATCH_N(ilog2(N), ROSETTA_LAUNCH(k_ntt_forward<S>, dim3(count), dim3(S::T),
                                                ntt_lds_bytes<S>(), st, in, out, tb.zeta));
  }
  return hipGetLastError();
}

hipError_t launch_poly_mul(const uint64_t *a, const uint64_t *b, uint64_t *c, size_t count,
                           uint32_t N, const Tables &tb, hipStream_t st) {
  ROSETTA_DISPATCH_N(ilog2(N), ROSETTA_LAUNCH(k_poly_mul<S>, dim3(count), dim3(S::T),
                                              ntt_lds_bytes<S>(), st, a, b, c, tb.zeta,
                                              tb.ninv));
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Elementwise field arithmetic (diagnostic entry point)
// ---------------------------------------------------------------------------

template <int OP>
__global__ void __launch_bounds__(256)
k_field_op(const u64 *__restrict__ a, const u64 *__restrict__ b, const u64 *__restrict__ c,
           u64 *__restrict__ out, size_t count) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= count) return;
  if constexpr (OP == ROSETTA_FIELD_ADD) {
    out[i] = gl_add(a[i], b[i]);
  } else if constexpr (OP == ROSETTA_FIELD_SUB) {
    out[i] = gl_sub(a[i], b[i]);
  } else if constexpr (OP == ROSETTA_FIELD_MUL) {
    out[i] = gl_mul(a[i], b[i]);
  } else if constexpr (OP == ROSETTA_FIELD_MUL_ADD) {
    out[i] = gl_mul_add(a[i], b[i], c[i]);
  } else if constexpr (OP == ROSETTA_FIELD_ADD_WEAK) {
    out[i] = gl_add_weak(a[i], b[i]);
  } else if constexpr (OP == ROSETTA_FIELD_MUL_ADD_WEAK) {
    out[i] = gl_mul_add_weak(a[i], b[i], c[i]);
  } else {
    out[i] = gl_mul_pow2<OP - ROSETTA_FIELD_MUL_POW2>(a[i]);
  }
}

// The decomposition's rounding of a at s, as the transform kernels compute
// it (the 32-bit high-word form from s = 34 up), sign-extended.
__global__ void __launch_bounds__(256)
k_field_round(const u64 *__restrict__ a, u64 *__restrict__ out, size_t count, int s) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= count) return;
  const i64 r = s >= 34 ? (i64)gl_round_top32(a[i], s) : gl_round_top(a[i], s);
  out[i] = (u64)r;
}

template <int E>
static hipError_t launch_field_pow2(int e, const u64 *a, u64 *out, size_t count, dim3 grid,
                                    hipStream_t st) {
  if constexpr (E < 96) {
    if (e != E) return launch_field_pow2<E + 1>(e, a, out, count, grid, st);
    hipLaunchKernelGGL(k_field_op<ROSETTA_FIELD_MUL_POW2 + E>, grid, dim3(256), 0, st, a,
                       nullptr, nullptr, out, count);
    return hipGetLastError();
  } else {
    return hipErrorInvalidValue;
  }
}

hipError_t launch_field_op(int op, const uint64_t *a, const uint64_t *b, const uint64_t *c,
                           uint64_t *out, size_t count, hipStream_t st) {
  const dim3 grid((unsigned)((count + 255) / 256));
  switch (op) {
    case ROSETTA_FIELD_ADD:
      hipLaunchKernelGGL(k_field_op<ROSETTA_FIELD_ADD>, grid, dim3(256), 0, st, a, b, c, out,
                         count);
      break;
    case ROSETTA_FIELD_SUB:
      hipLaunchKernelGGL(k_field_op<ROSETTA_FIELD_SUB>, grid, dim3(256), 0, st, a, b, c, out,
                         count);
      break;
    case ROSETTA_FIELD_MUL:
      hipLaunchKernelGGL(k_field_op<ROSETTA_FIELD_MUL>, grid, dim3(256), 0, st, a, b, c, out,
                         count);
      break;
    case ROSETTA_FIELD_MUL_ADD:
      hipLaunchKernelGGL(k_field_op<ROSETTA_FIELD_MUL_ADD>, grid, dim3(256), 0, st, a, b, c,
                         out, count);
      break;
    case ROSETTA_FIELD_ADD_WEAK:
      hipLaunchKernelGGL(k_field_op<ROSETTA_FIELD_ADD_WEAK>, grid, dim3(256), 0, st, a, b, c,
                         out, count);
      break;
    case ROSETTA_FIELD_MUL_ADD_WEAK:
      hipLaunchKernelGGL(k_field_op<ROSETTA_FIELD_MUL_ADD_WEAK>, grid, dim3(256), 0, st, a, b,
                         c, out, count);
      break;
    default:
      if (op > ROSETTA_FIELD_ROUND_TOP && op < ROSETTA_FIELD_ROUND_TOP + 64) {
        hipLaunchKernelGGL(k_field_round, grid, dim3(256), 0, st, a, out, count,
                           op - ROSETTA_FIELD_ROUND_TOP);
        break;
      }
      return launch_field_pow2<0>(op - ROSETTA_FIELD_MUL_POW2, a, out, count, grid, st);
  }
  return hipGetLastError();
}

// Eight independent product chains per thread, all in registers.
__global__ void __launch_bounds__(256)
k_modmul_chain(u64 seed, uint32_t threads, uint32_t iters, u64 *__restrict__ out) {
  const uint32_t t = blockIdx.x * 256 + threadIdx.x;
  if (t >= threads) return;
  u64 w = (seed ^ ((u64)t * 0x9E3779B97F4A7C15ull)) % GL_P;
  if (w < 2) w = 3;
  u64 x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = (seed + 8ull * t + j + 1) % GL_P;
  for (uint32_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = gl_mul(x[j], w);
  }
  u64 r = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) r ^= x[j];
  out[t] = r;
}

hipError_t launch_modmul_chain(uint64_t seed, uint32_t threads, uint32_t iters, uint64_t *out,
                               hipStream_t st) {
  hipLaunchKernelGGL(k_modmul_chain, dim3((threads + 255) / 256), dim3(256), 0, st, seed,
                     threads, iters, out);
  return hipGetLastError();
}

}  // namespace rosetta
