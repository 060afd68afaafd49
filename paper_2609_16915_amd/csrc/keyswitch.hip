// Key switching kernels (step a8) and the preparation of their key: the
// int8 matrix-core kernel for parameter sets whose digits fit a signed byte
// (ks_on_matrix_cores), the VALU kernel for the others.
//
// Kept apart from kernels.hip because they are compiled with the compiler's
// default instruction scheduling: both are streams of independent
// multiply-accumulates (matrix products, or 32x32-bit products into 64-bit
// accumulators), which the default occupancy-first schedule already
// interleaves, while the transform kernels are built with the ILP-first one.
#include <hip/hip_runtime.h>

#include "gl.hpp"
#include "internal.hpp"

namespace rosetta {

// Prepared key-switching key: the standard [N*l_ks][n+1] words followed by
// h * (sum over rows of column c), h = 2^(beta_ks - 1), for the offset-digit
// accumulation of k_keyswitch.
__global__ void k_ksk_colsum(const u64 *__restrict__ ksk, u64 *__restrict__ out, size_t rows,
                             int cols, u64 half) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= cols) return;
  u64 s = 0;
  for (size_t r = 0; r < rows; ++r) s = gl_add(s, ksk[r * cols + c]);
  out[c] = gl_mul(s, half);
}

// ---------------------------------------------------------------------------
// Key switching
// ---------------------------------------------------------------------------

// out[b][c] = (c == n ? b'_b : 0) - sum_{j,t} d_{b,j,t} KSK[j][t][c].
// A workgroup covers KS_BT ciphertexts x 256 output columns.  Digits are
// produced in LDS per chunk of KS_JC input coefficients in offset form
// d + h in [0, 2h] (h = 2^(beta_ks-1)); the offset is removed at the end
// with the column sums stored after the key (k_ksk_colsum).  Sums of
// offset digit x 32-bit half-word products stay below N l_ks 2^beta_ks
// 2^32 < 2^64, so the two 64-bit accumulators per output never wrap.
constexpr int KS_BT = 16;
constexpr int KS_JC = 32;
constexpr int KS_TPB = 256;

template <int LKS>
__global__ void __launch_bounds__(KS_TPB)
k_keyswitch(const u64 *__restrict__ big, const u64 *__restrict__ ksk, u64 *__restrict__ out,
            size_t batch, int n, int N, int beta) {
  __shared__ u32 dig[KS_JC][LKS][KS_BT];
  __shared__ u64 body[KS_BT];
  const int tid = threadIdx.x;
  const int c = blockIdx.y * KS_TPB + tid;
  const size_t b0 = (size_t)blockIdx.x * KS_BT;
  const int cols = n + 1;
  const int s = 64 - LKS * beta;
  const i64 h = (i64)1 << (beta - 1);
  const i64 mask = ((i64)1 << beta) - 1;

  u64 acc_lo[KS_BT], acc_hi[KS_BT];
#pragma unroll
  for (int b = 0; b < KS_BT; ++b) acc_lo[b] = acc_hi[b] = 0;
  if (tid < KS_BT) body[tid] = (b0 + tid < batch) ? big[(b0 + tid) * (size_t)(N + 1) + N] : 0;

  for (int j0 = 0; j0 < N; j0 += KS_JC) {
    __syncthreads();
    for (int e = tid; e < KS_BT * KS_JC; e += KS_TPB) {
      const int bb = e / KS_JC, jj = e % KS_JC;
      const size_t q = b0 + bb;
      const u64 a = q < batch ? big[q * (size_t)(N + 1) + j0 + jj] : 0;
      i64 r = gl_round_top(a, s);
#pragma unroll
      for (int t = LKS - 1; t >= 1; --t) {
        const i64 d = ((r + h) & mask) - h;
        r = (r - d) >> beta;
        dig[jj][t][bb] = (u32)(d + h);
      }
      dig[jj][0][bb] = (u32)(r + h);
    }
    __syncthreads();
    if (c < cols) {
      const u64 *kp = ksk + (size_t)j0 * LKS * cols + c;
#pragma unroll 4
      for (int jj = 0; jj < KS_JC; ++jj) {
#pragma unroll
        for (int t = 0; t < LKS; ++t) {
          const u64 w = kp[(size_t)(jj * LKS + t) * cols];
          const u32 wl = (u32)w, wh = (u32)(w >> 32);
#pragma unroll
          for (int b = 0; b < KS_BT; ++b) {
            const u32 d = dig[jj][t][b];
            acc_lo[b] += (u64)d * wl;
            acc_hi[b] += (u64)d * wh;
          }
        }
      }
    }
  }
  if (c < cols) {
    const u64 hc = ksk[(size_t)N * LKS * cols + c];
#pragma unroll
    for (int b = 0; b < KS_BT; ++b) {
      const size_t q = b0 + b;
      if (q >= batch) break;
      u64 lo = acc_lo[b] + (acc_hi[b] << 32);
      const u64 hi = (acc_hi[b] >> 32) + (lo < acc_lo[b] ? 1 : 0);
      const u64 sum = gl_reduce128(lo, hi);
      u64 r = gl_sub(c == n ? body[b] : 0, sum);
      out[q * (size_t)cols + c] = gl_add(r, hc);
    }
  }
}

// ---------------------------------------------------------------------------
// Key switching on the int8 matrix cores
// ---------------------------------------------------------------------------

// Over a batch the key switch is one integer matrix product: digits
// D[b][kappa] (batch x N l_ks) times key K[kappa][c] ((N l_ks) x (n+1)),
// kappa = t N + j for digit level t of input coefficient j (any order of
// the contraction index gives the same sum).  Each key word K in [0, p) is
// replaced by V = K or K - p, whichever lies in the range of 8 balanced
// base-256 digits [-128 S, 127 S], S = (2^64 - 1) / 255; V = sum_m 256^m k_m
// with k_m in [-128, 127], so D K = sum_m 256^m (D k_m) (mod p) with eight
// exact int8 x int8 -> int32 products.  X = V + 128 S lies in [0, 2^64) and
// its plain base-256 digits are k_m + 128, so byte m of X with its top bit
// flipped is k_m as a signed byte; X is K + 128 S, plus 2^32 - 1 (= -p mod
// 2^64) when V = K - p.
//
// Byte-plane layout, in 8-byte words: word ((cb KB + kb) 8 + m) 128
// + 2 lane + cc holds, in byte i, k_m[kappa][c] with kappa = 32 kb +
// 8 (lane / 16) + i and c = 32 cb + 16 cc + lane % 16 (0 past the last
// column): the B operand of a 16 x 16 x 32 int8 product (lane l supplies
// rows 8 (l / 16) .. + 7 of column l % 16) for column tile cc of column
// block cb, plane m, k block kb (KB = N l_ks / 32 of them).  The 1024
// words of one (cb, kb) are contiguous, and a lane's two column tiles are
// adjacent.
constexpr u64 KS_S128 = 0x8080808080808080ull;   // 128 S
constexpr u64 KS_S127 = 0x7F7F7F7F7F7F7F7Full;   // 127 S

__global__ void k_ksk_planes(const u64 *__restrict__ ksk, u64 *__restrict__ planes, int N,
                             int lks, int cols, size_t words) {
  const size_t w = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (w >= words) return;
  const int cc = (int)(w & 1), lane = (int)((w >> 1) & 63), m = (int)((w >> 7) & 7);
  const size_t blk = w >> 10;              // cb KB + kb
  const size_t KB = (size_t)N * lks / 32;
  const int kb = (int)(blk % KB), cb = (int)(blk / KB);
  const int c = 32 * cb + 16 * cc + lane % 16;
  u64 word = 0;
  for (int i = 0; i < 8; ++i) {
    const int kappa = 32 * kb + 8 * (lane / 16) + i;
    const int t = kappa / N, j = kappa % N;
    const u64 K = c < cols ? ksk[((size_t)j * lks + t) * cols + c] : 0;
    const u64 X = K + KS_S128 + (K <= KS_S127 ? 0 : GL_EPS);
    word |= (((X >> (8 * m)) & 0xFF) ^ 0x80) << (8 * i);
  }
  planes[w] = word;
}

typedef int32_t ks_v4i __attribute__((ext_vector_type(4)));

// out[b][c] = (c == n ? b'_b : 0) - sum_kappa D[b][kappa] K[kappa][c].
// Workgroup = 4 waves on one 32-column block, each wave on its own 32
// ciphertexts: two 16-ciphertext row tiles x two 16-column tiles x 8 byte
// planes of int32 accumulators.  The contraction runs over k blocks in the
// order (32-coefficient chunk, level from the bottom); the workgroup
// stages each k block's 8 KB of key fragments in LDS (double-buffered, one
// barrier per k block, the next block's global loads in flight during the
// current one's products), so the key is fetched once per 128 ciphertexts.
// At a chunk's first level a lane rounds its 8 coefficients of each row
// tile (loaded one chunk ahead) and issues the next chunk's loads; every
// level peels one balanced digit from the bottom (the A operand of level
// t: row l % 16, coefficients 8 (l / 16) .. + 7) and issues 32 products.
// The planes are recombined exactly: with |acc| < 2^31, lo = sum_{m<4}
// 256^m acc_m and hi = sum_{m>=4} 256^(m-4) acc_m are below 2^56 in
// magnitude, and the sum is lo + 2^32 hi mod p.  A wave with no
// ciphertexts still takes part in the staging and the barriers.
//
// Two waves per SIMD: the register cap of 256 holds the 128 accumulators,
// the key fragments and the prefetched coefficients without spills (left
// to itself the compiler takes 256 + 128 registers and one wave).
constexpr int KSM_WAVES = 4;

template <int LKS>
__global__ void __launch_bounds__(64 * KSM_WAVES) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_keyswitch_mfma(const u64 *__restrict__ big, const u64 *__restrict__ planes,
                 u64 *__restrict__ out, size_t batch, int n, int N, int beta) {
  __shared__ __attribute__((aligned(16))) u64 kbuf[2][1024];
  const int tid = threadIdx.x;
  const int wv = tid >> 6, l = tid & 63;
  const int cb = blockIdx.y;
  const int cols = n + 1;
  const size_t b0 = ((size_t)blockIdx.x * KSM_WAVES + wv) * 32;
  const bool active = b0 < batch;
  const int s = 64 - LKS * beta;
  const int32_t h = 1 << (beta - 1), mask = (1 << beta) - 1;
  const int NB = N / 32, KB = NB * LKS;
  // this thread's 32 bytes of each k block's 8 KB
  const ulonglong2 *gsrc = (const ulonglong2 *)(planes + (size_t)cb * KB * 1024) + 2 * tid;

  const u64 *arow[2];
  bool aok[2];
#pragma unroll
  for (int bt = 0; bt < 2; ++bt) {
    const size_t q = b0 + 16 * bt + (l & 15);
    aok[bt] = q < batch;
    arow[bt] = big + (aok[bt] ? q : 0) * (size_t)(N + 1) + 8 * (l >> 4);
  }
  ks_v4i acc[2][2][8];
#pragma unroll
  for (int bt = 0; bt < 2; ++bt)
#pragma unroll
    for (int cc = 0; cc < 2; ++cc)
#pragma unroll
      for (int m = 0; m < 8; ++m) acc[bt][cc][m] = ks_v4i{0, 0, 0, 0};

  {
    const ulonglong2 g0 = gsrc[(size_t)(LKS - 1) * NB * 512], g1 = gsrc[(size_t)(LKS - 1) * NB * 512 + 1];
    ((ulonglong2 *)kbuf[0])[2 * tid] = g0;
    ((ulonglong2 *)kbuf[0])[2 * tid + 1] = g1;
  }
  __syncthreads();

  // raw coefficients of the next chunk, loaded a whole chunk (l_ks k
  // blocks) before they are rounded
  u64 cn[2][8];
#pragma unroll
  for (int bt = 0; bt < 2; ++bt)
#pragma unroll
    for (int i = 0; i < 8; ++i) cn[bt][i] = (active && aok[bt]) ? arow[bt][i] : 0;
  int32_t r[2][8];
  const int total = NB * LKS;
#pragma unroll 1
  for (int it = 0; it < total; ++it) {
    const int jb = it / LKS, t = LKS - 1 - (it - jb * LKS);
    // next k block: (jb, t - 1), or (jb + 1, LKS - 1)
    ulonglong2 p0, p1;
    const bool more = it + 1 < total;
    if (more) {
      const int kn = t > 0 ? (t - 1) * NB + jb : (LKS - 1) * NB + jb + 1;
      p0 = gsrc[(size_t)kn * 512];
      p1 = gsrc[(size_t)kn * 512 + 1];
    }
    if (active) {
      if (t == LKS - 1) {
#pragma unroll
        for (int bt = 0; bt < 2; ++bt)
#pragma unroll
          for (int i = 0; i < 8; ++i) r[bt][i] = gl_round_top32(cn[bt][i], s);
        if (jb + 1 < NB) {
#pragma unroll
          for (int bt = 0; bt < 2; ++bt)
#pragma unroll
            for (int i = 0; i < 8; ++i) cn[bt][i] = aok[bt] ? arow[bt][32 * (jb + 1) + i] : 0;
        }
      }
      long a[2];
#pragma unroll
      for (int bt = 0; bt < 2; ++bt) {
        u32 w0 = 0, w1 = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          int32_t d = r[bt][i];
          if (t > 0) {
            d = ((d + h) & mask) - h;
            r[bt][i] = (r[bt][i] - d) >> beta;
          }
          const u32 byte = (u32)d & 0xFFu;
          if (i < 4) w0 |= byte << (8 * i);
          else w1 |= byte << (8 * (i - 4));
        }
        a[bt] = (long)gl_mk(w0, w1);
      }
      const ulonglong2 *kb2 = (const ulonglong2 *)kbuf[it & 1] + l;
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        const ulonglong2 f = kb2[64 * m];
#pragma unroll
        for (int bt = 0; bt < 2; ++bt) {
          acc[bt][0][m] = __builtin_amdgcn_mfma_i32_16x16x32_i8(a[bt], (long)f.x, acc[bt][0][m], 0, 0, 0);
          acc[bt][1][m] = __builtin_amdgcn_mfma_i32_16x16x32_i8(a[bt], (long)f.y, acc[bt][1][m], 0, 0, 0);
        }
      }
    }
    if (more) {
      ((ulonglong2 *)kbuf[(it + 1) & 1])[2 * tid] = p0;
      ((ulonglong2 *)kbuf[(it + 1) & 1])[2 * tid + 1] = p1;
    }
    __syncthreads();
  }
  if (!active) return;

#pragma unroll
  for (int bt = 0; bt < 2; ++bt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const size_t q = b0 + 16 * bt + 4 * (l >> 4) + i;
      if (q >= batch) continue;
      const u64 body = big[q * (size_t)(N + 1) + N];
#pragma unroll
      for (int cc = 0; cc < 2; ++cc) {
        const int c = 32 * cb + 16 * cc + (l & 15);
        if (c >= cols) continue;
        int64_t lo = 0, hi = 0;
#pragma unroll
        for (int m = 3; m >= 0; --m) {
          lo = lo * 256 + acc[bt][cc][m][i];
          hi = hi * 256 + acc[bt][cc][m + 4][i];
        }
        const u64 lop = (u64)lo + (lo < 0 ? GL_P : 0);
        const u64 hi_p = (u64)hi + (hi < 0 ? GL_P : 0);
        const u64 sum = gl_add(lop, gl_mul_pow2<32>(hi_p));
        out[q * (size_t)cols + c] = gl_sub(c == n ? body : 0, sum);
      }
    }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

hipError_t launch_ksk_prepare(const uint64_t *ksk_std, uint64_t *ksk_dev,
                              const rosetta_params &p, hipStream_t st) {
  const size_t rows = (size_t)p.N * p.ks_level;
  const int cols = (int)p.n + 1;
  if (ks_on_matrix_cores(p)) {
    const size_t words = ks_matrix_key_words(p);
    hipLaunchKernelGGL(k_ksk_planes, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, st,
                       ksk_std, ksk_dev, (int)p.N, (int)p.ks_level, cols, words);
    return hipGetLastError();
  }
  hipError_t e = hipMemcpyAsync(ksk_dev, ksk_std, rows * cols * sizeof(u64),
                                hipMemcpyDeviceToDevice, st);
  if (e != hipSuccess) return e;
  const u64 half = 1ull << (p.ks_base_log - 1);
  hipLaunchKernelGGL(k_ksk_colsum, dim3((cols + 255) / 256), dim3(256), 0, st, ksk_std,
                     ksk_dev + rows * cols, rows, cols, half);
  return hipGetLastError();
}

hipError_t launch_keyswitch(const uint64_t *big, const uint64_t *ksk_dev, uint64_t *out,
                            size_t batch, const rosetta_params &p, hipStream_t st) {
  if (ks_on_matrix_cores(p)) {
    const dim3 grid((unsigned)((batch + 32 * KSM_WAVES - 1) / (32 * KSM_WAVES)),
                    (p.n + 1 + 31) / 32);
    const int n = (int)p.n, N = (int)p.N, beta = (int)p.ks_base_log;
#define ROSETTA_KSM_CASE(LK)                                                               \
  case LK:                                                                                 \
    hipLaunchKernelGGL(k_keyswitch_mfma<LK>, grid, dim3(64 * KSM_WAVES), 0, st, big, ksk_dev, \
                       out, batch, n, N, beta);                                            \
    break;
    switch (p.ks_level) {
      ROSETTA_KSM_CASE(1)
      ROSETTA_KSM_CASE(2)
      ROSETTA_KSM_CASE(3)
      ROSETTA_KSM_CASE(4)
      ROSETTA_KSM_CASE(5)
      ROSETTA_KSM_CASE(6)
      ROSETTA_KSM_CASE(7)
      ROSETTA_KSM_CASE(8)
      default:
        return hipErrorInvalidValue;
    }
#undef ROSETTA_KSM_CASE
    return hipGetLastError();
  }
  const dim3 grid((unsigned)((batch + KS_BT - 1) / KS_BT), (p.n + 1 + KS_TPB - 1) / KS_TPB);
  const int n = (int)p.n, N = (int)p.N, beta = (int)p.ks_base_log;
#define ROSETTA_KS_CASE(LK)                                                                 \
  case LK:                                                                                  \
    hipLaunchKernelGGL(k_keyswitch<LK>, grid, dim3(KS_TPB), 0, st, big, ksk_dev, out, batch, \
                       n, N, beta);                                                         \
    break;
  switch (p.ks_level) {
    ROSETTA_KS_CASE(1)
    ROSETTA_KS_CASE(2)
    ROSETTA_KS_CASE(3)
    ROSETTA_KS_CASE(4)
    ROSETTA_KS_CASE(5)
    ROSETTA_KS_CASE(6)
    ROSETTA_KS_CASE(7)
    ROSETTA_KS_CASE(8)
    default:
      return hipErrorInvalidValue;
  }
#undef ROSETTA_KS_CASE
  return hipGetLastError();
}

}  // namespace rosetta
