// Key switching kernels (step a8) and the preparation of their key.
//
// Kept apart from kernels.hip because they are compiled with the compiler's
// default instruction scheduling: the key switch is a stream of independent
// 32x32-bit multiply-accumulates into 64-bit accumulators, which the
// default occupancy-first schedule already interleaves, while the transform
// kernels are built with the ILP-first one.
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
// Launchers
// ---------------------------------------------------------------------------

hipError_t launch_ksk_prepare(const uint64_t *ksk_std, uint64_t *ksk_dev,
                              const rosetta_params &p, hipStream_t st) {
  const size_t rows = (size_t)p.N * p.ks_level;
  const int cols = (int)p.n + 1;
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
