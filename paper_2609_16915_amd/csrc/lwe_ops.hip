// Word-by-word linear combinations of LWE arrays (the scaling and
// subtractions of the refined comparison in Step 1 of the lookup).  The work
// is a few words per ciphertext, bound by memory traffic: one coalesced
// pass, each thread one word.
#include <hip/hip_runtime.h>

#include "gl.hpp"
#include "internal.hpp"

namespace rosetta {

// out[i] = alpha a[i] + beta b[i] + gamma c[i] mod p (b, c optional); each
// term a product reduced mod p, the sum kept canonical.
__global__ void __launch_bounds__(256)
k_lwe_combine(const u64 *a, u64 alpha, const u64 *b, u64 beta, const u64 *c, u64 gamma,
              u64 *out, size_t words) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= words) return;
  u64 v = gl_mul(a[i], alpha);
  if (b) v = gl_add(v, gl_mul(b[i], beta));
  if (c) v = gl_add(v, gl_mul(c[i], gamma));
  out[i] = v;
}

hipError_t launch_lwe_combine(const uint64_t *a, uint64_t alpha, const uint64_t *b, uint64_t beta,
                              const uint64_t *c, uint64_t gamma, uint64_t *out, size_t words,
                              hipStream_t st) {
  hipLaunchKernelGGL(k_lwe_combine, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, st, a,
                     alpha, b, beta, c, gamma, out, words);
  return hipGetLastError();
}

}  // namespace rosetta
