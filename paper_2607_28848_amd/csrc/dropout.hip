// dropout.hip -- LoRA dropout on the adapter input of the training rows
// (Sec. 4.1 trains the adapter with dropout 0.05; inference rows run without).
//
// Masks come from Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel
// random numbers: as easy as 1, 2, 3", SC 2011), a counter-based generator,
// so any element's draw is recomputable: element (i, k) of compact training
// row i and input column k takes output word k % 4 of the generator at
// counter (k / 4, i, offset low, offset high) and key (seed low, seed high),
// and is dropped when that word is below floor(p * 2^32).  The kept elements
// are scaled by 1 / (1 - p) (inverted dropout); the scale is applied to fp32
// sums, so the bf16 inputs enter the matrix cores unrounded.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "plan.h"

namespace dsv {
namespace {

__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
  constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;  // round multipliers
  constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;  // key increments
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += W0;
      k1 += W1;
    }
    const uint64_t p0 = (uint64_t)M0 * c[0], p1 = (uint64_t)M1 * c[2];
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
}

// One 32-bit word of the kept-element bitmask per thread: bit b of word w of
// row i keeps column 32 w + b.
__global__ __launch_bounds__(256) void dropout_mask_kernel(uint32_t* __restrict__ bits, int32_t Tt,
                                                           int32_t words, uint32_t thr, uint32_t s0, uint32_t s1,
                                                           uint32_t o0, uint32_t o1) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)Tt * words) return;
  const uint32_t i = (uint32_t)(idx / words), w = (uint32_t)(idx % words);
  uint32_t m = 0;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    uint32_t c[4] = {8u * w + (uint32_t)q, i, o0, o1};
    philox4x32_10(c, s0, s1);
#pragma unroll
    for (int e = 0; e < 4; ++e) m |= (c[e] >= thr ? 1u : 0u) << (4 * q + e);
  }
  bits[idx] = m;
}

}  // namespace

hipError_t launch_dropout_mask(uint32_t* bits, int32_t Tt, int32_t K, const DropoutSpec& d, hipStream_t s) {
  if (Tt <= 0) return hipSuccess;
  const int32_t words = (K + 31) / 32;
  const int64_t n = (int64_t)Tt * words;
  hipLaunchKernelGGL(dropout_mask_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, bits, Tt, words,
                     d.thr, (uint32_t)d.seed, (uint32_t)(d.seed >> 32), (uint32_t)d.offset,
                     (uint32_t)(d.offset >> 32));
  return hipGetLastError();
}

}  // namespace dsv
