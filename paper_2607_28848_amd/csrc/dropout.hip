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
    const uint32_t hi0 = __umulhi(M0, c[0]), lo0 = M0 * c[0];
    const uint32_t hi1 = __umulhi(M1, c[2]), lo1 = M1 * c[2];
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

// Low-rank term of dX under dropout (bf16 path): for compact training row i,
// delta[i][k] = scale * keep(i, k) * sum_j g[i][j] A_a[j][k], fp32, added to
// dy W in the dX GEMM's epilogue.  8 columns per thread.
__global__ __launch_bounds__(256) void dropout_dx_low_kernel(DropoutDxArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int kb = a.K / 8;
  if (idx >= (int64_t)a.Tt * kb) return;
  const int i = (int)(idx / kb), k0 = 8 * (int)(idx % kb);
  const int ad = a.train_adapter[i], r = a.ranks[ad];
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const uint16_t* gi = a.G + (int64_t)i * a.ldg;
  const uint16_t* Aa = a.A + (int64_t)ad * a.r_max * a.K + k0;
  for (int j = 0; j < r; ++j) {
    const float gj = __uint_as_float((uint32_t)gi[j] << 16);
    const uint4 v = *reinterpret_cast<const uint4*>(Aa + (int64_t)j * a.K);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] = fmaf(gj, __uint_as_float(w[e] << 16), acc[2 * e]);
      acc[2 * e + 1] = fmaf(gj, __uint_as_float(w[e] & 0xffff0000u), acc[2 * e + 1]);
    }
  }
  const uint32_t m = (a.keep[(int64_t)i * a.keep_words + (k0 >> 5)] >> (k0 & 31)) & 0xffu;
  float* out = a.delta + (int64_t)i * a.K + k0;
  float4 lo, hi;
  lo.x = (m & 1u) ? a.scale * acc[0] : 0.f;
  lo.y = (m & 2u) ? a.scale * acc[1] : 0.f;
  lo.z = (m & 4u) ? a.scale * acc[2] : 0.f;
  lo.w = (m & 8u) ? a.scale * acc[3] : 0.f;
  hi.x = (m & 16u) ? a.scale * acc[4] : 0.f;
  hi.y = (m & 32u) ? a.scale * acc[5] : 0.f;
  hi.z = (m & 64u) ? a.scale * acc[6] : 0.f;
  hi.w = (m & 128u) ? a.scale * acc[7] : 0.f;
  *reinterpret_cast<float4*>(out) = lo;
  *reinterpret_cast<float4*>(out + 4) = hi;
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

hipError_t launch_dropout_dx_low(const DropoutDxArgs& a, hipStream_t s) {
  if (a.Tt <= 0) return hipSuccess;
  const int64_t n = (int64_t)a.Tt * (a.K / 8);
  hipLaunchKernelGGL(dropout_dx_low_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dsv
