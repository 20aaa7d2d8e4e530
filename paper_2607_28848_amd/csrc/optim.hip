// optim.hip -- fused AdamW step of the training adapters (the optimizer
// update that follows the LoRA backward, Sec. 3.2 "Backward subprocess";
// AdamW with decoupled weight decay, Sec. 4.1 training configuration).
//
// Per parameter element (fp32 master p, moments m and v, gradient g, step t):
//   p <- p (1 - lr wd)
//   m <- b1 m + (1 - b1) g,   v <- b2 v + (1 - b2) g^2
//   p <- p - (lr / (1 - b1^t)) m / (sqrt(v) / sqrt(1 - b2^t) + eps)
// and the parameter copy the forward reads is p rounded once (bf16: to
// nearest even).  Elementwise and HBM-bound: 4 B of gradient, 12 B of state
// read and 12 B written, plus the copy, per element.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "plan.h"

namespace dsv {
namespace {

__device__ __forceinline__ uint16_t f2bf_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rounded = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  const uint32_t quiet = (u >> 16) | 0x40u;
  return (uint16_t)(((u & 0x7fffffffu) > 0x7f800000u) ? quiet : rounded);
}

__device__ __forceinline__ void adamw_one(const AdamWArgs& a, float g, float& p, float& m, float& v) {
  p *= a.decay;
  m = a.b1 * m + a.c1 * g;
  v = a.b2 * v + a.c2 * g * g;
  p -= a.step_size * m / (sqrtf(v) / a.sqrt_bc2 + a.eps);
}

// blockIdx.y: training adapter; x: 256-thread blocks over the adapter's A part
// (r_a rows of K, contiguous: 4 elements per thread) then its B part (N rows of
// r_a entries with stride r_max: 1 element per thread).
__global__ __launch_bounds__(256) void adamw_kernel(AdamWArgs a) {
  const int ad = a.train_ads[blockIdx.y];
  const int r = a.ranks[ad];
  const int64_t nA4 = (int64_t)r * a.K / 4, nB = (int64_t)a.N * r;
  const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (u < nA4) {
    const int64_t e = (int64_t)ad * a.r_max * a.K + 4 * u;  // rows j < r are contiguous
    const float4 g = *reinterpret_cast<const float4*>(a.dA + e);
    float4 p = *reinterpret_cast<const float4*>(a.pA + e);
    float4 m = *reinterpret_cast<const float4*>(a.mA + e);
    float4 v = *reinterpret_cast<const float4*>(a.vA + e);
    adamw_one(a, g.x, p.x, m.x, v.x);
    adamw_one(a, g.y, p.y, m.y, v.y);
    adamw_one(a, g.z, p.z, m.z, v.z);
    adamw_one(a, g.w, p.w, m.w, v.w);
    *reinterpret_cast<float4*>(a.pA + e) = p;
    *reinterpret_cast<float4*>(a.mA + e) = m;
    *reinterpret_cast<float4*>(a.vA + e) = v;
    if (a.A && a.bf16) {
      const uint32_t lo = (uint32_t)f2bf_rne(p.x) | ((uint32_t)f2bf_rne(p.y) << 16);
      const uint32_t hi = (uint32_t)f2bf_rne(p.z) | ((uint32_t)f2bf_rne(p.w) << 16);
      *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.A) + e) = make_uint2(lo, hi);
    } else if (a.A) {
      *reinterpret_cast<float4*>(static_cast<float*>(a.A) + e) = p;
    }
  } else if (u - nA4 < nB) {
    const int64_t q = u - nA4, n = q / r, j = q - n * r;
    const int64_t e = (int64_t)ad * a.N * a.r_max + n * a.r_max + j;
    float p = a.pB[e], m = a.mB[e], v = a.vB[e];
    adamw_one(a, a.dB[e], p, m, v);
    a.pB[e] = p;
    a.mB[e] = m;
    a.vB[e] = v;
    if (a.B && a.bf16) static_cast<uint16_t*>(a.B)[e] = f2bf_rne(p);
    else if (a.B) static_cast<float*>(a.B)[e] = p;
  }
}

}  // namespace

hipError_t launch_adamw(const AdamWArgs& a, int32_t n_tads, hipStream_t s) {
  if (n_tads <= 0) return hipSuccess;
  // blocks enough for the largest rank (r_max); threads past an adapter's count exit
  const int64_t units = (int64_t)a.r_max * a.K / 4 + (int64_t)a.N * a.r_max;
  hipLaunchKernelGGL(adamw_kernel, dim3((unsigned)((units + 255) / 256), (unsigned)n_tads), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dsv
