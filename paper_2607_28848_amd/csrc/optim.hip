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

__device__ __forceinline__ void adamw4(const AdamWArgs& a, float4 g, float4& p, float4& m, float4& v) {
  adamw_one(a, g.x, p.x, m.x, v.x);
  adamw_one(a, g.y, p.y, m.y, v.y);
  adamw_one(a, g.z, p.z, m.z, v.z);
  adamw_one(a, g.w, p.w, m.w, v.w);
}

// One float4 unit at element e of a slice: gradient, master and moments read,
// master and moments written, the rounded copy written (if any).
__device__ __forceinline__ void unit4(const AdamWArgs& a, int64_t e, const float* dg, float* pm, float* mm,
                                      float* vm, void* copy) {
  const float4 g = *reinterpret_cast<const float4*>(dg + e);
  float4 p = *reinterpret_cast<const float4*>(pm + e);
  float4 m = *reinterpret_cast<const float4*>(mm + e);
  float4 v = *reinterpret_cast<const float4*>(vm + e);
  adamw4(a, g, p, m, v);
  *reinterpret_cast<float4*>(pm + e) = p;
  *reinterpret_cast<float4*>(mm + e) = m;
  *reinterpret_cast<float4*>(vm + e) = v;
  if (copy && a.bf16) {
    const uint32_t lo = (uint32_t)f2bf_rne(p.x) | ((uint32_t)f2bf_rne(p.y) << 16);
    const uint32_t hi = (uint32_t)f2bf_rne(p.z) | ((uint32_t)f2bf_rne(p.w) << 16);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(copy) + e) = make_uint2(lo, hi);
  } else if (copy) {
    *reinterpret_cast<float4*>(static_cast<float*>(copy) + e) = p;
  }
}

// One block: 256 units of one (projection, training adapter) pair.  The
// projection is found from the block index (blk_begin ascending), then the
// adapter slot and the block's place inside the adapter's A-then-B units.
__global__ __launch_bounds__(256) void adamw_kernel(AdamWArgs a) {
  const int32_t bid = (int32_t)blockIdx.x;
  int p = 0;
#pragma unroll
  for (int q = 1; q < kMaxGroup; ++q)
    if (q < a.n_proj && bid >= a.proj[q].blk_begin) p = q;
  const AdamWProj& P = a.proj[p];
  // the host keeps every per-adapter unit count below 2^31: 32-bit index math
  const uint32_t local = (uint32_t)(bid - P.blk_begin);
  const uint32_t slot = local / (uint32_t)P.bpa;
  const int ad = a.train_ads[slot];
  const uint32_t r = (uint32_t)a.ranks[ad];
  const uint32_t nA4 = r * ((uint32_t)P.K / 4u);
  const uint32_t u = (local - slot * (uint32_t)P.bpa) * 256u + threadIdx.x;
  if (u < nA4) {
    // rows j < r of the adapter's A slice are contiguous
    unit4(a, (int64_t)ad * a.r_max * P.K + 4 * (int64_t)u, P.dA, P.pA, P.mA, P.vA, P.A);
    return;
  }
  const uint32_t q = u - nA4;
  const int64_t base = (int64_t)ad * P.N * a.r_max;
  if (a.bvec) {
    // B row n holds entries j < r at n * r_max + j; r and r_max multiples of 4
    const uint32_t r4 = r >> 2;
    if (q < (uint32_t)P.N * r4) {
      const uint32_t n = q / r4, j4 = q - n * r4;
      unit4(a, base + (int64_t)n * a.r_max + 4 * j4, P.dB, P.pB, P.mB, P.vB, P.B);
    }
  } else if (q < (uint32_t)P.N * r) {
    const uint32_t n = q / r, j = q - n * r;
    const int64_t e = base + (int64_t)n * a.r_max + j;
    float pv = P.pB[e], m = P.mB[e], v = P.vB[e];
    adamw_one(a, P.dB[e], pv, m, v);
    P.pB[e] = pv;
    P.mB[e] = m;
    P.vB[e] = v;
    if (P.B && a.bf16) static_cast<uint16_t*>(P.B)[e] = f2bf_rne(pv);
    else if (P.B) static_cast<float*>(P.B)[e] = pv;
  }
}

}  // namespace

hipError_t launch_adamw(const AdamWArgs& a, int64_t n_blocks, hipStream_t s) {
  if (n_blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL(adamw_kernel, dim3((unsigned)n_blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dsv
