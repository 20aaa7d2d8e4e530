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
// row i keeps column 32 w + b.  The grid covers every projection of the group
// back to back, each in whole workgroups (entry p owns workgroups
// [blk[p], blk[p + 1])), so the entry is the same for a whole workgroup.
struct MaskLaunch {
  uint32_t* bits[kMaxGroup];
  int32_t words[kMaxGroup];
  uint32_t thr[kMaxGroup], s0[kMaxGroup], s1[kMaxGroup], o0[kMaxGroup], o1[kMaxGroup];
  int64_t total[kMaxGroup];  // Tt * words
  int32_t blk[kMaxGroup + 1];
  int32_t n;
};

__global__ __launch_bounds__(256) void dropout_mask_kernel(MaskLaunch L) {
  int p = 0;
  while (p + 1 < L.n && (int32_t)blockIdx.x >= L.blk[p + 1]) ++p;
  const int64_t loc = (int64_t)((int32_t)blockIdx.x - L.blk[p]) * 256 + threadIdx.x;
  if (loc >= L.total[p]) return;
  const uint32_t words = (uint32_t)L.words[p];
  const uint32_t i = (uint32_t)(loc / words), w = (uint32_t)(loc % words);
  uint32_t m = 0;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    uint32_t c[4] = {8u * w + (uint32_t)q, i, L.o0[p], L.o1[p]};
    philox4x32_10(c, L.s0[p], L.s1[p]);
#pragma unroll
    for (int e = 0; e < 4; ++e) m |= (c[e] >= L.thr[p] ? 1u : 0u) << (4 * q + e);
  }
  L.bits[p][loc] = m;
}

}  // namespace

hipError_t launch_dropout_mask_group(const DropoutMaskGroup& g, int32_t Tt, hipStream_t s) {
  if (Tt <= 0 || g.n <= 0) return hipSuccess;
  if (g.n > kMaxGroup) return hipErrorInvalidValue;
  MaskLaunch L{};
  for (int p = 0; p < g.n; ++p) {
    if (!g.bits[p]) continue;
    const int q = L.n++;
    L.bits[q] = g.bits[p];
    L.words[q] = (g.K[p] + 31) / 32;
    L.thr[q] = g.d[p].thr;
    L.s0[q] = (uint32_t)g.d[p].seed;
    L.s1[q] = (uint32_t)(g.d[p].seed >> 32);
    L.o0[q] = (uint32_t)g.d[p].offset;
    L.o1[q] = (uint32_t)(g.d[p].offset >> 32);
    L.total[q] = (int64_t)Tt * L.words[q];
    const int64_t end = L.blk[q] + (L.total[q] + 255) / 256;
    if (end > INT32_MAX) return hipErrorInvalidValue;
    L.blk[q + 1] = (int32_t)end;
  }
  if (L.n == 0 || L.blk[L.n] == 0) return hipSuccess;
  hipLaunchKernelGGL(dropout_mask_kernel, dim3((unsigned)L.blk[L.n]), dim3(256), 0, s, L);
  return hipGetLastError();
}

hipError_t launch_dropout_mask(uint32_t* bits, int32_t Tt, int32_t K, const DropoutSpec& d, hipStream_t s) {
  DropoutMaskGroup g{};
  g.bits[0] = bits;
  g.K[0] = K;
  g.d[0] = d;
  g.n = 1;
  return launch_dropout_mask_group(g, Tt, s);
}

}  // namespace dsv
