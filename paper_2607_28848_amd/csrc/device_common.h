// device_common.h -- device-side helpers shared by the bf16 kernels (GEMM and
// rank-r / reduction kernels): vector types, 16-byte and masked loads, the
// bf16 roundings, dropout-mask helpers, LDS address-space types.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"

namespace dsv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 as_bf(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ u32x4 zero4() { return u32x4{0u, 0u, 0u, 0u}; }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest even (NaN stays NaN): gfx950's conversion
// instruction, two values per instruction.
__device__ __forceinline__ uint32_t f2bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Eight bf16 values with element e zeroed unless bit e of b is set (dropout).
__device__ __forceinline__ u32x4 keep8(u32x4 v, uint32_t b) {
  u32x4 o;
#pragma unroll
  for (int d = 0; d < 4; ++d)
    o[d] = v[d] & (((b >> (2 * d)) & 1u ? 0x0000ffffu : 0u) | ((b >> (2 * d + 1)) & 1u ? 0xffff0000u : 0u));
  return o;
}

// Byte of the dropout bitmask that covers columns c .. c+7 (c a multiple of 8).
__device__ __forceinline__ uint32_t keep_byte(const uint32_t* keep, int keep_words, int row, int c) {
  return (keep[(int64_t)row * keep_words + (c >> 5)] >> (c & 31)) & 0xffu;
}

// Eight bf16 values p[e * stride], e < n_valid (1 <= n_valid), the rest zero.
// Every lane loads all eight (the index is clamped to n_valid - 1, so every
// address is one the caller vouches for): straight-line code, no branches.
__device__ __forceinline__ u32x4 ld8_sel(const uint16_t* p, int64_t stride, int n_valid) {
  uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t x = (uint32_t)p[(int64_t)min(e, n_valid - 1) * stride];
    w[e >> 1] |= (e < n_valid ? x : 0u) << (16 * (e & 1));
  }
  return u32x4{w[0], w[1], w[2], w[3]};
}

// Eight bf16 values read with a per-element predicate, from p[e * stride].
__device__ __forceinline__ u32x4 ld8_masked(const uint16_t* p, int64_t stride, int n_valid) {
  uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    uint32_t v = (e < n_valid) ? (uint32_t)p[e * stride] : 0u;
    w[e >> 1] |= v << (16 * (e & 1));
  }
  return u32x4{w[0], w[1], w[2], w[3]};
}

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) uint32_t lds_u32;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// s_waitcnt immediate (gfx9 encoding): wait until at most n vector-memory
// operations of this wave are outstanding; lgkm and exp counters untouched.
constexpr int vmcnt_imm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }
__device__ __forceinline__ void vmem_wait_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

}  // namespace
}  // namespace dsv
