// kernels_f32.hip -- fp32 mode of the co-batched multi-LoRA layer: plain
// fp32 FMA kernels, one thread per output element, with the same semantics,
// layouts and fixed summation orders as the bf16 path (no matrix cores: this
// mode exists for tight-tolerance checks, not for throughput).
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "plan.h"

namespace dsv {
namespace {

// Dropout: is element k of compact training row i kept?
__device__ __forceinline__ bool kept(const F32Args& g, int i, int k) {
  return (g.keep[(int64_t)i * g.keep_words + (k >> 5)] >> (k & 31)) & 1u;
}

// h = x A_a^T for every row (j < r_a); training rows also into H_save.
__global__ void f32_shrink(F32Args g) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int t = (int)(idx / g.r_max), j = (int)(idx % g.r_max);
  if (t >= g.T) return;
  const int a = g.row_adapter[t];
  if (j >= g.ranks[a]) return;
  const float* x = g.X + (int64_t)t * g.ldx;
  const float* Aj = g.A + ((int64_t)a * g.r_max + j) * g.K;
  const int tr = g.row_train[t];
  const bool drop = g.keep && tr >= 0;  // dropout on a training row's low-rank input
  float acc = 0.f;
  for (int k = 0; k < g.K; ++k) acc = fmaf((drop && !kept(g, tr, k)) ? 0.f : x[k], Aj[k], acc);
  if (drop) acc *= g.drop_scale;
  g.Hall[(int64_t)t * g.r_max + j] = acc;
  if (tr >= 0 && g.Hsave) g.Hsave[(int64_t)tr * g.r_max + j] = acc;
}

// Backward without a kept H_save: h of the training rows again, in the same
// order of operations as f32_shrink (so the same values).
__global__ void f32_hrec(F32Args g) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int i = (int)(idx / g.r_max), j = (int)(idx % g.r_max);
  if (i >= g.Tt) return;
  const int a = g.train_adapter[i];
  if (j >= g.ranks[a]) return;
  const float* x = g.X + (int64_t)g.train_rows[i] * g.ldx;
  const float* Aj = g.A + ((int64_t)a * g.r_max + j) * g.K;
  const bool drop = g.keep != nullptr;
  float acc = 0.f;
  for (int k = 0; k < g.K; ++k) acc = fmaf((drop && !kept(g, i, k)) ? 0.f : x[k], Aj[k], acc);
  if (drop) acc *= g.drop_scale;
  g.Hrec[(int64_t)i * g.r_max + j] = acc;
}

// y = x W^T + s_a h B_a^T, fp32 sum, one store.
__global__ void f32_out(F32Args g) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int t = (int)(idx / g.N), n = (int)(idx % g.N);
  if (t >= g.T) return;
  const int a = g.row_adapter[t], r = g.ranks[a];
  const float* x = g.X + (int64_t)t * g.ldx;
  const float* w = g.W + (int64_t)n * g.ldw;
  float low = 0.f;
  const float* h = g.Hall + (int64_t)t * g.r_max;
  const float* b = g.B + ((int64_t)a * g.N + n) * g.r_max;
  for (int j = 0; j < r; ++j) low = fmaf(h[j], b[j], low);
  float acc = g.scales[a] * low;
  for (int k = 0; k < g.K; ++k) acc = fmaf(x[k], w[k], acc);
  g.Y[(int64_t)t * g.ldy + n] = acc;
}

// g = s_a dy B_a for every training row.
__global__ void f32_gmat(F32Args g) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int i = (int)(idx / g.r_max), j = (int)(idx % g.r_max);
  if (i >= g.Tt) return;
  const int a = g.train_adapter[i];
  if (j >= g.ranks[a]) return;
  const float* dy = g.dY + (int64_t)i * g.lddy;
  const float* b = g.B + (int64_t)a * g.N * g.r_max + j;
  float acc = 0.f;
  for (int n = 0; n < g.N; ++n) acc = fmaf(dy[n], b[(int64_t)n * g.r_max], acc);
  g.G[(int64_t)i * g.r_max + j] = g.scales[a] * acc;
}

// dB[a][n][j] (+)= s_a sum_i H_save[i][j] dy[i][n]; training rows of a in
// compact order (chunk list), fixed order.
__global__ void f32_db(F32Args g) {
  const int slot = blockIdx.y;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n = (int)(idx / g.r_max), j = (int)(idx % g.r_max);
  if (n >= g.N) return;
  const int a = g.train_ads[slot];
  if (j >= g.ranks[a]) return;
  float acc = 0.f;
  for (int p = g.tad_ptr[slot]; p < g.tad_ptr[slot + 1]; ++p) {
    const int32_t* ck = g.chunks + (int64_t)g.tad_chunks[p] * kItemWords;
    for (int i = ck[1]; i < ck[1] + ck[2]; ++i)
      acc = fmaf(g.Hs[(int64_t)i * g.r_max + j], g.dY[(int64_t)i * g.lddy + n], acc);
  }
  float* o = g.dB + ((int64_t)a * g.N + n) * g.r_max + j;
  const float v = g.scales[a] * acc;
  *o = g.accumulate ? *o + v : v;
}

// dA[a][j][k] (+)= sum_i g[i][j] x[t_i][k].
__global__ void f32_da(F32Args g) {
  const int slot = blockIdx.y;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int j = (int)(idx / g.K), k = (int)(idx % g.K);
  if (j >= g.r_max) return;
  const int a = g.train_ads[slot];
  if (j >= g.ranks[a]) return;
  float acc = 0.f;
  for (int p = g.tad_ptr[slot]; p < g.tad_ptr[slot + 1]; ++p) {
    const int32_t* ck = g.chunks + (int64_t)g.tad_chunks[p] * kItemWords;
    for (int i = ck[1]; i < ck[1] + ck[2]; ++i) {
      const float x = g.X[(int64_t)g.train_rows[i] * g.ldx + k];
      acc = fmaf(g.G[(int64_t)i * g.r_max + j], (g.keep && !kept(g, i, k)) ? 0.f : x, acc);
    }
  }
  if (g.keep) acc *= g.drop_scale;
  float* o = g.dA + ((int64_t)a * g.r_max + j) * g.K + k;
  *o = g.accumulate ? *o + acc : acc;
}

// dx = dy W + g A_a.
__global__ void f32_dx(F32Args g) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int i = (int)(idx / g.K), k = (int)(idx % g.K);
  if (i >= g.Tt) return;
  const int a = g.train_adapter[i], r = g.ranks[a];
  float acc = 0.f;
  const float* gi = g.G + (int64_t)i * g.r_max;
  const float* Aa = g.A + (int64_t)a * g.r_max * g.K + k;
  for (int j = 0; j < r; ++j) acc = fmaf(gi[j], Aa[(int64_t)j * g.K], acc);
  if (g.keep) acc = kept(g, i, k) ? acc * g.drop_scale : 0.f;  // through the dropout mask
  const float* dy = g.dY + (int64_t)i * g.lddy;
  for (int n = 0; n < g.N; ++n) acc = fmaf(dy[n], g.W[(int64_t)n * g.ldw + k], acc);
  g.dX[(int64_t)i * g.lddx + k] = acc;
}

unsigned blocks(int64_t n) { return (unsigned)((n + 255) / 256); }

}  // namespace

hipError_t launch_f32_fwd(const F32Args& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  hipLaunchKernelGGL(f32_shrink, dim3(blocks((int64_t)a.T * a.r_max)), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(f32_out, dim3(blocks((int64_t)a.T * a.N)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_f32_bwd(const F32Args& a0, hipStream_t s) {
  if (a0.Tt <= 0) return hipSuccess;
  F32Args a = a0;
  hipError_t e;
  if (!a.Hs) {
    hipLaunchKernelGGL(f32_hrec, dim3(blocks((int64_t)a.Tt * a.r_max)), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    a.Hs = a.Hrec;
  }
  hipLaunchKernelGGL(f32_gmat, dim3(blocks((int64_t)a.Tt * a.r_max)), dim3(256), 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(f32_db, dim3(blocks((int64_t)a.N * a.r_max), a.n_tads), dim3(256), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(f32_da, dim3(blocks((int64_t)a.r_max * a.K), a.n_tads), dim3(256), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.dX) {
    hipLaunchKernelGGL(f32_dx, dim3(blocks((int64_t)a.Tt * a.K)), dim3(256), 0, s, a);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace dsv
