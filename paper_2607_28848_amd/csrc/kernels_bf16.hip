// kernels_bf16.hip -- CDNA4 (gfx950) kernels of the co-batched multi-LoRA
// layer in bf16 with fp32 accumulation.
//
// Forward (Sec. 2.2 multi-LoRA batching, Sec. 3.2 mixed forward batch):
//   shrink           h = x A_a^T for every row, grouped by adapter; rounded
//                    once to bf16; training rows also land in H_save.
//   gather_expand    fp32 low-rank term s_a h B_a^T of the rows that do not
//                    ride a GEMM tile group (short segments, e.g. decode),
//                    reading each touched adapter's B once per column block.
//   gemm (NT)        y = x W^T on the matrix cores; the tile's own adapter
//                    groups add s_a h B_a^T in the prologue, gathered rows add
//                    their fp32 term; one rounding to bf16 at the end.
// Backward (Sec. 3.2 backward of the training rows):
//   transpose_b/h    small transposed copies of B_a and H_save.
//   gmat             g = s_a dy B_a (contraction over N).
//   token_reduce     fp32 per-chunk partials of dy^T h and x^T g.
//   reduce_out       fixed-order sum of the partials into dB / dA.
//   gemm (NN)        dx = dy W + g A_a (prologue adds g A_a).
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "plan.h"

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

// fp32 -> bf16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

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

// 8x8 transpose of 16-bit elements held as 8 rows of 4 dwords:
// out[c] element e = in[e] element c.
__device__ __forceinline__ void transpose8x8(const u32x4 in[8], u32x4 out[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int d = c >> 1;
    const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = __builtin_amdgcn_perm(in[2 * e + 1][d], in[2 * e][d], sel);
    out[c] = u32x4{w[0], w[1], w[2], w[3]};
  }
}

// ---------------------------------------------------------------------------
// GEMM: 256 x 256 output tile per workgroup, 4 waves in a 2 x 2 grid, each
// wave 128 x 128 = 4 x 4 tiles of v_mfma_f32_32x32x16_bf16.  K-steps of 64,
// double-buffered LDS tiles of [256][64] bf16 for each operand, 16-byte
// chunks XOR-swizzled so that both the staging stores and the fragment reads
// are free of bank conflicts.
// ---------------------------------------------------------------------------
constexpr int TN = 256, TK = 64;
constexpr int kStageLd = TN + 8;  // epilogue staging row stride (elements)
constexpr int kLdsElems = (2 * 2 * kTileM * TK > kTileM * kStageLd) ? 2 * 2 * kTileM * TK
                                                                     : kTileM * kStageLd;

__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }

__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * TK + ((chunk ^ swz(row)) << 3);
}

template <bool NN>
__global__ __launch_bounds__(256) void gemm_lora_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[kLdsElems];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Workgroup -> tile.  Consecutive workgroup ids land on different XCDs
  // (round robin over 8); renumber so that each XCD owns a contiguous range
  // of tiles, then walk that range in groups of 8 row tiles so the tiles
  // running together on one XCD share row and column panels in its L2.
  const int nblk = gridDim.x, bid = blockIdx.x;
  const int per = nblk >> 3, rem = nblk & 7, xcd = bid & 7;
  const int logical = xcd * per + min(xcd, rem) + (bid >> 3);
  const int GM = 8;
  const int span = GM * g.n_ntiles;
  const int grp = logical / span, first_m = grp * GM;
  const int gsz = min(g.n_mtiles - first_m, GM);
  const int mt = first_m + (logical % span) % gsz;
  const int nt = (logical % span) / gsz;

  const int32_t* td = g.tiles + (int64_t)mt * kTileWords;
  const int m0 = td[0], ngroups = td[1], has_gather = td[2], nrows = td[3];
  const int n0 = nt * TN;

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // ---- low-rank prologue: tile groups on the matrix cores -----------------
  for (int gi = 0; gi < ngroups; ++gi) {
    const int a = td[4 + 3 * gi], lo = td[5 + 3 * gi], hi = td[6 + 3 * gi];
    const int r = g.ranks[a];
    const uint16_t* lq = g.Lq + (int64_t)a * g.lq_ad;
    for (int j0 = 0; j0 < r; j0 += 16) {
      const int jb = j0 + 8 * (lane >> 5);
      const int nv = min(8, r - jb);
      bf16x8 af[4], bq[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = wm * 128 + 32 * i + (lane & 31);
        u32x4 v = zero4();
        if (row >= lo && row < hi && nv > 0) {
          const uint16_t* p = g.Lp + (int64_t)(m0 + row) * g.ldl + jb;
          v = (nv == 8) ? ld16(p) : ld8_masked(p, 1, nv);
        }
        af[i] = as_bf(v);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = n0 + wn * 128 + 32 * j + (lane & 31);
        u32x4 v = zero4();
        if (col < g.Nout && nv > 0) v = ld8_masked(lq + (int64_t)jb * g.lq_j + (int64_t)col * g.lq_col, g.lq_j, nv);
        bq[j] = as_bf(v);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bq[j], acc[i][j], 0, 0, 0);
    }
  }
  if (g.scales != nullptr && ngroups > 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = wm * 128 + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        float s = 1.f;
        for (int gi = 0; gi < ngroups; ++gi)
          if (row >= td[5 + 3 * gi] && row < td[6 + 3 * gi]) s = g.scales[td[4 + 3 * gi]];
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j][v] *= s;
      }
  }
  if (has_gather && g.delta != nullptr) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = wm * 128 + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        if (row < nrows) {
          const int gs = g.gslot[m0 + row];
          if (gs >= 0) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int col = n0 + wn * 128 + 32 * j + (lane & 31);
              if (col < g.Nout) acc[i][j][v] += g.delta[(int64_t)gs * g.Nout + col];
            }
          }
        }
      }
  }

  // ---- main loop -----------------------------------------------------------
  // buffer b: A-operand tile at smem + b * 2 * kTileM * TK, B-operand tile right after it
  auto sA = [&](int b) { return smem + b * (2 * kTileM * TK); };
  auto sB = [&](int b) { return smem + b * (2 * kTileM * TK) + kTileM * TK; };
  const int nk = (g.C + TK - 1) / TK;
  u32x4 ra[8], rb[8];

  auto load_tile = [&](int kt) {
    const int k0 = kt * TK;
    const int ch = tid & 7;
    const int kk = k0 + ch * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = (tid >> 3) + 32 * i;
      ra[i] = (row < nrows && kk < g.C) ? ld16(g.P + (int64_t)(m0 + row) * g.ldp + kk) : zero4();
    }
    if constexpr (!NN) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int col = (tid >> 3) + 32 * i;
        rb[i] = (n0 + col < g.Nout && kk < g.C) ? ld16(g.Q + (int64_t)(n0 + col) * g.ldq + kk) : zero4();
      }
    } else {
      const int cb = tid >> 5, ob = tid & 31;
      const int ncol = n0 + 8 * ob;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int crow = k0 + 8 * cb + e;
        rb[e] = (crow < g.C && ncol < g.Nout) ? ld16(g.Q + (int64_t)crow * g.ldq + ncol) : zero4();
      }
    }
  };
  auto store_tile = [&](int buf) {
    const int ch = tid & 7;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = (tid >> 3) + 32 * i;
      *reinterpret_cast<u32x4*>(sA(buf) + lds_off(row, ch)) = ra[i];
    }
    if constexpr (!NN) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int col = (tid >> 3) + 32 * i;
        *reinterpret_cast<u32x4*>(sB(buf) + lds_off(col, ch)) = rb[i];
      }
    } else {
      const int cb = tid >> 5, ob = tid & 31;
      u32x4 tb[8];
      transpose8x8(rb, tb);
#pragma unroll
      for (int c = 0; c < 8; ++c)
        *reinterpret_cast<u32x4*>(sB(buf) + lds_off(8 * ob + c, cb)) = tb[c];
    }
  };

  if (nk > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_tile(kt + 1);
#pragma unroll
    for (int s = 0; s < TK / 16; ++s) {
      const int ch = 2 * s + (lane >> 5);
      bf16x8 af[4], bq[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = wm * 128 + 32 * i + (lane & 31);
        af[i] = as_bf(*reinterpret_cast<const u32x4*>(sA(buf) + lds_off(row, ch)));
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = wn * 128 + 32 * j + (lane & 31);
        bq[j] = as_bf(*reinterpret_cast<const u32x4*>(sB(buf) + lds_off(col, ch)));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bq[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_tile(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: one rounding, staged through LDS for 16-byte stores ------
  uint16_t* st = smem;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = wm * 128 + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        const int col = wn * 128 + 32 * j + (lane & 31);
        st[row * kStageLd + col] = f2bf(acc[i][j][v]);
      }
  __syncthreads();
#pragma unroll 4
  for (int it = 0; it < (kTileM * TN / 8) / 256; ++it) {
    const int idx = tid + 256 * it;
    const int row = idx >> 5, ch = idx & 31;
    const int col = n0 + ch * 8;
    if (row < nrows && col < g.Nout)
      *reinterpret_cast<u32x4*>(g.out + (int64_t)(m0 + row) * g.ldo + col) =
          *reinterpret_cast<const u32x4*>(st + row * kStageLd + ch * 8);
  }
}

// ---------------------------------------------------------------------------
// Skinny rank-r contraction: one workgroup per item of <= 16 rows of one
// adapter; the 4 waves take interleaved 32-wide slices of the contraction
// with v_mfma_f32_16x16x32_bf16 and combine them in LDS in a fixed order.
// ---------------------------------------------------------------------------
template <int MODE>  // 0: shrink (h -> H_all, H_save), 1: g (-> G, G^T)
__global__ __launch_bounds__(256) void skinny_kernel(SkinnyArgs g) {
  __shared__ float red[4][16][DSV_MAX_RANK + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* it = g.items + (int64_t)blockIdx.x * kItemWords;
  const int a = it[0], begin = it[1], cnt = it[2];
  const int r = g.ranks[a];
  const int slot = g.qsel ? g.qsel[a] : a;
  const uint16_t* Qa = g.Q + (int64_t)slot * g.q_ad;
  const int i = lane & 15;
  const int prow = (i < cnt) ? (g.rows ? g.rows[begin + i] : begin + i) : -1;
  f32x4 acc[4];
#pragma unroll
  for (int jt = 0; jt < 4; ++jt) acc[jt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nsteps = (g.C + 31) / 32;
  for (int step = wave; step < nsteps; step += 4) {
    const int k = step * 32 + 8 * (lane >> 4);
    const bool kin = k < g.C;
    const u32x4 av = (prow >= 0 && kin) ? ld16(g.P + (int64_t)prow * g.ldp + k) : zero4();
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
      if (16 * jt < r) {
        const int j = 16 * jt + (lane & 15);
        const u32x4 bv = (j < r && kin) ? ld16(Qa + (int64_t)j * g.ldq + k) : zero4();
        acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(av), as_bf(bv), acc[jt], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int jt = 0; jt < 4; ++jt)
#pragma unroll
    for (int v = 0; v < 4; ++v) red[wave][4 * (lane >> 4) + v][16 * jt + (lane & 15)] = acc[jt][v];
  __syncthreads();
  const float s = g.scales ? g.scales[a] : 1.f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int idx = tid + 256 * q;
    const int row = idx >> 6, j = idx & 63;
    if (row < cnt && j < r) {
      const float sum = ((red[0][row][j] + red[1][row][j]) + red[2][row][j]) + red[3][row][j];
      const int pr = g.rows ? g.rows[begin + row] : begin + row;
      if (MODE == 0) {
        const uint16_t hb = f2bf(sum);
        g.out1[(int64_t)pr * g.ld1 + j] = hb;
        if (g.out2) {
          const int tr = g.row_train[pr];
          if (tr >= 0) g.out2[(int64_t)tr * g.ld2 + j] = hb;
        }
      } else {
        const uint16_t gb = f2bf(s * sum);
        g.out1[(int64_t)pr * g.ld1 + j] = gb;
        g.out2[(int64_t)j * g.ld2 + pr] = gb;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Gathered low-rank term: item = <= 16 gathered rows of one adapter, one
// workgroup per (item, 256-column block); fp32 result, already scaled.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gather_expand_kernel(
    const uint16_t* __restrict__ H, int64_t ldh, const uint16_t* __restrict__ B, int32_t N,
    int32_t r_max, const int32_t* __restrict__ items, const int32_t* __restrict__ gather_rows,
    const int32_t* __restrict__ ranks, const float* __restrict__ scales, float* __restrict__ delta) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* it = items + (int64_t)blockIdx.x * kItemWords;
  const int a = it[0], sbeg = it[1], cnt = it[2];
  const int r = ranks[a];
  const int i = lane & 15;
  const int row = (i < cnt) ? gather_rows[sbeg + i] : -1;
  const uint16_t* Ba = B + (int64_t)a * N * r_max;
  const int nb = blockIdx.y * 256 + wave * 64;
  f32x4 acc[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int j0 = 0; j0 < r; j0 += 32) {
    const int jb = j0 + 8 * (lane >> 4);
    const int nv = min(8, r - jb);
    u32x4 av = zero4();
    if (row >= 0 && nv > 0) {
      const uint16_t* p = H + (int64_t)row * ldh + jb;
      av = (nv == 8) ? ld16(p) : ld8_masked(p, 1, nv);
    }
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const int n = nb + 16 * ct + (lane & 15);
      u32x4 bv = zero4();
      if (n < N && nv > 0) bv = ld8_masked(Ba + (int64_t)n * r_max + jb, 1, nv);
      acc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(av), as_bf(bv), acc[ct], 0, 0, 0);
    }
  }
  const float s = scales[a];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int ii = 4 * (lane >> 4) + v;
      const int n = nb + 16 * ct + (lane & 15);
      if (ii < cnt && n < N) delta[(int64_t)(sbeg + ii) * N + n] = s * acc[ct][v];
    }
}

// ---------------------------------------------------------------------------
// Reduction over training tokens, per single-adapter chunk:
//   part[chunk][c][j] = sum_t P[prow(t)][c] Qt[j][t]
// A lane loads an 8 (tokens) x 8 (columns) block, transposes it in registers
// and feeds the 8 columns as A-operands of 8 v_mfma_f32_16x16x32_bf16 tiles
// (tile m, row rho <-> column c = base + 8 rho + m).  Each wave covers 128
// columns, a workgroup 512.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void token_reduce_kernel(TokenReduceArgs g) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* ck = g.chunks + (int64_t)blockIdx.x * kItemWords;
  const int a = ck[0], begin = ck[1], cnt = ck[2];
  const int r = g.ranks[a];
  const int q = lane >> 4, rho = lane & 15;
  const int cbase = blockIdx.y * 512 + wave * 128;
  const int c0 = cbase + 8 * rho;
  f32x4 acc[8][4];
#pragma unroll
  for (int m = 0; m < 8; ++m)
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) acc[m][jt] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int t0 = 0; t0 < cnt; t0 += 32) {
    const int tb = t0 + 8 * q;
    u32x4 v[8], V[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int t = tb + e;
      v[e] = zero4();
      if (t < cnt && c0 < g.C) {
        const int pr = g.prow ? g.prow[begin + t] : begin + t;
        v[e] = ld16(g.P + (int64_t)pr * g.ldp + c0);
      }
    }
    transpose8x8(v, V);
    const int nt = min(8, cnt - tb);
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
      if (16 * jt < r) {
        const int j = 16 * jt + rho;
        u32x4 bv = zero4();
        if (j < r && nt > 0) bv = ld8_masked(g.Qt + (int64_t)j * g.ldqt + begin + tb, 1, nt);
#pragma unroll
        for (int m = 0; m < 8; ++m)
          acc[m][jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(V[m]), as_bf(bv), acc[m][jt], 0, 0, 0);
      }
    }
  }
  float* out = g.part + (int64_t)blockIdx.x * g.C * g.r_max;
#pragma unroll
  for (int m = 0; m < 8; ++m)
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
      for (int vv = 0; vv < 4; ++vv) {
        const int rr = 4 * q + vv;
        const int c = cbase + 8 * rr + m;
        const int j = 16 * jt + rho;
        if (j < r && c < g.C) out[(int64_t)c * g.r_max + j] = acc[m][jt][vv];
      }
}

// Fixed-order sum of one training adapter's chunk partials.
__global__ __launch_bounds__(256) void reduce_out_kernel(
    const float* __restrict__ part, int32_t C, int32_t r_max, const int32_t* __restrict__ train_ads,
    const int32_t* __restrict__ tad_ptr, const int32_t* __restrict__ tad_chunks,
    const int32_t* __restrict__ ranks, const float* __restrict__ scales, int a_layout,
    int32_t accumulate, float* __restrict__ out) {
  const int ta = blockIdx.y;
  const int a = train_ads[ta], r = ranks[a];
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  int c, j;
  if (a_layout) {  // out[a][j][c], c fastest
    j = (int)(idx / C);
    c = (int)(idx % C);
  } else {  // out[a][c][j], j fastest
    c = (int)(idx / r_max);
    j = (int)(idx % r_max);
  }
  if (c >= C || j >= r) return;
  float sum = 0.f;
  for (int p = tad_ptr[ta]; p < tad_ptr[ta + 1]; ++p)
    sum += part[((int64_t)tad_chunks[p] * C + c) * r_max + j];
  if (scales) sum *= scales[a];
  float* o = a_layout ? out + ((int64_t)a * r_max + j) * C + c : out + ((int64_t)a * C + c) * r_max + j;
  *o = accumulate ? *o + sum : sum;
}

// Bt[slot][j][n] = B[a][n][j]  (j < r_a; other rows zero).
__global__ __launch_bounds__(256) void transpose_b_kernel(const uint16_t* __restrict__ B, int32_t N,
                                                          int32_t r_max, const int32_t* __restrict__ train_ads,
                                                          const int32_t* __restrict__ ranks,
                                                          uint16_t* __restrict__ Bt) {
  const int slot = blockIdx.z, j = blockIdx.y;
  const int n = blockIdx.x * 256 + threadIdx.x;
  if (n >= N) return;
  const int a = train_ads[slot];
  const uint16_t v = (j < ranks[a]) ? B[((int64_t)a * N + n) * r_max + j] : (uint16_t)0;
  Bt[((int64_t)slot * r_max + j) * N + n] = v;
}

// Ht[j][t] = H_save[t][j]  (j < rank of row t; other entries zero).
__global__ __launch_bounds__(256) void transpose_h_kernel(const uint16_t* __restrict__ Hs, int32_t Tt,
                                                          int32_t r_max, const int32_t* __restrict__ train_adapter,
                                                          const int32_t* __restrict__ ranks,
                                                          uint16_t* __restrict__ Ht, int64_t ldt) {
  const int j = blockIdx.y;
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= Tt) return;
  const uint16_t v = (j < ranks[train_adapter[t]]) ? Hs[(int64_t)t * r_max + j] : (uint16_t)0;
  Ht[(int64_t)j * ldt + t] = v;
}

}  // namespace

hipError_t launch_gemm_nt(const GemmArgs& a, hipStream_t s) {
  if (a.n_mtiles <= 0 || a.n_ntiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(gemm_lora_kernel<false>, dim3(a.n_mtiles * a.n_ntiles), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemm_nn(const GemmArgs& a, hipStream_t s) {
  if (a.n_mtiles <= 0 || a.n_ntiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(gemm_lora_kernel<true>, dim3(a.n_mtiles * a.n_ntiles), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_shrink(const SkinnyArgs& a, int32_t n_items, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(skinny_kernel<0>, dim3(n_items), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gmat(const SkinnyArgs& a, int32_t n_items, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(skinny_kernel<1>, dim3(n_items), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gather_expand(const uint16_t* H, int64_t ldh, const uint16_t* B, int32_t N,
                                int32_t r_max, const int32_t* items, int32_t n_items,
                                const int32_t* gather_rows, const int32_t* ranks,
                                const float* scales, float* delta, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_expand_kernel, dim3(n_items, (N + 255) / 256), dim3(256), 0, s, H, ldh,
                     B, N, r_max, items, gather_rows, ranks, scales, delta);
  return hipGetLastError();
}

hipError_t launch_token_reduce(const TokenReduceArgs& a, int32_t n_chunks, hipStream_t s) {
  if (n_chunks <= 0) return hipSuccess;
  hipLaunchKernelGGL(token_reduce_kernel, dim3(n_chunks, (a.C + 511) / 512), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_reduce_out(const float* part, int32_t C, int32_t r_max, const int32_t* train_ads,
                             int32_t n_tads, const int32_t* tad_ptr, const int32_t* tad_chunks,
                             const int32_t* ranks, const float* scales, bool a_layout,
                             int32_t accumulate, float* out, hipStream_t s) {
  if (n_tads <= 0) return hipSuccess;
  const int64_t total = (int64_t)C * r_max;
  hipLaunchKernelGGL(reduce_out_kernel, dim3((unsigned)((total + 255) / 256), n_tads), dim3(256), 0, s,
                     part, C, r_max, train_ads, tad_ptr, tad_chunks, ranks, scales, a_layout ? 1 : 0,
                     accumulate, out);
  return hipGetLastError();
}

hipError_t launch_transpose_b(const uint16_t* B, int32_t N, int32_t r_max, const int32_t* train_ads,
                              int32_t n_tads, const int32_t* ranks, uint16_t* Bt, hipStream_t s) {
  if (n_tads <= 0) return hipSuccess;
  hipLaunchKernelGGL(transpose_b_kernel, dim3((N + 255) / 256, r_max, n_tads), dim3(256), 0, s, B, N,
                     r_max, train_ads, ranks, Bt);
  return hipGetLastError();
}

hipError_t launch_transpose_h(const uint16_t* Hs, int32_t Tt, int32_t r_max,
                              const int32_t* train_adapter, const int32_t* ranks, uint16_t* Ht,
                              int64_t ldt, hipStream_t s) {
  if (Tt <= 0) return hipSuccess;
  hipLaunchKernelGGL(transpose_h_kernel, dim3((Tt + 255) / 256, r_max), dim3(256), 0, s, Hs, Tt, r_max,
                     train_adapter, ranks, Ht, ldt);
  return hipGetLastError();
}

}  // namespace dsv
