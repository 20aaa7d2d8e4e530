// kernels_bf16.hip -- CDNA4 (gfx950) rank-r and reduction kernels of the
// co-batched multi-LoRA layer in bf16 with fp32 accumulation (the GEMMs are in
// gemm_bf16.hip).
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
//   token_reduce     fp32 per-chunk partials of dy^T h (dB) that also
//                    contract the dy rows they stage with B_a: per-block
//                    partials of g = s_a dy B_a, so dy is read once for both.
//   g finish         fixed-order sum of g's block partials, rounded once.
//   token_reduce     fp32 per-chunk partials of x^T g (dA).
//   reduce_out       fixed-order sum of the partials into dB / dA.
//   gemm (NT / NN)   dx = dy W + g A_a (prologue adds g A_a).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "device_common.h"
#include "kernels.h"
#include "plan.h"

namespace dsv {
namespace {

// ---------------------------------------------------------------------------
// Skinny rank-r contraction out[row][j] = sum_k P[row][k] Q_a[j][k]: one
// workgroup per item of <= ROWS rows of one adapter, 8 waves.  The
// contraction runs in chunks of 256 columns; a chunk's ROWS input rows and
// 16*NJ adapter rows go from global memory straight into LDS, 512 contiguous
// bytes per row (two rows per wave instruction), double-buffered, so the input
// streams in long runs.  Wave w multiplies columns [32w, 32w+32) of every chunk
// with v_mfma_f32_16x16x32_bf16; the 8 partial sums of a row are combined in
// LDS in a fixed order, so a row's result does not depend on the item it sits
// in.  The LDS image of a row is swizzled (16-byte chunk c in slot c ^ (row & 7))
// so the fragment reads are free of bank conflicts.
// ---------------------------------------------------------------------------
constexpr int SW = 8;       // waves per rank-contraction workgroup
constexpr int SK_CK = 256;  // contraction columns per chunk

// Zeros in global memory: a direct-to-LDS load from here writes zeros, so a
// lane with nothing to load still issues its load and every wave issues the
// same number of loads per chunk (what a partial vmcnt wait relies on).
__device__ const u32x4 kZeroRow[64] = {};

typedef __attribute__((address_space(1))) const void global_cv;
extern "C" __device__ void llvm_amdgcn_global_load_lds(global_cv* src, lds_u32* lds, int size, int offset,
                                                       int aux) __asm("llvm.amdgcn.global.load.lds");

// Final value of one entry (item row `row`, rank column j) from its fp32 sum.
template <int MODE>
__device__ __forceinline__ void skinny_store(const SkinnyArgs& g, int a, int begin, int row, int j, float sum) {
  const int pr = g.rows ? g.rows[begin + row] : begin + row;
  if (MODE == 0) {
    if (g.keep && g.row_train[pr] >= 0) sum *= g.drop_scale;  // dropout of a training row
    const uint16_t hb = f2bf(sum);
    if (g.out1) g.out1[(int64_t)pr * g.ld1 + j] = hb;
    if (g.out2) {
      const int tr = g.row_train[pr];
      if (tr >= 0) g.out2[(int64_t)tr * g.ld2 + j] = hb;
    }
  } else {
    const float s = g.scales ? g.scales[a] : 1.f;
    g.out1[(int64_t)pr * g.ld1 + j] = f2bf(s * sum);
  }
}

// DROP (shrink only): the training rows' input passes through the dropout mask
// (a mask byte per 8 columns, applied to the fragment as it is read).
template <int MODE, int NJ, int ROWS, bool DROP>  // MODE 0: shrink (h -> H_all, H_save), 1: g (-> G)
__global__ __launch_bounds__(64 * SW) void skinny_kernel(SkinnyGroup G) {
  const SkinnyArgs g = G.a[G.slot_proj[blockIdx.y]];  // the projection's arguments (scalar registers)
  const int piece = G.slot_piece[blockIdx.y];
  constexpr int RT = ROWS / 16;           // 16-row tiles per item
  constexpr int SR = ROWS + 16 * NJ;      // LDS rows of a chunk: input rows, then adapter rows
  constexpr int RB = SK_CK * 2;           // bytes per LDS row
  constexpr int L = SR / 2 / SW;          // 1 KiB load instructions per wave per chunk
  constexpr int STAGE = SR * RB;
  static_assert(L * 2 * SW == SR, "loads per wave");
  // Chunks in flight: three buffers (two chunks loading while one is used)
  // where that keeps two workgroups per CU (72 KB of LDS), else two.  Under
  // dropout the mask loads share the vector-memory counter, so two.
  constexpr int NSTG = (!DROP && 3 * STAGE <= 72 * 1024) ? 3 : 2;
  __shared__ __attribute__((aligned(1024))) char smem[NSTG * STAGE];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int32_t* it = g.items + (int64_t)blockIdx.x * kItemWords;
  const int a = it[0], begin = it[1], cnt = it[2];
  const int r = g.ranks[a];
  const int qslot = g.qsel ? g.qsel[a] : a;
  const uint16_t* Qa = g.Q + (int64_t)qslot * g.q_ad;
  // Wave instruction q loads LDS rows 2q and 2q+1; lane = 32 * (row - 2q) +
  // slot.  Rows past the item repeat its last row (their sums are not stored),
  // adapter rows past the rank load nothing and are written with zeros, as are
  // the columns past the contraction.
  const int sub = lane >> 5, sl = lane & 31;
  const uint16_t* src[L];
  int kcap[L];  // columns the lane's row provides
#pragma unroll
  for (int i = 0; i < L; ++i) {
    const int q = wave * L + i;
    const int sr = 2 * q + sub;
    if (2 * q < ROWS) {
      const int e = max(min(sr, cnt - 1), 0);
      const int pr = g.rows ? g.rows[begin + e] : begin + e;
      src[i] = g.P + (int64_t)pr * g.ldp + 8 * (sl ^ (sr & 7));
      kcap[i] = g.C;
    } else {
      const int j = sr - ROWS;
      src[i] = Qa + (int64_t)min(j, r - 1) * g.ldq + 8 * (sl ^ (sr & 7));
      kcap[i] = j < r ? g.C : 0;
    }
  }
  auto issue = [&](int c, int st) {
    char* base = smem + st * STAGE;
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int q = wave * L + i;
      const int k = c * SK_CK + 8 * (sl ^ ((2 * q + sub) & 7));
      if constexpr (NSTG == 3) {  // every lane loads: L loads per wave per chunk
        const void* from = k < kcap[i] ? static_cast<const void*>(src[i] + c * SK_CK)
                                       : static_cast<const void*>(&kZeroRow[lane]);
        llvm_amdgcn_global_load_lds((global_cv*)from, (lds_u32*)(base + q * 1024), 16, 0, 0);
      } else if (k < kcap[i]) {
        llvm_amdgcn_global_load_lds((global_cv*)(src[i] + c * SK_CK), (lds_u32*)(base + q * 1024), 16, 0, 0);
      } else {
        *reinterpret_cast<u32x4*>(base + q * 1024 + 16 * lane) = zero4();
      }
    }
  };
  // dropout: compact training index of each fragment row of the lane (-1: none)
  int trl[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    trl[t] = -1;
    if constexpr (DROP) {
      const int i = 16 * t + (lane & 15);
      const int pr = g.rows ? g.rows[begin + min(i, cnt - 1)] : begin + min(i, cnt - 1);
      trl[t] = i < cnt ? g.row_train[pr] : -1;
    }
  }
  const int lc = 4 * wave + (lane >> 4);  // logical 16-byte chunk of the lane's fragments
  // this workgroup's chunks of the contraction: [c_beg, nch)
  const int c_beg = piece * g.cpp;
  const int nch = min((g.C + SK_CK - 1) / SK_CK, c_beg + g.cpp);
  f32x4 acc[RT][NJ];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int jt = 0; jt < NJ; ++jt) acc[t][jt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Mask bytes of chunk c + 1 are loaded during chunk c, into the other of two
  // register sets (the loop is unrolled by two), so the wait at the top of a
  // chunk covers them and nothing waits on a load issued after them.
  auto load_mask = [&](int c, uint32_t (&m)[RT]) {
    const int col = min(c * SK_CK + 8 * lc, 32 * g.keep_words - 8);
#pragma unroll
    for (int t = 0; t < RT; ++t) m[t] = keep_byte(g.keep, g.keep_words, max(trl[t], 0), col);
  };
  auto chunk = [&](int c, const uint32_t (&mu)[RT], uint32_t (&ml)[RT]) {
    if constexpr (NSTG == 3) {
      // This wave's loads of chunk c are in (chunk c + 1's L loads may still be
      // in flight), and after the barrier everyone's are.  A plain barrier: the
      // fence of __syncthreads would wait for every load in flight.
      if (c + 1 < nch) __builtin_amdgcn_s_waitcnt(vmcnt_imm(L));
      else vmem_wait_all();
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
    } else {
      vmem_wait_all();
      __syncthreads();  // chunk c is in; every wave is done with chunk c - 1's buffer
    }
    if (c + NSTG - 1 < nch) issue(c + NSTG - 1, (c + NSTG - 1 - c_beg) % NSTG);
    if constexpr (DROP) load_mask(min(c + 1, nch - 1), ml);  // unconditional: no merge to wait on
    const char* sb = smem + ((c - c_beg) % NSTG) * STAGE;
    bf16x8 xf[RT], qf[NJ];
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      const int row = 16 * t + (lane & 15);
      u32x4 x = *reinterpret_cast<const u32x4*>(sb + row * RB + 16 * (lc ^ (row & 7)));
      if constexpr (DROP) x = trl[t] >= 0 ? keep8(x, mu[t]) : x;
      xf[t] = as_bf(x);
    }
#pragma unroll
    for (int jt = 0; jt < NJ; ++jt) {
      const int row = ROWS + 16 * jt + (lane & 15);
      qf[jt] = as_bf(*reinterpret_cast<const u32x4*>(sb + row * RB + 16 * (lc ^ (row & 7))));
    }
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int jt = 0; jt < NJ; ++jt)
        acc[t][jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xf[t], qf[jt], acc[t][jt], 0, 0, 0);
  };
  uint32_t m0[RT] = {}, m1[RT] = {};
  if (c_beg < nch) {
    issue(c_beg, 0);
    if (NSTG == 3 && c_beg + 1 < nch) issue(c_beg + 1, 1);
    if constexpr (DROP) load_mask(c_beg, m0);
  }
  for (int c = c_beg; c < nch; c += 2) {
    chunk(c, m0, m1);
    if (c + 1 < nch) chunk(c + 1, m1, m0);
  }
  __syncthreads();  // the stage buffers become the reduction buffer
  constexpr int RW = 16 * NJ + 1;
  static_assert(SW * ROWS * RW * 4 <= NSTG * STAGE, "reduction buffer");
  float* red = reinterpret_cast<float*>(smem);  // [SW][ROWS][RW]
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int jt = 0; jt < NJ; ++jt)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        red[(wave * ROWS + 16 * t + 4 * (lane >> 4) + v) * RW + 16 * jt + (lane & 15)] = acc[t][jt][v];
  __syncthreads();
#pragma unroll
  for (int q = 0; q < (ROWS * 64 + 64 * SW - 1) / (64 * SW); ++q) {
    const int idx = tid + 64 * SW * q;
    const int row = idx >> 6, j = idx & 63;
    if (row < ROWS && row < cnt && j < r) {
      float sum = 0.f;
#pragma unroll
      for (int w = 0; w < SW; ++w) sum += red[(w * ROWS + row) * RW + j];
      if (g.pieces == 1)
        skinny_store<MODE>(g, a, begin, row, j, sum);
      else
        g.part[((int64_t)piece * g.part_n + begin + row) * g.r_max + j] = sum;
    }
  }
}

// Sum of the pieces of a split rank-r contraction, in piece order, and the
// store of the result: one workgroup per (item, split projection).
template <int MODE>
__global__ __launch_bounds__(256) void skinny_finish_kernel(SkinnyGroup G) {
  const SkinnyArgs& g = G.a[G.slot_proj[blockIdx.y]];
  const int32_t* it = g.items + (int64_t)blockIdx.x * kItemWords;
  const int a = it[0], begin = it[1], cnt = it[2];
  const int r = g.ranks[a];
  for (int idx = threadIdx.x; idx < cnt * r; idx += 256) {
    const int row = idx / r, j = idx - row * r;
    const float* src = g.part + (int64_t)(begin + row) * g.r_max + j;
    const int64_t stride = (int64_t)g.part_n * g.r_max;
    // eight loads in flight, added in piece order (the same sum as one at a time)
    float sum = 0.f;
    int q = 0;
    for (; q + 8 <= g.pieces; q += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = src[(q + u) * stride];
#pragma unroll
      for (int u = 0; u < 8; ++u) sum += v[u];
    }
    for (; q < g.pieces; ++q) sum += src[q * stride];
    skinny_store<MODE>(g, a, begin, row, j, sum);
  }
}

// ---------------------------------------------------------------------------
// Gathered low-rank term: item = <= 16 gathered rows of one adapter, one
// workgroup per (item, 256-column block); fp32 result, already scaled.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gather_expand_kernel(
    GatherGroup G, int64_t ldh, int32_t r_max, const int32_t* __restrict__ items,
    const int32_t* __restrict__ gather_rows, const int32_t* __restrict__ ranks, const float* __restrict__ scales) {
  int pj = 0;  // the projection: blockIdx.y runs over every projection's column blocks
  while (pj + 1 < G.n && (int)blockIdx.y >= G.yoff[pj + 1]) ++pj;
  const uint16_t* __restrict__ H = G.a[pj].H;
  const uint16_t* __restrict__ B = G.a[pj].B;
  const int32_t N = G.a[pj].N;
  float* __restrict__ delta = G.a[pj].delta;
  const int by = (int)blockIdx.y - G.yoff[pj];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* it = items + (int64_t)blockIdx.x * kItemWords;
  const int a = it[0], sbeg = it[1], cnt = it[2];
  const int r = ranks[a];
  const int i = lane & 15;
  const int row = (i < cnt) ? gather_rows[sbeg + i] : -1;
  const uint16_t* Ba = B + (int64_t)a * N * r_max;
  const int nb = by * 256 + wave * 64;
  // B rows start 16-byte aligned when r_max is a multiple of 8: a lane's 8
  // ranks are then one 16-byte load (else 8 element loads)
  const bool b16 = (r_max & 7) == 0;
  f32x4 acc[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
  // both 32-rank steps (r <= 64) are loaded before the first MFMA: one round
  // trip to memory per workgroup instead of one per step
  u32x4 av[2], bv[2][4];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int jb = 32 * s + 8 * (lane >> 4);
    const int nv = min(8, r - jb);
    av[s] = zero4();
    if (row >= 0 && nv > 0) {
      const uint16_t* p = H + (int64_t)row * ldh + jb;
      av[s] = (nv == 8) ? ld16(p) : ld8_masked(p, 1, nv);
    }
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const int n = nb + 16 * ct + (lane & 15);
      bv[s][ct] = zero4();
      if (n < N && nv > 0) {
        const uint16_t* p = Ba + (int64_t)n * r_max + jb;
        bv[s][ct] = (b16 && nv == 8) ? ld16(p) : ld8_masked(p, 1, nv);
      }
    }
  }
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    if (32 * s >= r) break;
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
      acc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(av[s]), as_bf(bv[s][ct]), acc[ct], 0, 0, 0);
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
//   part[chunk][c][j] = sum_t P[prow(t)][c] Q[t][j]
// One workgroup per (chunk, kTokenCols = 256 columns), 8 waves; wave w owns
// columns [32w, 32w+32).  Tokens go in steps of 32: the step's 32 P rows (512
// contiguous bytes each, two rows per wave instruction) go from global memory
// straight into LDS, double-buffered, and come out transposed
// (ds_read_b64_tr_b16), so a lane holds one column c and 8 consecutive tokens:
// the A operand of v_mfma_f32_16x16x32_bf16 with the columns as rows and the
// tokens as the contraction.  The B operand (rank j, 8 tokens of Q, the small
// rank-wide matrix) is read from global memory a step ahead.  A row of the
// LDS image keeps its 16-byte slot s at s ^ 2(t % 4), so the 4 rows x 32
// bytes of one transposed read hit distinct banks.  Tokens past the chunk and
// columns past C are written as zeros instead of loaded.  Each column's sum
// runs over the tokens in order, so it does not depend on the column blocking.
// ---------------------------------------------------------------------------
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// GP (the dB reductions, P = dY): the workgroup also writes the g partial of
// its column block.  The adapter's B rows of the block sit in LDS rank-major
// (bts[j][c], kBtRow-byte rows), loaded once; in every step waves 0 and 1
// take the step's tokens 0-15 and 16-31 as MFMA A-operands (rows read from the
// staged P image as they are, 16 bytes = 8 columns per lane) against B's
// columns, 8 contractions of 32 columns, and store the [16][r] partial.
constexpr int kBtRow = kTokenCols * 2 + 16;

template <int NJ, bool DROP, bool GP>
__global__ __launch_bounds__(512) void token_reduce_kernel(TokenReduceGroup G) {
  constexpr int TS = 32;                     // tokens per step
  constexpr int STAGE = TS * kTokenCols * 2;  // P bytes per stage
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE + (GP ? 16 * NJ * kBtRow : 0)];
  int k = 0;  // the reduction: blockIdx.y runs over every reduction's column blocks
  while (k + 1 < G.n && (int)blockIdx.y >= G.yoff[k + 1]) ++k;
  const TokenReduceArgs g = G.a[k];
  const int cb = (int)blockIdx.y - G.yoff[k], cbase = cb * kTokenCols;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int32_t* ck = g.chunks + (int64_t)blockIdx.x * kItemWords;
  const int a = ck[0], begin = ck[1], cnt = ck[2];
  const int r = g.ranks[a];
  const int nsteps = (cnt + TS - 1) / TS;
  const int sub = lane >> 5, sl = lane & 31;  // staging: row within the instruction, slot
  const int gq = lane >> 4, lam = lane & 15;  // fragments: token octet, column / rank
  // P rows 2q + sub of the step, q = 2 wave + i; slot sl holds the row's
  // 16-byte chunk sl ^ 2(row % 4).  The P row numbers of a step are looked up
  // a step before its loads are issued.
  auto rows_of = [&](int step, int (&pr)[2]) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int t = min(step * TS + 2 * (2 * wave + i) + sub, cnt - 1);
      pr[i] = g.prow ? g.prow[begin + t] : begin + t;
    }
  };
  auto issue = [&](int step, int st, const int (&pr)[2]) {
    char* base = smem + st * STAGE;
    const int t0 = step * TS;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = 2 * wave + i;
      const int row = 2 * q + sub;
      const int c = cbase + 8 * (sl ^ (2 * (row & 3)));
      char* dst = base + q * 1024;
      if (t0 + row < cnt && c < g.C)
        llvm_amdgcn_global_load_lds((global_cv*)(g.P + (int64_t)pr[i] * g.ldp + c), (lds_u32*)dst, 16, 0, 0);
      else
        *reinterpret_cast<u32x4*>(dst + 16 * lane) = zero4();
    }
  };
  // B fragments of a step: Q[begin + 8 gq + e][16 jt + lam], zero past the rank
  // and past the chunk (straight-line loads from clamped addresses)
  auto load_q = [&](int step, u32x4 (&bq)[NJ]) {
    const int t = step * TS + 8 * gq;
    const int nt = max(1, min(8, cnt - t));
    const uint16_t* row = g.Q + (int64_t)(begin + min(t, cnt - 1)) * g.ldq;
#pragma unroll
    for (int jt = 0; jt < NJ; ++jt) {
      const int j = 16 * jt + lam;
      const u32x4 v = ld8_sel(row + min(j, r - 1), g.ldq, nt);
      bq[jt] = (j < r && t < cnt) ? v : zero4();
    }
  };
  // dropout: each token's mask word for the wave's 32 columns, a step ahead
  const bool masked = DROP && g.keep != nullptr;  // DROP: the launch has masked reductions
  const int kw = masked ? min((cbase + 32 * wave) >> 5, g.keep_words - 1) : 0;
  auto load_mask = [&](int step, uint32_t (&m)[8]) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int t = min(step * TS + 8 * gq + e, cnt - 1);
      m[e] = g.keep[(int64_t)(begin + t) * g.keep_words + kw];
    }
  };
  if constexpr (GP) {
    // B_a[c][j] of the block's columns into bts[j][c]; zero past the rank and
    // past C (published by the first step's barrier)
    char* bts = smem + 2 * STAGE;
    const uint16_t* Ba = g.B + (int64_t)a * g.C * g.r_max;
    const bool b16 = (g.r_max & 7) == 0;  // a rank octet is one aligned 16-byte load
    for (int idx = tid; idx < kTokenCols * 2 * NJ; idx += 512) {
      const int cl = idx % kTokenCols, jo = idx / kTokenCols;  // column, rank octet
      const int c = cbase + cl, nv = min(8, r - 8 * jo);
      u32x4 v = zero4();
      if (c < g.C && nv > 0) {
        const uint16_t* src = Ba + (int64_t)c * g.r_max + 8 * jo;
        v = (b16 && nv == 8) ? ld16(src) : ld8_masked(src, 1, nv);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e)
        *reinterpret_cast<uint16_t*>(bts + (8 * jo + e) * kBtRow + 2 * cl) = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
    }
  }
  auto tr_read = [&](const char* p) -> u32x2 {
    const s16x4 h = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
    return u32x2{(uint32_t)(uint16_t)h[0] | ((uint32_t)(uint16_t)h[1] << 16),
                 (uint32_t)(uint16_t)h[2] | ((uint32_t)(uint16_t)h[3] << 16)};
  };
  f32x4 acc[2][NJ];
#pragma unroll
  for (int ct = 0; ct < 2; ++ct)
#pragma unroll
    for (int jt = 0; jt < NJ; ++jt) acc[ct][jt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // One step; the B fragments and mask words of the next step load into the
  // other register set (the loop is unrolled by two), so the wait at the top
  // of a step covers them and nothing waits on a load issued after them.
  auto step_fn = [&](int step, const u32x4 (&qu)[NJ], u32x4 (&ql)[NJ], const uint32_t (&mu)[8],
                     uint32_t (&ml)[8], const int (&pu)[2], int (&pl)[2]) {
    vmem_wait_all();
    __syncthreads();  // the step is in; every wave is done with the previous step's buffer
    // the step's fragments are read before the next step's loads into LDS are
    // issued, so no read has to wait for those loads
    const char* sb = smem + (step & 1) * STAGE;
    u32x4 x[2];
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) {
      u32x2 h[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int t = 8 * gq + 4 * hh + (lam >> 2);
        const int col = 32 * wave + 16 * ct + 4 * (lam & 3);  // within the block
        h[hh] = tr_read(sb + t * (kTokenCols * 2) + 16 * ((col >> 3) ^ (2 * (t & 3))) + 2 * (col & 7));
      }
      x[ct] = u32x4{h[0][0], h[0][1], h[1][0], h[1][1]};
    }
    if (step + 1 < nsteps) issue(step + 1, (step + 1) & 1, pu);
    rows_of(min(step + 2, nsteps - 1), pl);
    load_q(min(step + 1, nsteps - 1), ql);
    if (masked) load_mask(min(step + 1, nsteps - 1), ml);
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) {
      if (masked) {
        // element e is token 8 gq + e of column 32 wave + 16 ct + lam
        const int bit = 16 * ct + lam;
#pragma unroll
        for (int d = 0; d < 4; ++d)
          x[ct][d] &= (((mu[2 * d] >> bit) & 1u) ? 0x0000ffffu : 0u) | (((mu[2 * d + 1] >> bit) & 1u) ? 0xffff0000u : 0u);
      }
#pragma unroll
      for (int jt = 0; jt < NJ; ++jt)
        acc[ct][jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(x[ct]), as_bf(qu[jt]), acc[ct][jt], 0, 0, 0);
    }
    if constexpr (GP) {
      if (wave < 2) {
        const char* bts = smem + 2 * STAGE;
        const int t = 16 * wave + lam;  // the lane's token row of the step (A-operand row)
        f32x4 ga[NJ];
#pragma unroll
        for (int jt = 0; jt < NJ; ++jt) ga[jt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 2
        for (int kc = 0; kc < kTokenCols / 32; ++kc) {
          const int c8 = 4 * kc + gq;  // the lane's 16-byte column chunk
          const u32x4 av = *reinterpret_cast<const u32x4*>(sb + t * (kTokenCols * 2) + 16 * (c8 ^ (2 * (t & 3))));
#pragma unroll
          for (int jt = 0; jt < NJ; ++jt) {
            const u32x4 bv = *reinterpret_cast<const u32x4*>(bts + (16 * jt + lam) * kBtRow + 16 * c8);
            ga[jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(av), as_bf(bv), ga[jt], 0, 0, 0);
          }
        }
        // ga[jt][v]: token 16 wave + 4 gq + v of the step, rank 16 jt + lam
        float* gp = g.gpart + ((int64_t)cb * g.gpart_n + begin) * g.r_max;
#pragma unroll
        for (int jt = 0; jt < NJ; ++jt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int tok = step * TS + 16 * wave + 4 * gq + v, j = 16 * jt + lam;
            if (tok < cnt && j < r) gp[(int64_t)tok * g.r_max + j] = ga[jt][v];
          }
      }
    }
  };
  u32x4 q0[NJ], q1[NJ];
  uint32_t m0[8] = {}, m1[8] = {};
  int p0[2], p1[2];
  if (nsteps > 0) {
    rows_of(0, p0);
    issue(0, 0, p0);
    rows_of(min(1, nsteps - 1), p0);
    load_q(0, q0);
    if (masked) load_mask(0, m0);
  }
  // p0 holds the rows of the next step to issue, p1 receives the one after
  for (int step = 0; step < nsteps; step += 2) {
    step_fn(step, q0, q1, m0, m1, p0, p1);
    if (step + 1 < nsteps) step_fn(step + 1, q1, q0, m1, m0, p1, p0);
  }
  // acc[ct][jt][v]: column 32 wave + 16 ct + 4 gq + v of the block, rank 16 jt + lam
  float* out = g.part + (int64_t)blockIdx.x * g.C * g.r_max;
#pragma unroll
  for (int ct = 0; ct < 2; ++ct)
#pragma unroll
    for (int jt = 0; jt < NJ; ++jt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int c = cbase + 32 * wave + 16 * ct + 4 * gq + v;
        const int j = 16 * jt + lam;
        if (j < r && c < g.C) out[(int64_t)c * g.r_max + j] = acc[ct][jt][v];
      }
}

// ---------------------------------------------------------------------------
// The same reductions without dropout, pipelined two steps deep, for Q rows
// that are 16-byte aligned (ldq a multiple of 8).  The step's Q tile (32
// tokens x 16 ranks per wave below NJ) goes into LDS by direct loads beside
// the P tile and is read back transposed like it, so no step has to combine
// scalar loads it just issued.  Two buffers, each a separate array picked by
// a compile-time number (a read of one buffer then never waits for the
// direct loads into the other).  Step s waits for its own loads only, every
// wave reads its fragments (GP: waves 0 and 1 also store the previous step's
// g partial and compute this step's from the buffer), a second barrier frees
// the buffer, and the direct loads of step s + 2 go into it before the
// MFMAs: two steps stay in flight per workgroup.  The direct loads are the
// last vector-memory operations of a step, and every wave issues three of
// them in every step, also for the two steps past the end (lanes and waves
// with nothing to load read a zero row, the spare waves into a scratch tile
// of the buffer), so the wait at the top of a step is always "all but the
// last three".  The chunk's P row numbers sit in LDS, loaded once.  Sums,
// their order and the results are those of token_reduce_kernel.
// ---------------------------------------------------------------------------
template <int V>
struct int_c {
  static constexpr int value = V;
};

__device__ __forceinline__ u32x2 tr_read16(const char* p) {
  const s16x4 h = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
  return u32x2{(uint32_t)(uint16_t)h[0] | ((uint32_t)(uint16_t)h[1] << 16),
               (uint32_t)(uint16_t)h[2] | ((uint32_t)(uint16_t)h[3] << 16)};
}

// Up to 16 ranks: six waves per SIMD, so that three workgroups share a CU
// (their LDS fits as well).
template <int NJ, bool GP>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(NJ == 1 ? 6 : 1))) void token_reduce_pipe_kernel(
    TokenReduceGroup G) {
  constexpr int TS = 32;                   // tokens per step
  constexpr int PB = TS * kTokenCols * 2;  // P bytes per step
  constexpr int QB = 1024;                 // Q bytes per step and 16 ranks
  constexpr int NLD = 3;                   // direct loads per wave and step
  // [P tile][Q tiles][spare tile]
  __shared__ __attribute__((aligned(256))) char st0[PB + (NJ + 1) * QB];
  __shared__ __attribute__((aligned(256))) char st1[PB + (NJ + 1) * QB];
  __shared__ __attribute__((aligned(16))) char bts[GP ? 16 * NJ * kBtRow : 16];
  __shared__ int32_t prl[kChunkRows];
  int k = 0;  // the reduction: blockIdx.y runs over every reduction's column blocks
  while (k + 1 < G.n && (int)blockIdx.y >= G.yoff[k + 1]) ++k;
  const TokenReduceArgs g = G.a[k];
  const int cb = (int)blockIdx.y - G.yoff[k], cbase = cb * kTokenCols;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int32_t* ck = g.chunks + (int64_t)blockIdx.x * kItemWords;
  const int a = ck[0], begin = ck[1], cnt = min(ck[2], kChunkRows);
  const int r = g.ranks[a];
  const int nsteps = (cnt + TS - 1) / TS;
  const int sub = lane >> 5, sl = lane & 31;  // staging: row within the instruction, slot
  const int gq = lane >> 4, lam = lane & 15;  // fragments: token octet, column / rank
  for (int i = tid; i < cnt; i += 512) prl[i] = g.prow ? g.prow[begin + i] : begin + i;
  __syncthreads();
  // P rows 2q + sub of the step (q = 2 wave + i), slot sl holding the row's
  // 16-byte chunk sl ^ 2(row % 4); wave w < NJ loads Q[token][16w .. 16w+15]
  // as [32 tokens][32 bytes], one token half per lane
  auto issue = [&](int step, char* sb) {
    const int t0 = step * TS;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = 2 * wave + i, row = 2 * q + sub;
      const int c = cbase + 8 * (sl ^ (2 * (row & 3)));
      const bool in = t0 + row < cnt && c < g.C;
      const void* from = in ? static_cast<const void*>(g.P + (int64_t)prl[max(min(t0 + row, cnt - 1), 0)] * g.ldp + c)
                            : static_cast<const void*>(&kZeroRow[lane]);
      llvm_amdgcn_global_load_lds((global_cv*)from, (lds_u32*)(sb + (q * 1024)), 16, 0, 0);
    }
    const int tq = lane >> 1, j0 = 16 * wave + 8 * (lane & 1);
    const bool in = wave < NJ && t0 + tq < cnt && j0 < g.ldq;
    const void* from = in ? static_cast<const void*>(g.Q + (int64_t)(begin + t0 + tq) * g.ldq + j0)
                          : static_cast<const void*>(&kZeroRow[lane]);
    llvm_amdgcn_global_load_lds((global_cv*)from, (lds_u32*)(sb + (PB + min(wave, NJ) * QB)), 16, 0, 0);
  };
  issue(0, st0);
  issue(1, st1);
  if constexpr (GP) {
    // B_a[c][j] of the block's columns into bts[j][c]; zero past the rank and
    // past C (published by the first step's barrier)
    const uint16_t* Ba = g.B + (int64_t)a * g.C * g.r_max;
    const bool b16 = (g.r_max & 7) == 0;  // a rank octet is one aligned 16-byte load
    for (int idx = tid; idx < kTokenCols * 2 * NJ; idx += 512) {
      const int cl = idx % kTokenCols, jo = idx / kTokenCols;  // column, rank octet
      const int c = cbase + cl, nv = min(8, r - 8 * jo);
      u32x4 v = zero4();
      if (c < g.C && nv > 0) {
        const uint16_t* src = Ba + (int64_t)c * g.r_max + 8 * jo;
        v = (b16 && nv == 8) ? ld16(src) : ld8_masked(src, 1, nv);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e)
        *reinterpret_cast<uint16_t*>(bts + (8 * jo + e) * kBtRow + 2 * cl) = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
    }
  }
  f32x4 acc[2][NJ], ga[NJ];
#pragma unroll
  for (int jt = 0; jt < NJ; ++jt) {
    acc[0][jt] = acc[1][jt] = f32x4{0.f, 0.f, 0.f, 0.f};
    ga[jt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // GP: the g partial of a step, ga[jt][v] = token 16 wave + 4 gq + v of the
  // step, rank 16 jt + lam (waves 0 and 1)
  auto gp_store = [&](int step) {
    if (wave < 2) {
      float* gp = g.gpart + ((int64_t)cb * g.gpart_n + begin) * g.r_max;
#pragma unroll
      for (int jt = 0; jt < NJ; ++jt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int tok = step * TS + 16 * wave + 4 * gq + v, j = 16 * jt + lam;
          if (tok < cnt && j < r) gp[(int64_t)tok * g.r_max + j] = ga[jt][v];
        }
    }
  };
  // Byte offsets of the lane's fragment reads within a buffer (every LDS
  // address below is one offset from its array: the compiler then tells the
  // two buffers apart and waits only for the loads into the one read).  The
  // token t = 8 gq + 4 hh + lam / 4 has t % 4 = lam / 4 for both halves hh,
  // so the second half is 4 rows (2048 bytes) further.
  int off_x[2];
#pragma unroll
  for (int ct = 0; ct < 2; ++ct) {
    const int t = 8 * gq + (lam >> 2);
    const int col = 32 * wave + 16 * ct + 4 * (lam & 3);  // within the block
    off_x[ct] = t * (kTokenCols * 2) + 16 * ((col >> 3) ^ (2 * (t & 3))) + 2 * (col & 7);
  }
  const int off_q = PB + (8 * gq + (lam >> 2)) * 32 + 8 * (lam & 3);
  // GP: row t = 16 wave + lam, chunk (4 kc + gq) ^ 2(t % 4) = 8(kc / 2) + ((4(kc % 2) + gq) ^ 2(t % 4))
  int off_av[2], off_bt[NJ];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int t = 16 * wave + lam;
    off_av[b] = t * (kTokenCols * 2) + 16 * ((4 * b + gq) ^ (2 * (t & 3)));
  }
#pragma unroll
  for (int jt = 0; jt < NJ; ++jt) off_bt[jt] = (16 * jt + lam) * kBtRow + 16 * gq;
  auto step_fn = [&](int step, auto bsel) {
    char* sb = decltype(bsel)::value ? st1 : st0;
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(NLD));
    // every wave's part of the step is in (a plain barrier: a fence would
    // also wait for the next step's loads)
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    // x[ct]: columns 32 wave + 16 ct + lam, tokens 8 gq + e (the A operand);
    // xq[jt]: rank 16 jt + lam, the same tokens (the B operand)
    u32x4 x[2], xq[NJ];
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) {
      const u32x2 h0 = tr_read16(sb + off_x[ct]), h1 = tr_read16(sb + (off_x[ct] + 4 * (kTokenCols * 2)));
      x[ct] = u32x4{h0[0], h0[1], h1[0], h1[1]};
    }
#pragma unroll
    for (int jt = 0; jt < NJ; ++jt) {
      const u32x2 h0 = tr_read16(sb + (off_q + jt * QB)), h1 = tr_read16(sb + (off_q + jt * QB + 4 * 32));
      xq[jt] = (16 * jt + lam < r) ? u32x4{h0[0], h0[1], h1[0], h1[1]} : zero4();
    }
    // GP, waves 0 and 1: store the previous step's g partial, then this
    // step's: the lane's token row 16 wave + lam of the step as it is (16
    // bytes = 8 columns per chunk) against B's columns, 8 contractions of 32
    // columns, read from the buffer before it is released
    if constexpr (GP) {
      if (step > 0) gp_store(step - 1);
      if (wave < 2) {
#pragma unroll
        for (int jt = 0; jt < NJ; ++jt) ga[jt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < kTokenCols / 32; ++kc) {
          const u32x4 av = *reinterpret_cast<const u32x4*>(sb + (off_av[kc & 1] + 128 * (kc >> 1)));
#pragma unroll
          for (int jt = 0; jt < NJ; ++jt) {
            const u32x4 bv = *reinterpret_cast<const u32x4*>(bts + (off_bt[jt] + 64 * kc));
            ga[jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(av), as_bf(bv), ga[jt], 0, 0, 0);
          }
        }
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");  // the buffer is free
    issue(step + 2, sb);  // zeros past the chunk
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int jt = 0; jt < NJ; ++jt)
        acc[ct][jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf(x[ct]), as_bf(xq[jt]), acc[ct][jt], 0, 0, 0);
  };
  // pairs of steps, then a last even one: every path into a step has the
  // other buffer's loads issued after this buffer's
  int step = 0;
  for (; step + 1 < nsteps; step += 2) {
    step_fn(step, int_c<0>{});
    step_fn(step + 1, int_c<1>{});
  }
  if (step < nsteps) step_fn(step, int_c<0>{});
  vmem_wait_all();  // the loads of the two steps past the end are in before the LDS is released
  if constexpr (GP) {
    if (nsteps > 0) gp_store(nsteps - 1);
  }
  // acc[ct][jt][v]: column 32 wave + 16 ct + 4 gq + v of the block, rank 16 jt + lam
  float* out = g.part + (int64_t)blockIdx.x * g.C * g.r_max;
#pragma unroll
  for (int ct = 0; ct < 2; ++ct)
#pragma unroll
    for (int jt = 0; jt < NJ; ++jt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int c = cbase + 32 * wave + 16 * ct + 4 * gq + v;
        const int j = 16 * jt + lam;
        if (j < r && c < g.C) out[(int64_t)c * g.r_max + j] = acc[ct][jt][v];
      }
}

// Fixed-order sum of one training adapter's chunk partials.
// Every final sum of a (grouped) backward in one launch: blockIdx.y = which *
// n_tads + training adapter (which: dB, dA of the first projection, then the
// next projection's).
__global__ __launch_bounds__(256) void reduce_out_kernel(ReduceOutGroup G, int32_t r_max, int32_t r_sel,
                                                         const int32_t* __restrict__ train_ads, int32_t n_tads,
                                                         const int32_t* __restrict__ tad_ptr,
                                                         const int32_t* __restrict__ tad_chunks,
                                                         const int32_t* __restrict__ ranks, int32_t accumulate) {
  const int which = (int)blockIdx.y / n_tads;
  const ReduceOutArgs g = G.a[which];
  const int ta = (int)blockIdx.y - which * n_tads;
  const int C = g.C;
  const int a = train_ads[ta], r = ranks[a];
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)C * r_sel) return;
  // j fastest, the partials' layout: the reads are coalesced in both output
  // layouts (the partials outweigh the output by the number of chunks); the
  // threads cover the ranks below r_sel (>= every training adapter's rank)
  const int c = (int)(idx / r_sel), j = (int)(idx % r_sel);
  if (c >= C || j >= r) return;
  // eight chunk partials in flight, added in chunk order (the same sum as one
  // at a time); the chunk ids are the same for the whole workgroup
  const float* src = g.part + (int64_t)c * r_max + j;
  const int64_t cs = (int64_t)C * r_max;
  const int p1 = tad_ptr[ta + 1];
  float sum = 0.f;
  int p = tad_ptr[ta];
  for (; p + 8 <= p1; p += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = src[tad_chunks[p + u] * cs];
#pragma unroll
    for (int u = 0; u < 8; ++u) sum += v[u];
  }
  for (; p < p1; ++p) sum += src[tad_chunks[p] * cs];
  if (g.scales) sum *= g.scales[a];
  sum *= g.post;
  float* o = g.a_layout ? g.out + ((int64_t)a * r_max + j) * C + c : g.out + ((int64_t)a * C + c) * r_max + j;
  *o = accumulate ? *o + sum : sum;
}

}  // namespace

namespace {
template <int MODE, int NJ, int ROWS, bool DROP>
void launch_skinny_kernel(const SkinnyGroup& g, int32_t n_items, int32_t ny, hipStream_t s) {
  hipLaunchKernelGGL((skinny_kernel<MODE, NJ, ROWS, DROP>), dim3(n_items, ny), dim3(64 * SW), 0, s, g);
}

template <int MODE, int ROWS, bool DROP>
void launch_skinny_nj(const SkinnyGroup& g, int32_t n_items, int32_t ny, int32_t r_max, hipStream_t s) {
  if (r_max <= 16) launch_skinny_kernel<MODE, 1, ROWS, DROP>(g, n_items, ny, s);
  else if (r_max <= 32) launch_skinny_kernel<MODE, 2, ROWS, DROP>(g, n_items, ny, s);
  else launch_skinny_kernel<MODE, 4, ROWS, DROP>(g, n_items, ny, s);
}

// Every projection of a group takes the dropout path or none does.  Each
// projection's contraction may be split into pieces (skinny_split); the pieces
// are launched longest first (workgroups are dispatched row by row of the
// grid), so the long ones start first and the short ones fill in behind them.
// Split projections need their partial buffer (part, part_n, r_max); a second
// launch sums their pieces.
template <int MODE, int ROWS>
hipError_t launch_skinny(const SkinnyGroup& g0, int32_t n_items, int32_t r_max, hipStream_t s) {
  if (n_items <= 0 || g0.n <= 0) return hipSuccess;
  if (g0.n > kMaxGroup || r_max < 1 || r_max > 64) return hipErrorInvalidValue;
  for (int p = 1; p < g0.n; ++p)
    if ((g0.a[p].keep != nullptr) != (g0.a[0].keep != nullptr)) return hipErrorInvalidValue;
  SkinnyGroup g = g0;
  for (int p = 0; p < g.n; ++p) {
    skinny_split(g.a[p].C, g.a[p].split_items, &g.a[p].pieces, &g.a[p].cpp);
    if (g.a[p].pieces > 1 && (g.a[p].part == nullptr || g.a[p].part_n < 0 || g.a[p].r_max < r_max))
      return hipErrorInvalidValue;
  }
  // stable insertion sort by chunks per piece, longest first (at most kMaxGroup
  // entries; no temporary buffer, so the allocation-free forward stays so)
  for (int p = 1; p < g.n; ++p) {
    const SkinnyArgs x = g.a[p];
    int q = p;
    for (; q > 0 && g.a[q - 1].cpp < x.cpp; --q) g.a[q] = g.a[q - 1];
    g.a[q] = x;
  }
  int ny = 0;
  for (int p = 0; p < g.n; ++p)
    for (int q = 0; q < g.a[p].pieces; ++q) {
      g.slot_proj[ny] = p;
      g.slot_piece[ny++] = q;
    }
  if constexpr (MODE == 0) {
    if (g.a[0].keep != nullptr) launch_skinny_nj<MODE, ROWS, true>(g, n_items, ny, r_max, s);
    else launch_skinny_nj<MODE, ROWS, false>(g, n_items, ny, r_max, s);
  } else {
    launch_skinny_nj<MODE, ROWS, false>(g, n_items, ny, r_max, s);
  }
  int nf = 0;
  for (int p = 0; p < g.n; ++p)
    if (g.a[p].pieces > 1) g.slot_proj[nf++] = p;
  if (nf > 0) hipLaunchKernelGGL((skinny_finish_kernel<MODE>), dim3(n_items, nf), dim3(256), 0, s, g);
  return hipGetLastError();
}

SkinnyGroup one(const SkinnyArgs& a) {
  SkinnyGroup g{};
  g.a[0] = a;
  g.n = 1;
  return g;
}
}  // namespace

hipError_t launch_shrink(const SkinnyArgs& a, int32_t n_items, int32_t r_max, hipStream_t s) {
  return launch_skinny<0, kRankItemRows>(one(a), n_items, r_max, s);
}

hipError_t launch_shrink_train(const SkinnyArgs& a, int32_t n_items, int32_t r_max, hipStream_t s) {
  return launch_skinny<0, kItemRows>(one(a), n_items, r_max, s);
}

hipError_t launch_shrink_group(const SkinnyGroup& g, int32_t n_items, int32_t r_max, hipStream_t s) {
  return launch_skinny<0, kRankItemRows>(g, n_items, r_max, s);
}

hipError_t launch_shrink_train_group(const SkinnyGroup& g, int32_t n_items, int32_t r_max, hipStream_t s) {
  return launch_skinny<0, kItemRows>(g, n_items, r_max, s);
}

hipError_t launch_gather_group(const GatherGroup& g, int64_t ldh, int32_t r_max, const int32_t* items,
                               int32_t n_items, const int32_t* gather_rows, const int32_t* ranks,
                               const float* scales, hipStream_t s) {
  if (n_items <= 0 || g.n <= 0) return hipSuccess;
  if (g.n > kMaxGroup || g.yoff[0] != 0) return hipErrorInvalidValue;
  for (int p = 0; p < g.n; ++p)
    if (g.yoff[p + 1] - g.yoff[p] != (g.a[p].N + 255) / 256) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_expand_kernel, dim3(n_items, g.yoff[g.n]), dim3(256), 0, s, g, ldh, r_max, items,
                     gather_rows, ranks, scales);
  return hipGetLastError();
}

hipError_t launch_gather_expand(const uint16_t* H, int64_t ldh, const uint16_t* B, int32_t N,
                                int32_t r_max, const int32_t* items, int32_t n_items,
                                const int32_t* gather_rows, const int32_t* ranks,
                                const float* scales, float* delta, hipStream_t s) {
  GatherGroup g{};
  g.a[0] = GatherArgs{H, B, N, delta};
  g.yoff[1] = (N + 255) / 256;
  g.n = 1;
  return launch_gather_group(g, ldh, r_max, items, n_items, gather_rows, ranks, scales, s);
}

template <bool DROP, bool GP>
void launch_token_reduce_nj(const TokenReduceGroup& g, int32_t n_chunks, int32_t r_sel, hipStream_t s) {
  const dim3 grid(n_chunks, g.yoff[g.n]);
  // the pipelined kernel when every reduction's Q rows are 16-byte aligned
  bool q16 = !DROP;
  for (int k = 0; k < g.n; ++k)
    q16 = q16 && (g.a[k].ldq & 7) == 0 && (reinterpret_cast<uintptr_t>(g.a[k].Q) & 15) == 0;
  if (q16) {
    if (r_sel <= 16)
      hipLaunchKernelGGL((token_reduce_pipe_kernel<1, GP>), grid, dim3(512), 0, s, g);
    else if (r_sel <= 32)
      hipLaunchKernelGGL((token_reduce_pipe_kernel<2, GP>), grid, dim3(512), 0, s, g);
    else
      hipLaunchKernelGGL((token_reduce_pipe_kernel<4, GP>), grid, dim3(512), 0, s, g);
    return;
  }
  if (r_sel <= 16)
    hipLaunchKernelGGL((token_reduce_kernel<1, DROP, GP>), grid, dim3(512), 0, s, g);
  else if (r_sel <= 32)
    hipLaunchKernelGGL((token_reduce_kernel<2, DROP, GP>), grid, dim3(512), 0, s, g);
  else
    hipLaunchKernelGGL((token_reduce_kernel<4, DROP, GP>), grid, dim3(512), 0, s, g);
}

// A launch whose reductions include a masked one runs the kernel with the
// masking code; it masks the reductions that carry a mask.  A launch of
// reductions that carry B (the dB side) also writes the g partials.
hipError_t launch_token_reduce_group(const TokenReduceGroup& g, int32_t n_chunks, int32_t r_sel, hipStream_t s) {
  if (n_chunks <= 0 || g.n <= 0) return hipSuccess;
  if (g.n > 2 * kMaxGroup || g.yoff[0] != 0 || r_sel < 1 || r_sel > g.a[0].r_max) return hipErrorInvalidValue;
  bool any_keep = false;
  int n_b = 0;
  for (int k = 0; k < g.n; ++k) {
    if (g.a[k].r_max != g.a[0].r_max || g.yoff[k + 1] - g.yoff[k] != token_col_blocks(g.a[k].C))
      return hipErrorInvalidValue;
    any_keep |= g.a[k].keep != nullptr;
    if (g.a[k].B != nullptr) {
      if (g.a[k].gpart == nullptr || g.a[k].gpart_n < 1) return hipErrorInvalidValue;
      ++n_b;
    }
  }
  if (n_b != 0 && (n_b != g.n || any_keep)) return hipErrorInvalidValue;
  if (n_b) launch_token_reduce_nj<false, true>(g, n_chunks, r_sel, s);
  else if (any_keep) launch_token_reduce_nj<true, false>(g, n_chunks, r_sel, s);
  else launch_token_reduce_nj<false, false>(g, n_chunks, r_sel, s);
  return hipGetLastError();
}

hipError_t launch_g_finish_group(const SkinnyGroup& g0, int32_t n_items, hipStream_t s) {
  if (n_items <= 0 || g0.n <= 0) return hipSuccess;
  if (g0.n > kMaxGroup) return hipErrorInvalidValue;
  SkinnyGroup g = g0;
  for (int p = 0; p < g.n; ++p) {
    if (g.a[p].part == nullptr || g.a[p].pieces < 1 || g.a[p].out1 == nullptr) return hipErrorInvalidValue;
    g.slot_proj[p] = p;
  }
  hipLaunchKernelGGL((skinny_finish_kernel<1>), dim3(n_items, g.n), dim3(256), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_reduce_out_group(const ReduceOutGroup& g, int32_t r_max, int32_t r_sel, const int32_t* train_ads,
                                   int32_t n_tads, const int32_t* tad_ptr, const int32_t* tad_chunks,
                                   const int32_t* ranks, int32_t accumulate, hipStream_t s) {
  if (n_tads <= 0 || g.n <= 0) return hipSuccess;
  if (g.n > 2 * kMaxGroup || r_sel < 1 || r_sel > r_max) return hipErrorInvalidValue;
  int64_t cmax = 0;
  for (int k = 0; k < g.n; ++k) cmax = g.a[k].C > cmax ? g.a[k].C : cmax;
  const int64_t total = cmax * r_sel;
  hipLaunchKernelGGL(reduce_out_kernel, dim3((unsigned)((total + 255) / 256), g.n * n_tads), dim3(256), 0, s, g,
                     r_max, r_sel, train_ads, n_tads, tad_ptr, tad_chunks, ranks, accumulate);
  return hipGetLastError();
}

hipError_t launch_reduce_out(const ReduceOutArgs& o0, const ReduceOutArgs& o1, int32_t r_max, int32_t r_sel,
                             const int32_t* train_ads, int32_t n_tads, const int32_t* tad_ptr,
                             const int32_t* tad_chunks, const int32_t* ranks, int32_t accumulate, hipStream_t s) {
  ReduceOutGroup g{};
  g.a[0] = o0;
  g.a[1] = o1;
  g.n = 2;
  return launch_reduce_out_group(g, r_max, r_sel, train_ads, n_tads, tad_ptr, tad_chunks, ranks, accumulate, s);
}

}  // namespace dsv
