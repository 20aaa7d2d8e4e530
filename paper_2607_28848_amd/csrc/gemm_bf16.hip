// gemm_bf16.hip -- CDNA4 (gfx950) GEMM kernels of the co-batched multi-LoRA
// layer in bf16 with fp32 accumulation (Sec. 2.2 multi-LoRA batching, Sec. 3.2
// mixed forward batch and backward of the training rows):
//   forward (NT)     y = x W^T on the matrix cores; the tile's own adapter
//                    groups add s_a h B_a^T in the prologue, gathered rows add
//                    their fp32 term; one rounding to bf16 at the end.
//   dX (NT / NN)     dx = dy W + g A_a (the prologue adds g A_a), on the
//                    transposed weight (NT) or on W itself (NN).
//   split fixup      sums the pieces of contraction-split tiles.
// plus the GEMM launchers and their benchmark timing.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "device_common.h"
#include "kernels.h"
#include "plan.h"

namespace dsv {
namespace {

// ---------------------------------------------------------------------------
// GEMM with a low-rank prologue.  TM x TN output tile per workgroup: 256x256
// (8 waves in a 2 x 4 grid, each wave 128 x 64) or 128x128 (4 waves in a 2 x 2
// grid, each 64 x 64), FM x FN tiles of v_mfma_f32_32x32x16_bf16 per wave.
// K-steps of 64.
//
// Operand tiles go from global memory straight into LDS (buffer loads with
// the LDS destination, 16 bytes per lane, one contiguous KiB per wave
// instruction), double-buffered, one barrier per K-step.  Lanes are assigned
// global chunks so that the LDS image is swizzled:
//   K-contiguous tiles ([rows][64] bf16, 128-byte rows): 16-byte chunk c of
//   row r sits in slot c ^ swz(r); MFMA fragments are 16-byte reads.
//   N-contiguous weight tile of the dX GEMM ([64][TN] bf16): chunk c of row n
//   sits in slot c ^ 2(n & 3); fragments are read with ds_read_b64_tr_b16,
//   which hands each lane 4 contraction values of one output column.
// Both read patterns are free of bank conflicts.  Out-of-range lanes point
// past the buffer descriptor's range and receive zeros.
// ---------------------------------------------------------------------------
extern "C" __device__ void llvm_amdgcn_raw_buffer_load_lds(i32x4 rsrc, lds_u32* lds, int size,
                                                           int voffset, int soffset, int offset,
                                                           int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

// Buffer descriptor: 64-bit base, byte range, CDNA data-format word.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, uint64_t range) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t rg = range > 0xFFFFFFF0ull ? 0xFFFFFFF0u : (uint32_t)range;
  i32x4 r;
  r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r.y = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
  r.z = __builtin_amdgcn_readfirstlane((int)rg);
  r.w = 0x00020000;
  return r;
}

// K-contiguous tiles hold rows of TK bf16 (TK / 8 chunks of 16 bytes); the
// chunk slot is XOR-swizzled with a function of the row so that the 16 lanes
// of one LDS access phase (16 consecutive rows, same logical chunk) hit
// distinct banks.
template <int TK>
__device__ __forceinline__ int swz(int row) {
  if constexpr (TK == 64) return (row ^ (row >> 3)) & 7;
  else return (row >> 2) & 3;
}
__device__ __forceinline__ int nn_swz(int n) { return 2 * (n & 3); }

template <int TM, int TN, int WGM, int WGN, int TK, int NS>
struct GemmShape {
  static constexpr int NW = WGM * WGN, THREADS = 64 * NW;
  static constexpr int WM = TM / WGM, WN = TN / WGN, FM = WM / 32, FN = WN / 32;
  static constexpr int A_BYTES = TM * TK * 2, B_BYTES = TN * TK * 2;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int LDS = NS * STAGE;
};

// A compile-time flag passed as a value (selects a generic lambda's form).
template <bool B>
struct bool_c {
  static constexpr bool value = B;
};

// Workgroup id -> logical index.  Consecutive workgroup ids land on different
// XCDs (round robin over 8); the renumbering gives each XCD a contiguous
// range of logical indices, so work that runs together on one XCD is
// adjacent in the tile order and shares operand panels in that XCD's L2.
__device__ __forceinline__ int xcd_major(int bid, int n) {
  const int per = n >> 3, rem = n & 7, xcd = bid & 7;
  return xcd * per + min(xcd, rem) + (bid >> 3);
}

// Tile -> (row tile, column tile): groups of 4 row tiles are walked column by
// column, so tiles in flight together share row and column panels (4 measured
// faster than 2, 8 or 16 on the Llama-3-8B layer set).
__device__ __forceinline__ void tile_coords(const GemmArgs& g, int lin, int& mt, int& nt) {
  const int GM = 4;
  const int span = GM * g.n_ntiles;
  const int grp = lin / span, first_m = grp * GM;
  const int gsz = min(g.n_mtiles - first_m, GM);
  mt = first_m + (lin % span) % gsz;
  nt = (lin % span) / gsz;
}

// One piece of a tile: K-steps [kb, ke) of tile `lin`.  A piece that covers
// the whole K range writes the tile; a piece of a split tile (t_sk: its index
// among the split tiles) writes its fp32 partial to slot t_sk * split + piece.
template <bool NN, int TM, int TN, int WGM, int WGN, int TK, int NS, bool SK>
__device__ __forceinline__ void gemm_piece(const GemmArgs& g, char* smem, int tid, int lin,
                                           int t_sk, int piece, int kb, int ke, int nk) {
  using S = GemmShape<TM, TN, WGM, WGN, TK, NS>;
  constexpr int WM = S::WM, WN = S::WN, FM = S::FM, FN = S::FN, NW = S::NW;
  constexpr int ROWB = TK * 2;          // bytes per row of a K-contiguous tile
  constexpr int CPR = TK / 8;           // 16-byte chunks per row
  // With 8 waves (two per SIMD) the operand loads of a K-step are all issued
  // by waves 0-3, one per SIMD: a wave whose load issue stalls on the
  // texture-address queue holds back its own later MFMAs, and the other wave
  // of its SIMD, which issues no loads, keeps the matrix core busy meanwhile.
  constexpr int LW = NW >= 8 ? NW / 2 : NW;  // loading waves
  constexpr int A_LOADS = TM * ROWB / 1024 / LW, B_LOADS = TN * ROWB / 1024 / LW;
  static_assert(A_LOADS * 1024 * LW == TM * ROWB && B_LOADS * 1024 * LW == TN * ROWB, "loads per wave");
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;

  int mt, nt;
  tile_coords(g, lin, mt, nt);

  const int32_t* td = g.tiles + (int64_t)mt * kTileWords;
  const int m0 = td[0], ngroups = td[1], has_gather = td[2], nrows = td[3];
  const int n0 = nt * TN;
  const uint16_t* a_base = g.P + (int64_t)m0 * g.ldp;
  const int64_t a_rows = min((int64_t)TM, (int64_t)g.M - m0);
  const uint16_t* b_base = NN ? g.Q + n0 : g.Q + (int64_t)n0 * g.ldq;
  const int64_t b_cols = min((int64_t)TN, (int64_t)g.Nout - n0);

  // Direct-to-LDS loads of K-step kt into stage `stage`.
  //
  // Large tiles (8+ accumulator tiles per wave, all loads issued by waves
  // 0..LW-1, 8+ loads of each operand per wave): the per-lane offsets are
  // recomputed here from a freshly read lane id -- held in registers across
  // the main loop they would be spilled -- in a form that costs a few VALU
  // operations per load.  With q = wave * LOADS + i, LOADS a multiple of 8:
  //   K-contiguous tile (8 rows of 64 per 1 KiB load): row = 8q + ln/8 and the
  //     chunk swizzle is (ln%8) ^ (ln/8) ^ (i%8), so the lane part is fixed
  //     and i only selects a constant XOR;
  //   N-contiguous dX weight tile (2 rows of 256 per load): n = 2q + ln/32 and
  //     the slot swizzle is (ln%32) ^ 2(ln/32) ^ 4(i%2).
  // Only the last, partial K-step checks the contraction bound per lane.
  // Other tiles keep the offsets in registers.
  auto issue = [&](int kt, int stage) {
    if (LW < NW && wave >= LW) return;
    const int k0 = kt * TK;
    char* sa = smem + stage * S::STAGE;
    char* sb = sa + S::A_BYTES;
    // descriptors rebased on the K-step keep every offset well inside 32 bits
    const i32x4 ra = make_rsrc(a_base + k0, (uint64_t)(a_rows * g.ldp - k0) * 2);
    constexpr bool kFast = FM * FN >= 8 && TK == 64 && A_LOADS % 8 == 0 && B_LOADS % 8 == 0 && (!NN || TN == 256);
    if (kFast && k0 + TK <= g.C) {  // every K-step but a partial last one
      int ln;
      asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
      const int lr = ln >> 3, x16 = ((ln & 7) ^ lr) << 4;
      const int lpa = lr * (int)g.ldp * 2;
#pragma unroll
      for (int i = 0; i < A_LOADS; ++i) {
        const int q = wave * A_LOADS + i;
        const int sq = __builtin_amdgcn_readfirstlane(q * 16 * (int)g.ldp);  // row block: scalar
        llvm_amdgcn_raw_buffer_load_lds(ra, (lds_u32*)(sa + q * 1024), 16, (x16 ^ ((i & 7) << 4)) + lpa + sq,
                                        0, 0, 0);
      }
      if constexpr (!NN) {
        const i32x4 rb = make_rsrc(b_base + k0, (uint64_t)(b_cols * g.ldq - k0) * 2);
        const int lpb = lr * (int)g.ldq * 2;
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
          const int q = wave * B_LOADS + i;
          const int sq = __builtin_amdgcn_readfirstlane(q * 16 * (int)g.ldq);
          llvm_amdgcn_raw_buffer_load_lds(rb, (lds_u32*)(sb + q * 1024), 16, (x16 ^ ((i & 7) << 4)) + lpb + sq,
                                          0, 0, 0);
        }
      } else {
        const i32x4 rb = make_rsrc(b_base + (int64_t)k0 * g.ldq, (uint64_t)((int64_t)TK * g.ldq - n0) * 2);
        const int h = ln >> 5, y16 = ((ln & 31) ^ (2 * h)) << 4;
        const int lpb = h * (int)g.ldq * 2;
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
          const int q = wave * B_LOADS + i;
          const int sq = __builtin_amdgcn_readfirstlane(q * 4 * (int)g.ldq);
          llvm_amdgcn_raw_buffer_load_lds(rb, (lds_u32*)(sb + q * 1024), 16, (y16 ^ ((i & 1) << 6)) + lpb + sq,
                                          0, 0, 0);
        }
      }
    } else {
      int ln = lane;
      if constexpr (kFast)
        asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
#pragma unroll
      for (int i = 0; i < A_LOADS; ++i) {
        const int q = wave * A_LOADS + i;
        const int row = q * (1024 / ROWB) + ln / CPR;
        const int c = (ln % CPR) ^ swz<TK>(row);
        const int vo = (k0 + 8 * c < g.C) ? (row * (int)g.ldp + 8 * c) * 2 : (int)0x7FFFFFF0;
        llvm_amdgcn_raw_buffer_load_lds(ra, (lds_u32*)(sa + q * 1024), 16, vo, 0, 0, 0);
      }
      if constexpr (!NN) {
        const i32x4 rb = make_rsrc(b_base + k0, (uint64_t)(b_cols * g.ldq - k0) * 2);
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
          const int q = wave * B_LOADS + i;
          const int col = q * (1024 / ROWB) + ln / CPR;
          const int c = (ln % CPR) ^ swz<TK>(col);
          const int vo = (k0 + 8 * c < g.C) ? (col * (int)g.ldq + 8 * c) * 2 : (int)0x7FFFFFF0;
          llvm_amdgcn_raw_buffer_load_lds(rb, (lds_u32*)(sb + q * 1024), 16, vo, 0, 0, 0);
        }
      } else {
        // the TK contraction rows of this K-step (fewer at the tail)
        const i32x4 rb = make_rsrc(b_base + (int64_t)k0 * g.ldq,
                                   (uint64_t)((int64_t)min(TK, g.C - k0) * g.ldq - n0) * 2);
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
          const int q = wave * B_LOADS + i;
          const int byte = q * 1024 + 16 * ln;
          const int n = byte / (TN * 2), slot = (byte % (TN * 2)) / 16;
          const int vo = (k0 + n < g.C) ? (n * (int)g.ldq + 8 * (slot ^ nn_swz(n))) * 2 : (int)0x7FFFFFF0;
          llvm_amdgcn_raw_buffer_load_lds(rb, (lds_u32*)(sb + q * 1024), 16, vo, 0, 0, 0);
        }
      }
    }
  };

  // The first NS K-steps are in flight while the low-rank prologue runs.
#pragma unroll
  for (int p = 0; p < NS; ++p)
    if (kb + p < ke) issue(kb + p, p);

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // ---- low-rank prologue (the piece that starts the tile's K range) -----
  // acc += (s_a h) B_a for the rows of each group.  s_a h is formed in fp32
  // and split into bf16 hi + lo (|lo| <= 2^-9 |hi|), so the product carries
  // the scale to about 2^-16 relative with no VALU work on the accumulators;
  // with scale 1 (or a power of two) lo is exactly zero and is skipped.
  for (int gi = 0; kb == 0 && gi < ngroups; ++gi) {
    const int a = td[4 + 3 * gi], lo = td[5 + 3 * gi], hi = td[6 + 3 * gi];
    if (hi <= wm * WM || lo >= wm * WM + WM) continue;  // no row of this wave
    const int r = g.ranks[a];
    const float sc = g.scales ? g.scales[a] : 1.f;
    const uint16_t* lq = g.Lq + (int64_t)a * g.lq_ad;
    // Loads are straight-line: lanes outside the group's rows, past the rank or
    // past the columns read a valid element (row lo, rank 0, the last column)
    // and drop it.  With r a multiple of 16 every lane's 8 ranks are valid, and
    // the h rows (and, for contiguous ranks with an 8-aligned stride, the B
    // rows) are read 16 bytes at a time.
    const bool full16 = (r & 15) == 0;
    const bool lq_vec = full16 && g.lq_j == 1 && (g.lq_col & 7) == 0;
    for (int j0 = 0; j0 < r; j0 += 16) {
      const int jb = j0 + 8 * (lane >> 5);
      const int nv = min(8, r - jb);
      const int jbc = nv > 0 ? jb : 0, nvc = max(nv, 1);
      bf16x8 af_hi[FM], af_lo[FM], bq[FN];
      bool any_lo = false;
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = wm * WM + 32 * i + (lane & 31);
        const bool rin = row >= lo && row < hi && nv > 0;
        const uint16_t* p = g.Lp + (int64_t)(m0 + (rin ? row : lo)) * g.ldl + jbc;
        u32x4 v = full16 ? ld16(p) : ld8_sel(p, 1, nvc);
        v = rin ? v : zero4();
        uint32_t wh[4], wl[4];
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const float x0 = sc * __uint_as_float(v[d] << 16);
          const float x1 = sc * __uint_as_float(v[d] & 0xffff0000u);
          const uint16_t h0 = f2bf(x0), h1 = f2bf(x1);
          const uint16_t l0 = f2bf(x0 - bf2f(h0)), l1 = f2bf(x1 - bf2f(h1));
          wh[d] = (uint32_t)h0 | ((uint32_t)h1 << 16);
          wl[d] = (uint32_t)l0 | ((uint32_t)l1 << 16);
          any_lo |= (wl[d] & 0x7fff7fffu) != 0u;
        }
        af_hi[i] = as_bf(u32x4{wh[0], wh[1], wh[2], wh[3]});
        af_lo[i] = as_bf(u32x4{wl[0], wl[1], wl[2], wl[3]});
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = n0 + wn * WN + 32 * j + (lane & 31);
        const bool cin = col < g.Nout && nv > 0;
        const uint16_t* p = lq + (int64_t)jbc * g.lq_j + (int64_t)min(col, g.Nout - 1) * g.lq_col;
        u32x4 v = lq_vec ? ld16(p) : ld8_sel(p, g.lq_j, nvc);
        bq[j] = as_bf(cin ? v : zero4());
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bq[j], af_hi[i], acc[i][j], 0, 0, 0);
      if (__builtin_amdgcn_ballot_w64(any_lo) != 0) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bq[j], af_lo[i], acc[i][j], 0, 0, 0);
      }
    }
  }

  // ---- dropout of the low-rank term (dX under LoRA dropout) --------------
  // The prologue left g A_a in the accumulators; it passes through the input's
  // mask before dy W is added: kept elements scaled by 1 / (1 - p), dropped
  // ones zeroed.  A lane holds one row and 16 columns of each 32 x 32 block,
  // all inside one 32-column mask word: one word per block.
  if (kb == 0 && g.keep != nullptr) {  // dX GEMMs only (the forward passes no mask)
    const int wcol = (n0 + wn * WN) >> 5;  // first mask word of the wave's columns
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WM + 32 * i + (lane & 31);
      uint32_t mw[FN];
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const uint32_t x = g.keep[(int64_t)(m0 + min(row, nrows - 1)) * g.keep_words + min(wcol + j, g.keep_words - 1)];
        // arithmetic masking keeps the load unconditional (a select would let the
        // compiler move it under a branch with a wait of its own)
        mw[j] = x & (0u - (uint32_t)(row < nrows && wcol + j < g.keep_words));
      }
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int bit = 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
          acc[i][j][v] = ((mw[j] >> bit) & 1u) ? acc[i][j][v] * g.keep_scale : 0.f;
        }
    }
  }

  // ---- main loop ----------------------------------------------------------
  // Fragment reads in the order the MFMAs consume them (weight column block
  // j outer, row block i inner): bq[0], af[0..FM), then bq[1..FN), so the first
  // MFMA of a 16-wide step waits for two reads, not for all of them.
  auto load_frags = [&](const char* sa, const char* sb, int s, bf16x8* af, bf16x8* bq) {
    const int ch = 2 * s + (lane >> 5);
    auto read_a = [&](int i) {
      const int row = wm * WM + 32 * i + (lane & 31);
      af[i] = as_bf(*reinterpret_cast<const u32x4*>(sa + row * ROWB + 16 * (ch ^ swz<TK>(row))));
    };
    auto read_b = [&](int j) {
      if constexpr (!NN) {
        const int col = wn * WN + 32 * j + (lane & 31);
        bq[j] = as_bf(*reinterpret_cast<const u32x4*>(sb + col * ROWB + 16 * (ch ^ swz<TK>(col))));
      } else {
        const int gq = lane >> 4, lam = lane & 15;
        const int c = wn * WN + 32 * j + 16 * (gq & 1) + 4 * (lam & 3);
        s16x4 h[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int n = 16 * s + 8 * (gq >> 1) + 4 * hh + (lam >> 2);
          const char* p = sb + n * (TN * 2) + 16 * ((c >> 3) ^ nn_swz(n)) + 2 * (c & 7);
          h[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
        }
        u32x4 v;
        v[0] = (uint32_t)(uint16_t)h[0][0] | ((uint32_t)(uint16_t)h[0][1] << 16);
        v[1] = (uint32_t)(uint16_t)h[0][2] | ((uint32_t)(uint16_t)h[0][3] << 16);
        v[2] = (uint32_t)(uint16_t)h[1][0] | ((uint32_t)(uint16_t)h[1][1] << 16);
        v[3] = (uint32_t)(uint16_t)h[1][2] | ((uint32_t)(uint16_t)h[1][3] << 16);
        bq[j] = as_bf(v);
      }
    };
    read_b(0);
#pragma unroll
    for (int i = 0; i < FM; ++i) read_a(i);
#pragma unroll
    for (int j = 1; j < FN; ++j) read_b(j);
  };

  // Pipeline: NS K-steps in flight.  In iteration kt the barrier that
  // publishes step kt+1 sits before the last 16-wide MFMA step of kt (whose
  // fragments are already in registers).  After it the buffer of kt is free
  // and receives step kt+NS, and the first fragments of kt+1 are read while
  // the last MFMAs of kt issue.
  constexpr int kLoads = A_LOADS + B_LOADS;          // direct loads per wave per K-step
  constexpr int kReads = FM + (NN ? 2 : 1) * FN;     // LDS reads per 16-wide step
  constexpr int kMfma = FM * FN;                     // MFMAs per 16-wide step
  constexpr int kSteps = TK / 16;
  constexpr int L = (kSteps - 1) & 1;  // fragment buffer of the last step
  static_assert(L == 1, "an even number of 16-wide steps per K-step");
  if (ke - kb >= NS) __builtin_amdgcn_s_waitcnt(vmcnt_imm((NS - 1) * kLoads));  // first step landed
  else vmem_wait_all();
  __syncthreads();
  bf16x8 af[2][FM], bq[2][FN];
  load_frags(smem, smem + S::A_BYTES, 0, af[0], bq[0]);
  int stage = 0;
  for (int kt = kb; kt < ke; ++kt) {
    char* sa = smem + stage * S::STAGE;
    char* sb = sa + S::A_BYTES;
#pragma unroll
    for (int s = 0; s < kSteps - 1; ++s) {
      load_frags(sa, sb, s + 1, af[(s + 1) & 1], bq[(s + 1) & 1]);
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bq[s & 1][j], af[s & 1][i], acc[i][j], 0, 0, 0);
    }
#pragma unroll
    for (int s = 0; s < kSteps - 1; ++s) {
#pragma unroll
      for (int q = 0; q < kReads; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      if (kMfma > kReads) __builtin_amdgcn_sched_group_barrier(0x008, kMfma - kReads, 0);
    }
    const int next = (stage + 1 == NS) ? 0 : stage + 1;
    if (kt + 1 < ke) {
      // step kt+1 has landed once at most (steps issued after it) loads remain
      if (kt + NS <= ke) __builtin_amdgcn_s_waitcnt(vmcnt_imm((NS - 2) * kLoads));
      else vmem_wait_all();
      __syncthreads();  // everyone's part of kt+1 is in; buffer `stage` is free
      if (kt + NS < ke) issue(kt + NS, stage);
      char* na = smem + next * S::STAGE;
      load_frags(na, na + S::A_BYTES, 0, af[L ^ 1], bq[L ^ 1]);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int i = 0; i < FM; ++i)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bq[L][j], af[L][i], acc[i][j], 0, 0, 0);
    stage = next;
  }

  // Accumulator layout (the MFMAs take the weight fragment as their first
  // operand): acc[i][j][v] is output row wm*WM + 32i + lane%32, column
  // wn*WN + 32j + 8(v/4) + 4(lane/32) + v%4 -- four consecutive columns of one
  // row per group of four v.

  // ---- a piece of a split tile: its fp32 partial goes to its slot (row-major
  // tm x tn); a follow-up kernel sums the pieces and writes the tile ----
  if (SK && !(kb == 0 && ke == nk)) {
    float* part = g.sk_part + (int64_t)(t_sk * g.sk_split + piece) * (TM * TN);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WM + 32 * i + (lane & 31);
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = wn * WN + 32 * j + 8 * q + 4 * (lane >> 5);
          *reinterpret_cast<f32x4*>(part + row * TN + col) =
              f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        }
    }
    return;
  }

  // ---- epilogue: one rounding, staged through LDS for 16-byte stores ----
  // Each wave stages its own rows, 32 at a time, in a private slice of the
  // pipeline buffer that the last K-step did not use (no wave reads it again),
  // so no workgroup barrier is needed: a lane writes 4 columns (8 bytes) of its
  // row, then the wave reads the slice back as 16-byte row chunks and stores
  // whole 128-byte row segments.  The slice row stride (WN + 4 elements, 2
  // dwords past a multiple of 32 banks) keeps the 8-byte writes of 16
  // consecutive rows on distinct banks.
  constexpr int SRS = WN * 2 + 8;  // slice row stride in bytes
  static_assert(NS == 2 && NW * 32 * SRS <= S::STAGE, "epilogue slices fit the idle pipeline buffer");
  char* slice = smem + ((ke - kb) & 1) * S::STAGE + wave * 32 * SRS;
  const bool gathered = has_gather && g.delta != nullptr;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int row = wm * WM + 32 * i + (lane & 31);
    const int gs = (gathered && row < nrows) ? g.gslot[m0 + row] : -1;
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int col = wn * WN + 32 * j + 8 * q + 4 * (lane >> 5);
        f32x4 x = f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        // rows of the gathered path add their fp32 low-rank term before the
        // rounding (a straight-line load from a clamped address, then a select)
        if (gathered) {
          const f32x4 d = *reinterpret_cast<const f32x4*>(g.delta + (int64_t)max(gs, 0) * g.Nout +
                                                          min(n0 + col, g.Nout - 4));
          x += (gs >= 0 && n0 + col < g.Nout) ? d : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        const uint32_t w0 = f2bf2(x[0], x[1]), w1 = f2bf2(x[2], x[3]);
        *reinterpret_cast<uint2*>(slice + (lane & 31) * SRS + 2 * (col - wn * WN)) = make_uint2(w0, w1);
      }
    asm volatile("" ::: "memory");  // a wave's LDS accesses run in order: the slice is complete
    constexpr int CPR = WN / 8;  // 16-byte chunks per slice row
#pragma unroll
    for (int q = 0; q < 32 * CPR / 64; ++q) {
      const int id = 64 * q + lane;
      const int rr = id / CPR, ch = id % CPR;
      const uint2 lo = *reinterpret_cast<const uint2*>(slice + rr * SRS + 16 * ch);
      const uint2 hi = *reinterpret_cast<const uint2*>(slice + rr * SRS + 16 * ch + 8);
      const int orow = wm * WM + 32 * i + rr, ocol = n0 + wn * WN + 8 * ch;
      // streaming stores: the output is not read again by this launch, so its
      // lines should not displace the operand panels the XCD's tiles share in L2
      if (orow < nrows && ocol < g.Nout)
        __builtin_nontemporal_store(u32x4{lo.x, lo.y, hi.x, hi.y},
                                    reinterpret_cast<u32x4*>(g.out + (int64_t)(m0 + orow) * g.ldo + ocol));
    }
    asm volatile("" ::: "memory");  // the slice is read before the next rows overwrite it
  }
}

template <bool NN, int TM, int TN, int WGM, int WGN, int TK, int NS, bool SK>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_lora_kernel(GemmArgs g) {
  using S = GemmShape<TM, TN, WGM, WGN, TK, NS>;
  static_assert(S::FM >= 1 && S::FN >= 1 && NS >= 2, "tile shape");
  static_assert((TM * TK * 2) % (1024 * S::NW) == 0 && (TN * TK * 2) % (1024 * S::NW) == 0, "loads per wave");
  __shared__ __attribute__((aligned(1024))) char smem[S::LDS];
  const int tid0 = threadIdx.x;
  const int nk = (g.C + TK - 1) / TK;

  // Whole tiles first (XCD-major over the tile order), then the pieces of
  // the split tiles, numbered piece-major so that the pieces running together
  // on one XCD sit at the same K offset of neighbouring tiles.
  int lin, t_sk = -1, piece = 0, kb = 0, ke = nk;
  if (!SK || (int)blockIdx.x < g.dp_tiles) {
    lin = xcd_major(blockIdx.x, SK ? g.dp_tiles : gridDim.x);
  } else {
    const int q = xcd_major(blockIdx.x - g.dp_tiles, gridDim.x - g.dp_tiles);
    piece = q / g.sk_tiles;
    t_sk = q - piece * g.sk_tiles;
    lin = g.dp_tiles + t_sk;
    kb = (int)(((int64_t)piece * nk) / g.sk_split);
    ke = (int)(((int64_t)(piece + 1) * nk) / g.sk_split);
  }
  gemm_piece<NN, TM, TN, WGM, WGN, TK, NS, SK>(g, smem, tid0, lin, t_sk, piece, kb, ke, nk);
}

// Several projections' GEMMs in one launch: whole 256x256 tiles, workgroups
// [off[p], off[p+1]) take projection p's tiles (XCD-major within it).  The
// host orders the projections by contraction length, longest first, so the
// long tiles start first and the short ones fill the last wave.
template <bool NN>
__global__ __launch_bounds__(512) void gemm_group_kernel(GemmGroup G) {
  using S = GemmShape<256, 256, 2, 4, 64, 2>;
  __shared__ __attribute__((aligned(1024))) char smem[S::LDS];
  int pj = 0;
  while (pj + 1 < G.n && (int)blockIdx.x >= G.off[pj + 1]) ++pj;
  const GemmArgs g = G.a[pj];  // a copy: uniform fields held in scalar registers
  const int local = (int)blockIdx.x - G.off[pj];
  const int lin = xcd_major(local, G.off[pj + 1] - G.off[pj]);
  const int nk = (g.C + 63) / 64;
  gemm_piece<NN, 256, 256, 2, 4, 64, 2, false>(g, smem, threadIdx.x, lin, -1, 0, 0, nk, nk);
}

// ---------------------------------------------------------------------------
// GEMM, 16x16x32 form of the 256 x 256 tile (NT: Q is [Nout][C]): 4 waves in a
// 2 x 2 grid, one per SIMD, each wave 128 x 128 = 8 x 8 blocks of
// v_mfma_f32_16x16x32_bf16 with its 256 fp32 accumulators.  Against the 8-wave
// 32x32x16 tile this reads a third fewer LDS bytes per MFMA (a wave's 16
// fragments feed 64 MFMAs per 32-wide step) and keeps every per-lane address
// in registers, so the main loop issues no address arithmetic: fragment reads
// are a base register plus an immediate, operand loads a base register plus a
// scalar offset.  Same LDS image (K-contiguous rows, chunk c of row r in slot
// c ^ swz(r)), direct-to-LDS loads, two-stage pipeline, low-rank prologue
// semantics and single-rounding epilogue as gemm_piece.
//
// Accumulator layout (weight fragment as the first MFMA operand): acc[i][j][v]
// is output row wm*128 + 16i + lane%16, column wn*128 + 16j + 4(lane/16) + v.
// ---------------------------------------------------------------------------
typedef short s16x4v __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));

// Four bf16 values p[e * stride], e < n_valid (1 <= n_valid), the rest zero;
// straight-line loads from clamped addresses.
__device__ __forceinline__ u32x2v ld4_sel(const uint16_t* p, int64_t stride, int n_valid) {
  uint32_t w[2] = {0u, 0u};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t x = (uint32_t)p[(int64_t)min(e, n_valid - 1) * stride];
    w[e >> 1] |= (e < n_valid ? x : 0u) << (16 * (e & 1));
  }
  return u32x2v{w[0], w[1]};
}

// DROP: the instantiation that masks the low-rank term (dX under LoRA
// dropout); the others carry no masking code.
template <bool SK, bool DROP, bool NN>
__device__ __forceinline__ void gemm_piece16(const GemmArgs& g, char* smem0, char* smem1, int tid, int lin, int t_sk,
                                             int piece,
                                             int kb, int ke, int nk) {
  constexpr int TM = 256, TN = 256, TK = 64, NW = 4, WM = 128, WN = 128, FM = 8, FN = 8;
  constexpr int ROWB = TK * 2;                   // bytes per LDS row
  constexpr int A_BYTES = TM * ROWB, STAGE = A_BYTES + TN * ROWB;
  constexpr int LOADS = TM * ROWB / 1024 / 4;    // 1 KiB direct loads per wave per operand
  static_assert(LOADS == 8 && TN == TM, "load split");
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  // The two pipeline buffers are two LDS arrays: with the buffer index a
  // constant at a use (the main loop runs K-steps in pairs), the compiler sees
  // that an LDS read and the direct loads in flight into the other buffer are
  // disjoint, and makes no read wait for those loads.
  auto buf = [&](int stage) { return stage ? smem1 : smem0; };

  int mt, nt;
  tile_coords(g, lin, mt, nt);
  const int32_t* td = g.tiles + (int64_t)mt * kTileWords;
  // uniform rows: the first loads need not wait for the tile descriptor
  const int m0 = g.uniform_rows ? mt * TM : td[0];
  const int nrows = g.uniform_rows ? min(TM, g.M - m0) : td[3];
  const int n0 = nt * TN;
  // Everything the first low-rank group needs is read here, before the first
  // direct load: past those loads a read of kernel-visible memory can no
  // longer be a scalar load, and a vector load would wait for every load
  // issued before it (vector-memory operations complete in order).
  const int ngroups = td[1], has_gather = td[2];
  const int g0_a = td[4], g0_lo = td[5], g0_hi = td[6];  // zeros when the tile has no group
  const int g0_r = g.ranks[g0_a];
  const float g0_sc = g.scales ? g.scales[g0_a] : 1.f;
  // NT: both operands are contraction-contiguous rows; the lane offsets are
  // computed for the A rows' stride and shifted by lr (ldq - ldp) elements for
  // the B rows (zero when the strides agree).
  // NN: the weight is [C][Nout] (rows of the contraction, W itself); its tile
  // of a K-step is TK rows of TN columns, and the launcher checks that the
  // whole weight's byte offsets fit in 31 bits.
  const int ld = (int)g.ldp;
  const int ldq = (int)g.ldq;
  const int64_t a_rows = min((int64_t)TM, (int64_t)g.M - m0);
  const int64_t b_cols = min((int64_t)TN, (int64_t)g.Nout - n0);
  // Descriptors over the tile's row panels (rows past the operand read zeros);
  // a K-step adds 2 k0 bytes to the scalar offset.  A panel is at most 256
  // rows of 2^20 elements, so every offset fits in 32 bits.  NN: over the
  // weight from the tile's first column (rows past the contraction read zeros).
  const i32x4 ra = make_rsrc(g.P + (int64_t)m0 * ld, (uint64_t)a_rows * ld * 2);
  const i32x4 rb = NN ? make_rsrc(g.Q + n0, ((uint64_t)g.C * ldq - n0) * 2)
                      : make_rsrc(g.Q + (int64_t)n0 * ldq, (uint64_t)b_cols * ldq * 2);

  // Operand loads: load i of a wave fills LDS rows 8q .. 8q+7 (q = 8 wave + i),
  // lane ln taking row 8q + ln/8, logical chunk (ln%8) ^ swz(row), which is
  // (ln%8) ^ (ln/8) ^ i.  The lane parts of the offsets stay in registers; the
  // row block and the K-step go in the scalar offset.
  const int lr = lane >> 3;
  int voff[LOADS];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) voff[i] = ((((lane & 7) ^ lr ^ i) << 4)) + lr * ld * 2;
  // NN weight loads: load i fills tile rows 2q, 2q+1 (q = 8 wave + i, 512
  // bytes each), lane ln taking row 2q + ln/32, slot ln%32, which holds the
  // row's 16-byte chunk (ln%32) ^ nn_swz(row); nn_swz(row) depends on i%2 only.
  const int dq_lane = lr * (ldq - ld) * 2;  // NT: B row offset minus A row offset
  int voffb[2];
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    const int n_in = 2 * par + (lane >> 5);
    voffb[par] = ((lane >> 5) * ldq + 8 * ((lane & 31) ^ nn_swz(n_in))) * 2;
  }
  auto load_b = [&](int kt, char* sa, int i) {
    const int q = wave * LOADS + i;
    if constexpr (NN)
      llvm_amdgcn_raw_buffer_load_lds(rb, (lds_u32*)(sa + A_BYTES + q * 1024), 16, voffb[i & 1],
                                      __builtin_amdgcn_readfirstlane((kt * TK + 2 * q) * ldq * 2), 0, 0);
    else
      llvm_amdgcn_raw_buffer_load_lds(rb, (lds_u32*)(sa + A_BYTES + q * 1024), 16, voff[i] + dq_lane,
                                      __builtin_amdgcn_readfirstlane(q * 16 * ldq + kt * TK * 2), 0, 0);
  };
  // whole K-step kt into `stage` (k0 + TK <= C)
  auto issue_whole = [&](int kt, int stage) {
    const int kbytes = kt * TK * 2;
    char* sa = buf(stage);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int q = wave * LOADS + i;
      llvm_amdgcn_raw_buffer_load_lds(ra, (lds_u32*)(sa + q * 1024), 16, voff[i],
                                      __builtin_amdgcn_readfirstlane(q * 16 * ld + kbytes), 0, 0);
    }
#pragma unroll
    for (int i = 0; i < LOADS; ++i) load_b(kt, sa, i);
  };
  // any K-step: chunks past the contraction read nothing (zeros)
  auto issue = [&](int kt, int stage) {
    const int k0 = kt * TK;
    if (k0 + TK <= g.C) {
      issue_whole(kt, stage);
      return;
    }
    char* sa = buf(stage);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int q = wave * LOADS + i;
      const int row = 8 * q + lr;
      const int c = (lane & 7) ^ swz<TK>(row);
      const bool in_c = k0 + 8 * c < g.C;
      const int vo = in_c ? (row * ld + k0 + 8 * c) * 2 : (int)0x7FFFFFF0;
      llvm_amdgcn_raw_buffer_load_lds(ra, (lds_u32*)(sa + q * 1024), 16, vo, 0, 0, 0);
      if constexpr (NN) {
        load_b(kt, sa, i);  // rows past the contraction lie past the descriptor
      } else {
        const int vb = in_c ? (row * ldq + k0 + 8 * c) * 2 : (int)0x7FFFFFF0;
        llvm_amdgcn_raw_buffer_load_lds(rb, (lds_u32*)(sa + A_BYTES + q * 1024), 16, vb, 0, 0, 0);
      }
    }
  };

  issue(kb, 0);

  // The first group's first 16 ranks are loaded between the first two
  // K-steps, so the wait for them is the wait for the first K-step alone
  // (vector-memory operations complete in order) rather than for both.  This
  // covers the forward form (h and B rows with contiguous ranks, r a multiple
  // of 16) for a wave that has rows in the group; anything else loads below.
  const bool pre = !DROP && kb == 0 && ngroups > 0 && g.lq_j == 1 && (g.lq_col & 3) == 0 && (g0_r & 15) == 0 &&
                   g0_hi > wm * WM && g0_lo < wm * WM + WM;
  u32x2v pre_h[FM], pre_b[FN];
  if (pre) {
    const int a = g0_a, lo = g0_lo, hi = g0_hi;
    const uint16_t* lq = g.Lq + (int64_t)a * g.lq_ad;
    const int jb = 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WM + 16 * i + (lane & 15);
      const int rr = (row >= lo && row < hi) ? row : lo;
      pre_h[i] = *reinterpret_cast<const u32x2v*>(g.Lp + (int64_t)(m0 + rr) * g.ldl + jb);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = n0 + wn * WN + 16 * j + (lane & 15);
      pre_b[j] = *reinterpret_cast<const u32x2v*>(lq + jb + (int64_t)min(col, g.Nout - 1) * g.lq_col);
    }
  }
  if (kb + 1 < ke) issue(kb + 1, 1);

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // ---- low-rank prologue (the piece that starts the tile's K range) -----
  // acc += (s_a h) B_a for the rows of each group, with 16x16x16 MFMAs over
  // steps of 16 ranks (a lane holds 4 ranks of one row / column); s_a h is
  // split into bf16 hi + lo as in gemm_piece.
  auto lr_mfma = [&](const u32x2v (&hv)[FM], const u32x2v (&bv)[FN], int lo, int hi, int nv, float sc) {
    s16x4v af_hi[FM], af_lo[FM], bq[FN];
    bool any_lo = false;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WM + 16 * i + (lane & 15);
      const bool rin = row >= lo && row < hi && nv > 0;
      const u32x2v v = rin ? hv[i] : u32x2v{0u, 0u};
      uint32_t wh[2], wl[2];
#pragma unroll
      for (int d = 0; d < 2; ++d) {
        const float x0 = sc * __uint_as_float(v[d] << 16);
        const float x1 = sc * __uint_as_float(v[d] & 0xffff0000u);
        const uint16_t h0 = f2bf(x0), h1 = f2bf(x1);
        const uint16_t l0 = f2bf(x0 - bf2f(h0)), l1 = f2bf(x1 - bf2f(h1));
        wh[d] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        wl[d] = (uint32_t)l0 | ((uint32_t)l1 << 16);
        any_lo |= (wl[d] & 0x7fff7fffu) != 0u;
      }
      af_hi[i] = __builtin_bit_cast(s16x4v, u32x2v{wh[0], wh[1]});
      af_lo[i] = __builtin_bit_cast(s16x4v, u32x2v{wl[0], wl[1]});
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = n0 + wn * WN + 16 * j + (lane & 15);
      bq[j] = __builtin_bit_cast(s16x4v, (col < g.Nout && nv > 0) ? bv[j] : u32x2v{0u, 0u});
    }
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(bq[j], af_hi[i], acc[i][j], 0, 0, 0);
    if (__builtin_amdgcn_ballot_w64(any_lo) != 0) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(bq[j], af_lo[i], acc[i][j], 0, 0, 0);
    }
  };
  // Under dropout (the DROP instantiation, launched only with a mask) the
  // low-rank term is masked per element: it is built one 16-row block at a
  // time in ordinary registers (below), masked there and added to the block's
  // accumulators, which are still zero.
  // the prefetched step: its data arrive with the first K-step
  if (pre) lr_mfma(pre_h, pre_b, g0_lo, g0_hi, 4, g0_sc);
  // every other (group, 16-rank step) of the tile
  for (int gi = 0; !DROP && kb == 0 && gi < ngroups; ++gi) {
    const int a = gi == 0 ? g0_a : td[4 + 3 * gi], lo = gi == 0 ? g0_lo : td[5 + 3 * gi];
    const int hi = gi == 0 ? g0_hi : td[6 + 3 * gi];
    if (hi <= wm * WM || lo >= wm * WM + WM) continue;  // no row of this wave
    const int r = gi == 0 ? g0_r : g.ranks[a];
    const float sc = gi == 0 ? g0_sc : (g.scales ? g.scales[a] : 1.f);
    const uint16_t* lq = g.Lq + (int64_t)a * g.lq_ad;
    const bool full16 = (r & 15) == 0;
    const bool lq_vec = full16 && g.lq_j == 1 && (g.lq_col & 3) == 0;
    for (int j0 = (gi == 0 && pre) ? 16 : 0; j0 < r; j0 += 16) {
      const int jb = j0 + 4 * (lane >> 4);
      const int nv = min(4, r - jb);
      const int jbc = nv > 0 ? jb : 0, nvc = max(nv, 1);
      u32x2v hv[FM], bv[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = wm * WM + 16 * i + (lane & 15);
        const uint16_t* p = g.Lp + (int64_t)(m0 + ((row >= lo && row < hi) ? row : lo)) * g.ldl + jbc;
        hv[i] = full16 ? *reinterpret_cast<const u32x2v*>(p) : ld4_sel(p, 1, nvc);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = n0 + wn * WN + 16 * j + (lane & 15);
        const uint16_t* p = lq + (int64_t)jbc * g.lq_j + (int64_t)min(col, g.Nout - 1) * g.lq_col;
        bv[j] = lq_vec ? *reinterpret_cast<const u32x2v*>(p) : ld4_sel(p, g.lq_j, nvc);
      }
      lr_mfma(hv, bv, lo, hi, nv, sc);
    }
  }

  // ---- dropout of the low-rank term (dX under LoRA dropout) --------------
  // Row block i (rows wm*WM + 16i ..): t[j] = the unmasked term of its 8
  // column blocks, the same MFMA sequence per element as the plain prologue
  // (groups in order, 16-rank steps, bf16 hi then lo parts of s_a h); then
  // element (row, col) keeps t * keep_scale where its mask bit is set, else 0.
  // Column blocks 2h and 2h+1 of a wave share mask word (n0 + wn*WN)/32 + h
  // (n0 and wn*WN are multiples of 32).  The next row block's h and mask
  // words load while the current one is computed; a tile whose rows form one
  // group of rank <= 16 loads its adapter's B fragments once.  The barrier per
  // row block keeps the compiler from interleaving row blocks (and their
  // registers).
  if (DROP && kb == 0) {
    const int bit0 = 4 * (lane >> 4);
    const int wd0 = (n0 + wn * WN) >> 5;
    const int jb0 = 4 * (lane >> 4);
    const bool one = ngroups == 1 && g0_r <= 16;  // one group, one 16-rank step
    auto load_b = [&](const uint16_t* lq, int jbc, int nvc, bool lq_vec, u32x2v (&bv)[FN]) {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = n0 + wn * WN + 16 * j + (lane & 15);
        const uint16_t* p = lq + (int64_t)jbc * g.lq_j + (int64_t)min(col, g.Nout - 1) * g.lq_col;
        bv[j] = lq_vec ? *reinterpret_cast<const u32x2v*>(p) : ld4_sel(p, g.lq_j, nvc);
      }
    };
    u32x2v b1[FN];  // the single group's B fragments (one)
    if (one) {
      const int nv = min(4, g0_r - jb0);
      load_b(g.Lq + (int64_t)g0_a * g.lq_ad, nv > 0 ? jb0 : 0, max(nv, 1),
             (g0_r & 15) == 0 && g.lq_j == 1 && (g.lq_col & 3) == 0, b1);
    }
    // h of the single group's row and the mask words of row block i
    auto load_row = [&](int i, u32x2v& hv, uint32_t (&mw)[FN / 2]) {
      const int row = wm * WM + 16 * i + (lane & 15);
      const int nv = min(4, g0_r - jb0);
      const bool rin = row >= g0_lo && row < g0_hi;
      const uint16_t* hp = g.Lp + (int64_t)(m0 + (rin ? row : g0_lo)) * g.ldl + (nv > 0 ? jb0 : 0);
      hv = ((g0_r & 15) == 0) ? *reinterpret_cast<const u32x2v*>(hp) : ld4_sel(hp, 1, max(nv, 1));
      const uint32_t* kr = g.keep + (int64_t)(m0 + min(row, nrows - 1)) * g.keep_words;
#pragma unroll
      for (int h = 0; h < FN / 2; ++h) mw[h] = kr[min(wd0 + h, g.keep_words - 1)];
    };
    u32x2v hv_n = u32x2v{0u, 0u};
    uint32_t mw_n[FN / 2] = {0u, 0u, 0u, 0u};
    load_row(0, hv_n, mw_n);
    // t[j] += (s h) B for one (group, 16-rank step); rows outside [lo, hi) add zeros
    auto lr_row = [&](f32x4 (&t)[FN], u32x2v hv, const u32x2v (&bv)[FN], int row, int lo, int hi, int nv,
                      float sc) {
      const u32x2v v = (row >= lo && row < hi && nv > 0) ? hv : u32x2v{0u, 0u};
      uint32_t wh[2], wl[2];
      bool any_lo = false;
#pragma unroll
      for (int d = 0; d < 2; ++d) {
        const float x0 = sc * __uint_as_float(v[d] << 16);
        const float x1 = sc * __uint_as_float(v[d] & 0xffff0000u);
        const uint16_t h0 = f2bf(x0), h1 = f2bf(x1);
        const uint16_t l0 = f2bf(x0 - bf2f(h0)), l1 = f2bf(x1 - bf2f(h1));
        wh[d] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        wl[d] = (uint32_t)l0 | ((uint32_t)l1 << 16);
        any_lo |= (wl[d] & 0x7fff7fffu) != 0u;
      }
      const s16x4v af_hi = __builtin_bit_cast(s16x4v, u32x2v{wh[0], wh[1]});
      const s16x4v af_lo = __builtin_bit_cast(s16x4v, u32x2v{wl[0], wl[1]});
      const bool lo_pass = __builtin_amdgcn_ballot_w64(any_lo) != 0;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = n0 + wn * WN + 16 * j + (lane & 15);
        const s16x4v bq = __builtin_bit_cast(s16x4v, (col < g.Nout && nv > 0) ? bv[j] : u32x2v{0u, 0u});
        t[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(bq, af_hi, t[j], 0, 0, 0);
        if (lo_pass) t[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(bq, af_lo, t[j], 0, 0, 0);
      }
    };
    float sel[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) sel[v] = (lane & 15) == 4 * (lane >> 4) + v ? 1.f : 0.f;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int rb0 = wm * WM + 16 * i;
      const int row = rb0 + (lane & 15);
      const u32x2v hv1 = hv_n;
      uint32_t mw[FN / 2];
#pragma unroll
      for (int h = 0; h < FN / 2; ++h) mw[h] = (row < nrows && wd0 + h < g.keep_words) ? mw_n[h] : 0u;
      if (i + 1 < FM) load_row(i + 1, hv_n, mw_n);
      f32x4 t[FN];
#pragma unroll
      for (int j = 0; j < FN; ++j) t[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (one) {
        if (g0_hi > rb0 && g0_lo < rb0 + 16) lr_row(t, hv1, b1, row, g0_lo, g0_hi, min(4, g0_r - jb0), g0_sc);
      } else {
        for (int gi = 0; gi < ngroups; ++gi) {
          const int a = td[4 + 3 * gi], lo = td[5 + 3 * gi], hi = td[6 + 3 * gi];
          if (hi <= rb0 || lo >= rb0 + 16) continue;  // no row of this block
          const int r = g.ranks[a];
          const float sc = g.scales ? g.scales[a] : 1.f;
          const uint16_t* lq = g.Lq + (int64_t)a * g.lq_ad;
          const bool full16 = (r & 15) == 0;
          const bool lq_vec = full16 && g.lq_j == 1 && (g.lq_col & 3) == 0;
          const bool rin = row >= lo && row < hi;
          for (int j0 = 0; j0 < r; j0 += 16) {
            const int jb = j0 + jb0;
            const int nv = min(4, r - jb);
            const int jbc = nv > 0 ? jb : 0, nvc = max(nv, 1);
            const uint16_t* hp = g.Lp + (int64_t)(m0 + (rin ? row : lo)) * g.ldl + jbc;
            const u32x2v hv = full16 ? *reinterpret_cast<const u32x2v*>(hp) : ld4_sel(hp, 1, nvc);
            u32x2v bv[FN];
            load_b(lq, jbc, nvc, lq_vec, bv);
            lr_row(t, hv, bv, row, lo, hi, nv, sc);
          }
        }
      }
      // The masked term enters the (zero) accumulators as matrix-core
      // products, so they stay where the main loop keeps them: fp32 MFMA step
      // s (16x16x4) multiplies a 0/1 selector (lane holds A[lane%16][lane/16] =
      // [lane%16 == 4(lane/16) + s]) by the lane's own value v = s, which lands
      // each value, exactly, in its own accumulator entry.
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float m = ((mw[j >> 1] >> (16 * (j & 1) + bit0 + v)) & 1u) ? t[j][v] * g.keep_scale : 0.f;
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(sel[v], m, acc[i][j], 0, 0, 0);
        }
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // ---- main loop ----------------------------------------------------------
  // Fragment (i, 32-wide step s) of the A tile: row R + lane%16 with R =
  // wm*128 + 16i, logical chunk 4s + lane/16.  With row%8 = lane%8 and
  // (row/8)%8 = (2i + lane/8%2)%8 the slot is lanepart ^ (4s ^ 2i%8), so a
  // fragment is at one of four lane offsets, picked by the constant
  // 4s ^ 2i%8, plus the immediate R*128.  The B tile is the same with wn, j.
  const int l15 = lane & 15;
  const int lanepart = (lane >> 4) ^ (l15 & 7) ^ (l15 >> 3);
  int off_a[4], off_b[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    off_a[c] = (wm * WM + l15) * ROWB + 16 * (lanepart ^ (2 * c));
    off_b[c] = A_BYTES + (wn * WN + l15) * ROWB + 16 * (lanepart ^ (2 * c));
  }
  auto rd_a = [&](const char* st, int s, int i) {
    return as_bf(*reinterpret_cast<const u32x4*>(st + off_a[((2 * s) ^ i) & 3] + 16 * i * ROWB));
  };
  // NN: weight fragment j of step s = output column wn*128 + 16j + lane%16 and
  // contraction rows 32s + 8(lane/16) .. +7, as two transposing reads of four
  // rows each: read hh of lane (g4 = lane/16, l = lane%16) addresses row
  // 32s + 8 g4 + 4 hh + l/4, column wn*128 + 16j + 4(l%4), whose chunk
  // (c/8) ^ nn_swz(row) is wn*16 + 2((j%4) ^ (l/4)) + 8(j/4) + (l%4)/2.
  int off_bn[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
    off_bn[c] = A_BYTES + (8 * (lane >> 4) + (l15 >> 2)) * (TN * 2) + 256 * wn + 32 * (c ^ (l15 >> 2)) +
                16 * ((l15 & 3) >> 1) + 8 * (l15 & 1);
  auto rd_b = [&](const char* st, int s, int j) {
    if constexpr (NN) {
      const char* p = st + off_bn[j & 3] + 128 * (j >> 2) + s * 32 * (TN * 2);
      const s16x4 h0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
      const s16x4 h1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 4 * (TN * 2)));
      const u32x2v a0 = __builtin_bit_cast(u32x2v, h0), a1 = __builtin_bit_cast(u32x2v, h1);
      return as_bf(u32x4{a0[0], a0[1], a1[0], a1[1]});
    } else {
      return as_bf(*reinterpret_cast<const u32x4*>(st + off_b[((2 * s) ^ j) & 3] + 16 * j * ROWB));
    }
  };

  // Fragments: two A sets (the current step's and the next one's) and one B
  // set whose fragment j is replaced by the next step's once the 8 MFMAs of
  // column block j have been issued.
  bf16x8 fa0[FM], fa1[FM], fb[FN];
  if (ke - kb >= 2) __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * LOADS));  // first K-step landed
  else vmem_wait_all();
  __syncthreads();
#pragma unroll
  for (int j = 0; j < FN; ++j) fb[j] = rd_b(smem0, 0, j);
#pragma unroll
  for (int i = 0; i < FM; ++i) fa0[i] = rd_a(smem0, 0, i);

  // Direct loads of whole K-step kl into buffer ls: load n of the wave's 16
  // (A for n < 8, B after).  A texture unit takes a 1 KiB load in about 16
  // cycles, so the 64 loads a K-step needs per CU are spread evenly, two per
  // wave per column block (a block's 8 MFMAs take 128 cycles), over the
  // second step, after the barrier that frees their buffer.
  auto load_n = [&](int kl, int ls, int n) {
    const int i = n & 7;
    const int q = wave * LOADS + i;
    if (n >= 8)
      load_b(kl, buf(ls), i);
    else
      llvm_amdgcn_raw_buffer_load_lds(ra, (lds_u32*)(buf(ls) + q * 1024), 16, voff[i],
                                      __builtin_amdgcn_readfirstlane(q * 16 * ld + kl * TK * 2), 0, 0);
  };
  // One 32-wide step with fragments (cur, fb); reads the next step's
  // fragments (nxt, fb) from buffer `st_next` step s_next, in the order fixed
  // by scheduling fences, per column block j: its 8 MFMAs, then (when `load`)
  // loads 2j, 2j+1 of whole K-step kl into buffer ls, then the next B
  // fragment j (replacing fb[j] once block j's MFMAs are issued) and A
  // fragments 2j, 2j+1 (blocks 0-3).
  auto step = [&](bf16x8 (&cur)[FM], bf16x8 (&nxt)[FM], const char* st_next, int s_next, bool load, int kl,
                  int ls) {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[j], cur[i], acc[i][j], 0, 0, 0);
      if (load) {
        load_n(kl, ls, 2 * j);
        load_n(kl, ls, 2 * j + 1);
      }
      if (j < 4) {
        nxt[2 * j] = rd_a(st_next, s_next, 2 * j);
        nxt[2 * j + 1] = rd_a(st_next, s_next, 2 * j + 1);
      }
      fb[j] = rd_b(st_next, s_next, j);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // K-step kt in buffer `stage` with K-step kt+1 to follow: first step, then
  // the barrier that publishes kt+1 (every wave's loads of it were issued
  // during the previous K-step's second step) and frees buffer `stage`, then
  // the second step, which reads kt+1's first fragments and loads whole
  // K-step kt+2 into buffer `stage` (when `load`).
  auto kstep = [&](int kt, int stage, bool load) {
    step(fa0, fa1, buf(stage), 1, false, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    vmem_wait_all();  // kt+1 landed (its loads are the only ones in flight)
    __syncthreads();  // everyone's part of kt+1 is in; buffer `stage` is free
    __builtin_amdgcn_sched_barrier(0);
    if (!load && kt + 2 < ke) issue(kt + 2, stage);  // a partial last K-step
    step(fa1, fa0, buf(stage ^ 1), 0, load, kt + 2, stage);
  };
  int kt = kb, stage = 0;
  const int main_end = min(ke, g.C / TK) - 2;  // kt < main_end: kt+2 is whole and below ke
  if constexpr (NN) {
    for (; kt + 1 < main_end; kt += 2) {  // pairs: buffers 0 then 1, constant at every use
      kstep(kt, 0, true);
      kstep(kt + 1, 1, true);
    }
    if (kt < main_end) {
      kstep(kt, 0, true);
      ++kt;
      stage = 1;
    }
  } else {
    for (; kt < main_end; ++kt, stage ^= 1) kstep(kt, stage, true);
  }
  for (; kt + 1 < ke; ++kt, stage ^= 1) kstep(kt, stage, false);
  // the last K-step: no successor to read
  step(fa0, fa1, buf(stage), 1, false, 0, 0);
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int i = 0; i < FM; ++i)
      acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[j], fa1[i], acc[i][j], 0, 0, 0);
  const int last_stage = stage;

  // ---- a piece of a split tile: its fp32 partial goes to its slot --------
  if (SK && !(kb == 0 && ke == nk)) {
    float* part = g.sk_part + (int64_t)(t_sk * g.sk_split + piece) * (TM * TN);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WM + 16 * i + l15;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = wn * WN + 16 * j + 4 * (lane >> 4);
        *reinterpret_cast<f32x4*>(part + row * TN + col) = acc[i][j];
      }
    }
    return;
  }

  // ---- epilogue: one rounding, staged through LDS for 16-byte stores ----
  // Each wave stages its rows 32 at a time (fragment rows i = 2t, 2t+1) in its
  // own slice of the buffer the last K-step did not use; a lane writes 4
  // columns (8 bytes) of a row, then the wave reads the slice back as
  // 16-byte row chunks and stores 256-byte row segments.  Slice row stride
  // 272 bytes (68 dwords): the 8-byte writes of 16 rows x 2 column groups of
  // one half-wave fall on distinct banks.
  constexpr int SRS = WN * 2 + 16;
  static_assert(NW * 32 * SRS <= STAGE, "epilogue slices fit the idle pipeline buffer");
  constexpr int CPR = WN / 8;  // 16-byte chunks per slice row
  static_assert(CPR == 16, "a slice read step covers 4 rows of 16 chunks");
  char* slice = buf(last_stage ^ 1) + wave * 32 * SRS;
  // Read-back step q of slice t: lane ln takes chunk ln % 16 of slice row
  // 4q + ln / 16.  Its output address is a wave-uniform part (row
  // m0 + wm WM + 32t + 4q, column n0 + wn WN) plus a per-lane offset.
  const int64_t ldo2 = g.ldo * 2;
  const uint32_t lane_off = (uint32_t)((lane >> 4) * ldo2 + 16 * (lane & 15));
  char* const out_w = reinterpret_cast<char*>(g.out) + ((int64_t)(m0 + wm * WM) * g.ldo + n0 + wn * WN) * 2;
  // The plain form (a whole tile without gathered rows) is compiled apart
  // from the general one: its stores need no bounds checks and its values no
  // gathered terms, which would otherwise be selected and added everywhere.
  const bool gathered = has_gather && g.delta != nullptr;
  auto epilogue = [&](auto plain_c) {
    constexpr bool PLAIN = decltype(plain_c)::value;
    // Gathered rows add their fp32 term: the wave's row slots are read once
    // and each slice's terms are loaded while the slice before it is processed.
    int gsv[FM];
    f32x4 dn[2][FN];
    auto load_terms = [&](int t) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = wn * WN + 16 * j + 4 * (lane >> 4);
          const int gs = gsv[2 * t + h];
          const f32x4 d = *reinterpret_cast<const f32x4*>(g.delta + (int64_t)max(gs, 0) * g.Nout +
                                                          min(n0 + col, g.Nout - 4));
          dn[h][j] = (gs >= 0 && n0 + col < g.Nout) ? d : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    };
    if (!PLAIN && gathered) {
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = wm * WM + 16 * i + l15;
        gsv[i] = row < nrows ? g.gslot[m0 + row] : -1;
      }
      load_terms(0);
    }
#pragma unroll
    for (int t = 0; t < FM / 2; ++t) {
      f32x4 dc[2][FN];
      if (!PLAIN && gathered) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int j = 0; j < FN; ++j) dc[h][j] = dn[h][j];
        if (t + 1 < FM / 2) load_terms(t + 1);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int i = 2 * t + h;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = wn * WN + 16 * j + 4 * (lane >> 4);
          f32x4 x = acc[i][j];
          if (!PLAIN && gathered) x += dc[h][j];
          const uint32_t w0 = f2bf2(x[0], x[1]), w1 = f2bf2(x[2], x[3]);
          *reinterpret_cast<uint2*>(slice + (16 * h + l15) * SRS + 2 * (col - wn * WN)) = make_uint2(w0, w1);
        }
      }
      asm volatile("" ::: "memory");  // a wave's LDS accesses run in order: the slice is complete
#pragma unroll
      for (int q = 0; q < 32 * CPR / 64; ++q) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(slice + (4 * q + (lane >> 4)) * SRS + 16 * (lane & 15));
        char* const dst = out_w + (int64_t)(32 * t + 4 * q) * ldo2 + lane_off;
        if constexpr (PLAIN) {
          __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(dst));
        } else {
          const int orow = wm * WM + 32 * t + 4 * q + (lane >> 4), ocol = n0 + wn * WN + 8 * (lane & 15);
          if (orow < nrows && ocol < g.Nout) __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(dst));
        }
      }
      asm volatile("" ::: "memory");  // the slice is read before the next rows overwrite it
    }
  };
  if (!gathered && nrows >= TM && n0 + TN <= g.Nout)
    epilogue(bool_c<true>{});
  else
    epilogue(bool_c<false>{});
}

template <bool SK, bool DROP, bool NN>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm16_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(1024))) char smem0[2 * 256 * 64 * 2];
  __shared__ __attribute__((aligned(1024))) char smem1[2 * 256 * 64 * 2];
  const int nk = (g.C + 63) / 64;
  int lin, t_sk = -1, piece = 0, kb = 0, ke = nk;
  if (!SK || (int)blockIdx.x < g.dp_tiles) {
    lin = xcd_major(blockIdx.x, SK ? g.dp_tiles : gridDim.x);
  } else {
    const int q = xcd_major(blockIdx.x - g.dp_tiles, gridDim.x - g.dp_tiles);
    piece = q / g.sk_tiles;
    t_sk = q - piece * g.sk_tiles;
    lin = g.dp_tiles + t_sk;
    kb = (int)(((int64_t)piece * nk) / g.sk_split);
    ke = (int)(((int64_t)(piece + 1) * nk) / g.sk_split);
  }
  gemm_piece16<SK, DROP, NN>(g, smem0, smem1, threadIdx.x, lin, t_sk, piece, kb, ke, nk);
}

template <bool DROP, bool NN>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm16_group_kernel(GemmGroup G) {
  __shared__ __attribute__((aligned(1024))) char smem0[2 * 256 * 64 * 2];
  __shared__ __attribute__((aligned(1024))) char smem1[2 * 256 * 64 * 2];
  // the workgroup's projection: every boundary compared at once (one batch
  // of argument loads instead of one dependent load per projection)
  int pj = 0;
#pragma unroll
  for (int p = 1; p < kMaxGroup; ++p) pj += (p < G.n && (int)blockIdx.x >= G.off[p]) ? 1 : 0;
  const GemmArgs g = G.a[pj];
  const int local = (int)blockIdx.x - G.off[pj];
  const int lin = xcd_major(local, G.off[pj + 1] - G.off[pj]);
  const int nk = (g.C + 63) / 64;
  gemm_piece16<false, DROP, NN>(g, smem0, smem1, threadIdx.x, lin, -1, 0, 0, nk, nk);
}

// ---------------------------------------------------------------------------
// Split tiles: sum the fp32 partials of a tile's pieces in K order, add the
// gathered rows' term, round once to bf16 and store -- the GEMM epilogue for
// the tiles the GEMM left in pieces.  Elementwise: one thread per 4 columns
// of a row, (TM * TN / 4) / 256 workgroups per split tile.
// ---------------------------------------------------------------------------
template <bool NN, int TM, int TN>  // NN: the dX GEMM's tiles (the layout is the same)
__global__ __launch_bounds__(256) void split_fixup_kernel(GemmArgs g) {
  constexpr int PER_TILE = TM * TN / 4 / 256;
  const int t_sk = blockIdx.x / PER_TILE;
  const int idx = (blockIdx.x % PER_TILE) * 256 + threadIdx.x;
  const int row = idx / (TN / 4), c4 = idx % (TN / 4);
  int mt, nt;
  tile_coords(g, g.dp_tiles + t_sk, mt, nt);
  const int32_t* td = g.tiles + (int64_t)mt * kTileWords;
  const int m0 = td[0], has_gather = td[2], nrows = td[3];
  const int col = nt * TN + 4 * c4;
  if (row >= nrows || col >= g.Nout) return;  // Nout % 8 == 0: all 4 columns or none
  const f32x4* src = reinterpret_cast<const f32x4*>(g.sk_part + (int64_t)t_sk * g.sk_split * (TM * TN)) + idx;
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int p = 0; p < g.sk_split; ++p) acc += src[(int64_t)p * (TM * TN / 4)];
  if (has_gather && g.delta != nullptr) {
    // rows of the gathered path add their fp32 low-rank term before the rounding
    const int gs = g.gslot[m0 + row];
    if (gs >= 0) acc += *reinterpret_cast<const f32x4*>(g.delta + (int64_t)gs * g.Nout + col);
  }
  const uint32_t lo = (uint32_t)f2bf(acc[0]) | ((uint32_t)f2bf(acc[1]) << 16);
  const uint32_t hi = (uint32_t)f2bf(acc[2]) | ((uint32_t)f2bf(acc[3]) << 16);
  *reinterpret_cast<uint2*>(g.out + (int64_t)(m0 + row) * g.ldo + col) = make_uint2(lo, hi);
}

}  // namespace

namespace {
// Benchmark timing of the next GEMM launch (set_launch_events): the start
// event rides the launch's first kernel and the stop event its last one, as
// part of their dispatches (hipExtLaunchKernelGGL), so the timing adds no
// packets between kernels.
hipEvent_t g_ev_start = nullptr, g_ev_stop = nullptr;

template <typename F, typename... Args>
void launch_timed(F kernel, dim3 grid, dim3 block, hipStream_t s, bool first, bool last, Args... args) {
  hipEvent_t e0 = first ? g_ev_start : nullptr, e1 = last ? g_ev_stop : nullptr;
  if (e0 || e1)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, e0, e1, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
  if (first) g_ev_start = nullptr;
  if (last) g_ev_stop = nullptr;
}

// Tile configurations: (TM, TN, wave grid, K-step, pipeline stages); two
// waves per SIMD in each (8 waves per 256-row workgroup, or two 4-wave
// 128 x 128 workgroups per CU).
// The 16x16x32 NN form addresses the weight with 32-bit byte offsets from the
// tile's first column, one K-step past the contraction at most.
bool nn16_fits(const GemmArgs& a) { return ((int64_t)a.C + 64) * a.ldq * 2 < ((int64_t)1 << 31); }

template <bool NN>
hipError_t launch_gemm_tiled(const GemmArgs& a, int tm, int tn, hipStream_t s) {
  if (a.n_mtiles <= 0 || a.n_ntiles <= 0) return hipSuccess;
  const int64_t tiles = (int64_t)a.n_mtiles * a.n_ntiles;
  if (a.dp_tiles < 0 || a.sk_tiles < 0 || a.dp_tiles + (int64_t)a.sk_tiles != tiles) return hipErrorInvalidValue;
  if (a.sk_tiles > 0) {
    // split tiles: 256x256 only, whole tiles a multiple of 8 (the pieces keep
    // the hardware's XCD round robin), and at least one K-step per piece
    const int64_t nk = (a.C + 63) / 64;
    if (tm != 256 || tn != 256 || (a.dp_tiles & 7) || a.sk_split < 2 || a.sk_split > nk || !a.sk_part)
      return hipErrorInvalidValue;
  }
  const dim3 grid((unsigned)(a.dp_tiles + (int64_t)a.sk_tiles * (a.sk_tiles > 0 ? a.sk_split : 0)));
  if constexpr (!NN) {
    // 256 x 256 NT tiles: the 16x16x32 form (both operands rows of the
    // contraction, each with its own row stride)
    if (tm == 256 && tn == 256) {
      const bool drop = a.keep != nullptr;
      if (a.sk_tiles > 0) {
        if (drop) launch_timed(gemm16_kernel<true, true, false>, grid, dim3(256), s, true, false, a);
        else launch_timed(gemm16_kernel<true, false, false>, grid, dim3(256), s, true, false, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        launch_timed(split_fixup_kernel<NN, 256, 256>, dim3((unsigned)a.sk_tiles * (256 * 256 / 4 / 256)), dim3(256),
                     s, false, true, a);
      } else if (drop) {
        launch_timed(gemm16_kernel<false, true, false>, grid, dim3(256), s, true, true, a);
      } else {
        launch_timed(gemm16_kernel<false, false, false>, grid, dim3(256), s, true, true, a);
      }
      return hipGetLastError();
    }
  }
  if constexpr (NN) {  // 256 x 256 NN tiles (dX reading W through transposing LDS reads)
    if (tm == 256 && tn == 256 && nn16_fits(a)) {
      const bool drop = a.keep != nullptr;
      if (a.sk_tiles > 0) {
        if (drop) launch_timed(gemm16_kernel<true, true, true>, grid, dim3(256), s, true, false, a);
        else launch_timed(gemm16_kernel<true, false, true>, grid, dim3(256), s, true, false, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        launch_timed(split_fixup_kernel<NN, 256, 256>, dim3((unsigned)a.sk_tiles * (256 * 256 / 4 / 256)), dim3(256),
                     s, false, true, a);
      } else if (drop) {
        launch_timed(gemm16_kernel<false, true, true>, grid, dim3(256), s, true, true, a);
      } else {
        launch_timed(gemm16_kernel<false, false, true>, grid, dim3(256), s, true, true, a);
      }
      return hipGetLastError();
    }
    if (tm == 256 && tn == 256) {  // the 8-wave form, for weights past 2^31 bytes
      if (a.sk_tiles > 0) {
        launch_timed(gemm_lora_kernel<NN, 256, 256, 2, 4, 64, 2, true>, grid, dim3(512), s, true, false, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        launch_timed(split_fixup_kernel<NN, 256, 256>, dim3((unsigned)a.sk_tiles * (256 * 256 / 4 / 256)),
                     dim3(256), s, false, true, a);
      } else {
        launch_timed(gemm_lora_kernel<NN, 256, 256, 2, 4, 64, 2, false>, grid, dim3(512), s, true, true, a);
      }
      return hipGetLastError();
    }
  }
  if (tm == 128 && tn == 128)
    launch_timed(gemm_lora_kernel<NN, 128, 128, 2, 2, 64, 2, false>, grid, dim3(256), s, true, true, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}
}  // namespace

hipError_t launch_gemm_nt(const GemmArgs& a, int tm, int tn, hipStream_t s) {
  return launch_gemm_tiled<false>(a, tm, tn, s);
}

void set_launch_events(hipEvent_t start, hipEvent_t stop) {
  g_ev_start = start;
  g_ev_stop = stop;
}

bool launch_events_pending() { return g_ev_start != nullptr || g_ev_stop != nullptr; }

hipError_t launch_gemm_nn(const GemmArgs& a, int tm, int tn, hipStream_t s) {
  return launch_gemm_tiled<true>(a, tm, tn, s);
}

namespace {
template <bool NN>
hipError_t launch_gemm_group(const GemmGroup& g, hipStream_t s) {
  if (g.n <= 0 || g.n > kMaxGroup || g.off[0] != 0) return hipErrorInvalidValue;
  for (int p = 0; p < g.n; ++p) {
    const GemmArgs& a = g.a[p];
    if (g.off[p + 1] - g.off[p] != a.n_mtiles * a.n_ntiles || a.sk_tiles != 0) return hipErrorInvalidValue;
  }
  if (g.off[g.n] <= 0) return hipSuccess;
  if constexpr (!NN) {
    // the masked instantiation serves launches whose projections all carry a mask
    int n_keep = 0;
    for (int p = 0; p < g.n; ++p) n_keep += g.a[p].keep != nullptr;
    if (n_keep != 0 && n_keep != g.n) return hipErrorInvalidValue;
    const bool drop = n_keep > 0;
    if (drop) launch_timed(gemm16_group_kernel<true, false>, dim3((unsigned)g.off[g.n]), dim3(256), s, true, true, g);
    else launch_timed(gemm16_group_kernel<false, false>, dim3((unsigned)g.off[g.n]), dim3(256), s, true, true, g);
  } else {
    bool fits = true, drop = false;
    int n_keep = 0;
    for (int p = 0; p < g.n; ++p) {
      fits = fits && nn16_fits(g.a[p]);
      n_keep += g.a[p].keep != nullptr;
    }
    if (n_keep != 0 && n_keep != g.n) return hipErrorInvalidValue;
    drop = n_keep > 0;
    if (fits && drop)
      launch_timed(gemm16_group_kernel<true, true>, dim3((unsigned)g.off[g.n]), dim3(256), s, true, true, g);
    else if (fits)
      launch_timed(gemm16_group_kernel<false, true>, dim3((unsigned)g.off[g.n]), dim3(256), s, true, true, g);
    else
      launch_timed(gemm_group_kernel<NN>, dim3((unsigned)g.off[g.n]), dim3(512), s, true, true, g);
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_gemm_group_nt(const GemmGroup& g, hipStream_t s) { return launch_gemm_group<false>(g, s); }
hipError_t launch_gemm_group_nn(const GemmGroup& g, hipStream_t s) { return launch_gemm_group<true>(g, s); }

}  // namespace dsv
