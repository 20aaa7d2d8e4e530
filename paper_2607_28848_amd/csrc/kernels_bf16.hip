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
//   token_reduce     fp32 per-chunk partials of dy^T h (dB) that also
//                    contract the dy rows they stage with B_a: per-block
//                    partials of g = s_a dy B_a, so dy is read once for both.
//   g finish         fixed-order sum of g's block partials, rounded once.
//   token_reduce     fp32 per-chunk partials of x^T g (dA).
//   reduce_out       fixed-order sum of the partials into dB / dA.
//   gemm (NT / NN)   dx = dy W + g A_a (prologue adds g A_a).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

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
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) uint32_t lds_u32;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

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

__device__ __forceinline__ void vmem_wait_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

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

// s_waitcnt immediate (gfx9 encoding): wait until at most n vector-memory
// operations of this wave are outstanding; lgkm and exp counters untouched.
constexpr int vmcnt_imm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

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

// Issue order of the instructions before it in its block: NV pairs (MFMA,
// vector-memory read), then ND pairs (MFMA, LDS read), then the other MFMAs.
template <int NV, int ND, int NM>
__device__ __forceinline__ void sched_interleave() {
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
  }
#pragma unroll
  for (int q = 0; q < ND; ++q) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, NM - NV - ND, 0);
}

// DROP: the instantiation that masks the low-rank term (dX under LoRA
// dropout); the others carry no masking code.
template <bool SK, bool DROP>
__device__ __forceinline__ void gemm_piece16(const GemmArgs& g, char* smem, int tid, int lin, int t_sk, int piece,
                                             int kb, int ke, int nk) {
  constexpr int TM = 256, TN = 256, TK = 64, NW = 4, WM = 128, WN = 128, FM = 8, FN = 8;
  constexpr int ROWB = TK * 2;                   // bytes per LDS row
  constexpr int A_BYTES = TM * ROWB, STAGE = A_BYTES + TN * ROWB;
  constexpr int LOADS = TM * ROWB / 1024 / 4;    // 1 KiB direct loads per wave per operand
  static_assert(LOADS == 8 && TN == TM, "load split");
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

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
  // Both operands are contraction-contiguous rows of the same length (the
  // launcher checks ldp == ldq), so one set of lane offsets serves both.
  const int ld = (int)g.ldp;
  const int64_t a_rows = min((int64_t)TM, (int64_t)g.M - m0);
  const int64_t b_cols = min((int64_t)TN, (int64_t)g.Nout - n0);
  // Descriptors over the tile's row panels (rows past the operand read zeros);
  // a K-step adds 2 k0 bytes to the scalar offset.  A panel is at most 256
  // rows of 2^20 elements, so every offset fits in 32 bits.
  const i32x4 ra = make_rsrc(g.P + (int64_t)m0 * ld, (uint64_t)a_rows * ld * 2);
  const i32x4 rb = make_rsrc(g.Q + (int64_t)n0 * ld, (uint64_t)b_cols * ld * 2);

  // Operand loads: load i of a wave fills LDS rows 8q .. 8q+7 (q = 8 wave + i),
  // lane ln taking row 8q + ln/8, logical chunk (ln%8) ^ swz(row), which is
  // (ln%8) ^ (ln/8) ^ i.  The lane parts of the offsets stay in registers; the
  // row block and the K-step go in the scalar offset.
  const int lr = lane >> 3;
  int voff[LOADS];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) voff[i] = ((((lane & 7) ^ lr ^ i) << 4)) + lr * ld * 2;
  // whole K-step kt into `stage` (k0 + TK <= C)
  auto issue_whole = [&](int kt, int stage) {
    const int kbytes = kt * TK * 2;
    char* sa = smem + stage * STAGE;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int q = wave * LOADS + i;
      llvm_amdgcn_raw_buffer_load_lds(ra, (lds_u32*)(sa + q * 1024), 16, voff[i],
                                      __builtin_amdgcn_readfirstlane(q * 16 * ld + kbytes), 0, 0);
    }
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int q = wave * LOADS + i;
      llvm_amdgcn_raw_buffer_load_lds(rb, (lds_u32*)(sa + A_BYTES + q * 1024), 16, voff[i],
                                      __builtin_amdgcn_readfirstlane(q * 16 * ld + kbytes), 0, 0);
    }
  };
  // any K-step: chunks past the contraction read nothing (zeros)
  auto issue = [&](int kt, int stage) {
    const int k0 = kt * TK;
    if (k0 + TK <= g.C) {
      issue_whole(kt, stage);
      return;
    }
    char* sa = smem + stage * STAGE;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int q = wave * LOADS + i;
      const int row = 8 * q + lr;
      const int c = (lane & 7) ^ swz<TK>(row);
      const int vo = (k0 + 8 * c < g.C) ? (row * ld + k0 + 8 * c) * 2 : (int)0x7FFFFFF0;
      llvm_amdgcn_raw_buffer_load_lds(ra, (lds_u32*)(sa + q * 1024), 16, vo, 0, 0, 0);
      llvm_amdgcn_raw_buffer_load_lds(rb, (lds_u32*)(sa + A_BYTES + q * 1024), 16, vo, 0, 0, 0);
    }
  };

  issue(kb, 0);

  // The first group's first 16 ranks are loaded between the first two
  // K-steps, so the wait for them is the wait for the first K-step alone
  // (vector-memory operations complete in order) rather than for both.  This
  // covers the forward form (h and B rows with contiguous ranks, r a multiple
  // of 16) for a wave that has rows in the group; anything else loads below.
  const bool pre = kb == 0 && ngroups > 0 && g.lq_j == 1 && (g.lq_col & 3) == 0 && (g0_r & 15) == 0 &&
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
  // the prefetched step: its data arrive with the first K-step
  if (pre) lr_mfma(pre_h, pre_b, g0_lo, g0_hi, 4, g0_sc);
  // every other (group, 16-rank step) of the tile
  for (int gi = 0; kb == 0 && gi < ngroups; ++gi) {
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
  // A 16-column block lies inside one 32-column mask word.
  if (DROP && kb == 0 && g.keep != nullptr) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WM + 16 * i + (lane & 15);
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int c0 = n0 + wn * WN + 16 * j;
        const int wd = c0 >> 5;
        const uint32_t x = g.keep[(int64_t)(m0 + min(row, nrows - 1)) * g.keep_words + min(wd, g.keep_words - 1)];
        const uint32_t mw = x & (0u - (uint32_t)(row < nrows && wd < g.keep_words));
        const int bit = (c0 & 31) + 4 * (lane >> 4);
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[i][j][v] = ((mw >> (bit + v)) & 1u) ? acc[i][j][v] * g.keep_scale : 0.f;
      }
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
  auto rd_b = [&](const char* st, int s, int j) {
    return as_bf(*reinterpret_cast<const u32x4*>(st + off_b[((2 * s) ^ j) & 3] + 16 * j * ROWB));
  };

  // Fragments: two A sets (the current step's and the next one's) and one B
  // set whose fragment j is replaced by the next step's once the 8 MFMAs of
  // column block j have been issued.
  bf16x8 fa0[FM], fa1[FM], fb[FN];
  if (ke - kb >= 2) __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * LOADS));  // first K-step landed
  else vmem_wait_all();
  __syncthreads();
#pragma unroll
  for (int j = 0; j < FN; ++j) fb[j] = rd_b(smem, 0, j);
#pragma unroll
  for (int i = 0; i < FM; ++i) fa0[i] = rd_a(smem, 0, i);

  // Direct loads of whole K-step kl into buffer ls: load n of the wave's 16
  // (A for n < 8, B after).  A texture unit takes a 1 KiB load in about 16
  // cycles, so the 64 loads a K-step needs per CU are spread evenly, two per
  // wave per column block (a block's 8 MFMAs take 128 cycles), over the
  // second step, after the barrier that frees their buffer.
  auto load_n = [&](int kl, int ls, int n) {
    const int i = n & 7;
    const int q = wave * LOADS + i;
    llvm_amdgcn_raw_buffer_load_lds(n < 8 ? ra : rb, (lds_u32*)(smem + ls * STAGE + (n < 8 ? 0 : A_BYTES) + q * 1024),
                                    16, voff[i], __builtin_amdgcn_readfirstlane(q * 16 * ld + kl * TK * 2), 0, 0);
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
    step(fa0, fa1, smem + stage * STAGE, 1, false, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    vmem_wait_all();  // kt+1 landed (its loads are the only ones in flight)
    __syncthreads();  // everyone's part of kt+1 is in; buffer `stage` is free
    __builtin_amdgcn_sched_barrier(0);
    if (!load && kt + 2 < ke) issue(kt + 2, stage);  // a partial last K-step
    step(fa1, fa0, smem + (stage ^ 1) * STAGE, 0, load, kt + 2, stage);
  };
  int kt = kb, stage = 0;
  const int main_end = min(ke, g.C / TK) - 2;  // kt < main_end: kt+2 is whole and below ke
  for (; kt < main_end; ++kt, stage ^= 1) kstep(kt, stage, true);
  for (; kt + 1 < ke; ++kt, stage ^= 1) kstep(kt, stage, false);
  // the last K-step: no successor to read
  step(fa0, fa1, smem + stage * STAGE, 1, false, 0, 0);
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
  char* slice = smem + (last_stage ^ 1) * STAGE + wave * 32 * SRS;
  const bool gathered = has_gather && g.delta != nullptr;
#pragma unroll
  for (int t = 0; t < FM / 2; ++t) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int i = 2 * t + h;
      const int row = wm * WM + 16 * i + l15;
      const int gs = (gathered && row < nrows) ? g.gslot[m0 + row] : -1;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = wn * WN + 16 * j + 4 * (lane >> 4);
        f32x4 x = acc[i][j];
        if (gathered) {
          const f32x4 d = *reinterpret_cast<const f32x4*>(g.delta + (int64_t)max(gs, 0) * g.Nout +
                                                          min(n0 + col, g.Nout - 4));
          x += (gs >= 0 && n0 + col < g.Nout) ? d : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        const uint32_t w0 = f2bf2(x[0], x[1]), w1 = f2bf2(x[2], x[3]);
        *reinterpret_cast<uint2*>(slice + (16 * h + l15) * SRS + 2 * (col - wn * WN)) = make_uint2(w0, w1);
      }
    }
    asm volatile("" ::: "memory");  // a wave's LDS accesses run in order: the slice is complete
    constexpr int CPR = WN / 8;     // 16-byte chunks per slice row
#pragma unroll
    for (int q = 0; q < 32 * CPR / 64; ++q) {
      const int id = 64 * q + lane;
      const int rr = id / CPR, ch = id % CPR;
      const u32x4 v = *reinterpret_cast<const u32x4*>(slice + rr * SRS + 16 * ch);
      const int orow = wm * WM + 32 * t + rr, ocol = n0 + wn * WN + 8 * ch;
      if (orow < nrows && ocol < g.Nout)
        __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(g.out + (int64_t)(m0 + orow) * g.ldo + ocol));
    }
    asm volatile("" ::: "memory");  // the slice is read before the next rows overwrite it
  }
}

template <bool SK, bool DROP>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm16_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * 2 * 256 * 64 * 2];
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
  gemm_piece16<SK, DROP>(g, smem, threadIdx.x, lin, t_sk, piece, kb, ke, nk);
}

template <bool DROP>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm16_group_kernel(GemmGroup G) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * 2 * 256 * 64 * 2];
  int pj = 0;
  while (pj + 1 < G.n && (int)blockIdx.x >= G.off[pj + 1]) ++pj;
  const GemmArgs g = G.a[pj];
  const int local = (int)blockIdx.x - G.off[pj];
  const int lin = xcd_major(local, G.off[pj + 1] - G.off[pj]);
  const int nk = (g.C + 63) / 64;
  gemm_piece16<false, DROP>(g, smem, threadIdx.x, lin, -1, 0, 0, nk, nk);
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
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];
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
      if (k < kcap[i])
        llvm_amdgcn_global_load_lds((global_cv*)(src[i] + c * SK_CK), (lds_u32*)(base + q * 1024), 16, 0, 0);
      else
        *reinterpret_cast<u32x4*>(base + q * 1024 + 16 * lane) = zero4();
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
    vmem_wait_all();
    __syncthreads();  // chunk c is in; every wave is done with chunk c - 1's buffer
    if (c + 1 < nch) issue(c + 1, (c + 1 - c_beg) & 1);
    if constexpr (DROP) load_mask(min(c + 1, nch - 1), ml);  // unconditional: no merge to wait on
    const char* sb = smem + ((c - c_beg) & 1) * STAGE;
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
    if constexpr (DROP) load_mask(c_beg, m0);
  }
  for (int c = c_beg; c < nch; c += 2) {
    chunk(c, m0, m1);
    if (c + 1 < nch) chunk(c + 1, m1, m0);
  }
  __syncthreads();  // the stage buffers become the reduction buffer
  constexpr int RW = 16 * NJ + 1;
  static_assert(SW * ROWS * RW * 4 <= 2 * STAGE, "reduction buffer");
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
    // contraction, one row length)
    if (tm == 256 && tn == 256) {
      if (a.ldp != a.ldq) return hipErrorInvalidValue;
      const bool drop = a.keep != nullptr;
      if (a.sk_tiles > 0) {
        if (drop) launch_timed(gemm16_kernel<true, true>, grid, dim3(256), s, true, false, a);
        else launch_timed(gemm16_kernel<true, false>, grid, dim3(256), s, true, false, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        launch_timed(split_fixup_kernel<NN, 256, 256>, dim3((unsigned)a.sk_tiles * (256 * 256 / 4 / 256)), dim3(256),
                     s, false, true, a);
      } else if (drop) {
        launch_timed(gemm16_kernel<false, true>, grid, dim3(256), s, true, true, a);
      } else {
        launch_timed(gemm16_kernel<false, false>, grid, dim3(256), s, true, true, a);
      }
      return hipGetLastError();
    }
  }
  if constexpr (NN) {  // 256 x 256 NN tiles (dX reading W transposed in LDS)
    if (tm == 256 && tn == 256) {
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

template <bool NN>
hipError_t launch_gemm_group(const GemmGroup& g, hipStream_t s) {
  if (g.n <= 0 || g.n > kMaxGroup || g.off[0] != 0) return hipErrorInvalidValue;
  for (int p = 0; p < g.n; ++p) {
    const GemmArgs& a = g.a[p];
    if (g.off[p + 1] - g.off[p] != a.n_mtiles * a.n_ntiles || a.sk_tiles != 0) return hipErrorInvalidValue;
  }
  if (g.off[g.n] <= 0) return hipSuccess;
  if constexpr (!NN) {
    for (int p = 0; p < g.n; ++p)
      if (g.a[p].ldp != g.a[p].ldq) return hipErrorInvalidValue;
    bool drop = false;
    for (int p = 0; p < g.n; ++p) drop = drop || g.a[p].keep != nullptr;
    if (drop) launch_timed(gemm16_group_kernel<true>, dim3((unsigned)g.off[g.n]), dim3(256), s, true, true, g);
    else launch_timed(gemm16_group_kernel<false>, dim3((unsigned)g.off[g.n]), dim3(256), s, true, true, g);
  } else {
    launch_timed(gemm_group_kernel<NN>, dim3((unsigned)g.off[g.n]), dim3(512), s, true, true, g);
  }
  return hipGetLastError();
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

hipError_t launch_gemm_group_nt(const GemmGroup& g, hipStream_t s) { return launch_gemm_group<false>(g, s); }
hipError_t launch_gemm_group_nn(const GemmGroup& g, hipStream_t s) { return launch_gemm_group<true>(g, s); }

}  // namespace dsv
