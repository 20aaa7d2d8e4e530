// kernels.h -- argument blocks and host launchers of the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dsv {

// GEMM with a low-rank prologue:  out = P Q' + (low-rank term) rounded once.
//   NT (forward):  out[m][n] = sum_c P[m][c] Q[n][c]        Q is [Nout][C]
//   NN (dX):       out[m][n] = sum_c P[m][c] Q[c][n]        Q is [C][Nout]
// Low-rank term of a row m in tile group (a, lo, hi):
//   scale(a) * sum_j Lp[m][j] Lq(a, j, n),  j < rank(a),
//   Lq(a, j, n) = Lq[a * lq_ad + j * lq_j + n * lq_col]
// Rows gathered elsewhere add delta[gslot[m]][n] (fp32, already scaled).
struct GemmArgs {
  const uint16_t* P;
  int64_t ldp;
  const uint16_t* Q;
  int64_t ldq;
  uint16_t* out;
  int64_t ldo;
  int32_t M;             // rows of P (bounds of the operand loads)
  int32_t Nout, C;
  const int32_t* tiles;  // row tiles, kTileWords words each
  int32_t uniform_rows;  // 256-row tile mt is rows [256 mt, min(M, 256 mt + 256)): no descriptor read needed
  int32_t n_mtiles, n_ntiles;
  const uint16_t* Lp;
  int64_t ldl;
  const uint16_t* Lq;
  int64_t lq_ad, lq_j, lq_col;
  const int32_t* ranks;
  const float* scales;   // nullptr: scale 1
  const float* delta;    // nullptr: no gathered rows
  const int32_t* gslot;
  // Work split over n_mtiles * n_ntiles tiles (tile order: groups of 8 row
  // tiles walked column by column).  Workgroups [0, dp_tiles) take tiles
  // [0, dp_tiles) whole; tiles [dp_tiles, tiles) (sk_tiles of them) are each
  // split into sk_split equal K ranges, one workgroup per piece, dispatched
  // after the whole tiles.  Pieces write fp32 partials to sk_part (one tm * tn
  // slot per piece); a second kernel sums them and writes those tiles.
  int32_t dp_tiles, sk_tiles, sk_split;
  float* sk_part;
  // dX under LoRA dropout: the prologue's low-rank term of row r, column c is
  // kept (times keep_scale) when bit c % 32 of keep[r][c / 32] is set, else
  // zeroed, before the main loop adds the base product (keep == nullptr: none)
  const uint32_t* keep;
  int32_t keep_words;
  float keep_scale;
};

// Rank-r contraction of a few rows of one adapter (shrink h = x A^T, and
// g = s dy B in the backward).
struct SkinnyArgs {
  const uint16_t* P;
  int64_t ldp;
  const int32_t* rows;   // item element -> P row
  const int32_t* items;  // {adapter, begin, count, aux}
  const uint16_t* Q;     // per adapter slot: [r][C], row stride ldq
  int64_t q_ad, ldq;
  const int32_t* qsel;   // adapter -> Q slot (nullptr: the adapter id)
  const int32_t* ranks;
  const float* scales;   // nullptr: scale 1
  int32_t C;
  // outputs (mode-dependent)
  uint16_t* out1;        // [rows][ld1] (shrink: nullptr = not written)
  int64_t ld1;
  uint16_t* out2;        // shrink: H_save [T_t][ld2] via row_train (nullptr: none)
  int64_t ld2;
  const int32_t* row_train;
  // dropout of the training rows (shrink only; keep == nullptr: none):
  // masked input elements, sum scaled by drop_scale
  const uint32_t* keep;
  int32_t keep_words;
  float drop_scale;
  // Contraction split (skinny_split): with more than one piece, piece q
  // sums chunks [q * cpp, (q + 1) * cpp) and writes the fp32 sum of element
  // (begin + row, j) of the item list to part[(q * part_n + begin + row) *
  // r_max + j]; a second kernel adds the pieces in order and stores the result.
  float* part;           // [pieces][part_n][r_max] (unused with one piece)
  int32_t part_n;        // length of the item list (rows grouped by item)
  int32_t r_max;
  int32_t split_items;   // the plan's item count that sets the split
  int32_t pieces, cpp;   // set by the launcher
};

// Contraction split of the rank-r contractions: a launch whose items alone
// cannot cover the CUs (fewer than kSkinnySplitBelow items of one projection)
// splits each item's contraction (chunks of 256 columns) into up to
// kMaxSkinnyPieces pieces of at least kSkinnyMinChunks chunks, aiming at
// kSkinnySplitTarget workgroups; with more items the bandwidth is already
// shared by enough workgroups and a split only adds the second pass.  The
// split depends on C and on the plan's item count (split_items), not on the
// launch: the forward shrink and the backward's recomputed h take the shrink's
// item count, so both sum every row in the same order.
constexpr int kSkinnySplitBelow = 160;
constexpr int kSkinnySplitTarget = 384;
constexpr int kSkinnyMinChunks = 4;
constexpr int kMaxSkinnyPieces = 8;
inline void skinny_split(int32_t C, int32_t split_items, int32_t* pieces, int32_t* cpp) {
  const int32_t nch = (C + 255) / 256;
  int32_t p = 1;
  if (split_items > 0 && split_items < kSkinnySplitBelow) {
    p = (kSkinnySplitTarget + split_items - 1) / split_items;
    p = p > nch / kSkinnyMinChunks ? nch / kSkinnyMinChunks : p;
    p = p > kMaxSkinnyPieces ? kMaxSkinnyPieces : p;
    p = p < 1 ? 1 : p;
  }
  int32_t c = (nch + p - 1) / p;
  c = c < 1 ? 1 : c;
  *cpp = c;
  *pieces = nch > 0 ? (nch + c - 1) / c : 1;
}
// fp32 partial bytes a rank-r contraction over C needs for an item list of n
// elements (0 when it is not split).
inline size_t skinny_part_bytes(int32_t C, int32_t split_items, int64_t n, int32_t r_max) {
  int32_t pieces, cpp;
  skinny_split(C, split_items, &pieces, &cpp);
  return pieces > 1 ? (size_t)pieces * (size_t)n * (size_t)r_max * 4 : 0;
}

// Per-chunk fp32 partial sums over training tokens:
//   part[chunk][c][j] = sum_{t in chunk} P[prow(t)][c] Q[t][j]
// With B (the g launch, P = dY), the same workgroup also contracts the P rows
// it stages with the adapter's B over its 256-column block cb:
//   gpart[cb][t][j] = sum_{c in block cb} P[t][c] B_a[c][j]
// (g = s_a dy B_a once the blocks are summed in order, by launch_g_finish_group).
struct TokenReduceArgs {
  const uint16_t* P;
  int64_t ldp;
  const int32_t* prow;   // compact row -> P row (nullptr: identity)
  const uint16_t* Q;     // [T_t][ldq], compact rows
  int64_t ldq;
  const int32_t* chunks;
  const int32_t* ranks;
  int32_t C, r_max;
  float* part;
  const uint32_t* keep;  // dropout mask of P's elements (compact rows), nullptr: none
  int32_t keep_words;
  const uint16_t* B;     // g launch: adapter stacks [n_ad][C][r_max]
  float* gpart;          // g launch: [token_col_blocks(C)][gpart_n][r_max]
  int32_t gpart_n;       // T_t
};

// Grouped launches: one kernel runs the same step of up to kMaxGroup
// projections (same plan, per-projection operands), the projection picked
// from the workgroup id.  The single-projection launchers below are groups
// of one.
constexpr int kMaxGroup = 8;
// Columns per workgroup of the token reductions.
constexpr int kTokenCols = 256;
inline int32_t token_col_blocks(int32_t C) { return (C + kTokenCols - 1) / kTokenCols; }
struct SkinnyGroup {
  SkinnyArgs a[kMaxGroup];
  int32_t n;
  // set by the launcher: workgroup row y runs piece slot_piece[y] of a[slot_proj[y]]
  int32_t slot_proj[kMaxGroup * kMaxSkinnyPieces];
  int32_t slot_piece[kMaxGroup * kMaxSkinnyPieces];
};
struct GatherArgs {           // gathered low-rank term of one projection
  const uint16_t* H;          // h of every row [T][ldh]
  const uint16_t* B;          // adapter stacks [n_ad][N][r_max]
  int32_t N;
  float* delta;               // [n_gather][N] fp32 out
};
struct GatherGroup {
  GatherArgs a[kMaxGroup];
  int32_t yoff[kMaxGroup + 1];  // prefix of the 256-column blocks
  int32_t n;
};
struct TokenReduceGroup {
  TokenReduceArgs a[2 * kMaxGroup];
  int32_t yoff[2 * kMaxGroup + 1];  // prefix of the kTokenCols-column blocks
  int32_t n;
};
// GEMM group: whole 256x256 tiles, workgroups [off[p], off[p+1]) take the
// tiles of projection a[p] (XCD-major within the projection).
struct GemmGroup {
  GemmArgs a[kMaxGroup];
  int32_t off[kMaxGroup + 1];
  int32_t n;
};

// Device scratch of the allocation-free forward (dsv_cobatch_fwd_noalloc): a
// file-scope array of kNoAllocScratchBytes in the library's device memory,
// one copy per device.  noalloc_scratch() returns the current device's address
// of it (looked up with hipGetSymbolAddress on the device's first call and kept).
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
hipError_t noalloc_scratch(void** out);

// Launchers (bf16).  Each returns hipSuccess or the launch error.
// Tile shapes (tm x tn): 256x256 or 128x128; `tiles` must be the
// plan's row-tile list of height tm.  Split tiles (sk_tiles > 0) are
// supported for 256x256 only.
hipError_t launch_gemm_nt(const GemmArgs& a, int tm, int tn, hipStream_t s);
// Benchmark timing: the next GEMM launch (launch_gemm_nt / _nn / _group_*)
// records `start` as its first kernel begins and `stop` as its last kernel
// ends, within the kernels' dispatches.  launch_events_pending() is true while
// an event has not been handed to a launch (nothing was launched).
void set_launch_events(hipEvent_t start, hipEvent_t stop);
bool launch_events_pending();
hipError_t launch_gemm_nn(const GemmArgs& a, int tm, int tn, hipStream_t s);
// Rank-r contractions: r_sel bounds the rank of every item's adapter (it sizes
// the rank tiles); the partials of a split contraction have stride a.r_max.
hipError_t launch_shrink(const SkinnyArgs& a, int32_t n_items, int32_t r_sel, hipStream_t s);
// shrink over items of <= 16 rows (the training items): recomputes h for the backward
hipError_t launch_shrink_train(const SkinnyArgs& a, int32_t n_items, int32_t r_sel, hipStream_t s);
hipError_t launch_gather_expand(const uint16_t* H, int64_t ldh, const uint16_t* B, int32_t N,
                                int32_t r_max, const int32_t* items, int32_t n_items,
                                const int32_t* gather_rows, const int32_t* ranks,
                                const float* scales, float* delta, hipStream_t s);
// Fixed-order sum of one reduction's chunk partials into its output.
struct ReduceOutArgs {
  const float* part;
  int32_t C;
  const float* scales;  // nullptr: scale 1
  int32_t a_layout;     // 1: out[a][j][c] (dA), 0: out[a][c][j] (dB)
  float* out;
  float post;           // extra factor (dropout scale of dA), 1 otherwise
};
struct ReduceOutGroup {
  ReduceOutArgs a[2 * kMaxGroup];
  int32_t n;
};
// Both final sums of a backward in one launch.
hipError_t launch_reduce_out(const ReduceOutArgs& o0, const ReduceOutArgs& o1, int32_t r_max, int32_t r_sel,
                             const int32_t* train_ads, int32_t n_tads, const int32_t* tad_ptr,
                             const int32_t* tad_chunks, const int32_t* ranks, int32_t accumulate, hipStream_t s);
// Grouped forms (n >= 1 entries filled).
hipError_t launch_shrink_group(const SkinnyGroup& g, int32_t n_items, int32_t r_sel, hipStream_t s);
hipError_t launch_shrink_train_group(const SkinnyGroup& g, int32_t n_items, int32_t r_sel, hipStream_t s);
hipError_t launch_gather_group(const GatherGroup& g, int64_t ldh, int32_t r_max, const int32_t* items,
                               int32_t n_items, const int32_t* gather_rows, const int32_t* ranks,
                               const float* scales, hipStream_t s);
// Token reductions of a backward, every entry with one r_max.  r_sel: the
// largest rank of a training adapter (sizes the rank tiles; the partials keep
// the r_max stride).  Either every entry carries B (the dB reductions, which
// also write the g partials of their column blocks; no dropout mask) or none
// does (the dA reductions).
hipError_t launch_token_reduce_group(const TokenReduceGroup& g, int32_t n_chunks, int32_t r_sel, hipStream_t s);
// g = s_a * (sum of the column blocks' partials, in block order), rounded once
// to bf16, for every projection of the group: entry p sums a[p].pieces
// partials of a[p].part ([pieces][part_n][r_max]) over the items (compact
// training rows of one adapter) and stores a[p].out1[row][j], j < r_a.
hipError_t launch_g_finish_group(const SkinnyGroup& g, int32_t n_items, hipStream_t s);
hipError_t launch_reduce_out_group(const ReduceOutGroup& g, int32_t r_max, int32_t r_sel, const int32_t* train_ads,
                                   int32_t n_tads, const int32_t* tad_ptr, const int32_t* tad_chunks,
                                   const int32_t* ranks, int32_t accumulate, hipStream_t s);
hipError_t launch_gemm_group_nt(const GemmGroup& g, hipStream_t s);
hipError_t launch_gemm_group_nn(const GemmGroup& g, hipStream_t s);

// Fused AdamW step of the training adapters' A and B slices of up to
// kMaxGroup projections in one launch (fp32 master weights and moments in
// the A / B layouts; the parameter copy A / B is bf16 when bf16 != 0, fp32
// otherwise, or not written when nullptr).  Projection p owns blocks
// [blk_begin, blk_begin + n_tads * bpa): bpa blocks per training adapter, over
// the adapter's A slice (float4 units) and then its B slice (float4 units of
// four rank entries when bvec, single entries otherwise).
struct AdamWProj {
  int32_t K, N;
  int32_t blk_begin, bpa;
  const float *dA, *dB;
  float *pA, *pB, *mA, *vA, *mB, *vB;
  void *A, *B;
};
struct AdamWArgs {
  int32_t r_max, n_proj, bvec, bf16;
  const int32_t* train_ads;  // training adapters (device)
  const int32_t* ranks;
  float decay;               // 1 - lr * wd
  float b1, b2, c1, c2, eps; // beta1, beta2, 1 - beta1, 1 - beta2
  float step_size;           // lr / (1 - b1^t)
  float sqrt_bc2;            // sqrt(1 - b2^t)
  AdamWProj proj[kMaxGroup];
};
hipError_t launch_adamw(const AdamWArgs& a, int64_t n_blocks, hipStream_t s);

// LoRA dropout of the training rows: mask parameters (thr = floor(p 2^32),
// scale = 1 / (1 - p)) and the bitmask kernel.
struct DropoutSpec {
  uint32_t thr;
  float scale;
  uint64_t seed, offset;
};
// bits: [Tt][ceil(K / 32)] words, bit b of word w keeps column 32 w + b.
// The masks of up to kMaxGroup projections (same Tt) in one launch; entries
// with bits == nullptr are skipped.
struct DropoutMaskGroup {
  uint32_t* bits[kMaxGroup];
  int32_t K[kMaxGroup];
  DropoutSpec d[kMaxGroup];
  int32_t n;
};
hipError_t launch_dropout_mask_group(const DropoutMaskGroup& g, int32_t Tt, hipStream_t s);
hipError_t launch_dropout_mask(uint32_t* bits, int32_t Tt, int32_t K, const DropoutSpec& d, hipStream_t s);


// Launchers (fp32 mode: plain FMA kernels, same semantics).
struct F32Args {
  int32_t T, Tt, K, N, r_max;
  const int32_t* row_adapter;
  const int32_t* row_train;
  const int32_t* train_rows;
  const int32_t* train_adapter;
  const int32_t* train_ads;
  int32_t n_tads;
  const int32_t* tad_ptr;
  const int32_t* tad_chunks;
  const int32_t* chunks;
  const int32_t* ranks;
  const float* scales;
  const float *X, *W, *A, *B, *Hs, *dY;
  float *Y, *Hsave, *Hall, *G, *dA, *dB, *dX;
  int64_t ldx, ldw, ldy, lddy, lddx;  // row strides of X, W, Y, dY, dX
  float* Hrec;   // backward with Hs == nullptr: h of the training rows recomputed here
  const uint32_t* keep;  // dropout mask of the training rows (nullptr: none)
  int32_t keep_words;
  float drop_scale;
  int32_t accumulate;
};
hipError_t launch_f32_fwd(const F32Args& a, hipStream_t s);
hipError_t launch_f32_bwd(const F32Args& a, hipStream_t s);

}  // namespace dsv
