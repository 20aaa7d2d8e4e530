// plan.h -- host plan and packed device metadata of a co-batched batch.
//
// The segment table of one batch (Sec. 3.2: inference entries and
// fine-tuning samples, each bound to one adapter) is turned once into int32
// work lists that every projection of the batch reuses.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include "dsv.h"

namespace dsv {

// GEMM row tiles come in two heights (256 and 128 output rows per
// workgroup).  The low-rank term of a row either rides its tile (the tile adds
// it with matrix-core instructions for each "group" = run of rows of one
// adapter) or comes from the gathered path.  That choice is made per 128-row
// block: its up to kBlockGroups longest runs of at least kMinGroupRows rows
// ride the tile, every other row (short segments such as single-token decode
// entries) is gathered.  A 256-row tile carries the groups of its two blocks.
constexpr int kTileM = 256;
constexpr int kBlockM = 128;
constexpr int kBlockGroups = 4;
constexpr int kMaxGroups = 8;
constexpr int kMinGroupRows = 4;
// Rows per gathered / g work item (one 16-row matrix-core tile) and per
// shrink item (two 16-row tiles sharing the adapter operand).
constexpr int kItemRows = 16;
constexpr int kRankItemRows = 32;
// Training rows per chunk of the backward reductions over tokens.
constexpr int kChunkRows = 256;

// tile descriptor: {row0, n_groups, has_gather, n_rows, {adapter, lo, hi} x kMaxGroups}
constexpr int kTileWords = 4 + 3 * kMaxGroups;
// item descriptor: {adapter, begin, count, aux}
constexpr int kItemWords = 4;

// Word offsets of each array inside the packed blob (int32 words).
struct MetaLayout {
  int64_t row_adapter;   // [T]   adapter of each token row
  int64_t row_train;     // [T]   compact training index or -1
  int64_t train_rows;    // [T_t] token row of each compact training index
  int64_t train_adapter; // [T_t] adapter of each compact training index
  int64_t shrink_rows;   // [T]   token rows sorted by (adapter, row)
  int64_t shrink_items;  // [n_shrink][4] {adapter, begin, count <= 32, 0} into shrink_rows
  int64_t gslot;         // [T]   slot of a gathered row or -1
  int64_t gather_rows;   // [T_g] token row of each gathered slot
  int64_t gather_items;  // [n_gitems][4] {adapter, slot_begin, count, 0}
  int64_t fwd_tiles;     // [n_ftiles][kTileWords] 256-row tiles over token rows
  int64_t fwd_tiles128;  // [n_ftiles128][kTileWords] 128-row tiles over token rows
  int64_t bwd_tiles;     // [n_btiles][kTileWords] <= 256-row tiles over compact training rows
  int64_t bwd_tiles128;  // [n_btiles128][kTileWords] <= 128-row tiles
  int64_t chunks;        // [n_chunks][4] {adapter, begin, count, train_adapter_slot}
  int64_t train_items;   // [n_titems][4] {adapter, begin, count, 0}: <= 16 compact rows
  int64_t train_ads;     // [n_tads] adapters owning training rows (ascending)
  int64_t ad_slot;       // [n_ad]  index into train_ads or -1
  int64_t tad_chunk_ptr; // [n_tads + 1] CSR over chunk ids per training adapter
  int64_t tad_chunks;    // [n_chunks]   chunk ids, grouped by training adapter
  int64_t ranks;         // [n_ad]  rank of each adapter
  int64_t scales;        // [n_ad]  scale of each adapter (float bits)
  int64_t total_words;
};

}  // namespace dsv

struct dsv_plan {
  int32_t T = 0, n_ad = 0, r_max = 0, T_t = 0;
  // largest rank among the adapters with rows / with training rows: the rank-r
  // kernels size their rank tiles for these rather than for r_max
  int32_t r_used = 0, r_train = 0;
  int32_t n_ftiles = 0, n_shrink = 0, n_gather = 0, n_gitems = 0, n_btiles = 0,
          n_chunks = 0, n_tads = 0, n_titems = 0, n_ftiles128 = 0, n_btiles128 = 0;
  // every 256-row backward tile t covers compact rows [256 t, min(T_t, 256 t + 256))
  // (no tile ends early at the adapter-run limit), as every forward tile does
  bool btiles_uniform = false;
  std::vector<int32_t> ranks;
  std::vector<float> scales;
  std::vector<int32_t> train_rows;     // host copy, compact order
  std::vector<int32_t> gather_rows;    // host copy, slot order
  std::vector<int32_t> tad_max_chunks; // chunks per training adapter (host copy)
  std::vector<int32_t> meta;           // packed blob, host image
  dsv::MetaLayout lay{};
  void* d_meta = nullptr;              // device copy (nullptr: host-only plan)
  void* copy_done = nullptr;           // hipEvent_t recorded after the upload
  const int32_t* dptr(int64_t off) const {
    return static_cast<const int32_t*>(d_meta) + off;
  }
};
