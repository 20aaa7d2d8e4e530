// plan.cpp -- validation and packing of a batch's segment table (host only,
// plus one asynchronous host-to-device copy of the packed blob).
//
// Sec. 3.2 of the paper admits each fine-tuning sample as one more entry of
// the host batch, bound to the reserved training adapter, next to inference
// entries on their own adapters (multi-LoRA batching, Sec. 2.2).  The table
// is the same for every projection of the batch, so everything that depends
// only on it is computed here, once.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <numeric>

#include "plan.h"

namespace {

using dsv::kChunkRows;
using dsv::kItemRows;
using dsv::kRankItemRows;
using dsv::kItemWords;
using dsv::kMaxGroups;
using dsv::kMinGroupRows;
using dsv::kBlockGroups;
using dsv::kBlockM;
using dsv::kTileM;
using dsv::kTileWords;

struct Run {
  int32_t lo, hi, adapter;  // [lo, hi) rows, relative to whatever they index
};

// Maximal runs of equal adapter id in ad[lo, hi).
std::vector<Run> runs_of(const int32_t* ad, int32_t lo, int32_t hi) {
  std::vector<Run> out;
  int32_t s = lo;
  for (int32_t t = lo + 1; t <= hi; ++t) {
    if (t == hi || ad[t] != ad[s]) {
      out.push_back({s, t, ad[s]});
      s = t;
    }
  }
  return out;
}

int build(const dsv_segment* segs, int32_t n_segs, int32_t T, const int32_t* rank,
          const float* scale, int32_t n_ad, int32_t r_max, dsv_plan& p) {
  if (n_segs < 0 || T < 0 || n_ad < 1) return DSV_ERR_ARG;
  if ((n_segs > 0 && !segs) || !rank || !scale) return DSV_ERR_ARG;
  if (r_max < 1 || r_max > DSV_MAX_RANK) return DSV_ERR_RANGE;
  for (int32_t a = 0; a < n_ad; ++a) {
    if (rank[a] < 1 || rank[a] > r_max) return DSV_ERR_RANGE;
    if (!std::isfinite(scale[a])) return DSV_ERR_RANGE;
  }
  // Canonical order: non-empty entries by start (table index breaks ties).
  std::vector<int32_t> order;
  order.reserve(n_segs);
  for (int32_t i = 0; i < n_segs; ++i) {
    const dsv_segment& s = segs[i];
    if (s.adapter < 0 || s.adapter >= n_ad) return DSV_ERR_RANGE;
    if (s.is_train != 0 && s.is_train != 1) return DSV_ERR_RANGE;
    if (s.len < 0 || s.start < 0 || (int64_t)s.start + s.len > T) return DSV_ERR_LAYOUT;
    if (s.len > 0) order.push_back(i);
  }
  std::stable_sort(order.begin(), order.end(),
                   [&](int32_t x, int32_t y) { return segs[x].start < segs[y].start; });
  int64_t pos = 0;
  for (int32_t i : order) {
    if (segs[i].start != pos) return DSV_ERR_LAYOUT;  // gap or overlap
    pos += segs[i].len;
  }
  if (pos != T) return DSV_ERR_LAYOUT;

  p.T = T;
  p.n_ad = n_ad;
  p.r_max = r_max;
  p.ranks.assign(rank, rank + n_ad);
  p.scales.assign(scale, scale + n_ad);

  std::vector<int32_t> row_adapter(T), row_train(T, -1);
  std::vector<char> is_train(T, 0);
  for (int32_t i : order) {
    const dsv_segment& s = segs[i];
    for (int32_t t = s.start; t < s.start + s.len; ++t) {
      row_adapter[t] = s.adapter;
      is_train[t] = (char)s.is_train;
    }
  }
  // Compact training order: ascending token row.
  std::vector<int32_t> train_rows, train_adapter;
  for (int32_t t = 0; t < T; ++t)
    if (is_train[t]) {
      row_train[t] = (int32_t)train_rows.size();
      train_rows.push_back(t);
      train_adapter.push_back(row_adapter[t]);
    }
  const int32_t Tt = (int32_t)train_rows.size();
  p.T_t = Tt;
  p.train_rows = train_rows;

  // Shrink work list: rows grouped by adapter (ascending row inside), split
  // into items of kRankItemRows rows; each item reads its adapter's A once.
  std::vector<int32_t> shrink_rows(T);
  std::iota(shrink_rows.begin(), shrink_rows.end(), 0);
  std::stable_sort(shrink_rows.begin(), shrink_rows.end(),
                   [&](int32_t x, int32_t y) { return row_adapter[x] < row_adapter[y]; });
  std::vector<int32_t> shrink_items;
  for (int32_t i = 0; i < T;) {
    int32_t a = row_adapter[shrink_rows[i]], j = i;
    while (j < T && row_adapter[shrink_rows[j]] == a && j - i < kRankItemRows) ++j;
    shrink_items.insert(shrink_items.end(), {a, i, j - i, 0});
    i = j;
  }

  // Forward GEMM row tiles.  Per 128-row block, the longest same-adapter runs
  // of at least kMinGroupRows rows (up to kBlockGroups of them) ride the tile;
  // every other row is gathered by adapter and its fp32 low-rank term is
  // computed beforehand, reading each adapter once.
  std::vector<std::vector<Run>> block_groups;
  std::vector<int32_t> block_gather;
  std::vector<char> gathered(T, 0);
  for (int32_t r0 = 0; r0 < T; r0 += kBlockM) {
    const int32_t r1 = std::min(T, r0 + kBlockM);
    std::vector<Run> runs = runs_of(row_adapter.data(), r0, r1);
    std::vector<int32_t> idx(runs.size());
    std::iota(idx.begin(), idx.end(), 0);
    std::stable_sort(idx.begin(), idx.end(), [&](int32_t x, int32_t y) {
      return runs[x].hi - runs[x].lo > runs[y].hi - runs[y].lo;
    });
    std::vector<Run> groups;
    for (int32_t k : idx)
      if ((int32_t)groups.size() < kBlockGroups && runs[k].hi - runs[k].lo >= kMinGroupRows)
        groups.push_back(runs[k]);
    std::sort(groups.begin(), groups.end(), [](const Run& x, const Run& y) { return x.lo < y.lo; });
    int32_t has_gather = 0;
    for (const Run& r : runs) {
      bool in_group = false;
      for (const Run& g : groups) in_group |= (g.lo == r.lo);
      if (!in_group) {
        has_gather = 1;
        for (int32_t t = r.lo; t < r.hi; ++t) gathered[t] = 1;
      }
    }
    block_groups.push_back(groups);
    block_gather.push_back(has_gather);
  }
  // Tiles of `tm` rows (a multiple of kBlockM): the groups of their blocks,
  // adjacent groups of one adapter merged.
  auto fwd_tiles_of = [&](int32_t tm) {
    std::vector<int32_t> out;
    const int32_t per = tm / kBlockM;
    for (int32_t b0 = 0; b0 < (int32_t)block_groups.size(); b0 += per) {
      const int32_t r0 = b0 * kBlockM, r1 = std::min(T, r0 + tm);
      std::vector<Run> groups;
      int32_t has_gather = 0;
      for (int32_t b = b0; b < std::min<int32_t>(b0 + per, (int32_t)block_groups.size()); ++b) {
        has_gather |= block_gather[b];
        for (const Run& g : block_groups[b]) {
          if (!groups.empty() && groups.back().hi == g.lo && groups.back().adapter == g.adapter)
            groups.back().hi = g.hi;
          else
            groups.push_back(g);
        }
      }
      int32_t w[kTileWords] = {r0, (int32_t)groups.size(), has_gather, r1 - r0};
      for (size_t g = 0; g < groups.size(); ++g) {
        w[4 + 3 * g] = groups[g].adapter;
        w[5 + 3 * g] = groups[g].lo - r0;
        w[6 + 3 * g] = groups[g].hi - r0;
      }
      out.insert(out.end(), w, w + kTileWords);
    }
    return out;
  };
  std::vector<int32_t> fwd_tiles = fwd_tiles_of(kTileM);
  std::vector<int32_t> fwd_tiles128 = fwd_tiles_of(kBlockM);
  // Gathered rows: slots ordered by (adapter, row); items of kItemRows slots.
  std::vector<int32_t> gather_rows, gslot(T, -1), gather_items;
  for (int32_t i = 0; i < T; ++i)
    if (gathered[shrink_rows[i]]) gather_rows.push_back(shrink_rows[i]);
  for (size_t s = 0; s < gather_rows.size(); ++s) gslot[gather_rows[s]] = (int32_t)s;
  p.gather_rows = gather_rows;
  for (int32_t i = 0; i < (int32_t)gather_rows.size();) {
    int32_t a = row_adapter[gather_rows[i]], j = i;
    while (j < (int32_t)gather_rows.size() && row_adapter[gather_rows[j]] == a && j - i < kItemRows) ++j;
    gather_items.insert(gather_items.end(), {a, i, j - i, 0});
    i = j;
  }

  // Backward GEMM row tiles over compact training rows: at most `tm` rows
  // and at most kMaxGroups adapter runs each (a tile ends early otherwise),
  // so every training row's low-rank term rides its tile.
  auto bwd_tiles_of = [&](int32_t tm) {
    std::vector<int32_t> out;
    std::vector<Run> runs = runs_of(train_adapter.data(), 0, Tt);
    size_t k = 0;  // run containing row `cur`
    int32_t r0 = 0;
    while (r0 < Tt) {
      const int32_t limit = std::min(Tt, r0 + tm);
      int32_t w[kTileWords] = {r0, 0, 0, 0};
      int32_t cur = r0, ng = 0;
      while (cur < limit && ng < kMaxGroups) {
        const int32_t hi = std::min(runs[k].hi, limit);
        w[4 + 3 * ng] = runs[k].adapter;
        w[5 + 3 * ng] = cur - r0;
        w[6 + 3 * ng] = hi - r0;
        ++ng;
        cur = hi;
        if (cur == runs[k].hi) ++k;
      }
      w[1] = ng;
      w[3] = cur - r0;
      out.insert(out.end(), w, w + kTileWords);
      r0 = cur;
    }
    return out;
  };
  std::vector<int32_t> bwd_tiles = bwd_tiles_of(kTileM);
  p.btiles_uniform = true;
  for (size_t t = 0; t * kTileWords < bwd_tiles.size(); ++t) {
    const int32_t r0 = bwd_tiles[t * kTileWords], n = bwd_tiles[t * kTileWords + 3];
    if (r0 != (int32_t)t * kTileM || n != std::min<int32_t>(kTileM, Tt - r0)) p.btiles_uniform = false;
  }
  std::vector<int32_t> bwd_tiles128 = bwd_tiles_of(kBlockM);

  // Adapters owning training rows, and single-adapter chunks of the compact
  // rows for the deterministic reductions over tokens.
  std::vector<int32_t> ad_slot(n_ad, -1), train_ads;
  for (int32_t a : train_adapter) ad_slot[a] = 1;
  for (int32_t a = 0; a < n_ad; ++a)
    if (ad_slot[a] == 1) {
      ad_slot[a] = (int32_t)train_ads.size();
      train_ads.push_back(a);
    }
  std::vector<int32_t> chunks;
  for (const Run& r : runs_of(train_adapter.data(), 0, Tt))
    for (int32_t b = r.lo; b < r.hi; b += kChunkRows)
      chunks.insert(chunks.end(), {r.adapter, b, std::min(kChunkRows, r.hi - b), ad_slot[r.adapter]});
  const int32_t n_chunks = (int32_t)chunks.size() / kItemWords;
  // Items of <= kItemRows compact rows of one adapter (the g contraction).
  std::vector<int32_t> train_items;
  for (const Run& r : runs_of(train_adapter.data(), 0, Tt))
    for (int32_t b = r.lo; b < r.hi; b += kItemRows)
      train_items.insert(train_items.end(), {r.adapter, b, std::min(kItemRows, r.hi - b), 0});
  const int32_t n_tads = (int32_t)train_ads.size();
  p.r_used = p.r_train = 0;
  for (int32_t t = 0; t < T; ++t) p.r_used = std::max(p.r_used, p.ranks[row_adapter[t]]);
  for (int32_t a : train_ads) p.r_train = std::max(p.r_train, p.ranks[a]);
  std::vector<int32_t> tad_ptr(n_tads + 1, 0), tad_chunks;
  p.tad_max_chunks.assign(n_tads, 0);
  for (int32_t s = 0; s < n_tads; ++s) {
    for (int32_t c = 0; c < n_chunks; ++c)
      if (chunks[c * kItemWords + 3] == s) tad_chunks.push_back(c);
    tad_ptr[s + 1] = (int32_t)tad_chunks.size();
    p.tad_max_chunks[s] = tad_ptr[s + 1] - tad_ptr[s];
  }

  // Pack.  Each array starts on a 64-word (256-byte) boundary.
  std::vector<int32_t>& m = p.meta;
  m.clear();
  auto put = [&](const int32_t* src, size_t n) -> int64_t {
    m.resize((m.size() + 63) & ~size_t(63), 0);
    int64_t off = (int64_t)m.size();
    m.insert(m.end(), src, src + n);
    return off;
  };
  std::vector<int32_t> scale_bits(n_ad);
  std::memcpy(scale_bits.data(), scale, sizeof(float) * n_ad);
  dsv::MetaLayout& L = p.lay;
  L.row_adapter = put(row_adapter.data(), T);
  L.row_train = put(row_train.data(), T);
  L.train_rows = put(train_rows.data(), Tt);
  L.train_adapter = put(train_adapter.data(), Tt);
  L.shrink_rows = put(shrink_rows.data(), T);
  L.shrink_items = put(shrink_items.data(), shrink_items.size());
  L.gslot = put(gslot.data(), T);
  L.gather_rows = put(gather_rows.data(), gather_rows.size());
  L.gather_items = put(gather_items.data(), gather_items.size());
  L.fwd_tiles = put(fwd_tiles.data(), fwd_tiles.size());
  L.fwd_tiles128 = put(fwd_tiles128.data(), fwd_tiles128.size());
  L.bwd_tiles = put(bwd_tiles.data(), bwd_tiles.size());
  L.bwd_tiles128 = put(bwd_tiles128.data(), bwd_tiles128.size());
  L.chunks = put(chunks.data(), chunks.size());
  L.train_items = put(train_items.data(), train_items.size());
  L.train_ads = put(train_ads.data(), train_ads.size());
  L.ad_slot = put(ad_slot.data(), ad_slot.size());
  L.tad_chunk_ptr = put(tad_ptr.data(), tad_ptr.size());
  L.tad_chunks = put(tad_chunks.data(), tad_chunks.size());
  L.ranks = put(rank, n_ad);
  L.scales = put(scale_bits.data(), n_ad);
  m.resize((m.size() + 63) & ~size_t(63), 0);
  L.total_words = (int64_t)m.size();

  p.n_ftiles = (int32_t)(fwd_tiles.size() / kTileWords);
  p.n_shrink = (int32_t)(shrink_items.size() / kItemWords);
  p.n_gather = (int32_t)gather_rows.size();
  p.n_gitems = (int32_t)(gather_items.size() / kItemWords);
  p.n_btiles = (int32_t)(bwd_tiles.size() / kTileWords);
  p.n_ftiles128 = (int32_t)(fwd_tiles128.size() / kTileWords);
  p.n_btiles128 = (int32_t)(bwd_tiles128.size() / kTileWords);
  p.n_chunks = n_chunks;
  p.n_tads = n_tads;
  p.n_titems = (int32_t)(train_items.size() / kItemWords);
  return DSV_OK;
}

}  // namespace

extern "C" int dsv_segments_build(const dsv_segment* segs, int32_t n_segs, int32_t n_tokens,
                                  const int32_t* adapter_rank, const float* adapter_scale,
                                  int32_t n_adapters, int32_t r_max, void* d_meta,
                                  size_t* meta_bytes, void* hip_stream, dsv_plan** out_plan) {
  if (out_plan) *out_plan = nullptr;
  if (!meta_bytes) return DSV_ERR_ARG;
  dsv_plan* p = nullptr;
  try {
    p = new dsv_plan();
    int rc = build(segs, n_segs, n_tokens, adapter_rank, adapter_scale, n_adapters, r_max, *p);
    if (rc != DSV_OK) {
      delete p;
      return rc;
    }
  } catch (const std::bad_alloc&) {
    delete p;
    return DSV_ERR_SIZE;
  } catch (...) {
    delete p;
    return DSV_ERR_ARG;
  }
  const size_t need = (size_t)p->lay.total_words * sizeof(int32_t);
  if (d_meta) {
    if (reinterpret_cast<uintptr_t>(d_meta) % 256 != 0) {
      delete p;
      return DSV_ERR_ARG;
    }
    if (*meta_bytes < need) {
      *meta_bytes = need;
      delete p;
      return DSV_ERR_SIZE;
    }
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    hipEvent_t ev = nullptr;
    hipError_t e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e == hipSuccess)
      e = hipMemcpyAsync(d_meta, p->meta.data(), need, hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = hipEventRecord(ev, st);
    if (e != hipSuccess) {
      if (ev) (void)hipEventDestroy(ev);
      delete p;
      return DSV_ERR_DEVICE;
    }
    p->copy_done = ev;
    p->d_meta = d_meta;
  }
  *meta_bytes = need;
  if (out_plan)
    *out_plan = p;
  else
    delete p;
  return DSV_OK;
}

extern "C" int32_t dsv_plan_train_rows(const dsv_plan* p) { return p ? p->T_t : -1; }

extern "C" int32_t dsv_plan_train_row_index(const dsv_plan* p, int32_t* host_out) {
  if (!p || (!host_out && p->T_t > 0)) return DSV_ERR_ARG;
  if (p->T_t > 0) std::memcpy(host_out, p->train_rows.data(), sizeof(int32_t) * p->T_t);
  return p->T_t;
}

extern "C" int32_t dsv_plan_gathered_rows(const dsv_plan* p, int32_t* host_out) {
  if (!p || (!host_out && p->n_gather > 0)) return DSV_ERR_ARG;
  if (p->n_gather > 0)
    std::memcpy(host_out, p->gather_rows.data(), sizeof(int32_t) * p->n_gather);
  return p->n_gather;
}

extern "C" int dsv_plan_meta_copy(const dsv_plan* p, void* host_out, size_t bytes) {
  if (!p || !host_out) return DSV_ERR_ARG;
  const size_t need = p->meta.size() * sizeof(int32_t);
  if (bytes < need) return DSV_ERR_SIZE;
  std::memcpy(host_out, p->meta.data(), need);
  return DSV_OK;
}

extern "C" int dsv_plan_counts(const dsv_plan* p, int32_t out[10]) {
  if (!p || !out) return DSV_ERR_ARG;
  out[0] = p->n_ftiles;
  out[1] = p->n_shrink;
  out[2] = p->n_gather;
  out[3] = p->n_gitems;
  out[4] = p->n_btiles;
  out[5] = p->n_chunks;
  out[6] = p->n_tads;
  out[7] = p->n_titems;
  out[8] = p->n_ftiles128;
  out[9] = p->n_btiles128;
  return DSV_OK;
}

extern "C" void dsv_plan_free(dsv_plan* p) {
  if (!p) return;
  if (p->copy_done) {
    // the host image is the source of the asynchronous upload: wait for it
    hipEvent_t ev = static_cast<hipEvent_t>(p->copy_done);
    (void)hipEventSynchronize(ev);
    (void)hipEventDestroy(ev);
  }
  delete p;
}

extern "C" const char* dsv_status_string(int s) {
  switch (s) {
    case DSV_OK: return "DSV_OK";
    case DSV_ERR_ARG: return "DSV_ERR_ARG: null or misaligned pointer, bad count, or plan not on device";
    case DSV_ERR_RANGE: return "DSV_ERR_RANGE: adapter id, rank, r_max, scale or flag out of range";
    case DSV_ERR_LAYOUT: return "DSV_ERR_LAYOUT: segments do not tile [0, n_tokens) exactly";
    case DSV_ERR_SIZE: return "DSV_ERR_SIZE: buffer too small or unsupported shape";
    case DSV_ERR_DEVICE: return "DSV_ERR_DEVICE: a HIP call or kernel launch failed";
    default: return "unknown dsv status";
  }
}
