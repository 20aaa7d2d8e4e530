// api.cpp -- the C entry points: argument checks on the host, workspace
// carving, and the launch sequence of the forward and backward passes.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>

#include "kernels.h"
#include "plan.h"

namespace {

using namespace dsv;

constexpr int64_t kMaxDim = 1 << 20;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }
int64_t ld_rank(int32_t r_max) { return (r_max + 7) & ~7; }  // 16-byte rows of rank entries

// Compute units of the current device (0 if the query fails).
int device_cus() {
  static int cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
  if (dev < 64 && cached[dev] > 0) return cached[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (dev < 64) cached[dev] = n;
  return n;
}

// GEMM launch plan: tile shape and work split.  Candidates, costed in
// CU-time (one 128 x 128 x C tile on one CU = 1):
//   128 x 128, two workgroups per CU, whole tiles in whole waves of 2 * CUs;
//   256 x 256 (4 units, at a relative matrix-core efficiency kEff256), one
//     workgroup per CU, whole tiles in whole waves of CUs;
//   the same with the r tiles of a last, partial wave split into
//     s = CUs / r equal K ranges (one workgroup per piece, at least
//     kMinSkIters K-steps each), so that wave takes 1/s of a tile's time,
//     plus kSplitCost64 for the pieces' fp32 partials and the kernel that sums
//     them (relative to a tile of 64 K-steps, so smaller for longer tiles).
// The constants were fitted to timings of the Llama-3-8B projections
// (forward and dX) on MI355X.
struct GemmPlan {
  int tm = 128, tn = 128;
  int32_t n_mtiles = 0, n_ntiles = 0;
  int32_t dp_tiles = 0, sk_tiles = 0, sk_split = 0;
};
constexpr int kMinSkIters = 8;
constexpr double kEff256 = 1.12;
constexpr double kSplitCost64 = 0.4;

GemmPlan plan_gemm(int32_t m256, int32_t m128, int32_t n_out, int32_t C, bool allow_split = true) {
  GemmPlan best;
  best.n_mtiles = m128;
  best.n_ntiles = (n_out + 127) / 128;
  best.dp_tiles = best.n_mtiles * best.n_ntiles;
  const int cus = device_cus();
  if (cus <= 0) return best;
  const int64_t t128 = (int64_t)m128 * best.n_ntiles;
  const double cost128 = (double)((t128 + 2 * cus - 1) / (2 * cus)) * 2.0;

  const int64_t n256 = (n_out + 255) / 256, t256 = (int64_t)m256 * n256;
  const int64_t nk = (C + 63) / 64;
  if (t256 <= 0) return best;
  GemmPlan p;
  p.tm = p.tn = 256;
  p.n_mtiles = m256;
  p.n_ntiles = (int32_t)n256;
  p.dp_tiles = (int32_t)t256;
  const int64_t full = t256 / cus, r = t256 % cus;
  double cost256 = (double)(full + (r > 0)) * 4.0 / kEff256;
  const int64_t split = r > 0 ? std::min<int64_t>(cus / r, nk / kMinSkIters) : 0;
  if (allow_split && split >= 2 && ((full * cus) & 7) == 0) {
    const double cost_split =
        ((double)full + 1.0 / (double)split) * 4.0 / kEff256 + kSplitCost64 * 64.0 / (double)nk;
    if (cost_split < cost256) {
      cost256 = cost_split;
      p.dp_tiles = (int32_t)(full * cus);
      p.sk_tiles = (int32_t)r;
      p.sk_split = (int32_t)split;
    }
  }
  return cost256 < cost128 ? p : best;
}

struct FwdWs {
  size_t h_all, delta, keep, sk_part, rk_part, total;
};
struct BwdWs {
  size_t g, hrec, part_b, part_a, keep, sk_part, g_part, h_part, total;
};

// Dropout bitmask of the training rows: ceil(K / 32) words per row.
size_t keep_bytes(const dsv_plan& p, int32_t K) { return (size_t)p.T_t * ((K + 31) / 32) * 4; }

// Split-tile scratch of a GEMM plan: one fp32 partial tile per piece.
size_t carve_sk(const GemmPlan& gp, size_t off, size_t* part) {
  *part = off;
  if (gp.sk_tiles <= 0) return off;
  return align256(off + (size_t)gp.sk_tiles * gp.sk_split * gp.tm * gp.tn * 4);
}

FwdWs fwd_ws(const dsv_plan& p, dsv_dtype dt, int32_t K, int32_t N, const GemmPlan& gp) {
  FwdWs w{};
  size_t off = 0;
  if (dt == DSV_BF16) {
    w.h_all = off;
    off = align256(off + (size_t)p.T * ld_rank(p.r_max) * 2);
    w.delta = off;
    off = align256(off + (size_t)p.n_gather * N * 4);
    off = carve_sk(gp, off, &w.sk_part);
    w.rk_part = off;  // pieces of a split shrink
    off = align256(off + skinny_part_bytes(K, p.n_shrink, p.T, p.r_max));
  } else {
    w.h_all = off;
    off = align256(off + (size_t)p.T * p.r_max * 4);
    w.delta = off;
  }
  w.keep = off;  // dropout mask of the training rows
  off = align256(off + keep_bytes(p, K));
  w.total = off;
  return w;
}

BwdWs bwd_ws(const dsv_plan& p, dsv_dtype dt, int32_t K, int32_t N, const GemmPlan& gp) {
  BwdWs w{};
  size_t off = 0;
  if (dt == DSV_BF16) {
    w.g = off;
    off = align256(off + (size_t)p.T_t * ld_rank(p.r_max) * 2);
    w.hrec = off;  // h of the training rows, recomputed when H_save is not kept
    off = align256(off + (size_t)p.T_t * ld_rank(p.r_max) * 2);
    w.part_b = off;
    off = align256(off + (size_t)p.n_chunks * N * p.r_max * 4);
    w.part_a = off;
    off = align256(off + (size_t)p.n_chunks * K * p.r_max * 4);
    off = carve_sk(gp, off, &w.sk_part);
    w.g_part = off;  // g's partials, one per 256-column block of N
    off = align256(off + (size_t)token_col_blocks(N) * p.T_t * p.r_max * 4);
    w.h_part = off;  // pieces of a split recomputed h
    off = align256(off + skinny_part_bytes(K, p.n_shrink, p.T_t, p.r_max));
  } else {
    w.g = off;
    off = align256(off + (size_t)p.T_t * p.r_max * 4);
    w.hrec = off;
    off = align256(off + (size_t)p.T_t * p.r_max * 4);
  }
  w.keep = off;  // dropout mask of the training rows
  off = align256(off + keep_bytes(p, K));
  w.total = off;
  return w;
}

GemmPlan fwd_gemm_plan(const dsv_plan& p, dsv_dtype dt, int32_t K, int32_t N, bool allow_split = true) {
  if (dt != DSV_BF16 || p.T == 0) return GemmPlan{};
  return plan_gemm(p.n_ftiles, p.n_ftiles128, N, K, allow_split);
}
GemmPlan bwd_gemm_plan(const dsv_plan& p, dsv_dtype dt, int32_t K, int32_t N) {
  if (dt != DSV_BF16 || p.T_t == 0) return GemmPlan{};
  return plan_gemm(p.n_btiles, p.n_btiles128, K, N);
}

int check_common(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N) {
  if (!p) return DSV_ERR_ARG;
  if (dt != DSV_BF16 && dt != DSV_F32) return DSV_ERR_RANGE;
  if (K <= 0 || N <= 0 || (K & 7) || (N & 7) || K > kMaxDim || N > kMaxDim) return DSV_ERR_SIZE;
  return DSV_OK;
}

int ptr_ok(const void* p) { return p && aligned16(p); }

// Row strides (elements) of one projection's caller buffers: X [T][x],
// W [N][w], Y [T][y], dY [T_t][dy], dX [T_t][dx], Wt [K][wt].
struct Strides {
  int64_t x, w, y, dy, dx, wt;
};
Strides dense_strides(int32_t K, int32_t N) { return Strides{K, K, N, N, K, N}; }
// A caller's stride: 0 is the dense row length; any other value must hold a
// row (>= len), keep rows 16-byte aligned (a multiple of 8 elements) and
// stay within the kernels' 32-bit panel offsets (<= kMaxDim).
int row_stride(int32_t given, int32_t len, int64_t* out) {
  if (given == 0) {
    *out = len;
    return DSV_OK;
  }
  if (given < len || (given & 7) || given > kMaxDim) return DSV_ERR_SIZE;
  *out = given;
  return DSV_OK;
}
int fwd_strides(const dsv_fwd_proj& q, Strides* st) {
  *st = dense_strides(q.K, q.N);
  int rc = row_stride(q.ldx, q.K, &st->x);
  if (rc == DSV_OK) rc = row_stride(q.ldw, q.K, &st->w);
  if (rc == DSV_OK) rc = row_stride(q.ldy, q.N, &st->y);
  return rc;
}
int bwd_strides(const dsv_bwd_proj& q, Strides* st) {
  *st = dense_strides(q.K, q.N);
  int rc = row_stride(q.ldx, q.K, &st->x);
  if (rc == DSV_OK) rc = row_stride(q.ldw, q.K, &st->w);
  if (rc == DSV_OK) rc = row_stride(q.lddy, q.N, &st->dy);
  if (rc == DSV_OK) rc = row_stride(q.lddx, q.K, &st->dx);
  if (rc == DSV_OK) rc = row_stride(q.ldwt, q.N, &st->wt);
  return rc;
}

template <typename T>
T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}

void set_split(GemmArgs& g, const GemmPlan& gp, void* ws, size_t part_off) {
  g.n_mtiles = gp.n_mtiles;
  g.n_ntiles = gp.n_ntiles;
  g.dp_tiles = gp.dp_tiles;
  g.sk_tiles = gp.sk_tiles;
  g.sk_split = gp.sk_split;
  g.sk_part = gp.sk_tiles > 0 ? at<float>(ws, part_off) : nullptr;
}

// Benchmark timing of the GEMM launches (dsv_timing_enable / dsv_timing_read).
struct Timing {
  static constexpr int kMaxPairs = 4096;
  bool on = false;
  int n = 0;
  hipEvent_t ev[kMaxPairs][2] = {};
  int kind[kMaxPairs] = {};  // 0 forward GEMM, 1 dX GEMM
};
Timing g_timing;

// Hands the events of a timed launch to the next GEMM launch (they are
// recorded within its kernels' dispatches); returns the pair index or -1.
int timing_begin(int kind, hipStream_t s) {
  (void)s;
  Timing& t = g_timing;
  if (!t.on || t.n >= Timing::kMaxPairs) return -1;
  const int i = t.n;
  for (int k = 0; k < 2; ++k)
    if (!t.ev[i][k] && hipEventCreate(&t.ev[i][k]) != hipSuccess) return -1;
  set_launch_events(t.ev[i][0], t.ev[i][1]);
  t.kind[i] = kind;
  t.n = i + 1;
  return i;
}

// A pair whose launch launched nothing (or failed before its last kernel) is
// dropped: its events were never recorded.
void timing_end(int i, hipStream_t s) {
  (void)s;
  if (i < 0 || !launch_events_pending()) return;
  set_launch_events(nullptr, nullptr);
  if (i == g_timing.n - 1) g_timing.n = i;
}

}  // namespace

extern "C" int dsv_timing_enable(int32_t on) {
  g_timing.on = on != 0;
  return DSV_OK;
}

extern "C" int dsv_timing_read(double* fwd_ms, int32_t* fwd_n, double* bwd_ms, int32_t* bwd_n) {
  double ms[2] = {0.0, 0.0};
  int32_t cnt[2] = {0, 0};
  int rc = DSV_OK;
  for (int i = 0; i < g_timing.n; ++i) {
    float e = 0.f;
    if (hipEventSynchronize(g_timing.ev[i][1]) != hipSuccess ||
        hipEventElapsedTime(&e, g_timing.ev[i][0], g_timing.ev[i][1]) != hipSuccess) {
      rc = DSV_ERR_DEVICE;
      continue;
    }
    ms[g_timing.kind[i]] += e;
    cnt[g_timing.kind[i]] += 1;
  }
  g_timing.n = 0;
  if (fwd_ms) *fwd_ms = ms[0];
  if (fwd_n) *fwd_n = cnt[0];
  if (bwd_ms) *bwd_ms = ms[1];
  if (bwd_n) *bwd_n = cnt[1];
  return rc;
}

namespace {

// AdamW of up to DSV_MAX_GROUP projections in one launch (dsv_adamw_step is a
// group of one): validation first, nothing launched on any error.
int adamw_impl(const dsv_plan* p, dsv_dtype dt, int32_t n, const dsv_adamw_proj* projs, int32_t step,
               const dsv_adamw_hparams* hp, hipStream_t stream) {
  if (!p) return DSV_ERR_ARG;
  if (n < 1 || n > DSV_MAX_GROUP) return DSV_ERR_RANGE;
  if (!projs) return DSV_ERR_ARG;
  for (int32_t i = 0; i < n; ++i) {
    const int rc = check_common(p, dt, projs[i].K, projs[i].N);
    if (rc != DSV_OK) return rc;
  }
  if (!p->d_meta || !hp) return DSV_ERR_ARG;
  if (step < 1 || !std::isfinite(hp->lr) || hp->lr < 0.0 || !std::isfinite(hp->weight_decay) ||
      hp->weight_decay < 0.0 || !(hp->beta1 >= 0.0 && hp->beta1 < 1.0) ||
      !(hp->beta2 >= 0.0 && hp->beta2 < 1.0) || !(hp->eps > 0.0) || !std::isfinite(hp->eps))
    return DSV_ERR_RANGE;
  for (int32_t i = 0; i < n; ++i) {
    const dsv_adamw_proj& q = projs[i];
    if (!ptr_ok(q.dA) || !ptr_ok(q.dB) || !ptr_ok(q.A_master) || !ptr_ok(q.B_master) || !ptr_ok(q.A_m) ||
        !ptr_ok(q.A_v) || !ptr_ok(q.B_m) || !ptr_ok(q.B_v) || (q.A && !aligned16(q.A)) ||
        (q.B && !aligned16(q.B)))
      return DSV_ERR_ARG;
  }
  if (p->n_tads == 0) return DSV_OK;
  AdamWArgs a{};
  a.r_max = p->r_max;
  a.n_proj = n;
  a.bf16 = dt == DSV_BF16;
  a.train_ads = p->dptr(p->lay.train_ads);
  a.ranks = p->dptr(p->lay.ranks);
  // B in float4 units when every training rank and the rank stride are multiples of 4
  bool bvec = (p->r_max & 3) == 0;
  for (int32_t s = 0; s < p->n_tads; ++s) bvec = bvec && (p->ranks[p->meta[p->lay.train_ads + s]] & 3) == 0;
  a.bvec = bvec ? 1 : 0;
  // factors formed in double on the host, rounded once to fp32
  const double bc1 = 1.0 - std::pow(hp->beta1, (double)step);
  const double bc2 = 1.0 - std::pow(hp->beta2, (double)step);
  a.decay = (float)(1.0 - hp->lr * hp->weight_decay);
  a.b1 = (float)hp->beta1;
  a.b2 = (float)hp->beta2;
  a.c1 = (float)(1.0 - hp->beta1);
  a.c2 = (float)(1.0 - hp->beta2);
  a.eps = (float)hp->eps;
  a.step_size = (float)(hp->lr / bc1);
  a.sqrt_bc2 = (float)std::sqrt(bc2);
  int64_t blocks = 0;
  for (int32_t i = 0; i < n; ++i) {
    const dsv_adamw_proj& q = projs[i];
    // units of the largest training rank; smaller ranks leave threads idle
    const int64_t r = p->r_train;
    const int64_t units = r * q.K / 4 + (bvec ? (int64_t)q.N * r / 4 : (int64_t)q.N * r);
    const int64_t bpa = (units + 255) / 256;
    if (bpa * 256 > INT32_MAX) return DSV_ERR_SIZE;  // the kernel indexes units in 32 bits
    AdamWProj& d = a.proj[i];
    d.K = q.K;
    d.N = q.N;
    d.blk_begin = (int32_t)blocks;
    d.bpa = (int32_t)bpa;
    d.dA = q.dA;
    d.dB = q.dB;
    d.pA = q.A_master;
    d.pB = q.B_master;
    d.mA = q.A_m;
    d.vA = q.A_v;
    d.mB = q.B_m;
    d.vB = q.B_v;
    d.A = q.A;
    d.B = q.B;
    blocks += bpa * p->n_tads;
    if (blocks > INT32_MAX) return DSV_ERR_SIZE;
  }
  return launch_adamw(a, blocks, stream) == hipSuccess ? DSV_OK : DSV_ERR_DEVICE;
}

}  // namespace

extern "C" int dsv_adamw_step(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N, int32_t step,
                              const dsv_adamw_hparams* hp, const float* dA, const float* dB, float* A_master,
                              float* B_master, float* A_m, float* A_v, float* B_m, float* B_v, void* A,
                              void* B, void* hip_stream) {
  const dsv_adamw_proj one{K, N, dA, dB, A_master, B_master, A_m, A_v, B_m, B_v, A, B};
  return adamw_impl(p, dt, 1, &one, step, hp, static_cast<hipStream_t>(hip_stream));
}

extern "C" int dsv_adamw_step_grouped(const dsv_plan* p, dsv_dtype dt, int32_t n_proj,
                                      const dsv_adamw_proj* projs, int32_t step, const dsv_adamw_hparams* hp,
                                      void* hip_stream) {
  return adamw_impl(p, dt, n_proj, projs, step, hp, static_cast<hipStream_t>(hip_stream));
}

extern "C" int dsv_gemm_config(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N, int32_t pass,
                               int32_t out[6]) {
  int rc = check_common(p, dt, K, N);
  if (rc != DSV_OK) return rc;
  if (!out || (pass != 0 && pass != 1)) return DSV_ERR_ARG;
  for (int i = 0; i < 6; ++i) out[i] = 0;
  if (dt != DSV_BF16 || (pass == 0 ? p->T : p->T_t) == 0) return DSV_OK;
  const GemmPlan gp = pass == 0 ? fwd_gemm_plan(*p, dt, K, N) : bwd_gemm_plan(*p, dt, K, N);
  out[0] = gp.tm;
  out[1] = gp.tn;
  out[2] = gp.n_mtiles;
  out[3] = gp.n_ntiles;
  out[4] = gp.sk_tiles;
  out[5] = gp.sk_split;
  return DSV_OK;
}

extern "C" int dsv_cobatch_fwd_workspace(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N,
                                         size_t* bytes) {
  int rc = check_common(p, dt, K, N);
  if (rc != DSV_OK) return rc;
  if (!bytes) return DSV_ERR_ARG;
  *bytes = fwd_ws(*p, dt, K, N, fwd_gemm_plan(*p, dt, K, N)).total;
  return DSV_OK;
}

extern "C" int dsv_lora_bwd_workspace(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N,
                                      size_t* bytes) {
  int rc = check_common(p, dt, K, N);
  if (rc != DSV_OK) return rc;
  if (!bytes) return DSV_ERR_ARG;
  *bytes = bwd_ws(*p, dt, K, N, bwd_gemm_plan(*p, dt, K, N)).total;
  return DSV_OK;
}

extern "C" int dsv_lora_bwd_dropout_workspace(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N,
                                              size_t* bytes) {
  int rc = check_common(p, dt, K, N);
  if (rc != DSV_OK) return rc;
  if (!bytes) return DSV_ERR_ARG;
  *bytes = bwd_ws(*p, dt, K, N, bwd_gemm_plan(*p, dt, K, N)).total;
  return DSV_OK;
}

namespace {

// Dropout parameters -> mask spec; false when they are out of range.
bool dropout_spec(const dsv_dropout* d, DropoutSpec* out) {
  if (!d || !std::isfinite(d->p) || d->p < 0.0 || d->p >= 1.0) return false;
  const double t = std::floor(d->p * 4294967296.0);
  out->thr = t >= 4294967295.0 ? 0xFFFFFFFFu : (uint32_t)t;
  out->scale = (float)(1.0 / (1.0 - d->p));
  out->seed = d->seed;
  out->offset = d->offset;
  return true;
}

// The caller's mask buffer must hold 32-bit words.
bool mask_aligned(const dsv_dropout* d) { return !d || !d->mask || (reinterpret_cast<uintptr_t>(d->mask) & 3) == 0; }

// Where a projection's mask lives: the caller's buffer, else the workspace.
uint32_t* mask_buffer(const dsv_dropout* d, void* ws_keep) {
  return d && d->mask ? d->mask : static_cast<uint32_t*>(ws_keep);
}

// noalloc: the allocation-free form (dsv_cobatch_fwd_noalloc): the workspace is
// the library's device scratch, the GEMM plan splits no tile along the
// contraction (a split needs a partial tile per piece, tens of MB), and no
// benchmark timing events are created.
int fwd_impl(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N, const void* X, const void* W, const void* A,
             const void* B, void* Y, void* H_save, const dsv_dropout* drop, void* workspace,
             size_t workspace_bytes, void* hip_stream, const Strides* lds = nullptr, bool noalloc = false) {
  int rc = check_common(p, dt, K, N);
  if (rc != DSV_OK) return rc;
  const Strides ld = lds ? *lds : dense_strides(K, N);
  DropoutSpec ds{};
  if (drop && !dropout_spec(drop, &ds)) return DSV_ERR_RANGE;
  if (!mask_aligned(drop)) return DSV_ERR_ARG;
  const bool dropping = drop && drop->p > 0.0 && p->T_t > 0;
  if (!p->d_meta) return DSV_ERR_ARG;
  if (p->T == 0) return DSV_OK;  // empty batch: nothing to read or write
  if (!ptr_ok(X) || !ptr_ok(W) || !ptr_ok(A) || !ptr_ok(B) || !ptr_ok(Y)) return DSV_ERR_ARG;
  if (H_save && !aligned16(H_save)) return DSV_ERR_ARG;
  const GemmPlan gp = fwd_gemm_plan(*p, dt, K, N, !noalloc);
  const FwdWs ws = fwd_ws(*p, dt, K, N, gp);
  if (ws.total > 0) {
    if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255)) return DSV_ERR_ARG;
    if (workspace_bytes < ws.total) return DSV_ERR_SIZE;
  }
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const MetaLayout& L = p->lay;
  const int32_t* ranks = p->dptr(L.ranks);
  const float* scales = reinterpret_cast<const float*>(p->dptr(L.scales));
  hipError_t e = hipSuccess;

  // 0. dropout mask of the training rows' adapter input (into the caller's
  //    buffer when one is given, for the backward to read).
  uint32_t* keep_w = dropping ? mask_buffer(drop, at<uint32_t>(workspace, ws.keep)) : nullptr;
  const uint32_t* keep = keep_w;
  const int32_t keep_words = (K + 31) / 32;
  if (dropping && (e = launch_dropout_mask(keep_w, p->T_t, K, ds, s)) != hipSuccess) return DSV_ERR_DEVICE;

  if (dt == DSV_F32) {
    F32Args a{};
    a.T = p->T;
    a.Tt = p->T_t;
    a.K = K;
    a.N = N;
    a.r_max = p->r_max;
    a.keep = keep;
    a.keep_words = keep_words;
    a.drop_scale = ds.scale;
    a.row_adapter = p->dptr(L.row_adapter);
    a.row_train = p->dptr(L.row_train);
    a.ranks = ranks;
    a.scales = scales;
    a.X = static_cast<const float*>(X);
    a.W = static_cast<const float*>(W);
    a.A = static_cast<const float*>(A);
    a.B = static_cast<const float*>(B);
    a.Y = static_cast<float*>(Y);
    a.ldx = ld.x;
    a.ldw = ld.w;
    a.ldy = ld.y;
    a.Hsave = p->T_t > 0 ? static_cast<float*>(H_save) : nullptr;
    a.Hall = at<float>(workspace, ws.h_all);
    e = launch_f32_fwd(a, s);
    return e == hipSuccess ? DSV_OK : DSV_ERR_DEVICE;
  }

  const int64_t ldh = ld_rank(p->r_max);
  uint16_t* h_all = at<uint16_t>(workspace, ws.h_all);
  float* delta = p->n_gather > 0 ? at<float>(workspace, ws.delta) : nullptr;

  // 1. shrink: h of every row, grouped by adapter.
  SkinnyArgs sk{};
  sk.P = static_cast<const uint16_t*>(X);
  sk.ldp = ld.x;
  sk.rows = p->dptr(L.shrink_rows);
  sk.items = p->dptr(L.shrink_items);
  sk.Q = static_cast<const uint16_t*>(A);
  sk.q_ad = (int64_t)p->r_max * K;
  sk.ldq = K;
  sk.qsel = nullptr;
  sk.ranks = ranks;
  sk.scales = nullptr;
  sk.C = K;
  sk.out1 = h_all;
  sk.ld1 = ldh;
  sk.out2 = p->T_t > 0 ? static_cast<uint16_t*>(H_save) : nullptr;
  sk.ld2 = p->r_max;
  sk.row_train = p->dptr(L.row_train);
  sk.keep = keep;
  sk.keep_words = keep_words;
  sk.drop_scale = ds.scale;
  sk.part = at<float>(workspace, ws.rk_part);
  sk.part_n = p->T;
  sk.r_max = p->r_max;
  sk.split_items = p->n_shrink;
  if ((e = launch_shrink(sk, p->n_shrink, p->r_used, s)) != hipSuccess) return DSV_ERR_DEVICE;

  // 2. gathered rows: fp32 low-rank term, each touched adapter read once.
  if (p->n_gather > 0) {
    e = launch_gather_expand(h_all, ldh, static_cast<const uint16_t*>(B), N, p->r_max,
                             p->dptr(L.gather_items), p->n_gitems, p->dptr(L.gather_rows), ranks,
                             scales, delta, s);
    if (e != hipSuccess) return DSV_ERR_DEVICE;
  }

  // 3. base GEMM with the low-rank prologue, one rounding.
  GemmArgs g{};
  g.P = static_cast<const uint16_t*>(X);
  g.ldp = ld.x;
  g.Q = static_cast<const uint16_t*>(W);
  g.ldq = ld.w;
  g.out = static_cast<uint16_t*>(Y);
  g.ldo = ld.y;
  g.M = p->T;
  g.Nout = N;
  g.C = K;
  g.tiles = p->dptr(gp.tm == 256 ? L.fwd_tiles : L.fwd_tiles128);
  g.uniform_rows = gp.tm == 256;
  set_split(g, gp, workspace, ws.sk_part);
  g.Lp = h_all;
  g.ldl = ldh;
  g.Lq = static_cast<const uint16_t*>(B);
  g.lq_ad = (int64_t)N * p->r_max;
  g.lq_j = 1;
  g.lq_col = p->r_max;
  g.ranks = ranks;
  g.scales = scales;
  g.delta = delta;
  g.gslot = p->dptr(L.gslot);
  const int tk = noalloc ? -1 : timing_begin(0, s);
  e = launch_gemm_nt(g, gp.tm, gp.tn, s);
  timing_end(tk, s);
  if (e != hipSuccess) return DSV_ERR_DEVICE;
  return DSV_OK;
}

// Wt (optional, bf16): the frozen weight transposed, [K][N]; the dX GEMM then
// reads it K-contiguous like the forward's W instead of transposing W on the fly.
// A second stream of the current device (default priority, non-blocking)
// and two events, created on first use: the grouped bf16 backward runs its
// dA reductions and final sums there, beside the dX GEMMs on the caller's
// stream, which need neither.  The fork and join are enqueued under a lock, so calls
// from several host threads do not interleave on the shared events; the side
// work of successive calls queues up on the one side stream.
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
std::mutex g_side_mu;
SideStream g_side[64];

// The current device's side stream (created if needed), or nullptr.
SideStream* side_stream() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  SideStream& sd = g_side[dev];
  if (!sd.s) {
    hipStream_t st = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (hipStreamCreateWithFlags(&st, hipStreamNonBlocking) != hipSuccess) return nullptr;
    if (hipEventCreateWithFlags(&e0, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&e1, hipEventDisableTiming) != hipSuccess) {
      if (e0) (void)hipEventDestroy(e0);
      (void)hipStreamDestroy(st);
      return nullptr;
    }
    sd.fork = e0;
    sd.join = e1;
    sd.s = st;
  }
  return &sd;
}

int bwd_impl(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N, const void* X, const void* W, const void* A,
             const void* B, const void* H_save, const void* dY, float* dA, float* dB, void* dX,
             int32_t accumulate, const dsv_dropout* drop, const void* Wt, void* workspace,
             size_t workspace_bytes, void* hip_stream, const Strides* lds = nullptr) {
  int rc = check_common(p, dt, K, N);
  if (rc != DSV_OK) return rc;
  const Strides ld = lds ? *lds : dense_strides(K, N);
  DropoutSpec ds{};
  if (drop && !dropout_spec(drop, &ds)) return DSV_ERR_RANGE;
  if (!mask_aligned(drop)) return DSV_ERR_ARG;
  const bool dropping = drop && drop->p > 0.0;
  if (accumulate != 0 && accumulate != 1) return DSV_ERR_RANGE;
  if (!p->d_meta) return DSV_ERR_ARG;
  if (p->T_t == 0) return DSV_OK;  // no training rows: nothing to read or write
  if (!ptr_ok(X) || !ptr_ok(W) || !ptr_ok(A) || !ptr_ok(B) || !ptr_ok(dA) || !ptr_ok(dB))
    return DSV_ERR_ARG;
  if (dX && !aligned16(dX)) return DSV_ERR_ARG;
  if (!ptr_ok(dY) || (H_save && !aligned16(H_save)) || (Wt && !aligned16(Wt))) return DSV_ERR_ARG;
  const GemmPlan gp = bwd_gemm_plan(*p, dt, K, N);
  const BwdWs ws = bwd_ws(*p, dt, K, N, gp);
  if (ws.total > 0) {
    if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255)) return DSV_ERR_ARG;
    if (workspace_bytes < ws.total) return DSV_ERR_SIZE;
  }
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const MetaLayout& L = p->lay;
  const int32_t* ranks = p->dptr(L.ranks);
  const float* scales = reinterpret_cast<const float*>(p->dptr(L.scales));
  hipError_t e = hipSuccess;

  // 0. the forward's dropout mask: the caller's buffer, or regenerated from
  //    the same seed and offset.
  uint32_t* keep = dropping ? mask_buffer(drop, at<uint32_t>(workspace, ws.keep)) : nullptr;
  const int32_t keep_words = (K + 31) / 32;
  if (dropping && !drop->mask && (e = launch_dropout_mask(keep, p->T_t, K, ds, s)) != hipSuccess)
    return DSV_ERR_DEVICE;

  if (dt == DSV_F32) {
    F32Args a{};
    a.T = p->T;
    a.Tt = p->T_t;
    a.K = K;
    a.N = N;
    a.r_max = p->r_max;
    a.keep = keep;
    a.keep_words = keep_words;
    a.drop_scale = ds.scale;
    a.train_rows = p->dptr(L.train_rows);
    a.train_adapter = p->dptr(L.train_adapter);
    a.train_ads = p->dptr(L.train_ads);
    a.n_tads = p->n_tads;
    a.tad_ptr = p->dptr(L.tad_chunk_ptr);
    a.tad_chunks = p->dptr(L.tad_chunks);
    a.chunks = p->dptr(L.chunks);
    a.ranks = ranks;
    a.scales = scales;
    a.X = static_cast<const float*>(X);
    a.W = static_cast<const float*>(W);
    a.A = static_cast<const float*>(A);
    a.B = static_cast<const float*>(B);
    a.Hs = static_cast<const float*>(H_save);
    a.Hrec = at<float>(workspace, ws.hrec);
    a.dY = static_cast<const float*>(dY);
    a.G = at<float>(workspace, ws.g);
    a.dA = dA;
    a.dB = dB;
    a.dX = static_cast<float*>(dX);
    a.ldx = ld.x;
    a.ldw = ld.w;
    a.lddy = ld.dy;
    a.lddx = ld.dx;
    a.accumulate = accumulate;
    e = launch_f32_bwd(a, s);
    return e == hipSuccess ? DSV_OK : DSV_ERR_DEVICE;
  }

  const int64_t ldh = ld_rank(p->r_max);
  uint16_t* gm = at<uint16_t>(workspace, ws.g);
  float* part_b = at<float>(workspace, ws.part_b);
  float* part_a = at<float>(workspace, ws.part_a);
  const int32_t* train_ads = p->dptr(L.train_ads);

  // 1. H_save not kept (residual-only retention): recompute h of the training
  //    rows from X with the forward's shrink (same values, bit for bit).
  const uint16_t* hs = static_cast<const uint16_t*>(H_save);
  int64_t ldhs = p->r_max;
  if (!hs) {
    uint16_t* hrec = at<uint16_t>(workspace, ws.hrec);
    SkinnyArgs sh{};
    sh.P = static_cast<const uint16_t*>(X);
    sh.ldp = ld.x;
    sh.rows = p->dptr(L.train_rows);
    sh.items = p->dptr(L.train_items);
    sh.Q = static_cast<const uint16_t*>(A);
    sh.q_ad = (int64_t)p->r_max * K;
    sh.ldq = K;
    sh.qsel = nullptr;
    sh.ranks = ranks;
    sh.scales = nullptr;
    sh.C = K;
    sh.out1 = nullptr;
    sh.out2 = hrec;
    sh.ld2 = ldh;
    sh.row_train = p->dptr(L.row_train);
    sh.keep = keep;
    sh.keep_words = keep_words;
    sh.drop_scale = ds.scale;
    sh.part = at<float>(workspace, ws.h_part);
    sh.part_n = p->T_t;
    sh.r_max = p->r_max;
    sh.split_items = p->n_shrink;  // the forward shrink's split: the same sums
    if ((e = launch_shrink_train(sh, p->n_titems, p->r_train, s)) != hipSuccess) return DSV_ERR_DEVICE;
    hs = hrec;
    ldhs = ldh;
  }

  // 2. per-chunk fp32 partials of dy^T h (-> dB); the same pass writes the
  //    per-column-block partials of dy B_a (-> g), reading dy once.
  TokenReduceGroup tb{};
  tb.n = 1;
  TokenReduceArgs& rb = tb.a[0];
  rb.P = static_cast<const uint16_t*>(dY);
  rb.ldp = ld.dy;
  rb.prow = nullptr;
  rb.Q = hs;
  rb.ldq = ldhs;
  rb.chunks = p->dptr(L.chunks);
  rb.ranks = ranks;
  rb.C = N;
  rb.r_max = p->r_max;
  rb.part = part_b;
  rb.B = static_cast<const uint16_t*>(B);
  rb.gpart = at<float>(workspace, ws.g_part);
  rb.gpart_n = p->T_t;
  tb.yoff[1] = token_col_blocks(N);
  if ((e = launch_token_reduce_group(tb, p->n_chunks, p->r_train, s)) != hipSuccess) return DSV_ERR_DEVICE;

  // 3. g = s_a dy B_a: the block partials summed in order, rounded once -> G [T_t][ldh]
  SkinnyGroup gf{};
  gf.n = 1;
  SkinnyArgs& sk = gf.a[0];
  sk.items = p->dptr(L.train_items);
  sk.ranks = ranks;
  sk.scales = scales;
  sk.out1 = gm;
  sk.ld1 = ldh;
  sk.part = rb.gpart;
  sk.part_n = p->T_t;
  sk.r_max = p->r_max;
  sk.pieces = token_col_blocks(N);
  if ((e = launch_g_finish_group(gf, p->n_titems, s)) != hipSuccess) return DSV_ERR_DEVICE;

  // 4. per-chunk fp32 partials of x^T g (-> dA)
  TokenReduceGroup ta{};
  ta.n = 1;
  TokenReduceArgs& ra = ta.a[0];
  ra.P = static_cast<const uint16_t*>(X);
  ra.ldp = ld.x;
  ra.prow = p->dptr(L.train_rows);
  ra.Q = gm;
  ra.ldq = ldh;
  ra.chunks = p->dptr(L.chunks);
  ra.ranks = ranks;
  ra.C = K;
  ra.r_max = p->r_max;
  ra.part = part_a;
  ra.keep = keep;  // dA contracts the masked input
  ra.keep_words = keep_words;
  ta.yoff[1] = token_col_blocks(K);

  // 5. fixed-order sums into dB (scaled by s_a) and dA.
  const int32_t* tad_ptr = p->dptr(L.tad_chunk_ptr);
  const int32_t* tad_chunks = p->dptr(L.tad_chunks);
  const ReduceOutArgs ob{part_b, N, scales, 0, dB, 1.f};
  const ReduceOutArgs oa{part_a, K, nullptr, 1, dA, dropping ? ds.scale : 1.f};
  auto dA_and_sums = [&](hipStream_t sx) -> int {
    if (launch_token_reduce_group(ta, p->n_chunks, p->r_train, sx) != hipSuccess) return DSV_ERR_DEVICE;
    if (launch_reduce_out(ob, oa, p->r_max, p->r_train, train_ads, p->n_tads, tad_ptr, tad_chunks, ranks, accumulate,
                          sx) != hipSuccess)
      return DSV_ERR_DEVICE;
    return DSV_OK;
  };
  if (!dX) return dA_and_sums(s);

  // 6. dx = dy W + g A_a on the matrix cores (W read with a transposing load).
  //    Under dropout g A_a passes through the input's mask (in the accumulators,
  //    between the low-rank prologue and the main loop).
  auto dx_gemm = [&](hipStream_t s) -> int {
    GemmArgs g{};
    g.P = static_cast<const uint16_t*>(dY);
    g.ldp = ld.dy;
    g.Q = static_cast<const uint16_t*>(Wt ? Wt : W);
    g.ldq = Wt ? ld.wt : ld.w;
    g.out = static_cast<uint16_t*>(dX);
    g.ldo = ld.dx;
    g.M = p->T_t;
    g.Nout = K;
    g.C = N;
    g.tiles = p->dptr(gp.tm == 256 ? L.bwd_tiles : L.bwd_tiles128);
    g.uniform_rows = gp.tm == 256 && p->btiles_uniform;
    set_split(g, gp, workspace, ws.sk_part);
    g.Lp = gm;
    g.ldl = ldh;
    g.Lq = static_cast<const uint16_t*>(A);
    g.lq_ad = (int64_t)p->r_max * K;
    g.lq_j = K;
    g.lq_col = 1;
    g.ranks = ranks;
    g.scales = nullptr;
    g.delta = nullptr;
    g.gslot = nullptr;
    g.keep = keep;
    g.keep_words = keep_words;
    g.keep_scale = ds.scale;
    const int tk = timing_begin(1, s);
    const hipError_t e = Wt ? launch_gemm_nt(g, gp.tm, gp.tn, s) : launch_gemm_nn(g, gp.tm, gp.tn, s);
    timing_end(tk, s);
    return e == hipSuccess ? DSV_OK : DSV_ERR_DEVICE;
  };
  // One projection's dA work is too small to pay for a fork to the side
  // stream (the grouped call forks): everything on the caller's stream.
  if ((rc = dA_and_sums(s)) != DSV_OK) return rc;
  return dx_gemm(s);
}

}  // namespace

extern "C" int dsv_cobatch_fwd(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N, const void* X,
                               const void* W, const void* A, const void* B, void* Y, void* H_save,
                               void* workspace, size_t workspace_bytes, void* hip_stream) {
  return fwd_impl(p, dt, K, N, X, W, A, B, Y, H_save, nullptr, workspace, workspace_bytes, hip_stream);
}

extern "C" int dsv_cobatch_fwd_noalloc(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N, const void* X,
                                       const void* W, const void* A, const void* B, void* Y, void* H_save,
                                       void* hip_stream) {
  // the device scratch replaces the workspace: its address on the current
  // device (looked up on the device's first call), never the array's name
  void* scratch = nullptr;
  if (noalloc_scratch(&scratch) != hipSuccess) return DSV_ERR_DEVICE;
  return fwd_impl(p, dt, K, N, X, W, A, B, Y, H_save, nullptr, scratch, kNoAllocScratchBytes, hip_stream,
                  /*lds=*/nullptr, /*noalloc=*/true);
}

extern "C" int dsv_cobatch_fwd_dropout(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N, const void* X,
                                       const void* W, const void* A, const void* B, void* Y, void* H_save,
                                       const dsv_dropout* dropout, void* workspace, size_t workspace_bytes,
                                       void* hip_stream) {
  if (!dropout) return DSV_ERR_ARG;
  return fwd_impl(p, dt, K, N, X, W, A, B, Y, H_save, dropout, workspace, workspace_bytes, hip_stream);
}

extern "C" int dsv_lora_bwd(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N, const void* X,
                            const void* W, const void* A, const void* B, const void* H_save,
                            const void* dY, float* dA, float* dB, void* dX, int32_t accumulate,
                            void* workspace, size_t workspace_bytes, void* hip_stream) {
  return bwd_impl(p, dt, K, N, X, W, A, B, H_save, dY, dA, dB, dX, accumulate, nullptr, nullptr, workspace,
                  workspace_bytes, hip_stream);
}

extern "C" int dsv_lora_bwd_dropout(const dsv_plan* p, dsv_dtype dt, int32_t K, int32_t N, const void* X,
                                    const void* W, const void* A, const void* B, const void* H_save,
                                    const void* dY, float* dA, float* dB, void* dX, int32_t accumulate,
                                    const dsv_dropout* dropout, void* workspace, size_t workspace_bytes,
                                    void* hip_stream) {
  if (!dropout) return DSV_ERR_ARG;
  return bwd_impl(p, dt, K, N, X, W, A, B, H_save, dY, dA, dB, dX, accumulate, dropout, nullptr, workspace,
                  workspace_bytes, hip_stream);
}

// ---------------------------------------------------------------------------
// Grouped launches: several projections of one batch (one plan) with one
// launch per step kind.  GEMMs take whole 256x256 tiles of every projection in
// one launch, longest contraction first, so the tail of one projection is
// filled by the tiles of the next instead of being split.
// ---------------------------------------------------------------------------
namespace {

static_assert(kMaxGroup == DSV_MAX_GROUP, "group size of the kernels and the interface");

GemmPlan whole256(int32_t m256, int32_t n_out) {
  GemmPlan g;
  g.tm = g.tn = 256;
  g.n_mtiles = m256;
  g.n_ntiles = (n_out + 255) / 256;
  g.dp_tiles = g.n_mtiles * g.n_ntiles;
  return g;
}

int check_group(const dsv_plan* p, dsv_dtype dt, int32_t n, const void* projs) {
  if (!p || !projs) return DSV_ERR_ARG;
  if (n < 1 || n > DSV_MAX_GROUP) return DSV_ERR_RANGE;
  if (dt != DSV_BF16 && dt != DSV_F32) return DSV_ERR_RANGE;
  return DSV_OK;
}

// Workspace of a grouped call: each projection's single-call regions (without
// split-tile partials for bf16), one after the other.
size_t fwd_group_ws(const dsv_plan& p, dsv_dtype dt, int32_t n, const dsv_fwd_proj* pr, size_t* base,
                    FwdWs* w) {
  size_t off = 0;
  for (int i = 0; i < n; ++i) {
    const GemmPlan gp = dt == DSV_BF16 ? whole256(p.n_ftiles, pr[i].N) : GemmPlan{};
    w[i] = fwd_ws(p, dt, pr[i].K, pr[i].N, gp);
    base[i] = off;
    off = align256(off + w[i].total);
  }
  return off;
}

size_t bwd_group_ws(const dsv_plan& p, dsv_dtype dt, int32_t n, const dsv_bwd_proj* pr, size_t* base,
                    BwdWs* w) {
  size_t off = 0;
  for (int i = 0; i < n; ++i) {
    const GemmPlan gp = dt == DSV_BF16 ? whole256(p.n_btiles, pr[i].K) : GemmPlan{};
    w[i] = bwd_ws(p, dt, pr[i].K, pr[i].N, gp);
    base[i] = off;
    off = align256(off + w[i].total);
  }
  return off;
}

// projections in launch order: longest contraction first (stable)
void by_contraction(int32_t n, const int32_t* C, int32_t* order) {
  for (int i = 0; i < n; ++i) order[i] = i;
  std::stable_sort(order, order + n, [&](int32_t a, int32_t b) { return C[a] > C[b]; });
}

}  // namespace

extern "C" int32_t dsv_row_stride(int32_t n, dsv_dtype dt) {
  if (n <= 0 || (dt != DSV_BF16 && dt != DSV_F32)) return 0;
  if (dt == DSV_BF16 && n > 8192 && ((int64_t)n * 2) % 4096 == 0) return n + 64;
  return n;
}

extern "C" int dsv_cobatch_fwd_grouped_workspace(const dsv_plan* p, dsv_dtype dt, int32_t n_proj,
                                                 const dsv_fwd_proj* projs, size_t* bytes) {
  int rc = check_group(p, dt, n_proj, projs);
  if (rc != DSV_OK) return rc;
  if (!bytes) return DSV_ERR_ARG;
  if (n_proj == 1) return dsv_cobatch_fwd_workspace(p, dt, projs[0].K, projs[0].N, bytes);
  for (int i = 0; i < n_proj; ++i)
    if ((rc = check_common(p, dt, projs[i].K, projs[i].N)) != DSV_OK) return rc;
  size_t base[DSV_MAX_GROUP];
  FwdWs w[DSV_MAX_GROUP];
  *bytes = fwd_group_ws(*p, dt, n_proj, projs, base, w);
  return DSV_OK;
}

extern "C" int dsv_lora_bwd_grouped_workspace(const dsv_plan* p, dsv_dtype dt, int32_t n_proj,
                                              const dsv_bwd_proj* projs, size_t* bytes) {
  int rc = check_group(p, dt, n_proj, projs);
  if (rc != DSV_OK) return rc;
  if (!bytes) return DSV_ERR_ARG;
  if (n_proj == 1) return dsv_lora_bwd_workspace(p, dt, projs[0].K, projs[0].N, bytes);
  for (int i = 0; i < n_proj; ++i)
    if ((rc = check_common(p, dt, projs[i].K, projs[i].N)) != DSV_OK) return rc;
  size_t base[DSV_MAX_GROUP];
  BwdWs w[DSV_MAX_GROUP];
  *bytes = bwd_group_ws(*p, dt, n_proj, projs, base, w);
  return DSV_OK;
}

namespace {

// Dropout of a grouped call: every projection's mask spec (projections with
// p = 0 get an all-keeping mask of scale 1 when another one drops, which
// leaves their results bit for bit as without dropout).
int group_dropout(const dsv_dropout* drops, int32_t n, int32_t T_t, DropoutSpec* ds, bool* any) {
  *any = false;
  for (int i = 0; i < n; ++i) ds[i] = DropoutSpec{0u, 1.f, 0, 0};
  if (!drops) return DSV_OK;
  for (int i = 0; i < n; ++i) {
    if (!dropout_spec(&drops[i], &ds[i])) return DSV_ERR_RANGE;
    if (!mask_aligned(&drops[i])) return DSV_ERR_ARG;
    if (drops[i].p > 0.0 && T_t > 0) *any = true;
  }
  return DSV_OK;
}

int fwd_grouped_impl(const dsv_plan* p, dsv_dtype dt, int32_t n_proj, const dsv_fwd_proj* projs,
                     const dsv_dropout* drops, void* workspace, size_t workspace_bytes, void* hip_stream) {
  int rc = check_group(p, dt, n_proj, projs);
  if (rc != DSV_OK) return rc;
  Strides st[DSV_MAX_GROUP];
  if (n_proj == 1) {
    const dsv_fwd_proj& q = projs[0];
    if ((rc = check_common(p, dt, q.K, q.N)) != DSV_OK || (rc = fwd_strides(q, &st[0])) != DSV_OK) return rc;
    return fwd_impl(p, dt, q.K, q.N, q.X, q.W, q.A, q.B, q.Y, q.H_save, drops, workspace, workspace_bytes,
                    hip_stream, &st[0]);
  }
  // every check before any launch
  for (int i = 0; i < n_proj; ++i) {
    const dsv_fwd_proj& q = projs[i];
    if ((rc = check_common(p, dt, q.K, q.N)) != DSV_OK) return rc;
    if ((rc = fwd_strides(q, &st[i])) != DSV_OK) return rc;
  }
  DropoutSpec ds[DSV_MAX_GROUP];
  bool dropping = false;
  if ((rc = group_dropout(drops, n_proj, p->T_t, ds, &dropping)) != DSV_OK) return rc;
  if (!p->d_meta) return DSV_ERR_ARG;
  if (p->T == 0) return DSV_OK;
  for (int i = 0; i < n_proj; ++i) {
    const dsv_fwd_proj& q = projs[i];
    if (!ptr_ok(q.X) || !ptr_ok(q.W) || !ptr_ok(q.A) || !ptr_ok(q.B) || !ptr_ok(q.Y)) return DSV_ERR_ARG;
    if (q.H_save && !aligned16(q.H_save)) return DSV_ERR_ARG;
  }
  size_t base[DSV_MAX_GROUP];
  FwdWs w[DSV_MAX_GROUP];
  const size_t total = fwd_group_ws(*p, dt, n_proj, projs, base, w);
  if (total > 0) {
    if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255)) return DSV_ERR_ARG;
    if (workspace_bytes < total) return DSV_ERR_SIZE;
  }
  char* wsb = static_cast<char*>(workspace);
  if (dt == DSV_F32) {  // the fp32 check path: the single-projection kernels, one projection at a time
    for (int i = 0; i < n_proj; ++i) {
      const dsv_fwd_proj& q = projs[i];
      rc = fwd_impl(p, dt, q.K, q.N, q.X, q.W, q.A, q.B, q.Y, q.H_save, drops ? &drops[i] : nullptr, wsb + base[i],
                    w[i].total, hip_stream, &st[i]);
      if (rc != DSV_OK) return rc;
    }
    return DSV_OK;
  }
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const MetaLayout& L = p->lay;
  const int32_t* ranks = p->dptr(L.ranks);
  const float* scales = reinterpret_cast<const float*>(p->dptr(L.scales));
  const int64_t ldh = ld_rank(p->r_max);

  // 0. dropout masks of the training rows' adapter input, every projection in
  //    one launch (into the caller's buffers where given)
  uint32_t* keepg[DSV_MAX_GROUP] = {};
  if (dropping) {
    DropoutMaskGroup mg{};
    mg.n = n_proj;
    for (int i = 0; i < n_proj; ++i) {
      keepg[i] = mask_buffer(&drops[i], at<uint32_t>(wsb + base[i], w[i].keep));
      mg.bits[i] = keepg[i];
      mg.K[i] = projs[i].K;
      mg.d[i] = ds[i];
    }
    if (launch_dropout_mask_group(mg, p->T_t, s) != hipSuccess) return DSV_ERR_DEVICE;
  }

  // 1. shrink of every projection in one launch
  SkinnyGroup sg{};
  sg.n = n_proj;
  for (int i = 0; i < n_proj; ++i) {
    const dsv_fwd_proj& q = projs[i];
    SkinnyArgs& sk = sg.a[i];
    sk.P = static_cast<const uint16_t*>(q.X);
    sk.ldp = st[i].x;
    sk.rows = p->dptr(L.shrink_rows);
    sk.items = p->dptr(L.shrink_items);
    sk.Q = static_cast<const uint16_t*>(q.A);
    sk.q_ad = (int64_t)p->r_max * q.K;
    sk.ldq = q.K;
    sk.ranks = ranks;
    sk.C = q.K;
    sk.out1 = at<uint16_t>(wsb + base[i], w[i].h_all);
    sk.ld1 = ldh;
    sk.out2 = p->T_t > 0 ? static_cast<uint16_t*>(q.H_save) : nullptr;
    sk.ld2 = p->r_max;
    sk.row_train = p->dptr(L.row_train);
    sk.part = at<float>(wsb + base[i], w[i].rk_part);
    sk.part_n = p->T;
    sk.r_max = p->r_max;
    sk.split_items = p->n_shrink;
    if (dropping) {
      sk.keep = keepg[i];
      sk.keep_words = (q.K + 31) / 32;
      sk.drop_scale = ds[i].scale;
    }
  }
  if (launch_shrink_group(sg, p->n_shrink, p->r_used, s) != hipSuccess) return DSV_ERR_DEVICE;

  // 2. gathered rows of every projection in one launch
  if (p->n_gather > 0) {
    GatherGroup gg{};
    gg.n = n_proj;
    for (int i = 0; i < n_proj; ++i) {
      gg.a[i] = GatherArgs{sg.a[i].out1, static_cast<const uint16_t*>(projs[i].B), projs[i].N,
                           at<float>(wsb + base[i], w[i].delta)};
      gg.yoff[i + 1] = gg.yoff[i] + (projs[i].N + 255) / 256;
    }
    if (launch_gather_group(gg, ldh, p->r_max, p->dptr(L.gather_items), p->n_gitems, p->dptr(L.gather_rows),
                            ranks, scales, s) != hipSuccess)
      return DSV_ERR_DEVICE;
  }

  // 3. every base GEMM in one launch, longest contraction first
  int32_t Cs[DSV_MAX_GROUP], order[DSV_MAX_GROUP];
  for (int i = 0; i < n_proj; ++i) Cs[i] = projs[i].K;
  by_contraction(n_proj, Cs, order);
  GemmGroup G{};
  G.n = n_proj;
  for (int k = 0; k < n_proj; ++k) {
    const int i = order[k];
    const dsv_fwd_proj& q = projs[i];
    GemmArgs& g = G.a[k];
    g.P = static_cast<const uint16_t*>(q.X);
    g.ldp = st[i].x;
    g.Q = static_cast<const uint16_t*>(q.W);
    g.ldq = st[i].w;
    g.out = static_cast<uint16_t*>(q.Y);
    g.ldo = st[i].y;
    g.M = p->T;
    g.Nout = q.N;
    g.C = q.K;
    g.tiles = p->dptr(L.fwd_tiles);
    g.uniform_rows = 1;
    set_split(g, whole256(p->n_ftiles, q.N), nullptr, 0);
    g.Lp = sg.a[i].out1;
    g.ldl = ldh;
    g.Lq = static_cast<const uint16_t*>(q.B);
    g.lq_ad = (int64_t)q.N * p->r_max;
    g.lq_j = 1;
    g.lq_col = p->r_max;
    g.ranks = ranks;
    g.scales = scales;
    g.delta = p->n_gather > 0 ? at<float>(wsb + base[i], w[i].delta) : nullptr;
    g.gslot = p->dptr(L.gslot);
    G.off[k + 1] = G.off[k] + g.n_mtiles * g.n_ntiles;
  }
  const int tk = timing_begin(0, s);
  const hipError_t e = launch_gemm_group_nt(G, s);
  timing_end(tk, s);
  return e == hipSuccess ? DSV_OK : DSV_ERR_DEVICE;
}

int bwd_grouped_impl(const dsv_plan* p, dsv_dtype dt, int32_t n_proj, const dsv_bwd_proj* projs, int32_t accumulate,
                     const dsv_dropout* drops, void* workspace, size_t workspace_bytes, void* hip_stream) {
  int rc = check_group(p, dt, n_proj, projs);
  if (rc != DSV_OK) return rc;
  Strides st[DSV_MAX_GROUP];
  if (n_proj == 1) {
    const dsv_bwd_proj& q = projs[0];
    if ((rc = check_common(p, dt, q.K, q.N)) != DSV_OK || (rc = bwd_strides(q, &st[0])) != DSV_OK) return rc;
    return bwd_impl(p, dt, q.K, q.N, q.X, q.W, q.A, q.B, q.H_save, q.dY, q.dA, q.dB, q.dX, accumulate, drops, q.Wt,
                    workspace, workspace_bytes, hip_stream, &st[0]);
  }
  for (int i = 0; i < n_proj; ++i) {
    if ((rc = check_common(p, dt, projs[i].K, projs[i].N)) != DSV_OK) return rc;
    if ((rc = bwd_strides(projs[i], &st[i])) != DSV_OK) return rc;
  }
  DropoutSpec ds[DSV_MAX_GROUP];
  bool dropping = false;
  if ((rc = group_dropout(drops, n_proj, p->T_t, ds, &dropping)) != DSV_OK) return rc;
  if (accumulate != 0 && accumulate != 1) return DSV_ERR_RANGE;
  if (!p->d_meta) return DSV_ERR_ARG;
  if (p->T_t == 0) return DSV_OK;
  for (int i = 0; i < n_proj; ++i) {
    const dsv_bwd_proj& q = projs[i];
    if (!ptr_ok(q.X) || !ptr_ok(q.W) || !ptr_ok(q.A) || !ptr_ok(q.B) || !ptr_ok(q.dA) || !ptr_ok(q.dB) ||
        !ptr_ok(q.dY))
      return DSV_ERR_ARG;
    if ((q.dX && !aligned16(q.dX)) || (q.H_save && !aligned16(q.H_save)) || (q.Wt && !aligned16(q.Wt)))
      return DSV_ERR_ARG;
  }
  size_t base[DSV_MAX_GROUP];
  BwdWs w[DSV_MAX_GROUP];
  const size_t total = bwd_group_ws(*p, dt, n_proj, projs, base, w);
  if (total > 0) {
    if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255)) return DSV_ERR_ARG;
    if (workspace_bytes < total) return DSV_ERR_SIZE;
  }
  char* wsb = static_cast<char*>(workspace);
  if (dt == DSV_F32) {
    for (int i = 0; i < n_proj; ++i) {
      const dsv_bwd_proj& q = projs[i];
      rc = bwd_impl(p, dt, q.K, q.N, q.X, q.W, q.A, q.B, q.H_save, q.dY, q.dA, q.dB, q.dX, accumulate,
                    drops ? &drops[i] : nullptr, q.Wt, wsb + base[i], w[i].total, hip_stream, &st[i]);
      if (rc != DSV_OK) return rc;
    }
    return DSV_OK;
  }
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const MetaLayout& L = p->lay;
  const int32_t* ranks = p->dptr(L.ranks);
  const float* scales = reinterpret_cast<const float*>(p->dptr(L.scales));
  const int64_t ldh = ld_rank(p->r_max);
  const int32_t* train_ads = p->dptr(L.train_ads);
  uint16_t* gm[DSV_MAX_GROUP];
  uint32_t* keep[DSV_MAX_GROUP];
  for (int i = 0; i < n_proj; ++i) {
    gm[i] = at<uint16_t>(wsb + base[i], w[i].g);
    keep[i] = dropping ? mask_buffer(&drops[i], at<uint32_t>(wsb + base[i], w[i].keep)) : nullptr;
  }

  // 0. the forward's dropout masks: the caller's buffers, or regenerated from
  //    the same seeds and offsets (one launch for those)
  if (dropping) {
    DropoutMaskGroup mg{};
    mg.n = n_proj;
    for (int i = 0; i < n_proj; ++i) {
      mg.bits[i] = drops[i].mask ? nullptr : keep[i];
      mg.K[i] = projs[i].K;
      mg.d[i] = ds[i];
    }
    if (launch_dropout_mask_group(mg, p->T_t, s) != hipSuccess) return DSV_ERR_DEVICE;
  }

  // 1. h of the training rows for projections whose forward kept no H_save
  const uint16_t* hs[DSV_MAX_GROUP];
  int64_t ldhs[DSV_MAX_GROUP];
  SkinnyGroup rg{};
  for (int i = 0; i < n_proj; ++i) {
    const dsv_bwd_proj& q = projs[i];
    hs[i] = static_cast<const uint16_t*>(q.H_save);
    ldhs[i] = p->r_max;
    if (hs[i]) continue;
    uint16_t* hrec = at<uint16_t>(wsb + base[i], w[i].hrec);
    SkinnyArgs& sh = rg.a[rg.n++];
    sh.P = static_cast<const uint16_t*>(q.X);
    sh.ldp = st[i].x;
    sh.rows = p->dptr(L.train_rows);
    sh.items = p->dptr(L.train_items);
    sh.Q = static_cast<const uint16_t*>(q.A);
    sh.q_ad = (int64_t)p->r_max * q.K;
    sh.ldq = q.K;
    sh.ranks = ranks;
    sh.C = q.K;
    sh.out2 = hrec;
    sh.ld2 = ldh;
    sh.row_train = p->dptr(L.row_train);
    sh.keep = keep[i];
    sh.keep_words = (q.K + 31) / 32;
    sh.drop_scale = ds[i].scale;
    sh.part = at<float>(wsb + base[i], w[i].h_part);
    sh.part_n = p->T_t;
    sh.r_max = p->r_max;
    sh.split_items = p->n_shrink;  // the forward shrink's split: the same sums
    hs[i] = hrec;
    ldhs[i] = ldh;
  }
  if (rg.n > 0 && launch_shrink_train_group(rg, p->n_titems, p->r_train, s) != hipSuccess) return DSV_ERR_DEVICE;

  // 2. chunk partials of dy^T h (dB), every projection; the same pass writes
  //    the column-block partials of dy B_a (g), reading dy once
  TokenReduceGroup tbg{};
  tbg.n = n_proj;
  for (int i = 0; i < n_proj; ++i) {
    const dsv_bwd_proj& q = projs[i];
    TokenReduceArgs& tb = tbg.a[i];
    tb.P = static_cast<const uint16_t*>(q.dY);
    tb.ldp = st[i].dy;
    tb.Q = hs[i];
    tb.ldq = ldhs[i];
    tb.chunks = p->dptr(L.chunks);
    tb.ranks = ranks;
    tb.C = q.N;
    tb.r_max = p->r_max;
    tb.part = at<float>(wsb + base[i], w[i].part_b);
    tb.B = static_cast<const uint16_t*>(q.B);
    tb.gpart = at<float>(wsb + base[i], w[i].g_part);
    tb.gpart_n = p->T_t;
    tbg.yoff[i + 1] = tbg.yoff[i] + token_col_blocks(q.N);
  }
  if (launch_token_reduce_group(tbg, p->n_chunks, p->r_train, s) != hipSuccess) return DSV_ERR_DEVICE;

  // 3. g = s_a dy B_a of every projection: block partials summed in order, rounded once
  SkinnyGroup gf{};
  gf.n = n_proj;
  for (int i = 0; i < n_proj; ++i) {
    SkinnyArgs& sk = gf.a[i];
    sk.items = p->dptr(L.train_items);
    sk.ranks = ranks;
    sk.scales = scales;
    sk.out1 = gm[i];
    sk.ld1 = ldh;
    sk.part = tbg.a[i].gpart;
    sk.part_n = p->T_t;
    sk.r_max = p->r_max;
    sk.pieces = token_col_blocks(projs[i].N);
  }
  if (launch_g_finish_group(gf, p->n_titems, s) != hipSuccess) return DSV_ERR_DEVICE;

  // 4. chunk partials of x^T g (dA), every projection
  TokenReduceGroup tag{};
  tag.n = n_proj;
  for (int i = 0; i < n_proj; ++i) {
    const dsv_bwd_proj& q = projs[i];
    TokenReduceArgs& ta = tag.a[i];
    ta.P = static_cast<const uint16_t*>(q.X);
    ta.ldp = st[i].x;
    ta.prow = p->dptr(L.train_rows);
    ta.Q = gm[i];
    ta.ldq = ldh;
    ta.chunks = p->dptr(L.chunks);
    ta.ranks = ranks;
    ta.C = q.K;
    ta.r_max = p->r_max;
    ta.part = at<float>(wsb + base[i], w[i].part_a);
    ta.keep = keep[i];  // dA contracts the masked input
    ta.keep_words = (q.K + 31) / 32;
    tag.yoff[i + 1] = tag.yoff[i] + token_col_blocks(q.K);
  }

  // 5. fixed-order sums into dB (scaled by s_a) and dA, every projection
  ReduceOutGroup og{};
  og.n = 2 * n_proj;
  for (int i = 0; i < n_proj; ++i) {
    og.a[2 * i] = ReduceOutArgs{tbg.a[i].part, projs[i].N, scales, 0, projs[i].dB, 1.f};
    og.a[2 * i + 1] = ReduceOutArgs{tag.a[i].part, projs[i].K, nullptr, 1, projs[i].dA,
                                    dropping ? ds[i].scale : 1.f};
  }
  auto dA_and_sums = [&](hipStream_t sx) -> int {
    if (launch_token_reduce_group(tag, p->n_chunks, p->r_train, sx) != hipSuccess) return DSV_ERR_DEVICE;
    if (launch_reduce_out_group(og, p->r_max, p->r_train, train_ads, p->n_tads, p->dptr(L.tad_chunk_ptr),
                                p->dptr(L.tad_chunks), ranks, accumulate, sx) != hipSuccess)
      return DSV_ERR_DEVICE;
    return DSV_OK;
  };

  // 6. every dX GEMM in one launch, longest contraction first (projections with a
  //    transposed weight in one NT launch, the others in one NN launch)
  auto dx_all = [&](hipStream_t s) -> int {
    int32_t Cs[DSV_MAX_GROUP], order[DSV_MAX_GROUP];
    for (int i = 0; i < n_proj; ++i) Cs[i] = projs[i].N;
    by_contraction(n_proj, Cs, order);
    for (int nt = 1; nt >= 0; --nt) {
      GemmGroup G{};
      for (int k = 0; k < n_proj; ++k) {
        const int i = order[k];
        const dsv_bwd_proj& q = projs[i];
        if (!q.dX || (q.Wt != nullptr) != (nt == 1)) continue;
        GemmArgs& g = G.a[G.n];
        g.P = static_cast<const uint16_t*>(q.dY);
        g.ldp = st[i].dy;
        g.Q = static_cast<const uint16_t*>(nt ? q.Wt : q.W);
        g.ldq = nt ? st[i].wt : st[i].w;
        g.out = static_cast<uint16_t*>(q.dX);
        g.ldo = st[i].dx;
        g.M = p->T_t;
        g.Nout = q.K;
        g.C = q.N;
        g.tiles = p->dptr(L.bwd_tiles);
        g.uniform_rows = p->btiles_uniform;
        set_split(g, whole256(p->n_btiles, q.K), nullptr, 0);
        g.Lp = gm[i];
        g.ldl = ldh;
        g.Lq = static_cast<const uint16_t*>(q.A);
        g.lq_ad = (int64_t)p->r_max * q.K;
        g.lq_j = q.K;
        g.lq_col = 1;
        g.ranks = ranks;
        g.keep = keep[i];  // dropout: g A_a through the input's mask
        g.keep_words = (q.K + 31) / 32;
        g.keep_scale = ds[i].scale;
        G.off[G.n + 1] = G.off[G.n] + g.n_mtiles * g.n_ntiles;
        ++G.n;
      }
      if (G.n > 0) {
        const int tk = timing_begin(1, s);
        const hipError_t e = nt ? launch_gemm_group_nt(G, s) : launch_gemm_group_nn(G, s);
        timing_end(tk, s);
        if (e != hipSuccess) return DSV_ERR_DEVICE;
      }
    }
    return DSV_OK;
  };

  // dX needs g only: the dA reduction and the final sums run beside it on the
  // side stream (joined back into the caller's stream before the call returns)
  {
    std::lock_guard<std::mutex> lk(g_side_mu);
    if (SideStream* sd = side_stream()) {
      if (hipEventRecord(sd->fork, s) != hipSuccess) return DSV_ERR_DEVICE;
      if ((rc = dx_all(s)) != DSV_OK) return rc;
      if (hipStreamWaitEvent(sd->s, sd->fork, 0) != hipSuccess) return DSV_ERR_DEVICE;
      if ((rc = dA_and_sums(sd->s)) != DSV_OK) return rc;
      if (hipEventRecord(sd->join, sd->s) != hipSuccess || hipStreamWaitEvent(s, sd->join, 0) != hipSuccess)
        return DSV_ERR_DEVICE;
      return DSV_OK;
    }
  }
  if ((rc = dA_and_sums(s)) != DSV_OK) return rc;
  return dx_all(s);
}

}  // namespace

extern "C" int dsv_cobatch_fwd_grouped(const dsv_plan* p, dsv_dtype dt, int32_t n_proj, const dsv_fwd_proj* projs,
                                       void* workspace, size_t workspace_bytes, void* hip_stream) {
  return fwd_grouped_impl(p, dt, n_proj, projs, nullptr, workspace, workspace_bytes, hip_stream);
}

extern "C" int dsv_cobatch_fwd_grouped_dropout(const dsv_plan* p, dsv_dtype dt, int32_t n_proj,
                                               const dsv_fwd_proj* projs, const dsv_dropout* dropouts,
                                               void* workspace, size_t workspace_bytes, void* hip_stream) {
  if (!dropouts) return DSV_ERR_ARG;
  return fwd_grouped_impl(p, dt, n_proj, projs, dropouts, workspace, workspace_bytes, hip_stream);
}

extern "C" int dsv_lora_bwd_grouped(const dsv_plan* p, dsv_dtype dt, int32_t n_proj, const dsv_bwd_proj* projs,
                                    int32_t accumulate, void* workspace, size_t workspace_bytes, void* hip_stream) {
  return bwd_grouped_impl(p, dt, n_proj, projs, accumulate, nullptr, workspace, workspace_bytes, hip_stream);
}

extern "C" int dsv_lora_bwd_grouped_dropout(const dsv_plan* p, dsv_dtype dt, int32_t n_proj,
                                            const dsv_bwd_proj* projs, int32_t accumulate,
                                            const dsv_dropout* dropouts, void* workspace, size_t workspace_bytes,
                                            void* hip_stream) {
  if (!dropouts) return DSV_ERR_ARG;
  return bwd_grouped_impl(p, dt, n_proj, projs, accumulate, dropouts, workspace, workspace_bytes, hip_stream);
}
