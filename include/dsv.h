/*
 * dsv.h -- C ABI of the co-batched multi-LoRA linear layer for AMD MI355X (gfx950).
 *
 * One linear layer runs a mixed batch of inference tokens (prefill or decode)
 * and LoRA fine-tuning tokens in a single pass, as in DeltaServe
 * (arXiv 2607.28848):
 *   - Sec. 2.2 ("Parameter-Efficient Fine-Tuning"): a frozen weight W of shape
 *     d x k receives the low-rank update B A, A of shape r x k, B of shape d x r;
 *     multi-LoRA batching lets tokens of different adapters share one pass of
 *     the frozen base while each applies its own adapter.
 *   - Sec. 3.2 ("Co-Serving Model", "Mixed forward batch"): each fine-tuning
 *     sample is one more batch entry bound to a reserved training adapter; only
 *     its rows keep activations for the backward.
 *   - Sec. 3.2 ("Backward subprocess"): the backward computes the LoRA
 *     gradients of the training rows; the base weight stays frozen.
 *   - Sec. 4.1 ("Fine-tuning Workload"): rank 16 with alpha 32; each adapter
 *     here carries its own scale s_a (alpha / r for the paper's adapter).
 *
 * For a token row x bound to adapter a (row-vector form):
 *     h = x A_a^T                  (rank r_a; kept for training rows)
 *     y = x W^T + s_a h B_a^T      (one rounding of the fp32 sum)
 * and, for training rows with upstream gradient dy:
 *     g   = s_a dy B_a             (gradient reaching h)
 *     dB_a += s_a dy^T h,  dA_a += g^T x,  dx = dy W + g A_a.
 *
 * LAYOUTS.  Every matrix is dense row-major in the paper's orientation, which
 * is also the torch.nn.Linear / PEFT parameter layout (K = in features,
 * N = out features, T = tokens in the batch, T_t = training tokens):
 *     X      [T][K]                 input rows of the whole batch
 *     W      [N][K]                 frozen base weight
 *     A      [n_ad][r_max][K]       stacked adapter down-projections
 *     B      [n_ad][N][r_max]       stacked adapter up-projections
 *     Y      [T][N]                 output
 *     H_save [T_t][r_max]           h of the training rows (pre-scale)
 *     dY     [T_t][N]               upstream gradient of the training rows
 *     dX     [T_t][K]               input gradient of the training rows
 *     dA     [n_ad][r_max][K] fp32, dB [n_ad][N][r_max] fp32
 * Training rows are numbered in ascending token-row order ("compact order");
 * H_save, dY and dX use it.  Rank-padding entries (index j >= r_a) are never
 * read or written.  Element type: bf16 (DSV_BF16) or fp32 (DSV_F32) for every
 * tensor except dA / dB, which are fp32 in both modes.  bf16 arithmetic
 * accumulates in fp32; h is rounded to bf16 once and that same value feeds
 * both the output and H_save.
 *
 * OWNERSHIP.  The caller owns every device buffer (metadata blob, inputs,
 * outputs, workspaces).  The library allocates no device memory; it owns only
 * the host-side plan.  Every launch is asynchronous on the caller's HIP stream
 * (NULL = default stream); a plan is immutable once built and may serve any
 * number of projections and streams.
 *
 * ERRORS.  Every check runs on the host before any launch; a call that
 * returns an error has launched nothing and written nothing.  Launch failures
 * are reported as DSV_ERR_DEVICE.  No C++ exception crosses this interface.
 */
#ifndef DSV_H
#define DSV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* One batch entry: tokens [start, start + len) of the batch, bound to
 * `adapter`; is_train = 1 marks a fine-tuning sample (Sec. 3.2). */
typedef struct {
  int32_t start;
  int32_t len;
  int32_t adapter;
  int32_t is_train;
} dsv_segment;

typedef enum { DSV_BF16 = 0, DSV_F32 = 1 } dsv_dtype;

enum {
  DSV_OK = 0,
  DSV_ERR_ARG = -1,    /* null / misaligned pointer, negative count, plan not on device */
  DSV_ERR_RANGE = -2,  /* adapter id, rank, r_max, scale or flag out of range */
  DSV_ERR_LAYOUT = -3, /* segments do not tile [0, n_tokens) exactly */
  DSV_ERR_SIZE = -4,   /* buffer too small, K / N not a positive multiple of 8, too large */
  DSV_ERR_DEVICE = -5  /* a HIP call or kernel launch failed */
};

typedef struct dsv_plan dsv_plan;

/* Largest supported adapter rank stride. */
#define DSV_MAX_RANK 64

/*
 * dsv_segments_build -- validate and pack the batch's segment table.
 *
 * segs[n_segs]: the batch entries, in any order.  They must tile
 * [0, n_tokens) exactly; zero-length entries are no-ops (0 <= start <=
 * n_tokens) and are otherwise ignored.  adapter_rank[n_adapters] in
 * [1, r_max], adapter_scale[n_adapters] finite, 1 <= r_max <= DSV_MAX_RANK.
 *
 * The plan records the per-row adapter map, the compact training-row order,
 * the rows of each adapter for the rank-r shrink, the split between rows
 * whose low-rank term rides the GEMM tile and rows grouped by adapter for the
 * gathered path (many short segments, e.g. decode), the GEMM tile list and
 * the per-adapter chunks of the backward reductions.
 *
 * d_meta == NULL: validation and size query only.  *meta_bytes receives the
 *   device blob size; if out_plan is not NULL a host-only plan is returned
 *   that the dsv_plan_* queries accept but fwd / bwd reject (DSV_ERR_ARG).
 * d_meta != NULL: a 256-byte aligned device buffer of at least *meta_bytes
 *   bytes; the packed metadata is copied into it with one asynchronous copy
 *   on hip_stream, and the returned plan refers to it.  d_meta must stay
 *   allocated while the plan is used.  The copy is ordered on hip_stream
 *   only: work queued on another stream that still reads an earlier plan in
 *   the same buffer must finish first, and launches on another stream must
 *   wait for the copy (an event recorded on hip_stream after this call).
 *   Uploading on a side stream into alternating buffers lets the copy of the
 *   next batch's metadata overlap the current batch's kernels.
 * On error *out_plan is set to NULL (when out_plan is not NULL).
 */
int dsv_segments_build(const dsv_segment* segs, int32_t n_segs, int32_t n_tokens,
                       const int32_t* adapter_rank, const float* adapter_scale,
                       int32_t n_adapters, int32_t r_max, void* d_meta,
                       size_t* meta_bytes, void* hip_stream, dsv_plan** out_plan);

/* Number of training tokens T_t (rows of H_save, dY and dX); -1 if plan is NULL. */
int32_t dsv_plan_train_rows(const dsv_plan* plan);

/* Copies the compact training-row order (T_t token rows, ascending) into
 * host_out.  Returns T_t or a negative status. */
int32_t dsv_plan_train_row_index(const dsv_plan* plan, int32_t* host_out);

/* Copies the token rows served by the gathered low-rank path (slot order:
 * by adapter, then row) into host_out.  Returns their count or a negative
 * status. */
int32_t dsv_plan_gathered_rows(const dsv_plan* plan, int32_t* host_out);

/* Copies the host image of the packed metadata (meta_bytes bytes) into
 * host_out, for inspection.  Returns DSV_OK or a negative status. */
int dsv_plan_meta_copy(const dsv_plan* plan, void* host_out, size_t bytes);

/* Counts of the plan's work lists, in this order: fwd 256-row GEMM tiles,
 * shrink items, gathered rows, gathered items, bwd 256-row GEMM tiles, bwd
 * chunks, adapters owning training rows, bwd rank-r items, fwd 128-row GEMM
 * tiles, bwd 128-row GEMM tiles.  Returns DSV_OK or DSV_ERR_ARG. */
int dsv_plan_counts(const dsv_plan* plan, int32_t out[10]);

/* Releases the host plan (NULL is a no-op).  If the plan was uploaded, first
 * waits until its asynchronous metadata copy has completed.  Does not touch
 * d_meta; kernels already queued keep reading it from there. */
void dsv_plan_free(dsv_plan* plan);

/*
 * dsv_cobatch_fwd_workspace -- bytes of device workspace dsv_cobatch_fwd
 * needs for this plan, dtype and shape (h of every row, plus the fp32
 * low-rank terms of the gathered rows).
 */
int dsv_cobatch_fwd_workspace(const dsv_plan* plan, dsv_dtype dtype, int32_t K, int32_t N,
                              size_t* bytes);

/*
 * dsv_cobatch_fwd -- Y = X W^T + s_a (X A_a^T) B_a^T for every row, and
 * H_save = X A_a^T for the training rows (Sec. 2.2, Sec. 3.2).
 * H_save == NULL keeps nothing for the backward (residual-only retention,
 * Sec. 3.2 "Mixed forward batch": the caller keeps X and dsv_lora_bwd
 * recomputes h).  K and N must be positive multiples of 8; every pointer
 * 16-byte aligned; workspace of at least dsv_cobatch_fwd_workspace bytes,
 * 256-byte aligned.
 */
int dsv_cobatch_fwd(const dsv_plan* plan, dsv_dtype dtype, int32_t K, int32_t N,
                    const void* X, const void* W, const void* A, const void* B, void* Y,
                    void* H_save, void* workspace, size_t workspace_bytes, void* hip_stream);

/*
 * dsv_cobatch_fwd_noalloc -- dsv_cobatch_fwd for callers that cannot allocate
 * device memory or pass a workspace: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  It calls no allocating
 * routine (no hipMalloc / hipFree, no library allocation): its intermediates
 * (h of every row, the fp32 low-rank terms of the gathered rows, the partial
 * sums of a split shrink) live in a fixed scratch array in the library's own
 * device memory, DSV_NOALLOC_SCRATCH_BYTES per device, held from the first
 * call on a device until the process ends.  The caller still passes inputs and
 * outputs; arguments, layouts and alignment as dsv_cobatch_fwd.
 * A batch whose intermediates exceed the scratch (dsv_cobatch_fwd_workspace of
 * the same plan and shape is an upper bound of what is used) returns
 * DSV_ERR_SIZE before any launch.  The base GEMM splits no tile along the
 * contraction (a split keeps a partial tile per piece): where
 * dsv_cobatch_fwd splits one (dsv_gemm_config pass 0 reports split tiles), Y
 * may differ from it in the last bit (another summation order); otherwise
 * Y and H_save are bit-identical to dsv_cobatch_fwd.
 * Every call on a device uses that device's one scratch array, which keeps
 * the last call's contents (no call relies on them): calls that overlap on
 * one device -- on different streams without ordering, or from several
 * threads -- race on it and give wrong results.  Calls ordered on one stream
 * are safe.
 */
#define DSV_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int dsv_cobatch_fwd_noalloc(const dsv_plan* plan, dsv_dtype dtype, int32_t K, int32_t N,
                            const void* X, const void* W, const void* A, const void* B, void* Y,
                            void* H_save, void* hip_stream);

/*
 * dsv_lora_bwd_workspace -- bytes of device workspace dsv_lora_bwd needs
 * (transposed copies of the small operands, g, and the fp32 partial sums of
 * the deterministic reductions over training tokens).
 */
int dsv_lora_bwd_workspace(const dsv_plan* plan, dsv_dtype dtype, int32_t K, int32_t N,
                           size_t* bytes);

/*
 * dsv_lora_bwd -- LoRA backward of the training rows (Sec. 3.2, "Backward
 * subprocess"): with g = s_a dY B_a,
 *     dB_a  (+)=  s_a dY^T H_save      dA_a  (+)=  g^T X_train
 *     dX     =   dY W + g A_a          (skipped when dX is NULL)
 * where the sums run over the training rows of adapter a.  accumulate = 0
 * overwrites, accumulate = 1 adds to, the dA / dB slices of adapters that own
 * training rows; other slices are untouched.  The reductions over tokens are
 * deterministic (fixed-order fp32 partial sums, no atomics): repeated calls
 * give bit-identical results.  H_save == NULL recomputes h of the training
 * rows from X and A first (the forward's own shrink, so the same values bit
 * for bit; 2 T_t K r FLOP and one read of X's training rows), for a forward
 * that kept no H_save.  With no training rows the call is a no-op.
 */
int dsv_lora_bwd(const dsv_plan* plan, dsv_dtype dtype, int32_t K, int32_t N,
                 const void* X, const void* W, const void* A, const void* B,
                 const void* H_save, const void* dY, float* dA, float* dB, void* dX,
                 int32_t accumulate, void* workspace, size_t workspace_bytes,
                 void* hip_stream);

/*
 * LoRA dropout of the training rows (Sec. 4.1 fine-tunes the adapter with
 * dropout 0.05).  The low-rank branch of a training row reads its input
 * through a mask: x~[i][k] = x[i][k] keep(i, k) / (1 - p); the base product
 * X W^T and the inference rows are unchanged.  keep(i, k) for compact training
 * row i (ascending token order) and column k is decided by Philox4x32-10
 * (Salmon et al., SC 2011): output word k mod 4 of the generator at counter
 * (k / 4, i, offset mod 2^32, offset / 2^32) and key (seed mod 2^32,
 * seed / 2^32) is compared with floor(p 2^32); words below it drop the
 * element.  The mask is a pure function of (seed, offset, i, k): the backward
 * regenerates the forward's mask from the same three values, and a caller
 * draws a fresh mask per step by advancing offset.  0 <= p < 1; p = 0 gives
 * the plain entry points' results bit for bit.
 *
 * mask (optional, NULL: none): a device buffer of T_t * ceil(K / 32) 32-bit
 * words (4-byte aligned, bit b of word w of row i keeps column 32 w + b),
 * owned by the caller, one per projection.  A forward given it draws the mask
 * into it instead of into its workspace; a backward given it reads the mask
 * from it instead of drawing it again.  The buffer must then hold what the
 * forward of the same plan, K, p, seed and offset wrote, unmodified since.
 * Results are bit-identical with and without the buffer; it saves the
 * backward's draw (about 8 Philox4x32-10 blocks per 32 elements).
 */
typedef struct {
  double p;
  uint64_t seed;
  uint64_t offset;
  uint32_t* mask;
} dsv_dropout;

/*
 * dsv_cobatch_fwd_dropout -- dsv_cobatch_fwd with LoRA dropout on the
 * training rows:  y = x W^T + s_a (x~ A_a^T) B_a^T,  H_save = x~ A_a^T.
 * Same arguments, layouts and workspace size (dsv_cobatch_fwd_workspace) as
 * dsv_cobatch_fwd.  Returns DSV_ERR_ARG for a NULL dropout, DSV_ERR_RANGE for
 * p outside [0, 1), else as dsv_cobatch_fwd.
 */
int dsv_cobatch_fwd_dropout(const dsv_plan* plan, dsv_dtype dtype, int32_t K, int32_t N,
                            const void* X, const void* W, const void* A, const void* B,
                            void* Y, void* H_save, const dsv_dropout* dropout, void* workspace,
                            size_t workspace_bytes, void* hip_stream);

/*
 * dsv_lora_bwd_dropout_workspace -- bytes of device workspace
 * dsv_lora_bwd_dropout needs (the regenerated mask, T_t ceil(K / 32) words,
 * lives in it; at present the same size as dsv_lora_bwd_workspace).
 */
int dsv_lora_bwd_dropout_workspace(const dsv_plan* plan, dsv_dtype dtype, int32_t K, int32_t N,
                                   size_t* bytes);

/*
 * dsv_lora_bwd_dropout -- backward of dsv_cobatch_fwd_dropout with the same
 * dropout values: with g = s_a dY B_a and x~ the forward's masked, scaled
 * adapter input,
 *     dB_a  (+)=  s_a dY^T H_save      dA_a  (+)=  g^T X~_train
 *     dX     =   dY W + (g A_a) masked and scaled like the input
 * H_save is the forward's (already masked); H_save == NULL recomputes it from
 * X through the regenerated mask.  Arguments as dsv_lora_bwd, workspace of at
 * least dsv_lora_bwd_dropout_workspace bytes.  Returns DSV_ERR_ARG for a NULL
 * dropout, DSV_ERR_RANGE for p outside [0, 1), else as dsv_lora_bwd.
 */
int dsv_lora_bwd_dropout(const dsv_plan* plan, dsv_dtype dtype, int32_t K, int32_t N,
                         const void* X, const void* W, const void* A, const void* B,
                         const void* H_save, const void* dY, float* dA, float* dB, void* dX,
                         int32_t accumulate, const dsv_dropout* dropout, void* workspace,
                         size_t workspace_bytes, void* hip_stream);

/*
 * Grouped launches over several projections of one batch (the paper's layer
 * set: q/k/v/o and gate/up/down all see the same segment table, Sec. 4.1).
 * dsv_cobatch_fwd_grouped and dsv_lora_bwd_grouped compute, for every entry of
 * projs[0 .. n_proj), exactly what dsv_cobatch_fwd / dsv_lora_bwd compute for
 * it, with one launch per step for all projections instead of one per
 * projection: the rank-r kernels, token reductions and final sums run the
 * projections side by side, and the base GEMMs of all projections form one
 * launch of whole 256 x 256 tiles ordered by contraction length (longest
 * first), so one projection's last partial wave is filled by the next one's
 * tiles.  Operands may alias across entries (q/k/v read one X); outputs must
 * not.  1 <= n_proj <= DSV_MAX_GROUP; n_proj = 1 is the single-projection
 * call.  Each entry follows the single call's shape, layout and alignment
 * rules; any entry that fails them fails the whole call before any launch.
 * The bf16 results may differ from the single calls in the last bit where
 * those split a tile along the contraction (another summation order);
 * repeated grouped calls are bit-identical.  The workspace holds the
 * single-call regions of every projection, 256-byte aligned, of at least the
 * *_grouped_workspace size.  The _dropout forms take dropouts[n_proj], one
 * dsv_dropout per projection (a caller gives each projection its own seed or
 * offset), and compute what dsv_cobatch_fwd_dropout / dsv_lora_bwd_dropout
 * compute for each entry; they return DSV_ERR_ARG for a NULL dropouts and
 * DSV_ERR_RANGE for any p outside [0, 1), and use the same workspace sizes.
 *
 * Streams (the grouped bf16 backward of two or more projections): dX needs g
 * only, so the dA reductions and the final sums of dA and dB run beside the dX GEMMs
 * on a second stream of the current device that the library creates on first
 * use (default priority, non-blocking, kept until the process ends), so
 * hip_stream must belong to the current device.  That
 * work is forked from hip_stream after g is complete and joined back into
 * hip_stream by an event wait before the call returns: everything the call
 * writes is complete in hip_stream order, as with one stream, and the results
 * are the same bits.  The fork and join are enqueued under a library lock, so
 * calls from several host threads stay correct; their side work queues up on
 * the one side stream.  Under stream capture the second stream joins the
 * capture through the fork event.  If the second stream cannot be created the
 * call runs everything on hip_stream.
 *
 * dsv_bwd_proj.Wt: the frozen weight is never updated, so a caller may keep it
 * a second time, transposed ([K][N], 16-byte aligned, the same bf16 values).
 * With it the dX GEMM reads its weight tile contraction-contiguous, as the
 * forward reads W, instead of transposing W inside the kernel (about 20%
 * faster on the Llama-3-8B set on MI355X); the results are bit-identical
 * either way.  Ignored for fp32; NULL reads W.
 *
 * Row strides (ldx, ldw, ldy; ldx, ldw, lddy, lddx, ldwt), in elements: the
 * distance between consecutive rows of that caller buffer.  0 means dense,
 * the row length (K for X, W and dX; N for Y, dY and Wt).  A non-zero stride
 * must be at least the row length, a multiple of 8 (rows stay 16-byte
 * aligned) and at most 2^20, else DSV_ERR_SIZE before any launch.  Only the
 * first K (or N) elements of a row are read or written; the elements between
 * rows are never touched, and the results are bit-identical to those on dense
 * buffers holding the same values.  Strides matter for speed where the dense
 * row length makes the rows of a GEMM tile collide in the memory system:
 * dsv_row_stride gives the stride the library recommends.
 */
#define DSV_MAX_GROUP 8

/*
 * dsv_row_stride -- the row stride (elements) recommended for caller buffers
 * whose rows hold n elements of dtype: n + 64 for bf16 rows of more than 8192
 * elements whose byte length is a multiple of 4096, else n.  (On MI355X the
 * base GEMM's contraction loop ran about 18% slower over dense bf16 rows of
 * 14336 elements than over rows 64 elements longer, with the same tile order
 * and data.)  Returns 0 for n <= 0 or an unknown dtype.
 */
int32_t dsv_row_stride(int32_t n, dsv_dtype dtype);

typedef struct {
  int32_t K, N;           /* in / out features of this projection */
  const void* X;          /* [T][K] */
  const void* W;          /* [N][K] */
  const void* A;          /* [n_ad][r_max][K] */
  const void* B;          /* [n_ad][N][r_max] */
  void* Y;                /* [T][N] out */
  void* H_save;           /* [T_t][r_max] out, or NULL (residual-only retention) */
  int32_t ldx, ldw, ldy;  /* row strides of X, W, Y (elements; 0: dense) */
} dsv_fwd_proj;

typedef struct {
  int32_t K, N;
  const void* X;          /* [T][K] */
  const void* W;          /* [N][K] */
  const void* A;          /* [n_ad][r_max][K] */
  const void* B;          /* [n_ad][N][r_max] */
  const void* H_save;     /* [T_t][r_max], or NULL: recomputed from X */
  const void* dY;         /* [T_t][N] */
  float* dA;              /* [n_ad][r_max][K] fp32 */
  float* dB;              /* [n_ad][N][r_max] fp32 */
  void* dX;               /* [T_t][K], or NULL: not computed */
  const void* Wt;         /* optional, bf16: W transposed, [K][N] row-major (see below), or NULL */
  int32_t ldx, ldw;       /* row strides of X, W (elements; 0: dense) */
  int32_t lddy, lddx;     /* row strides of dY, dX */
  int32_t ldwt;           /* row stride of Wt */
} dsv_bwd_proj;

int dsv_cobatch_fwd_grouped_workspace(const dsv_plan* plan, dsv_dtype dtype, int32_t n_proj,
                                      const dsv_fwd_proj* projs, size_t* bytes);
int dsv_cobatch_fwd_grouped(const dsv_plan* plan, dsv_dtype dtype, int32_t n_proj,
                            const dsv_fwd_proj* projs, void* workspace, size_t workspace_bytes,
                            void* hip_stream);
int dsv_lora_bwd_grouped_workspace(const dsv_plan* plan, dsv_dtype dtype, int32_t n_proj,
                                   const dsv_bwd_proj* projs, size_t* bytes);
int dsv_lora_bwd_grouped(const dsv_plan* plan, dsv_dtype dtype, int32_t n_proj,
                         const dsv_bwd_proj* projs, int32_t accumulate, void* workspace,
                         size_t workspace_bytes, void* hip_stream);
int dsv_cobatch_fwd_grouped_dropout(const dsv_plan* plan, dsv_dtype dtype, int32_t n_proj,
                                    const dsv_fwd_proj* projs, const dsv_dropout* dropouts,
                                    void* workspace, size_t workspace_bytes, void* hip_stream);
int dsv_lora_bwd_grouped_dropout(const dsv_plan* plan, dsv_dtype dtype, int32_t n_proj,
                                 const dsv_bwd_proj* projs, int32_t accumulate,
                                 const dsv_dropout* dropouts, void* workspace,
                                 size_t workspace_bytes, void* hip_stream);

/*
 * Kernel timing: benchmark instrumentation only, not part of the layer's
 * computation (the results of every other call are the same with it on or
 * off).  Its state is process-global: one set of event pairs shared by every
 * thread, stream and device of the process.  While enabled (on = 1), every
 * dsv_cobatch_fwd / dsv_lora_bwd call records a HIP event pair on its own
 * stream immediately around its matrix-core GEMM launch (forward: the base
 * GEMM with its low-rank prologue; backward: the dX GEMM; in both, when tiles
 * are split along the contraction, also the kernel that sums their pieces).  Up to 4096 pairs
 * are kept; further launches are not timed.  dsv_timing_read waits for the
 * recorded events, returns the summed milliseconds and launch counts of the
 * forward and backward GEMMs, and releases the pairs.  Not thread-safe:
 * enable it only in a single-threaded benchmark.  Returns DSV_OK, or
 * DSV_ERR_DEVICE if a HIP event call failed.
 */
int dsv_timing_enable(int32_t on);
int dsv_timing_read(double* fwd_ms, int32_t* fwd_launches, double* bwd_ms,
                    int32_t* bwd_launches);

/*
 * dsv_adamw_step -- one fused AdamW step of the plan's training adapters
 * (the optimizer update that follows the LoRA backward, Sec. 3.2 "Backward
 * subprocess"; AdamW with decoupled weight decay, Sec. 4.1: lr 1e-3, weight
 * decay 0.01).  For every adapter with training rows in the plan and every
 * element of its A slice (rows j < r_a) and B slice (columns j < r_a):
 *     p <- p (1 - lr wd)
 *     m <- beta1 m + (1 - beta1) g,      v <- beta2 v + (1 - beta2) g^2
 *     p <- p - lr m_hat / (sqrt(v_hat) + eps),
 *          m_hat = m / (1 - beta1^step), v_hat = v / (1 - beta2^step)
 * with g from dA / dB (as dsv_lora_bwd leaves them), then writes p rounded
 * once (bf16: to nearest even; fp32: copied) into the parameter stacks A / B
 * that dsv_cobatch_fwd reads.  A_master / B_master, A_m, A_v, B_m, B_v are
 * fp32 in the dA / dB layouts ([n_ad][r_max][K], [n_ad][N][r_max]), owned by
 * the caller (moments start at zero, masters at the fp32 value of A / B).
 * A or B may be NULL to skip that copy.  step >= 1 is the 1-based step
 * count.  Other adapters and rank-padding entries are neither read nor
 * written.  Returns DSV_OK, DSV_ERR_ARG (NULL / misaligned pointer, plan not
 * on device), DSV_ERR_RANGE (step < 1, lr or wd < 0 or not finite, beta not
 * in [0, 1), eps <= 0), DSV_ERR_SIZE or DSV_ERR_DEVICE.
 */
typedef struct {
  double lr;
  double beta1;
  double beta2;
  double eps;
  double weight_decay;
} dsv_adamw_hparams;  /* double: 1 - beta is formed on the host before rounding to fp32 */

int dsv_adamw_step(const dsv_plan* plan, dsv_dtype dtype, int32_t K, int32_t N, int32_t step,
                   const dsv_adamw_hparams* hp, const float* dA, const float* dB, float* A_master,
                   float* B_master, float* A_m, float* A_v, float* B_m, float* B_v, void* A,
                   void* B, void* hip_stream);

/*
 * dsv_adamw_step_grouped -- the same AdamW step for the adapters of up to
 * DSV_MAX_GROUP projections of one layer (q, k, v, o, gate, up, down share
 * the batch's training adapters but have their own K x N), in one launch.
 * projs[n_proj] holds each projection's shape and the buffers dsv_adamw_step
 * takes (same layouts, ownership and NULL rules).  Every element is computed
 * exactly as dsv_adamw_step computes it, so a group and the single calls give
 * bit-identical results.  Returns DSV_ERR_RANGE for n_proj outside
 * [1, DSV_MAX_GROUP], DSV_ERR_ARG for a NULL projs, else as dsv_adamw_step
 * (any bad entry fails the whole call before anything is launched).
 */
typedef struct {
  int32_t K, N;
  const float* dA;        /* [n_ad][r_max][K] */
  const float* dB;        /* [n_ad][N][r_max] */
  float* A_master;        /* [n_ad][r_max][K] fp32 */
  float* B_master;        /* [n_ad][N][r_max] fp32 */
  float* A_m;
  float* A_v;
  float* B_m;
  float* B_v;
  void* A;                /* parameter copy (bf16 or fp32), or NULL */
  void* B;
} dsv_adamw_proj;

int dsv_adamw_step_grouped(const dsv_plan* plan, dsv_dtype dtype, int32_t n_proj,
                           const dsv_adamw_proj* projs, int32_t step, const dsv_adamw_hparams* hp,
                           void* hip_stream);

/* GEMM launch configuration that dsv_cobatch_fwd (pass 0) or dsv_lora_bwd
 * (pass 1, the dX GEMM) uses for this plan, dtype and K x N on the current
 * device, for benchmarks and tests.  out[6] receives: tile rows, tile
 * columns, row tiles, column tiles, the number of tiles split along the
 * contraction and the number of pieces each of them is split into (0 and 0
 * when none is split).  The bf16 path picks, per launch, the tile shape and
 * split with the smallest estimated time; fp32 and empty passes report zeros.
 * Returns DSV_OK, DSV_ERR_ARG (NULL plan or out, pass not 0 or 1) or the
 * dsv_cobatch_fwd size and dtype errors. */
int dsv_gemm_config(const dsv_plan* plan, dsv_dtype dtype, int32_t K, int32_t N, int32_t pass,
                    int32_t out[6]);

/* Static description of a status code. */
const char* dsv_status_string(int status);

#ifdef __cplusplus
}
#endif
#endif /* DSV_H */
