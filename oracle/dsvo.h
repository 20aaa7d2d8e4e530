/*
 * dsvo.h -- fp64 reference ("oracle") for the co-batched multi-LoRA linear layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * bench's CPU-baseline leg may load this library.  It shares no code, header,
 * table or helper with the HIP library under paper_2607_28848_amd/.
 *
 * What it computes (DeltaServe, arXiv 2607.28848):
 *   - LoRA (Sec. 2.2, "Parameter-Efficient Fine-Tuning"): a frozen weight
 *     W in R^{d x k} gets a trainable update  dW = B A  with  A in R^{r x k},
 *     B in R^{d x r};  the effective weight is  W + B A.
 *   - Multi-LoRA batching (Sec. 2.2): tokens on different adapters share one
 *     base-model pass and apply adapter-specific low-rank factors.
 *   - Mixed forward batch (Sec. 3.2, "Co-Serving Model"): a fine-tuning sample
 *     is one more segment of the batch, bound to the reserved training adapter;
 *     only its rows keep activations for the backward.
 *   - Backward (Sec. 3.2, "Backward subprocess"): LoRA gradients for the
 *     training rows; the base weight is frozen and gets none.
 *   - Scale: the paper trains with r = 16 and alpha = 32 (Sec. 4.1,
 *     "Fine-tuning Workload"); every adapter here carries its own scale s_a.
 *
 * Storage (row-major, the paper's own orientation, identical to the
 * torch.nn.Linear / PEFT parameter layout; d = N output features,
 * k = K input features):
 *   X [T][K]   W [N][K]   A [n_ad][r_max][K]   B [n_ad][N][r_max]
 * With x a token row, the layer output is  y = x W^T + s_a (x A_a^T) B_a^T.
 *
 * Segment table: n_seg entries of 4 int32 each: {start, len, adapter, is_train}.
 * The segments must tile [0, T) exactly (len 0 allowed).  Training rows are
 * numbered in ascending token-row order; that compact order indexes H_save,
 * dY and dX.
 *
 * All arithmetic is fp64; inputs are the (already dtype-rounded) values
 * widened to double.  Entries of A / B / H at rank index j >= r_a are never
 * read or written.
 */
#ifndef DSVO_H
#define DSVO_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Fills row_adapter[T] (adapter of each token row) and train_rows[] (ascending
 * training rows).  Returns T_t >= 0, or -1 if the table does not tile [0,T)
 * or names an adapter outside [0, n_ad). */
int dsvo_rows(int T, int n_seg, const int32_t* seg, int n_ad,
              int32_t* row_adapter, int32_t* train_rows);

/* Forward for the token rows listed in rows[0..n_rows):
 *   H[i][j] = sum_k X[t][k] A[a][j][k]                       (j < r_a)
 *   Y[i][n] = sum_k X[t][k] W[n][k] + s_a sum_j H[i][j] B[a][n][j]
 * with t = rows[i], a = adapter of row t.  Y is [n_rows][N], H [n_rows][r_max].
 * LoRA dropout (Sec. 4.1 trains with dropout 0.05 on the adapter input): when
 * drop is not NULL it holds [T_t][K] multipliers (the kept-element mask times
 * 1 / (1 - p), compact training order) and a training row's low-rank path
 * reads x[k] * drop[i][k] instead of x[k]; the base path and inference rows
 * are unchanged.  Returns 0, or -1 on an invalid table / row. */
int dsvo_forward(int T, int K, int N, int n_seg, const int32_t* seg,
                 int n_ad, const int32_t* rank, const double* scale, int r_max,
                 const double* X, const double* W, const double* A, const double* B,
                 const double* drop, int n_rows, const int32_t* rows, double* Y, double* H);

/* Backward for the training rows (compact index i, token row t = train_rows[i]):
 *   G[i][j]    = s_a sum_n dY[i][n] B[a][n][j]
 *   dB[a][n][j] = s_a sum_{i of a} H[i][j] dY[i][n]      (H recomputed exactly)
 *   dA[a][j][k] = sum_{i of a} G[i][j] X[t][k]
 *   dX[m][k]   = sum_n dY[i][n] W[n][k] + sum_j G[i][j] A[a][j][k],  i = dx_rows[m]
 * With drop (see dsvo_forward) X[t][k] in H and dA reads X[t][k] drop[i][k],
 * and the low-rank term of dX[m][k] is multiplied by drop[i][k] (the chain
 * rule through the fixed mask).
 * These are the exact gradients of L = sum_i <dY[i], Y[t]>.  dA and dB slices
 * of adapters that own training rows are overwritten; other slices are left
 * untouched.  G is [T_t][r_max], dX [n_dx][K].  Returns 0 or -1. */
int dsvo_backward(int T, int K, int N, int n_seg, const int32_t* seg,
                  int n_ad, const int32_t* rank, const double* scale, int r_max,
                  const double* X, const double* W, const double* A, const double* B,
                  const double* drop, const double* dY, double* G, double* dA, double* dB,
                  int n_dx, const int32_t* dx_rows, double* dX);

/* OpenMP threads of the loops above (1 without OpenMP). */
int dsvo_threads(void);

#ifdef __cplusplus
}
#endif
#endif
