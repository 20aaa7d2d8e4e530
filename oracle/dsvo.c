/*
 * dsvo.c -- fp64 reference ("oracle") of the co-batched multi-LoRA layer.
 *
 * TEST INFRASTRUCTURE ONLY (tests, smoke check, the bench's CPU baseline).
 * Plain loops in double precision, OpenMP over independent output rows only;
 * no blocking, no fusion, no reordering of any sum beyond what the
 * definitions below state.  Every sum over k, n, j or training rows runs in
 * ascending index order.  See dsvo.h for the layouts and the paper passages.
 */
#include "dsvo.h"
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Segment table -> per-row adapter and the ascending list of training rows.
 * The table must tile [0,T): every row is covered exactly once (Sec. 3.2:
 * each batch entry, inference or fine-tuning, is one contiguous run of
 * tokens bound to one adapter). */
int dsvo_rows(int T, int n_seg, const int32_t* seg, int n_ad,
              int32_t* row_adapter, int32_t* train_rows) {
  if (T < 0 || n_seg < 0) return -1;
  char* is_train = (char*)calloc((size_t)T + 1, 1);
  int32_t* seen = (int32_t*)calloc((size_t)T + 1, sizeof(int32_t));
  if (!is_train || !seen) { free(is_train); free(seen); return -1; }
  int bad = 0;
  for (int s = 0; s < n_seg && !bad; ++s) {
    int32_t st = seg[4 * s], len = seg[4 * s + 1], a = seg[4 * s + 2], tr = seg[4 * s + 3];
    if (st < 0 || len < 0 || (int64_t)st + len > T || a < 0 || a >= n_ad) { bad = 1; break; }
    for (int32_t t = st; t < st + len; ++t) {
      seen[t] += 1;
      row_adapter[t] = a;
      is_train[t] = tr != 0;
    }
  }
  for (int t = 0; t < T && !bad; ++t)
    if (seen[t] != 1) bad = 1;
  int tt = 0;
  if (!bad)
    for (int t = 0; t < T; ++t)
      if (is_train[t]) train_rows[tt++] = t;
  free(is_train);
  free(seen);
  return bad ? -1 : tt;
}

/* H = x A_a^T for one token row (Sec. 2.2: the low-rank path first maps the
 * row into the r-dimensional space of adapter a). */
static void shrink_row(int K, int r, int r_max, const double* x, const double* Aa, double* h) {
  for (int j = 0; j < r; ++j) {
    double acc = 0.0;
    for (int k = 0; k < K; ++k) acc += x[k] * Aa[(size_t)j * K + k];
    h[j] = acc;
  }
  (void)r_max;
}

/* The input of the low-rank path of token row t: x itself, or for a training
 * row under dropout x[k] * drop[i][k] (i = compact index of t). */
static void lora_input(int K, const double* x, const double* drop_row, double* out) {
  for (int k = 0; k < K; ++k) out[k] = drop_row ? x[k] * drop_row[k] : x[k];
}

int dsvo_forward(int T, int K, int N, int n_seg, const int32_t* seg,
                 int n_ad, const int32_t* rank, const double* scale, int r_max,
                 const double* X, const double* W, const double* A, const double* B,
                 const double* drop, int n_rows, const int32_t* rows, double* Y, double* H) {
  if (K <= 0 || N <= 0 || r_max <= 0) return -1;
  int32_t* row_adapter = (int32_t*)malloc(sizeof(int32_t) * ((size_t)T + 1));
  int32_t* train_rows = (int32_t*)malloc(sizeof(int32_t) * ((size_t)T + 1));
  if (!row_adapter || !train_rows) { free(row_adapter); free(train_rows); return -1; }
  int tt = dsvo_rows(T, n_seg, seg, n_ad, row_adapter, train_rows);
  int bad = tt < 0;
  for (int i = 0; i < n_rows && !bad; ++i)
    if (rows[i] < 0 || rows[i] >= T) bad = 1;
  for (int a = 0; a < n_ad && !bad; ++a)
    if (rank[a] < 1 || rank[a] > r_max) bad = 1;
  int32_t* compact = NULL;  /* token row -> compact training index, or -1 */
  if (!bad) {
    compact = (int32_t*)malloc(sizeof(int32_t) * ((size_t)T + 1));
    if (!compact) bad = 1;
  }
  if (!bad) {
    for (int t = 0; t < T; ++t) compact[t] = -1;
    for (int i = 0; i < tt; ++i) compact[train_rows[i]] = i;
#pragma omp parallel for schedule(dynamic, 4)
    for (int i = 0; i < n_rows; ++i) {
      const int t = rows[i];
      const int a = row_adapter[t];
      const int r = rank[a];
      const double s = scale[a];
      const double* x = X + (size_t)t * K;
      const double* Aa = A + (size_t)a * r_max * K;
      const double* Ba = B + (size_t)a * N * r_max;
      double* h = H + (size_t)i * r_max;
      double* xl = (double*)malloc(sizeof(double) * (size_t)K);
      lora_input(K, x, (drop && compact[t] >= 0) ? drop + (size_t)compact[t] * K : NULL, xl);
      shrink_row(K, r, r_max, xl, Aa, h);
      free(xl);
      for (int n = 0; n < N; ++n) {
        /* base term: the frozen weight, shared by every row (Sec. 2.2) */
        double base = 0.0;
        const double* wn = W + (size_t)n * K;
        for (int k = 0; k < K; ++k) base += x[k] * wn[k];
        /* low-rank term of the row's own adapter, scaled by s_a */
        double low = 0.0;
        const double* bn = Ba + (size_t)n * r_max;
        for (int j = 0; j < r; ++j) low += h[j] * bn[j];
        Y[(size_t)i * N + n] = base + s * low;
      }
    }
  }
  free(compact);
  free(row_adapter);
  free(train_rows);
  return bad ? -1 : 0;
}

int dsvo_backward(int T, int K, int N, int n_seg, const int32_t* seg,
                  int n_ad, const int32_t* rank, const double* scale, int r_max,
                  const double* X, const double* W, const double* A, const double* B,
                  const double* drop, const double* dY, double* G, double* dA, double* dB,
                  int n_dx, const int32_t* dx_rows, double* dX) {
  if (K <= 0 || N <= 0 || r_max <= 0) return -1;
  int32_t* row_adapter = (int32_t*)malloc(sizeof(int32_t) * ((size_t)T + 1));
  int32_t* train_rows = (int32_t*)malloc(sizeof(int32_t) * ((size_t)T + 1));
  if (!row_adapter || !train_rows) { free(row_adapter); free(train_rows); return -1; }
  const int tt = dsvo_rows(T, n_seg, seg, n_ad, row_adapter, train_rows);
  int bad = tt < 0;
  for (int a = 0; a < n_ad && !bad; ++a)
    if (rank[a] < 1 || rank[a] > r_max) bad = 1;
  for (int m = 0; m < n_dx && !bad; ++m)
    if (dx_rows[m] < 0 || dx_rows[m] >= tt) bad = 1;
  double* Hs = NULL;
  double* XL = NULL;  /* low-rank-path input of every training row */
  char* owns = NULL;
  if (!bad) {
    Hs = (double*)malloc(sizeof(double) * ((size_t)tt * r_max + 1));
    XL = (double*)malloc(sizeof(double) * ((size_t)tt * K + 1));
    owns = (char*)calloc((size_t)n_ad, 1);
    if (!Hs || !XL || !owns) bad = 1;
  }
  if (!bad) {
    for (int i = 0; i < tt; ++i) owns[row_adapter[train_rows[i]]] = 1;

    /* H of every training row, recomputed exactly from its low-rank input. */
#pragma omp parallel for schedule(static)
    for (int i = 0; i < tt; ++i) {
      const int t = train_rows[i], a = row_adapter[t];
      lora_input(K, X + (size_t)t * K, drop ? drop + (size_t)i * K : NULL, XL + (size_t)i * K);
      shrink_row(K, rank[a], r_max, XL + (size_t)i * K, A + (size_t)a * r_max * K,
                 Hs + (size_t)i * r_max);
    }

    /* G[i][j] = s_a * sum_n dY[i][n] B[a][n][j]: the gradient reaching H. */
#pragma omp parallel for schedule(static)
    for (int i = 0; i < tt; ++i) {
      const int a = row_adapter[train_rows[i]], r = rank[a];
      const double* Ba = B + (size_t)a * N * r_max;
      for (int j = 0; j < r; ++j) {
        double acc = 0.0;
        for (int n = 0; n < N; ++n) acc += dY[(size_t)i * N + n] * Ba[(size_t)n * r_max + j];
        G[(size_t)i * r_max + j] = scale[a] * acc;
      }
    }

    /* dB[a][n][j] = s_a * sum_{i of a} H[i][j] dY[i][n]; rows of dB in parallel. */
#pragma omp parallel for schedule(static)
    for (int n = 0; n < N; ++n) {
      for (int a = 0; a < n_ad; ++a) {
        if (!owns[a]) continue;
        const int r = rank[a];
        for (int j = 0; j < r; ++j) {
          double acc = 0.0;
          for (int i = 0; i < tt; ++i) {
            if (row_adapter[train_rows[i]] != a) continue;
            acc += Hs[(size_t)i * r_max + j] * dY[(size_t)i * N + n];
          }
          dB[((size_t)a * N + n) * r_max + j] = scale[a] * acc;
        }
      }
    }

    /* dA[a][j][k] = sum_{i of a} G[i][j] XL[i][k] (XL: the low-rank input of
     * training row i); columns k in parallel. */
#pragma omp parallel for schedule(static)
    for (int k = 0; k < K; ++k) {
      for (int a = 0; a < n_ad; ++a) {
        if (!owns[a]) continue;
        const int r = rank[a];
        for (int j = 0; j < r; ++j) {
          double acc = 0.0;
          for (int i = 0; i < tt; ++i) {
            const int t = train_rows[i];
            if (row_adapter[t] != a) continue;
            acc += G[(size_t)i * r_max + j] * XL[(size_t)i * K + k];
          }
          dA[((size_t)a * r_max + j) * K + k] = acc;
        }
      }
    }

    /* dX[m][k] = sum_n dY[i][n] W[n][k] + sum_j G[i][j] A[a][j][k]. */
#pragma omp parallel for schedule(dynamic, 4)
    for (int m = 0; m < n_dx; ++m) {
      const int i = dx_rows[m];
      const int a = row_adapter[train_rows[i]], r = rank[a];
      const double* Aa = A + (size_t)a * r_max * K;
      for (int k = 0; k < K; ++k) {
        double base = 0.0;
        for (int n = 0; n < N; ++n) base += dY[(size_t)i * N + n] * W[(size_t)n * K + k];
        double low = 0.0;
        for (int j = 0; j < r; ++j) low += G[(size_t)i * r_max + j] * Aa[(size_t)j * K + k];
        if (drop) low *= drop[(size_t)i * K + k];  /* through the fixed mask */
        dX[(size_t)m * K + k] = base + low;
      }
    }
  }
  free(Hs);
  free(XL);
  free(owns);
  free(row_adapter);
  free(train_rows);
  return bad ? -1 : 0;
}

/* Threads the OpenMP loops above run with (1 without OpenMP): reported next to
 * the reference's measured rate. */
int dsvo_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
