/*
 * CPU oracle for the sparse-weight x dense-activation product of SparseDNN
 * (Wang, "SparseDNN: Fast Sparse Deep Learning Inference on CPUs", arXiv 2101.07948).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or calls this
 * file; only the test suite, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header or table with the GPU library.
 *
 * What it computes, and where the paper defines it:
 *
 *   oracle_spmm_f64  The plain definition of the operator of Sec. 2.2 / Sec. 3.2.2
 *                    (sparse matrix times dense matrix), with the fused element-wise
 *                    epilogue of Sec. 3.1 (layer fusion): for every output element
 *                        C[i][n] = act( sum_p values[p] * B[col_idx[p]][n] + bias[i] )
 *                    summed in double over row i's stored entries in ascending column
 *                    order, bias added in double, activation applied in double.
 *                    Also returns, per element, sum_p |values[p]| * |B[col_idx[p]][n]|
 *                    (the scale of the fp32 rounding bound used by the parity tests).
 *
 *   oracle_spmm_f32  The same definition with a float accumulator and the same loop
 *                    order; it is the CPU baseline that the benchmark times.  No
 *                    blocking, no intrinsics, no BLAS; OpenMP splits rows only.
 *
 *   oracle_conv3x3_f64  The sparse 3x3 convolution of Sec. 3.2.3 (stride 1, zero padding
 *                    of 1, as in the paper's convolution benchmark, Sec. 4.1) by its
 *                    definition: for output channel o, pixel (y, x) and image b,
 *                        C[o][y][x][b] = act( sum over the stored filter taps (i, ky, kx)
 *                            of filter o of  w * X[i][y + ky - 1][x + kx - 1][b]
 *                            (zero outside the image)  + bias[o] )
 *                    in double.  The filters are an OC x (IC * 9) CSR whose column is
 *                    i * 9 + ky * 3 + kx (the paper's OC by IC x Fx x Fy filter matrix);
 *                    activations are IC x H x W x NB (channel, row, column, image).
 *                    Also returns sum |w * x| per output element.
 *
 *   oracle_reorder   The greedy weight-row permutation of Sec. 3.1.2 (Algorithm 1):
 *                    the first row is the one with the most nonzeros, and each next
 *                    row is the remaining row whose nonzero column set overlaps most
 *                    with the previously placed row.  Readings where the paper is
 *                    silent: rows are 0..M-1 and exactly M are placed; ties in the
 *                    first pick go to the lower row index; ties in later picks go to
 *                    the larger nonzero count, then the lower row index; "nonzero"
 *                    means a stored CSR entry.  Column sets are kept as sorted lists
 *                    and overlaps are counted by a two-pointer merge.
 *
 * Activations (epi): 0 none, 1 ReLU = max(x, 0), 2 GELU = x * Phi(x) in its exact
 * erf form 0.5 * x * (1 + erf(x / sqrt(2))) -- the paper names GELU in Sec. 5 and
 * cites Hendrycks & Gimpel for it; the tanh approximation is not used.
 *
 * Input contract (checked by the callers, not here): row_ptr[0] = 0, row_ptr is
 * non-decreasing, row_ptr[M] = nnz, 0 <= col_idx[p] < K, columns strictly
 * increasing within a row, B is K x N row-major, bias is length M or NULL.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double act_f64(double x, int epi) {
  if (epi == 1) return x > 0.0 ? x : 0.0;
  if (epi == 2) return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));
  return x;
}

static float act_f32(float x, int epi) {
  if (epi == 1) return x > 0.0f ? x : 0.0f;
  if (epi == 2) return (float)(0.5 * (double)x * (1.0 + erf((double)x / sqrt(2.0))));
  return x;
}

/* Parity reference.  C_out is M x N doubles (unrounded); bound_out is M x N doubles
 * holding sum_p |w_p * B[c_p][n]| (may be NULL).  Returns 0. */
int oracle_spmm_f64(int32_t M, int32_t K, int32_t N, const int32_t* row_ptr,
                    const int32_t* col_idx, const float* values, const float* B,
                    const float* bias, int32_t epi, double* C_out, double* bound_out) {
  (void)K;
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < M; ++i) {
    double* acc = C_out + (size_t)i * N;
    double* bnd = bound_out ? bound_out + (size_t)i * N : NULL;
    for (int32_t n = 0; n < N; ++n) {
      acc[n] = 0.0;
      if (bnd) bnd[n] = 0.0;
    }
    /* ascending column order: the CSR row is sorted by column */
    for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
      const double w = (double)values[p];
      const float* brow = B + (size_t)col_idx[p] * N;
      for (int32_t n = 0; n < N; ++n) {
        const double t = w * (double)brow[n];
        acc[n] += t;
        if (bnd) bnd[n] += fabs(t);
      }
    }
    const double bi = bias ? (double)bias[i] : 0.0;
    for (int32_t n = 0; n < N; ++n) acc[n] = act_f64(acc[n] + bi, epi);
  }
  return 0;
}

/* Timed CPU baseline: float accumulator, same loop order as the reference. */
int oracle_spmm_f32(int32_t M, int32_t K, int32_t N, const int32_t* row_ptr,
                    const int32_t* col_idx, const float* values, const float* B,
                    const float* bias, int32_t epi, float* C_out) {
  (void)K;
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < M; ++i) {
    float* acc = C_out + (size_t)i * N;
    for (int32_t n = 0; n < N; ++n) acc[n] = 0.0f;
    for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
      const float w = values[p];
      const float* brow = B + (size_t)col_idx[p] * N;
      for (int32_t n = 0; n < N; ++n) acc[n] += w * brow[n];
    }
    const float bi = bias ? bias[i] : 0.0f;
    for (int32_t n = 0; n < N; ++n) acc[n] = act_f32(acc[n] + bi, epi);
  }
  return 0;
}

/* Sparse 3x3 convolution, stride 1, padding 1, by its definition (see the header).
 * X is IC x H x W x NB, C_out and bound_out are OC x H x W x NB doubles.  Returns 0. */
int oracle_conv3x3_f64(int32_t OC, int32_t IC, int32_t H, int32_t W, int32_t NB,
                       const int32_t* row_ptr, const int32_t* col_idx, const float* values,
                       const float* X, const float* bias, int32_t epi, double* C_out,
                       double* bound_out) {
  (void)IC;
  const size_t plane = (size_t)H * W * NB;
#pragma omp parallel for schedule(static)
  for (int32_t o = 0; o < OC; ++o) {
    const double bo = bias ? (double)bias[o] : 0.0;
    for (int32_t y = 0; y < H; ++y)
      for (int32_t x = 0; x < W; ++x)
        for (int32_t b = 0; b < NB; ++b) {
          double acc = 0.0, bnd = 0.0;
          for (int32_t p = row_ptr[o]; p < row_ptr[o + 1]; ++p) {
            const int32_t tap = col_idx[p];
            const int32_t i = tap / 9, ky = (tap % 9) / 3, kx = tap % 3;
            int32_t yy = y + ky - 1, xx = x + kx - 1;
            if (yy < 0 || yy >= H || xx < 0 || xx >= W) continue;
            const double t = (double)values[p] * (double)X[i * plane + ((size_t)yy * W + xx) * NB + b];
            acc += t;
            bnd += fabs(t);
          }
          const size_t at = (size_t)o * plane + ((size_t)y * W + x) * NB + b;
          C_out[at] = act_f64(acc + bo, epi);
          if (bound_out) bound_out[at] = bnd;
        }
  }
  return 0;
}

/* |cols(a) ∩ cols(b)| for two sorted column lists, by a two-pointer merge. */
static int32_t overlap_sorted(const int32_t* a, int32_t na, const int32_t* b, int32_t nb) {
  int32_t i = 0, j = 0, common = 0;
  while (i < na && j < nb) {
    if (a[i] == b[j]) {
      ++common;
      ++i;
      ++j;
    } else if (a[i] < b[j]) {
      ++i;
    } else {
      ++j;
    }
  }
  return common;
}

/* Algorithm 1 (Sec. 3.1.2).  perm_out[i] = original row placed at position i. */
int oracle_reorder(int32_t M, int32_t K, const int32_t* row_ptr, const int32_t* col_idx,
                   int32_t* perm_out) {
  (void)K;
  if (M <= 0) return 0;
  char* remaining = (char*)malloc((size_t)M);
  if (!remaining) return 1;
  memset(remaining, 1, (size_t)M);

  /* first pick: the row with the most nonzeros (lowest index among equals) */
  int32_t first = 0;
  for (int32_t x = 1; x < M; ++x) {
    const int32_t nx = row_ptr[x + 1] - row_ptr[x];
    const int32_t nf = row_ptr[first + 1] - row_ptr[first];
    if (nx > nf) first = x;
  }
  perm_out[0] = first;
  remaining[first] = 0;

  /* each next pick: most overlap with the previously placed row */
  for (int32_t i = 1; i < M; ++i) {
    const int32_t prev = perm_out[i - 1];
    const int32_t* pc = col_idx + row_ptr[prev];
    const int32_t pn = row_ptr[prev + 1] - row_ptr[prev];
    int32_t best = -1, best_ov = -1, best_nnz = -1;
    for (int32_t x = 0; x < M; ++x) {
      if (!remaining[x]) continue;
      const int32_t xn = row_ptr[x + 1] - row_ptr[x];
      const int32_t ov = overlap_sorted(pc, pn, col_idx + row_ptr[x], xn);
      /* scanning x upward, a strict improvement keeps the lowest index on ties */
      if (ov > best_ov || (ov == best_ov && xn > best_nnz)) {
        best = x;
        best_ov = ov;
        best_nnz = xn;
      }
    }
    perm_out[i] = best;
    remaining[best] = 0;
  }
  free(remaining);
  return 0;
}

/* Number of OpenMP threads the two SpMM routines use (for reporting). */
int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Sets the OpenMP thread count of later calls (n >= 1); for timing at chosen counts. */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
