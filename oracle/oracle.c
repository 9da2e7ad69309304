/*
 * CPU oracle for the SpMM hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may call this code.  The GPU library never links it, and this file shares
 * no header, helper, table or constant with the GPU library.
 *
 * Everything here is a plain, slow, sequential-per-row definition:
 *
 *   SpMM (Sec. "Sparse Matrix Operators on GPUs": C = A B, each nonzero of A
 *   drives one multiply-add per column of B):
 *     C64[i][j] = sum_{p = rowptr[i]}^{rowptr[i+1]-1} (double)val[p] * (double)B[col[p]][j]
 *     S[i][j]   = sum_p |val[p]| * |B[col[p]][j]|
 *   summed left to right in CSR order in fp64.  An fp32 x fp32 product is exact
 *   in fp64 (24 + 24 significand bits <= 53), so only the additions round.
 *   Rows are independent, so the OpenMP split over rows does not change any
 *   bit of the result.
 *
 *   Representations (Sec. "Structural Features and Overhead Modeling",
 *   Eq. format-expansion; Appendix "Compilation-Plan Design Space"):
 *     BSR(b): block-row floor(i/b), block-column floor(k/b); occupied blocks
 *       sorted by block-column within a block-row; values b*b row-major
 *       within a block, absent entries +0.0f.
 *     Blocked-ELL(b): BSR padded to W = max blocks per block-row; padding
 *       blocks have column -1 and zero values.
 *     Transpose: counting sort by column, entries of a transposed row in
 *       ascending original row order, values copied bitwise.
 *     ELL: rows padded to W = max row length, row-major, padding column -1
 *       and value +0.0f.
 *     SELL-C-sigma: rows sorted by non-increasing length within windows of
 *       sigma rows (stable), slices of C sorted rows, row-major within a
 *       slice, each row padded to the slice's longest (column -1, +0.0f).
 *     Column windows: over the heavy-split layout, windows of R light rows
 *       (in list order); per window its staged columns (used by >= 2 of its
 *       rows, at most `cap`, the most used kept) ascending; a code per entry,
 *       -2 - p (staged position p) or the column itself.
 *
 *   Schedules (Appendix "Case Studies", SpMM web-graph case; merge-path
 *   decomposition of Merrill and Garland cited in the background section):
 *     heavy split (T, c): rows with r_i < T are light (ascending order); a row
 *       with r_i >= T is cut into ceil(r_i / c) chunks [begin, min(begin+c, end)).
 *       The library may process the light rows in another order (by last
 *       column, oracle_light_by_last_col) and the chunks in another order (by
 *       middle column, oracle_chunks_by_mid_col); the set and the chunks are
 *       the same.
 *     merge-path split (U units): the merge of the row-end list rowptr[1..m]
 *       with the nonzero indices 0..nnz-1 is walked one step at a time; a row
 *       end is taken before the nonzero index equal to it.  With
 *       L = ceil((m + nnz) / U), unit u starts at path position
 *       min(u*L, m + nnz), recorded as (rows consumed, nonzeros consumed).
 *
 *   Structural statistics (Sec. "Structural Features and Overhead Modeling"):
 *     integer counts, and fp64 fields computed from exact integer sums by one
 *     fixed formula each, listed at oracle_stats.
 *
 * The row-length shape class follows a reading of the paper, which names the
 * classes without thresholds; the thresholds are stated at oracle_stats.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- SpMM --- */

static void spmm_row(const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t n,
                     const float *B, int32_t i, double *c, double *s) {
  for (int32_t j = 0; j < n; ++j) {
    c[j] = 0.0;
    s[j] = 0.0;
  }
  for (int32_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
    const double a = (double)vals[p];
    const float *brow = B + (int64_t)colidx[p] * n;
    for (int32_t j = 0; j < n; ++j) {
      c[j] += a * (double)brow[j];
      s[j] += fabs(a) * fabs((double)brow[j]);
    }
  }
}

/* C64, S: m x n row-major (S may be NULL). */
void oracle_spmm_csr(int32_t m, int32_t k, const int32_t *rowptr, const int32_t *colidx,
                     const float *vals, int32_t n, const float *B, double *C64, double *S) {
  (void)k;
#pragma omp parallel
  {
    double *tmp = S ? NULL : (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
#pragma omp for schedule(dynamic, 64)
    for (int32_t i = 0; i < m; ++i)
      spmm_row(rowptr, colidx, vals, n, B, i, C64 + (int64_t)i * n, S ? S + (int64_t)i * n : tmp);
    free(tmp);
  }
}

/* Selected rows only: row rows[t] of the product goes to C64[t][*], S[t][*]. */
void oracle_spmm_csr_rows(const int32_t *rows, int64_t nrows, const int32_t *rowptr, const int32_t *colidx,
                          const float *vals, int32_t n, const float *B, double *C64, double *S) {
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t t = 0; t < nrows; ++t)
    spmm_row(rowptr, colidx, vals, n, B, rows[t], C64 + t * n, S + t * n);
}

/* C = A^T B computed as a scatter over A's rows in ascending row order:
 * C[col[p]][*] += val[p] * B[i][*].  For each output row the terms arrive in
 * ascending i, the same order as a CSR walk of the transposed matrix.
 * C64, S: k x n, B: m x n.  Sequential (the scatter has write conflicts). */
void oracle_spmm_csr_transposed(int32_t m, int32_t k, const int32_t *rowptr, const int32_t *colidx,
                                const float *vals, int32_t n, const float *B, double *C64, double *S) {
  memset(C64, 0, sizeof(double) * (size_t)k * (size_t)n);
  memset(S, 0, sizeof(double) * (size_t)k * (size_t)n);
  for (int32_t i = 0; i < m; ++i)
    for (int32_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
      const double a = (double)vals[p];
      double *c = C64 + (int64_t)colidx[p] * n;
      double *s = S + (int64_t)colidx[p] * n;
      const float *brow = B + (int64_t)i * n;
      for (int32_t j = 0; j < n; ++j) {
        c[j] += a * (double)brow[j];
        s[j] += fabs(a) * fabs((double)brow[j]);
      }
    }
}

/* Block SpMM: for each row of a block-row, blocks in stored order
 * (ascending block-column), then in-block columns ascending; every stored
 * slot (including the zero fill) is a term.  Columns >= k (the padding of
 * the last block-column) are skipped.  bptr == NULL means Blocked-ELL with
 * `width` slots per block-row and column -1 marking padding.  C64, S: m x n. */
void oracle_spmm_blocks(int32_t m, int32_t k, int32_t b, const int32_t *bptr, int32_t width,
                        const int32_t *bcol, const float *bval, int32_t n, const float *B, double *C64,
                        double *S) {
  const int32_t mb = (m + b - 1) / b;
#pragma omp parallel for schedule(dynamic, 4)
  for (int32_t br = 0; br < mb; ++br) {
    int64_t q0 = bptr ? bptr[br] : (int64_t)br * width;
    int64_t q1 = bptr ? bptr[br + 1] : (int64_t)(br + 1) * width;
    for (int32_t rr = 0; rr < b; ++rr) {
      int32_t i = br * b + rr;
      if (i >= m) break;
      double *c = C64 + (int64_t)i * n;
      double *s = S + (int64_t)i * n;
      for (int32_t j = 0; j < n; ++j) {
        c[j] = 0.0;
        s[j] = 0.0;
      }
      for (int64_t q = q0; q < q1; ++q) {
        if (bcol[q] < 0) continue;
        for (int32_t cc = 0; cc < b; ++cc) {
          int64_t kk = (int64_t)bcol[q] * b + cc;
          if (kk >= k) break;
          const double a = (double)bval[(q * b + rr) * b + cc];
          const float *brow = B + kk * n;
          for (int32_t j = 0; j < n; ++j) {
            c[j] += a * (double)brow[j];
            s[j] += fabs(a) * fabs((double)brow[j]);
          }
        }
      }
    }
  }
}

/* ----------------------------------------------------------- Transpose --- */

/* trowptr: k+1, tcolidx/tvals: nnz. */
void oracle_transpose(int32_t m, int32_t k, const int32_t *rowptr, const int32_t *colidx, const float *vals,
                      int32_t *trowptr, int32_t *tcolidx, float *tvals) {
  for (int32_t j = 0; j <= k; ++j) trowptr[j] = 0;
  for (int32_t p = 0; p < rowptr[m]; ++p) trowptr[colidx[p] + 1]++;
  for (int32_t j = 0; j < k; ++j) trowptr[j + 1] += trowptr[j];
  int32_t *next = (int32_t *)malloc(sizeof(int32_t) * (size_t)(k > 0 ? k : 1));
  for (int32_t j = 0; j < k; ++j) next[j] = trowptr[j];
  for (int32_t i = 0; i < m; ++i)
    for (int32_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
      int32_t q = next[colidx[p]]++;
      tcolidx[q] = i;
      memcpy(&tvals[q], &vals[p], sizeof(float));
    }
  free(next);
}

/* --------------------------------------------------------------- Blocks --- */

static int cmp_i32(const void *a, const void *b) {
  int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return (x > y) - (x < y);
}

/* Sorted distinct block-columns of block-row br into out (returns count).
 * scratch must hold every nonzero of the block-row. */
static int32_t block_cols(int32_t m, const int32_t *rowptr, const int32_t *colidx, int32_t b, int32_t br,
                          int32_t *scratch) {
  int32_t r0 = br * b, r1 = r0 + b < m ? r0 + b : m;
  int32_t cnt = 0;
  for (int32_t p = rowptr[r0]; p < rowptr[r1]; ++p) scratch[cnt++] = colidx[p] / b;
  qsort(scratch, (size_t)cnt, sizeof(int32_t), cmp_i32);
  int32_t w = 0;
  for (int32_t q = 0; q < cnt; ++q)
    if (w == 0 || scratch[w - 1] != scratch[q]) scratch[w++] = scratch[q];
  return w;
}

static int32_t max_block_row_nnz(int32_t m, const int32_t *rowptr, int32_t b) {
  int32_t best = 1;
  for (int32_t r0 = 0; r0 < m; r0 += b) {
    int32_t r1 = r0 + b < m ? r0 + b : m;
    if (rowptr[r1] - rowptr[r0] > best) best = rowptr[r1] - rowptr[r0];
  }
  return best;
}

/* Occupied-block count per block-row into counts[mb] (may be NULL);
 * returns the total. */
int64_t oracle_block_counts(int32_t m, const int32_t *rowptr, const int32_t *colidx, int32_t b, int32_t *counts) {
  const int32_t mb = (m + b - 1) / b;
  int32_t *scratch = (int32_t *)malloc(sizeof(int32_t) * (size_t)max_block_row_nnz(m, rowptr, b));
  int64_t total = 0;
  for (int32_t br = 0; br < mb; ++br) {
    int32_t w = block_cols(m, rowptr, colidx, b, br, scratch);
    if (counts) counts[br] = w;
    total += w;
  }
  free(scratch);
  return total;
}

/* BSR: bptr[mb+1], bcol[nnzb], bval[nnzb*b*b]. */
void oracle_to_bsr(int32_t m, const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t b,
                   int32_t *bptr, int32_t *bcol, float *bval) {
  const int32_t mb = (m + b - 1) / b;
  int32_t *scratch = (int32_t *)malloc(sizeof(int32_t) * (size_t)max_block_row_nnz(m, rowptr, b));
  int64_t q0 = 0;
  for (int32_t br = 0; br < mb; ++br) {
    bptr[br] = (int32_t)q0;
    int32_t w = block_cols(m, rowptr, colidx, b, br, scratch);
    for (int32_t t = 0; t < w; ++t) bcol[q0 + t] = scratch[t];
    memset(bval + q0 * b * b, 0, sizeof(float) * (size_t)w * b * b);
    for (int32_t i = br * b; i < m && i < (br + 1) * b; ++i)
      for (int32_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
        int32_t bc = colidx[p] / b;
        int32_t t = 0;
        while (scratch[t] != bc) ++t; /* linear search: plain, not fast */
        memcpy(&bval[((q0 + t) * b + (i - br * b)) * b + colidx[p] % b], &vals[p], sizeof(float));
      }
    q0 += w;
  }
  bptr[mb] = (int32_t)q0;
  free(scratch);
}

/* Blocked-ELL: width = max blocks per block-row; bcol[mb*width] (-1 pad),
 * bval[mb*width*b*b]. */
void oracle_to_bell(int32_t m, const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t b,
                    int32_t width, int32_t *bcol, float *bval) {
  const int32_t mb = (m + b - 1) / b;
  int32_t *scratch = (int32_t *)malloc(sizeof(int32_t) * (size_t)max_block_row_nnz(m, rowptr, b));
  memset(bval, 0, sizeof(float) * (size_t)mb * width * b * b);
  for (int32_t br = 0; br < mb; ++br) {
    int64_t q0 = (int64_t)br * width;
    int32_t w = block_cols(m, rowptr, colidx, b, br, scratch);
    for (int32_t t = 0; t < width; ++t) bcol[q0 + t] = t < w ? scratch[t] : -1;
    for (int32_t i = br * b; i < m && i < (br + 1) * b; ++i)
      for (int32_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
        int32_t bc = colidx[p] / b;
        int32_t t = 0;
        while (scratch[t] != bc) ++t;
        memcpy(&bval[((q0 + t) * b + (i - br * b)) * b + colidx[p] % b], &vals[p], sizeof(float));
      }
  }
  free(scratch);
}

/* ------------------------------------------------------------------ ELL --- */

/* ELL (Sec. "Structural Features and Overhead Modeling", rho_ELL; Appendix
 * "Case Studies", SpMV uniform-row case): every row padded to width W =
 * max r_i, row-major [m][W]; row i's entries in CSR order, then column -1 and
 * value +0.0f. */
void oracle_to_ell(int32_t m, const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t width,
                   int32_t *ecol, float *eval) {
  for (int32_t i = 0; i < m; ++i) {
    int32_t r = rowptr[i + 1] - rowptr[i];
    for (int32_t t = 0; t < width; ++t) {
      int64_t q = (int64_t)i * width + t;
      if (t < r) {
        ecol[q] = colidx[rowptr[i] + t];
        memcpy(&eval[q], &vals[rowptr[i] + t], sizeof(float));
      } else {
        ecol[q] = -1;
        eval[q] = 0.0f;
      }
    }
  }
}

/* ELL SpMM: slots in order, padding (column -1) skipped.  C64, S: m x n. */
void oracle_spmm_ell(int32_t m, int32_t width, const int32_t *ecol, const float *eval, int32_t n, const float *B,
                     double *C64, double *S) {
#pragma omp parallel for schedule(dynamic, 64)
  for (int32_t i = 0; i < m; ++i) {
    double *c = C64 + (int64_t)i * n;
    double *s = S + (int64_t)i * n;
    for (int32_t j = 0; j < n; ++j) {
      c[j] = 0.0;
      s[j] = 0.0;
    }
    for (int32_t t = 0; t < width; ++t) {
      int64_t q = (int64_t)i * width + t;
      if (ecol[q] < 0) continue;
      const double a = (double)eval[q];
      const float *brow = B + (int64_t)ecol[q] * n;
      for (int32_t j = 0; j < n; ++j) {
        c[j] += a * (double)brow[j];
        s[j] += fabs(a) * fabs((double)brow[j]);
      }
    }
  }
}

/* ------------------------------------------------------ Column windows --- */

/* Packed column windows (Sec. "Agentic Lowering and Refinement": the
 * mechanism library's packed column windows for SpMM, after Sextans; Appendix
 * "Compilation-Plan Design Space", SpMM row: window descriptors, B staged in
 * shared memory, C held in registers), over the heavy-split layout
 * (oracle_split_layout): heavy rows
 * keep their chunks, and the light rows, in list order, are cut into windows
 * of R consecutive list positions.
 *
 * A window's staged columns are those that two or more of its light rows
 * use.  When more than `cap` columns qualify, the `cap` most used are kept,
 * ties to the smaller column.  They are stored ascending:
 * win_ptr[w] .. win_ptr[w+1] indexes window w's in win_cols.  code[] runs
 * parallel to the layout's colidx: an entry of a light row in window w whose
 * column is staged at position p holds -2 - p; every other entry (heavy rows
 * included) holds its column.  Returns the total number of staged columns
 * (call with win_cols == NULL to size; win_ptr and code may be NULL then). */
typedef struct {
  int32_t col, uses;
} oracle_col_use;

static int cmp_more_uses(const void *a, const void *b) {
  const oracle_col_use *x = (const oracle_col_use *)a, *y = (const oracle_col_use *)b;
  if (x->uses != y->uses) return x->uses > y->uses ? -1 : 1;
  return (x->col > y->col) - (x->col < y->col);
}

int64_t oracle_split_windows(int64_t n_light, const int32_t *lptr, const int32_t *colidx, int64_t nnz, int32_t R,
                             int32_t cap, int32_t *win_ptr, int32_t *win_cols, int32_t *code) {
  const int64_t nw = (n_light + R - 1) / R;
  int64_t total = 0, widest = 1;
  for (int64_t w = 0; w < nw; ++w) {
    const int64_t t1 = (w + 1) * R < n_light ? (w + 1) * R : n_light;
    if (lptr[t1] - lptr[w * R] > widest) widest = lptr[t1] - lptr[w * R];
  }
  int32_t *cols = (int32_t *)malloc(sizeof(int32_t) * (size_t)widest);
  oracle_col_use *cand = (oracle_col_use *)malloc(sizeof(oracle_col_use) * (size_t)widest);
  int32_t *staged = (int32_t *)malloc(sizeof(int32_t) * (size_t)widest);
  for (int64_t w = 0; w < nw; ++w) {
    const int64_t t0 = w * R, t1 = (w + 1) * R < n_light ? (w + 1) * R : n_light;
    const int64_t p0 = lptr[t0], p1 = lptr[t1];
    int32_t cnt = 0, nc = 0;
    for (int64_t p = p0; p < p1; ++p) cols[cnt++] = colidx[p];
    qsort(cols, (size_t)cnt, sizeof(int32_t), cmp_i32);
    /* a run of equal columns in the sorted list counts the rows that use it */
    for (int32_t q = 0; q < cnt;) {
      int32_t e = q;
      while (e < cnt && cols[e] == cols[q]) ++e;
      if (e - q >= 2) {
        cand[nc].col = cols[q];
        cand[nc].uses = e - q;
        ++nc;
      }
      q = e;
    }
    if (nc > cap) {
      qsort(cand, (size_t)nc, sizeof(oracle_col_use), cmp_more_uses);
      nc = cap;
    }
    for (int32_t q = 0; q < nc; ++q) staged[q] = cand[q].col;
    qsort(staged, (size_t)nc, sizeof(int32_t), cmp_i32);
    if (win_ptr) win_ptr[w] = (int32_t)total;
    if (win_cols) {
      for (int32_t q = 0; q < nc; ++q) win_cols[total + q] = staged[q];
      for (int64_t p = p0; p < p1; ++p) {
        int32_t pos = -1;
        for (int32_t q = 0; q < nc; ++q) /* linear search: plain, not fast */
          if (staged[q] == colidx[p]) pos = q;
        code[p] = pos >= 0 ? -2 - pos : colidx[p];
      }
    }
    total += nc;
  }
  if (win_ptr) win_ptr[nw] = (int32_t)total;
  if (code)
    for (int64_t p = n_light > 0 ? lptr[n_light] : 0; p < nnz; ++p) code[p] = colidx[p];
  free(cols);
  free(cand);
  free(staged);
  return total;
}

/* SpMM over the windowed split layout: light row light[t] sums its entries
 * [lptr[t], lptr[t+1]); a heavy row sums its chunks' entries (consecutive in
 * the layout and in the chunk list).  An entry reads B[c] for a code c >= 0
 * and column win_cols[win_ptr[t / R] + p] for a code -2 - p.  Each row is
 * summed left to right in its CSR order. */
void oracle_spmm_split_windows(int32_t m, int64_t n_light, const int32_t *light, const int32_t *lptr,
                               int64_t n_chunks, const int32_t *chunks, const int32_t *code, const float *vals,
                               int32_t R, const int32_t *win_ptr, const int32_t *win_cols, int32_t n, const float *B,
                               double *C64, double *S) {
  /* per row: its entry range in the layout and its window (-1: heavy) */
  int64_t *rb = (int64_t *)malloc(sizeof(int64_t) * (size_t)(m > 0 ? m : 1));
  int64_t *re = (int64_t *)malloc(sizeof(int64_t) * (size_t)(m > 0 ? m : 1));
  int64_t *rw = (int64_t *)malloc(sizeof(int64_t) * (size_t)(m > 0 ? m : 1));
  for (int32_t i = 0; i < m; ++i) rb[i] = re[i] = 0, rw[i] = -1;
  for (int64_t t = 0; t < n_light; ++t) {
    rb[light[t]] = lptr[t];
    re[light[t]] = lptr[t + 1];
    rw[light[t]] = t / R;
  }
  for (int64_t q = 0; q < n_chunks; ++q) {
    const int32_t r = chunks[3 * q];
    if (q == 0 || chunks[3 * (q - 1)] != r) rb[r] = chunks[3 * q + 1];
    re[r] = chunks[3 * q + 2];
  }
#pragma omp parallel for schedule(dynamic, 64)
  for (int32_t i = 0; i < m; ++i) {
    double *c = C64 + (int64_t)i * n;
    double *s = S + (int64_t)i * n;
    for (int32_t j = 0; j < n; ++j) {
      c[j] = 0.0;
      s[j] = 0.0;
    }
    for (int64_t p = rb[i]; p < re[i]; ++p) {
      const int32_t cd = code[p];
      const int32_t col = cd >= 0 ? cd : win_cols[win_ptr[rw[i]] + (-2 - cd)];
      const double a = (double)vals[p];
      const float *brow = B + (int64_t)col * n;
      for (int32_t j = 0; j < n; ++j) {
        c[j] += a * (double)brow[j];
        s[j] += fabs(a) * fabs((double)brow[j]);
      }
    }
  }
  free(rb);
  free(re);
  free(rw);
}

/* ------------------------------------------------------------ SELL-C-sigma --- */

/* SELL-C-sigma (Appendix "Compilation-Plan Design Space", SpMV row: sliced ELL
 * with slice height C and sort window sigma).  Rows are sorted by
 * non-increasing length inside consecutive windows of sigma rows (stable:
 * equal lengths keep their order); perm[i] is the original row at sorted
 * position i.  Sorted rows are cut into slices of C; slice s holds its rows
 * row-major, each padded to the slice's longest row (column -1, value +0.0f),
 * starting at slice_ptr[s].  Returns the total number of slots (call with
 * col == NULL to size; perm and slice_ptr are always filled). */
typedef struct {
  int32_t len, row;
} len_row_t;

static int cmp_len_desc(const void *a, const void *b) {
  const len_row_t *x = (const len_row_t *)a, *y = (const len_row_t *)b;
  if (x->len != y->len) return x->len > y->len ? -1 : 1;
  return (x->row > y->row) - (x->row < y->row); /* stable: original order among equals */
}

int64_t oracle_to_sell(int32_t m, const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t C,
                       int32_t sigma, int32_t *perm, int64_t *slice_ptr, int32_t *col, float *val) {
  len_row_t *w = (len_row_t *)malloc(sizeof(len_row_t) * (size_t)(sigma > 0 ? sigma : 1));
  for (int32_t b = 0; b < m; b += sigma) {
    const int32_t e = b + sigma < m ? b + sigma : m;
    for (int32_t i = b; i < e; ++i) {
      w[i - b].len = rowptr[i + 1] - rowptr[i];
      w[i - b].row = i;
    }
    qsort(w, (size_t)(e - b), sizeof(len_row_t), cmp_len_desc);
    for (int32_t i = b; i < e; ++i) perm[i] = w[i - b].row;
  }
  free(w);
  const int32_t ns = (m + C - 1) / C;
  int64_t total = 0;
  for (int32_t sl = 0; sl < ns; ++sl) {
    const int32_t r0 = sl * C, r1 = r0 + C < m ? r0 + C : m;
    int32_t width = 0;
    for (int32_t i = r0; i < r1; ++i) {
      const int32_t len = rowptr[perm[i] + 1] - rowptr[perm[i]];
      if (len > width) width = len;
    }
    slice_ptr[sl] = total;
    if (col) {
      for (int32_t i = r0; i < r1; ++i) {
        const int32_t r = perm[i], len = rowptr[r + 1] - rowptr[r];
        for (int32_t t = 0; t < width; ++t) {
          const int64_t slot = total + (int64_t)(i - r0) * width + t;
          if (t < len) {
            col[slot] = colidx[rowptr[r] + t];
            memcpy(&val[slot], &vals[rowptr[r] + t], sizeof(float));
          } else {
            col[slot] = -1;
            val[slot] = 0.0f;
          }
        }
      }
    }
    total += (int64_t)(r1 - r0) * width;
  }
  slice_ptr[ns] = total;
  return total;
}

/* SELL SpMM: sorted row i of slice s writes C row perm[i]. */
void oracle_spmm_sell(int32_t m, int32_t C, const int32_t *perm, const int64_t *slice_ptr, const int32_t *col,
                      const float *val, int32_t n, const float *B, double *C64, double *S) {
#pragma omp parallel for schedule(dynamic, 64)
  for (int32_t i = 0; i < m; ++i) {
    const int32_t sl = i / C, r0 = sl * C, r1 = r0 + C < m ? r0 + C : m;
    const int64_t width = (slice_ptr[sl + 1] - slice_ptr[sl]) / (r1 - r0);
    double *c = C64 + (int64_t)perm[i] * n;
    double *s = S + (int64_t)perm[i] * n;
    for (int32_t j = 0; j < n; ++j) {
      c[j] = 0.0;
      s[j] = 0.0;
    }
    for (int64_t t = 0; t < width; ++t) {
      const int64_t slot = slice_ptr[sl] + (int64_t)(i - r0) * width + t;
      if (col[slot] < 0) continue;
      const double a = (double)val[slot];
      const float *brow = B + (int64_t)col[slot] * n;
      for (int32_t j = 0; j < n; ++j) {
        c[j] += a * (double)brow[j];
        s[j] += fabs(a) * fabs((double)brow[j]);
      }
    }
  }
}

/* ------------------------------------------------------------ Schedules --- */

/* Heavy-row split.  light (may be NULL): light row ids; chunks (may be
 * NULL): (row, begin, end) triples.  counts[0] = #light, counts[1] = #chunks. */
void oracle_heavy_split(int32_t m, const int32_t *rowptr, int32_t T, int32_t c, int32_t *light, int32_t *chunks,
                        int64_t *counts) {
  int64_t nl = 0, nc = 0;
  for (int32_t i = 0; i < m; ++i) {
    int32_t r = rowptr[i + 1] - rowptr[i];
    if (r < T) {
      if (light) light[nl] = i;
      ++nl;
    } else {
      for (int32_t begin = rowptr[i]; begin < rowptr[i + 1]; begin += c) {
        if (chunks) {
          chunks[3 * nc + 0] = i;
          chunks[3 * nc + 1] = begin;
          chunks[3 * nc + 2] = (rowptr[i + 1] - begin < c) ? rowptr[i + 1] : begin + c;
        }
        ++nc;
      }
    }
  }
  counts[0] = nl;
  counts[1] = nc;
}

/* Light-row order "by last column": the light rows (given ascending) sorted
 * by the column of their last nonzero, ties by row; an empty row's key is k
 * (it goes last).  A schedule choice of this library, not of the paper: rows
 * whose largest columns are equal run together. */
typedef struct {
  int32_t key, row;
} oracle_keyed_row;

static int cmp_keyed_row(const void *a, const void *b) {
  const oracle_keyed_row *x = (const oracle_keyed_row *)a, *y = (const oracle_keyed_row *)b;
  if (x->key != y->key) return x->key < y->key ? -1 : 1;
  return (x->row > y->row) - (x->row < y->row);
}

void oracle_light_by_last_col(int32_t k, const int32_t *rowptr, const int32_t *colidx, int64_t n_light,
                              const int32_t *light_in, int32_t *light_out) {
  oracle_keyed_row *t = (oracle_keyed_row *)malloc(sizeof(oracle_keyed_row) * (size_t)(n_light > 0 ? n_light : 1));
  for (int64_t i = 0; i < n_light; ++i) {
    const int32_t r = light_in[i];
    t[i].row = r;
    t[i].key = rowptr[r + 1] > rowptr[r] ? colidx[rowptr[r + 1] - 1] : k;
  }
  qsort(t, (size_t)n_light, sizeof(oracle_keyed_row), cmp_keyed_row);
  for (int64_t i = 0; i < n_light; ++i) light_out[i] = t[i].row;
  free(t);
}

/* Chunk processing order "by middle column": the chunks (row, begin, end)
 * of the split layout (colidx in its coordinates) sorted by the column of
 * the entry at position floor((begin + end) / 2), ties by chunk index.  A
 * schedule choice of this library, not of the paper: chunks of different
 * heavy rows that cover the same region of columns run together.  The chunk
 * list itself (and so the order of partial sums per row) is unchanged. */
void oracle_chunks_by_mid_col(const int32_t *colidx, int64_t n_chunks, const int32_t *chunks, int32_t *order) {
  oracle_keyed_row *t = (oracle_keyed_row *)malloc(sizeof(oracle_keyed_row) * (size_t)(n_chunks > 0 ? n_chunks : 1));
  for (int64_t q = 0; q < n_chunks; ++q) {
    const int64_t b = chunks[3 * q + 1], e = chunks[3 * q + 2];
    t[q].row = (int32_t)q;
    t[q].key = colidx[(b + e) / 2];
  }
  qsort(t, (size_t)n_chunks, sizeof(oracle_keyed_row), cmp_keyed_row);
  for (int64_t q = 0; q < n_chunks; ++q) order[q] = t[q].row;
  free(t);
}

/* Split layout: the entries of the light rows, in the order of `light`,
 * followed by those of the heavy rows (r >= T) in ascending row order.
 * lptr (n_light + 1): light row i of the list spans [lptr[i], lptr[i+1]);
 * chunks (row, begin, end) cut each heavy row into pieces of at most c
 * nonzeros, in the new coordinates.  out_colidx / out_vals hold rowptr[m]. */
void oracle_split_layout(int32_t m, const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t T,
                         int32_t c, int64_t n_light, const int32_t *light, int32_t *lptr, int32_t *out_colidx,
                         float *out_vals, int32_t *chunks) {
  int64_t pos = 0, nc = 0;
  for (int64_t i = 0; i < n_light; ++i) {
    const int32_t r = light[i];
    lptr[i] = (int32_t)pos;
    for (int32_t p = rowptr[r]; p < rowptr[r + 1]; ++p, ++pos) {
      out_colidx[pos] = colidx[p];
      out_vals[pos] = vals[p];
    }
  }
  lptr[n_light] = (int32_t)pos;
  for (int32_t r = 0; r < m; ++r) {
    if (rowptr[r + 1] - rowptr[r] < T) continue;
    const int64_t start = pos;
    for (int32_t p = rowptr[r]; p < rowptr[r + 1]; ++p, ++pos) {
      out_colidx[pos] = colidx[p];
      out_vals[pos] = vals[p];
    }
    for (int64_t b = start; b < pos; b += c) {
      chunks[3 * nc + 0] = r;
      chunks[3 * nc + 1] = (int32_t)b;
      chunks[3 * nc + 2] = (int32_t)(pos - b < c ? pos : b + c);
      ++nc;
    }
  }
}

/* Merge-path split by an explicit walk of the merged path.
 * coords: 2*(U+1) int32, pairs (rows consumed, nonzeros consumed). */
void oracle_merge_split(int32_t m, const int32_t *rowptr, int32_t U, int32_t *coords) {
  const int64_t nnz = rowptr[m];
  const int64_t total = (int64_t)m + nnz;
  int64_t L = (total + U - 1) / U;
  if (L < 1) L = 1;
  int64_t i = 0, j = 0;
  int32_t u = 0;
  for (int64_t d = 0;; ++d) {
    while (u <= U && (int64_t)u * L <= d) {
      /* every unit whose start position is d (positions past the end clamp to it) */
      coords[2 * u] = (int32_t)i;
      coords[2 * u + 1] = (int32_t)j;
      ++u;
    }
    if (d == total) break;
    if (i < m && rowptr[i + 1] <= j)
      ++i; /* row i has no nonzero left: take its end first */
    else
      ++j;
  }
  for (; u <= U; ++u) {
    coords[2 * u] = m;
    coords[2 * u + 1] = (int32_t)nnz;
  }
}

/* ----------------------------------------------------------- Statistics --- */

/*
 * ints[]:  0 m, 1 k, 2 nnz, 3 row_min, 4 row_max, 5 row_q25, 6 row_q50,
 *          7 row_q75, 8 empty_rows, 9 col_deg_max, 10 row_span_median,
 *          11 diag_nnz, 12 nnzb4, 13 nnzb8, 14 nnzb16, 15 dense_tiles16,
 *          16 dense_tile_nnz16, 17 bell16_width, 18 sell16_slots,
 *          19 sell32_slots, 20 sell512_slots, 21 shape_class
 * reals[]: 0 density, 1 row_mean, 2 row_cv, 3 empty_row_frac, 4 col_deg_mean,
 *          5 col_deg_cv, 6 row_span_mean, 7 row_span_norm, 8 col_gap_mean,
 *          9 diag_frac, 10 tile16_coverage, 11 dense_tile_frac,
 *          12 dense_tile_nnz_frac, 13 rho_ell, 14 rho_sell16, 15 rho_sell32,
 *          16 rho_sell512, 17 rho_bsr4, 18 rho_bsr8, 19 rho_bsr16,
 *          20 rho_bell16, 21 nnz_per_tile16
 * row_hist[33]: bin 0 holds r = 0, bin t holds 2^(t-1) <= r < 2^t.
 * fill_hist[8]: occupied 16x16 tiles by nonzero count c, bin (c-1)/32.
 *
 * Quartiles are lower nearest-rank: sorted[floor(p (m-1))].  The median row
 * span is the lower median over non-empty rows of (last col - first col + 1).
 * CV is the population CV: sqrt(sum(x^2)/n - mean^2) / mean.  The mean gap is
 * pooled: sum over rows with r >= 2 of (span - 1), over the sum of (r - 1).
 */
static double cv_of(int64_t sum, int64_t sumsq, int64_t count) {
  if (count <= 0 || sum <= 0) return 0.0;
  double mean = (double)sum / (double)count;
  double var = (double)sumsq / (double)count - mean * mean;
  return var > 0.0 ? sqrt(var) / mean : 0.0;
}

static int cmp_i64(const void *a, const void *b) {
  int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
  return (x > y) - (x < y);
}

static int64_t sell_slots(int32_t m, const int32_t *rowptr, int32_t c) {
  int64_t slots = 0;
  for (int32_t s0 = 0; s0 < m; s0 += c) {
    int32_t s1 = s0 + c < m ? s0 + c : m;
    int32_t mx = 0;
    for (int32_t i = s0; i < s1; ++i)
      if (rowptr[i + 1] - rowptr[i] > mx) mx = rowptr[i + 1] - rowptr[i];
    slots += (int64_t)(s1 - s0) * mx;
  }
  return slots;
}

void oracle_stats(int32_t m, int32_t k, const int32_t *rowptr, const int32_t *colidx, int32_t dense_thr,
                  int64_t *ints, double *reals, int64_t *row_hist, int64_t *fill_hist) {
  const int64_t nnz = m > 0 ? rowptr[m] : 0;
  memset(ints, 0, sizeof(int64_t) * 22);
  memset(reals, 0, sizeof(double) * 22);
  memset(row_hist, 0, sizeof(int64_t) * 33);
  memset(fill_hist, 0, sizeof(int64_t) * 8);
  ints[0] = m;
  ints[1] = k;
  ints[2] = nnz;

  /* rows */
  int64_t *len = (int64_t *)malloc(sizeof(int64_t) * (size_t)(m > 0 ? m : 1));
  int64_t sumsq = 0, empty = 0;
  for (int32_t i = 0; i < m; ++i) {
    len[i] = rowptr[i + 1] - rowptr[i];
    sumsq += len[i] * len[i];
    if (len[i] == 0) ++empty;
    int t = 0;
    while (t < 32 && len[i] >= ((int64_t)1 << t)) ++t;
    row_hist[t]++;
  }
  qsort(len, (size_t)m, sizeof(int64_t), cmp_i64);
  if (m > 0) {
    ints[3] = len[0];
    ints[4] = len[m - 1];
    ints[5] = len[(m - 1) / 4];
    ints[6] = len[(m - 1) / 2];
    ints[7] = len[3 * (int64_t)(m - 1) / 4];
  }
  free(len);
  ints[8] = empty;
  if (m > 0 && k > 0) reals[0] = (double)nnz / ((double)m * (double)k);
  if (m > 0) {
    reals[1] = (double)nnz / (double)m;
    reals[2] = cv_of(nnz, sumsq, m);
    reals[3] = (double)empty / (double)m;
  }

  /* columns */
  int64_t *deg = (int64_t *)calloc((size_t)(k > 0 ? k : 1), sizeof(int64_t));
  for (int64_t p = 0; p < nnz; ++p) deg[colidx[p]]++;
  int64_t dmax = 0, dsq = 0;
  for (int32_t j = 0; j < k; ++j) {
    if (deg[j] > dmax) dmax = deg[j];
    dsq += deg[j] * deg[j];
  }
  free(deg);
  ints[9] = dmax;
  if (k > 0) {
    reals[4] = (double)nnz / (double)k;
    reals[5] = cv_of(nnz, dsq, k);
  }

  /* spans, gaps, diagonal */
  int64_t *spans = (int64_t *)malloc(sizeof(int64_t) * (size_t)(m > 0 ? m : 1));
  int64_t nspan = 0, span_sum = 0, gap_num = 0, gap_den = 0, diag = 0;
  for (int32_t i = 0; i < m; ++i) {
    int32_t r = rowptr[i + 1] - rowptr[i];
    for (int32_t p = rowptr[i]; p < rowptr[i + 1]; ++p)
      if (colidx[p] == i) ++diag;
    if (r == 0) continue;
    int64_t span = (int64_t)colidx[rowptr[i + 1] - 1] - colidx[rowptr[i]] + 1;
    spans[nspan++] = span;
    span_sum += span;
    if (r >= 2) {
      gap_num += span - 1;
      gap_den += r - 1;
    }
  }
  qsort(spans, (size_t)nspan, sizeof(int64_t), cmp_i64);
  if (nspan > 0) {
    ints[10] = spans[(nspan - 1) / 2];
    reals[6] = (double)span_sum / (double)nspan;
    if (k > 0) reals[7] = reals[6] / (double)k;
  }
  free(spans);
  if (gap_den > 0) reals[8] = (double)gap_num / (double)gap_den;
  ints[11] = diag;
  int32_t mn = m < k ? m : k;
  if (mn > 0) reals[9] = (double)diag / (double)mn;

  /* blocks */
  int64_t nnzb[3];
  const int32_t bs[3] = {4, 8, 16};
  for (int t = 0; t < 3; ++t) nnzb[t] = oracle_block_counts(m, rowptr, colidx, bs[t], NULL);
  ints[12] = nnzb[0];
  ints[13] = nnzb[1];
  ints[14] = nnzb[2];
  /* 16x16 tile fills: sort the tile keys of each block-row */
  {
    const int32_t mb = (m + 15) / 16;
    int32_t *scratch = (int32_t *)malloc(sizeof(int32_t) * (size_t)max_block_row_nnz(m, rowptr, 16));
    int64_t dense_tiles = 0, dense_nnz = 0;
    int32_t width = 0;
    for (int32_t br = 0; br < mb; ++br) {
      int32_t r0 = br * 16, r1 = r0 + 16 < m ? r0 + 16 : m;
      int32_t cnt = 0;
      for (int32_t p = rowptr[r0]; p < rowptr[r1]; ++p) scratch[cnt++] = colidx[p] / 16;
      qsort(scratch, (size_t)cnt, sizeof(int32_t), cmp_i32);
      int32_t tiles = 0;
      for (int32_t q = 0; q < cnt;) {
        int32_t e = q;
        while (e < cnt && scratch[e] == scratch[q]) ++e;
        int32_t fill = e - q;
        fill_hist[(fill - 1) / 32]++;
        if (fill >= dense_thr) {
          ++dense_tiles;
          dense_nnz += fill;
        }
        ++tiles;
        q = e;
      }
      if (tiles > width) width = tiles;
    }
    free(scratch);
    ints[15] = dense_tiles;
    ints[16] = dense_nnz;
    ints[17] = width;
    if (m > 0 && k > 0) reals[10] = (double)nnzb[2] / ((double)((m + 15) / 16) * (double)((k + 15) / 16));
    if (nnzb[2] > 0) {
      reals[11] = (double)dense_tiles / (double)nnzb[2];
      reals[21] = (double)nnz / (double)nnzb[2];
    }
    if (nnz > 0) reals[12] = (double)dense_nnz / (double)nnz;
  }

  /* representation expansion, Eq. format-expansion */
  ints[18] = sell_slots(m, rowptr, 16);
  ints[19] = sell_slots(m, rowptr, 32);
  ints[20] = sell_slots(m, rowptr, 512);
  if (nnz > 0) {
    reals[13] = (double)((int64_t)m * ints[4]) / (double)nnz;
    reals[14] = (double)ints[18] / (double)nnz;
    reals[15] = (double)ints[19] / (double)nnz;
    reals[16] = (double)ints[20] / (double)nnz;
    reals[17] = (double)(16 * nnzb[0]) / (double)nnz;
    reals[18] = (double)(64 * nnzb[1]) / (double)nnz;
    reals[19] = (double)(256 * nnzb[2]) / (double)nnz;
    reals[20] = (double)(256 * ints[17] * (int64_t)((m + 15) / 16)) / (double)nnz;
  }

  /* shape class (a reading: the paper gives no thresholds):
   * 0 uniform     CV < 0.1 (or no nonzeros);
   * 4 bimodal     else, two local maxima of the log2 row-length histogram at
   *               least 2 bins apart, each holding >= 10 % of the rows;
   * 1 moderate    else CV < 0.5;
   * 3 power-law   else CV >= 1 and max >= 50 mean;
   * 2 skewed      otherwise. */
  {
    double cv = reals[2], mean = reals[1];
    int cls;
    int bimodal = 0;
    for (int a = 0; a < 33 && !bimodal; ++a) {
      int amax = (a == 0 || row_hist[a] > row_hist[a - 1]) && (a == 32 || row_hist[a] >= row_hist[a + 1]);
      if (!amax || 10 * row_hist[a] < m) continue;
      for (int c2 = a + 2; c2 < 33; ++c2) {
        int cmax = (row_hist[c2] > row_hist[c2 - 1]) && (c2 == 32 || row_hist[c2] >= row_hist[c2 + 1]);
        if (cmax && 10 * row_hist[c2] >= m) { bimodal = 1; break; }
      }
    }
    if (nnz == 0 || cv < 0.1) cls = 0;
    else if (bimodal) cls = 4;
    else if (cv < 0.5) cls = 1;
    else if (cv >= 1.0 && (double)ints[4] >= 50.0 * mean) cls = 3;
    else cls = 2;
    ints[21] = cls;
  }
}

/* Thread count of the OpenMP row loops above.  Results do not depend on it:
 * each row is summed sequentially by one thread.  n > 0 sets it; returns the
 * count in effect. */
int32_t oracle_threads(int32_t n) {
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
}
