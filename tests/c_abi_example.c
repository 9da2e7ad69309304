/* The library from plain C: analyse, plan and run C = A.B through the C ABI
 * with device buffers from the HIP runtime, no Python and no torch.
 *
 * A is the m x m tridiagonal matrix with 2 on the diagonal and -1 beside it,
 * and B holds small integers, so every product and partial sum is an integer
 * below 2^24 and the exact result is known in closed form:
 *   C[i][c] = 2 B[i][c] - B[i-1][c] - B[i+1][c]   (missing neighbours dropped).
 * The program checks every element bitwise for several widths (each width
 * selects a different kernel geometry).
 *
 * Exit status: 0 all widths exact, 1 a mismatch or an error, 2 no GPU (the
 * library loaded and planned on the host only). */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "sparseditto.h"

#define CHECK_SD(call)                                                          \
  do {                                                                          \
    int st_ = (call);                                                           \
    if (st_ != SD_OK) {                                                         \
      fprintf(stderr, "%s: %s (%s)\n", #call, sd_status_string(st_), sd_last_error()); \
      return 1;                                                                 \
    }                                                                           \
  } while (0)

static int run_width(const sd_csr_t *A, int32_t n) {
  const int32_t m = A->m;
  float *hb = malloc(sizeof(float) * (size_t)m * n), *hc = malloc(sizeof(float) * (size_t)m * n);
  if (!hb || !hc) return 1;
  for (int32_t i = 0; i < m; ++i)
    for (int32_t c = 0; c < n; ++c) hb[(size_t)i * n + c] = (float)((i * 7 + c * 3) % 19 - 9);
  float *db = NULL, *dc = NULL;
  if (hipMalloc((void **)&db, sizeof(float) * (size_t)m * n) != hipSuccess ||
      hipMalloc((void **)&dc, sizeof(float) * (size_t)m * n) != hipSuccess ||
      hipMemcpy(db, hb, sizeof(float) * (size_t)m * n, hipMemcpyHostToDevice) != hipSuccess) {
    fprintf(stderr, "hip allocation or copy failed\n");
    return 1;
  }
  sd_plan_t plan = NULL;
  CHECK_SD(sd_plan(A, n, &plan));
  sd_plan_info_t info;
  CHECK_SD(sd_plan_info(plan, &info));
  CHECK_SD(sd_spmm(plan, db, dc, NULL));
  if (hipDeviceSynchronize() != hipSuccess ||
      hipMemcpy(hc, dc, sizeof(float) * (size_t)m * n, hipMemcpyDeviceToHost) != hipSuccess) {
    fprintf(stderr, "hip synchronise or copy failed\n");
    return 1;
  }
  long bad = 0;
  for (int32_t i = 0; i < m; ++i)
    for (int32_t c = 0; c < n; ++c) {
      float want = 2.0f * hb[(size_t)i * n + c];
      if (i > 0) want -= hb[(size_t)(i - 1) * n + c];
      if (i + 1 < m) want -= hb[(size_t)(i + 1) * n + c];
      if (memcmp(&want, &hc[(size_t)i * n + c], sizeof(float)) != 0) ++bad;
    }
  printf("n=%d family=%d lanes_per_row=%d row_slices=%d mismatches=%ld\n", n, info.family, info.lanes_per_row,
         info.row_slices, bad);
  sd_plan_destroy(plan);
  hipFree(db);
  hipFree(dc);
  free(hb);
  free(hc);
  return bad == 0 ? 0 : 1;
}

int main(void) {
  const int32_t m = 4099;  /* not a multiple of any tile */
  const int64_t nnz = 3 * (int64_t)m - 2;
  int32_t *rowptr = malloc(sizeof(int32_t) * (m + 1)), *colidx = malloc(sizeof(int32_t) * nnz);
  float *vals = malloc(sizeof(float) * nnz);
  if (!rowptr || !colidx || !vals) return 1;
  int64_t p = 0;
  for (int32_t i = 0; i < m; ++i) {
    rowptr[i] = (int32_t)p;
    for (int32_t j = i - 1; j <= i + 1; ++j)
      if (j >= 0 && j < m) {
        colidx[p] = j;
        vals[p] = j == i ? 2.0f : -1.0f;
        ++p;
      }
  }
  rowptr[m] = (int32_t)p;
  sd_csr_t A = {m, m, nnz, rowptr, colidx, vals};

  sd_stats_t stats;
  CHECK_SD(sd_analyze(&A, 0, &stats));
  printf("analyse: m=%lld nnz=%lld row_max=%lld diag_frac=%.3f\n", (long long)stats.m, (long long)stats.nnz,
         (long long)stats.row_max, stats.diag_frac);

  int devices = 0;
  if (hipGetDeviceCount(&devices) != hipSuccess || devices == 0) {
    sd_plan_opts_t o;
    memset(&o, 0, sizeof(o));
    o.placement = 2; /* host only */
    sd_plan_t plan = NULL;
    CHECK_SD(sd_plan_ex(&A, 8, &o, &plan));
    const int st = sd_spmm(plan, NULL, NULL, NULL);
    sd_plan_destroy(plan);
    printf("no GPU: host-only plan built, sd_spmm says %s\n", sd_status_string(st));
    return st == SD_ERR_INVALID_VALUE || st == SD_ERR_NO_DEVICE ? 2 : 1;
  }
  const int32_t widths[] = {1, 3, 8, 32, 64, 100};
  for (size_t w = 0; w < sizeof(widths) / sizeof(widths[0]); ++w)
    if (run_width(&A, widths[w]) != 0) return 1;
  free(rowptr);
  free(colidx);
  free(vals);
  printf("ok\n");
  return 0;
}
