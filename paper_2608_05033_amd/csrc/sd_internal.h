// Internal declarations shared by the host-side C++ and the HIP runtime of
// the SpMM library.  Nothing here is part of the C ABI.
#pragma once

#include <cstdint>
#include <cstddef>
#include <string>
#include <vector>

#include "../../include/sparseditto.h"

namespace sd {

// Records the HIP error's text for sd_last_error on this thread and returns
// SD_ERR_HIP.
int report_hip_error(int hip_error);

// MI355X (gfx950) figures used when no device is attached to a plan
// (host-only plans): 256 compute units, 4 MiB L2 per XCD, 256 MiB
// Infinity Cache, 160 KiB LDS per CU (64 KiB addressable per workgroup by
// default), 1024 threads per workgroup, 512 VGPRs per lane per SIMD.
constexpr int32_t kDefaultCUs = 256;
constexpr int64_t kDefaultL2 = 4ll << 20;
constexpr int64_t kMallBytes = 256ll << 20;
constexpr int32_t kDefaultMaxThreads = 1024;
constexpr int32_t kDefaultMaxLds = 64 << 10;
constexpr int32_t kBlockThreads = 256;  // every kernel runs 4 wave64 per workgroup
// Packed column windows: default light rows per window, and the LDS the
// staged B rows of one window may take (a window keeps its most used columns
// that fit).  16 KiB leaves room for eight workgroups per compute unit: on the
// power-law workloads 64 KiB (two per unit) ran 1.5-2.6x slower than 16.
constexpr int32_t kDefaultWindowRows = 64;
constexpr int64_t kWindowLdsBudget = 16 << 10;

// Host view of a validated CSR matrix (non-owning).
struct CsrView {
  int32_t m = 0, k = 0;
  int64_t nnz = 0;
  const int32_t *rowptr = nullptr;
  const int32_t *colidx = nullptr;
  const float *values = nullptr;
};

// Owned CSR (used for the materialised transpose).
struct CsrOwned {
  int32_t m = 0, k = 0;
  std::vector<int32_t> rowptr, colidx;
  std::vector<float> values;
  CsrView view() const {
    CsrView v;
    v.m = m;
    v.k = k;
    v.nnz = rowptr.empty() ? 0 : rowptr.back();
    v.rowptr = rowptr.data();
    v.colidx = colidx.data();
    v.values = values.data();
    return v;
  }
};

// host_csr.cpp
int validate_csr(const sd_csr_t *A, CsrView *out);
int analyze(const CsrView &A, int32_t dense_threshold, sd_stats_t *out);
// Exact integer sums behind the fp64 statistics (population CVs, span mean,
// column-gap mean).  finish_stats computes every fp64 field, the expansion
// factors and the shape class from the integer fields of *out and these sums,
// so host and device analysis give bit-identical statistics.
struct StatsSums {
  int64_t row_sumsq = 0, col_sumsq = 0, span_sum = 0, nonempty = 0, gap_num = 0, gap_den = 0;
};
void finish_stats(const StatsSums &sum, sd_stats_t *out);
int64_t kth_from_hist(const std::vector<int64_t> &hist, int64_t kth);
int transpose(const CsrView &A, CsrOwned *out);

// host_plan.cpp: conversions and partitions
// order 1: light rows ascending; 2: by the column of their last nonzero (ties
// by row, empty rows last).
void heavy_split(const CsrView &A, int32_t T, int32_t c, int32_t order, std::vector<int32_t> *light,
                 std::vector<int32_t> *chunks, std::vector<int32_t> *heavy_rows,
                 std::vector<int32_t> *heavy_ptr);
void merge_split(const CsrView &A, int32_t U, std::vector<int32_t> *coords, int64_t *L);
void block_convert(const CsrView &A, int32_t b, bool ell, std::vector<int32_t> *bptr,
                   std::vector<int32_t> *bcol, std::vector<float> *bval, int32_t *width);

// ELL: rows padded to the longest row, row-major [m][W], padding column -1
// and value +0.0f.
void ell_convert(const CsrView &A, std::vector<int32_t> *ecol, std::vector<float> *eval, int32_t *width);

// SELL-C-sigma: perm[i] = original row of sorted row i (stable sort by
// non-increasing length inside windows of sigma rows); slices of C sorted
// rows, row-major, padded to the slice's longest row (column -1, +0.0f);
// slice_ptr[s] = first slot of slice s.
void sell_convert(const CsrView &A, int32_t C, int32_t sigma, std::vector<int32_t> *perm,
                  std::vector<int64_t> *slice_ptr, std::vector<int32_t> *col, std::vector<float> *val);

// Packed column windows over the heavy-split layout: the light rows, in list
// order, are cut into windows of R list positions; a window stages the
// columns that two or more of its rows use (at most cap, the most used kept,
// ties to the smaller column), ascending in wcols[wptr[w] .. wptr[w+1]].  In
// colidx (the layout's columns, |light| rows of lptr first) an entry of a
// light row whose column its window stages becomes -2 - p (staged position
// p); every other entry keeps its column.  wmax is the largest staged count of
// a window, staged_uses the entries that read a staged column.
void split_windows(int32_t k, const std::vector<int32_t> &lptr, int64_t n_light, std::vector<int32_t> *colidx,
                   int32_t R, int32_t cap, std::vector<int32_t> *wptr, std::vector<int32_t> *wcols, int32_t *wmax,
                   int64_t *staged_uses);

// Tiered gather policy: bit 31 of a column index marks a cold column (its B
// row is gathered non-temporally).  Hot columns are those with degree >= D,
// D the smallest degree >= 2 for which they number at most `budget_rows`.
void tag_cold_columns(const CsrView &A, int64_t budget_rows, std::vector<int32_t> *tagged, int64_t *hot_cols,
                      int64_t *hot_nnz);

// Planner rules (family choice and default parameters).
struct PlanChoice {
  int32_t family = SD_FMT_CSR_ROW;
  int32_t engine = SD_ENGINE_AUTO;
  int32_t T = 0, c = 0, U = 0;
  int32_t policy = 1;  // 1 normal, 2 tiered, 3 non-temporal
  int32_t wg_order = 2;  // 1 contiguous rows per XCD, 2 hardware round-robin
};
// G is the number of lanes that share one sparse row for width n.
PlanChoice choose_plan(const sd_stats_t &st, int32_t n, int32_t cu_count, int32_t G, const sd_plan_opts_t &o);
// Median over non-empty rows of the largest |column - row| (lower median).
int64_t median_row_reach(const CsrView &A);
// Chunk size S for the chunked round-robin workgroup order: the largest power
// of two in [8, 64] such that one round of 8 chunks divides the reach in
// workgroups, so a row and its farthest typical neighbour run on the same XCD;
// 0 if there is none (keep the plain round-robin).
int32_t chunk_for_reach(int64_t reach, int64_t rows_per_wg);
// Row batching for the row kernels: rows per lane group J in {1, 2, 4}
// (J <= G) and B-row gathers per row per batch UNR in {4, 8}.
void row_batch_for(const sd_stats_t &st, int64_t rows, int32_t G, int32_t cu_count, int32_t req_J,
                   int32_t req_unr, int32_t *J, int32_t *unr);
// Nonzeros each slice of a sliced row takes per round (the B-row gathers in
// flight per lane).
constexpr int32_t kSliceRound = 4;
// The heavy-split layout: the light rows' entries in the order of `light`,
// then the heavy rows' (r >= T) ascending.  lptr (|light| + 1) points into it
// by list position; chunks (row, begin, end) are in its coordinates.
void split_layout(const CsrView &A, int32_t T, int32_t c, const std::vector<int32_t> &light,
                  std::vector<int32_t> *lptr, std::vector<int32_t> *colidx, std::vector<float> *vals,
                  std::vector<int32_t> *chunks);
// Processing order of the split layout's chunks: order 2 sorts the chunk
// indices by the column of each chunk's middle entry colidx[(begin + end) / 2]
// (ties by index), so chunks of different heavy rows that cover the same
// columns run together; order 1 keeps the chunk list.
void chunk_order(const std::vector<int32_t> &colidx, const std::vector<int32_t> &chunks, int32_t order,
                 std::vector<int32_t> *corder);
// Lane groups sharing one row in the CSR row and heavy-split kernels (1 = one
// group per row); a power of two with G * S <= 64, above 1 only for G <= 8.
int32_t slices_for(const sd_stats_t &st, int32_t family, int32_t n, int32_t G);

}  // namespace sd

// The opaque plan.  Host arrays are kept for host-only plans; device plans
// release them once uploaded and export from device memory instead.
struct sd_plan_s {
  sd_plan_info_t info{};
  int32_t device = -1;  // -1: host only
  int32_t col_tile_req = 0;  // requested dense columns per lane group (0: whole width)

  // host arrays
  std::vector<int32_t> h_rowptr, h_colidx, h_coltag, h_light, h_chunks, h_corder, h_heavy_rows, h_heavy_ptr, h_coords,
      h_bptr, h_bcol, h_ecol, h_wptr, h_wcols, h_perm;
  std::vector<int64_t> h_sptr;
  std::vector<float> h_vals, h_bval, h_eval;

  // device arrays
  int32_t *d_corder = nullptr;  // CSR_SPLIT: chunk processing order
  int32_t *d_rowptr = nullptr, *d_colidx = nullptr, *d_light = nullptr, *d_chunks = nullptr,
          *d_heavy_rows = nullptr, *d_heavy_ptr = nullptr, *d_coords = nullptr, *d_bptr = nullptr,
          *d_bcol = nullptr, *d_carry_row = nullptr, *d_ecol = nullptr, *d_wptr = nullptr, *d_wcols = nullptr,
          *d_perm = nullptr;
  int64_t *d_sptr = nullptr;
  float *d_vals = nullptr, *d_bval = nullptr, *d_ws = nullptr, *d_eval = nullptr;
  float *d_zrow = nullptr;  // block families: n zero floats, the B row of slots without one
  std::vector<void *> allocations;
};
