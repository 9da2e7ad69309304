// Launch interface of the SpMM kernels (HIP, gfx950).  All pointers are
// device pointers; every launch is asynchronous on `stream`.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>
#include <functional>

#include "../../include/sparseditto.h"
#include "sd_internal.h"

namespace sd {

struct CsrOperand {
  const int32_t *rowptr;
  const int32_t *colidx;
  const float *vals;
  int32_t m;  // rows of the operand (= rows of C)
  int32_t k;  // columns of the operand (= rows of B)
};

struct DenseIO {
  const float *B;
  float *C;
  int32_t n;
  int32_t vec4;    // 1: B and C 16-byte aligned and n % 4 == 0
  int32_t policy;  // B-gather cache policy: 0 normal, 1 tiered by the column tag, 2 non-temporal
  int32_t col_tile;  // dense columns per lane group (power of two >= 4), 0 = whole width
  int32_t order;     // workgroup order: 1 one contiguous range of rows per XCD, 0 hardware round-robin,
                     // S >= 2 round-robin over chunks of S consecutive workgroups
};

// Lane-group geometry for a dense width: G lanes per sparse row, VW floats
// per lane, coltiles column tiles of G*VW columns.
struct Geometry {
  int32_t G, VW, coltiles;
};
Geometry geometry_for(int32_t n, int32_t vec4, int32_t col_tile = 0);

// slices > 1 (G <= 8 only): S = slices lane groups share each row, each taking
// every S-th nonzero (rows_per_group and unroll are then unused).
hipError_t launch_csr_rows(const CsrOperand &A, const DenseIO &io, int32_t rows_per_group, int32_t unroll,
                           int32_t slices, hipStream_t s);

// corder: the chunk processing order, a permutation of [0, nchunks).
hipError_t launch_csr_split(const CsrOperand &A, const int32_t *light, int32_t nlight, const int32_t *chunks,
                            const int32_t *corder, int32_t nchunks, const int32_t *heavy_rows,
                            const int32_t *heavy_ptr, int32_t nheavy, float *ws, const DenseIO &io,
                            int32_t rows_per_group, int32_t unroll, int32_t slices, hipStream_t s);

// Merge path over `units` pieces.  rows: 2 units int32 (carry rows, then head
// rows); part: 2 units n floats (carry partials, then head partials).
hipError_t launch_csr_merge(const CsrOperand &A, const int32_t *coords, int32_t units, int32_t *rows,
                            float *part, const DenseIO &io, hipStream_t s);

// Block formats: bptr == nullptr selects Blocked-ELL with `width` slots per
// block-row.  engine: 1 MFMA (any width: 64-, 32- and 16-column tiles, the
// last one partial; 16-column tiles of single floats without vec4), 2 VALU.
// zero_block: index of a block with column -1 and zero values that follows the
// stored blocks (the MFMA kernel fetches it for slots past a block-row's end).
// zrow: io.n zero floats (16-byte aligned), the MFMA kernel's B operand for
// every slot without a B row.
hipError_t launch_bsr(int32_t mb, int32_t m, int32_t k, const int32_t *bptr, int32_t width,
                      const int32_t *bcol, const float *bval, int64_t zero_block, const float *zrow,
                      int32_t engine, const DenseIO &io, hipStream_t s);

// ELL: ecol/eval [m][width], column -1 = padding.  passes >= 1 and width <= G
// (the lane-group size) select the pipelined kernel with `passes` row passes
// per workgroup; otherwise one row per lane group.
hipError_t launch_ell(const int32_t *ecol, const float *eval, int32_t width, int32_t m, int32_t passes,
                      const DenseIO &io, hipStream_t s);

// SELL-C-sigma: perm [m], slice pointers sptr [ceil(m/C)+1] (int64), slots
// scol/sval row-major per slice, column -1 = padding.
hipError_t launch_sell(const int32_t *perm, const int64_t *sptr, const int32_t *scol, const float *sval,
                       int32_t C, int32_t m, const DenseIO &io, hipStream_t s);

// Packed column windows over the heavy-split layout: A.rowptr holds the light
// rows' pointers by list position and A.colidx the entry codes (-2 - p for the
// window's staged column p, else the column); light-list windows of R
// positions stage wcols[wptr[w] .. wptr[w+1]] (at most wmax); the chunks and
// the fix-up are those of launch_csr_split.  Dynamic LDS:
// window_lds_bytes(n, vec4, col_tile, wmax).
size_t window_lds_bytes(int32_t n, int32_t vec4, int32_t col_tile, int32_t staged);
hipError_t launch_win_split(const CsrOperand &A, const int32_t *light, int32_t nlight, const int32_t *chunks,
                            const int32_t *corder, int32_t nchunks, const int32_t *heavy_rows,
                            const int32_t *heavy_ptr, int32_t nheavy, float *ws, const int32_t *wptr,
                            const int32_t *wcols, int32_t R, int32_t wmax, const DenseIO &io, hipStream_t s);

// Reads `bytes` of `buf` (16-byte aligned, zero-filled) so that L2 and the
// Infinity Cache no longer hold earlier data; `sink` is one float that is
// never written for a zero-filled buffer.
hipError_t launch_cache_flush(const void *buf, size_t bytes, float *sink, hipStream_t s);

// convert.hip: conversions and partitions on the device, producing exactly
// the arrays of the host conversions (ell_convert, merge_split, heavy_split).
hipError_t dev_ell(const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t m, int32_t W,
                   int32_t *ecol, float *eval, hipStream_t s);
hipError_t dev_merge_coords(const int32_t *rowptr, int32_t m, int64_t nnz, int32_t U, int64_t L, int32_t *coords,
                            hipStream_t s);
// per row max(|first col - row|, |last col - row|), -1 for an empty row
// 16x16 BSR (ell_width < 0: nnzb blocks, bptr [mb+1]) or Blocked-ELL
// (ell_width >= 0: mb * ell_width slots, -1 padding) of a valid CSR in device
// memory, into caller-owned bcol [slots+1] and bval [(slots+1)*256] (one zero
// block after the stored ones); bptr may be null for Blocked-ELL.  nnzb and
// ell_width come from the analysis; a disagreement returns
// hipErrorInvalidValue before any block is written.  Waits for the stream.
hipError_t dev_block16(const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t m, int32_t k,
                       int64_t nnz, int64_t nnzb, int32_t ell_width, int32_t *bptr, int32_t *bcol, float *bval,
                       hipStream_t s);
// SELL-C-sigma of a valid CSR in device memory (rows sorted longest first
// within windows of sigma rows, slices of C rows padded to their longest row,
// column -1 / value 0 padding).  perm [m] and slice_ptr [ns+1] come from
// alloc; *slots is the padded size.  When it exceeds max_slots nothing more is
// built (col and val stay null); else col and val [slots] come from alloc.
// Waits for the stream.
hipError_t dev_sell(const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t m, int32_t row_max,
                    int32_t C, int32_t sigma, int64_t max_slots, const std::function<void *(size_t)> &alloc,
                    hipStream_t s, int32_t **perm, int64_t **sptr, int32_t **scol, float **sval, int64_t *slots);
// Tiered-policy tags of a valid CSR's columns in device memory: tagged [nnz]
// (caller-owned) holds each column, with bit 31 set where the column is
// cold, i.e. below the smallest degree D >= 2 whose columns at or above it
// number at most budget_rows.  Waits for the stream.
hipError_t dev_tag_cold(const int32_t *colidx, int64_t nnz, int32_t k, int64_t budget_rows, int32_t *tagged,
                        int64_t *hot_cols, int64_t *hot_nnz, hipStream_t s);
// Hash of a CSR pattern: the sum modulo 2^64 of mix64(salt ^ (i << 32 | a[i]))
// over the row pointers (salt kPatternSalt[0]) and the column indices
// (kPatternSalt[1]); pattern_hash_host computes the same value.  Waits for
// the stream.
constexpr uint64_t kPatternSalt[2] = {0x243f6a8885a308d3ull, 0x13198a2e03707344ull};
hipError_t dev_pattern_hash(const int32_t *rowptr, const int32_t *colidx, int32_t m, int64_t nnz, hipStream_t s,
                            uint64_t *out);
uint64_t pattern_hash_host(const int32_t *rowptr, const int32_t *colidx, int32_t m, int64_t nnz);
// CSR of A^T (k rows, m columns) from a valid CSR A in device memory, into
// caller-owned t_rowptr [k+1], t_colidx [nnz], t_vals [nnz]; rows of each
// column ascending.  Waits for the stream.
hipError_t dev_transpose(const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t m, int32_t k,
                         int64_t nnz, int32_t *t_rowptr, int32_t *t_colidx, float *t_vals, hipStream_t s);
hipError_t dev_row_reach(const int32_t *rowptr, const int32_t *colidx, int32_t m, int64_t *reach, hipStream_t s);
// alloc(bytes) returns plan-owned device memory (nullptr on failure); waits for s
// Writes the heavy-split layout into lptr (|light| + 1), colidx_out and
// vals_out (nnz each): the light rows' entries in list order, then the heavy
// rows' in the order of heavy_rows; moves each heavy row's chunks (heavy_ptr
// groups them; their begin and end are in the input's coordinates on entry)
// to the new coordinates.  The inputs must not alias the outputs.
hipError_t dev_split_layout(const int32_t *rowptr, const int32_t *colidx, const float *vals, int64_t nnz,
                            const int32_t *light, int64_t n_light, const int32_t *heavy_rows,
                            const int32_t *heavy_ptr, int64_t n_heavy, int32_t *lptr, int32_t *colidx_out,
                            float *vals_out, int32_t *chunks, hipStream_t s);
// Packed column windows over a split layout in device memory (lptr [n_light
// + 1], colidx [nnz], the layout's columns): windows of R light-list
// positions stage the columns two or more of their rows use, at most cap, the
// most used kept (ties to the smaller column), ascending.  The light entries'
// columns in colidx become codes (-2 - staged position, else the column);
// wptr [windows + 1] and wcols [staged] come from alloc.  Waits for the
// stream.  The same arrays as the host's split_windows.
hipError_t dev_split_windows(const int32_t *lptr, int64_t n_light, int32_t *colidx, int32_t R, int32_t cap,
                             const std::function<void *(size_t)> &alloc, hipStream_t s, int32_t **wptr,
                             int32_t **wcols, int32_t *wmax, int64_t *n_staged, int64_t *staged_uses);
// Chunk processing order of a split layout: by the column of each chunk's
// middle entry colidx[(begin + end) / 2], ties by chunk index (order 2), or
// the chunk list itself (order 1).  corder: n_chunks int32.
hipError_t dev_chunk_order(const int32_t *colidx, const int32_t *chunks, int64_t n_chunks, int32_t k, int32_t order,
                           int32_t *corder, hipStream_t s);
// Reorders the light rows (device, ascending on entry) by the column of their
// last nonzero, ties by row, empty rows last (a stable radix sort by key).
hipError_t dev_light_by_last_col(const int32_t *rowptr, const int32_t *colidx, int32_t k, int32_t *light,
                                 int64_t n_light, hipStream_t s);
hipError_t dev_heavy_split(const int32_t *rowptr, int32_t m, int32_t T, int32_t c,
                           const std::function<void *(size_t)> &alloc, hipStream_t s, int32_t **light,
                           int32_t **chunks, int32_t **heavy_rows, int32_t **heavy_ptr, int64_t *n_light,
                           int64_t *n_heavy, int64_t *n_chunks);

// analyze.hip: sd_analyze on a CSR matrix whose arrays are device pointers;
// runs on stream s and waits for it.  Same statistics as the host analysis.
int analyze_device(const sd_csr_t *A, int32_t dense_threshold, sd_stats_t *out, hipStream_t s);

// Kernel attributes of the main kernel a plan will launch (for the
// resource-bound legality check).
// width: ELL/WIN slots per row.
hipError_t kernel_attributes(int32_t family, int32_t engine, int32_t n, int32_t vec4, int32_t rows_per_group,
                             int32_t unroll, int32_t slices, int32_t col_tile, int32_t width,
                             hipFuncAttributes *attr);

}  // namespace sd
