/*
 * sparseditto.h -- C ABI of the MI355X SpMM library.
 *
 * The library computes C = A.B (or C = A^T.B) for a sparse A given in CSR
 * (int32 indices, fp32 values) and dense, row-major fp32 B and C, through a
 * representation and schedule chosen from A's structure.  The paper frames
 * this as a compilation plan Pi = <R, S, theta_H> (Sec. "SparseDitto Design",
 * Eq. compilation-plan): a representation R (layout + metadata), a schedule S
 * (parallel decomposition + dataflow) and target-specific parameters.
 *
 * Calls:
 *   sd_analyze      structural statistics            (Sec. "Structural Features and
 *                                                     Overhead Modeling", Eq. format-expansion)
 *   sd_plan[_ex]    choose + size + convert + upload (Sec. "Architecture-Aware
 *                                                     Compilation-Plan Synthesis", Eqs.
 *                                                     representation-footprint,
 *                                                     candidate-working-set, l2-scale-ratios,
 *                                                     resource-bounds)
 *   sd_spmm         run a plan on a HIP stream       (the per-call compute step; one-time
 *                                                     preprocessing stays in sd_plan, as in
 *                                                     the paper's measurement protocol)
 *   sd_analyze_device, sd_plan_device
 *                   the same two steps for a CSR already in device memory
 *   sd_plan_cache_size / _save / _load
 *                   measured plan choices kept and reused across processes
 *   sd_plan_info / sd_plan_export / sd_plan_destroy / sd_status_string / sd_last_error
 *
 * Conventions shared by every call:
 *   - Every function except sd_plan_destroy and sd_status_string returns an
 *     sd_status; 0 (SD_OK) is success.  On failure, outputs are left untouched
 *     unless stated otherwise, and nothing is leaked.
 *   - Host pointers are plain CPU memory; device pointers are HIP device
 *     memory on the plan's device.
 *   - No call keeps a pointer to caller memory after it returns.
 *   - Calls on distinct plans are thread-safe; a single plan must not be used
 *     by two threads or two streams at the same time (its workspace is shared).
 */
#ifndef SPARSEDITTO_H
#define SPARSEDITTO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ statuses --- */
typedef enum {
  SD_OK = 0,
  SD_ERR_INVALID_VALUE = 1, /* null pointer, n < 1, unknown enum, bad option */
  SD_ERR_INVALID_CSR = 2,   /* CSR breaks one of the rules of sd_csr_t */
  SD_ERR_UNSUPPORTED = 3,   /* forced family or parameters infeasible for this input */
  SD_ERR_OUT_OF_MEMORY = 4, /* host or device allocation failed */
  SD_ERR_HIP = 5,           /* HIP runtime or launch error (message via sd_last_error) */
  SD_ERR_OVERFLOW = 6,      /* a size does not fit the index types */
  SD_ERR_NO_DEVICE = 7,     /* the plan has no device part (host-only plan) */
  SD_ERR_IO = 8             /* plan-cache file cannot be opened, read or written, or is malformed */
} sd_status;

/* ----------------------------------------------------------------- CSR --- */
/* A sparse m x k matrix in CSR, in HOST memory (DEVICE memory for
 * sd_analyze_device and sd_plan_device).
 * Rules checked by sd_analyze and sd_plan (else SD_ERR_INVALID_CSR):
 *   m >= 0, k >= 0, rowptr[0] = 0, rowptr non-decreasing, rowptr[m] = nnz,
 *   0 <= colidx[p] < k, and columns strictly ascending within each row
 *   (canonical CSR: no duplicates).  nnz < 2^31 (else SD_ERR_OVERFLOW).
 * values may hold any fp32 bit patterns (they are copied bitwise). */
typedef struct {
  int32_t m, k;
  int64_t nnz;
  const int32_t *rowptr; /* m + 1 */
  const int32_t *colidx; /* nnz */
  const float *values;   /* nnz */
} sd_csr_t;

/* ---------------------------------------------------------- statistics --- */
/* Structural statistics of A (Sec. "Structural Features and Overhead
 * Modeling": intrinsic pattern features and representation-induced overhead
 * features, Eq. format-expansion).  r_i is the nonzero count of row i.
 * Integer fields are exact counts.  Each fp64 field is computed from exact
 * integer sums by exactly the formula given, so results are reproducible bit
 * for bit; every ratio is 0 when its denominator is 0. */
typedef struct {
  int64_t m, k, nnz;
  int64_t row_min, row_max;
  int64_t row_q25, row_q50, row_q75; /* lower nearest rank: sorted r at floor(p (m-1)) */
  int64_t empty_rows;
  int64_t col_deg_max;     /* max over columns of the column nonzero count */
  int64_t row_span_median; /* lower median over non-empty rows of (last col - first col + 1):
                              the "median row bandwidth" of the case studies */
  int64_t diag_nnz;        /* #{p : colidx[p] == row(p)} */
  int64_t nnzb4, nnzb8, nnzb16; /* occupied b x b blocks, block (floor(i/b), floor(j/b)) */
  int64_t dense_tiles16;   /* occupied 16x16 tiles holding >= dense_threshold nonzeros */
  int64_t dense_tile_nnz16;/* nonzeros inside those tiles */
  int64_t bell16_width;    /* max occupied 16x16 blocks in one block-row */
  int64_t sell16_slots, sell32_slots, sell512_slots; /* sum over slices s of c rows of |s| max r_i */
  int64_t shape_class;     /* 0 uniform, 1 moderate, 2 skewed, 3 power-law, 4 bimodal (heuristic) */
  int64_t dense_threshold; /* the threshold used (128 = half-full tile) */

  double density;          /* nnz / (m * k) */
  double row_mean;         /* nnz / m */
  double row_cv;           /* population CV: sqrt(sum r^2 / m - mean^2) / mean */
  double empty_row_frac;   /* empty_rows / m */
  double col_deg_mean;     /* nnz / k */
  double col_deg_cv;       /* population CV of the column counts over all k columns */
  double row_span_mean;    /* sum of spans / #non-empty rows */
  double row_span_norm;    /* row_span_mean / k */
  double col_gap_mean;     /* sum over rows with r >= 2 of (span - 1), over sum of (r - 1) */
  double diag_frac;        /* diag_nnz / min(m, k) */
  double tile16_coverage;  /* nnzb16 / (ceil(m/16) ceil(k/16)) */
  double dense_tile_frac;  /* dense_tiles16 / nnzb16 */
  double dense_tile_nnz_frac; /* dense_tile_nnz16 / nnz */
  double rho_ell;          /* m * row_max / nnz */
  double rho_sell16, rho_sell32, rho_sell512; /* sellC_slots / nnz */
  double rho_bsr4, rho_bsr8, rho_bsr16;       /* b^2 nnzb_b / nnz */
  double rho_bell16;       /* 256 * bell16_width * ceil(m/16) / nnz */
  double nnz_per_tile16;   /* nnz / nnzb16 */

  int64_t row_hist[33];    /* bin 0: r = 0; bin t: 2^(t-1) <= r < 2^t */
  int64_t fill16_hist[8];  /* occupied 16x16 tiles by count c, bin (c - 1) / 32 */
} sd_stats_t;

/* A is read and not kept.  dense_threshold in [1, 256] (0 = default 128).
 * Host-only; needs no GPU.  Errors: SD_ERR_INVALID_VALUE (null A or out),
 * SD_ERR_INVALID_CSR, SD_ERR_OVERFLOW, SD_ERR_OUT_OF_MEMORY. */
int sd_analyze(const sd_csr_t *A, int32_t dense_threshold, sd_stats_t *out);

/* sd_analyze for a matrix already in device memory: A->rowptr, A->colidx and
 * A->values are device pointers of the current HIP device (values are not
 * read).  The statistics are computed by HIP kernels on `stream` (a
 * hipStream_t; NULL = the null stream) as exact integer aggregates and
 * finished on the host exactly as sd_analyze finishes them, so *out is
 * bit-identical to sd_analyze on the same matrix.  Waits for the stream
 * before returning.  Allocates and frees device scratch of about
 * 4 k + 8 (row_max + max row span) + m/4 bytes.
 * Errors: as sd_analyze (the CSR checks run on the device), SD_ERR_NO_DEVICE,
 * SD_ERR_HIP. */
int sd_analyze_device(const sd_csr_t *A, int32_t dense_threshold, sd_stats_t *out, void *stream);

/* --------------------------------------------------------------- plans --- */
/* Plan families: the CSR, nonzero-balanced CSR and block formats of the SpMM
 * template set (Sec. "Energy-Based Model for Optimization Templates"), plus
 * the padded-row, packed-window and sliced layouts of the design space
 * (Appendix "Compilation-Plan Design Space", SpMM and SpMV rows):
 *   CSR_ROW    CSR; a lane group per row covers the dense width with 128-bit
 *              loads of B rows; one write of each C row.
 *   CSR_SPLIT  CSR; rows with r_i >= heavy_threshold are cut into chunks of at
 *              most chunk_nnz nonzeros (Appendix "Case Studies", SpMM web
 *              graph).  Chunk partials go to a workspace and a fix-up kernel
 *              sums them in a fixed order: no atomics, deterministic.
 *   CSR_MERGE  CSR; the merge path of row ends and nonzeros is cut into `units`
 *              equal pieces (nonzero-balanced decomposition); each piece
 *              writes the rows that end inside it and leaves a carry for its
 *              last, unfinished row; a fix-up adds carries in unit order.
 *   BSR        16x16 blocks, block-column ascending per block-row, values
 *              row-major within a block, zero fill; fp32 MFMA (or VALU).
 *   BELL       Blocked-ELL: BSR padded to the widest block-row (column -1,
 *              zero values for padding); same kernels as BSR.
 *   ELL        rows padded to the longest row, row-major [m][W], padding
 *              column -1 and value 0 (the rho_ELL representation of Eq.
 *              format-expansion; Appendix "Case Studies", uniform rows): a
 *              row's entries sit at row * W, so no row pointer is read.
 *   WIN        packed column windows (Sec. "Agentic Lowering and Refinement":
 *              packed column windows for SpMM, after Sextans; Appendix
 *              "Compilation-Plan Design Space", SpMM row: window descriptors,
 *              B staged in shared memory, C held in registers) over the
 *              CSR_SPLIT layout: heavy rows run as the split's chunks, and
 *              the light rows, in list order, are cut into windows of R list
 *              positions, one workgroup each.  A window stages the columns
 *              that two or more of its rows use (at most as many as fit
 *              16 KiB of LDS, the most used kept); their B rows are copied to
 *              LDS once per window and every use reads them there.  Each
 *              entry of the layout carries an int32 code: -2 - p for the
 *              window's staged column p, else the column read from B.
 *   SELL       SELL-C-sigma (Appendix "Compilation-Plan Design Space", SpMV
 *              row: slice height C, sort window sigma).  Rows are sorted by
 *              non-increasing length inside windows of sigma rows (stable);
 *              slices of C sorted rows are padded to their longest row and
 *              stored row-major (one lane group loads a row's entries
 *              contiguously; the classic layout is column-major, for one row
 *              per SIMD lane).  C is the rows one wave64 processes (64/G). */
typedef enum {
  SD_FMT_AUTO = 0,
  SD_FMT_CSR_ROW = 1,
  SD_FMT_CSR_SPLIT = 2,
  SD_FMT_CSR_MERGE = 3,
  SD_FMT_BSR = 4,
  SD_FMT_BELL = 5,
  SD_FMT_ELL = 6,
  SD_FMT_WIN = 7,
  SD_FMT_SELL = 8
} sd_format_t;

/* BSR / BELL engine.  MFMA (fp32 matrix cores) serves any width: column tiles
 * of 64, 32 and 16 (the last one partial) with 16-byte aligned B and C, and
 * 16-column tiles of single floats otherwise.  VALU: one FMA per lane per
 * block entry. */
typedef enum { SD_ENGINE_AUTO = 0, SD_ENGINE_MFMA = 1, SD_ENGINE_VALU = 2 } sd_engine_t;

/* Options; zero-initialised fields take their defaults. */
typedef struct {
  int32_t force;           /* sd_format_t; SD_FMT_AUTO lets the planner choose */
  int32_t heavy_threshold; /* CSR_SPLIT: T, rows with r >= T are split (0 = planner default) */
  int32_t chunk_nnz;       /* CSR_SPLIT: c, nonzeros per chunk (0 = default) */
  int32_t units;           /* CSR_MERGE: U, number of path pieces (0 = default) */
  int32_t engine;          /* sd_engine_t for BSR/BELL */
  int32_t transpose;       /* nonzero: the plan computes C = A^T B (A^T materialised) */
  int32_t placement;       /* 0 = current HIP device (default), 1 = device `device`,
                              2 = host only: no device memory and no HIP call;
                              sd_spmm returns SD_ERR_NO_DEVICE, info and export work */
  int32_t device;          /* HIP device ordinal when placement == 1 */
  int32_t dense_threshold; /* passed to the analysis (0 = 128) */
  int32_t rows_per_group;  /* CSR_ROW / CSR_SPLIT light rows: rows batched by one lane
                              group, 1, 2 or 4.  ELL: rows one lane group walks in turn,
                              loading the next row's entries while the current row's
                              gathers are in flight, 1, 2, 4, 8 or 16 (0 = planner default) */
  int32_t gather_unroll;   /* B-row gathers per row issued before the FMAs, 4 or 8
                              (0 = planner default) */
  int32_t cache_policy;    /* CSR_MERGE B-row gathers: 0 = planner default, 1 = normal
                              loads, 2 = tiered (rows of hot columns normal, the rest
                              non-temporal), 3 = all non-temporal */
  int32_t hot_budget_kib;  /* tiered policy: bytes of B rows kept hot, in KiB (0 = default) */
  int32_t search;          /* nonzero: measured plan selection (the paper keeps, for reuse,
                              the quickest candidate that passes validation: Introduction,
                              and Sec. "Architecture-Aware Compilation-Plan Synthesis"
                              on returning the fastest valid branch): build a
                              bounded set of candidate plans, time each on the device with
                              scratch operands, check each against the rule-based plan on
                              sampled rows, keep the fastest.  The choice is cached in the
                              process by (structure hash, m, k, nnz, n, transpose, device).
                              Needs a device; the other fields are ignored. */
  int32_t col_tile;        /* CSR and ELL families: dense columns per lane group (the K-tile
                              width of the paper's SpMM hardware mapping), a power of two
                              >= 4; the dense width is processed in ceil(n / col_tile)
                              column passes (0 = the whole width, up to 256) */
  int32_t window_rows;     /* WIN: light rows per window R, >= 1 (0 = 64); a window
                              stages at most the columns whose B rows fit 16 KiB of
                              LDS, its most used */
  int32_t wg_order;        /* workgroup order of the row, merge and block kernels over the
                              8 XCDs (each with its own L2): 0 = planner default,
                              1 = each XCD takes one contiguous range of rows,
                              2 = the hardware's round-robin (all XCDs on one band of
                              rows, sharing what they fetch through the Infinity Cache),
                              3 = round-robin over chunks of wg_chunk consecutive
                              workgroups (each XCD a contiguous sub-band, neighbouring XCDs
                              the adjacent ones) */
  int32_t wg_chunk;        /* wg_order 3: workgroups per chunk, >= 2 (0 = 64) */
  int32_t sell_sigma;      /* SELL: sort window in rows, >= 1 (0 = 8 slices) */
  int32_t row_slices;      /* CSR_ROW / CSR_SPLIT at narrow widths (lanes per row G <= 8,
                              i.e. n <= 32 with 128-bit accesses): lane groups that share
                              one row (or chunk), each taking every row_slices-th nonzero,
                              their partial sums added across lanes in a fixed order.
                              A power of two with G * row_slices <= 64; 1 = one lane group
                              per row (0 = planner default) */
  int32_t light_order;     /* CSR_SPLIT: order in which the light rows are processed
                              (the output is the same): 1 = ascending row, 2 = by the
                              column of the row's last nonzero, ties by row (rows whose
                              largest columns agree run together; an empty row last);
                              0 = planner default (2) */
  int32_t chunk_order;     /* CSR_SPLIT: order in which the heavy rows' chunks are processed
                              (the output is the same: each row still adds its chunks'
                              partial sums in one fixed order): 1 = chunk-list order (ascending
                              row, then position), 2 = by the column of the chunk's middle
                              entry (the one at floor((begin + end) / 2)), ties by chunk
                              index, so chunks of different rows that cover the same
                              columns run together; 0 = planner default (2) */
} sd_plan_opts_t;

typedef struct sd_plan_s *sd_plan_t;

/* Builds a plan for dense width n: validates A, analyses it, picks a family
 * (or takes opts->force), sizes it (footprints, legality against the device's
 * thread/register/LDS limits), converts A on the host and copies the plan's
 * arrays to device memory once.  A may be freed afterwards.
 * Errors: SD_ERR_INVALID_VALUE (null A/out, n < 1, bad option),
 * SD_ERR_INVALID_CSR, SD_ERR_OVERFLOW, SD_ERR_UNSUPPORTED (forced family
 * infeasible), SD_ERR_OUT_OF_MEMORY, SD_ERR_HIP.  *out is set only on SD_OK. */
int sd_plan(const sd_csr_t *A, int32_t n, sd_plan_t *out);
int sd_plan_ex(const sd_csr_t *A, int32_t n, const sd_plan_opts_t *opts, sd_plan_t *out);

/* sd_plan_ex for a matrix already in device memory (the preparation stage of
 * Sec. "Architecture-Aware Compilation-Plan Synthesis" moved next to the
 * data): A->rowptr, A->colidx and A->values are device pointers of the
 * current HIP device, read on `stream` (a hipStream_t; NULL = the null stream)
 * after the caller's earlier work there.  The statistics come from
 * sd_analyze_device (of A^T for a transpose plan, itself built on the device
 * once A has passed the checks); every family is then built by HIP kernels
 * straight into the plan's device memory (info.device_built = 1).  A search
 * (opts->search) times its candidates the same way, built from device memory,
 * and shares the choice cache with sd_plan_ex (the same key for the same
 * pattern).  Only placement != 0 copies A to the host and calls sd_plan_ex.  Either way the plan's info, exports and results are
 * those sd_plan_ex gives for the same matrix and options.  A is not kept and
 * may be freed once this returns; the call waits for `stream`.
 * Errors: as sd_plan_ex (the CSR checks of sd_analyze_device run on the
 * device), SD_ERR_NO_DEVICE (no HIP device). */
int sd_plan_device(const sd_csr_t *A, int32_t n, const sd_plan_opts_t *opts, void *stream, sd_plan_t *out);

/* C = A.B (C = A^T.B for a transpose plan), enqueued on `stream` (a
 * hipStream_t; NULL = the null stream); returns without waiting.
 * B: device, rows_B x n row-major, leading dimension n (rows_B = k, or m for
 * a transpose plan).  C: device, rows_C x n row-major (rows_C = m, or k), fully
 * overwritten (no accumulation).  B and C must not overlap (checked:
 * SD_ERR_INVALID_VALUE).  B and C are used
 * with 128-bit accesses when both are 16-byte aligned and n % 4 == 0, else
 * with 32-bit accesses.  No allocation, no host synchronisation, no memset:
 * the call may be captured into a HIP graph and replayed (the plan's
 * workspace is fixed at plan time; replays on one plan must not overlap).
 * Errors: SD_ERR_INVALID_VALUE (null plan/pointers, overlapping B and C), SD_ERR_NO_DEVICE,
 * SD_ERR_HIP (launch failure; the stream's state is whatever HIP reports). */
int sd_spmm(sd_plan_t plan, const float *B, float *C, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): C = A.B by
 * the CSR_MERGE family's kernels, straight from a CSR in device memory, with
 * no plan and no allocation.  A->rowptr, A->colidx and A->values are device
 * pointers of the current HIP device; A must follow the rules of sd_csr_t,
 * which this call does not check (sd_analyze_device checks a pattern once).
 * B: device, k x n row-major; C: device, m x n row-major, fully overwritten;
 * they must not overlap.  units: merge-path pieces (0 = the planner's default,
 * halved until they fit the scratch).
 * The split coordinates and the pieces' carry and head partials live in a
 * library-owned device array of 16 MiB per device (held until the process
 * ends), which needs 8 (units + 1) + 8 units + 8 n units bytes (each of the
 * first two parts rounded up to 256): SD_ERR_UNSUPPORTED when that exceeds
 * 16 MiB.  Every call on one device shares that array, and each call writes
 * every part of it that it reads, so calls need no clearing between them; but
 * calls that overlap on one device race (issue them on one stream, or
 * synchronise between streams).  Enqueued on `stream` (NULL = null stream);
 * returns without waiting; calls no hipMalloc, hipFree or allocating library
 * routine.  The same units give the same bits as sd_spmm on a CSR_MERGE plan
 * with those units.
 * Errors: SD_ERR_INVALID_VALUE (null pointers, n < 1, units < 0, negative
 * sizes, overlapping B and C), SD_ERR_OVERFLOW (nnz >= 2^31),
 * SD_ERR_UNSUPPORTED (scratch too small for units and n), SD_ERR_NO_DEVICE,
 * SD_ERR_HIP. */
int sd_spmm_merge_noalloc(const sd_csr_t *A, int32_t n, int32_t units, const float *B, float *C, void *stream);

typedef struct {
  int32_t family;          /* sd_format_t actually used */
  int32_t engine;          /* sd_engine_t actually used (BSR/BELL) */
  int32_t transpose;
  int32_t device;          /* -1 for host-only plans */
  int64_t m, k, n, nnz;    /* of the operand the kernels see (A^T for a transpose plan) */
  int64_t heavy_threshold, chunk_nnz, n_light, n_heavy, n_chunks;
  int64_t units, merge_len;
  int64_t block, nnzb, bell_width, block_rows;
  /* Workload-scale analysis (Eqs. representation-footprint, candidate-working-set,
   * l2-scale-ratios), bytes: */
  int64_t m_rep;           /* stored values + metadata of the representation */
  int64_t workspace;       /* W: temporary storage of the dataflow */
  int64_t d_r, d_s;        /* dense operand B and output C */
  int64_t m_r, m_t;        /* m_rep + W + D_R, and m_r + D_S */
  int64_t compulsory_bytes;/* 8 nnz + 4 (m + 1) + 4 k n + 4 m n: the traffic model */
  int64_t l2_bytes, mall_bytes;
  double q_r, q_t;         /* m_r / l2_bytes, m_t / l2_bytes */
  double q_r_mall, q_t_mall;
  int64_t work_units;      /* rows, chunks + light rows, path pieces, or block-rows */
  double units_per_cu;
  int32_t cu_count;
  /* Hardware mapping legality (Eq. resource-bounds) for the main kernel: */
  int32_t block_threads, max_threads, regs_per_thread, lds_bytes, max_lds_bytes;
  int32_t legal;           /* 1 if block_threads <= max_threads, regs * threads within the
                              register file and lds_bytes <= max_lds_bytes */
  int32_t rows_per_group;  /* rows batched per lane group by the row kernels */
  int32_t lanes_per_row;   /* G: lanes of a wave64 that share one row */
  int32_t gather_unroll;   /* B-row gathers per row per batch */
  int32_t cache_policy;    /* policy used (1 normal, 2 tiered, 3 non-temporal; 0 = not a CSR plan) */
  int32_t row_slices;      /* CSR_ROW / CSR_SPLIT: lane groups sharing a row (1 = none) */
  int32_t light_order;     /* CSR_SPLIT: light-row order used (1 ascending, 2 by last column) */
  int32_t chunk_order;     /* CSR_SPLIT: chunk order used (1 chunk list, 2 by middle column) */
  int32_t reserved[1];
  int64_t hot_columns;     /* tiered policy: columns whose B rows are gathered with normal loads */
  int64_t hot_nnz;         /* nonzeros in those columns */
  int64_t ell_width;       /* ELL: slots per row (= longest row) */
  int32_t search_candidates; /* plans timed by the search (0: no search) */
  int32_t search_cache_hit;  /* 1 if the choice came from the in-process cache */
  double search_best_ms;     /* measured time of the chosen plan (ms per sd_spmm) */
  double search_rule_ms;     /* measured time of the rule-based plan */
  int32_t col_tile;          /* dense columns per lane group (CSR and ELL families) */
  int32_t col_passes;        /* column passes over the dense width */
  int32_t window_rows;       /* WIN: rows per window R */
  int32_t window_max;        /* WIN: most staged columns in one window (sets the LDS size) */
  int64_t window_staged;     /* WIN: staged columns over all windows (B rows copied to LDS) */
  int64_t window_staged_uses;/* WIN: nonzeros whose B row is read from LDS */
  int32_t wg_order;          /* 1 contiguous rows per XCD, 2 round-robin, 3 chunked round-robin */
  int32_t wg_chunk;          /* wg_order 3: workgroups per chunk */
  int32_t device_built;      /* 1 if sd_plan_device built the representation on the device */
  int32_t reserved2[1];
  int64_t reach;             /* ELL / CSR_ROW: median over rows of the largest |column - row|
                                (sets the default chunked order; 0 if not computed) */
  int32_t sell_c;            /* SELL: slice height C (rows per slice) */
  int32_t sell_sigma;        /* SELL: sort window */
  int64_t sell_slices;       /* SELL: number of slices */
  int64_t sell_slots;        /* SELL: stored slots, padding included */
} sd_plan_info_t;

int sd_plan_info(sd_plan_t plan, sd_plan_info_t *out);

/* Copies one of the plan's converted arrays into host memory, for bit-exact
 * checks.  `bytes` must be at least the array's size (sd_plan_export_size). */
typedef enum {
  SD_EXPORT_ROWPTR = 1,       /* int32 [m+1]   (of A, or A^T for a transpose plan).  A CSR_SPLIT
                                 or WIN plan holds the split layout instead: ROWPTR [n_light+1]
                                 points by list position over the light rows (in LIGHT_ROWS
                                 order), whose entries come first in COLIDX / VALUES, followed
                                 by the heavy rows' entries in ascending row order (WIN: the
                                 columns are exported as WIN_CODE) */
  SD_EXPORT_COLIDX = 2,       /* int32 [nnz] */
  SD_EXPORT_VALUES = 3,       /* fp32  [nnz] */
  SD_EXPORT_LIGHT_ROWS = 4,   /* int32 [n_light]          CSR_SPLIT */
  SD_EXPORT_CHUNKS = 5,       /* int32 [n_chunks][3]      CSR_SPLIT: (row, begin, end), begin and
                                 end in the split layout's coordinates */
  SD_EXPORT_MERGE_COORDS = 6, /* int32 [units+1][2]       CSR_MERGE: (rows, nonzeros) consumed */
  SD_EXPORT_BLOCK_PTR = 7,    /* int32 [block_rows+1]     BSR */
  SD_EXPORT_BLOCK_COL = 8,    /* int32 [nnzb] (BSR) or [block_rows][bell_width] (BELL, -1 pad) */
  SD_EXPORT_BLOCK_VAL = 9,    /* fp32  [slots][16][16], row-major within a block */
  SD_EXPORT_ELL_COL = 10,     /* int32 [m][ell_width]      ELL, -1 = padding */
  SD_EXPORT_ELL_VAL = 11,     /* fp32  [m][ell_width]      ELL, 0 = padding */
  SD_EXPORT_WIN_PTR = 12,     /* int32 [windows+1]         WIN: staged-column range per window
                                 (windows = ceil(n_light / window_rows)) */
  SD_EXPORT_WIN_COLS = 13,    /* int32 [window_staged]     WIN: staged columns, ascending per window */
  SD_EXPORT_WIN_CODE = 14,    /* int32 [nnz]               WIN: per entry of the split layout, -2 - p
                                 for staged column p, else the column */
  SD_EXPORT_WIN_VAL = 15,     /* fp32  [nnz]               WIN: the split layout's values */
  SD_EXPORT_SELL_PERM = 16,   /* int32 [m]                 SELL: original row of each sorted row */
  SD_EXPORT_SELL_SLICE_PTR = 17, /* int64 [sell_slices+1] SELL: first slot of each slice */
  SD_EXPORT_SELL_COL = 18,    /* int32 [sell_slots]        SELL, -1 = padding */
  SD_EXPORT_SELL_VAL = 19,    /* fp32  [sell_slots]        SELL, 0 = padding */
  SD_EXPORT_CHUNK_ORDER = 20  /* int32 [n_chunks]          CSR_SPLIT: chunk indices in processing order */
} sd_export_t;

int sd_plan_export_size(sd_plan_t plan, int32_t what, size_t *bytes);
int sd_plan_export(sd_plan_t plan, int32_t what, void *host_dst, size_t bytes);

/* Empties the in-process cache of measured plan choices. */
void sd_plan_cache_clear(void);

/* Keyed reuse of measured choices across processes (the paper keeps the
 * fastest valid plan found for an input and reuses it; Sec.
 * "Architecture-Aware Compilation-Plan Synthesis").  A search (opts->search)
 * records, per key, the options of the plan it chose; the key hashes A's
 * sizes and pattern (row pointers and columns, not values), n, the transpose
 * flag and the device's architecture name, CU count, L2 and LDS sizes.
 *
 * sd_plan_cache_size: number of recorded choices.
 * sd_plan_cache_save: writes every recorded choice to `path` (created or
 *   replaced; native byte order, so a file is for machines of the same
 *   endianness).
 * sd_plan_cache_load: adds the choices in a file written by
 *   sd_plan_cache_save, replacing recorded choices with the same key; later
 *   searches with a matching key build the recorded plan without timing
 *   (info.search_cache_hit = 1).  The file is checked as a whole before
 *   anything is added.
 * Host-only.  Errors: SD_ERR_INVALID_VALUE (null argument), SD_ERR_IO (cannot
 * open, read or write; wrong tag, record size or length; a record that is not
 * a valid plan choice), SD_ERR_OUT_OF_MEMORY. */
int sd_plan_cache_size(int64_t *entries);
int sd_plan_cache_save(const char *path);
int sd_plan_cache_load(const char *path);

/* Frees the plan's host and device memory.  NULL is a no-op.  The caller must
 * make sure no sd_spmm on this plan is still running (synchronise its stream). */
void sd_plan_destroy(sd_plan_t plan);

/* Static strings; never NULL. */
const char *sd_status_string(int status);
/* The last HIP error text seen by this thread ("" if none). */
const char *sd_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SPARSEDITTO_H */
