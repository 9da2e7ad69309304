// Device-side structural analysis (sd_analyze_device): the statistics of
// sd_analyze for a CSR matrix whose arrays live in device memory.
//
// The kernels compute only exact integer aggregates (counts, sums, maxima,
// histograms); the host turns them into sd_stats_t with the same finishing
// step as the host analysis, so both give bit-identical statistics.
//
//  * rows      one thread per row: length, log2 histogram, squares, span,
//              column gaps, row-pointer checks;
//  * nonzeros  one thread per 16 consecutive nonzeros (one binary search for
//              the first row, then a walk): column range and ascending-order
//              checks, column degrees, the diagonal, and for b in {4, 8, 16}
//              whether the nonzero is the first of its b x b block (no smaller
//              column of the same block in its row, and none of the block's
//              columns in the earlier rows of its block-row, by binary search).
//              The first nonzero of a 16x16 block also counts the block's
//              nonzeros (binary searches in the block-row's 16 rows) for the
//              fill histogram, the dense-tile counters and the block-row width;
//  * slices    one thread per slice of c rows for the SELL-c slot counts;
//  * quartiles histograms of row lengths and spans, read back and walked on
//              the host (lower nearest rank, as on the host).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <vector>

#include "sd_internal.h"

namespace {

typedef unsigned long long u64;

struct DevAgg {
  u64 row_sumsq, col_sumsq, span_sum, nonempty, gap_num, gap_den, diag, empty;
  u64 nnzb[3], dense_tiles, dense_nnz, sell_slots[3];
  u64 row_hist[33], fill16_hist[8];
  int32_t rmax, rmin, smax, dmax, width16, bad;
};

__device__ __forceinline__ int log2_bin_dev(int64_t r) {
  int t = 0;
  while (t < 32 && r >= ((int64_t)1 << t)) ++t;
  return t;
}

// smallest p in [lo, hi) with col[p] >= v (hi if none)
__device__ __forceinline__ int32_t lower_bound_dev(const int32_t *__restrict__ col, int32_t lo, int32_t hi, int32_t v) {
  while (lo < hi) {
    const int32_t mid = lo + ((hi - lo) >> 1);
    if (col[mid] < v) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Wave-wide reductions (every lane of the wave must call them): the shared
// counters get one atomic per wave instead of one per thread, which matters
// on millions of rows.
__device__ __forceinline__ u64 wave_sum(u64 v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ int32_t wave_max(int32_t v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ int32_t wave_min(int32_t v) {
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ void add_once(u64 *dst, u64 v) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0 && v) atomicAdd(dst, v);
}

// Histogram update with equal values combined across the wave: the lanes
// holding the leader's value add their count with one atomic (a stencil's
// rows mostly share one length and one span).  Every lane must call it.
__device__ __forceinline__ void wave_hist_add(u64 *__restrict__ hist, int64_t v, bool valid) {
  uint64_t pending = __ballot(valid);
  while (pending) {
    const int leader = __ffsll((long long)pending) - 1;
    const int64_t lv = __shfl(v, leader, 64);
    const uint64_t same = __ballot(valid && v == lv) & pending;
    if ((threadIdx.x & 63) == leader) atomicAdd(&hist[lv], (u64)__popcll(same));
    pending &= ~same;
  }
}

__global__ __launch_bounds__(256) void k_an_rows(const int32_t *__restrict__ rowptr, const int32_t *__restrict__ colidx,
                                                 int32_t m, int64_t nnz, DevAgg *__restrict__ agg) {
  __shared__ u64 hist[33];
  for (int t = threadIdx.x; t < 33; t += 256) hist[t] = 0;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  u64 sumsq = 0, empty = 0, nonempty = 0, span_sum = 0, gap_num = 0, gap_den = 0;
  int32_t rmax = 0, rmin = INT32_MAX, smax = 0, bad = 0;
  if (i < m) {
    const int32_t p0 = rowptr[i], p1 = rowptr[i + 1];
    if (p1 < p0 || p0 < 0 || (int64_t)p1 > nnz) {
      bad = 1;
    } else {
      const int64_t r = p1 - p0;
      atomicAdd(&hist[log2_bin_dev(r)], 1ull);
      sumsq = (u64)(r * r);
      rmax = (int32_t)r;
      rmin = (int32_t)r;
      if (r == 0) {
        empty = 1;
      } else {
        const int64_t span = (int64_t)colidx[p1 - 1] - colidx[p0] + 1;
        nonempty = 1;
        span_sum = (u64)span;
        smax = (int32_t)span;
        if (r >= 2) {
          gap_num = (u64)(span - 1);
          gap_den = (u64)(r - 1);
        }
      }
    }
  }
  add_once(&agg->row_sumsq, sumsq);
  add_once(&agg->empty, empty);
  add_once(&agg->nonempty, nonempty);
  add_once(&agg->span_sum, span_sum);
  add_once(&agg->gap_num, gap_num);
  add_once(&agg->gap_den, gap_den);
  rmax = wave_max(rmax);
  rmin = wave_min(rmin);
  smax = wave_max(smax);
  bad = wave_max(bad);
  if ((threadIdx.x & 63) == 0) {
    atomicMax(&agg->rmax, rmax);
    atomicMin(&agg->rmin, rmin);
    atomicMax(&agg->smax, smax);
    if (bad) atomicOr(&agg->bad, 1);
  }
  __syncthreads();
  for (int t = threadIdx.x; t < 33; t += 256)
    if (hist[t]) atomicAdd(&agg->row_hist[t], hist[t]);
}

// Second row pass, once the maxima are known: histograms of lengths and spans.
__global__ __launch_bounds__(256) void k_an_row_hists(const int32_t *__restrict__ rowptr,
                                                      const int32_t *__restrict__ colidx, int32_t m,
                                                      u64 *__restrict__ lhist, u64 *__restrict__ shist) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  int64_t len = 0, span = 0;
  if (i < m) {
    const int32_t p0 = rowptr[i], p1 = rowptr[i + 1];
    len = p1 - p0;
    if (p1 > p0) span = (int64_t)colidx[p1 - 1] - colidx[p0] + 1;
  }
  wave_hist_add(lhist, len, i < m);
  wave_hist_add(shist, span, i < m && len > 0);
}

constexpr int kPerThread = 16;  // nonzeros walked by one thread

__global__ __launch_bounds__(256) void k_an_nnz(const int32_t *__restrict__ rowptr, const int32_t *__restrict__ colidx,
                                                int32_t m, int32_t k, int64_t nnz, int32_t dense_threshold,
                                                int32_t *__restrict__ deg, int32_t *__restrict__ bwidth,
                                                DevAgg *__restrict__ agg) {
  const int64_t p_begin = ((int64_t)blockIdx.x * 256 + threadIdx.x) * kPerThread;
  const int64_t p_end = min(nnz, p_begin + kPerThread);
  u64 diag = 0, nb[3] = {0, 0, 0}, dense_tiles = 0, dense_nnz = 0, fh[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  int32_t bad = 0;
  if (p_begin < nnz) {
    // row of p_begin: the last i with rowptr[i] <= p_begin (rows may be empty)
    int32_t lo = 0, hi = m;
    while (lo < hi) {
      const int32_t mid = lo + ((hi - lo + 1) >> 1);
      if (rowptr[mid] <= p_begin) lo = mid;
      else hi = mid - 1;
    }
    int32_t row = lo;
    int32_t bw_row = -1, bw_count = 0;  // 16x16 blocks found in block-row bw_row, flushed on change
    for (int64_t p = p_begin; p < p_end; ++p) {
      while (row < m - 1 && rowptr[row + 1] <= p) ++row;
      const int32_t c = colidx[p];
      const int32_t rs = rowptr[row];
      if (c < 0 || c >= k || (p > rs && colidx[p - 1] >= c)) {
        bad = 1;
        continue;
      }
      atomicAdd(&deg[c], 1);
      diag += (c == row);
      const int32_t bsz[3] = {4, 8, 16};
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const int32_t b = bsz[t];
        const int32_t bc = c / b;
        if (p > rs && colidx[p - 1] / b == bc) continue;  // not the first of its block in this row
        const int32_t r0 = row / b * b;
        bool first = true;
        for (int32_t rr = r0; rr < row && first; ++rr) {
          const int32_t q = lower_bound_dev(colidx, rowptr[rr], rowptr[rr + 1], bc * b);
          if (q < rowptr[rr + 1] && colidx[q] < bc * b + b) first = false;
        }
        if (!first) continue;
        ++nb[t];
        if (b == 16) {
          int32_t f = 0;
          const int32_t r1 = min(m, r0 + 16);
          for (int32_t rr = r0; rr < r1; ++rr) {
            const int32_t a = lower_bound_dev(colidx, rowptr[rr], rowptr[rr + 1], bc * 16);
            const int32_t e = lower_bound_dev(colidx, a, rowptr[rr + 1], bc * 16 + 16);
            f += e - a;
          }
          if (f < 1 || f > 256) {  // only an unsorted row (an invalid matrix) gets here
            bad = 1;
            continue;
          }
          ++fh[(f - 1) / 32];
          if (f >= dense_threshold) {
            ++dense_tiles;
            dense_nnz += (u64)f;
          }
          if (row / 16 != bw_row) {
            if (bw_count) atomicAdd(&bwidth[bw_row], bw_count);
            bw_row = row / 16;
            bw_count = 0;
          }
          ++bw_count;
        }
      }
    }
    if (bw_count) atomicAdd(&bwidth[bw_row], bw_count);
  }
  bad = wave_max(bad);
  if ((threadIdx.x & 63) == 0 && bad) atomicOr(&agg->bad, 1);
  add_once(&agg->diag, diag);
  for (int t = 0; t < 3; ++t) add_once(&agg->nnzb[t], nb[t]);
  add_once(&agg->dense_tiles, dense_tiles);
  add_once(&agg->dense_nnz, dense_nnz);
  for (int t = 0; t < 8; ++t) add_once(&agg->fill16_hist[t], fh[t]);
}

__global__ __launch_bounds__(256) void k_an_cols(const int32_t *__restrict__ deg, int32_t k, DevAgg *__restrict__ agg) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t d = j < k ? deg[j] : 0;
  add_once(&agg->col_sumsq, (u64)(d * d));
  const int32_t mx = wave_max((int32_t)d);
  if ((threadIdx.x & 63) == 0 && mx) atomicMax(&agg->dmax, mx);
}

__global__ __launch_bounds__(256) void k_an_width(const int32_t *__restrict__ bwidth, int32_t mb,
                                                  DevAgg *__restrict__ agg) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int32_t mx = wave_max(j < mb ? bwidth[j] : 0);
  if ((threadIdx.x & 63) == 0 && mx) atomicMax(&agg->width16, mx);
}

__global__ __launch_bounds__(256) void k_an_sell(const int32_t *__restrict__ rowptr, int32_t m, int32_t c, int t,
                                                 DevAgg *__restrict__ agg) {
  const int64_t s0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * c;
  u64 slots = 0;
  if (s0 < m) {
    const int64_t s1 = min((int64_t)m, s0 + c);
    int32_t mx = 0;
    for (int64_t i = s0; i < s1; ++i) mx = max(mx, rowptr[i + 1] - rowptr[i]);
    slots = (u64)((s1 - s0) * mx);
  }
  add_once(&agg->sell_slots[t], slots);
}

uint32_t grid_for(int64_t items) { return (uint32_t)((items + 255) / 256); }

struct DevBuf {
  void *p = nullptr;
  ~DevBuf() {
    if (p) (void)hipFree(p);
  }
};

// Declared after the buffers it protects, so it is destroyed first: every
// return waits for the stream before the buffers are freed (an early error
// return may leave kernels that use them in flight).
struct StreamDrain {
  hipStream_t s;
  ~StreamDrain() { (void)hipStreamSynchronize(s); }
};

int hip_status(hipError_t e) {
  if (e == hipSuccess) return SD_OK;
  return e == hipErrorOutOfMemory ? SD_ERR_OUT_OF_MEMORY : SD_ERR_HIP;
}

}  // namespace

namespace sd {

int analyze_device(const sd_csr_t *A, int32_t dense_threshold, sd_stats_t *out, hipStream_t s) {
  if (!A || !out) return SD_ERR_INVALID_VALUE;
  if (dense_threshold == 0) dense_threshold = 128;
  if (dense_threshold < 1 || dense_threshold > 256) return SD_ERR_INVALID_VALUE;
  const int32_t m = A->m, k = A->k;
  const int64_t nnz = A->nnz;
  if (m < 0 || k < 0 || nnz < 0) return SD_ERR_INVALID_CSR;
  if (nnz >= ((int64_t)1 << 31)) return SD_ERR_OVERFLOW;
  if (!A->rowptr || (nnz > 0 && (!A->colidx || !A->values))) return SD_ERR_INVALID_VALUE;
  if (nnz > 0 && (m == 0 || k == 0)) return SD_ERR_INVALID_CSR;
  // rowptr[0] == 0 and rowptr[m] == nnz
  int32_t ends[2] = {0, 0};
  hipError_t e = hipMemcpyAsync(&ends[0], A->rowptr, sizeof(int32_t), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipMemcpyAsync(&ends[1], A->rowptr + m, sizeof(int32_t), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_status(e);
  if (ends[0] != 0 || ends[1] != nnz) return SD_ERR_INVALID_CSR;

  DevBuf agg_b, deg_b, bw_b, lh_b, sh_b;
  StreamDrain drain{s};
  const int32_t mb16 = (m + 15) / 16;
  if ((e = hipMalloc(&agg_b.p, sizeof(DevAgg))) != hipSuccess) return hip_status(e);
  if ((e = hipMalloc(&deg_b.p, sizeof(int32_t) * (size_t)std::max(1, k))) != hipSuccess) return hip_status(e);
  if ((e = hipMalloc(&bw_b.p, sizeof(int32_t) * (size_t)std::max(1, mb16))) != hipSuccess) return hip_status(e);
  DevAgg init;
  std::memset(&init, 0, sizeof(init));
  init.rmin = m > 0 ? INT32_MAX : 0;
  DevAgg *agg = static_cast<DevAgg *>(agg_b.p);
  int32_t *deg = static_cast<int32_t *>(deg_b.p), *bw = static_cast<int32_t *>(bw_b.p);
  if ((e = hipMemcpyAsync(agg, &init, sizeof(init), hipMemcpyHostToDevice, s)) != hipSuccess ||
      (e = hipMemsetAsync(deg, 0, sizeof(int32_t) * (size_t)std::max(1, k), s)) != hipSuccess ||
      (e = hipMemsetAsync(bw, 0, sizeof(int32_t) * (size_t)std::max(1, mb16), s)) != hipSuccess)
    return hip_status(e);

  if (m > 0) hipLaunchKernelGGL(k_an_rows, dim3(grid_for(m)), dim3(256), 0, s, A->rowptr, A->colidx, m, nnz, agg);
  if ((e = hipGetLastError()) != hipSuccess) return hip_status(e);
  DevAgg h;
  if ((e = hipMemcpyAsync(&h, agg, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return hip_status(e);
  if (h.bad) return SD_ERR_INVALID_CSR;

  // column checks first: the block pass indexes rows by the (now checked) row pointers
  if (nnz > 0) {
    hipLaunchKernelGGL(k_an_nnz, dim3(grid_for((nnz + kPerThread - 1) / kPerThread)), dim3(256), 0, s, A->rowptr,
                       A->colidx, m, k, nnz, dense_threshold, deg, bw, agg);
    if ((e = hipGetLastError()) != hipSuccess) return hip_status(e);
  }
  // spans (which size and index the span histogram below) are only meaningful
  // once the columns have passed the checks
  if ((e = hipMemcpyAsync(&h, agg, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return hip_status(e);
  if (h.bad) return SD_ERR_INVALID_CSR;
  if (k > 0) hipLaunchKernelGGL(k_an_cols, dim3(grid_for(k)), dim3(256), 0, s, deg, k, agg);
  if (mb16 > 0) hipLaunchKernelGGL(k_an_width, dim3(grid_for(mb16)), dim3(256), 0, s, bw, mb16, agg);
  const int32_t cs[3] = {16, 32, 512};
  for (int t = 0; t < 3 && m > 0; ++t)
    hipLaunchKernelGGL(k_an_sell, dim3(grid_for(((int64_t)m + cs[t] - 1) / cs[t])), dim3(256), 0, s, A->rowptr, m,
                       cs[t], t, agg);
  if ((e = hipGetLastError()) != hipSuccess) return hip_status(e);

  // quartile histograms, sized by the maxima of the first pass
  const int64_t lh_n = (int64_t)h.rmax + 1, sh_n = (int64_t)h.smax + 1;
  std::vector<u64> lh((size_t)lh_n, 0), sh((size_t)sh_n, 0);
  if (m > 0) {
    if ((e = hipMalloc(&lh_b.p, sizeof(u64) * (size_t)lh_n)) != hipSuccess ||
        (e = hipMalloc(&sh_b.p, sizeof(u64) * (size_t)sh_n)) != hipSuccess ||
        (e = hipMemsetAsync(lh_b.p, 0, sizeof(u64) * (size_t)lh_n, s)) != hipSuccess ||
        (e = hipMemsetAsync(sh_b.p, 0, sizeof(u64) * (size_t)sh_n, s)) != hipSuccess)
      return hip_status(e);
    hipLaunchKernelGGL(k_an_row_hists, dim3(grid_for(m)), dim3(256), 0, s, A->rowptr, A->colidx, m,
                       static_cast<u64 *>(lh_b.p), static_cast<u64 *>(sh_b.p));
    if ((e = hipGetLastError()) != hipSuccess ||
        (e = hipMemcpyAsync(lh.data(), lh_b.p, sizeof(u64) * (size_t)lh_n, hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipMemcpyAsync(sh.data(), sh_b.p, sizeof(u64) * (size_t)sh_n, hipMemcpyDeviceToHost, s)) != hipSuccess)
      return hip_status(e);
  }
  if ((e = hipMemcpyAsync(&h, agg, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return hip_status(e);
  if (h.bad) return SD_ERR_INVALID_CSR;

  sd_stats_t st;
  std::memset(&st, 0, sizeof(st));
  st.m = m;
  st.k = k;
  st.nnz = nnz;
  st.dense_threshold = dense_threshold;
  st.row_min = m > 0 ? h.rmin : 0;
  st.row_max = h.rmax;
  st.empty_rows = (int64_t)h.empty;
  for (int t = 0; t < 33; ++t) st.row_hist[t] = (int64_t)h.row_hist[t];
  std::vector<int64_t> lhist(lh.begin(), lh.end()), shist(sh.begin(), sh.end());
  if (m > 0) {
    st.row_q25 = kth_from_hist(lhist, (int64_t)(m - 1) / 4);
    st.row_q50 = kth_from_hist(lhist, (int64_t)(m - 1) / 2);
    st.row_q75 = kth_from_hist(lhist, 3 * (int64_t)(m - 1) / 4);
  }
  if (h.nonempty > 0) st.row_span_median = kth_from_hist(shist, ((int64_t)h.nonempty - 1) / 2);
  st.col_deg_max = h.dmax;
  st.diag_nnz = (int64_t)h.diag;
  st.nnzb4 = (int64_t)h.nnzb[0];
  st.nnzb8 = (int64_t)h.nnzb[1];
  st.nnzb16 = (int64_t)h.nnzb[2];
  st.dense_tiles16 = (int64_t)h.dense_tiles;
  st.dense_tile_nnz16 = (int64_t)h.dense_nnz;
  st.bell16_width = h.width16;
  for (int t = 0; t < 8; ++t) st.fill16_hist[t] = (int64_t)h.fill16_hist[t];
  st.sell16_slots = (int64_t)h.sell_slots[0];
  st.sell32_slots = (int64_t)h.sell_slots[1];
  st.sell512_slots = (int64_t)h.sell_slots[2];
  StatsSums sum;
  sum.row_sumsq = (int64_t)h.row_sumsq;
  sum.col_sumsq = (int64_t)h.col_sumsq;
  sum.span_sum = (int64_t)h.span_sum;
  sum.nonempty = (int64_t)h.nonempty;
  sum.gap_num = (int64_t)h.gap_num;
  sum.gap_den = (int64_t)h.gap_den;
  finish_stats(sum, &st);
  *out = st;
  return SD_OK;
}

}  // namespace sd
