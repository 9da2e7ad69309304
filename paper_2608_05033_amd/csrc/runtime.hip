// C ABI of the SpMM library: plan construction (validation, analysis,
// family choice, conversion, footprints, legality, one upload to device
// memory) and the per-call sd_spmm launch on the caller's stream.
//
// Footprints follow Sec. "Architecture-Aware Compilation-Plan Synthesis":
// Eq. representation-footprint (M_rep = value slots x 4 B + metadata fields x
// their byte widths), Eq. candidate-working-set (M_R = M_rep + W + D_R,
// M_T = M_R + D_S with D_R = B and D_S = C for SpMM), Eq. l2-scale-ratios
// (q = M / C_L2) plus the same ratios against the 256 MiB Infinity Cache, the
// work units per compute unit, and the legality check of Eq. resource-bounds
// (threads, registers x threads, LDS) from the compiled kernel's attributes.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "kernels.h"
#include "sd_internal.h"

namespace {

thread_local std::string g_last_error;

int hip_fail(hipError_t e) {
  g_last_error = hipGetErrorString(e);
  return SD_ERR_HIP;
}

int hip_alloc_copy(sd_plan_s *p, void **dst, const void *src, size_t bytes) {
  if (bytes == 0) bytes = 4;  // keep every pointer valid
  void *d = nullptr;
  hipError_t e = hipMalloc(&d, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    g_last_error = hipGetErrorString(e);
    return e == hipErrorOutOfMemory ? SD_ERR_OUT_OF_MEMORY : SD_ERR_HIP;
  }
  p->allocations.push_back(d);
  *dst = d;
  if (src) {
    e = hipMemcpy(d, src, bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e);
  }
  return SD_OK;
}

template <typename T>
int upload(sd_plan_s *p, T **dst, const std::vector<T> &v) {
  return hip_alloc_copy(p, reinterpret_cast<void **>(dst), v.empty() ? nullptr : v.data(), v.size() * sizeof(T));
}

void release(sd_plan_s *p) {
  if (p->device >= 0 && !p->allocations.empty()) {
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(p->device);
    for (void *d : p->allocations) (void)hipFree(d);
    (void)hipSetDevice(cur);
  }
  p->allocations.clear();
}

struct DeviceGuard {
  int prev = -1;
  bool active = false;
  int enter(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) return SD_ERR_HIP;
    if (prev != dev) {
      hipError_t e = hipSetDevice(dev);
      if (e != hipSuccess) return hip_fail(e);
      active = true;
    }
    return SD_OK;
  }
  ~DeviceGuard() {
    if (active) (void)hipSetDevice(prev);
  }
};

// Returned by build_plan for a device source whose plan needs a host
// path (explicit placement); sd_plan_device then copies A to the host.  Not a
// public status.
constexpr int kNeedHost = -100;

// Median over non-empty rows of the row reach, from the device (the same
// lower median as median_row_reach on the host).
int device_median_reach(const sd_csr_t *dev, hipStream_t s, int64_t *out) {
  *out = 0;
  if (dev->m == 0) return SD_OK;
  int64_t *d = nullptr;
  hipError_t e = hipMalloc(&d, sizeof(int64_t) * (size_t)dev->m);
  if (e != hipSuccess) return hip_fail(e);
  std::vector<int64_t> h((size_t)dev->m);
  e = sd::dev_row_reach(dev->rowptr, dev->colidx, dev->m, d, s);
  if (e == hipSuccess) e = hipMemcpyAsync(h.data(), d, sizeof(int64_t) * h.size(), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  else (void)hipStreamSynchronize(s);  // nothing may still use d when it is freed
  (void)hipFree(d);
  if (e != hipSuccess) return hip_fail(e);
  h.erase(std::remove(h.begin(), h.end(), (int64_t)-1), h.end());
  if (h.empty()) return SD_OK;
  const size_t mid = (h.size() - 1) / 2;
  std::nth_element(h.begin(), h.begin() + (long)mid, h.end());
  *out = h[mid];
  return SD_OK;
}

// A^T of a device CSR, in device memory owned here; freed after the stream
// it was built on has drained.
struct DeviceTranspose {
  sd_csr_t csr{};
  hipStream_t s = nullptr;
  void *p[3] = {nullptr, nullptr, nullptr};
  ~DeviceTranspose() {
    if (p[0] || p[1] || p[2]) (void)hipStreamSynchronize(s);
    for (void *q : p)
      if (q) (void)hipFree(q);
  }
};

int device_transpose(const sd_csr_t *A, hipStream_t s, DeviceTranspose *T) {
  T->s = s;
  const size_t sizes[3] = {4 * ((size_t)A->k + 1), 4 * (size_t)std::max<int64_t>(1, A->nnz),
                           4 * (size_t)std::max<int64_t>(1, A->nnz)};
  for (int t = 0; t < 3; ++t) {
    hipError_t e = hipMalloc(&T->p[t], sizes[t]);
    if (e != hipSuccess) return hip_fail(e);
  }
  T->csr.m = A->k;
  T->csr.k = A->m;
  T->csr.nnz = A->nnz;
  T->csr.rowptr = static_cast<int32_t *>(T->p[0]);
  T->csr.colidx = static_cast<int32_t *>(T->p[1]);
  T->csr.values = static_cast<float *>(T->p[2]);
  hipError_t e = sd::dev_transpose(A->rowptr, A->colidx, A->values, A->m, A->k, A->nnz,
                                   const_cast<int32_t *>(T->csr.rowptr), const_cast<int32_t *>(T->csr.colidx),
                                   const_cast<float *>(T->csr.values), s);
  return e == hipSuccess ? SD_OK : hip_fail(e);
}

// dev != nullptr: A lives in device memory (dev's pointers, on the current
// device, stream ds); statistics come from the device analysis and the CSR,
// heavy-split, merge-path and ELL representations are built on the device.
// Packed column windows: the most staged columns one window may keep, those
// whose B rows (one tile of the dense width in the 128-bit geometry, never
// narrower than the 32-bit one used for unaligned B or C) fit the LDS budget.
int32_t window_cap(int32_t n, int32_t vec4, int32_t col_tile, int32_t max_lds) {
  const int64_t row_bytes = std::max<int64_t>(1, (int64_t)sd::window_lds_bytes(n, vec4, col_tile, 1));
  const int64_t budget = std::min<int64_t>(sd::kWindowLdsBudget, max_lds);
  return (int32_t)std::min<int64_t>(INT32_MAX, budget / row_bytes);
}

int build_plan(const sd_csr_t *A_in, int32_t n, const sd_plan_opts_t &o, sd_plan_s *p,
               const sd_csr_t *src = nullptr, hipStream_t ds = nullptr) {
  sd::CsrView A;
  int st;
  sd::CsrOwned At;
  sd_stats_t stats;
  DeviceTranspose Tt;
  if (src) {
    if (o.placement != 0) return kNeedHost;
    if (o.transpose) {  // A is checked (by its analysis) before it is transposed
      if ((st = sd::analyze_device(src, o.dense_threshold, &stats, ds)) != SD_OK) return st;
      if ((st = device_transpose(src, ds, &Tt)) != SD_OK) return st;
      src = &Tt.csr;
    }
    if ((st = sd::analyze_device(src, o.dense_threshold, &stats, ds)) != SD_OK) return st;
    A.m = src->m;  // sizes only: no host array is read on this path
    A.k = src->k;
    A.nnz = src->nnz;
  } else {
    st = sd::validate_csr(A_in, &A);
    if (st != SD_OK) return st;
    if (o.transpose) {
      st = sd::transpose(A, &At);
      if (st != SD_OK) return st;
      A = At.view();
    }
    st = sd::analyze(A, o.dense_threshold, &stats);
    if (st != SD_OK) return st;
  }

  // ---- device and its limits
  sd_plan_info_t &I = p->info;
  I.cu_count = sd::kDefaultCUs;
  I.l2_bytes = sd::kDefaultL2;
  I.max_threads = sd::kDefaultMaxThreads;
  I.max_lds_bytes = sd::kDefaultMaxLds;
  int32_t regs_per_cu = 512 * 64 * 4;  // VGPRs per CU (4 SIMDs x 512 x 64 lanes)
  p->device = -1;
  if (o.placement != 2) {
    int dev = 0;
    if (o.placement == 1) {
      int count = 0;
      hipError_t e = hipGetDeviceCount(&count);
      if (e != hipSuccess) return hip_fail(e);
      if (o.device < 0 || o.device >= count) return SD_ERR_INVALID_VALUE;
      dev = o.device;
    } else {
      hipError_t e = hipGetDevice(&dev);
      if (e != hipSuccess) return hip_fail(e);
    }
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return hip_fail(e);
    p->device = dev;
    I.cu_count = prop.multiProcessorCount;
    I.l2_bytes = prop.l2CacheSize;
    I.max_threads = prop.maxThreadsPerBlock;
    I.max_lds_bytes = (int32_t)prop.sharedMemPerBlock;
    regs_per_cu = prop.regsPerMultiprocessor > 0 ? prop.regsPerMultiprocessor : regs_per_cu;
  }
  I.device = p->device;

  // ---- family and parameters
  const int32_t vec4 = (n % 4 == 0) ? 1 : 0;
  // K tiles: when the dense operand is larger than half the Infinity Cache,
  // 64-column passes halve the gathered footprint per pass (measured on the
  // power-law workloads at N = 128: -10 to -14 %; no gain at N <= 64).
  int32_t col_tile = o.col_tile;
  if (col_tile == 0 && n > 64 && 4 * (int64_t)A.k * n > sd::kMallBytes / 2) col_tile = 64;
  const sd::Geometry geo = sd::geometry_for(n, vec4, col_tile);
  p->col_tile_req = col_tile;
  I.lanes_per_row = geo.G;
  I.col_tile = geo.G * geo.VW;
  I.col_passes = geo.coltiles;
  sd::PlanChoice pc = sd::choose_plan(stats, n, I.cu_count, geo.G, o);
  if (pc.family < SD_FMT_CSR_ROW || pc.family > SD_FMT_SELL) return SD_ERR_INVALID_VALUE;
  if (pc.T < 1 || pc.c < 1 || pc.U < 1) return SD_ERR_INVALID_VALUE;
  if (pc.engine < SD_ENGINE_AUTO || pc.engine > SD_ENGINE_VALU) return SD_ERR_INVALID_VALUE;
  I.family = pc.family;
  I.device_built = src ? 1 : 0;
  // Light rows by the column of their last nonzero unless asked otherwise:
  // measured with B streamed from HBM, R-MAT 2^20 at N = 128 ran 1.08 against
  // 1.18 ms and the four GCN products 13.9-14.1 against 14.3-14.4 ms (rows
  // whose largest, mostly cold, columns agree then share those B rows in L2).
  const int32_t light_order = o.light_order > 0 ? o.light_order : 2;
  const int32_t chunk_ord = o.chunk_order > 0 ? o.chunk_order : 2;
  I.wg_order = o.wg_order > 0 ? o.wg_order : pc.wg_order;
  I.wg_chunk = I.wg_order == 3 ? (o.wg_chunk >= 2 ? o.wg_chunk : 64) : 0;
  I.engine = (pc.family == SD_FMT_BSR || pc.family == SD_FMT_BELL) ? pc.engine : SD_ENGINE_AUTO;
  I.transpose = o.transpose ? 1 : 0;
  I.m = A.m;
  I.k = A.k;
  I.n = n;
  I.nnz = A.nnz;

  // ---- representation and partition, host side
  int64_t m_rep = 8 * A.nnz + 4 * ((int64_t)A.m + 1);  // CSR: fp32 value + int32 column per nonzero
  int64_t ws = 0;
  int64_t units = A.m;
  try {
    if (pc.family == SD_FMT_BSR || pc.family == SD_FMT_BELL) {
      const int64_t mb = (A.m + 15) / 16;
      const int64_t slots = pc.family == SD_FMT_BSR ? stats.nnzb16 : stats.bell16_width * mb;
      if (slots * 256 > ((int64_t)1 << 36)) return SD_ERR_UNSUPPORTED;  // > 256 GiB of block values
      int32_t width = 0;
      if (src) {
        // device copies carry one zero block (column -1) after the stored ones
        width = (int32_t)stats.bell16_width;
        const bool bsr = pc.family == SD_FMT_BSR;
        if ((bsr && (st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_bptr), nullptr, 4 * ((size_t)mb + 1))) !=
                        SD_OK) ||
            (st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_bcol), nullptr, 4 * ((size_t)slots + 1))) !=
                SD_OK ||
            (st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_bval), nullptr, 1024 * ((size_t)slots + 1))) !=
                SD_OK)
          return st;
        hipError_t e = sd::dev_block16(src->rowptr, src->colidx, src->values, A.m, A.k, A.nnz, stats.nnzb16,
                                       bsr ? -1 : width, bsr ? p->d_bptr : nullptr, p->d_bcol, p->d_bval, ds);
        if (e != hipSuccess) return hip_fail(e);
      } else {
        sd::block_convert(A, 16, pc.family == SD_FMT_BELL, &p->h_bptr, &p->h_bcol, &p->h_bval, &width);
        if (pc.family == SD_FMT_BELL) p->h_bptr.clear();
      }
      I.block = 16;
      I.nnzb = stats.nnzb16;
      I.bell_width = width;
      I.block_rows = mb;
      m_rep = slots * 256 * 4 + slots * 4 + (pc.family == SD_FMT_BSR ? 4 * (mb + 1) : 0);
      units = mb;
    } else if (pc.family == SD_FMT_ELL) {
      int32_t w = 0;
      if ((int64_t)A.m * std::max<int64_t>(1, stats.row_max) > ((int64_t)1 << 34)) return SD_ERR_UNSUPPORTED;
      if (src) {
        w = (int32_t)stats.row_max;
        const size_t slots = (size_t)A.m * (size_t)w;
        if ((st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_ecol), nullptr, 4 * slots)) != SD_OK ||
            (st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_eval), nullptr, 4 * slots)) != SD_OK)
          return st;
        hipError_t e = sd::dev_ell(src->rowptr, src->colidx, src->values, A.m, w, p->d_ecol, p->d_eval, ds);
        if (e != hipSuccess) return hip_fail(e);
      } else {
        sd::ell_convert(A, &p->h_ecol, &p->h_eval, &w);
      }
      I.ell_width = w;
      m_rep = 8 * (int64_t)A.m * w;
      // Rows per lane group, walked with the next row's entries loaded behind the
      // current gathers (when a row fits one entry load per lane, W <= G).  One
      // by default: with B streamed from HBM, more rows per group measured slower
      // on the 7-point Laplacian (40 vs 37 us at 4 rows).
      I.rows_per_group = o.rows_per_group > 0 ? o.rows_per_group : 1;
    } else if (pc.family == SD_FMT_SELL) {
      // slice height: the rows one wave processes in the 128-bit geometry
      const int32_t C = std::max(1, 64 / geo.G);
      const int32_t sigma = o.sell_sigma > 0 ? o.sell_sigma : 8 * C;
      I.sell_c = C;
      I.sell_sigma = sigma;
      I.sell_slices = ((int64_t)A.m + C - 1) / C;
      if (src) {
        auto alloc = [&](size_t bytes) -> void * {
          void *q = nullptr;
          return hip_alloc_copy(p, &q, nullptr, bytes) == SD_OK ? q : nullptr;
        };
        hipError_t e = sd::dev_sell(src->rowptr, src->colidx, src->values, A.m, (int32_t)stats.row_max, C, sigma,
                                    (int64_t)1 << 34, alloc, ds, &p->d_perm, &p->d_sptr, &p->d_ecol, &p->d_eval,
                                    &I.sell_slots);
        if (e != hipSuccess) return hip_fail(e);
      } else {
        sd::sell_convert(A, C, sigma, &p->h_perm, &p->h_sptr, &p->h_ecol, &p->h_eval);
        I.sell_slots = p->h_sptr.back();
      }
      if (I.sell_slots > ((int64_t)1 << 34)) return SD_ERR_UNSUPPORTED;
      m_rep = 8 * I.sell_slots + 4 * (int64_t)A.m + 8 * (I.sell_slices + 1);
      units = I.sell_slices;
    } else if (pc.family == SD_FMT_WIN && !src) {
      // Packed column windows over the heavy-split layout (host conversion;
      // the device one is below, with the split's)
      I.cache_policy = 1;
      p->h_vals.assign(A.values, A.values + A.nnz);
      sd::heavy_split(A, pc.T, pc.c, light_order, &p->h_light, &p->h_chunks, &p->h_heavy_rows, &p->h_heavy_ptr);
      sd::split_layout(A, pc.T, pc.c, p->h_light, &p->h_rowptr, &p->h_colidx, &p->h_vals, &p->h_chunks);
      sd::chunk_order(p->h_colidx, p->h_chunks, chunk_ord, &p->h_corder);
      I.chunk_order = chunk_ord;
      I.light_order = light_order;
      I.heavy_threshold = pc.T;
      I.chunk_nnz = pc.c;
      I.n_light = (int64_t)p->h_light.size();
      I.n_heavy = (int64_t)p->h_heavy_rows.size();
      I.n_chunks = (int64_t)p->h_chunks.size() / 3;
      // LDS per staged column: one tile of the dense width (the 128-bit geometry,
      // which is never narrower than the 32-bit one used for unaligned B or C);
      // a window keeps at most the columns that fit the budget, its most used
      const int32_t cap = window_cap(n, vec4, col_tile, I.max_lds_bytes);
      const int32_t R = o.window_rows > 0 ? o.window_rows : sd::kDefaultWindowRows;
      int32_t wmax = 0;
      int64_t uses = 0;
      sd::split_windows(A.k, p->h_rowptr, I.n_light, &p->h_colidx, R, cap, &p->h_wptr, &p->h_wcols, &wmax, &uses);
      I.window_rows = R;
      I.window_max = wmax;
      I.window_staged = (int64_t)p->h_wcols.size();
      I.window_staged_uses = uses;
      const int64_t n_windows = (I.n_light + R - 1) / R;
      m_rep += 4 * I.n_light + 16 * I.n_chunks + 4 * I.n_heavy + 4 * (I.n_heavy + 1) + 4 * (n_windows + 1) +
               4 * I.window_staged;
      ws = 4 * (int64_t)n * I.n_chunks;
      units = I.n_chunks + n_windows;
    } else if (src) {
      // CSR families from device memory: device-to-device copies, then the
      // partitions on the device
      I.cache_policy = pc.family == SD_FMT_CSR_MERGE ? pc.policy : 1;
      if ((st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_rowptr), nullptr, 4 * ((size_t)A.m + 1))) !=
              SD_OK ||
          (st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_colidx), nullptr, 4 * (size_t)A.nnz)) != SD_OK ||
          (st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_vals), nullptr, 4 * (size_t)A.nnz)) != SD_OK)
        return st;
      hipError_t e = hipMemcpyAsync(p->d_rowptr, src->rowptr, 4 * ((size_t)A.m + 1), hipMemcpyDeviceToDevice, ds);
      if (e == hipSuccess && I.cache_policy == 2) {  // tiered: the columns with their cold tags
        const int64_t budget = (o.hot_budget_kib > 0 ? (int64_t)o.hot_budget_kib << 10 : (int64_t)2 << 20);
        e = sd::dev_tag_cold(src->colidx, A.nnz, A.k, std::max<int64_t>(1, budget / (4 * (int64_t)n)), p->d_colidx,
                             &I.hot_columns, &I.hot_nnz, ds);
      } else if (e == hipSuccess && A.nnz) {
        e = hipMemcpyAsync(p->d_colidx, src->colidx, 4 * (size_t)A.nnz, hipMemcpyDeviceToDevice, ds);
      }
      if (e == hipSuccess && A.nnz)
        e = hipMemcpyAsync(p->d_vals, src->values, 4 * (size_t)A.nnz, hipMemcpyDeviceToDevice, ds);
      if (e != hipSuccess) return hip_fail(e);
      if (pc.family == SD_FMT_CSR_SPLIT || pc.family == SD_FMT_WIN) {
        auto alloc = [&](size_t bytes) -> void * {
          void *q = nullptr;
          return hip_alloc_copy(p, &q, nullptr, bytes) == SD_OK ? q : nullptr;
        };
        e = sd::dev_heavy_split(src->rowptr, A.m, pc.T, pc.c, alloc, ds, &p->d_light, &p->d_chunks,
                                &p->d_heavy_rows, &p->d_heavy_ptr, &I.n_light, &I.n_heavy, &I.n_chunks);
        if (e == hipSuccess && light_order == 2)
          e = sd::dev_light_by_last_col(src->rowptr, src->colidx, A.k, p->d_light, I.n_light, ds);
        // the split layout, over the copies just made of rowptr / colidx / values
        if (e == hipSuccess)
          e = sd::dev_split_layout(src->rowptr, src->colidx, src->values, A.nnz, p->d_light, I.n_light,
                                   p->d_heavy_rows, p->d_heavy_ptr, I.n_heavy, p->d_rowptr, p->d_colidx,
                                   p->d_vals, p->d_chunks, ds);
        if (e != hipSuccess) return hip_fail(e);
        if ((st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_corder), nullptr, 4 * (size_t)I.n_chunks)) !=
            SD_OK)
          return st;
        e = sd::dev_chunk_order(p->d_colidx, p->d_chunks, I.n_chunks, A.k, chunk_ord, p->d_corder, ds);
        if (e != hipSuccess) return hip_fail(e);
        I.chunk_order = chunk_ord;
        I.light_order = light_order;
        I.heavy_threshold = pc.T;
        I.chunk_nnz = pc.c;
        m_rep += 4 * I.n_light + 16 * I.n_chunks + 4 * I.n_heavy + 4 * (I.n_heavy + 1);
        ws = 4 * (int64_t)n * I.n_chunks;
        units = I.n_light + I.n_chunks;
        if (pc.family == SD_FMT_WIN) {  // windows over the light rows of that layout
          const int32_t R = o.window_rows > 0 ? o.window_rows : sd::kDefaultWindowRows;
          int32_t wmax = 0;
          int64_t staged = 0, uses = 0;
          e = sd::dev_split_windows(p->d_rowptr, I.n_light, p->d_colidx, R,
                                    window_cap(n, vec4, col_tile, I.max_lds_bytes), alloc, ds, &p->d_wptr,
                                    &p->d_wcols, &wmax, &staged, &uses);
          if (e != hipSuccess) return hip_fail(e);
          I.window_rows = R;
          I.window_max = wmax;
          I.window_staged = staged;
          I.window_staged_uses = uses;
          const int64_t n_windows = (I.n_light + R - 1) / R;
          m_rep += 4 * (n_windows + 1) + 4 * staged;
          units = I.n_chunks + n_windows;
        }
      } else if (pc.family == SD_FMT_CSR_MERGE) {
        const int64_t total = (int64_t)A.m + A.nnz;
        const int64_t L = std::max<int64_t>(1, (total + pc.U - 1) / pc.U);
        if ((st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_coords), nullptr,
                                 8 * ((size_t)pc.U + 1))) != SD_OK)
          return st;
        e = sd::dev_merge_coords(src->rowptr, A.m, A.nnz, pc.U, L, p->d_coords, ds);
        if (e != hipSuccess) return hip_fail(e);
        I.units = pc.U;
        I.merge_len = L;
        m_rep += 8 * ((int64_t)pc.U + 1);
        ws = 8 * (int64_t)n * pc.U + 8 * (int64_t)pc.U;  // carries and heads
        units = pc.U;
      }
    } else {
      p->h_rowptr.assign(A.rowptr, A.rowptr + A.m + 1);
      p->h_colidx.assign(A.colidx, A.colidx + A.nnz);
      // only the merge-path kernel carries the tiered / non-temporal gathers
      I.cache_policy = pc.family == SD_FMT_CSR_MERGE ? pc.policy : 1;
      if (I.cache_policy == 2) {
        const int64_t budget = (o.hot_budget_kib > 0 ? (int64_t)o.hot_budget_kib << 10 : (int64_t)2 << 20);
        sd::tag_cold_columns(A, std::max<int64_t>(1, budget / (4 * (int64_t)n)), &p->h_coltag, &I.hot_columns,
                             &I.hot_nnz);
      }
      p->h_vals.resize((size_t)A.nnz);
      if (A.nnz) std::memcpy(p->h_vals.data(), A.values, sizeof(float) * (size_t)A.nnz);
      if (pc.family == SD_FMT_CSR_SPLIT) {
        sd::heavy_split(A, pc.T, pc.c, light_order, &p->h_light, &p->h_chunks, &p->h_heavy_rows, &p->h_heavy_ptr);
        // the kernels read the split layout: light rows in list order, then heavy rows
        sd::split_layout(A, pc.T, pc.c, p->h_light, &p->h_rowptr, &p->h_colidx, &p->h_vals, &p->h_chunks);
        sd::chunk_order(p->h_colidx, p->h_chunks, chunk_ord, &p->h_corder);
        I.chunk_order = chunk_ord;
        I.light_order = light_order;
        I.heavy_threshold = pc.T;
        I.chunk_nnz = pc.c;
        I.n_light = (int64_t)p->h_light.size();
        I.n_heavy = (int64_t)p->h_heavy_rows.size();
        I.n_chunks = (int64_t)p->h_chunks.size() / 3;
        m_rep += 4 * I.n_light + 16 * I.n_chunks + 4 * I.n_heavy + 4 * (I.n_heavy + 1);
        ws = 4 * (int64_t)n * I.n_chunks;
        units = I.n_light + I.n_chunks;
      } else if (pc.family == SD_FMT_CSR_MERGE) {
        int64_t L = 0;
        sd::merge_split(A, pc.U, &p->h_coords, &L);
        I.units = pc.U;
        I.merge_len = L;
        m_rep += 8 * ((int64_t)pc.U + 1);
        ws = 8 * (int64_t)n * pc.U + 8 * (int64_t)pc.U;  // carries and heads
        units = pc.U;
      }
    }
  } catch (const std::bad_alloc &) {
    return SD_ERR_OUT_OF_MEMORY;
  }
  if ((int64_t)n * A.m > ((int64_t)1 << 40) || (int64_t)n * A.k > ((int64_t)1 << 40)) return SD_ERR_OVERFLOW;
  if (I.family == SD_FMT_CSR_ROW || I.family == SD_FMT_CSR_SPLIT) {
    sd::row_batch_for(stats, I.family == SD_FMT_CSR_ROW ? A.m : I.n_light, geo.G, I.cu_count, o.rows_per_group,
                      o.gather_unroll, &I.rows_per_group, &I.gather_unroll);
    // narrow widths: lane groups that share a row
    if (o.row_slices > 1 && (geo.G > 8 || geo.G * o.row_slices > 64)) return SD_ERR_UNSUPPORTED;
    I.row_slices = o.row_slices > 0 ? o.row_slices : sd::slices_for(stats, I.family, n, geo.G);
    if (I.row_slices > 1) {
      I.rows_per_group = 1;
      I.gather_unroll = sd::kSliceRound;
    }
    I.lanes_per_row = geo.G * I.row_slices;
  }
  // Row families under the default order: chunked round-robin when the rows'
  // typical farthest neighbour is a whole number of rounds away, which keeps
  // both on one XCD (7-point Laplacian 64^3, ELL: 34 against 38 us).
  if (o.wg_order == 0 && (I.family == SD_FMT_ELL || I.family == SD_FMT_CSR_ROW)) {
    const int64_t rows_per_wg = (int64_t)(sd::kBlockThreads / (geo.G * std::max(1, I.row_slices))) *
                                (I.family == SD_FMT_CSR_ROW ? std::max(1, I.rows_per_group) : 1);
    if (src) {
      if ((st = device_median_reach(src, ds, &I.reach)) != SD_OK) return st;
    } else {
      I.reach = sd::median_row_reach(A);
    }
    const int32_t S = sd::chunk_for_reach(I.reach, rows_per_wg);
    if (S > 0) {
      I.wg_order = 3;
      I.wg_chunk = S;
    }
  }


  // ---- workload-scale analysis
  I.m_rep = m_rep;
  I.workspace = ws;
  I.d_r = 4 * (int64_t)A.k * n;
  I.d_s = 4 * (int64_t)A.m * n;
  I.m_r = m_rep + ws + I.d_r;
  I.m_t = I.m_r + I.d_s;
  I.compulsory_bytes = 8 * A.nnz + 4 * ((int64_t)A.m + 1) + I.d_r + I.d_s;
  I.mall_bytes = sd::kMallBytes;
  I.q_r = I.l2_bytes > 0 ? (double)I.m_r / (double)I.l2_bytes : 0.0;
  I.q_t = I.l2_bytes > 0 ? (double)I.m_t / (double)I.l2_bytes : 0.0;
  I.q_r_mall = (double)I.m_r / (double)I.mall_bytes;
  I.q_t_mall = (double)I.m_t / (double)I.mall_bytes;
  I.work_units = units;
  I.units_per_cu = I.cu_count > 0 ? (double)units / (double)I.cu_count : 0.0;
  I.block_threads = sd::kBlockThreads;

  if (p->device < 0) {
    I.legal = I.block_threads <= I.max_threads ? 1 : 0;
    return SD_OK;
  }

  // ---- upload (once) and legality from the compiled kernel
  DeviceGuard guard;
  st = guard.enter(p->device);
  if (st != SD_OK) return st;
  hipFuncAttributes attr;
  std::memset(&attr, 0, sizeof(attr));
  hipError_t e =
      sd::kernel_attributes(I.family, I.engine, n, vec4, I.rows_per_group, I.gather_unroll, I.row_slices, col_tile,
                            (int32_t)I.ell_width, &attr);
  if (e != hipSuccess) return hip_fail(e);
  I.regs_per_thread = attr.numRegs;
  I.lds_bytes = (int32_t)attr.sharedSizeBytes;
  if (I.family == SD_FMT_WIN) I.lds_bytes += (int32_t)sd::window_lds_bytes(n, vec4, col_tile, I.window_max);
  I.legal = (I.block_threads <= I.max_threads && I.block_threads <= attr.maxThreadsPerBlock &&
             (int64_t)attr.numRegs * I.block_threads <= regs_per_cu && I.lds_bytes <= I.max_lds_bytes)
                ? 1
                : 0;
  if (!I.legal) return SD_ERR_UNSUPPORTED;

  if (I.family == SD_FMT_ELL || I.family == SD_FMT_SELL) {
    if (I.family == SD_FMT_SELL && !src) {
      if ((st = upload(p, &p->d_perm, p->h_perm)) != SD_OK) return st;
      if ((st = upload(p, &p->d_sptr, p->h_sptr)) != SD_OK) return st;
      std::vector<int32_t>().swap(p->h_perm);
      std::vector<int64_t>().swap(p->h_sptr);
    }
    if (!src) {
      if ((st = upload(p, &p->d_ecol, p->h_ecol)) != SD_OK) return st;
      if ((st = upload(p, &p->d_eval, p->h_eval)) != SD_OK) return st;
    }
    std::vector<int32_t>().swap(p->h_ecol);
    std::vector<float>().swap(p->h_eval);
  } else if (I.family == SD_FMT_BSR || I.family == SD_FMT_BELL) {
    {
      const std::vector<float> zeros((size_t)std::max<int64_t>(I.n, 4), 0.0f);
      if ((st = upload(p, &p->d_zrow, zeros)) != SD_OK) return st;
    }
    if (!src) {
      if (I.family == SD_FMT_BSR && (st = upload(p, &p->d_bptr, p->h_bptr)) != SD_OK) return st;
      // device copies carry one extra block after the stored ones: column -1 and
      // zero values (the MFMA kernel's fetch target past a block-row's end);
      // exports copy only the stored blocks
      p->h_bcol.push_back(-1);
      p->h_bval.resize(p->h_bval.size() + 256, 0.0f);
      if ((st = upload(p, &p->d_bcol, p->h_bcol)) != SD_OK) return st;
      if ((st = upload(p, &p->d_bval, p->h_bval)) != SD_OK) return st;
      std::vector<int32_t>().swap(p->h_bcol);
      std::vector<float>().swap(p->h_bval);
    }
  } else {
    if (!src) {
      if ((st = upload(p, &p->d_rowptr, p->h_rowptr)) != SD_OK) return st;
      if ((st = upload(p, &p->d_colidx, I.cache_policy == 2 ? p->h_coltag : p->h_colidx)) != SD_OK) return st;
      std::vector<int32_t>().swap(p->h_coltag);
      if ((st = upload(p, &p->d_vals, p->h_vals)) != SD_OK) return st;
      std::vector<int32_t>().swap(p->h_colidx);
      std::vector<float>().swap(p->h_vals);
    }
    if (I.family == SD_FMT_WIN && !src) {
      if ((st = upload(p, &p->d_wptr, p->h_wptr)) != SD_OK) return st;
      if ((st = upload(p, &p->d_wcols, p->h_wcols)) != SD_OK) return st;
      std::vector<int32_t>().swap(p->h_wptr);
      std::vector<int32_t>().swap(p->h_wcols);
    }
    if (I.family == SD_FMT_CSR_SPLIT || I.family == SD_FMT_WIN) {
      if (!src) {
        if ((st = upload(p, &p->d_light, p->h_light)) != SD_OK) return st;
        if ((st = upload(p, &p->d_chunks, p->h_chunks)) != SD_OK) return st;
        if ((st = upload(p, &p->d_corder, p->h_corder)) != SD_OK) return st;
        if ((st = upload(p, &p->d_heavy_rows, p->h_heavy_rows)) != SD_OK) return st;
        if ((st = upload(p, &p->d_heavy_ptr, p->h_heavy_ptr)) != SD_OK) return st;
      }
      if ((st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_ws), nullptr, (size_t)ws)) != SD_OK) return st;
    } else if (I.family == SD_FMT_CSR_MERGE) {
      if (!src && (st = upload(p, &p->d_coords, p->h_coords)) != SD_OK) return st;
      // carry and head rows, carry and head partials
      if ((st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_carry_row), nullptr, 8 * (size_t)I.units)) !=
          SD_OK)
        return st;
      if ((st = hip_alloc_copy(p, reinterpret_cast<void **>(&p->d_ws), nullptr, 8 * (size_t)n * (size_t)I.units)) !=
          SD_OK)
        return st;
    }
  }
  if (src) {  // the device conversions ran on the caller's stream
    hipError_t e2 = hipStreamSynchronize(ds);
    if (e2 != hipSuccess) return hip_fail(e2);
  }
  return SD_OK;
}

}  // namespace

namespace {

struct ExportRef {
  const void *host = nullptr;
  const void *dev = nullptr;
  size_t bytes = 0;
  bool ok = false;
};

template <typename T>
ExportRef ref_of(const std::vector<T> &h, const T *d, size_t count, bool device_plan) {
  ExportRef r;
  r.ok = true;
  r.bytes = count * sizeof(T);
  if (device_plan && d) r.dev = d;
  else r.host = h.data();
  return r;
}

ExportRef export_ref(const sd_plan_s *p, int32_t what) {
  const sd_plan_info_t &I = p->info;
  const bool dev = p->device >= 0;
  const bool csr = I.family >= SD_FMT_CSR_ROW && I.family <= SD_FMT_CSR_MERGE;
  const bool split = I.family == SD_FMT_CSR_SPLIT || I.family == SD_FMT_WIN;  // the split layout
  const bool blk = I.family == SD_FMT_BSR || I.family == SD_FMT_BELL;
  switch (what) {
    case SD_EXPORT_ROWPTR:
      // a heavy-split plan holds its split layout: |light| + 1 pointers by list position
      if (csr || split)
        return ref_of(p->h_rowptr, p->d_rowptr, split ? (size_t)I.n_light + 1 : (size_t)I.m + 1, dev);
      break;
    case SD_EXPORT_COLIDX:
      if (csr) return ref_of(p->h_colidx, p->d_colidx, (size_t)I.nnz, dev);
      break;
    case SD_EXPORT_VALUES:
      if (csr || split) return ref_of(p->h_vals, p->d_vals, (size_t)I.nnz, dev);
      break;
    case SD_EXPORT_LIGHT_ROWS:
      if (split) return ref_of(p->h_light, p->d_light, (size_t)I.n_light, dev);
      break;
    case SD_EXPORT_CHUNKS:
      if (split) return ref_of(p->h_chunks, p->d_chunks, 3 * (size_t)I.n_chunks, dev);
      break;
    case SD_EXPORT_CHUNK_ORDER:
      if (split) return ref_of(p->h_corder, p->d_corder, (size_t)I.n_chunks, dev);
      break;
    case SD_EXPORT_MERGE_COORDS:
      if (I.family == SD_FMT_CSR_MERGE) return ref_of(p->h_coords, p->d_coords, 2 * ((size_t)I.units + 1), dev);
      break;
    case SD_EXPORT_BLOCK_PTR:
      if (I.family == SD_FMT_BSR) return ref_of(p->h_bptr, p->d_bptr, (size_t)I.block_rows + 1, dev);
      break;
    case SD_EXPORT_ELL_COL:
      if (I.family == SD_FMT_ELL) return ref_of(p->h_ecol, p->d_ecol, (size_t)(I.m * I.ell_width), dev);
      break;
    case SD_EXPORT_ELL_VAL:
      if (I.family == SD_FMT_ELL) return ref_of(p->h_eval, p->d_eval, (size_t)(I.m * I.ell_width), dev);
      break;
    case SD_EXPORT_WIN_PTR:
      if (I.family == SD_FMT_WIN)
        return ref_of(p->h_wptr, p->d_wptr, (size_t)((I.n_light + I.window_rows - 1) / I.window_rows) + 1, dev);
      break;
    case SD_EXPORT_WIN_COLS:
      if (I.family == SD_FMT_WIN) return ref_of(p->h_wcols, p->d_wcols, (size_t)I.window_staged, dev);
      break;
    case SD_EXPORT_WIN_CODE:
      if (I.family == SD_FMT_WIN) return ref_of(p->h_colidx, p->d_colidx, (size_t)I.nnz, dev);
      break;
    case SD_EXPORT_WIN_VAL:
      if (I.family == SD_FMT_WIN) return ref_of(p->h_vals, p->d_vals, (size_t)I.nnz, dev);
      break;
    case SD_EXPORT_SELL_PERM:
      if (I.family == SD_FMT_SELL) return ref_of(p->h_perm, p->d_perm, (size_t)I.m, dev);
      break;
    case SD_EXPORT_SELL_SLICE_PTR:
      if (I.family == SD_FMT_SELL) return ref_of(p->h_sptr, p->d_sptr, (size_t)I.sell_slices + 1, dev);
      break;
    case SD_EXPORT_SELL_COL:
      if (I.family == SD_FMT_SELL) return ref_of(p->h_ecol, p->d_ecol, (size_t)I.sell_slots, dev);
      break;
    case SD_EXPORT_SELL_VAL:
      if (I.family == SD_FMT_SELL) return ref_of(p->h_eval, p->d_eval, (size_t)I.sell_slots, dev);
      break;
    case SD_EXPORT_BLOCK_COL:
      if (blk) {
        const size_t slots = I.family == SD_FMT_BSR ? (size_t)I.nnzb : (size_t)(I.bell_width * I.block_rows);
        return ref_of(p->h_bcol, p->d_bcol, slots, dev);
      }
      break;
    case SD_EXPORT_BLOCK_VAL:
      if (blk) {
        const size_t slots = I.family == SD_FMT_BSR ? (size_t)I.nnzb : (size_t)(I.bell_width * I.block_rows);
        return ref_of(p->h_bval, p->d_bval, slots * 256, dev);
      }
      break;
  }
  return ExportRef{};
}

}  // namespace

namespace {
int search_plan(const sd_csr_t *A, int32_t n, const sd_plan_opts_t &o, sd_plan_t *out,
                const sd_csr_t *src = nullptr, hipStream_t ds = nullptr);
int check_opts(const sd_plan_opts_t &o);
int make_plan(const sd_csr_t *A, int32_t n, const sd_plan_opts_t &o, const sd_csr_t *src, hipStream_t s,
              sd_plan_t *out);
}  // namespace

extern "C" {

int sd_analyze(const sd_csr_t *A, int32_t dense_threshold, sd_stats_t *out) {
  if (!A || !out) return SD_ERR_INVALID_VALUE;
  sd::CsrView v;
  int st = sd::validate_csr(A, &v);
  if (st != SD_OK) return st;
  return sd::analyze(v, dense_threshold, out);
}

int sd_analyze_device(const sd_csr_t *A, int32_t dense_threshold, sd_stats_t *out, void *stream) {
  if (!A || !out) return SD_ERR_INVALID_VALUE;
  int count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count == 0) {
    (void)hipGetLastError();
    return SD_ERR_NO_DEVICE;
  }
  return sd::analyze_device(A, dense_threshold, out, reinterpret_cast<hipStream_t>(stream));
}

int sd_plan(const sd_csr_t *A, int32_t n, sd_plan_t *out) { return sd_plan_ex(A, n, nullptr, out); }

int sd_plan_ex(const sd_csr_t *A, int32_t n, const sd_plan_opts_t *opts, sd_plan_t *out) {
  if (!A || !out || n < 1) return SD_ERR_INVALID_VALUE;
  sd_plan_opts_t o;
  std::memset(&o, 0, sizeof(o));
  if (opts) o = *opts;
  if (o.search) {
    if (o.placement == 2) return SD_ERR_NO_DEVICE;
    return search_plan(A, n, o, out);
  }
  int st = check_opts(o);
  if (st != SD_OK) return st;
  return make_plan(A, n, o, nullptr, nullptr, out);
}

int sd_plan_device(const sd_csr_t *A, int32_t n, const sd_plan_opts_t *opts, void *stream, sd_plan_t *out) {
  if (!A || !out || n < 1) return SD_ERR_INVALID_VALUE;
  if (A->m < 0 || A->k < 0 || A->nnz < 0) return SD_ERR_INVALID_CSR;
  if (!A->rowptr || (A->nnz > 0 && (!A->colidx || !A->values))) return SD_ERR_INVALID_VALUE;
  sd_plan_opts_t o;
  std::memset(&o, 0, sizeof(o));
  if (opts) o = *opts;
  int st = check_opts(o);
  if (st != SD_OK) return st;
  int count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count <= 0) {
    (void)hipGetLastError();
    return SD_ERR_NO_DEVICE;
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (o.placement == 0) {
    try {
      st = o.search ? search_plan(nullptr, n, o, out, A, s) : make_plan(nullptr, n, o, A, s, out);
    } catch (const std::bad_alloc &) {
      st = SD_ERR_OUT_OF_MEMORY;
    }
    if (st != kNeedHost) return st;
  }
  // Host conversion: the matrix is copied to the host (ordered after the
  // caller's work on `stream`) and planned as sd_plan_ex plans it.
  std::vector<int32_t> rowptr, colidx;
  std::vector<float> vals;
  try {
    rowptr.resize((size_t)A->m + 1);
    colidx.resize((size_t)A->nnz);
    vals.resize((size_t)A->nnz);
  } catch (const std::bad_alloc &) {
    return SD_ERR_OUT_OF_MEMORY;
  }
  hipError_t e = hipMemcpyAsync(rowptr.data(), A->rowptr, 4 * rowptr.size(), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess && A->nnz)
    e = hipMemcpyAsync(colidx.data(), A->colidx, 4 * colidx.size(), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess && A->nnz) e = hipMemcpyAsync(vals.data(), A->values, 4 * vals.size(), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e);
  const sd_csr_t H{A->m, A->k, A->nnz, rowptr.data(), colidx.data(), vals.data()};
  return sd_plan_ex(&H, n, &o, out);
}

}  // extern "C"

namespace {

int check_opts(const sd_plan_opts_t &o) {
  if ((o.rows_per_group != 0 && o.rows_per_group != 1 && o.rows_per_group != 2 && o.rows_per_group != 4 &&
       o.rows_per_group != 8 && o.rows_per_group != 16) ||
      (o.gather_unroll != 0 && o.gather_unroll != 4 && o.gather_unroll != 8))
    return SD_ERR_INVALID_VALUE;
  if (o.cache_policy < 0 || o.cache_policy > 3 || o.hot_budget_kib < 0) return SD_ERR_INVALID_VALUE;
  if (o.col_tile != 0 && (o.col_tile < 4 || (o.col_tile & (o.col_tile - 1)) != 0)) return SD_ERR_INVALID_VALUE;
  if (o.window_rows < 0 || o.wg_order < 0 || o.wg_order > 3 || o.wg_chunk < 0 || o.sell_sigma < 0)
    return SD_ERR_INVALID_VALUE;
  if (o.row_slices < 0 || o.row_slices > 64 || (o.row_slices & (o.row_slices - 1)) != 0) return SD_ERR_INVALID_VALUE;
  if (o.light_order < 0 || o.light_order > 2) return SD_ERR_INVALID_VALUE;
  if (o.chunk_order < 0 || o.chunk_order > 2) return SD_ERR_INVALID_VALUE;
  if (o.force < SD_FMT_AUTO || o.force > SD_FMT_SELL || o.placement < 0 || o.placement > 2 ||
      o.heavy_threshold < 0 || o.chunk_nnz < 0 || o.units < 0 || o.engine < 0 || o.engine > SD_ENGINE_VALU)
    return SD_ERR_INVALID_VALUE;
  return SD_OK;
}

// Builds one plan from host CSR A, or from device CSR src on stream s.
int make_plan(const sd_csr_t *A, int32_t n, const sd_plan_opts_t &o, const sd_csr_t *src, hipStream_t s,
              sd_plan_t *out) {
  sd_plan_s *p = nullptr;
  try {
    p = new sd_plan_s();
  } catch (const std::bad_alloc &) {
    return SD_ERR_OUT_OF_MEMORY;
  }
  int st;
  try {
    st = build_plan(A, n, o, p, src, s);
  } catch (const std::bad_alloc &) {
    st = SD_ERR_OUT_OF_MEMORY;
  }
  if (st != SD_OK) {
    if (src) (void)hipStreamSynchronize(s);  // no conversion may still write the memory freed here
    release(p);
    delete p;
    return st;
  }
  *out = p;
  return SD_OK;
}

}  // namespace

extern "C" {

int sd_spmm(sd_plan_t p, const float *B, float *C, void *stream) {
  if (!p) return SD_ERR_INVALID_VALUE;
  if (p->device < 0) return SD_ERR_NO_DEVICE;
  const sd_plan_info_t &I = p->info;
  if (I.m == 0) return SD_OK;  // empty output
  if (!C || (!B && I.k > 0)) return SD_ERR_INVALID_VALUE;
  {  // B (k x n) and C (m x n) must not overlap: the kernels write C while others still read B
    const uintptr_t b0 = reinterpret_cast<uintptr_t>(B), c0 = reinterpret_cast<uintptr_t>(C);
    const uintptr_t b1 = b0 + (uintptr_t)I.k * (uintptr_t)I.n * sizeof(float);
    const uintptr_t c1 = c0 + (uintptr_t)I.m * (uintptr_t)I.n * sizeof(float);
    if (I.k > 0 && b0 < c1 && c0 < b1) return SD_ERR_INVALID_VALUE;
  }
  DeviceGuard guard;
  int st = guard.enter(p->device);
  if (st != SD_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  sd::DenseIO io;
  io.B = B;
  io.C = C;
  io.n = (int32_t)I.n;
  io.vec4 = (I.n % 4 == 0) && ((reinterpret_cast<uintptr_t>(B) | reinterpret_cast<uintptr_t>(C)) % 16 == 0);
  io.policy = I.cache_policy == 2 ? 1 : I.cache_policy == 3 ? 2 : 0;
  io.col_tile = p->col_tile_req;
  io.order = I.wg_order == 1 ? 1 : I.wg_order == 3 ? std::max(2, I.wg_chunk) : 0;
  sd::CsrOperand A{p->d_rowptr, p->d_colidx, p->d_vals, (int32_t)I.m, (int32_t)I.k};
  hipError_t e = hipSuccess;
  switch (I.family) {
    case SD_FMT_CSR_ROW:
      e = sd::launch_csr_rows(A, io, I.rows_per_group, I.gather_unroll, I.row_slices, s);
      break;
    case SD_FMT_CSR_SPLIT:
      e = sd::launch_csr_split(A, p->d_light, (int32_t)I.n_light, p->d_chunks, p->d_corder, (int32_t)I.n_chunks,
                               p->d_heavy_rows,
                               p->d_heavy_ptr, (int32_t)I.n_heavy, p->d_ws, io, I.rows_per_group,
                               I.gather_unroll, I.row_slices, s);
      break;
    case SD_FMT_CSR_MERGE:
      e = sd::launch_csr_merge(A, p->d_coords, (int32_t)I.units, p->d_carry_row, p->d_ws, io, s);
      break;
    case SD_FMT_ELL:
      e = sd::launch_ell(p->d_ecol, p->d_eval, (int32_t)I.ell_width, (int32_t)I.m, I.rows_per_group, io, s);
      break;
    case SD_FMT_SELL:
      e = sd::launch_sell(p->d_perm, p->d_sptr, p->d_ecol, p->d_eval, I.sell_c, (int32_t)I.m, io, s);
      break;
    case SD_FMT_WIN:
      e = sd::launch_win_split(A, p->d_light, (int32_t)I.n_light, p->d_chunks, p->d_corder, (int32_t)I.n_chunks,
                               p->d_heavy_rows, p->d_heavy_ptr, (int32_t)I.n_heavy, p->d_ws, p->d_wptr,
                               p->d_wcols, I.window_rows, I.window_max, io, s);
      break;
    case SD_FMT_BSR:
    case SD_FMT_BELL: {
      const int32_t engine = I.engine;  // MFMA serves any width and alignment (sliced column tiles)
      const int64_t zero_block = I.family == SD_FMT_BSR ? I.nnzb : I.bell_width * I.block_rows;
      e = sd::launch_bsr((int32_t)I.block_rows, (int32_t)I.m, (int32_t)I.k,
                         I.family == SD_FMT_BSR ? p->d_bptr : nullptr, (int32_t)I.bell_width, p->d_bcol, p->d_bval,
                         zero_block, p->d_zrow, engine, io, s);
      break;
    }
    default:
      return SD_ERR_INVALID_VALUE;
  }
  if (e != hipSuccess) return hip_fail(e);
  return SD_OK;
}

int sd_plan_info(sd_plan_t p, sd_plan_info_t *out) {
  if (!p || !out) return SD_ERR_INVALID_VALUE;
  *out = p->info;
  return SD_OK;
}

int sd_plan_export_size(sd_plan_t p, int32_t what, size_t *bytes) {
  if (!p || !bytes) return SD_ERR_INVALID_VALUE;
  ExportRef r = export_ref(p, what);
  if (!r.ok) return SD_ERR_INVALID_VALUE;
  *bytes = r.bytes;
  return SD_OK;
}

int sd_plan_export(sd_plan_t p, int32_t what, void *host_dst, size_t bytes) {
  if (!p || (!host_dst && bytes)) return SD_ERR_INVALID_VALUE;
  ExportRef r = export_ref(p, what);
  if (!r.ok || bytes < r.bytes) return SD_ERR_INVALID_VALUE;
  if (r.bytes == 0) return SD_OK;
  if (r.dev) {
    DeviceGuard guard;
    int st = guard.enter(p->device);
    if (st != SD_OK) return st;
    hipError_t e = hipMemcpy(host_dst, r.dev, r.bytes, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e);
    if (what == SD_EXPORT_COLIDX && p->info.cache_policy == 2) {  // drop the cold-column tags
      int32_t *c = static_cast<int32_t *>(host_dst);
      for (size_t i = 0; i < r.bytes / sizeof(int32_t); ++i) c[i] &= 0x7fffffff;
    }
  } else {
    std::memcpy(host_dst, r.host, r.bytes);
  }
  return SD_OK;
}

void sd_plan_destroy(sd_plan_t p) {
  if (!p) return;
  release(p);
  delete p;
}

const char *sd_status_string(int status) {
  switch (status) {
    case SD_OK: return "SD_OK";
    case SD_ERR_INVALID_VALUE: return "SD_ERR_INVALID_VALUE: invalid argument";
    case SD_ERR_INVALID_CSR: return "SD_ERR_INVALID_CSR: malformed CSR";
    case SD_ERR_UNSUPPORTED: return "SD_ERR_UNSUPPORTED: plan infeasible for this input";
    case SD_ERR_OUT_OF_MEMORY: return "SD_ERR_OUT_OF_MEMORY: allocation failed";
    case SD_ERR_HIP: return "SD_ERR_HIP: HIP runtime or launch error";
    case SD_ERR_OVERFLOW: return "SD_ERR_OVERFLOW: size exceeds index range";
    case SD_ERR_NO_DEVICE: return "SD_ERR_NO_DEVICE: host-only plan";
    case SD_ERR_IO: return "SD_ERR_IO: cache file unreadable, unwritable or malformed";
  }
  return "unknown sd_status";
}

const char *sd_last_error(void) { return g_last_error.c_str(); }

void sd_plan_cache_clear(void);

}  // extern "C"

namespace sd {
int report_hip_error(int hip_error) { return hip_fail(static_cast<hipError_t>(hip_error)); }
}  // namespace sd

// ------------------------------------------------------ measured selection ---
// Among its candidate plans the paper keeps the quickest one that passes
// validation, and reuses that choice per input (Introduction; Sec. "Architecture-Aware Compilation-Plan
// Synthesis"; Sec. "Agentic Lowering and Refinement"; Sec. "Evaluation",
// measurement protocol).  Here the candidates are this library's families and
// parameter sets allowed by the operand's statistics; each is built, timed on
// the device with scratch operands, and checked against the rule-based plan.
namespace {

std::mutex g_cache_mu;
std::unordered_map<uint64_t, sd_plan_opts_t> g_cache;

uint64_t fnv1a(uint64_t h, const void *p, size_t bytes) {
  const unsigned char *c = static_cast<const unsigned char *>(p);
  for (size_t i = 0; i < bytes; ++i) {
    h ^= c[i];
    h *= 1099511628211ull;
  }
  return h;
}

// The device enters the key by its architecture and size, not its ordinal, so
// a saved cache applies to any GPU of the same kind.
int device_signature(int dev, uint64_t *sig) {
  hipDeviceProp_t prop;
  hipError_t e = hipGetDeviceProperties(&prop, dev);
  if (e != hipSuccess) return hip_fail(e);
  const int64_t sizes[3] = {prop.multiProcessorCount, (int64_t)prop.l2CacheSize, (int64_t)prop.sharedMemPerBlock};
  uint64_t h = fnv1a(1469598103934665603ull, prop.gcnArchName, strnlen(prop.gcnArchName, sizeof(prop.gcnArchName)));
  *sig = fnv1a(h, sizes, sizeof(sizes));
  return SD_OK;
}

// The pattern enters the key through a sum of mixed (position, value) terms
// (sd::pattern_hash_host), so a matrix in device memory gets the same key
// from the same hash computed on the device.
uint64_t structure_key(int64_t m, int64_t k, int64_t nnz, uint64_t pattern, int32_t n, int32_t transpose,
                       uint64_t device_sig) {
  uint64_t h = 1469598103934665603ull;
  const int64_t hdr[7] = {m, k, nnz, n, transpose, (int64_t)device_sig, (int64_t)pattern};
  return fnv1a(h, hdr, sizeof(hdr));
}

struct Scratch {
  float *B = nullptr, *Cref = nullptr, *C = nullptr;
  void *flush = nullptr;  // zero-filled, read before every timed launch (nullptr: no flush)
  float *sink = nullptr;
  size_t flush_bytes = 0;
  hipStream_t s = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  ~Scratch() {
    if (flush) (void)hipFree(flush);
    if (sink) (void)hipFree(sink);
    if (B) (void)hipFree(B);
    if (Cref) (void)hipFree(Cref);
    if (C) (void)hipFree(C);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    if (s) (void)hipStreamDestroy(s);
  }
};

// Mean ms per sd_spmm with the dense operand coming from HBM, as in use:
// before every timed launch a read of twice the Infinity Cache's size
// (outside the events) evicts the previous launch's B rows from L2 and the
// Infinity Cache.  Timed warm, the candidates rank differently (the
// Laplacian's ELL plan runs 31 us warm in contiguous-per-XCD order and 41 us
// cold, against 38 and 37 us in round-robin order).
int time_plan(sd_plan_t p, Scratch &sc, float *C, double *ms) {
  int st;
  if ((st = sd_spmm(p, sc.B, C, sc.s)) != SD_OK) return st;
  hipError_t e = hipSuccess;
  double total = 0.0;
  int reps = 3;
  for (int i = 0; i < reps && e == hipSuccess; ++i) {
    if (sc.flush) e = sd::launch_cache_flush(sc.flush, sc.flush_bytes, sc.sink, sc.s);
    if (e == hipSuccess) e = hipEventRecord(sc.e0, sc.s);
    if (e == hipSuccess && (st = sd_spmm(p, sc.B, C, sc.s)) != SD_OK) return st;
    if (e == hipSuccess) e = hipEventRecord(sc.e1, sc.s);
    if (e == hipSuccess) e = hipEventSynchronize(sc.e1);
    float one = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&one, sc.e0, sc.e1);
    total += one;
    // about 20 ms of timed work in all, between 3 and 12 launches
    if (i == 0 && e == hipSuccess) reps = (int)std::min(12.0, std::max(3.0, 20.0 / std::max(1e-3, (double)one)));
  }
  if (e != hipSuccess) return hip_fail(e);
  *ms = total / reps;
  return SD_OK;
}

// Strided sample of up to 1024 rows of C into host memory.
int sample_rows(const float *C, int64_t m, int64_t n, std::vector<float> *out, int64_t *stride, int64_t *rows) {
  *stride = std::max<int64_t>(1, m / 1024);
  *rows = (m + *stride - 1) / *stride;
  out->resize((size_t)(*rows * n));
  hipError_t e = hipMemcpy2D(out->data(), sizeof(float) * n, C, sizeof(float) * n * *stride, sizeof(float) * n,
                             (size_t)*rows, hipMemcpyDeviceToHost);
  return e == hipSuccess ? SD_OK : hip_fail(e);
}

}  // namespace

extern "C" void sd_plan_cache_clear(void) {
  std::lock_guard<std::mutex> lk(g_cache_mu);
  g_cache.clear();
}

// Cache file: 8-byte tag, u32 size of sd_plan_opts_t, u32 zero, u64 count,
// then count records of (u64 key, sd_plan_opts_t), keys ascending; native
// byte order.
namespace {
constexpr char kCacheTag[8] = {'S', 'D', 'P', 'L', 'A', 'N', 'C', '2'};

struct FileCloser {
  std::FILE *f;
  ~FileCloser() {
    if (f) std::fclose(f);
  }
};
}  // namespace

extern "C" int sd_plan_cache_size(int64_t *entries) {
  if (!entries) return SD_ERR_INVALID_VALUE;
  std::lock_guard<std::mutex> lk(g_cache_mu);
  *entries = (int64_t)g_cache.size();
  return SD_OK;
}

extern "C" int sd_plan_cache_save(const char *path) {
  if (!path) return SD_ERR_INVALID_VALUE;
  std::vector<std::pair<uint64_t, sd_plan_opts_t>> rows;
  {
    std::lock_guard<std::mutex> lk(g_cache_mu);
    rows.assign(g_cache.begin(), g_cache.end());
  }
  std::sort(rows.begin(), rows.end(),
            [](const std::pair<uint64_t, sd_plan_opts_t> &a, const std::pair<uint64_t, sd_plan_opts_t> &b) {
              return a.first < b.first;
            });
  FileCloser fc{std::fopen(path, "wb")};
  if (!fc.f) return SD_ERR_IO;
  const uint32_t hdr[2] = {(uint32_t)sizeof(sd_plan_opts_t), 0};
  const uint64_t count = rows.size();
  bool ok = std::fwrite(kCacheTag, 1, sizeof(kCacheTag), fc.f) == sizeof(kCacheTag) &&
            std::fwrite(hdr, sizeof(hdr), 1, fc.f) == 1 && std::fwrite(&count, sizeof(count), 1, fc.f) == 1;
  for (size_t i = 0; ok && i < rows.size(); ++i)
    ok = std::fwrite(&rows[i].first, sizeof(uint64_t), 1, fc.f) == 1 &&
         std::fwrite(&rows[i].second, sizeof(sd_plan_opts_t), 1, fc.f) == 1;
  ok = std::fclose(fc.f) == 0 && ok;
  fc.f = nullptr;
  return ok ? SD_OK : SD_ERR_IO;
}

extern "C" int sd_plan_cache_load(const char *path) {
  if (!path) return SD_ERR_INVALID_VALUE;
  FileCloser fc{std::fopen(path, "rb")};
  if (!fc.f) return SD_ERR_IO;
  char tag[8];
  uint32_t hdr[2];
  uint64_t count = 0;
  if (std::fread(tag, 1, sizeof(tag), fc.f) != sizeof(tag) || std::memcmp(tag, kCacheTag, sizeof(tag)) != 0 ||
      std::fread(hdr, sizeof(hdr), 1, fc.f) != 1 || hdr[0] != sizeof(sd_plan_opts_t) || hdr[1] != 0 ||
      std::fread(&count, sizeof(count), 1, fc.f) != 1 || count > ((uint64_t)1 << 24))
    return SD_ERR_IO;
  std::vector<std::pair<uint64_t, sd_plan_opts_t>> rows;
  try {
    rows.resize((size_t)count);
  } catch (const std::bad_alloc &) {
    return SD_ERR_OUT_OF_MEMORY;
  }
  for (auto &r : rows) {
    if (std::fread(&r.first, sizeof(uint64_t), 1, fc.f) != 1 ||
        std::fread(&r.second, sizeof(sd_plan_opts_t), 1, fc.f) != 1)
      return SD_ERR_IO;
    // a record must be a plain plan choice (no search, a known family and valid options)
    if (r.second.search != 0 || r.second.force < SD_FMT_CSR_ROW || r.second.force > SD_FMT_SELL ||
        check_opts(r.second) != SD_OK)
      return SD_ERR_IO;
  }
  if (std::fgetc(fc.f) != EOF) return SD_ERR_IO;  // trailing bytes: not a file this library wrote
  std::lock_guard<std::mutex> lk(g_cache_mu);
  for (const auto &r : rows) g_cache[r.first] = r.second;
  return SD_OK;
}

namespace {

// A: host CSR; or src: device CSR on stream ds (A unused).  Returns kNeedHost
// when a device-source plan needs a host conversion.
int search_plan(const sd_csr_t *A, int32_t n, const sd_plan_opts_t &o, sd_plan_t *out, const sd_csr_t *src,
                hipStream_t ds) {
  sd::CsrView v;
  int st;
  sd_stats_t stats;
  if (src) {  // checks A and gives its statistics
    if ((st = sd::analyze_device(src, o.dense_threshold, &stats, ds)) != SD_OK) return st;
  } else if ((st = sd::validate_csr(A, &v)) != SD_OK) {
    return st;
  }
  auto build = [&](const sd_plan_opts_t &q, sd_plan_t *p) -> int {
    if (!src) return sd_plan_ex(A, n, &q, p);
    const int cs = check_opts(q);
    return cs != SD_OK ? cs : make_plan(nullptr, n, q, src, ds, p);
  };
  int dev = 0;
  hipError_t e = o.placement == 1 ? hipSuccess : hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e);
  if (o.placement == 1) dev = o.device;
  sd_plan_opts_t base = o;
  base.search = 0;
  uint64_t sig = 0;
  if ((st = device_signature(dev, &sig)) != SD_OK) return st;
  uint64_t pattern = 0;
  if (src) {
    hipError_t he = sd::dev_pattern_hash(src->rowptr, src->colidx, src->m, src->nnz, ds, &pattern);
    if (he != hipSuccess) return hip_fail(he);
  } else {
    pattern = sd::pattern_hash_host(v.rowptr, v.colidx, v.m, v.nnz);
  }
  const sd_csr_t *dims = src ? src : A;
  const uint64_t key = structure_key(dims->m, dims->k, dims->nnz, pattern, n, o.transpose ? 1 : 0, sig);
  bool hit = false;
  sd_plan_opts_t cached;
  {
    std::lock_guard<std::mutex> lk(g_cache_mu);
    auto it = g_cache.find(key);
    if (it != g_cache.end()) {
      hit = true;
      cached = it->second;
    }
  }
  if (hit) {
    st = build(cached, out);
    if (st == SD_OK) (*out)->info.search_cache_hit = 1;
    return st;
  }
  // statistics of the operand the kernels will see
  sd::CsrOwned At;
  DeviceTranspose Tt;
  if (o.transpose) {
    if (src) {
      if ((st = device_transpose(src, ds, &Tt)) != SD_OK) return st;
      if ((st = sd::analyze_device(&Tt.csr, o.dense_threshold, &stats, ds)) != SD_OK) return st;
    } else {
      if ((st = sd::transpose(v, &At)) != SD_OK) return st;
      v = At.view();
    }
  }
  if (!src && (st = sd::analyze(v, o.dense_threshold, &stats)) != SD_OK) return st;

  // the rule-based plan is the reference and the first candidate
  sd_plan_t best = nullptr;
  base.force = SD_FMT_AUTO;
  if ((st = build(base, &best)) != SD_OK) return st;
  const int64_t m = best->info.m, kk = best->info.k;
  if (m == 0) {
    *out = best;
    return SD_OK;
  }
  DeviceGuard guard;
  if ((st = guard.enter(best->device)) != SD_OK) {
    sd_plan_destroy(best);
    return st;
  }
  Scratch sc;
  std::vector<float> hb((size_t)std::max<int64_t>(1, kk * n));
  uint64_t x = 0x9e3779b97f4a7c15ull;
  for (auto &f : hb) {  // deterministic operand in [-1, 1)
    x = x * 6364136223846793005ull + 1442695040888963407ull;
    f = (float)((int32_t)(x >> 40) - (1 << 23)) * (1.0f / 8388608.0f);
  }
  const size_t cbytes = sizeof(float) * (size_t)(m * n);
  if ((e = hipMalloc(&sc.B, sizeof(float) * hb.size())) != hipSuccess || (e = hipMalloc(&sc.Cref, cbytes)) != hipSuccess ||
      (e = hipMalloc(&sc.C, cbytes)) != hipSuccess ||
      (e = hipMemcpy(sc.B, hb.data(), sizeof(float) * hb.size(), hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipStreamCreate(&sc.s)) != hipSuccess || (e = hipEventCreate(&sc.e0)) != hipSuccess ||
      (e = hipEventCreate(&sc.e1)) != hipSuccess) {
    (void)hipGetLastError();
    sd_plan_destroy(best);
    return e == hipErrorOutOfMemory ? SD_ERR_OUT_OF_MEMORY : hip_fail(e);
  }
  // the cache-flush buffer: 2 x the Infinity Cache; without it the search times warm
  sc.flush_bytes = 2 * (size_t)sd::kMallBytes;
  if (hipMalloc(&sc.flush, sc.flush_bytes) != hipSuccess || hipMalloc(&sc.sink, sizeof(float)) != hipSuccess ||
      hipMemset(sc.flush, 0, sc.flush_bytes) != hipSuccess) {
    (void)hipGetLastError();
    if (sc.flush) (void)hipFree(sc.flush);
    sc.flush = nullptr;
  }
  double best_ms = 0.0;
  if ((st = time_plan(best, sc, sc.Cref, &best_ms)) != SD_OK) {
    sd_plan_destroy(best);
    return st;
  }
  const double rule_ms = best_ms;
  std::vector<float> ref, got;
  int64_t stride = 1, rows = 0;
  if ((st = sample_rows(sc.Cref, m, n, &ref, &stride, &rows)) != SD_OK) {
    sd_plan_destroy(best);
    return st;
  }
  std::vector<double> rowmax((size_t)rows, 0.0);
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t j = 0; j < n; ++j) rowmax[r] = std::max(rowmax[r], (double)std::fabs(ref[r * n + j]));

  // candidates allowed by the statistics
  std::vector<sd_plan_opts_t> cands;
  // order 0 takes the family's default workgroup order; the other order is a
  // candidate of its own for the families that have one
  auto add = [&](int32_t fam, int32_t T, int32_t c, int32_t engine, int32_t order, int32_t chunk = 0,
                 int32_t slices = 0) {
    sd_plan_opts_t q = base;
    q.force = fam;
    q.heavy_threshold = T;
    q.chunk_nnz = c;
    q.engine = engine;
    q.wg_order = order;
    q.wg_chunk = chunk;
    q.row_slices = slices;
    if (fam == best->info.family && (fam != SD_FMT_CSR_SPLIT || (T == best->info.heavy_threshold &&
                                                              c == best->info.chunk_nnz)) &&
        (engine == 0 || engine == best->info.engine) &&
        (order == 0 || (order == best->info.wg_order && (order != 3 || chunk == best->info.wg_chunk))) &&
        (slices == 0 || slices == best->info.row_slices))
      return;  // the reference itself
    cands.push_back(q);
  };
  auto add_orders = [&](int32_t fam, int32_t engine) {
    add(fam, 0, 0, engine, 0);
    const bool block = fam == SD_FMT_BSR || fam == SD_FMT_BELL;
    add(fam, 0, 0, engine, block ? 2 : 1);
    if (!block) {  // chunked round-robin
      add(fam, 0, 0, engine, 3, 16);
      add(fam, 0, 0, engine, 3, 32);
    }
  };
  add_orders(SD_FMT_CSR_ROW, 0);
  if (stats.nnz > 0 && stats.rho_ell <= 3.0 && stats.row_max <= 1024) add_orders(SD_FMT_ELL, 0);
  if (stats.nnz > 0) add(SD_FMT_WIN, 0, 0, 0, 0);
  if (stats.nnz > 0 && stats.row_cv >= 0.3 && stats.row_max < 256) add(SD_FMT_SELL, 0, 0, 0, 0);
  if (stats.row_max >= 256) add(SD_FMT_CSR_SPLIT, 256, 256, 0, 0);
  if (stats.row_max >= 4096) add(SD_FMT_CSR_SPLIT, 512, 4096, 0, 0);
  if (stats.row_max >= 64) add(SD_FMT_CSR_SPLIT, 64, 64, 0, 0);
  add_orders(SD_FMT_CSR_MERGE, 0);
  // narrow widths: rows shared by S lane groups (G lanes cover the width)
  const int32_t G = best->info.col_tile / (n % 4 == 0 ? 4 : 1);
  if (G >= 1 && G <= 8 && stats.nnz > 0) {
    for (int32_t S = 1; S <= 64 / G; S *= 2) {
      add(SD_FMT_CSR_ROW, 0, 0, 0, 0, 0, S);
      if (stats.row_max >= 512) add(SD_FMT_CSR_SPLIT, 512, 2048, 0, 0, 0, S);
      if (stats.row_max >= 256 && S >= 4) add(SD_FMT_CSR_SPLIT, 256, 256 * (S / 2), 0, 0, 0, S);
    }
  }
  if (stats.row_max >= 512) {  // the split (default sizes) with its light rows ascending, its chunks in list order
    sd_plan_opts_t q = base;
    q.force = SD_FMT_CSR_SPLIT;
    q.light_order = 1;
    cands.push_back(q);
    q.light_order = 0;
    q.chunk_order = 1;
    cands.push_back(q);
  }
  if (stats.nnz > 0 && stats.rho_bsr16 <= 4.0) {
    add_orders(SD_FMT_BSR, SD_ENGINE_MFMA);
    add(SD_FMT_BSR, 0, 0, SD_ENGINE_VALU, 0);
  }
  int32_t timed = 1;
  for (const sd_plan_opts_t &q : cands) {
    sd_plan_t p = nullptr;
    if (build(q, &p) != SD_OK) continue;  // infeasible candidate: skipped
    double ms = 0.0;
    bool ok = time_plan(p, sc, sc.C, &ms) == SD_OK && sample_rows(sc.C, m, n, &got, &stride, &rows) == SD_OK;
    for (int64_t r = 0; ok && r < rows; ++r)
      for (int64_t j = 0; j < n; ++j) {
        const double a = got[r * n + j], b = ref[r * n + j];
        if (!(std::fabs(a - b) <= 1e-4 * (1.0 + rowmax[r])) && !(std::isnan(a) && std::isnan(b))) {
          ok = false;  // invalid candidate
          break;
        }
      }
    ++timed;
    if (ok && ms < best_ms) {
      sd_plan_destroy(best);
      best = p;
      best_ms = ms;
    } else {
      sd_plan_destroy(p);
    }
  }
  best->info.search_candidates = timed;
  best->info.search_best_ms = best_ms;
  best->info.search_rule_ms = rule_ms;
  sd_plan_opts_t chosen = base;
  chosen.force = best->info.family;
  chosen.engine = best->info.engine;
  chosen.heavy_threshold = (int32_t)best->info.heavy_threshold;
  chosen.chunk_nnz = (int32_t)best->info.chunk_nnz;
  chosen.units = (int32_t)best->info.units;
  chosen.wg_order = best->info.wg_order;
  chosen.wg_chunk = best->info.wg_chunk;
  chosen.sell_sigma = best->info.sell_sigma;
  chosen.window_rows = best->info.window_rows;
  chosen.row_slices = best->info.row_slices;
  chosen.light_order = best->info.light_order;
  chosen.chunk_order = best->info.chunk_order;
  {
    std::lock_guard<std::mutex> lk(g_cache_mu);
    g_cache[key] = chosen;
  }
  *out = best;
  return SD_OK;
}

}  // namespace
