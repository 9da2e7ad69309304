// Device-side conversions and partitions for plans built from a CSR matrix
// already in device memory (sd_plan_device).  Each produces exactly the
// arrays of its host counterpart in host_plan.cpp:
//
//  * ELL        rows padded to W slots, column -1 / value +0.0f padding;
//  * merge path U + 1 split coordinates (rows, nonzeros consumed), one binary
//               search per coordinate on the merged sequence of row ends and
//               nonzero indices;
//  * heavy split light rows (r < T) in row order; for heavy rows, chunks
//               (row, begin, end) of at most c nonzeros in row and chunk order,
//               the heavy rows and the first chunk of each (plus the total),
//               placed by exclusive prefix sums (hipCUB) of per-row counts;
//  * row reach  per row, the larger of |first column - row| and
//               |last column - row| (-1 for an empty row).
#include <hip/hip_runtime.h>
#include <hipcub/hipcub.hpp>

#include <algorithm>
#include <cstdint>
#include <functional>

#include "kernels.h"

namespace sd {
namespace {

__global__ __launch_bounds__(256) void k_ell_fill(const int32_t *__restrict__ rowptr,
                                                  const int32_t *__restrict__ colidx,
                                                  const float *__restrict__ vals, int32_t m, int32_t W,
                                                  int32_t *__restrict__ ecol, float *__restrict__ eval) {
  const int64_t slot = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (slot >= (int64_t)m * W) return;
  const int64_t i = slot / W, t = slot - i * W;
  const int32_t p0 = rowptr[i], r = rowptr[i + 1] - p0;
  if (t < r) {
    ecol[slot] = colidx[p0 + t];
    eval[slot] = vals[p0 + t];  // a bit copy: loads and stores move the pattern unchanged
  } else {
    ecol[slot] = -1;
    eval[slot] = 0.0f;
  }
}

__global__ __launch_bounds__(256) void k_merge_coords(const int32_t *__restrict__ rowptr, int32_t m, int64_t nnz,
                                                      int32_t U, int64_t L, int32_t *__restrict__ coords) {
  const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (u > U) return;
  const int64_t total = (int64_t)m + nnz;
  const int64_t d = min(u * L, total);
  int64_t lo = max((int64_t)0, d - nnz), hi = min(d, (int64_t)m);
  while (lo < hi) {
    const int64_t mid = (lo + hi) / 2;
    if ((int64_t)rowptr[mid + 1] + mid >= d) hi = mid;
    else lo = mid + 1;
  }
  coords[2 * u] = (int32_t)lo;
  coords[2 * u + 1] = (int32_t)(d - lo);
}

__global__ __launch_bounds__(256) void k_split_counts(const int32_t *__restrict__ rowptr, int32_t m, int32_t T,
                                                      int32_t c, int32_t *__restrict__ light,
                                                      int32_t *__restrict__ heavy, int32_t *__restrict__ pieces) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= m) return;
  const int64_t r = rowptr[i + 1] - rowptr[i];
  const bool is_light = r < T;
  light[i] = is_light ? 1 : 0;
  heavy[i] = is_light ? 0 : 1;
  pieces[i] = is_light ? 0 : (int32_t)((r + c - 1) / c);
}

__global__ __launch_bounds__(256) void k_split_fill(const int32_t *__restrict__ rowptr, int32_t m, int32_t T,
                                                    int32_t c, const int64_t *__restrict__ light_pos,
                                                    const int64_t *__restrict__ heavy_pos,
                                                    const int64_t *__restrict__ chunk_pos,
                                                    int32_t *__restrict__ light, int32_t *__restrict__ chunks,
                                                    int32_t *__restrict__ heavy_rows,
                                                    int32_t *__restrict__ heavy_ptr) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= m) return;
  const int32_t p0 = rowptr[i], p1 = rowptr[i + 1];
  if (p1 - p0 < T) {
    light[light_pos[i]] = (int32_t)i;
    return;
  }
  const int64_t h = heavy_pos[i], first = chunk_pos[i];
  heavy_rows[h] = (int32_t)i;
  heavy_ptr[h] = (int32_t)first;
  const int32_t n_pieces = (int32_t)(((int64_t)(p1 - p0) + c - 1) / c);
  for (int32_t q = 0; q < n_pieces; ++q) {
    const int32_t b = p0 + q * c;
    int32_t *ch = chunks + 3 * (first + q);
    ch[0] = (int32_t)i;
    ch[1] = b;
    ch[2] = min(p1, b + c);
  }
}

__global__ __launch_bounds__(256) void k_row_reach(const int32_t *__restrict__ rowptr,
                                                   const int32_t *__restrict__ colidx, int32_t m,
                                                   int64_t *__restrict__ reach) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= m) return;
  const int32_t p0 = rowptr[i], p1 = rowptr[i + 1];
  int64_t v = -1;  // empty rows are marked and skipped by the caller
  if (p1 > p0) {
    const int64_t a = colidx[p0] - i, b = colidx[p1 - 1] - i;
    v = max(a < 0 ? -a : a, b < 0 ? -b : b);
  }
  reach[i] = v;
}

uint32_t grid_for(int64_t items) { return (uint32_t)((items + 255) / 256); }

struct Scratch {
  void *p[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  ~Scratch() {
    for (void *q : p)
      if (q) (void)hipFree(q);
  }
};

}  // namespace

hipError_t dev_ell(const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t m, int32_t W,
                   int32_t *ecol, float *eval, hipStream_t s) {
  const int64_t slots = (int64_t)m * W;
  if (slots == 0) return hipSuccess;
  hipLaunchKernelGGL(k_ell_fill, dim3(grid_for(slots)), dim3(256), 0, s, rowptr, colidx, vals, m, W, ecol, eval);
  return hipGetLastError();
}

hipError_t dev_merge_coords(const int32_t *rowptr, int32_t m, int64_t nnz, int32_t U, int64_t L, int32_t *coords,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_merge_coords, dim3(grid_for((int64_t)U + 1)), dim3(256), 0, s, rowptr, m, nnz, U, L, coords);
  return hipGetLastError();
}

hipError_t dev_row_reach(const int32_t *rowptr, const int32_t *colidx, int32_t m, int64_t *reach, hipStream_t s) {
  if (m == 0) return hipSuccess;
  hipLaunchKernelGGL(k_row_reach, dim3(grid_for(m)), dim3(256), 0, s, rowptr, colidx, m, reach);
  return hipGetLastError();
}

hipError_t dev_heavy_split(const int32_t *rowptr, int32_t m, int32_t T, int32_t c,
                           const std::function<void *(size_t)> &alloc, hipStream_t s, int32_t **light,
                           int32_t **chunks, int32_t **heavy_rows, int32_t **heavy_ptr, int64_t *n_light,
                           int64_t *n_heavy, int64_t *n_chunks) {
  *light = *chunks = *heavy_rows = *heavy_ptr = nullptr;
  *n_light = *n_heavy = *n_chunks = 0;
  const size_t mm = (size_t)std::max(1, m);
  Scratch sc;  // flags / counts (int32 x 3) and their exclusive prefix sums (int64 x 3)
  hipError_t e;
  if ((e = hipMalloc(&sc.p[0], 3 * sizeof(int32_t) * mm)) != hipSuccess) return e;
  if ((e = hipMalloc(&sc.p[1], 3 * sizeof(int64_t) * (mm + 1))) != hipSuccess) return e;
  int32_t *f = static_cast<int32_t *>(sc.p[0]);
  int64_t *pos = static_cast<int64_t *>(sc.p[1]);
  int32_t *fl = f, *fh = f + mm, *fp = f + 2 * mm;
  int64_t *pl = pos, *ph = pos + (mm + 1), *pp = pos + 2 * (mm + 1);
  if (m > 0) {
    hipLaunchKernelGGL(k_split_counts, dim3(grid_for(m)), dim3(256), 0, s, rowptr, m, T, c, fl, fh, fp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // exclusive sums over the m rows; each total is the last prefix plus the last count
    size_t tmp_bytes = 0;
    if ((e = hipcub::DeviceScan::ExclusiveSum(nullptr, tmp_bytes, fl, pl, m, s)) != hipSuccess) return e;
    if ((e = hipMalloc(&sc.p[2], std::max<size_t>(tmp_bytes, 1))) != hipSuccess) return e;
    for (int t = 0; t < 3; ++t) {
      int32_t *in = t == 0 ? fl : t == 1 ? fh : fp;
      int64_t *out = t == 0 ? pl : t == 1 ? ph : pp;
      size_t b = tmp_bytes;
      if ((e = hipcub::DeviceScan::ExclusiveSum(sc.p[2], b, in, out, m, s)) != hipSuccess) return e;
    }
  }
  // totals: last prefix + last count
  int64_t last_pos[3] = {0, 0, 0};
  int32_t last_cnt[3] = {0, 0, 0};
  if (m > 0) {
    for (int t = 0; t < 3; ++t) {
      const int64_t *out = t == 0 ? pl : t == 1 ? ph : pp;
      const int32_t *in = t == 0 ? fl : t == 1 ? fh : fp;
      if ((e = hipMemcpyAsync(&last_pos[t], out + (m - 1), sizeof(int64_t), hipMemcpyDeviceToHost, s)) !=
              hipSuccess ||
          (e = hipMemcpyAsync(&last_cnt[t], in + (m - 1), sizeof(int32_t), hipMemcpyDeviceToHost, s)) != hipSuccess)
        return e;
    }
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
  }
  *n_light = last_pos[0] + last_cnt[0];
  *n_heavy = last_pos[1] + last_cnt[1];
  *n_chunks = last_pos[2] + last_cnt[2];
  *light = static_cast<int32_t *>(alloc(sizeof(int32_t) * (size_t)std::max<int64_t>(1, *n_light)));
  *chunks = static_cast<int32_t *>(alloc(3 * sizeof(int32_t) * (size_t)std::max<int64_t>(1, *n_chunks)));
  *heavy_rows = static_cast<int32_t *>(alloc(sizeof(int32_t) * (size_t)std::max<int64_t>(1, *n_heavy)));
  *heavy_ptr = static_cast<int32_t *>(alloc(sizeof(int32_t) * (size_t)(*n_heavy + 1)));
  if (!*light || !*chunks || !*heavy_rows || !*heavy_ptr) return hipErrorOutOfMemory;
  if (m > 0) {
    hipLaunchKernelGGL(k_split_fill, dim3(grid_for(m)), dim3(256), 0, s, rowptr, m, T, c, pl, ph, pp, *light,
                       *chunks, *heavy_rows, *heavy_ptr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const int32_t total = (int32_t)*n_chunks;
  if ((e = hipMemcpyAsync(*heavy_ptr + *n_heavy, &total, sizeof(int32_t), hipMemcpyHostToDevice, s)) != hipSuccess)
    return e;
  return hipStreamSynchronize(s);  // the scratch arrays are freed on return
}

}  // namespace sd
