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
//               |last column - row| (-1 for an empty row);
//  * transpose  the CSR of A^T: a stable radix sort (hipCUB) of the nonzero
//               positions by column keeps each column's rows ascending, as the
//               host's counting sort does; row pointers by binary search in
//               the sorted keys, source rows by binary search in A's rowptr;
//  * 16x16 BSR / Blocked-ELL  a stable radix sort of the nonzeros by
//               (block-row, block-column); the first nonzero of each key opens
//               a block, an inclusive scan numbers the blocks (block-columns
//               ascending within a block-row), block-row pointers by binary
//               search, then one thread per nonzero writes its value into the
//               zero-filled block (row-major inside the block);
//  * SELL-C-sigma  a stable radix sort of the rows by (sort window, longest
//               first) gives the permutation; slice widths, slice offsets by
//               an exclusive sum, then one thread per sorted row copies its
//               entries into the padded slice;
//  * windows    a stable radix sort of the nonzeros by (window, column): a
//               run of two or more equal keys is a staged column of that
//               window; scans number the runs and the staged columns, window
//               pointers by binary search, then one thread per nonzero writes
//               its code (staged position or column) and value;
//  * cold tags  column degrees by integer atomics; the hot threshold is taken
//               on the host from the degrees exactly as the host conversion
//               takes it; then one thread per nonzero sets bit 31 of a cold
//               column;
//  * pattern hash  the sum, modulo 2^64, of a mixed (array, position, value)
//               term per row pointer and column index: the same on the host
//               (pattern_hash in runtime.hip) and, being a sum, computed in any
//               order on the device.
#include <hip/hip_runtime.h>
#include <hipcub/hipcub.hpp>

#include <algorithm>
#include <cstdint>
#include <functional>
#include <vector>

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

// the row holding nonzero p of a valid CSR (m >= 1): the last row starting at
// or before p
__device__ inline int32_t row_of(const int32_t *__restrict__ rowptr, int32_t m, int64_t p) {
  int32_t lo = 0, hi = m - 1;
  while (lo < hi) {
    const int32_t mid = lo + (hi - lo + 1) / 2;
    if (rowptr[mid] <= p) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__global__ __launch_bounds__(256) void k_iota(int32_t *__restrict__ x, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) x[i] = (int32_t)i;
}

// t_rowptr[j] = number of sorted keys below j, for j in [0, k]
__global__ __launch_bounds__(256) void k_transpose_rowptr(const uint32_t *__restrict__ keys, int64_t nnz, int32_t k,
                                                          int32_t *__restrict__ t_rowptr) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j > k) return;
  int64_t lo = 0, hi = nnz;
  while (lo < hi) {
    const int64_t mid = (lo + hi) / 2;
    if ((int64_t)keys[mid] < j) lo = mid + 1;
    else hi = mid;
  }
  t_rowptr[j] = (int32_t)lo;
}

// entry q of A^T is A's nonzero perm[q]: its row (the last row starting at or
// before it) becomes the column, its value is copied bit for bit
__global__ __launch_bounds__(256) void k_transpose_fill(const int32_t *__restrict__ rowptr, int32_t m,
                                                        const float *__restrict__ vals,
                                                        const int32_t *__restrict__ perm, int64_t nnz,
                                                        int32_t *__restrict__ t_colidx, float *__restrict__ t_vals) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= nnz) return;
  const int32_t p = perm[q];
  t_colidx[q] = row_of(rowptr, m, p);
  t_vals[q] = vals[p];
}

__global__ __launch_bounds__(256) void k_block_keys(const int32_t *__restrict__ rowptr,
                                                    const int32_t *__restrict__ colidx, int32_t m, int64_t nnz,
                                                    int64_t kb, uint64_t *__restrict__ keys,
                                                    int32_t *__restrict__ pos) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= nnz) return;
  const int32_t i = row_of(rowptr, m, p);
  keys[p] = (uint64_t)(i / 16) * (uint64_t)kb + (uint64_t)(colidx[p] / 16);
  pos[p] = (int32_t)p;
}

__global__ __launch_bounds__(256) void k_block_heads(const uint64_t *__restrict__ skeys, int64_t nnz,
                                                     int32_t *__restrict__ head) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= nnz) return;
  head[q] = (q == 0 || skeys[q] != skeys[q - 1]) ? 1 : 0;
}

// ukey[b] = key of block b (blocks numbered by the inclusive scan of heads)
__global__ __launch_bounds__(256) void k_block_list(const uint64_t *__restrict__ skeys,
                                                    const int32_t *__restrict__ head,
                                                    const int32_t *__restrict__ incl, int64_t nnz,
                                                    uint64_t *__restrict__ ukey) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= nnz || !head[q]) return;
  ukey[incl[q] - 1] = skeys[q];
}

// bptr[br] = blocks in the block-rows before br, for br in [0, mb]
__global__ __launch_bounds__(256) void k_block_ptr(const uint64_t *__restrict__ ukey, int64_t nnzb, int64_t mb,
                                                   int64_t kb, int32_t *__restrict__ bptr) {
  const int64_t br = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (br > mb) return;
  const uint64_t target = (uint64_t)br * (uint64_t)kb;
  int64_t lo = 0, hi = nnzb;
  while (lo < hi) {
    const int64_t mid = (lo + hi) / 2;
    if (ukey[mid] < target) lo = mid + 1;
    else hi = mid;
  }
  bptr[br] = (int32_t)lo;
}

// block b's slot: b itself (BSR, ell_width < 0) or br * ell_width + its rank
// in the block-row (Blocked-ELL)
__device__ inline int64_t block_slot(int64_t b, uint64_t key, int64_t kb, const int32_t *__restrict__ bptr,
                                     int32_t ell_width) {
  if (ell_width < 0) return b;
  const int64_t br = (int64_t)(key / (uint64_t)kb);
  return br * ell_width + (b - bptr[br]);
}

__global__ __launch_bounds__(256) void k_block_cols(const uint64_t *__restrict__ ukey, int64_t nnzb, int64_t kb,
                                                    const int32_t *__restrict__ bptr, int32_t ell_width,
                                                    int32_t *__restrict__ bcol) {
  const int64_t b = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (b >= nnzb) return;
  const uint64_t key = ukey[b];
  bcol[block_slot(b, key, kb, bptr, ell_width)] = (int32_t)(key % (uint64_t)kb);
}

__global__ __launch_bounds__(256) void k_block_vals(const int32_t *__restrict__ rowptr,
                                                    const int32_t *__restrict__ colidx,
                                                    const float *__restrict__ vals, int32_t m, int64_t nnz,
                                                    const uint64_t *__restrict__ skeys,
                                                    const int32_t *__restrict__ perm,
                                                    const int32_t *__restrict__ incl, int64_t kb,
                                                    const int32_t *__restrict__ bptr, int32_t ell_width,
                                                    float *__restrict__ bval) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= nnz) return;
  const int32_t p = perm[q];
  const int32_t i = row_of(rowptr, m, p), c = colidx[p];
  const int64_t slot = block_slot(incl[q] - 1, skeys[q], kb, bptr, ell_width);
  bval[slot * 256 + (i % 16) * 16 + (c % 16)] = vals[p];
}

// ---- SELL-C-sigma
__global__ __launch_bounds__(256) void k_sell_keys(const int32_t *__restrict__ rowptr, int32_t m, int32_t sigma,
                                                   int32_t row_max, uint64_t *__restrict__ keys,
                                                   int32_t *__restrict__ rows) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= m) return;
  const int32_t len = rowptr[i + 1] - rowptr[i];
  keys[i] = (uint64_t)(i / sigma) * (uint64_t)(row_max + 1) + (uint64_t)(row_max - len);
  rows[i] = (int32_t)i;
}

__global__ __launch_bounds__(256) void k_sell_sizes(const int32_t *__restrict__ rowptr,
                                                    const int32_t *__restrict__ perm, int32_t m, int32_t C,
                                                    int64_t ns, int64_t *__restrict__ size) {
  const int64_t sl = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (sl >= ns) return;
  const int64_t r0 = sl * C, r1 = min((int64_t)m, r0 + C);
  int32_t w = 0;
  for (int64_t i = r0; i < r1; ++i) {
    const int32_t r = perm[i];
    w = max(w, rowptr[r + 1] - rowptr[r]);
  }
  size[sl] = (r1 - r0) * w;
}

__global__ __launch_bounds__(256) void k_sell_fill(const int32_t *__restrict__ rowptr,
                                                   const int32_t *__restrict__ colidx,
                                                   const float *__restrict__ vals, const int32_t *__restrict__ perm,
                                                   const int64_t *__restrict__ sptr, int32_t m, int32_t C,
                                                   int32_t *__restrict__ scol, float *__restrict__ sval) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= m) return;
  const int64_t sl = i / C, r0 = sl * C, rows = min((int64_t)m, r0 + C) - r0;
  const int64_t w = (sptr[sl + 1] - sptr[sl]) / rows;
  const int32_t r = perm[i], p0 = rowptr[r], len = rowptr[r + 1] - p0;
  const int64_t base = sptr[sl] + (i - r0) * w;
  for (int32_t t = 0; t < len; ++t) {
    scol[base + t] = colidx[p0 + t];
    sval[base + t] = vals[p0 + t];
  }
}

__global__ __launch_bounds__(256) void k_col_degree(const int32_t *__restrict__ colidx, int64_t nnz,
                                                    int32_t *__restrict__ deg) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p < nnz) atomicAdd(&deg[colidx[p]], 1);
}

__global__ __launch_bounds__(256) void k_tag_cold(const int32_t *__restrict__ colidx, int64_t nnz,
                                                  const int32_t *__restrict__ deg, int32_t D,
                                                  int32_t *__restrict__ tagged) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= nnz) return;
  const int32_t c = colidx[p];
  tagged[p] = deg[c] >= D ? c : (int32_t)((uint32_t)c | 0x80000000u);
}

// splitmix64's finaliser
__device__ __host__ inline uint64_t mix64(uint64_t x) {
  x ^= x >> 30;
  x *= 0xbf58476d1ce4e5b9ull;
  x ^= x >> 27;
  x *= 0x94d049bb133111ebull;
  x ^= x >> 31;
  return x;
}

__global__ __launch_bounds__(256) void k_pattern_hash(const int32_t *__restrict__ a, int64_t len, uint64_t salt,
                                                      unsigned long long *__restrict__ sum) {
  uint64_t acc = 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < len; i += (int64_t)gridDim.x * 256)
    acc += mix64(salt ^ ((uint64_t)i << 32 | (uint32_t)a[i]));
  atomicAdd(sum, (unsigned long long)acc);  // a sum: the same total in any order
}

__global__ __launch_bounds__(256) void k_fill_i32(int32_t *__restrict__ x, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) x[i] = v;
}

uint32_t grid_for(int64_t items) { return (uint32_t)((items + 255) / 256); }

// Device scratch of one conversion.  Freed on return, after the stream has
// drained: an early error return may leave kernels that use it in flight.
struct Scratch {
  hipStream_t s;
  void *p[12] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                 nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  explicit Scratch(hipStream_t stream) : s(stream) {}
  ~Scratch() {
    bool any = false;
    for (void *q : p) any = any || q;
    if (any) (void)hipStreamSynchronize(s);
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

__global__ void k_last_col_keys(const int32_t *__restrict__ rowptr, const int32_t *__restrict__ colidx, int32_t k,
                                const int32_t *__restrict__ light, int64_t n, int32_t *__restrict__ keys) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t r = light[i];
  keys[i] = rowptr[r + 1] > rowptr[r] ? colidx[rowptr[r + 1] - 1] : k;
}

hipError_t dev_light_by_last_col(const int32_t *rowptr, const int32_t *colidx, int32_t k, int32_t *light,
                                 int64_t n_light, hipStream_t s) {
  if (n_light < 2) return hipSuccess;
  if (n_light > INT32_MAX) return hipErrorInvalidValue;
  const int n = (int)n_light;
  Scratch sc(s);  // keys in / out, rows out, sort workspace
  hipError_t e;
  if ((e = hipMalloc(&sc.p[0], 2 * sizeof(int32_t) * (size_t)n)) != hipSuccess) return e;
  if ((e = hipMalloc(&sc.p[1], sizeof(int32_t) * (size_t)n)) != hipSuccess) return e;
  int32_t *kin = static_cast<int32_t *>(sc.p[0]), *kout = kin + n, *rout = static_cast<int32_t *>(sc.p[1]);
  hipLaunchKernelGGL(k_last_col_keys, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, rowptr, colidx, k, light,
                     n_light, kin);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  int bits = 1;
  while (bits < 31 && ((int64_t)1 << bits) <= (int64_t)k) ++bits;  // keys lie in [0, k]
  size_t tmp = 0;
  if ((e = hipcub::DeviceRadixSort::SortPairs(nullptr, tmp, kin, kout, light, rout, n, 0, bits, s)) != hipSuccess)
    return e;
  if ((e = hipMalloc(&sc.p[2], std::max<size_t>(tmp, 1))) != hipSuccess) return e;
  if ((e = hipcub::DeviceRadixSort::SortPairs(sc.p[2], tmp, kin, kout, light, rout, n, 0, bits, s)) != hipSuccess)
    return e;
  if ((e = hipMemcpyAsync(light, rout, sizeof(int32_t) * (size_t)n, hipMemcpyDeviceToDevice, s)) != hipSuccess)
    return e;
  return hipStreamSynchronize(s);  // the scratch arrays are freed on return
}

__global__ void k_chunk_mid_keys(const int32_t *__restrict__ colidx, const int32_t *__restrict__ chunks, int64_t n,
                                 int32_t *__restrict__ keys, int32_t *__restrict__ idx) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= n) return;
  const int64_t b = chunks[3 * q + 1], e = chunks[3 * q + 2];
  keys[q] = colidx[(b + e) / 2];
  idx[q] = (int32_t)q;
}

hipError_t dev_chunk_order(const int32_t *colidx, const int32_t *chunks, int64_t n_chunks, int32_t k, int32_t order,
                           int32_t *corder, hipStream_t s) {
  if (n_chunks == 0) return hipSuccess;
  if (n_chunks > INT32_MAX) return hipErrorInvalidValue;
  const int n = (int)n_chunks;
  if (order != 2 || n < 2) {
    hipLaunchKernelGGL(k_iota, dim3(grid_for(n)), dim3(256), 0, s, corder, (int64_t)n);
    return hipGetLastError();
  }
  Scratch sc(s);  // keys in / out, indices in, sort workspace
  hipError_t e;
  if ((e = hipMalloc(&sc.p[0], 2 * sizeof(int32_t) * (size_t)n)) != hipSuccess) return e;
  if ((e = hipMalloc(&sc.p[1], sizeof(int32_t) * (size_t)n)) != hipSuccess) return e;
  int32_t *kin = static_cast<int32_t *>(sc.p[0]), *kout = kin + n, *iin = static_cast<int32_t *>(sc.p[1]);
  hipLaunchKernelGGL(k_chunk_mid_keys, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, colidx, chunks,
                     (int64_t)n, kin, iin);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  int bits = 1;
  while (bits < 31 && ((int64_t)1 << bits) < (int64_t)k) ++bits;  // keys lie in [0, k)
  size_t tmp = 0;
  // a radix sort is stable: equal keys keep ascending chunk indices
  if ((e = hipcub::DeviceRadixSort::SortPairs(nullptr, tmp, kin, kout, iin, corder, n, 0, bits, s)) != hipSuccess)
    return e;
  if ((e = hipMalloc(&sc.p[2], std::max<size_t>(tmp, 1))) != hipSuccess) return e;
  if ((e = hipcub::DeviceRadixSort::SortPairs(sc.p[2], tmp, kin, kout, iin, corder, n, 0, bits, s)) != hipSuccess)
    return e;
  return hipStreamSynchronize(s);  // the scratch arrays are freed on return
}

__global__ void k_row_lengths(const int32_t *__restrict__ rowptr, const int32_t *__restrict__ rows, int64_t n,
                              int64_t *__restrict__ len) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) len[i] = (int64_t)rowptr[rows[i] + 1] - rowptr[rows[i]];
}

// One wave per listed row: its entries to [start[i], start[i] + length).
__global__ void k_move_rows(const int32_t *__restrict__ rowptr, const int32_t *__restrict__ colidx,
                            const float *__restrict__ vals, const int32_t *__restrict__ rows,
                            const int64_t *__restrict__ start, int64_t base, int64_t n,
                            int32_t *__restrict__ colidx_out, float *__restrict__ vals_out) {
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= n) return;
  const int32_t r = rows[i];
  const int32_t p0 = rowptr[r], len = rowptr[r + 1] - p0;
  const int64_t q0 = base + start[i];
  for (int32_t t = threadIdx.x & 63; t < len; t += 64) {
    colidx_out[q0 + t] = colidx[p0 + t];
    vals_out[q0 + t] = vals[p0 + t];
  }
}

__global__ void k_lptr_from_starts(const int64_t *__restrict__ start, const int64_t *__restrict__ len, int64_t n,
                                   int32_t *__restrict__ lptr) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) lptr[i] = (int32_t)start[i];
  if (i == n - 1) lptr[n] = (int32_t)(start[i] + len[i]);
}

// Heavy row h: its chunks move by (new start - old start).
__global__ void k_shift_chunks(const int32_t *__restrict__ rowptr, const int32_t *__restrict__ heavy_rows,
                               const int32_t *__restrict__ heavy_ptr, const int64_t *__restrict__ start,
                               int64_t base, int64_t n_heavy, int32_t *__restrict__ chunks) {
  const int64_t h = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (h >= n_heavy) return;
  const int64_t shift = base + start[h] - rowptr[heavy_rows[h]];
  for (int32_t q = heavy_ptr[h]; q < heavy_ptr[h + 1]; ++q) {
    chunks[3 * (int64_t)q + 1] = (int32_t)(chunks[3 * (int64_t)q + 1] + shift);
    chunks[3 * (int64_t)q + 2] = (int32_t)(chunks[3 * (int64_t)q + 2] + shift);
  }
}

hipError_t dev_split_layout(const int32_t *rowptr, const int32_t *colidx, const float *vals, int64_t nnz,
                            const int32_t *light, int64_t n_light, const int32_t *heavy_rows,
                            const int32_t *heavy_ptr, int64_t n_heavy, int32_t *lptr, int32_t *colidx_out,
                            float *vals_out, int32_t *chunks, hipStream_t s) {
  (void)nnz;
  Scratch sc(s);  // lengths and starts (int64) of the light rows, then of the heavy rows; scan workspace
  hipError_t e;
  const int64_t nl = std::max<int64_t>(1, n_light), nh = std::max<int64_t>(1, n_heavy);
  if ((e = hipMalloc(&sc.p[0], 2 * sizeof(int64_t) * (size_t)(nl + nh))) != hipSuccess) return e;
  int64_t *len_l = static_cast<int64_t *>(sc.p[0]), *st_l = len_l + nl, *len_h = st_l + nl, *st_h = len_h + nh;
  int64_t light_total = 0;
  if (n_light > 0) {
    const uint32_t g = (uint32_t)((n_light + 255) / 256);
    hipLaunchKernelGGL(k_row_lengths, dim3(g), dim3(256), 0, s, rowptr, light, n_light, len_l);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    size_t tmp = 0;
    if ((e = hipcub::DeviceScan::ExclusiveSum(nullptr, tmp, len_l, st_l, (int)n_light, s)) != hipSuccess) return e;
    if ((e = hipMalloc(&sc.p[1], std::max<size_t>(tmp, 1))) != hipSuccess) return e;
    if ((e = hipcub::DeviceScan::ExclusiveSum(sc.p[1], tmp, len_l, st_l, (int)n_light, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_lptr_from_starts, dim3(g), dim3(256), 0, s, st_l, len_l, n_light, lptr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_move_rows, dim3((uint32_t)((n_light + 3) / 4)), dim3(256), 0, s, rowptr, colidx, vals, light,
                       st_l, (int64_t)0, n_light, colidx_out, vals_out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    int64_t last[2] = {0, 0};
    if ((e = hipMemcpyAsync(&last[0], st_l + n_light - 1, sizeof(int64_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipMemcpyAsync(&last[1], len_l + n_light - 1, sizeof(int64_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
      return e;
    light_total = last[0] + last[1];
  } else {
    const int32_t zero = 0;
    if ((e = hipMemcpyAsync(lptr, &zero, sizeof(int32_t), hipMemcpyHostToDevice, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
      return e;
  }
  if (n_heavy > 0) {
    const uint32_t g = (uint32_t)((n_heavy + 255) / 256);
    hipLaunchKernelGGL(k_row_lengths, dim3(g), dim3(256), 0, s, rowptr, heavy_rows, n_heavy, len_h);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    size_t tmp = 0;
    if ((e = hipcub::DeviceScan::ExclusiveSum(nullptr, tmp, len_h, st_h, (int)n_heavy, s)) != hipSuccess) return e;
    if ((e = hipMalloc(&sc.p[2], std::max<size_t>(tmp, 1))) != hipSuccess) return e;
    if ((e = hipcub::DeviceScan::ExclusiveSum(sc.p[2], tmp, len_h, st_h, (int)n_heavy, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_move_rows, dim3((uint32_t)((n_heavy + 3) / 4)), dim3(256), 0, s, rowptr, colidx, vals,
                       heavy_rows, st_h, light_total, n_heavy, colidx_out, vals_out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_shift_chunks, dim3(g), dim3(256), 0, s, rowptr, heavy_rows, heavy_ptr, st_h, light_total,
                       n_heavy, chunks);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipStreamSynchronize(s);  // the scratch arrays are freed on return
}

// ---- packed column windows over the split layout
// Light entry p belongs to the light row t with lptr[t] <= p < lptr[t + 1]
// (the last such t when empty rows share a pointer) and to window t / R; its
// key is (window << 32) | column.
__global__ __launch_bounds__(256) void k_win_entry_keys(const int32_t *__restrict__ lptr, int64_t n_light,
                                                        const int32_t *__restrict__ colidx, int64_t E, int32_t R,
                                                        uint64_t *__restrict__ keys) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= E) return;
  int64_t lo = 0, hi = n_light - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) / 2;
    if (lptr[mid] <= p) lo = mid;
    else hi = mid - 1;
  }
  keys[p] = ((uint64_t)(lo / R) << 32) | (uint32_t)colidx[p];
}

// Runs of equal (window, column) keys: a run of two or more is a candidate,
// keyed (window, uses descending, column) so that a window's most used come
// first; the rest sort to the end.
__global__ __launch_bounds__(256) void k_win_candidates(const uint64_t *__restrict__ run_key,
                                                        const int32_t *__restrict__ run_len,
                                                        const int32_t *__restrict__ n_runs, int32_t cbits,
                                                        uint64_t *__restrict__ key2) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= *n_runs) return;
  const uint64_t w = run_key[i] >> 32, col = run_key[i] & 0xffffffffull;
  const uint64_t inv = ((1ull << cbits) - 1) - (uint64_t)run_len[i];
  key2[i] = run_len[i] >= 2 ? (w << (cbits + 32)) | (inv << 32) | col : ~0ull;
}

// Candidate i (sorted) is kept when fewer than cap candidates of its window
// precede it; kept ones are re-keyed (window, column), the others sort last.
__global__ __launch_bounds__(256) void k_win_keep(const uint64_t *__restrict__ key2, const int32_t *__restrict__ n_runs,
                                                  int32_t cbits, int32_t cap, uint64_t *__restrict__ key3,
                                                  int32_t *__restrict__ kept) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= *n_runs) return;
  const uint64_t k = key2[i];
  kept[i] = 0;
  if (k == ~0ull) {
    key3[i] = ~0ull;
    return;
  }
  const uint64_t w = k >> (cbits + 32);
  const uint64_t first_key = w << (cbits + 32);
  int64_t lo = 0, hi = i;  // first index whose key is >= first_key
  while (lo < hi) {
    const int64_t mid = (lo + hi) / 2;
    if (key2[mid] < first_key) lo = mid + 1;
    else hi = mid;
  }
  key3[i] = (i - lo < cap) ? (w << 32) | (k & 0xffffffffull) : ~0ull;
  kept[i] = (i - lo < cap) ? 1 : 0;
}

// wptr[w] = first staged key of window w (keys sorted, kept ones first).
__global__ __launch_bounds__(256) void k_win_ptr_cols(const uint64_t *__restrict__ key3, int64_t n_kept, int64_t nw,
                                                      int32_t *__restrict__ wptr, int32_t *__restrict__ wcols) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n_kept) wcols[i] = (int32_t)(key3[i] & 0xffffffffull);
  if (i > nw) return;
  const uint64_t target = (uint64_t)i << 32;
  int64_t lo = 0, hi = n_kept;
  while (lo < hi) {
    const int64_t mid = (lo + hi) / 2;
    if (key3[mid] < target) lo = mid + 1;
    else hi = mid;
  }
  wptr[i] = (int32_t)lo;
}

// Entry codes: -2 - (position among its window's staged columns), else the
// column; staged[p] = 1 for an entry that reads a staged column.
__global__ __launch_bounds__(256) void k_win_codes(const uint64_t *__restrict__ entry_key,
                                                   const int32_t *__restrict__ wptr, const int32_t *__restrict__ wcols,
                                                   int64_t E, int32_t *__restrict__ code, int32_t *__restrict__ staged) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= E) return;
  const int64_t w = (int64_t)(entry_key[p] >> 32);
  const int32_t col = (int32_t)(entry_key[p] & 0xffffffffull);
  int64_t lo = wptr[w], hi = wptr[w + 1];
  while (lo < hi) {
    const int64_t mid = (lo + hi) / 2;
    if (wcols[mid] < col) lo = mid + 1;
    else hi = mid;
  }
  const bool hit = lo < wptr[w + 1] && wcols[lo] == col;
  code[p] = hit ? (int32_t)(-2 - (lo - wptr[w])) : col;
  staged[p] = hit ? 1 : 0;
}

hipError_t dev_split_windows(const int32_t *lptr, int64_t n_light, int32_t *colidx, int32_t R, int32_t cap,
                             const std::function<void *(size_t)> &alloc, hipStream_t s, int32_t **wptr,
                             int32_t **wcols, int32_t *wmax, int64_t *n_staged, int64_t *staged_uses) {
  *wmax = 0;
  *n_staged = 0;
  *staged_uses = 0;
  const int64_t nw = (n_light + R - 1) / R;
  hipError_t e;
  int32_t E32 = 0;
  if (n_light > 0) {
    if ((e = hipMemcpyAsync(&E32, lptr + n_light, sizeof(int32_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
      return e;
  }
  const int64_t E = E32;
  *wptr = static_cast<int32_t *>(alloc(sizeof(int32_t) * (size_t)(nw + 1)));
  if (!*wptr) return hipErrorOutOfMemory;
  if (E == 0 || cap < 1 || R < 2) {  // nothing can be staged: every code is its column
    hipLaunchKernelGGL(k_fill_i32, dim3(grid_for(nw + 1)), dim3(256), 0, s, *wptr, nw + 1, 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    *wcols = static_cast<int32_t *>(alloc(sizeof(int32_t)));
    if (!*wcols) return hipErrorOutOfMemory;
    return hipStreamSynchronize(s);
  }
  if (E > INT32_MAX / 2) return hipErrorInvalidValue;
  const int n = (int)E;
  Scratch sc(s);
  // entry keys, sorted keys, run keys, run lengths + run count, candidate keys (x2), kept keys (x2), flags, temp
  if ((e = hipMalloc(&sc.p[0], sizeof(uint64_t) * (size_t)n)) != hipSuccess) return e;
  if ((e = hipMalloc(&sc.p[1], sizeof(uint64_t) * (size_t)n)) != hipSuccess) return e;
  if ((e = hipMalloc(&sc.p[2], sizeof(uint64_t) * (size_t)n)) != hipSuccess) return e;
  if ((e = hipMalloc(&sc.p[3], sizeof(int32_t) * ((size_t)n + 1))) != hipSuccess) return e;
  if ((e = hipMalloc(&sc.p[4], 2 * sizeof(uint64_t) * (size_t)n)) != hipSuccess) return e;
  if ((e = hipMalloc(&sc.p[5], sizeof(int32_t) * (size_t)n)) != hipSuccess) return e;
  if ((e = hipMalloc(&sc.p[6], sizeof(int64_t))) != hipSuccess) return e;
  uint64_t *ekey = static_cast<uint64_t *>(sc.p[0]), *skey = static_cast<uint64_t *>(sc.p[1]);
  uint64_t *rkey = static_cast<uint64_t *>(sc.p[2]);
  int32_t *rlen = static_cast<int32_t *>(sc.p[3]), *nruns = rlen + n;
  uint64_t *k2 = static_cast<uint64_t *>(sc.p[4]), *k2s = k2 + n;
  int32_t *flag = static_cast<int32_t *>(sc.p[5]);
  int64_t *uses_d = static_cast<int64_t *>(sc.p[6]);
  int wbits = 1;
  while (wbits < 31 && ((int64_t)1 << wbits) < nw) ++wbits;
  int cbits = 1;  // uses are at most R (each row uses a column once)
  while (cbits < 31 && ((int64_t)1 << cbits) <= (int64_t)R) ++cbits;
  if (wbits + cbits > 32) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_win_entry_keys, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, lptr, n_light, colidx, E, R,
                     ekey);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  size_t t1 = 0, t2 = 0, t3 = 0, t4 = 0, t5 = 0;
  if ((e = hipcub::DeviceRadixSort::SortKeys(nullptr, t1, ekey, skey, n, 0, 32 + wbits, s)) != hipSuccess) return e;
  if ((e = hipcub::DeviceRunLengthEncode::Encode(nullptr, t2, skey, rkey, rlen, nruns, n, s)) != hipSuccess) return e;
  if ((e = hipcub::DeviceRadixSort::SortKeys(nullptr, t3, k2, k2s, n, 0, 64, s)) != hipSuccess) return e;
  if ((e = hipcub::DeviceReduce::Sum(nullptr, t4, flag, uses_d, n, s)) != hipSuccess) return e;
  t5 = std::max({t1, t2, t3, t4, (size_t)1});
  if ((e = hipMalloc(&sc.p[7], t5)) != hipSuccess) return e;
  if ((e = hipcub::DeviceRadixSort::SortKeys(sc.p[7], t1, ekey, skey, n, 0, 32 + wbits, s)) != hipSuccess) return e;
  if ((e = hipcub::DeviceRunLengthEncode::Encode(sc.p[7], t2, skey, rkey, rlen, nruns, n, s)) != hipSuccess)
    return e;
  hipLaunchKernelGGL(k_win_candidates, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, rkey, rlen, nruns, cbits,
                     k2);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  int32_t runs = 0;
  if ((e = hipMemcpyAsync(&runs, nruns, sizeof(int32_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return e;
  if ((e = hipcub::DeviceRadixSort::SortKeys(sc.p[7], t3, k2, k2s, runs, 0, 64, s)) != hipSuccess) return e;
  // kept candidates re-keyed (window, column) into k2, then sorted into skey
  hipLaunchKernelGGL(k_win_keep, dim3((uint32_t)((runs + 255) / 256)), dim3(256), 0, s, k2s, nruns, cbits, cap, k2,
                     flag);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = hipcub::DeviceRadixSort::SortKeys(sc.p[7], t3, k2, skey, runs, 0, 64, s)) != hipSuccess) return e;
  int64_t n_kept = 0;  // the kept keys sort first
  if ((e = hipcub::DeviceReduce::Sum(sc.p[7], t4, flag, uses_d, runs, s)) != hipSuccess ||
      (e = hipMemcpyAsync(&n_kept, uses_d, sizeof(int64_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return e;
  *wcols = static_cast<int32_t *>(alloc(sizeof(int32_t) * (size_t)std::max<int64_t>(1, n_kept)));
  if (!*wcols) return hipErrorOutOfMemory;
  hipLaunchKernelGGL(k_win_ptr_cols, dim3(grid_for(std::max<int64_t>(n_kept, nw + 1))), dim3(256), 0, s, skey, n_kept,
                     nw, *wptr, *wcols);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_win_codes, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, ekey, *wptr, *wcols, E, colidx,
                     flag);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = hipcub::DeviceReduce::Sum(sc.p[7], t4, flag, uses_d, n, s)) != hipSuccess) return e;
  std::vector<int32_t> hw((size_t)nw + 1);
  if ((e = hipMemcpyAsync(hw.data(), *wptr, sizeof(int32_t) * hw.size(), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipMemcpyAsync(staged_uses, uses_d, sizeof(int64_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return e;
  for (int64_t w = 0; w < nw; ++w) *wmax = std::max(*wmax, hw[(size_t)w + 1] - hw[(size_t)w]);
  *n_staged = n_kept;
  return hipSuccess;  // synchronised above; the scratch arrays are freed on return
}

hipError_t dev_heavy_split(const int32_t *rowptr, int32_t m, int32_t T, int32_t c,
                           const std::function<void *(size_t)> &alloc, hipStream_t s, int32_t **light,
                           int32_t **chunks, int32_t **heavy_rows, int32_t **heavy_ptr, int64_t *n_light,
                           int64_t *n_heavy, int64_t *n_chunks) {
  *light = *chunks = *heavy_rows = *heavy_ptr = nullptr;
  *n_light = *n_heavy = *n_chunks = 0;
  const size_t mm = (size_t)std::max(1, m);
  Scratch sc(s);  // flags / counts (int32 x 3) and their exclusive prefix sums (int64 x 3)
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

hipError_t dev_block16(const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t m, int32_t k,
                       int64_t nnz, int64_t nnzb, int32_t ell_width, int32_t *bptr, int32_t *bcol, float *bval,
                       hipStream_t s) {
  const int64_t mb = ((int64_t)m + 15) / 16, kb = std::max<int64_t>(1, ((int64_t)k + 15) / 16);
  const int64_t slots = ell_width >= 0 ? mb * ell_width : nnzb;
  hipError_t e;
  Scratch sc(s);  // keys, sorted keys, positions, sorted positions, heads, block numbers, block keys, temporary, bptr
  int32_t *ptr = bptr;
  if (!ptr) {
    if ((e = hipMalloc(&sc.p[8], sizeof(int32_t) * (size_t)(mb + 1))) != hipSuccess) return e;
    ptr = static_cast<int32_t *>(sc.p[8]);
  }
  // padding, and the zero block after the stored ones
  if ((e = hipMemsetAsync(bval, 0, sizeof(float) * 256 * (size_t)(slots + 1), s)) != hipSuccess) return e;
  hipLaunchKernelGGL(k_fill_i32, dim3(grid_for(slots + 1)), dim3(256), 0, s, bcol, slots + 1, -1);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (nnz == 0) {
    if (nnzb != 0) return hipErrorInvalidValue;
    if ((e = hipMemsetAsync(ptr, 0, sizeof(int32_t) * (size_t)(mb + 1), s)) != hipSuccess) return e;
    return hipStreamSynchronize(s);
  }
  const size_t n4 = sizeof(int32_t) * (size_t)nnz, n8 = sizeof(uint64_t) * (size_t)nnz;
  if ((e = hipMalloc(&sc.p[0], n8)) != hipSuccess || (e = hipMalloc(&sc.p[1], n8)) != hipSuccess ||
      (e = hipMalloc(&sc.p[2], n4)) != hipSuccess || (e = hipMalloc(&sc.p[3], n4)) != hipSuccess ||
      (e = hipMalloc(&sc.p[4], n4)) != hipSuccess || (e = hipMalloc(&sc.p[5], n4)) != hipSuccess ||
      (e = hipMalloc(&sc.p[6], sizeof(uint64_t) * (size_t)std::max<int64_t>(1, nnzb))) != hipSuccess)
    return e;
  uint64_t *keys = static_cast<uint64_t *>(sc.p[0]), *skeys = static_cast<uint64_t *>(sc.p[1]);
  int32_t *pos = static_cast<int32_t *>(sc.p[2]), *perm = static_cast<int32_t *>(sc.p[3]);
  int32_t *head = static_cast<int32_t *>(sc.p[4]), *incl = static_cast<int32_t *>(sc.p[5]);
  uint64_t *ukey = static_cast<uint64_t *>(sc.p[6]);
  hipLaunchKernelGGL(k_block_keys, dim3(grid_for(nnz)), dim3(256), 0, s, rowptr, colidx, m, nnz, kb, keys, pos);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const uint64_t n_keys = (uint64_t)mb * (uint64_t)kb;  // every key is below this
  int end_bit = 1;
  while (end_bit < 64 && ((uint64_t)1 << end_bit) < n_keys) ++end_bit;
  size_t tmp_sort = 0, tmp_scan = 0;
  if ((e = hipcub::DeviceRadixSort::SortPairs(nullptr, tmp_sort, keys, skeys, pos, perm, (int)nnz, 0, end_bit,
                                               s)) != hipSuccess ||
      (e = hipcub::DeviceScan::InclusiveSum(nullptr, tmp_scan, head, incl, (int)nnz, s)) != hipSuccess)
    return e;
  size_t tmp = std::max<size_t>({tmp_sort, tmp_scan, 1});
  if ((e = hipMalloc(&sc.p[7], tmp)) != hipSuccess) return e;
  if ((e = hipcub::DeviceRadixSort::SortPairs(sc.p[7], tmp_sort, keys, skeys, pos, perm, (int)nnz, 0, end_bit,
                                               s)) != hipSuccess)
    return e;
  hipLaunchKernelGGL(k_block_heads, dim3(grid_for(nnz)), dim3(256), 0, s, skeys, nnz, head);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = hipcub::DeviceScan::InclusiveSum(sc.p[7], tmp_scan, head, incl, (int)nnz, s)) != hipSuccess) return e;
  // nothing is written by block number before the count agrees with the
  // storage sized from the analysis
  int32_t total = 0;
  if ((e = hipMemcpyAsync(&total, incl + (nnz - 1), sizeof(int32_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return e;
  if ((int64_t)total != nnzb) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_block_list, dim3(grid_for(nnz)), dim3(256), 0, s, skeys, head, incl, nnz, ukey);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_block_ptr, dim3(grid_for(mb + 1)), dim3(256), 0, s, ukey, nnzb, mb, kb, ptr);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (ell_width >= 0) {  // every block-row must fit the padded width
    std::vector<int32_t> h((size_t)mb + 1);
    if ((e = hipMemcpyAsync(h.data(), ptr, sizeof(int32_t) * h.size(), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
      return e;
    for (int64_t br = 0; br < mb; ++br)
      if (h[br + 1] - h[br] > ell_width) return hipErrorInvalidValue;
  }
  hipLaunchKernelGGL(k_block_cols, dim3(grid_for(nnzb)), dim3(256), 0, s, ukey, nnzb, kb, ptr, ell_width, bcol);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_block_vals, dim3(grid_for(nnz)), dim3(256), 0, s, rowptr, colidx, vals, m, nnz, skeys, perm,
                     incl, kb, ptr, ell_width, bval);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return hipStreamSynchronize(s);  // the scratch arrays are freed on return
}

hipError_t dev_sell(const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t m, int32_t row_max,
                    int32_t C, int32_t sigma, int64_t max_slots, const std::function<void *(size_t)> &alloc,
                    hipStream_t s, int32_t **perm, int64_t **sptr, int32_t **scol, float **sval, int64_t *slots) {
  *perm = nullptr;
  *sptr = nullptr;
  *scol = nullptr;
  *sval = nullptr;
  *slots = 0;
  const int64_t ns = ((int64_t)m + C - 1) / C;
  hipError_t e;
  *perm = static_cast<int32_t *>(alloc(sizeof(int32_t) * (size_t)std::max(1, m)));
  *sptr = static_cast<int64_t *>(alloc(sizeof(int64_t) * (size_t)(ns + 1)));
  if (!*perm || !*sptr) return hipErrorOutOfMemory;
  if (m == 0) {
    if ((e = hipMemsetAsync(*sptr, 0, sizeof(int64_t), s)) != hipSuccess) return e;
    *scol = static_cast<int32_t *>(alloc(sizeof(int32_t)));
    *sval = static_cast<float *>(alloc(sizeof(float)));
    if (!*scol || !*sval) return hipErrorOutOfMemory;
    return hipStreamSynchronize(s);
  }
  Scratch sc(s);  // keys, sorted keys, rows, slice sizes, temporary
  const size_t mm = (size_t)m;
  if ((e = hipMalloc(&sc.p[0], 8 * mm)) != hipSuccess || (e = hipMalloc(&sc.p[1], 8 * mm)) != hipSuccess ||
      (e = hipMalloc(&sc.p[2], 4 * mm)) != hipSuccess || (e = hipMalloc(&sc.p[3], 8 * (size_t)ns)) != hipSuccess)
    return e;
  uint64_t *keys = static_cast<uint64_t *>(sc.p[0]), *skeys = static_cast<uint64_t *>(sc.p[1]);
  int32_t *rows = static_cast<int32_t *>(sc.p[2]);
  int64_t *size = static_cast<int64_t *>(sc.p[3]);
  hipLaunchKernelGGL(k_sell_keys, dim3(grid_for(m)), dim3(256), 0, s, rowptr, m, sigma, row_max, keys, rows);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const uint64_t n_keys = (uint64_t)((m + (int64_t)sigma - 1) / sigma) * (uint64_t)(row_max + 1);
  int end_bit = 1;
  while (end_bit < 64 && ((uint64_t)1 << end_bit) < n_keys) ++end_bit;
  size_t tmp_sort = 0, tmp_scan = 0;
  if ((e = hipcub::DeviceRadixSort::SortPairs(nullptr, tmp_sort, keys, skeys, rows, *perm, m, 0, end_bit, s)) !=
          hipSuccess ||
      (e = hipcub::DeviceScan::ExclusiveSum(nullptr, tmp_scan, size, *sptr, (int)ns, s)) != hipSuccess)
    return e;
  if ((e = hipMalloc(&sc.p[4], std::max<size_t>({tmp_sort, tmp_scan, 1}))) != hipSuccess) return e;
  if ((e = hipcub::DeviceRadixSort::SortPairs(sc.p[4], tmp_sort, keys, skeys, rows, *perm, m, 0, end_bit, s)) !=
      hipSuccess)
    return e;
  hipLaunchKernelGGL(k_sell_sizes, dim3(grid_for(ns)), dim3(256), 0, s, rowptr, *perm, m, C, ns, size);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = hipcub::DeviceScan::ExclusiveSum(sc.p[4], tmp_scan, size, *sptr, (int)ns, s)) != hipSuccess) return e;
  int64_t last[2] = {0, 0};
  if ((e = hipMemcpyAsync(&last[0], *sptr + (ns - 1), sizeof(int64_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipMemcpyAsync(&last[1], size + (ns - 1), sizeof(int64_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return e;
  *slots = last[0] + last[1];
  if (*slots > max_slots) return hipSuccess;  // the caller rejects the plan; nothing more is built
  if ((e = hipMemcpyAsync(*sptr + ns, slots, sizeof(int64_t), hipMemcpyHostToDevice, s)) != hipSuccess) return e;
  *scol = static_cast<int32_t *>(alloc(sizeof(int32_t) * (size_t)std::max<int64_t>(1, *slots)));
  *sval = static_cast<float *>(alloc(sizeof(float) * (size_t)std::max<int64_t>(1, *slots)));
  if (!*scol || !*sval) return hipErrorOutOfMemory;
  if (*slots > 0) {
    hipLaunchKernelGGL(k_fill_i32, dim3(grid_for(*slots)), dim3(256), 0, s, *scol, *slots, -1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = hipMemsetAsync(*sval, 0, sizeof(float) * (size_t)*slots, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_sell_fill, dim3(grid_for(m)), dim3(256), 0, s, rowptr, colidx, vals, *perm, *sptr, m, C,
                       *scol, *sval);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipStreamSynchronize(s);  // the scratch arrays are freed on return
}

hipError_t dev_tag_cold(const int32_t *colidx, int64_t nnz, int32_t k, int64_t budget_rows, int32_t *tagged,
                        int64_t *hot_cols, int64_t *hot_nnz, hipStream_t s) {
  *hot_cols = *hot_nnz = 0;
  hipError_t e;
  Scratch sc(s);
  const size_t kk = (size_t)std::max(1, k);
  if ((e = hipMalloc(&sc.p[0], 4 * kk)) != hipSuccess) return e;
  int32_t *deg = static_cast<int32_t *>(sc.p[0]);
  if ((e = hipMemsetAsync(deg, 0, 4 * kk, s)) != hipSuccess) return e;
  if (nnz > 0) {
    hipLaunchKernelGGL(k_col_degree, dim3(grid_for(nnz)), dim3(256), 0, s, colidx, nnz, deg);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  std::vector<int32_t> h(kk);
  if ((e = hipMemcpyAsync(h.data(), deg, 4 * kk, hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return e;
  h.resize((size_t)k);
  // smallest D >= 2 with #{deg >= D} <= budget_rows (the host conversion's rule)
  int32_t dmax = 0;
  for (int32_t d : h) dmax = std::max(dmax, d);
  std::vector<int64_t> hist((size_t)dmax + 2, 0);
  for (int32_t d : h) hist[d]++;
  int64_t above = 0;
  int32_t D = dmax + 1;
  for (int32_t d = dmax; d >= 2; --d) {
    if (above + hist[d] > budget_rows) break;
    above += hist[d];
    D = d;
  }
  int64_t hn = 0;
  for (int32_t d : h)
    if (d >= D) hn += d;
  *hot_cols = above;
  *hot_nnz = hn;
  if (nnz > 0) {
    hipLaunchKernelGGL(k_tag_cold, dim3(grid_for(nnz)), dim3(256), 0, s, colidx, nnz, deg, D, tagged);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipStreamSynchronize(s);
}

uint64_t pattern_hash_host(const int32_t *rowptr, const int32_t *colidx, int32_t m, int64_t nnz) {
  uint64_t h = 0;
  for (int64_t i = 0; i <= m; ++i) h += mix64(kPatternSalt[0] ^ ((uint64_t)i << 32 | (uint32_t)rowptr[i]));
  for (int64_t p = 0; p < nnz; ++p) h += mix64(kPatternSalt[1] ^ ((uint64_t)p << 32 | (uint32_t)colidx[p]));
  return h;
}

hipError_t dev_pattern_hash(const int32_t *rowptr, const int32_t *colidx, int32_t m, int64_t nnz, hipStream_t s,
                            uint64_t *out) {
  Scratch sc(s);
  hipError_t e;
  if ((e = hipMalloc(&sc.p[0], sizeof(unsigned long long))) != hipSuccess) return e;
  unsigned long long *sum = static_cast<unsigned long long *>(sc.p[0]);
  if ((e = hipMemsetAsync(sum, 0, sizeof(unsigned long long), s)) != hipSuccess) return e;
  const int64_t lens[2] = {(int64_t)m + 1, nnz};
  const int32_t *arrs[2] = {rowptr, colidx};
  for (int t = 0; t < 2; ++t) {
    if (lens[t] == 0) continue;
    const uint32_t grid = (uint32_t)std::min<int64_t>(2048, (lens[t] + 255) / 256);
    hipLaunchKernelGGL(k_pattern_hash, dim3(grid), dim3(256), 0, s, arrs[t], lens[t], kPatternSalt[t], sum);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  unsigned long long h = 0;
  if ((e = hipMemcpyAsync(&h, sum, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return e;
  *out = (uint64_t)h;
  return hipSuccess;
}

hipError_t dev_transpose(const int32_t *rowptr, const int32_t *colidx, const float *vals, int32_t m, int32_t k,
                         int64_t nnz, int32_t *t_rowptr, int32_t *t_colidx, float *t_vals, hipStream_t s) {
  hipError_t e;
  if (nnz > 0) {
    Scratch sc(s);  // sorted keys, positions, sorted positions, sort temporary
    const size_t bytes = sizeof(int32_t) * (size_t)nnz;
    for (int t = 0; t < 3; ++t)
      if ((e = hipMalloc(&sc.p[t], bytes)) != hipSuccess) return e;
    uint32_t *keys_out = static_cast<uint32_t *>(sc.p[0]);
    int32_t *pos = static_cast<int32_t *>(sc.p[1]), *perm = static_cast<int32_t *>(sc.p[2]);
    hipLaunchKernelGGL(k_iota, dim3(grid_for(nnz)), dim3(256), 0, s, pos, nnz);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    int end_bit = 1;  // columns are in [0, k): sort on the bits that can be set
    while (end_bit < 31 && ((int64_t)1 << end_bit) < (int64_t)k) ++end_bit;
    const uint32_t *keys_in = reinterpret_cast<const uint32_t *>(colidx);  // valid columns are non-negative
    size_t tmp = 0;
    if ((e = hipcub::DeviceRadixSort::SortPairs(nullptr, tmp, keys_in, keys_out, pos, perm, (int)nnz, 0, end_bit,
                                                 s)) != hipSuccess)
      return e;
    if ((e = hipMalloc(&sc.p[3], std::max<size_t>(tmp, 1))) != hipSuccess) return e;
    if ((e = hipcub::DeviceRadixSort::SortPairs(sc.p[3], tmp, keys_in, keys_out, pos, perm, (int)nnz, 0, end_bit,
                                                 s)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(k_transpose_rowptr, dim3(grid_for((int64_t)k + 1)), dim3(256), 0, s, keys_out, nnz, k,
                       t_rowptr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_transpose_fill, dim3(grid_for(nnz)), dim3(256), 0, s, rowptr, m, vals, perm, nnz, t_colidx,
                       t_vals);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return hipStreamSynchronize(s);  // the scratch arrays are freed on return
  }
  if ((e = hipMemsetAsync(t_rowptr, 0, sizeof(int32_t) * ((size_t)k + 1), s)) != hipSuccess) return e;
  return hipStreamSynchronize(s);
}

}  // namespace sd
