// sd_spmm_merge_noalloc: the merge-path SpMM of a CSR already in device
// memory, with no plan and no allocation.
//
// sd_spmm on a CSR_MERGE plan keeps the split coordinates and the pieces'
// carry and head partials in device memory the plan allocated.  This variant
// keeps them in `scratch`, a fixed device array of kNoAllocScratchBytes that
// the code object itself provides (each device holds its own copy until the
// process ends), and computes the split coordinates on the device on every
// call, so it calls no allocator at all.  The kernels are the plan path's:
// k_merge_coords, k_csr_merge and k_merge_fixup, given the scratch's device
// address as they are given the plan's buffers.
//
// In host code `scratch` names a host-side stand-in, not device memory; only
// the address hipGetSymbolAddress returns for the current device is passed to
// kernels.  That lookup runs once per device, on the first call made with that
// device current.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <mutex>

#include "kernels.h"
#include "sd_internal.h"

static constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;

struct DeviceScratch {
  std::once_flag once;
  hipError_t status = hipSuccess;
  unsigned char *ptr = nullptr;  // device address of this device's scratch
  int32_t cu_count = 0;
};
DeviceScratch g_scratch[kMaxDevices];

// Bytes one call needs for U pieces of width n: the (U + 1) split
// coordinates, 2 U carry and head rows, and 2 U n carry and head partials,
// each region 256-byte aligned.
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
size_t scratch_bytes(int64_t U, int64_t n) {
  return align256(8 * (size_t)(U + 1)) + align256(8 * (size_t)U) + 8 * (size_t)U * (size_t)n;
}

}  // namespace

extern "C" int sd_spmm_merge_noalloc(const sd_csr_t *A, int32_t n, int32_t units, const float *B, float *C,
                                     void *stream) {
  if (!A || n < 1 || units < 0 || A->m < 0 || A->k < 0 || A->nnz < 0) return SD_ERR_INVALID_VALUE;
  if (A->nnz > INT32_MAX) return SD_ERR_OVERFLOW;
  if (A->m == 0) return SD_OK;  // empty output
  if (!A->rowptr || !C || (A->nnz > 0 && (!A->colidx || !A->values)) || (!B && A->k > 0))
    return SD_ERR_INVALID_VALUE;
  {  // B (k x n) and C (m x n) must not overlap
    const uintptr_t b0 = reinterpret_cast<uintptr_t>(B), c0 = reinterpret_cast<uintptr_t>(C);
    const uintptr_t b1 = b0 + (uintptr_t)A->k * (uintptr_t)n * sizeof(float);
    const uintptr_t c1 = c0 + (uintptr_t)A->m * (uintptr_t)n * sizeof(float);
    if (A->k > 0 && b0 < c1 && c0 < b1) return SD_ERR_INVALID_VALUE;
  }
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0) return SD_ERR_NO_DEVICE;
  if (dev >= kMaxDevices) return SD_ERR_UNSUPPORTED;
  DeviceScratch &ds = g_scratch[dev];
  std::call_once(ds.once, [&] {
    ds.status = hipGetSymbolAddress(reinterpret_cast<void **>(&ds.ptr), HIP_SYMBOL(scratch));
    if (ds.status == hipSuccess) ds.status = hipDeviceGetAttribute(&ds.cu_count, hipDeviceAttributeMultiprocessorCount, dev);
  });
  if (ds.status != hipSuccess || !ds.ptr) return sd::report_hip_error(ds.status != hipSuccess ? ds.status
                                                                                             : hipErrorInvalidSymbol);

  const int32_t vec4 = (n % 4 == 0) && ((reinterpret_cast<uintptr_t>(B) | reinterpret_cast<uintptr_t>(C)) % 16 == 0);
  const sd::Geometry geo = sd::geometry_for(n, vec4, 0);
  const int64_t total = (int64_t)A->m + A->nnz;
  int64_t U = units;
  if (U == 0) {
    // the plan path's default: lane groups for about 32 waves per compute
    // unit and at least 64 path steps per piece, then as many pieces as fit
    const int64_t groups = (int64_t)std::max(1, ds.cu_count) * 32 * (64 / geo.G);
    const int64_t per_unit = std::max<int64_t>(64, (total + groups - 1) / groups);
    U = (total + per_unit - 1) / per_unit;
    while (U > 1 && scratch_bytes(U, n) > kNoAllocScratchBytes) U = (U + 1) / 2;
  }
  if (U < 1 || scratch_bytes(U, n) > kNoAllocScratchBytes) return SD_ERR_UNSUPPORTED;
  const int64_t L = std::max<int64_t>(1, (total + U - 1) / U);

  int32_t *coords = reinterpret_cast<int32_t *>(ds.ptr);
  int32_t *rows = reinterpret_cast<int32_t *>(ds.ptr + align256(8 * (size_t)(U + 1)));
  float *part = reinterpret_cast<float *>(ds.ptr + align256(8 * (size_t)(U + 1)) + align256(8 * (size_t)U));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  // every coordinate, row slot and partial the fix-up reads is written by
  // this call's kernels first, so nothing in the scratch needs clearing
  e = sd::dev_merge_coords(A->rowptr, A->m, A->nnz, (int32_t)U, L, coords, s);
  if (e != hipSuccess) return sd::report_hip_error(e);
  sd::DenseIO io;
  io.B = B;
  io.C = C;
  io.n = n;
  io.vec4 = vec4;
  io.policy = 0;
  io.col_tile = 0;
  io.order = 0;  // the merge plan's default: the hardware's round-robin
  const sd::CsrOperand Aop{A->rowptr, A->colidx, A->values, A->m, A->k};
  e = sd::launch_csr_merge(Aop, coords, (int32_t)U, rows, part, io, s);
  if (e != hipSuccess) return sd::report_hip_error(e);
  return SD_OK;
}
