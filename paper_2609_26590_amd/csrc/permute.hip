// gtr_scan_permute: token rows between spatial and scan order (paper Sec. 3.1,
// "Directional scanning"). A pure copy of whole rows, so bit-exact.
//
// One thread moves one vector unit (16, 8, 4, 2 or 1 bytes, the widest that
// divides the row and both base addresses). Consecutive threads take
// consecutive units of a row, so every row is read and written as one
// contiguous run; the permutation only decides which row goes where.
#include <hip/hip_runtime.h>

#include "gtr.h"
#include "gtr_device.h"
#include "gtr_internal.h"

namespace gtr {

template <typename U>
__global__ void __launch_bounds__(256) permute_kernel(const U* __restrict__ src, U* __restrict__ dst,
                                                      int64_t rows_total, int64_t units_per_row, int32_t H,
                                                      int32_t W, int dir, int inverse) {
  const int64_t L = (int64_t)H * W;
  const int64_t n = rows_total * units_per_row;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = i / units_per_row;
    const int64_t u = i - row * units_per_row;
    const int64_t o = row / L;
    const int64_t s = row - o * L;
    const int64_t sp = scan_to_spatial(s, H, W, dir);
    const int64_t from = inverse ? s : sp;
    const int64_t to = inverse ? sp : s;
    dst[(o * L + to) * units_per_row + u] = src[(o * L + from) * units_per_row + u];
  }
}

}  // namespace gtr

using namespace gtr;

extern "C" gtr_status gtr_scan_permute(const void* src, void* dst, int64_t outer, int32_t H, int32_t W,
                                       int64_t row_elems, gtr_dtype dt, gtr_scan dir, int32_t inverse,
                                       hipStream_t stream) {
  if (!src || !dst) return GTR_ERR_NULL;
  if (outer <= 0 || H <= 0 || W <= 0 || row_elems <= 0) return GTR_ERR_SHAPE;
  const size_t es = dtype_size(dt);
  if (es == 0) return GTR_ERR_UNSUPPORTED;
  if (dir < GTR_SCAN_ROW || dir > GTR_SCAN_COL_REV) return GTR_ERR_UNSUPPORTED;
  if (inverse != 0 && inverse != 1) return GTR_ERR_UNSUPPORTED;
  int64_t L, rows, row_bytes, total;
  if (__builtin_mul_overflow((int64_t)H, (int64_t)W, &L) || __builtin_mul_overflow(outer, L, &rows) ||
      __builtin_mul_overflow(row_elems, (int64_t)es, &row_bytes) || __builtin_mul_overflow(rows, row_bytes, &total))
    return GTR_ERR_SHAPE;
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (s0 < d0 + (uintptr_t)total && d0 < s0 + (uintptr_t)total) return GTR_ERR_ALIAS;

  const uintptr_t mix = s0 | d0 | (uintptr_t)row_bytes;
  int vec = 16;
  while (vec > 1 && (mix & (uintptr_t)(vec - 1))) vec >>= 1;
  const int64_t upr = row_bytes / vec;
  const int64_t n = rows * upr;
  const int64_t want = (n + 255) / 256;
  const unsigned blocks = (unsigned)(want < 1024 ? want : 1024);
  switch (vec) {
    case 16:
      hipLaunchKernelGGL(permute_kernel<uint4>, dim3(blocks), dim3(256), 0, stream, static_cast<const uint4*>(src),
                         static_cast<uint4*>(dst), rows, upr, H, W, (int)dir, (int)inverse);
      break;
    case 8:
      hipLaunchKernelGGL(permute_kernel<uint2>, dim3(blocks), dim3(256), 0, stream, static_cast<const uint2*>(src),
                         static_cast<uint2*>(dst), rows, upr, H, W, (int)dir, (int)inverse);
      break;
    case 4:
      hipLaunchKernelGGL(permute_kernel<uint32_t>, dim3(blocks), dim3(256), 0, stream,
                         static_cast<const uint32_t*>(src), static_cast<uint32_t*>(dst), rows, upr, H, W, (int)dir,
                         (int)inverse);
      break;
    case 2:
      hipLaunchKernelGGL(permute_kernel<uint16_t>, dim3(blocks), dim3(256), 0, stream,
                         static_cast<const uint16_t*>(src), static_cast<uint16_t*>(dst), rows, upr, H, W, (int)dir,
                         (int)inverse);
      break;
    default:
      hipLaunchKernelGGL(permute_kernel<uint8_t>, dim3(blocks), dim3(256), 0, stream,
                         static_cast<const uint8_t*>(src), static_cast<uint8_t*>(dst), rows, upr, H, W, (int)dir,
                         (int)inverse);
      break;
  }
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}
