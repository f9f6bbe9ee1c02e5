// Device-to-device row copies for the keep buffers of a row-prefix offload
// (the rows of a chunk that stay on the device while its region is reused).
// A kernel on the caller's stream rather than a device-to-device
// hipMemcpy: the runtime may serve the latter with a copy engine or queue it
// where other streams' copies are waiting, which was measured to add about
// 80 ms to a 128K-token step once several offloading contexts (and their
// copy streams) were alive; a kernel keeps the move in plain stream order.
//
// HBM-bound: `height` rows of `width` bytes, read and written once.  Rows
// move as 16-byte vectors when every address and size allows it, else as
// 4-byte words (widths and pitches are multiples of 4 bytes).
#include "sppo_kernels.h"
#include "tile_common.h"

namespace sppo {
namespace {

template <typename V>
__global__ __launch_bounds__(256) void copy_rows_kernel(char* __restrict__ dst, int64_t dpitch,
                                                        const char* __restrict__ src, int64_t spitch,
                                                        int64_t per_row, int64_t total) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += stride) {
    const int64_t row = t / per_row, col = (t - row * per_row) * (int64_t)sizeof(V);
    *reinterpret_cast<V*>(dst + row * dpitch + col) = *reinterpret_cast<const V*>(src + row * spitch + col);
  }
}

}  // namespace

hipError_t launch_copy_rows(void* dst, size_t dpitch, const void* src, size_t spitch, size_t width, size_t height,
                            hipStream_t stream) {
  if (width == 0 || height == 0) return hipSuccess;
  if (width % 4 || dpitch % 4 || spitch % 4 || (reinterpret_cast<uintptr_t>(dst) & 3) ||
      (reinterpret_cast<uintptr_t>(src) & 3))
    return hipErrorInvalidValue;
  const bool v16 = width % 16 == 0 && dpitch % 16 == 0 && spitch % 16 == 0 &&
                   (reinterpret_cast<uintptr_t>(dst) & 15) == 0 && (reinterpret_cast<uintptr_t>(src) & 15) == 0;
  const int64_t per_row = (int64_t)(width / (v16 ? 16 : 4));
  const int64_t total = per_row * (int64_t)height;
  const int64_t blocks = (total + 255) / 256;
  const dim3 grid((unsigned)(blocks < 4096 ? blocks : 4096)), block(256);
  char* d = static_cast<char*>(dst);
  const char* s = static_cast<const char*>(src);
  if (v16) {
    hipLaunchKernelGGL(copy_rows_kernel<u32x4>, grid, block, 0, stream, d, (int64_t)dpitch, s, (int64_t)spitch,
                       per_row, total);
  } else {
    hipLaunchKernelGGL(copy_rows_kernel<uint32_t>, grid, block, 0, stream, d, (int64_t)dpitch, s, (int64_t)spitch,
                       per_row, total);
  }
  return hipGetLastError();
}

}  // namespace sppo
