// Finalize step of the reverse walk.  Key j receives gradient only from
// query rows r >= j, and the backward walk visits the chunks N-1, ..., 0
// (Sec. 5.2), so once chunk i's backward has run no later call touches the
// dK/dV rows [c_i, c_{i+1}) again: those rows are final and can be rounded
// from the fp32 accumulators to the problem's element type.
//
// HBM-bound: per element 8 bytes read (dK, dV fp32) and 4 written (bf16).
// One thread per 8 consecutive elements of the [B, rows, W] span, W = Hkv*D
// (a multiple of 64), 16-byte loads of the accumulators and 16-byte bf16
// stores.
#include "sppo_kernels.h"
#include "tile_common.h"

namespace sppo {
namespace {

__global__ __launch_bounds__(256) void finalize_bf16_kernel(const float* __restrict__ dk, const float* __restrict__ dv,
                                                            uint16_t* __restrict__ ok, uint16_t* __restrict__ ov,
                                                            int64_t row0, int64_t rows, int64_t S, int64_t W,
                                                            int64_t n8) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= n8) return;
  const int64_t e = t * 8, per_b = rows * W;
  const int64_t b = e / per_b;
  const int64_t off = (b * S + row0) * W + (e - b * per_b);
  const f32x4 k0 = *reinterpret_cast<const f32x4*>(dk + off), k1 = *reinterpret_cast<const f32x4*>(dk + off + 4);
  const f32x4 v0 = *reinterpret_cast<const f32x4*>(dv + off), v1 = *reinterpret_cast<const f32x4*>(dv + off + 4);
  *reinterpret_cast<bf16x8*>(ok + off) = pack_bf16x8(k0[0], k0[1], k0[2], k0[3], k1[0], k1[1], k1[2], k1[3]);
  *reinterpret_cast<bf16x8*>(ov + off) = pack_bf16x8(v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]);
}

// fp32 problems: the final rows are copied as they are.
__global__ __launch_bounds__(256) void finalize_f32_kernel(const float* __restrict__ dk, const float* __restrict__ dv,
                                                           float* __restrict__ ok, float* __restrict__ ov,
                                                           int64_t row0, int64_t rows, int64_t S, int64_t W,
                                                           int64_t n8) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= n8) return;
  const int64_t e = t * 8, per_b = rows * W;
  const int64_t b = e / per_b;
  const int64_t off = (b * S + row0) * W + (e - b * per_b);
#pragma unroll
  for (int h = 0; h < 8; h += 4) {
    *reinterpret_cast<f32x4*>(ok + off + h) = *reinterpret_cast<const f32x4*>(dk + off + h);
    *reinterpret_cast<f32x4*>(ov + off + h) = *reinterpret_cast<const f32x4*>(dv + off + h);
  }
}

}  // namespace

hipError_t launch_finalize(const FinalizeArgs& a, hipStream_t stream) {
  if (a.B <= 0 || a.rows <= 0 || a.W <= 0 || a.W % 8 || a.row0 < 0 || a.row0 + a.rows > a.S)
    return hipErrorInvalidValue;
  const int64_t n8 = a.B * a.rows * a.W / 8;
  const dim3 grid((unsigned)((n8 + 255) / 256)), block(256);
  if (a.bf16) {
    hipLaunchKernelGGL(finalize_bf16_kernel, grid, block, 0, stream, a.dk, a.dv, static_cast<uint16_t*>(a.out_k),
                       static_cast<uint16_t*>(a.out_v), a.row0, a.rows, a.S, a.W, n8);
  } else {
    hipLaunchKernelGGL(finalize_f32_kernel, grid, block, 0, stream, a.dk, a.dv, static_cast<float*>(a.out_k),
                       static_cast<float*>(a.out_v), a.row0, a.rows, a.S, a.W, n8);
  }
  return hipGetLastError();
}

}  // namespace sppo
