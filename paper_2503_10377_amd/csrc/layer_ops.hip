// Row-wise and elementwise kernels of a full transformer layer chunk (the
// non-attention, non-GEMM steps): LayerNorm forward and backward, the GELU
// recomputation, the weight transpose, and the packing of the chunk's
// [dQ | dK | dV] rows for the QKV projection's backward.  bf16 activations,
// fp32 statistics and parameter gradients.
#include "sppo_kernels.h"
#include "tile_common.h"

namespace sppo {
namespace {

constexpr int kLnThreads = 256;
constexpr int kLnMaxPer = 4;  // 16-byte groups per thread: H <= 256 * 8 * 4 = 8192

__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();  // red may still be read by a previous reduction
  if (lane == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

__device__ __forceinline__ void unpack8(const u32x4& x, float (&f)[8]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f[2 * e] = __uint_as_float(x[e] << 16);
    f[2 * e + 1] = __uint_as_float(x[e] & 0xffff0000u);
  }
}
__device__ __forceinline__ u32x4 pack8(const float (&f)[8]) {
  const bf16x8 b = pack_bf16x8(f[0], f[1], f[2], f[3], f[4], f[5], f[6], f[7]);
  return __builtin_bit_cast(u32x4, b);
}

// y = (x - mean) * rstd * gamma + beta per row, with biased variance; one
// workgroup per row.  mean and rstd are kept for the backward.
__global__ __launch_bounds__(kLnThreads) void ln_fwd_kernel(LnArgs a) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const uint16_t* x = a.x + row * a.ldx;
  const int H = a.H, tid = threadIdx.x;
  float v[kLnMaxPer][8];
  float s = 0.f;
#pragma unroll
  for (int p = 0; p < kLnMaxPer; ++p) {
    const int c = 8 * (tid + kLnThreads * p);
    if (c < H) {
      unpack8(ld_global16(x + c), v[p]);
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[p][e];
    }
  }
  const float mean = block_sum(s, red) / H;
  float q = 0.f;
#pragma unroll
  for (int p = 0; p < kLnMaxPer; ++p) {
    const int c = 8 * (tid + kLnThreads * p);
    if (c < H) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = v[p][e] - mean;
        q += d * d;
      }
    }
  }
  const float rstd = 1.f / sqrtf(block_sum(q, red) / H + a.eps);
  uint16_t* y = a.y + row * a.ldy;
#pragma unroll
  for (int p = 0; p < kLnMaxPer; ++p) {
    const int c = 8 * (tid + kLnThreads * p);
    if (c < H) {
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (v[p][e] - mean) * rstd * a.gamma[c + e] + a.beta[c + e];
      *reinterpret_cast<u32x4*>(y + c) = pack8(o);
    }
  }
  if (tid == 0 && a.mean) {
    a.mean[row] = mean;
    a.rstd[row] = rstd;
  }
}

// N block-wide sums at once (four waves): one shuffle tree per value, one
// round through LDS.
template <int N>
__device__ __forceinline__ void block_sum_n(float (&v)[N], float* red) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v[i] += __shfl_xor(v[i], off);
  }
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();  // red may still be read by a previous reduction
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < N; ++i) red[w * N + i] = v[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = red[i] + red[N + i] + red[2 * N + i] + red[3 * N + i];
}

// Backward of y = xhat * gamma + beta, xhat = (x - mean) * rstd, per row:
//   dx = dres + rstd * (g - mean_j(g) - xhat * mean_j(g * xhat)),  g = dy * gamma
// (dres: the gradient that reaches x around the LayerNorm, the residual
// branch).  Workgroup b handles rows [b R, b R + R), two rows at a time (one
// reduction for both), and writes its partial sums of dy * xhat and dy over
// those rows (the gamma and beta gradients) to part[b]; ln_reduce adds the
// partials.  PER 16-byte column groups per thread (H <= 2048 PER).
template <int PER>
__global__ __launch_bounds__(kLnThreads) void ln_bwd_kernel(LnArgs a) {
  __shared__ float red[4 * 4];
  const int H = a.H, tid = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * a.rows_per_block;
  const int64_t r1 = r0 + a.rows_per_block < a.rows ? r0 + a.rows_per_block : a.rows;
  float pg[PER][8], pb[PER][8];
#pragma unroll
  for (int p = 0; p < PER; ++p) {
#pragma unroll
    for (int e = 0; e < 8; ++e) pg[p][e] = pb[p][e] = 0.f;
  }
  for (int64_t row = r0; row < r1; row += 2) {
    const bool two = row + 1 < r1;
    float xh[2][PER][8], gg[2][PER][8];
    float sums[4] = {0.f, 0.f, 0.f, 0.f};
    float mean[2], rstd[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t rr = j == 0 || two ? row + j : row;  // a lone last row is read twice, used once
      mean[j] = a.mean[rr];
      rstd[j] = a.rstd[rr];
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        const int c = 8 * (tid + kLnThreads * p);
        if (c < H) {
          float xv[8], dv[8];
          unpack8(ld_global16(a.x + rr * a.ldx + c), xv);
          unpack8(ld_global16(a.dy + rr * a.lddy + c), dv);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            xh[j][p][e] = (xv[e] - mean[j]) * rstd[j];
            gg[j][p][e] = dv[e] * a.gamma[c + e];
            sums[2 * j] += gg[j][p][e];
            sums[2 * j + 1] += gg[j][p][e] * xh[j][p][e];
            if (j == 0 || two) {
              pg[p][e] += dv[e] * xh[j][p][e];
              pb[p][e] += dv[e];
            }
          }
        }
      }
    }
    block_sum_n<4>(sums, red);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (j == 1 && !two) break;
      const int64_t rr = row + j;
      const float m1 = sums[2 * j] / H, m2 = sums[2 * j + 1] / H;
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        const int c = 8 * (tid + kLnThreads * p);
        if (c < H) {
          float rv[8], o[8];
          unpack8(ld_global16(a.dres + rr * a.lddres + c), rv);
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = rv[e] + rstd[j] * (gg[j][p][e] - m1 - xh[j][p][e] * m2);
          *reinterpret_cast<u32x4*>(a.y + rr * a.ldy + c) = pack8(o);
        }
      }
    }
  }
  float* part = a.part + (int64_t)blockIdx.x * 2 * H;
#pragma unroll
  for (int p = 0; p < PER; ++p) {
    const int c = 8 * (tid + kLnThreads * p);
    if (c < H) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        part[c + e] = pg[p][e];
        part[H + c + e] = pb[p][e];
      }
    }
  }
}

// dgamma[c] (+)= sum_b part[b][c], dbeta[c] (+)= sum_b part[b][H + c].  A
// workgroup covers 32 columns of the 2H partial row with 8 row groups: group
// t sums the blocks b = t, t + 8, ... in order, then the eight group sums
// are added in group order (a fixed order: the result is deterministic).
constexpr int kRedCols = 32, kRedGroups = 8;
__global__ __launch_bounds__(kRedCols * kRedGroups) void ln_reduce_kernel(LnArgs a) {
  __shared__ float red[kRedGroups][kRedCols];
  const int lc = threadIdx.x % kRedCols, t = threadIdx.x / kRedCols;
  const int c = blockIdx.x * kRedCols + lc;  // column of the [2H] partial row
  const int W = 2 * a.H;
  float s = 0.f;
  if (c < W) {
    for (int b = t; b < a.nblocks; b += kRedGroups) s += a.part[(int64_t)b * W + c];
  }
  red[t][lc] = s;
  __syncthreads();
  if (t == 0 && c < W) {
    float tot = red[0][lc];
#pragma unroll
    for (int u = 1; u < kRedGroups; ++u) tot += red[u][lc];
    float* dst = c < a.H ? a.dgamma + c : a.dbeta + (c - a.H);
    if (a.accumulate) *dst += tot;
    else *dst = tot;
  }
}

// y = gelu(x) elementwise over n bf16 values (n % 8 == 0).
__global__ __launch_bounds__(256) void gelu_kernel(const uint16_t* x, uint16_t* y, int64_t n) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (i >= n) return;
  float v[8];
  unpack8(ld_global16(x + i), v);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = gelu_tanh(v[e]);
  *reinterpret_cast<u32x4*>(y + i) = pack8(v);
}

// out[c][r] = in[r][c] for a [R, C] bf16 matrix, 64 x 64 tiles through LDS.
__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* in, uint16_t* out, int64_t R, int64_t C) {
  __shared__ uint16_t t[64][66];
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int y = ty; y < 64; y += 4) {
    const int64_t r = r0 + y, c = c0 + tx;
    t[y][tx] = (r < R && c < C) ? in[r * C + c] : 0;
  }
  __syncthreads();
  for (int y = ty; y < 64; y += 4) {
    const int64_t c = c0 + y, r = r0 + tx;
    if (c < C && r < R) out[c * R + r] = t[tx][y];
  }
}

// Row t of dqkv = [dQ_i[t] | bf16(dK[c + t]) | bf16(dV[c + t])] for the
// chunk's rows (B = 1): dQ_i is [s, Hq D] bf16, dK/dV [S, Hkv D] fp32.
__global__ __launch_bounds__(256) void pack_dqkv_kernel(PackArgs a) {
  const int64_t t = blockIdx.x;
  const int wq = a.wq, wkv = a.wkv;
  uint16_t* out = a.out + t * (int64_t)(wq + 2 * wkv);
  for (int c = threadIdx.x * 8; c < wq; c += 256 * 8)
    *reinterpret_cast<u32x4*>(out + c) = ld_global16(a.dq + t * (int64_t)wq + c);
  const float* dk = a.dk + (a.c + t) * (int64_t)wkv;
  const float* dv = a.dv + (a.c + t) * (int64_t)wkv;
  for (int c = threadIdx.x * 8; c < wkv; c += 256 * 8) {
    float f[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = dk[c + e];
    *reinterpret_cast<u32x4*>(out + wq + c) = pack8(f);
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = dv[c + e];
    *reinterpret_cast<u32x4*>(out + wq + wkv + c) = pack8(f);
  }
}

}  // namespace

hipError_t launch_ln_fwd(const LnArgs& a, hipStream_t stream) {
  if (a.rows <= 0 || a.H <= 0 || a.H % 8 || a.H > kLnThreads * 8 * kLnMaxPer) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ln_fwd_kernel, dim3((unsigned)a.rows), dim3(kLnThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_ln_bwd(const LnArgs& a, hipStream_t stream) {
  if (a.rows <= 0 || a.H <= 0 || a.H % 8 || a.H > kLnThreads * 8 * kLnMaxPer || a.rows_per_block <= 0)
    return hipErrorInvalidValue;
  LnArgs b = a;
  b.nblocks = (int)((a.rows + a.rows_per_block - 1) / a.rows_per_block);
  const dim3 grid((unsigned)b.nblocks), block(kLnThreads);
  switch ((a.H + 2047) / 2048) {
    case 1: hipLaunchKernelGGL(ln_bwd_kernel<1>, grid, block, 0, stream, b); break;
    case 2: hipLaunchKernelGGL(ln_bwd_kernel<2>, grid, block, 0, stream, b); break;
    case 3: hipLaunchKernelGGL(ln_bwd_kernel<3>, grid, block, 0, stream, b); break;
    default: hipLaunchKernelGGL(ln_bwd_kernel<4>, grid, block, 0, stream, b); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(ln_reduce_kernel, dim3((unsigned)((2 * a.H + kRedCols - 1) / kRedCols)),
                     dim3(kRedCols * kRedGroups), 0, stream, b);
  return hipGetLastError();
}

hipError_t launch_gelu(const uint16_t* x, uint16_t* y, int64_t n, hipStream_t stream) {
  if (n <= 0 || n % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gelu_kernel, dim3((unsigned)((n / 8 + 255) / 256)), dim3(256), 0, stream, x, y, n);
  return hipGetLastError();
}

hipError_t launch_transpose(const uint16_t* in, uint16_t* out, int64_t R, int64_t C, hipStream_t stream) {
  if (R <= 0 || C <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(transpose_kernel, dim3((unsigned)((C + 63) / 64), (unsigned)((R + 63) / 64)), dim3(256), 0,
                     stream, in, out, R, C);
  return hipGetLastError();
}

hipError_t launch_pack_dqkv(const PackArgs& a, hipStream_t stream) {
  if (a.rows <= 0 || a.wq % 8 || a.wkv % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_dqkv_kernel, dim3((unsigned)a.rows), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sppo
