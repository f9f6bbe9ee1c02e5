// fp32 forward and backward of one chunk of sequence-chunked causal
// attention (the fp32 configuration is a parity case: small, latency-bound,
// and held to 1e-4 absolute error, so it uses plain fp32 FMA loops with
// correctly rounded expf/logf rather than bf16 matrix cores).
//
// Same chunk semantics as the bf16 path: queries [c0, c1) attend to keys
// [0, c1), causally masked on the diagonal (Sec. 5.1 of SPPO); backward
// accumulates dK/dV over the reverse chunk walk (Sec. 5.2).
//   fwd   : one thread per query row; K/V tiles of 64 keys in LDS.
//   pre   : Delta_r = <dO_r, O_r>.
//   dq    : one thread per query row.
//   dkdv  : one thread per key row; Q/dO tiles of 64 rows in LDS, every
//           query head of the key's GQA group.
#include "sppo_kernels.h"

namespace sppo {
namespace {

constexpr int kT = 64;  // threads per block = rows per tile

template <int D>
__global__ __launch_bounds__(kT) void fwd_f32_kernel(ChunkArgs a) {
  __shared__ float Ks[kT][D];
  __shared__ float Vs[kT][D];
  const int tid = threadIdx.x, h = blockIdx.y;
  const int64_t b = blockIdx.z;
  const int hk = h / (a.Hq / a.Hkv);
  const int64_t c0 = a.c0, c1 = a.c1, s = c1 - c0;
  const int64_t q0 = c0 + (int64_t)blockIdx.x * kT;
  const int64_t r = q0 + tid;
  const bool rvalid = r < c1;
  const int64_t kend = (q0 + kT < c1) ? q0 + kT : c1;
  const float* qrow = static_cast<const float*>(a.q) + ((b * s + (r - c0)) * a.Hq + h) * D;
  float q[D], o[D];
  for (int d = 0; d < D; ++d) {
    q[d] = rvalid ? qrow[d] : 0.f;
    o[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const float* kb = static_cast<const float*>(a.k) + (b * a.S * a.Hkv + hk) * D;
  const float* vb = static_cast<const float*>(a.v) + (b * a.S * a.Hkv + hk) * D;
  const int64_t stride = (int64_t)a.Hkv * D;
  for (int64_t k0 = 0; k0 < kend; k0 += kT) {
    __syncthreads();
    for (int x = tid; x < kT * D; x += kT) {
      const int jj = x / D, d = x % D;
      const int64_t j = k0 + jj;
      Ks[jj][d] = j < c1 ? kb[j * stride + d] : 0.f;
      Vs[jj][d] = j < c1 ? vb[j * stride + d] : 0.f;
    }
    __syncthreads();
    for (int jj = 0; jj < kT; ++jj) {
      const int64_t j = k0 + jj;
      if (j > r || j >= c1) break;
      float dot = 0.f;
      for (int d = 0; d < D; ++d) dot = fmaf(q[d], Ks[jj][d], dot);
      const float sv = dot * a.scale;
      if (sv > m) {
        const float corr = expf(m - sv);
        l *= corr;
        for (int d = 0; d < D; ++d) o[d] *= corr;
        m = sv;
      }
      const float p = expf(sv - m);
      l += p;
      for (int d = 0; d < D; ++d) o[d] = fmaf(p, Vs[jj][d], o[d]);
    }
  }
  if (rvalid) {
    float* orow = static_cast<float*>(a.o) + ((b * s + (r - c0)) * a.Hq + h) * D;
    const float inv = 1.f / l;
    for (int d = 0; d < D; ++d) orow[d] = o[d] * inv;
    a.lse[(b * a.Hq + h) * s + (r - c0)] = m + logf(l);
  }
}

template <int D>
__global__ __launch_bounds__(256) void pre_f32_kernel(ChunkArgs a) {
  const int64_t s = a.c1 - a.c0;
  const int64_t item = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (item >= a.B * s * a.Hq) return;
  const float* orow = static_cast<const float*>(a.o) + item * D;
  const float* drow = static_cast<const float*>(a.dout) + item * D;
  float acc = 0.f;
  for (int d = 0; d < D; ++d) acc = fmaf(orow[d], drow[d], acc);
  const int64_t h = item % a.Hq, rr = (item / a.Hq) % s, b = item / (a.Hq * s);
  a.delta[(b * a.Hq + h) * s + rr] = acc;
}

template <int D>
__global__ __launch_bounds__(kT) void dq_f32_kernel(ChunkArgs a) {
  __shared__ float Ks[kT][D];
  __shared__ float Vs[kT][D];
  const int tid = threadIdx.x, h = blockIdx.y;
  const int64_t b = blockIdx.z;
  const int hk = h / (a.Hq / a.Hkv);
  const int64_t c0 = a.c0, c1 = a.c1, s = c1 - c0;
  const int64_t q0 = c0 + (int64_t)blockIdx.x * kT;
  const int64_t r = q0 + tid;
  const bool rvalid = r < c1;
  const int64_t kend = (q0 + kT < c1) ? q0 + kT : c1;
  const int64_t off = ((b * s + (r - c0)) * a.Hq + h) * D;
  float q[D], dout[D], dq[D];
  for (int d = 0; d < D; ++d) {
    q[d] = rvalid ? static_cast<const float*>(a.q)[off + d] : 0.f;
    dout[d] = rvalid ? static_cast<const float*>(a.dout)[off + d] : 0.f;
    dq[d] = 0.f;
  }
  const float lse = rvalid ? a.lse[(b * a.Hq + h) * s + (r - c0)] : 0.f;
  const float delta = rvalid ? a.delta[(b * a.Hq + h) * s + (r - c0)] : 0.f;
  const float* kb = static_cast<const float*>(a.k) + (b * a.S * a.Hkv + hk) * D;
  const float* vb = static_cast<const float*>(a.v) + (b * a.S * a.Hkv + hk) * D;
  const int64_t stride = (int64_t)a.Hkv * D;
  for (int64_t k0 = 0; k0 < kend; k0 += kT) {
    __syncthreads();
    for (int x = tid; x < kT * D; x += kT) {
      const int jj = x / D, d = x % D;
      const int64_t j = k0 + jj;
      Ks[jj][d] = j < c1 ? kb[j * stride + d] : 0.f;
      Vs[jj][d] = j < c1 ? vb[j * stride + d] : 0.f;
    }
    __syncthreads();
    for (int jj = 0; jj < kT; ++jj) {
      const int64_t j = k0 + jj;
      if (j > r || j >= c1) break;
      float qk = 0.f, dp = 0.f;
      for (int d = 0; d < D; ++d) {
        qk = fmaf(q[d], Ks[jj][d], qk);
        dp = fmaf(dout[d], Vs[jj][d], dp);
      }
      const float p = expf(qk * a.scale - lse);
      const float ds = p * (dp - delta);
      for (int d = 0; d < D; ++d) dq[d] = fmaf(ds, Ks[jj][d], dq[d]);
    }
  }
  if (rvalid) {
    float* out = static_cast<float*>(a.dq) + off;
    for (int d = 0; d < D; ++d) out[d] = dq[d] * a.scale;
  }
}

template <int D>
__global__ __launch_bounds__(kT) void dkdv_f32_kernel(ChunkArgs a) {
  __shared__ float Qs[kT][D];
  __shared__ float Ds[kT][D];
  __shared__ float Ls[kT];
  __shared__ float Es[kT];
  const int tid = threadIdx.x, hk = blockIdx.y;
  const int64_t b = blockIdx.z;
  const int G = a.Hq / a.Hkv;
  const int64_t c0 = a.c0, c1 = a.c1, s = c1 - c0;
  const int64_t k0 = a.kv0 + (int64_t)blockIdx.x * kT;
  const int64_t j = k0 + tid;
  const bool jvalid = j < a.kv1;
  const int64_t kvoff = ((b * a.S + j) * a.Hkv + hk) * D;
  float kr[D], vr[D], dk[D], dv[D];
  for (int d = 0; d < D; ++d) {
    kr[d] = jvalid ? static_cast<const float*>(a.k)[kvoff + d] : 0.f;
    vr[d] = jvalid ? static_cast<const float*>(a.v)[kvoff + d] : 0.f;
    dk[d] = dv[d] = 0.f;
  }
  const int64_t qfirst = k0 > c0 ? k0 : c0;  // first query that sees a key here
  for (int hh = 0; hh < G; ++hh) {
    const int h = hk * G + hh;
    for (int64_t qa = qfirst; qa < c1; qa += kT) {
      __syncthreads();
      for (int x = tid; x < kT * D; x += kT) {
        const int ii = x / D, d = x % D;
        const int64_t rr = qa + ii - c0;
        const int64_t off = ((b * s + rr) * a.Hq + h) * D + d;
        const bool ok = qa + ii < c1;
        Qs[ii][d] = ok ? static_cast<const float*>(a.q)[off] : 0.f;
        Ds[ii][d] = ok ? static_cast<const float*>(a.dout)[off] : 0.f;
      }
      {
        const int64_t rr = qa + tid - c0;
        const bool ok = qa + tid < c1;
        Ls[tid] = ok ? a.lse[(b * a.Hq + h) * s + rr] : 0.f;
        Es[tid] = ok ? a.delta[(b * a.Hq + h) * s + rr] : 0.f;
      }
      __syncthreads();
      if (!jvalid) continue;
      for (int ii = 0; ii < kT; ++ii) {
        const int64_t qi = qa + ii;
        if (qi >= c1) break;
        if (qi < j) continue;
        float qk = 0.f, dp = 0.f;
        for (int d = 0; d < D; ++d) {
          qk = fmaf(Qs[ii][d], kr[d], qk);
          dp = fmaf(Ds[ii][d], vr[d], dp);
        }
        const float p = expf(qk * a.scale - Ls[ii]);
        const float ds = p * (dp - Es[ii]);
        for (int d = 0; d < D; ++d) {
          dv[d] = fmaf(p, Ds[ii][d], dv[d]);
          dk[d] = fmaf(ds, Qs[ii][d], dk[d]);
        }
      }
    }
  }
  if (jvalid) {
    float* dko = a.dk + kvoff;
    float* dvo = a.dv + kvoff;
    for (int d = 0; d < D; ++d) {
      const float kv = dk[d] * a.scale;
      if (a.accumulate) {
        dko[d] += kv;
        dvo[d] += dv[d];
      } else {
        dko[d] = kv;
        dvo[d] = dv[d];
      }
    }
  }
}

}  // namespace

hipError_t launch_fwd_f32(const ChunkArgs& a, hipStream_t stream) {
  const int64_t s = a.c1 - a.c0;
  dim3 grid((unsigned)((s + kT - 1) / kT), (unsigned)a.Hq, (unsigned)a.B);
  if (a.D == 64) {
    hipLaunchKernelGGL(fwd_f32_kernel<64>, grid, dim3(kT), 0, stream, a);
  } else if (a.D == 128) {
    hipLaunchKernelGGL(fwd_f32_kernel<128>, grid, dim3(kT), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_bwd_pre_f32(const ChunkArgs& a, hipStream_t stream) {
  const int64_t s = a.c1 - a.c0;
  dim3 grid((unsigned)((a.B * s * a.Hq + 255) / 256));
  if (a.D == 64) {
    hipLaunchKernelGGL(pre_f32_kernel<64>, grid, dim3(256), 0, stream, a);
  } else if (a.D == 128) {
    hipLaunchKernelGGL(pre_f32_kernel<128>, grid, dim3(256), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dkdv_f32(const ChunkArgs& a, hipStream_t stream) {
  if (a.kv0 < 0 || a.kv1 > a.c1 || a.kv0 >= a.kv1) return hipErrorInvalidValue;
  dim3 grid((unsigned)((a.kv1 - a.kv0 + kT - 1) / kT), (unsigned)a.Hkv, (unsigned)a.B);
  if (a.D == 64) {
    hipLaunchKernelGGL(dkdv_f32_kernel<64>, grid, dim3(kT), 0, stream, a);
  } else if (a.D == 128) {
    hipLaunchKernelGGL(dkdv_f32_kernel<128>, grid, dim3(kT), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dq_f32(const ChunkArgs& a, hipStream_t stream) {
  const int64_t s = a.c1 - a.c0;
  dim3 grid((unsigned)((s + kT - 1) / kT), (unsigned)a.Hq, (unsigned)a.B);
  if (a.D == 64) {
    hipLaunchKernelGGL(dq_f32_kernel<64>, grid, dim3(kT), 0, stream, a);
  } else if (a.D == 128) {
    hipLaunchKernelGGL(dq_f32_kernel<128>, grid, dim3(kT), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sppo
