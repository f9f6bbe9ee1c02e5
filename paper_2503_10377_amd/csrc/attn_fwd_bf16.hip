// Forward of one chunk of sequence-chunked causal attention, bf16 in / fp32
// accumulate, for gfx950 (MI355X).
//
// Chunk i's queries (rows [c0, c1)) attend to keys [0, c1): every earlier
// chunk fully, the diagonal block causally (two-level activation management,
// Sec. 5.1 of SPPO: K/V of all earlier subsequences stay resident on the GPU).
//
// One workgroup = 4 waves = 128 query rows of one head; each wave owns 32
// rows.  K/V tiles of 64 keys are staged through LDS in natural layout
// (swizzled, conflict-free), prefetched into registers one tile ahead; V^T
// operands come from ds_read_b64_tr_b16 transposed reads.  Per tile each wave
//   S^T[key][query] = K Q^T          (16x v_mfma_f32_32x32x16_bf16, D=128)
//   online softmax in base 2 (lane <-> query, so row statistics are in-lane
//   plus one exchange with lane^32)
//   O^T[d][query] += V^T P^T         (16 MFMAs, P^T fed from S^T's registers)
// The epilogue writes O = O^T / l (bf16) and LSE = ln2 * (m + log2 l).
#include "sppo_kernels.h"
#include "tile_common.h"

namespace sppo {
namespace {

constexpr int kFwdBR = 128;  // query rows per workgroup (4 waves x 32)
constexpr int kFwdBC = 64;   // keys per K/V tile
constexpr float kLazyMax = 8.f;  // log2 headroom before the running max moves

template <int D>
__global__ __launch_bounds__(256) void fwd_bf16_kernel(ChunkArgs a) {
  constexpr int BR = kFwdBR, BC = kFwdBC;
  using T = LdsTile<D>;
  constexpr int NK = D / 16;  // k-steps of K Q^T
  constexpr int ND = D / 32;  // 32-wide d blocks of O^T
  constexpr int CG = T::CG;
  constexpr int ITEMS = (BC / 4) * CG;
  constexpr int IPT = (ITEMS + 255) / 256;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[BC * T::P];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[BC * T::P];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g = lane >> 5;
  const int t = gridDim.x - 1 - blockIdx.x;  // longest (latest) query tiles first
  const int h = blockIdx.y;
  const int64_t b = blockIdx.z;
  const int hk = h / (a.Hq / a.Hkv);
  const int64_t c0 = a.c0, c1 = a.c1, s = c1 - c0;
  const int64_t q0 = c0 + (int64_t)t * BR;
  const int64_t r = q0 + w * 32 + l32;
  const bool rvalid = r < c1;
  const int64_t kend = (q0 + BR < c1) ? q0 + BR : c1;
  const int nkv = (int)((kend + BC - 1) / BC);
  const float C = a.scale * kLog2e;
  const auto nat = T::nat_base(lane);
  const auto trb = T::tr_base(lane);

  bf16x8 qf[NK];
  {
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) + ((b * s + (r - c0)) * a.Hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      qf[kk] = rvalid ? as_bf16x8(ld_global16(qrow + 16 * kk + 8 * g)) : bf16x8{};
    }
  }

  const int64_t kvstride = (int64_t)a.Hkv * D;
  const uint16_t* kbase = static_cast<const uint16_t*>(a.k) + (b * a.S * a.Hkv + hk) * D;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v) + (b * a.S * a.Hkv + hk) * D;

  f32x16 o[ND];
#pragma unroll
  for (int db = 0; db < ND; ++db) o[db] = f32x16{};
  float m = -INFINITY, lsum = 0.f;

  Block4x8 kreg[IPT], vreg[IPT];
  Block4x8Offsets boff[IPT];
#pragma unroll
  for (int u = 0; u < IPT; ++u) {
    const int c = tid + 256 * u;
    boff[u] = block4x8_offsets(c / CG, c % CG, kvstride);
  }
  auto load_tile = [&](int it) {
    const int64_t k0 = (int64_t)it * BC;
    const auto rk = tile_rsrc(kbase + k0 * kvstride, c1 - k0, BC, kvstride);
    const auto rv = tile_rsrc(vbase + k0 * kvstride, c1 - k0, BC, kvstride);
#pragma unroll
    for (int u = 0; u < IPT; ++u) {
      if (ITEMS % 256 == 0 || tid + 256 * u < ITEMS) {
        load_block4x8(kreg[u], rk, boff[u]);
        load_block4x8(vreg[u], rv, boff[u]);
      }
    }
  };

  load_tile(0);
  for (int it = 0; it < nkv; ++it) {
    const int64_t k0 = (int64_t)it * BC;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < IPT; ++u) {
      const int c = tid + 256 * u;
      if (ITEMS % 256 == 0 || c < ITEMS) {
        const int rg = c / CG, cg = c % CG;
        store_block_tile<D>(kreg[u], Ks, rg, cg);
        store_block_tile<D>(vreg[u], Vs, rg, cg);
      }
    }
    __syncthreads();
    if (it + 1 < nkv) load_tile(it + 1);

    // S^T = K Q^T for the tile's two 32-key blocks.
    f32x16 sv[2];
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      sv[jb] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        sv[jb] = mfma32(ld_lds_nat<D>(Ks, nat, 32 * jb, kk), qf[kk], sv[jb]);
      }
    }
    // Causal mask: only tiles that reach past the wave's first row need it.
    if (k0 + BC - 1 > q0 + 32 * w) {
      const int rel = (int)(r - k0);  // key offset within the tile of this row
#pragma unroll
      for (int jb = 0; jb < 2; ++jb) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          if (32 * jb + 8 * (v / 4) + 4 * g + (v % 4) > rel) sv[jb][v] = -INFINITY;
        }
      }
    }
  // Online softmax, base 2: x = s * scale * log2(e).  The running max m
    // is only moved when some row of the wave sees a tile max more than
    // kLazyMax above it (then O and l are rescaled); otherwise the stale m
    // is kept, so P = exp2(x - m) stays <= 2^kLazyMax -- exact in fp32, and
    // in range for bf16 -- and the 64-register O rescale is skipped.
    float mx = -INFINITY;
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sv[jb][v]);
    }
    mx = fmaxf(mx, xor32(mx)) * C;
    if (__any(mx > m + kLazyMax)) {
      const float mnew = fmaxf(m, mx);
      const float alpha = fast_exp2(m - mnew);  // m = -inf on the first tile: 0
      m = mnew;
      lsum *= alpha;
#pragma unroll
      for (int db = 0; db < ND; ++db) {
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
      }
    }
    bf16x8 pb[4];
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      float p[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        p[v] = fast_exp2(sv[jb][v] * C - m);
        lsum += p[v];
      }
      pb[2 * jb] = pack_bf16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
      pb[2 * jb + 1] = pack_bf16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
    }
    // O^T += V^T P^T.
#pragma unroll
    for (int db = 0; db < ND; ++db) {
#pragma unroll
      for (int kb = 0; kb < BC / 16; ++kb) {
        o[db] = mfma32(ld_lds_tr<D>(Vs, trb, 16 * kb, 32 * db), pb[kb], o[db]);
      }
    }
  }

  const float lt = lsum + xor32(lsum);
  if (rvalid) {
    const float inv = 1.f / lt;
    uint16_t* orow = static_cast<uint16_t*>(a.o) + ((b * s + (r - c0)) * a.Hq + h) * D;
#pragma unroll
    for (int db = 0; db < ND; ++db) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        *reinterpret_cast<u32x2*>(orow + 32 * db + 8 * q4 + 4 * g) =
            pack_bf16x4(o[db][4 * q4 + 0] * inv, o[db][4 * q4 + 1] * inv, o[db][4 * q4 + 2] * inv,
                        o[db][4 * q4 + 3] * inv);
      }
    }
    if (g == 0) a.lse[(b * a.Hq + h) * s + (r - c0)] = (m + fast_log2(lt)) * kLn2;
  }
}

}  // namespace

hipError_t launch_fwd_bf16(const ChunkArgs& a, hipStream_t stream) {
  const int64_t s = a.c1 - a.c0;
  dim3 grid((unsigned)((s + kFwdBR - 1) / kFwdBR), (unsigned)a.Hq, (unsigned)a.B);
  if (a.D == 128) {
    hipLaunchKernelGGL(fwd_bf16_kernel<128>, grid, dim3(256), 0, stream, a);
  } else if (a.D == 64) {
    hipLaunchKernelGGL(fwd_bf16_kernel<64>, grid, dim3(256), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sppo
