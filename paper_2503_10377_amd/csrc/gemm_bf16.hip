// Dense bf16 GEMM on MFMA (fp32 accumulation) for the projections and the
// MLP of a full transformer layer chunk:  C[M, N] (op)= sum_k A(m, k) B(k, n).
//
// Two operand layouts, both read by LDS-DMA into the swizzled tiles of
// tile_common.h:
//   NT  A [M, K], B [N, K] row-major (k contiguous in both; natural operand
//       reads).  The forward projections x W use the transposed weight W^T
//       [out, in] as B; the data gradients dY W^T use the weight W [in, out]
//       as B.
//   TN  A stored [K, M], B stored [K, N] row-major (k = row; transposed
//       operand reads): the weight gradients X^T dY, accumulated in fp32.
// Both operands of a product read the same k-slot map (natural or
// transposed), so their k values pair up.
//
// Workgroup tile 256 x 256, 8 waves (4 along M x 2 along N, each 64 x 128 =
// 2 x 4 MFMA tiles of 32 x 32), k-block 64, two LDS stages: the DMA of
// k-block kb+1 runs under the MFMAs of k-block kb.
#include "sppo_kernels.h"
#include "tile_common.h"

namespace sppo {
namespace {

constexpr int GBM = 256, GBN = 256, GBK = 64;

__device__ __forceinline__ float bf16_round(float x) { return (float)(__bf16)x; }


template <int TN, int EPI>
__global__ __launch_bounds__(512, 1) void gemm_bf16_kernel(GemmArgs g) {
  // The residual and GELU' epilogues read aux: they run with the MFMA
  // operands swapped (acc = C^T), which gives each lane four consecutive
  // columns and vector loads / stores (17% faster for GELU', 2% for the
  // residual); the others keep lane <-> column, whose stores cover whole
  // 64-byte row segments (the swapped layout was 4-13% slower for them).
  constexpr bool kColEpi = EPI == kEpiAddBf16 || EPI == kEpiDGelu;
  // Stage s: A tile then B tile.  NT: [256 rows][64] (XTile<64>); TN:
  // [64 k-rows][256] as two [64][128] halves (XTile<128>).
  constexpr int TILE = GBM * GBK;  // elements per operand tile
  __shared__ __attribute__((aligned(1024))) uint16_t A0[TILE], B0[TILE], A1[TILE], B1[TILE];
  using T64 = XTile<64>;
  using T128 = XTile<128>;

  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, gh = lane >> 5;
  const int wm = w & 3, wn = w >> 2;  // wave tile rows 64 wm.., cols 128 wn..
  const int64_t m0 = (int64_t)blockIdx.y * GBM, n0 = (int64_t)blockIdx.x * GBN;

  // ---- DMA: 32 wave instructions (1 KiB each) per operand tile, 4 per wave.
  int da[4], db[4];
  if constexpr (!TN) {
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      da[x] = T64::dma(lane, w * 4 + x, g.lda);
      db[x] = T64::dma(lane, w * 4 + x, g.ldb);
    }
  } else {
    // instruction u covers rows 4u.. of half u / 16
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int u = w * 4 + x, half = u >> 4;
      da[x] = T128::dma(lane, u & 15, g.lda) + half * 128 * 2;
      db[x] = T128::dma(lane, u & 15, g.ldb) + half * 128 * 2;
    }
  }
  auto issue = [&](int64_t k0, uint16_t* sa, uint16_t* sb) {
    if constexpr (!TN) {
      const int64_t va = g.M - m0, vb = g.N - n0;
      const int na = va <= 0 ? 0 : (va < GBM ? (int)va : GBM);
      const int nb = vb <= 0 ? 0 : (vb < GBN ? (int)vb : GBN);
      const auto ra = uniform_rsrc(reinterpret_cast<uint64_t>(g.a + m0 * g.lda + k0), na * (int)(g.lda * 2));
      const auto rb = uniform_rsrc(reinterpret_cast<uint64_t>(g.b + n0 * g.ldb + k0), nb * (int)(g.ldb * 2));
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        lds_dma16(ra, sa + (w * 4 + x) * 512, da[x]);
        lds_dma16(rb, sb + (w * 4 + x) * 512, db[x]);
      }
    } else {
      const int64_t vk = g.K - k0;
      const int nk = vk <= 0 ? 0 : (vk < GBK ? (int)vk : GBK);
      const auto ra = uniform_rsrc(reinterpret_cast<uint64_t>(g.a + k0 * g.lda + m0), nk * (int)(g.lda * 2));
      const auto rb = uniform_rsrc(reinterpret_cast<uint64_t>(g.b + k0 * g.ldb + n0), nk * (int)(g.ldb * 2));
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int u = w * 4 + x;  // half u / 16, rows 4 (u % 16) ..
        lds_dma16(ra, sa + (u >> 4) * (GBK * 128) + (u & 15) * 512, da[x]);
        lds_dma16(rb, sb + (u >> 4) * (GBK * 128) + (u & 15) * 512, db[x]);
      }
    }
  };

  // ---- operand reads
  int nat[4];
  int tro[4][2];
  if constexpr (!TN) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) nat[kk] = T64::nat(lane, kk);
  } else {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      tro[d][0] = T128::tr(lane, d, 0);
      tro[d][1] = T128::tr(lane, d, 1);
    }
  }
  // A operand of M tile mt, k-step kk; B operand of N tile nt.
  auto a_op = [&](const uint16_t* sa, int mt, int kk) {
    if constexpr (!TN) {
      return ld_nat(sa + (wm * 64 + 32 * mt) * 64, nat[kk]);
    } else {
      const int ml = wm * 64 + 32 * mt;  // column in the [64][256] tile
      const uint16_t* hb = sa + (ml >> 7) * (GBK * 128);
      const int d = (ml & 127) >> 5;
      return ld_tr(hb, tro[d][0] + 16 * kk * 128, tro[d][1] + 16 * kk * 128);
    }
  };
  auto b_op = [&](const uint16_t* sb, int nt, int kk) {
    if constexpr (!TN) {
      return ld_nat(sb + (wn * 128 + 32 * nt) * 64, nat[kk]);
    } else {
      const uint16_t* hb = sb + wn * (GBK * 128);
      return ld_tr(hb, tro[nt][0] + 16 * kk * 128, tro[nt][1] + 16 * kk * 128);
    }
  };

  f32x16 acc[2][4];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[mt][nt] = f32x16{};
  }
  // Four k-steps per stage, eight MFMAs each; the six operand reads of k-step
  // kk+1 are issued before the MFMAs of k-step kk (register double buffer),
  // and the second wave on the SIMD covers what latency remains.
  auto compute = [&](const uint16_t* sa, const uint16_t* sb) {
    bf16x8 ao[2][2], bo[2][4];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) ao[0][mt] = a_op(sa, mt, 0);
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) bo[0][nt] = b_op(sb, nt, 0);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int cur = kk & 1, nxt = cur ^ 1;
      if (kk < 3) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) ao[nxt][mt] = a_op(sa, mt, kk + 1);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) bo[nxt][nt] = b_op(sb, nt, kk + 1);
      }
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          if constexpr (kColEpi) acc[mt][nt] = mfma32(bo[cur][nt], ao[cur][mt], acc[mt][nt]);
          else acc[mt][nt] = mfma32(ao[cur][mt], bo[cur][nt], acc[mt][nt]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // k-blocks in pairs (buffers 0, 1), then an odd last one: the loop has a
  // single exit, so the accumulators stay in place.
  const int nkb = (int)((g.K + GBK - 1) / GBK);
  issue(0, A0, B0);
  int kb = 0;
  for (; kb + 2 <= nkb; kb += 2) {
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();  // k-block kb landed; every wave is done with kb-1
    issue((int64_t)(kb + 1) * GBK, A1, B1);
    compute(A0, B0);
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
    if (kb + 2 < nkb) issue((int64_t)(kb + 2) * GBK, A0, B0);
    compute(A1, B1);
  }
  if (kb < nkb) {
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
    compute(A0, B0);
  }

  constexpr bool kLoads = EPI == kEpiAddBf16 || EPI == kEpiDGelu || EPI == kEpiAccF32;
  if constexpr (!kColEpi) {
    // ---- epilogue, lane <-> column n, v <-> row m (8 (v/4) + 4 (l/32) + v%4);
    // one 32 x 32 tile at a time.  The fp32-accumulate epilogue loads eight
    // rows' old values before storing the eight results (one memory round
    // trip, not one per element); a tile whose 32 rows are all below M takes
    // a branch-free path.
    auto roff = [](int v) { return 8 * (v / 4) + (v % 4); };
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        __builtin_amdgcn_sched_barrier(0);
        const int64_t n = n0 + wn * 128 + 32 * nt + l32;
        const int64_t mb = m0 + wm * 64 + 32 * mt + 4 * gh;
        const bool full = m0 + wm * 64 + 32 * mt + 32 <= g.M;  // uniform over the wave
        // element offsets from C / aux fit 32 bits (checked by the C ABI): one
        // register per address, on the wave-uniform base pointer
        const uint32_t cb = (uint32_t)(mb * g.ldc + n), ab = (uint32_t)(mb * g.ldaux + n);
        const uint32_t cs = (uint32_t)g.ldc, as = (uint32_t)g.ldaux;
        if (n < g.N) {
          // in halves of eight rows: the eight loads, then the eight results
#pragma unroll
          for (int hb = 0; hb < 2; ++hb) {
            float in[8];
            if constexpr (kLoads) {
#pragma unroll
              for (int u = 0; u < 8; ++u) {
                const int v = 8 * hb + u;
                in[u] = 0.f;
                if (full || mb + roff(v) < g.M) {
                  if constexpr (EPI == kEpiAccF32) in[u] = static_cast<const float*>(g.c)[cb + roff(v) * cs];
                  else in[u] = (float)reinterpret_cast<const __bf16*>(g.aux)[ab + roff(v) * as];
                }
              }
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const int v = 8 * hb + u;
              if (full || mb + roff(v) < g.M) {
                const float x = acc[mt][nt][v];
                const uint32_t ic = cb + roff(v) * cs;
                if constexpr (EPI == kEpiBf16) {
                  static_cast<__bf16*>(g.c)[ic] = (__bf16)x;
                } else if constexpr (EPI == kEpiAddBf16) {
                  static_cast<__bf16*>(g.c)[ic] = (__bf16)(x + in[u]);
                } else if constexpr (EPI == kEpiGelu) {
                  const __bf16 pre = (__bf16)x;
                  reinterpret_cast<__bf16*>(g.aux)[ab + roff(v) * as] = pre;
                  static_cast<__bf16*>(g.c)[ic] = (__bf16)gelu_tanh((float)pre);
                } else if constexpr (EPI == kEpiDGelu) {
                  static_cast<__bf16*>(g.c)[ic] = (__bf16)(x * gelu_tanh_grad(in[u]));
                } else if constexpr (EPI == kEpiAccF32) {
                  static_cast<float*>(g.c)[ic] = in[u] + x;
                } else {
                  static_cast<float*>(g.c)[ic] = x;
                }
              }
            }
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      }
    }
  } else {
    // ---- epilogue.  The MFMAs take B as their first operand, so acc holds
    // C^T: lane l has row m = l % 32 of the 32 x 32 tile and, for v = 4q + e,
    // column n = 8 q + 4 (l / 32) + e -- four consecutive columns per q, one
    // 8-byte (bf16) or 16-byte (fp32) vector access each.  Epilogues that read
    // (residual, GELU pre-activation, fp32 accumulator) load the tile's four
    // vectors before storing any result.  Element offsets from C / aux fit 32
    // bits, and N, ldc, ldaux are multiples of 4 (checked by the C ABI).
    typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        __builtin_amdgcn_sched_barrier(0);
        const int64_t m = m0 + wm * 64 + 32 * mt + l32;
        const int64_t nb = n0 + wn * 128 + 32 * nt + 4 * gh;
        if (m < g.M) {
          const uint32_t cb = (uint32_t)(m * g.ldc + nb), ab = (uint32_t)(m * g.ldaux + nb);
          float in[16];
          if constexpr (kLoads) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              if (nb + 8 * q < g.N) {
                if constexpr (EPI == kEpiAccF32) {
                  const float4 t = *reinterpret_cast<const float4*>(static_cast<const float*>(g.c) + cb + 8 * q);
                  in[4 * q] = t.x; in[4 * q + 1] = t.y; in[4 * q + 2] = t.z; in[4 * q + 3] = t.w;
                } else {
                  const bf16x4_t t = *reinterpret_cast<const bf16x4_t*>(static_cast<const __bf16*>(g.aux) + ab + 8 * q);
#pragma unroll
                  for (int e = 0; e < 4; ++e) in[4 * q + e] = (float)t[e];
                }
              }
            }
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (nb + 8 * q < g.N) {
              const uint32_t ic = cb + 8 * q;
              float r[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const float x = acc[mt][nt][4 * q + e];
                if constexpr (EPI == kEpiAddBf16) r[e] = x + in[4 * q + e];
                else if constexpr (EPI == kEpiDGelu) r[e] = x * gelu_tanh_grad(in[4 * q + e]);
                else if constexpr (EPI == kEpiAccF32) r[e] = in[4 * q + e] + x;
                else r[e] = x;
              }
              if constexpr (EPI == kEpiAccF32 || EPI == kEpiF32) {
                *reinterpret_cast<float4*>(static_cast<float*>(g.c) + ic) = make_float4(r[0], r[1], r[2], r[3]);
              } else if constexpr (EPI == kEpiGelu) {
                const bf16x4_t pre = {(__bf16)r[0], (__bf16)r[1], (__bf16)r[2], (__bf16)r[3]};
                *reinterpret_cast<bf16x4_t*>(static_cast<__bf16*>(g.aux) + ab + 8 * q) = pre;
                const bf16x4_t o = {(__bf16)gelu_tanh((float)pre[0]), (__bf16)gelu_tanh((float)pre[1]),
                                    (__bf16)gelu_tanh((float)pre[2]), (__bf16)gelu_tanh((float)pre[3])};
                *reinterpret_cast<bf16x4_t*>(static_cast<__bf16*>(g.c) + ic) = o;
              } else {
                const bf16x4_t o = {(__bf16)r[0], (__bf16)r[1], (__bf16)r[2], (__bf16)r[3]};
                *reinterpret_cast<bf16x4_t*>(static_cast<__bf16*>(g.c) + ic) = o;
              }
            }
          }
        }
      }
    }
  }
}

template <int TN>
hipError_t launch_epi(const GemmArgs& g, dim3 grid, hipStream_t stream) {
  switch (g.epi) {
    case kEpiBf16: hipLaunchKernelGGL((gemm_bf16_kernel<TN, kEpiBf16>), grid, dim3(512), 0, stream, g); break;
    case kEpiAddBf16: hipLaunchKernelGGL((gemm_bf16_kernel<TN, kEpiAddBf16>), grid, dim3(512), 0, stream, g); break;
    case kEpiGelu: hipLaunchKernelGGL((gemm_bf16_kernel<TN, kEpiGelu>), grid, dim3(512), 0, stream, g); break;
    case kEpiDGelu: hipLaunchKernelGGL((gemm_bf16_kernel<TN, kEpiDGelu>), grid, dim3(512), 0, stream, g); break;
    case kEpiAccF32: hipLaunchKernelGGL((gemm_bf16_kernel<TN, kEpiAccF32>), grid, dim3(512), 0, stream, g); break;
    case kEpiF32: hipLaunchKernelGGL((gemm_bf16_kernel<TN, kEpiF32>), grid, dim3(512), 0, stream, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(const GemmArgs& g, hipStream_t stream) {
  if (g.M <= 0 || g.N <= 0 || g.K <= 0) return hipErrorInvalidValue;
  dim3 grid((unsigned)((g.N + GBN - 1) / GBN), (unsigned)((g.M + GBM - 1) / GBM));
  return g.tn ? launch_epi<1>(g, grid, stream) : launch_epi<0>(g, grid, stream);
}

}  // namespace sppo
