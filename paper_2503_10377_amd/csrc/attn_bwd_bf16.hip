// Backward of one chunk of sequence-chunked causal attention, bf16 in / fp32
// accumulate, for gfx950 (MI355X).  The reverse walk over chunks (Sec. 5.2
// of SPPO) calls this for i = N-1..0; dK/dV accumulate across calls in fp32.
//
// Three kernels, all on the caller's stream:
//   bwd_pre   Delta_r = <dO_r, O_r>                      (HBM-bound)
//   bwd_dkdv  one workgroup per 128 keys of one KV head (4 waves x 32 keys,
//             lane <-> key); streams the chunk's query tiles (64 rows, every
//             query head of the GQA group) through LDS (natural, swizzled
//             layout; Q^T and dO^T operands by transposed reads) and accumulates
//               dV += P^T dO,  dK += scale * dS^T Q
//             in registers; S = Q K^T and dP = dO V^T are recomputed.
//   bwd_dq    one workgroup per 128 query rows of one head (lane <-> query);
//             streams K/V tiles and accumulates dQ^T += K^T dS^T.
// P = exp2(S*scale*log2e - LSE*log2e), dS = P (dP - Delta).
#include <type_traits>

#include "sppo_kernels.h"
#include "tile_common.h"

namespace sppo {
namespace {

constexpr int kDqBR = 128;    // query rows per dq workgroup
constexpr int kDqBC = 64;     // keys per dq K/V tile
constexpr int kKvBKV = 128;   // keys per dkdv workgroup
constexpr int kKvBQ = 64;     // query rows per dkdv query tile

// ------------------------------------------------------------------ Delta
template <int D>
__global__ __launch_bounds__(256) void bwd_pre_bf16_kernel(ChunkArgs a) {
  constexpr int LPI = D / 8;  // lanes per (b, r, h) row, 8 bf16 each
  const int64_t s = a.c1 - a.c0;
  const int64_t nrows = a.B * s * a.Hq;
  const int64_t item = ((int64_t)blockIdx.x * 256 + threadIdx.x) / LPI;
  const int sub = threadIdx.x % LPI;
  float acc = 0.f;
  if (item < nrows) {
    const u32x4 ov = ld_global16(static_cast<const uint16_t*>(a.o) + item * D + 8 * sub);
    const u32x4 dv = ld_global16(static_cast<const uint16_t*>(a.dout) + item * D + 8 * sub);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc += __uint_as_float(ov[e] << 16) * __uint_as_float(dv[e] << 16);
      acc += __uint_as_float(ov[e] & 0xffff0000u) * __uint_as_float(dv[e] & 0xffff0000u);
    }
  }
#pragma unroll
  for (int off = LPI / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (item < nrows && sub == 0) {
    const int64_t h = item % a.Hq;
    const int64_t rr = (item / a.Hq) % s;
    const int64_t b = item / (a.Hq * s);
    a.delta[(b * a.Hq + h) * s + rr] = acc;
  }
}

// --------------------------------------------------------------------- dQ
template <int D>
__global__ __launch_bounds__(256) void bwd_dq_bf16_kernel(ChunkArgs a) {
  constexpr int BR = kDqBR, BC = kDqBC;
  using T = LdsTile<D>;
  constexpr int NK = D / 16, ND = D / 32, CG = T::CG;
  constexpr int ITEMS = (BC / 4) * CG;
  constexpr int IPT = (ITEMS + 255) / 256;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[BC * T::P];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[BC * T::P];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g = lane >> 5;
  const int t = gridDim.x - 1 - blockIdx.x;
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

  bf16x8 qf[NK], df[NK];
  float lse2 = INFINITY, dl = 0.f;
  if (rvalid) {
    const int64_t off = ((b * s + (r - c0)) * a.Hq + h) * D;
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) + off;
    const uint16_t* drow = static_cast<const uint16_t*>(a.dout) + off;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      qf[kk] = as_bf16x8(ld_global16(qrow + 16 * kk + 8 * g));
      df[kk] = as_bf16x8(ld_global16(drow + 16 * kk + 8 * g));
    }
    lse2 = a.lse[(b * a.Hq + h) * s + (r - c0)] * kLog2e;
    dl = a.delta[(b * a.Hq + h) * s + (r - c0)];
  } else {
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) qf[kk] = df[kk] = bf16x8{};
  }

  const int64_t kvstride = (int64_t)a.Hkv * D;
  const uint16_t* kbase = static_cast<const uint16_t*>(a.k) + (b * a.S * a.Hkv + hk) * D;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v) + (b * a.S * a.Hkv + hk) * D;

  f32x16 dq[ND];
#pragma unroll
  for (int db = 0; db < ND; ++db) dq[db] = f32x16{};

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

  // One K/V tile as scheduling regions (see the dK/dV kernel):
  //   1: natural K/V reads of keys 0..31
  //   2: S^T, dP^T MFMAs of keys 0..31  + natural reads of keys 32..63
  //   3: S^T, dP^T MFMAs of keys 32..63 + P, dS of keys 0..31 (VALU)
  //                                     + transposed K reads for keys 0..31
  //   4: dQ MFMAs over keys 0..31       + P, dS of keys 32..63
  //   5: transposed K reads for keys 32..63, then their dQ MFMAs
  auto tile_body = [&](int64_t k0, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int rel = (int)(r - k0);
    f32x16 sv[2], dp[2];
    bf16x8 dsb[4];
    bf16x8 nk[NK], nv[NK];
    bf16x8 tk[2][ND];

    auto nat_reads = [&](int jb) {
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        nk[kk] = ld_lds_nat<D>(Ks, nat, 32 * jb, kk);
        nv[kk] = ld_lds_nat<D>(Vs, nat, 32 * jb, kk);
      }
    };
    auto sdp_mfma = [&](int jb) {
      sv[jb] = f32x16{};
      dp[jb] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        sv[jb] = mfma32(nk[kk], qf[kk], sv[jb]);
        dp[jb] = mfma32(nv[kk], df[kk], dp[jb]);
      }
    };
    auto softmax = [&](int jb) {
      float ds[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float p = fast_exp2(sv[jb][v] * C - lse2);
        if (MASK && 32 * jb + 8 * (v / 4) + 4 * g + (v % 4) > rel) p = 0.f;
        ds[v] = p * (dp[jb][v] - dl);
      }
      dsb[2 * jb] = pack_bf16x8(ds[0], ds[1], ds[2], ds[3], ds[4], ds[5], ds[6], ds[7]);
      dsb[2 * jb + 1] = pack_bf16x8(ds[8], ds[9], ds[10], ds[11], ds[12], ds[13], ds[14], ds[15]);
    };
    auto tr_reads = [&](int jb) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
        for (int db = 0; db < ND; ++db) tk[hh][db] = ld_lds_tr<D>(Ks, trb, 16 * (2 * jb + hh), 32 * db);
      }
    };
    // dQ^T[d][query] += K^T dS^T: K^T comes from transposed reads of K.
    auto dq_mfma = [&](int jb) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
        for (int db = 0; db < ND; ++db) dq[db] = mfma32(tk[hh][db], dsb[2 * jb + hh], dq[db]);
      }
    };

    nat_reads(0);
    __builtin_amdgcn_sched_barrier(0);
    sdp_mfma(0);
    nat_reads(1);
    __builtin_amdgcn_sched_barrier(0);
    sdp_mfma(1);
    softmax(0);
    tr_reads(0);
    __builtin_amdgcn_sched_barrier(0);
    dq_mfma(0);
    softmax(1);
    __builtin_amdgcn_sched_barrier(0);
    tr_reads(1);
    __builtin_amdgcn_sched_barrier(0);
    dq_mfma(1);
    __builtin_amdgcn_sched_barrier(0);
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
    load_tile(it + 1 < nkv ? it + 1 : it);  // the last prefetch repeats a tile, harmlessly

    if (k0 + BC - 1 > q0 + 32 * w) {
      tile_body(k0, std::true_type{});
    } else {
      tile_body(k0, std::false_type{});
    }
  }

  if (rvalid) {
    uint16_t* qrow = static_cast<uint16_t*>(a.dq) + ((b * s + (r - c0)) * a.Hq + h) * D;
#pragma unroll
    for (int db = 0; db < ND; ++db) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        *reinterpret_cast<u32x2*>(qrow + 32 * db + 8 * q4 + 4 * g) =
            pack_bf16x4(dq[db][4 * q4 + 0] * a.scale, dq[db][4 * q4 + 1] * a.scale,
                        dq[db][4 * q4 + 2] * a.scale, dq[db][4 * q4 + 3] * a.scale);
      }
    }
  }
}

// ------------------------------------------------------------------ dK dV
template <int D>
__global__ __launch_bounds__(256) void bwd_dkdv_bf16_kernel(ChunkArgs a) {
  constexpr int BQ = kKvBQ;
  using T = LdsTile<D>;
  constexpr int NK = D / 16, ND = D / 32, CG = T::CG;
  constexpr int ITEMS = (BQ / 4) * CG;
  constexpr int IPT = (ITEMS + 255) / 256;
  __shared__ __attribute__((aligned(16))) uint16_t Qs[BQ * T::P];
  __shared__ __attribute__((aligned(16))) uint16_t Ds[BQ * T::P];
  __shared__ __attribute__((aligned(16))) float lse2s[BQ];
  __shared__ __attribute__((aligned(16))) float dls[BQ];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g = lane >> 5;
  const int hk = blockIdx.y;
  const int64_t b = blockIdx.z;
  const int G = a.Hq / a.Hkv;
  const int64_t c0 = a.c0, c1 = a.c1, s = c1 - c0;
  const int64_t kv1 = a.kv1;
  const int64_t k0 = a.kv0 + (int64_t)blockIdx.x * kKvBKV;
  const int64_t j = k0 + 32 * w + l32;  // this lane's key
  const float C = a.scale * kLog2e;
  const auto nat = T::nat_base(lane);
  const auto trb = T::tr_base(lane);

  bf16x8 kf[NK], vf[NK];
  {
    const int64_t off = ((b * a.S + j) * a.Hkv + hk) * D;
    const uint16_t* krow = static_cast<const uint16_t*>(a.k) + off;
    const uint16_t* vrow = static_cast<const uint16_t*>(a.v) + off;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      kf[kk] = j < kv1 ? as_bf16x8(ld_global16(krow + 16 * kk + 8 * g)) : bf16x8{};
      vf[kk] = j < kv1 ? as_bf16x8(ld_global16(vrow + 16 * kk + 8 * g)) : bf16x8{};
    }
  }

  f32x16 dk[ND], dv[ND];
#pragma unroll
  for (int db = 0; db < ND; ++db) dk[db] = dv[db] = f32x16{};

  // Query tiles (chunk-local) that can see a key of this workgroup.
  const int64_t qt_begin = k0 > c0 ? (k0 - c0) / BQ : 0;
  const int64_t nqt = (s + BQ - 1) / BQ;

  const int64_t qstride = (int64_t)a.Hq * D;
  Block4x8 qreg[IPT], dreg[IPT];
  Block4x8Offsets boff[IPT];
#pragma unroll
  for (int u = 0; u < IPT; ++u) {
    const int c = tid + 256 * u;
    boff[u] = block4x8_offsets(c / CG, c % CG, qstride);
  }
  float lse_r = INFINITY, dl_r = 0.f;
  auto load_tile = [&](int h, int64_t qt) {
    const int64_t tile0 = (b * s + qt * BQ) * a.Hq + h;  // first row of the tile, in D-element units
    const auto rq = tile_rsrc(static_cast<const uint16_t*>(a.q) + tile0 * D, s - qt * BQ, BQ, qstride);
    const auto rd = tile_rsrc(static_cast<const uint16_t*>(a.dout) + tile0 * D, s - qt * BQ, BQ, qstride);
#pragma unroll
    for (int u = 0; u < IPT; ++u) {
      if (ITEMS % 256 == 0 || tid + 256 * u < ITEMS) {
        load_block4x8(qreg[u], rq, boff[u]);
        load_block4x8(dreg[u], rd, boff[u]);
      }
    }
    if (tid < BQ) {
      const int64_t rr = qt * BQ + tid;
      lse_r = rr < s ? a.lse[(b * a.Hq + h) * s + rr] * kLog2e : INFINITY;
      dl_r = rr < s ? a.delta[(b * a.Hq + h) * s + rr] : 0.f;
    }
  };

  // One query tile, as five scheduling regions (sched_barrier between them
  // keeps the compiler from sinking LDS reads next to their MFMAs):
  //   1: natural reads of Q/dO rows 0..31
  //   2: S, dP MFMAs of rows 0..31        + natural reads of rows 32..63
  //   3: S, dP MFMAs of rows 32..63       + P, dS of rows 0..31 (VALU)
  //                                       + transposed Q/dO reads for rows 0..31
  //   4: dV, dK MFMAs of rows 0..31       + P, dS of rows 32..63
  //   5: transposed reads for rows 32..63, then their dV, dK MFMAs
  // so every MFMA batch has its operands in flight one region ahead and the
  // softmax VALU work of one row block can overlap the MFMAs of the other.
  // MASK selects the diagonal variant.
  auto tile_body = [&](int64_t q0, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int rel = (int)(j - q0);  // this lane's key relative to the query tile
    f32x16 sv[2], dp[2];
    bf16x8 pb[2][2], dsb[2][2];
    bf16x8 nq[NK], nd[NK];
    bf16x8 tq[2][ND], td[2][ND];

    auto nat_reads = [&](int ib) {
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        nq[kk] = ld_lds_nat<D>(Qs, nat, 32 * ib, kk);
        nd[kk] = ld_lds_nat<D>(Ds, nat, 32 * ib, kk);
      }
    };
    auto sdp_mfma = [&](int ib) {
      sv[ib] = f32x16{};
      dp[ib] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        sv[ib] = mfma32(nq[kk], kf[kk], sv[ib]);
        dp[ib] = mfma32(nd[kk], vf[kk], dp[ib]);
      }
    };
    auto softmax = [&](int ib) {
      float p[16], ds[16];
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const int qi = 32 * ib + 8 * v4 + 4 * g;
        const float4 l4 = *reinterpret_cast<const float4*>(lse2s + qi);
        const float4 d4 = *reinterpret_cast<const float4*>(dls + qi);
        const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
        const float dv4[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int v = 4 * v4 + e;
          float pv = fast_exp2(sv[ib][v] * C - lv[e]);
          if (MASK && rel > qi + e) pv = 0.f;
          p[v] = pv;
          ds[v] = pv * (dp[ib][v] - dv4[e]);
        }
      }
      pb[ib][0] = pack_bf16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
      pb[ib][1] = pack_bf16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
      dsb[ib][0] = pack_bf16x8(ds[0], ds[1], ds[2], ds[3], ds[4], ds[5], ds[6], ds[7]);
      dsb[ib][1] = pack_bf16x8(ds[8], ds[9], ds[10], ds[11], ds[12], ds[13], ds[14], ds[15]);
    };
    auto tr_reads = [&](int ib, int hh) {
#pragma unroll
      for (int db = 0; db < ND; ++db) {
        tq[hh][db] = ld_lds_tr<D>(Qs, trb, 16 * (2 * ib + hh), 32 * db);
        td[hh][db] = ld_lds_tr<D>(Ds, trb, 16 * (2 * ib + hh), 32 * db);
      }
    };
    auto dkdv_mfma = [&](int ib) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
        for (int db = 0; db < ND; ++db) {
          dv[db] = mfma32(pb[ib][hh], td[hh][db], dv[db]);
          dk[db] = mfma32(dsb[ib][hh], tq[hh][db], dk[db]);
        }
      }
    };

    nat_reads(0);
    __builtin_amdgcn_sched_barrier(0);
    sdp_mfma(0);
    nat_reads(1);
    __builtin_amdgcn_sched_barrier(0);
    sdp_mfma(1);
    softmax(0);
    tr_reads(0, 0);
    tr_reads(0, 1);
    __builtin_amdgcn_sched_barrier(0);
    dkdv_mfma(0);
    softmax(1);
    __builtin_amdgcn_sched_barrier(0);
    tr_reads(1, 0);
    tr_reads(1, 1);
    __builtin_amdgcn_sched_barrier(0);
    dkdv_mfma(1);
    __builtin_amdgcn_sched_barrier(0);
  };

  load_tile(hk * G, qt_begin);
  for (int hh = 0; hh < G; ++hh) {
    for (int64_t qt = qt_begin; qt < nqt; ++qt) {
      __syncthreads();
#pragma unroll
      for (int u = 0; u < IPT; ++u) {
        const int c = tid + 256 * u;
        if (ITEMS % 256 == 0 || c < ITEMS) {
          const int rg = c / CG, cg = c % CG;
          store_block_tile<D>(qreg[u], Qs, rg, cg);
          store_block_tile<D>(dreg[u], Ds, rg, cg);
        }
      }
      if (tid < BQ) {
        lse2s[tid] = lse_r;
        dls[tid] = dl_r;
      }
      __syncthreads();
      // Prefetch the next tile (the same one again after the last, harmless).
      {
        int nh = hh;
        int64_t nq = qt + 1;
        if (nq == nqt) {
          nq = qt_begin;
          nh = hh + 1 < G ? hh + 1 : hh;
        }
        load_tile(hk * G + nh, nq);
      }
      const int64_t q0 = c0 + qt * BQ;
      if (k0 + 32 * w + 31 > q0) {
        tile_body(q0, std::true_type{});
      } else {
        tile_body(q0, std::false_type{});
      }
    }
  }

  // Write back rows [k0, k0+128) n [kv0, kv1): lane <-> d, v <-> key.
#pragma unroll
  for (int db = 0; db < ND; ++db) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int64_t key = k0 + 32 * w + 8 * (v / 4) + 4 * g + (v % 4);
      if (key < kv1) {
        const int64_t idx = ((b * a.S + key) * a.Hkv + hk) * D + 32 * db + l32;
        const float kval = dk[db][v] * a.scale;
        const float vval = dv[db][v];
        if (a.accumulate) {
          a.dk[idx] += kval;
          a.dv[idx] += vval;
        } else {
          a.dk[idx] = kval;
          a.dv[idx] = vval;
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_bwd_pre_bf16(const ChunkArgs& a, hipStream_t stream) {
  const int64_t s = a.c1 - a.c0;
  const int64_t threads = a.B * s * a.Hq * (a.D / 8);
  dim3 grid((unsigned)((threads + 255) / 256));
  if (a.D == 128) {
    hipLaunchKernelGGL(bwd_pre_bf16_kernel<128>, grid, dim3(256), 0, stream, a);
  } else if (a.D == 64) {
    hipLaunchKernelGGL(bwd_pre_bf16_kernel<64>, grid, dim3(256), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dkdv_bf16(const ChunkArgs& a, hipStream_t stream) {
  if (a.kv0 < 0 || a.kv1 > a.c1 || a.kv0 >= a.kv1) return hipErrorInvalidValue;
  dim3 grid((unsigned)((a.kv1 - a.kv0 + kKvBKV - 1) / kKvBKV), (unsigned)a.Hkv, (unsigned)a.B);
  if (a.D == 128) {
    hipLaunchKernelGGL(bwd_dkdv_bf16_kernel<128>, grid, dim3(256), 0, stream, a);
  } else if (a.D == 64) {
    hipLaunchKernelGGL(bwd_dkdv_bf16_kernel<64>, grid, dim3(256), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dq_bf16(const ChunkArgs& a, hipStream_t stream) {
  const int64_t s = a.c1 - a.c0;
  dim3 grid((unsigned)((s + kDqBR - 1) / kDqBR), (unsigned)a.Hq, (unsigned)a.B);
  if (a.D == 128) {
    hipLaunchKernelGGL(bwd_dq_bf16_kernel<128>, grid, dim3(256), 0, stream, a);
  } else if (a.D == 64) {
    hipLaunchKernelGGL(bwd_dq_bf16_kernel<64>, grid, dim3(256), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sppo
