// Forward of one chunk of sequence-chunked causal attention, bf16 in / fp32
// accumulate, for gfx950 (MI355X).
//
// Chunk i's queries (rows [c0, c1)) attend to keys [0, c1): every earlier
// chunk fully, the diagonal block causally (two-level activation management,
// Sec. 5.1 of SPPO: K/V of all earlier subsequences stay resident on the GPU).
//
// One workgroup = 4 waves = 128 query rows of one head; each wave owns 32
// rows (lane <-> query, so row statistics are in-lane plus one exchange with
// lane^32).  Keys stream through LDS by LDS-DMA: K in a ring of four 32-key
// sub-block buffers, V in two 64-key tile buffers, one barrier per 64-key
// tile.  Per 32-key sub-block u each wave computes
//   S^T(u) = K(u) Q^T          (8x v_mfma_f32_32x32x16_bf16, D = 128)
//   P^T(u) = exp2(S^T C - m)   (online softmax in base 2, lazy rescale)
//   O^T   += V(u)^T P^T(u)     (8 MFMAs, P^T fed from S^T's registers)
// software pipelined: the MFMAs of S^T(u+1) run while the VALU turns S^T(u)
// into P^T(u), and the row max of S^T(u+1) is reduced while the PV MFMAs of
// u run.  Key tiles that reach the workgroup's own rows (the causal mask) are
// done afterwards, one at a time.  The epilogue writes O = O^T / l (bf16)
// and LSE = ln2 * (m + log2 l).
#include "sppo_kernels.h"
#include "tile_common.h"

namespace sppo {
namespace {

constexpr int kFwdBR = 128;      // query rows per workgroup (4 waves x 32)
constexpr int kFwdBC = 64;       // keys per V tile (two K sub-blocks)
constexpr float kLazyMax = 8.f;  // log2 headroom before the running max moves

#define SGB(mask, n) __builtin_amdgcn_sched_group_barrier(mask, n, 0)
constexpr int kSgMFMA = 0x008, kSgVALU = 0x002, kSgDSRead = 0x100, kSgTrans = 0x400;

template <int D>
__global__ __launch_bounds__(256, 2) void fwd_bf16_kernel(ChunkArgs a) {
  constexpr int BR = kFwdBR, BC = kFwdBC;
  using T = XTile<D>;
  constexpr int P = T::P;
  constexpr int NK = D / 16;  // k-steps of K Q^T
  constexpr int ND = D / 32;  // 32-wide d blocks of O^T
  constexpr int IPWK = (32 / T::RPI) / 4, IPWV = (BC / T::RPI) / 4;  // DMA instructions per wave
  static_assert(IPWK >= 1 && IPWK * 4 * T::RPI == 32 && IPWV * 4 * T::RPI == BC, "tiles split over 4 waves");
  __shared__ __attribute__((aligned(1024))) uint16_t K0[32 * P];
  __shared__ __attribute__((aligned(1024))) uint16_t K1[32 * P];
  __shared__ __attribute__((aligned(1024))) uint16_t K2[32 * P];
  __shared__ __attribute__((aligned(1024))) uint16_t K3[32 * P];
  __shared__ __attribute__((aligned(1024))) uint16_t V0[BC * P];
  __shared__ __attribute__((aligned(1024))) uint16_t V1[BC * P];
  auto kbuf = [&](auto I) -> uint16_t* {
    if constexpr (decltype(I)::value == 0) return K0;
    else if constexpr (decltype(I)::value == 1) return K1;
    else if constexpr (decltype(I)::value == 2) return K2;
    else return K3;
  };
  auto vbuf = [&](auto I) -> uint16_t* {
    if constexpr (decltype(I)::value == 0) return V0;
    else return V1;
  };
  auto kbuf_rt = [&](int i) -> uint16_t* { return i == 0 ? K0 : i == 1 ? K1 : i == 2 ? K2 : K3; };

  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  const GridPos gp = xcd_grouped();
  const int t = gridDim.x - 1 - gp.x;  // longest (latest) query tiles first
  const int h = gp.y;
  const int64_t b = gp.z;
  const int hk = h / (a.Hq / a.Hkv);
  const int64_t c0 = a.c0, c1 = a.c1, s = c1 - c0;
  const int64_t q0 = c0 + (int64_t)t * BR;
  const int64_t r = q0 + w * 32 + l32;
  const bool rvalid = r < c1;
  const int64_t kend = (q0 + BR < c1) ? q0 + BR : c1;
  const int nkv = (int)((kend + BC - 1) / BC);
  const int nsub = 2 * nkv;
  const int nfull = (int)(q0 / BC);  // tiles every row of the workgroup sees in full
  const float C = a.scale * kLog2e;

  int nat[NK];
#pragma unroll
  for (int kk = 0; kk < NK; ++kk) nat[kk] = T::nat(lane, kk);
  int tro[ND][2];
#pragma unroll
  for (int db = 0; db < ND; ++db) {
    tro[db][0] = T::tr(lane, db, 0);
    tro[db][1] = T::tr(lane, db, 1);
  }
  const int64_t kvstride = (int64_t)a.Hkv * D;
  int dmak[IPWK], dmav[IPWV];
#pragma unroll
  for (int x = 0; x < IPWK; ++x) dmak[x] = T::dma(lane, w * IPWK + x, kvstride);
#pragma unroll
  for (int x = 0; x < IPWV; ++x) dmav[x] = T::dma(lane, w * IPWV + x, kvstride);

  bf16x8 qf[NK];
  {
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) + ((b * s + (r - c0)) * a.Hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) qf[kk] = rvalid ? as_bf16x8(ld_global16(qrow + 16 * kk + 8 * g)) : bf16x8{};
  }
  const uint16_t* kbase = static_cast<const uint16_t*>(a.k) + (b * a.S * a.Hkv + hk) * D;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v) + (b * a.S * a.Hkv + hk) * D;

  // The next K sub-block (32 keys) or V tile (64 keys) into LDS; keys past
  // the chunk end load as zeros.  Both are issued in key order, so scalar
  // state walks K and V (no per-call index arithmetic).
  const int krow_bytes = (int)(kvstride * 2);
  uint64_t ka = uniform_u64(reinterpret_cast<uint64_t>(kbase)), va = uniform_u64(reinterpret_cast<uint64_t>(vbase));
  int remk = (int)c1, remv = (int)c1;  // keys left from the next sub-block / tile
  auto issue_k = [&](uint16_t* dst) {
    const int n = remk <= 0 ? 0 : (remk < 32 ? remk : 32);
    const auto rk = uniform_rsrc(ka, n * krow_bytes);
#pragma unroll
    for (int x = 0; x < IPWK; ++x) lds_dma16(rk, dst + (w * IPWK + x) * 512, dmak[x]);
    ka += (uint64_t)32 * krow_bytes;
    remk -= 32;
  };
  auto issue_v = [&](uint16_t* dst) {
    const int n = remv <= 0 ? 0 : (remv < BC ? remv : BC);
    const auto rv = uniform_rsrc(va, n * krow_bytes);
#pragma unroll
    for (int x = 0; x < IPWV; ++x) lds_dma16(rv, dst + (w * IPWV + x) * 512, dmav[x]);
    va += (uint64_t)BC * krow_bytes;
    remv -= BC;
  };

  f32x16 o[ND];
#pragma unroll
  for (int db = 0; db < ND; ++db) o[db] = f32x16{};
  float m = -INFINITY, lsum = 0.f;

  // The running max m moves only when some row of the wave sees a max more
  // than kLazyMax above it (then O and l are rescaled); otherwise the stale m
  // is kept, so P = exp2(x - m) stays <= 2^kLazyMax -- exact in fp32 and in
  // range for bf16 -- and the O rescale is skipped.
  auto rescale_if_needed = [&](float mx) {
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
  };
  // Row max (scaled to base 2) of a 32-key S^T block: 16 keys in-lane, the
  // other 16 in lane^32.
  auto row_max = [&](const f32x16& x) {
    const float a = max3_nc(x[0], x[1], x[2]), b = max3_nc(x[3], x[4], x[5]), c = max3_nc(x[6], x[7], x[8]);
    const float d = max3_nc(x[9], x[10], x[11]), e = max3_nc(x[12], x[13], x[14]);
    return max_xor32(max_nc(max3_nc(a, b, c), max3_nc(d, e, x[15]))) * C;
  };
  auto ld_vt = [&](const uint16_t* V, int db, int kb) {
    return ld_tr(V, tro[db][0] + 16 * kb * P, tro[db][1] + 16 * kb * P);
  };

  // One steady sub-block step: A then B.
  //   A: S^T(u+1) = K(u+1) Q^T (MFMA) | P^T(u) = exp2(S^T(u) C - m), bf16 pack (VALU)
  //   B: O^T += V(u)^T P^T(u)   (MFMA) | row sums of P(u), row max of S^T(u+1) (VALU)
  // Knext: sub-block u+1's K buffer; Vh: sub-block u's 32 V rows.
  auto step = [&](const f32x16& scur, f32x16& snext, const uint16_t* Knext, const uint16_t* Vh) -> float {
    bf16x8 kop[NK];
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) kop[kk] = ld_nat(Knext, nat[kk]);
    bf16x8 vop[ND][2];
#pragma unroll
    for (int db = 0; db < ND; ++db) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) vop[db][kb] = ld_vt(Vh, db, kb);
    }
    float p[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) p[v] = fast_exp2(scur[v] * C - m);
    bf16x8 pb[2];
    pb[0] = pack_bf16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
    pb[1] = pack_bf16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
    snext = mfma32(kop[0], qf[0], f32x16{});
#pragma unroll
    for (int kk = 1; kk < NK; ++kk) snext = mfma32(kop[kk], qf[kk], snext);
#pragma unroll
    for (int db = 0; db < ND; ++db) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) o[db] = mfma32(vop[db][kb], pb[kb], o[db]);
    }
    float s4[4];
#pragma unroll
    for (int y = 0; y < 4; ++y) s4[y] = (p[4 * y] + p[4 * y + 1]) + (p[4 * y + 2] + p[4 * y + 3]);
    lsum += (s4[0] + s4[1]) + (s4[2] + s4[3]);
    const float mx = row_max(snext);
    // A: four K reads and four exponent FMAs up front, then per MFMA one more
    // read, 16 / NK exps (the scheduling groups count transcendental ops
    // apart from other VALU ops) and ~4 VALU ops; no VALU right after the
    // last S^T MFMA (what is left is the row max of S^T(u+1), which would
    // wait for that MFMA to finish).
    SGB(kSgDSRead, 4);
    SGB(kSgVALU, 4);
#pragma unroll
    for (int i = 0; i < NK; ++i) {
      SGB(kSgMFMA, 1);
      if (i < NK - 4) {
        SGB(kSgDSRead, 1);
      } else {
        SGB(kSgDSRead, 2);
      }
      SGB(kSgTrans, 16 / NK);
      if (i < NK - 1) SGB(kSgVALU, 4);
    }
    // B: the first PV MFMA, the remaining V reads, then the other PV MFMAs
    // with the sums and the max.
    SGB(kSgMFMA, 1);
    SGB(kSgDSRead, 8);
    SGB(kSgVALU, 4);
#pragma unroll
    for (int i = 1; i < 2 * ND; ++i) {
      SGB(kSgMFMA, 1);
      SGB(kSgVALU, 4);
    }
    return mx;
  };

  // Prologue: K sub-blocks 0..2 and V tile 0.
  issue_k(K0);
  issue_v(V0);
  if (1 < nsub) issue_k(K1);
  if (2 < nsub) issue_k(K2);
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  __syncthreads();
  int klast = nsub < 3 ? nsub - 1 : 2, vlast = 0;  // last K sub-block / V tile issued

  if (nfull > 0) {
    const int U = 2 * nfull;
    f32x16 sa, sb;
    sa = mfma32(ld_nat(K0, nat[0]), qf[0], f32x16{});
#pragma unroll
    for (int kk = 1; kk < NK; ++kk) sa = mfma32(ld_nat(K0, nat[kk]), qf[kk], sa);
    rescale_if_needed(row_max(sa));
    __syncthreads();  // every wave is done with K0 before sub-block 4 lands there
    if (3 < nsub) issue_k(K3);
    if (4 < nsub) issue_k(K0);
    if (1 < nkv) issue_v(V1);
    // Tile j, parity PAR (every LDS base an immediate): sub-blocks 2j (S^T in
    // sa) and 2j+1 (S^T in sb).  At its start K sub-blocks <= 2j+2 and V tile
    // j have landed; sub-blocks 2j-1, 2j and V tile j-1 are free for
    // sub-blocks 2j+3, 2j+4 and V tile j+1.
    auto tile = [&](int j, auto par) {
      constexpr int PAR = decltype(par)::value;
      if (j > 0) {
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
        __syncthreads();
        if (2 * j + 3 < nsub) issue_k(kbuf(IC<(2 * PAR + 3) & 3>{}));
        if (2 * j + 4 < nsub) issue_k(kbuf(IC<(2 * PAR) & 3>{}));
        if (j + 1 < nkv) issue_v(vbuf(IC<(PAR + 1) & 1>{}));
      }
      const uint16_t* V = vbuf(IC<PAR>{});
      rescale_if_needed(step(sa, sb, kbuf(IC<(2 * PAR + 1) & 3>{}), V));
      const float mx = step(sb, sa, kbuf(IC<(2 * PAR + 2) & 3>{}), V + 32 * P);
      if (2 * j + 2 < U) rescale_if_needed(mx);  // past the last steady tile it is not a real max
    };
    int j = 0;
    for (; j + 2 <= nfull; j += 2) {
      tile(j, IC<0>{});
      tile(j + 1, IC<1>{});
    }
    if (j < nfull) tile(j, IC<0>{});
    klast = 2 * nfull + 2 < nsub - 1 ? 2 * nfull + 2 : nsub - 1;
    vlast = nfull < nkv - 1 ? nfull : nkv - 1;
  }

  // Diagonal tiles [nfull, nkv), with the causal mask, one 64-key tile at a
  // time; the first was loaded ahead by the steady loop (or the prologue).
  for (int j = nfull; j < nkv; ++j) {
    if (j > nfull) {
      __syncthreads();  // every wave is done with tile j-1
      for (int u = klast + 1; u <= 2 * j + 1 && u < nsub; ++u) issue_k(kbuf_rt(u & 3));
      if (2 * j + 1 > klast) klast = 2 * j + 1 < nsub - 1 ? 2 * j + 1 : nsub - 1;
      if (j > vlast) {
        issue_v((j & 1) ? V1 : V0);
        vlast = j;
      }
    }
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
    const int64_t k0 = (int64_t)j * BC;
    const uint16_t* V = (j & 1) ? V1 : V0;
    f32x16 sv[2];
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      const uint16_t* K = kbuf_rt((2 * j + jb) & 3);
      sv[jb] = mfma32(ld_nat(K, nat[0]), qf[0], f32x16{});
#pragma unroll
      for (int kk = 1; kk < NK; ++kk) sv[jb] = mfma32(ld_nat(K, nat[kk]), qf[kk], sv[jb]);
    }
    const int rel = (int)(r - k0);  // key offset within the tile of this row
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        if (32 * jb + 8 * (v / 4) + 4 * g + (v % 4) > rel) sv[jb][v] = -INFINITY;
      }
    }
    rescale_if_needed(fmaxf(row_max(sv[0]), row_max(sv[1])));
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      float p[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        p[v] = fast_exp2(sv[jb][v] * C - m);
        lsum += p[v];
      }
      bf16x8 pb[2];
      pb[0] = pack_bf16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
      pb[1] = pack_bf16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
#pragma unroll
      for (int db = 0; db < ND; ++db) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) o[db] = mfma32(ld_vt(V + 32 * jb * P, db, kb), pb[kb], o[db]);
      }
    }
  }

  const float lt = sum_xor32(lsum);
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
