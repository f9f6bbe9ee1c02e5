// Backward of one chunk of sequence-chunked causal attention, bf16 in / fp32
// accumulate, for gfx950 (MI355X).  The reverse walk over chunks (Sec. 5.2
// of SPPO) calls this for i = N-1..0; dK/dV accumulate across calls in fp32.
//
// Three kernels, all on the caller's stream:
//   bwd_pre   -Delta_r = -<dO_r, O_r> and LSE2_r = LSE_r * log2(e) into the
//             context's workspace (HBM-bound); -Delta is the initial value
//             of the dP accumulators, so the MFMAs produce dP - Delta
//   bwd_dkdv  one workgroup per 128 keys of one KV head at a time (4 waves x
//             32 keys, lane <-> key, K/V fragments in registers); the chunk's
//             query rows of every head of the GQA group stream through LDS in
//             32-row sub-blocks, and per sub-block
//               S = Q K^T, dP = dO V^T, P = exp2(S C - LSE2), dS = P (dP - Delta)
//               dV += P^T dO,  dK += dS^T Q
//             The kernel is persistent (as many workgroups as the CUs
//             hold at once, one per CU at its register use): each XCD
//             takes key tiles from its own queue, in the XCD-grouped order,
//             and once it is empty from the other XCDs' queues, so XCDs that
//             run faster than others do more of the work.
//   bwd_dq    one workgroup per 128 query rows of one head (lane <-> query);
//             keys stream through LDS in 32-key sub-blocks, and per sub-block
//               S^T = K Q^T, dP^T = V dO^T, dS^T as above, dQ^T += K^T dS^T
// Both stream their sub-blocks through a six-slot LDS ring by LDS-DMA, five
// sub-blocks ahead, one barrier per sub-block, and software-pipeline them:
// the MFMAs of sub-block n+1's S and dP run while the VALU forms sub-block
// n's P and dS, then the gradient MFMAs of sub-block n run.  The order of
// every step is fixed with sched_barrier, so operand reads sit a few MFMAs
// ahead of their use.  Sub-blocks that need the causal mask are done one at
// a time, outside the pipeline.
#include "sppo_kernels.h"
#include "tile_common.h"

namespace sppo {
namespace {

constexpr int kKvKeys = 128;  // keys per dK/dV workgroup (4 waves x 32)
constexpr int kDqRows = 128;  // query rows per dQ workgroup (4 waves x 32)
constexpr int kSB = 32;       // rows (dK/dV) or keys (dQ) per sub-block
constexpr int kRing = 6;      // LDS ring slots
constexpr int kAhead = 5;     // sub-blocks loaded ahead of the one in use
// LSE2 groups loaded ahead of their use in the softmax (0: right before;
// 1: 1.3% faster at 128K, measured when the Delta groups went with them;
// all four at the step start: 0.9%).
constexpr int kLdAhead = 1;
// The B phase's first three transposed reads are issued in the last MFMA
// slots of the A phase, which read nothing else (dQ 1% faster than issuing
// them right before B).
constexpr bool kEarlyTr = true;
// Each step's barrier also waits for sub-block n+2, so the B phase of step n
// can read A(n+1)'s first natural operands in its last MFMA slots (which read
// nothing else): dK/dV 0.6% faster than reading them right after the barrier.
constexpr bool kEarlyA = true;
constexpr bool kEarlyAq = true;  // the same for the dQ kernel: 2.1% faster
static_assert(kAhead == kRing - 1, "a slot is refilled right after its last reader");

// ------------------------------------------------------------------ Delta
template <int D>
__global__ __launch_bounds__(256) void bwd_pre_bf16_kernel(ChunkArgs a) {
  constexpr int LPI = D / 8;  // lanes per (b, r, h) row, 8 bf16 each
  const int64_t s = a.c1 - a.c0;
  const int64_t nrows = a.B * s * a.Hq;
  const int64_t item = ((int64_t)blockIdx.x * 256 + threadIdx.x) / LPI;
  const int sub = threadIdx.x % LPI;
  // A backward call's queues start from zero (the dK/dV launches leave them
  // so; cleared here as well, ahead of every call's first dK/dV launch).
  if (blockIdx.x == 0 && threadIdx.x < 9) atomicExch(a.tiles + threadIdx.x, 0);
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
    const int64_t idx = (b * a.Hq + h) * s + rr;
    a.delta[idx] = -acc;
    a.lse2[idx] = a.lse[idx] * kLog2e;
  }
}

// ------------------------------------------------------------------ dK dV
template <int D>
__global__ __launch_bounds__(256, 1) void bwd_dkdv_bf16_kernel(ChunkArgs a) {
  using T = XTile<D>;
  constexpr int P = T::P, NK = D / 16, ND = D / 32;
  constexpr int IPWQ = (kSB / T::RPI) / 4;  // DMA instructions per wave per tensor per sub-block
  static_assert(IPWQ >= 1 && IPWQ * 4 * T::RPI == kSB, "sub-block splits over 4 waves");
  constexpr int DMA_PER_SB = 2 * IPWQ + 1;  // Q, dO, and one for the [LSE2 | -Delta] record
  // One LDS object per ring slot, [Q rows | dO rows], and the slots' records,
  // [LSE2 (32 floats) | -Delta (32 floats)], in an array of their own at the
  // bottom of LDS, where the broadcast reads take their offsets as immediates.
  constexpr int SLOT = 2 * kSB * P;
  __shared__ __attribute__((aligned(1024))) float REC[kRing][64];
  __shared__ __attribute__((aligned(1024))) uint16_t R0[SLOT], R1[SLOT], R2[SLOT], R3[SLOT], R4[SLOT], R5[SLOT];
  auto slot = [&](auto I) -> uint16_t* {
    constexpr int i = decltype(I)::value;
    if constexpr (i == 0) return R0; else if constexpr (i == 1) return R1; else if constexpr (i == 2) return R2;
    else if constexpr (i == 3) return R3; else if constexpr (i == 4) return R4; else return R5;
  };
  auto qbuf = [&](auto I) -> uint16_t* { return slot(I); };
  auto obuf = [&](auto I) -> uint16_t* { return slot(I) + kSB * P; };
  auto lbuf = [&](auto I) -> float* { return REC[decltype(I)::value]; };

  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  // Key tiles in the XCD-grouped order (the tiles of a KV head one after
  // another): XCD x owns positions [x T / 8, (x+1) T / 8) of the T tiles.
  // Thread 0 takes the next position from this XCD's queue, or when that
  // is used up from the next XCD's, and hands it to the workgroup through
  // LDS; -1 when every queue is used up.
  const int nx = (int)((a.kv1 - a.kv0 + kKvKeys - 1) / kKvKeys), ny = a.Hkv;
  const int total = nx * ny * (int)a.B;
  __shared__ int s_tile;
  uint32_t xcc;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
  for (;;) {
  if (tid == 0) {
    int t = -1;
    for (int y = 0; y < 8 && t < 0; ++y) {
      const int x = (int)((xcc + y) & 7);
      const int lo = (int)((int64_t)x * total / 8), hi = (int)((int64_t)(x + 1) * total / 8);
      if (lo < hi) {
        const int n = atomicAdd(a.tiles + x, 1);
        if (lo + n < hi) t = lo + n;
      }
    }
    s_tile = t;
  }
  __syncthreads();
  const int tile = s_tile;
  if (tile < 0) break;
  const GridPos gp{tile % nx, (tile / nx) % ny, tile / (nx * ny)};
  const int hk = gp.y;
  const int64_t b = gp.z;
  const int G = a.Hq / a.Hkv;
  const int64_t c0 = a.c0, c1 = a.c1, s = c1 - c0;
  const int64_t kv1 = a.kv1;
  const int64_t k0 = a.kv0 + (int64_t)gp.x * kKvKeys;
  const int64_t j = k0 + 32 * w + l32;  // this lane's key
  const float C = a.scale * kLog2e;

  // Query sub-blocks (chunk-local, 32 rows from c0): [sb_begin, sb_u) need
  // the mask, [sb_u, nsb) see every key of the workgroup.
  const int nsb = (int)((s + kSB - 1) / kSB);
  const int sb_begin = k0 > c0 ? (int)((k0 - c0) / kSB) : 0;
  int sb_u = (int)((k0 + kKvKeys - c0 + kSB - 1) / kSB);
  if (sb_u > nsb) sb_u = nsb;
  if (sb_u < sb_begin) sb_u = sb_begin;
  const int N = nsb - sb_u;  // unmasked sub-blocks per head

  int nat[NK];
#pragma unroll
  for (int kk = 0; kk < NK; ++kk) nat[kk] = T::nat(lane, kk);
  int tro[ND][2];
#pragma unroll
  for (int db = 0; db < ND; ++db) {
    tro[db][0] = T::tr(lane, db, 0);
    tro[db][1] = T::tr(lane, db, 1);
  }
  const int64_t qstride = (int64_t)a.Hq * D;
  int dmaq[IPWQ];
#pragma unroll
  for (int x = 0; x < IPWQ; ++x) dmaq[x] = T::dma(lane, w * IPWQ + x, qstride);
  // The [LSE2 | -Delta] record: waves 0, 1 load LSE2 rows 0..15, 16..31,
  // waves 2, 3 -Delta, 16 lanes each.
  const int dmal = (16 * (w & 1) + (lane & 15)) * 4;
  const float* lsrc = (w < 2) ? a.lse2 : a.delta;
  const int ldst = 32 * (w >> 1) + 16 * (w & 1);

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

  // DMA of query sub-block sb of head h into a slot; rows past the chunk load
  // zeros, so every call issues DMA_PER_SB instructions per wave.
  auto issue = [&](int h, int sb, uint16_t* qd, uint16_t* od, float* ld) {
    const int64_t r0 = (int64_t)sb * kSB;
    const int64_t valid = s - r0;
    const int64_t tile0 = (b * s + r0) * a.Hq + h;
    const auto rq = tile_rsrc(static_cast<const uint16_t*>(a.q) + tile0 * D, valid, kSB, qstride);
    const auto ro = tile_rsrc(static_cast<const uint16_t*>(a.dout) + tile0 * D, valid, kSB, qstride);
#pragma unroll
    for (int x = 0; x < IPWQ; ++x) {
      lds_dma16(rq, qd + (w * IPWQ + x) * 512, dmaq[x]);
      lds_dma16(ro, od + (w * IPWQ + x) * 512, dmaq[x]);
    }
    const int64_t nrec = valid <= 0 ? 0 : (valid < kSB ? valid : kSB);
    const uint64_t lb = reinterpret_cast<uint64_t>(lsrc + (b * a.Hq + h) * s + r0);
    const uint64_t lbu = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(lb >> 32)) << 32) |
                         (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)lb);
    const auto rl = __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<float*>(lbu), (short)0,
                                                      __builtin_amdgcn_readfirstlane((int)(nrec * 4)), kBufferFlags);
    if (lane < 16) lds_dma4(rl, ld + ldst, dmal);
  };
  // The unmasked stream of a head issues its sub-blocks in order, so the
  // scalar state below walks Q, dO and the record one sub-block per call
  // (no per-call index arithmetic).  Past the chunk end the byte counts drop
  // to zero and the DMA fills zeros.
  const int64_t sbb = (int64_t)kSB * qstride * 2;  // bytes per sub-block of Q or dO
  const int qrow_bytes = (int)(qstride * 2);
  uint64_t qa = 0, oa = 0, la = 0;
  int rem = 0;
  auto stream_begin = [&](int h) {
    const int64_t r0 = (int64_t)sb_u * kSB;
    const int64_t tile0 = (b * s + r0) * a.Hq + h;
    qa = uniform_u64(reinterpret_cast<uint64_t>(static_cast<const uint16_t*>(a.q) + tile0 * D));
    oa = uniform_u64(reinterpret_cast<uint64_t>(static_cast<const uint16_t*>(a.dout) + tile0 * D));
    la = uniform_u64(reinterpret_cast<uint64_t>(lsrc + (b * a.Hq + h) * s + r0));
    rem = (int)(s - r0);
  };
  auto stream_issue = [&](uint16_t* qd, uint16_t* od, float* ld) {
    const int n = rem <= 0 ? 0 : (rem < kSB ? rem : kSB);
    const auto rq = uniform_rsrc(qa, n * qrow_bytes);
    const auto ro = uniform_rsrc(oa, n * qrow_bytes);
#pragma unroll
    for (int x = 0; x < IPWQ; ++x) {
      lds_dma16(rq, qd + (w * IPWQ + x) * 512, dmaq[x]);
      lds_dma16(ro, od + (w * IPWQ + x) * 512, dmaq[x]);
    }
    const auto rl = uniform_rsrc(la, n * 4);
    if (lane < 16) lds_dma4(rl, ld + ldst, dmal);
    qa += sbb;
    oa += sbb;
    la += kSB * 4;
    rem -= kSB;
  };
  auto tr_rd = [&](const uint16_t* X, int hh, int db) {
    return ld_tr(X, tro[db][0] + 16 * hh * P, tro[db][1] + 16 * hh * P);
  };
  // -Delta of the 16 rows 8 (v/4) + 4 g + v%4 of a sub-block, from its record:
  // the initial value of its dP accumulator.
  auto ndelta = [&](const float* ld) {
    f32x16 x;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float4 t = *reinterpret_cast<const float4*>(ld + 32 + 8 * k + 4 * g);
      x[4 * k] = t.x;
      x[4 * k + 1] = t.y;
      x[4 * k + 2] = t.z;
      x[4 * k + 3] = t.w;
    }
    return x;
  };
  // S = Q K^T and dP - Delta = dO V^T - Delta of one sub-block (lane <-> key);
  // dp holds -Delta on entry.
  auto sdp = [&](const uint16_t* Qs, const uint16_t* Os, f32x16& sv, f32x16& dp) {
    sv = mfma32(ld_nat(Qs, nat[0]), kf[0], f32x16{});
    dp = mfma32(ld_nat(Os, nat[0]), vf[0], dp);
#pragma unroll
    for (int kk = 1; kk < NK; ++kk) {
      sv = mfma32(ld_nat(Qs, nat[kk]), kf[kk], sv);
      dp = mfma32(ld_nat(Os, nat[kk]), vf[kk], dp);
    }
  };
  // dV += P^T dO, dK += dS^T Q of one sub-block.
  auto grads = [&](const uint16_t* Qs, const uint16_t* Os, const bf16x8 (&pb)[2], const bf16x8 (&dsb)[2]) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
      for (int db = 0; db < ND; ++db) {
        dv[db] = mfma32(pb[hh], tr_rd(Os, hh, db), dv[db]);
        dk[db] = mfma32(dsb[hh], tr_rd(Qs, hh, db), dk[db]);
      }
    }
  };

  // Heads of the GQA group one after another, each in row order: the masked
  // sub-blocks one at a time, then the unmasked stream.  A key's dK/dV thus
  // sums its rows in the same order whatever range of keys a launch covers
  // (rows before a key add exact zeros).
  for (int hh = 0; hh < G; ++hh) {
    const int h = hk * G + hh;
    // ---- sub-blocks with the causal mask, one at a time (slot 0)
    for (int sb = sb_begin; sb < sb_u; ++sb) {
      __syncthreads();
      issue(h, sb, qbuf(IC<0>{}), obuf(IC<0>{}), lbuf(IC<0>{}));
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
      __syncthreads();
      const float* ld = lbuf(IC<0>{});
      f32x16 sv, dp = ndelta(ld);
      sdp(qbuf(IC<0>{}), obuf(IC<0>{}), sv, dp);
      const int64_t r0g = c0 + (int64_t)sb * kSB;  // global row of the sub-block's first row
      float p[16], ds[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int qi = 8 * (v / 4) + 4 * g + (v % 4);
        float pv = fast_exp2(sv[v] * C - ld[qi]);
        if (j > r0g + qi) pv = 0.f;  // key j sees row r iff j <= r
        p[v] = pv;
        ds[v] = pv * dp[v];
      }
      bf16x8 pb[2], dsb[2];
      pb[0] = pack_bf16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
      pb[1] = pack_bf16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
      dsb[0] = pack_bf16x8(ds[0], ds[1], ds[2], ds[3], ds[4], ds[5], ds[6], ds[7]);
      dsb[1] = pack_bf16x8(ds[8], ds[9], ds[10], ds[11], ds[12], ds[13], ds[14], ds[15]);
      grads(qbuf(IC<0>{}), obuf(IC<0>{}), pb, dsb);
    }

    // ---- unmasked stream, software pipelined
    if (N == 0) continue;
    __syncthreads();  // every slot is free
    stream_begin(h);
    stream_issue(qbuf(IC<0>{}), obuf(IC<0>{}), lbuf(IC<0>{}));
    stream_issue(qbuf(IC<1>{}), obuf(IC<1>{}), lbuf(IC<1>{}));
    stream_issue(qbuf(IC<2>{}), obuf(IC<2>{}), lbuf(IC<2>{}));
    stream_issue(qbuf(IC<3>{}), obuf(IC<3>{}), lbuf(IC<3>{}));
    stream_issue(qbuf(IC<4>{}), obuf(IC<4>{}), lbuf(IC<4>{}));
    // With kEarlyA, sub-blocks 0 and 1 land before the loop and step 0's
    // first natural operands are read here; later steps get theirs from the
    // end of the previous B phase.
    __builtin_amdgcn_s_waitcnt(waitcnt_vm((kAhead - (kEarlyA ? 2 : 1)) * DMA_PER_SB));
    __syncthreads();
    f32x16 sa, da = ndelta(lbuf(IC<0>{})), sb2, db2;
    sdp(qbuf(IC<0>{}), obuf(IC<0>{}), sa, da);
    bf16x8 opn[4];
    if (kEarlyA) {
#pragma unroll
      for (int m = 0; m < 4; ++m) opn[m] = ld_nat((m & 1) ? obuf(IC<1>{}) : qbuf(IC<1>{}), nat[m >> 1]);
      db2 = ndelta(lbuf(IC<1>{}));
    }
    // Step n in slot I: A(n) reads slot I+1 (natural) and slot I's record;
    // B(n) reads slot I (transposed) and, in its last MFMA slots, A(n+1)'s
    // first natural operands from slot I+2.  At its start sub-blocks n+1 and
    // n+2 have landed (only n+3, n+4 may still be loading); then sub-block
    // n+5 goes to slot I+5 = I-1, free since step n-1.  dnext holds -Delta of
    // sub-block n+1 on entry (read in B(n-1)); B(n) leaves -Delta of n+2 in
    // dcur, which is step n+1's dnext.
    auto step = [&](int n, auto sl, f32x16& scur, f32x16& dcur, f32x16& snext, f32x16& dnext) {
      constexpr int I = decltype(sl)::value;
      constexpr int I1 = (I + 1) % kRing, I2 = (I + 2) % kRing, I5 = (I + kAhead) % kRing;
      __builtin_amdgcn_s_waitcnt(waitcnt_vm((kAhead - (kEarlyA ? 3 : 2)) * DMA_PER_SB));
      __syncthreads();
      stream_issue(qbuf(IC<I5>{}), obuf(IC<I5>{}), lbuf(IC<I5>{}));
      const uint16_t* Qn = qbuf(IC<I1>{});
      const uint16_t* On = obuf(IC<I1>{});
      const uint16_t* Qc = qbuf(IC<I>{});
      const uint16_t* Oc = obuf(IC<I>{});
      const float* ld = lbuf(IC<I>{});
      if (!kEarlyA) dnext = ndelta(lbuf(IC<I1>{}));
      // A(n): MFMA m (NA of them) is S(n+1) (m even) or dP(n+1) (m odd),
      // k-step m/2; its operand is read four MFMAs ahead.  The VALU turns the
      // 16 elements of S(n), dP(n) into P(n), dS(n), element i beside MFMA
      // i / (16 / NA).
      constexpr int NA = 2 * NK, EPM = 16 / NA;
      auto nat_op = [&](int m) { return ld_nat((m & 1) ? On : Qn, nat[m >> 1]); };
      bf16x8 op[NA];
#pragma unroll
      for (int m = 0; m < 4; ++m) op[m] = kEarlyA ? opn[m] : nat_op(m);
      // LSE2 of rows 8 k + 4 g .. + 3 (group k of four elements), loaded
      // kLdAhead groups before its use.
      float4 lgk[4];
      auto ld_group = [&](int k) { lgk[k] = *reinterpret_cast<const float4*>(ld + 8 * k + 4 * g); };
#pragma unroll
      for (int k = 0; k <= kLdAhead && k < 4; ++k) ld_group(k);
      float p[16], ds[16];
      bf16x8 pb[2], dsb[2];
      // B(n): MFMA jj is dV (jj even) or dK (jj odd) for k-half hh, d-block
      // db; its transposed operand is read three slots ahead (the first
      // three in the last MFMA slots of A(n), which read nothing else).
      constexpr int NB = 4 * ND;
      auto tr_op = [&](int jj) {
        const int blk = jj >> 1;
        return tr_rd((jj & 1) ? Qc : Oc, blk / ND, blk % ND);
      };
      bf16x8 top[NB];
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if (i % EPM == 0) {
          const int mi = i / EPM;
          if (mi & 1) {
            dnext = mfma32(op[mi], vf[mi >> 1], dnext);
          } else {
            snext = mfma32(op[mi], kf[mi >> 1], mi == 0 ? f32x16{} : snext);
          }
          if (mi + 4 < NA) op[mi + 4] = nat_op(mi + 4);
          else if (kEarlyTr && mi + 4 - NA < 3) top[mi + 4 - NA] = tr_op(mi + 4 - NA);
        }
        const int e = i & 3;
        const float4 l4 = lgk[i >> 2];
        const float lv = e == 0 ? l4.x : e == 1 ? l4.y : e == 2 ? l4.z : l4.w;
        // Element i's exp, element i-1's dS: an exp's result is not read by the
        // next instruction (that would cost a wait state).
        p[i] = fast_exp2(scur[i] * C - lv);
        if (i > 0) ds[i - 1] = p[i - 1] * dcur[i - 1];
        if (e == 3 && i < 15) {  // rows 8 (v/4) + 4 g + v%4 of the next group of four
          if ((i >> 2) + kLdAhead + 1 < 4) ld_group((i >> 2) + kLdAhead + 1);
        }
        if (i == 8) {
          pb[0] = pack_bf16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
          dsb[0] = pack_bf16x8(ds[0], ds[1], ds[2], ds[3], ds[4], ds[5], ds[6], ds[7]);
        }
        if (i % EPM == EPM - 1) __builtin_amdgcn_sched_barrier(0);
      }
      ds[15] = p[15] * dcur[15];
      pb[1] = pack_bf16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
      dsb[1] = pack_bf16x8(ds[8], ds[9], ds[10], ds[11], ds[12], ds[13], ds[14], ds[15]);
      if (!kEarlyTr) {
        top[0] = tr_op(0);
        top[1] = tr_op(1);
        top[2] = tr_op(2);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int jj = 0; jj < NB; ++jj) {
        const int blk = jj >> 1, hh = blk / ND, db = blk % ND;
        if (jj & 1) {
          dk[db] = mfma32(dsb[hh], top[jj], dk[db]);
        } else {
          dv[db] = mfma32(pb[hh], top[jj], dv[db]);
        }
        if (jj + 3 < NB) {
          top[jj + 3] = tr_op(jj + 3);
        } else if (kEarlyA) {  // A(n+1)'s first natural operands and -Delta, from sub-block n+2
          const int m0 = jj + 3 - NB;
          opn[m0] = ld_nat((m0 & 1) ? obuf(IC<I2>{}) : qbuf(IC<I2>{}), nat[m0 >> 1]);
          if (m0 == 2) {
            opn[3] = ld_nat(obuf(IC<I2>{}), nat[1]);
            dcur = ndelta(lbuf(IC<I2>{}));
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    // Past the last sub-block A still computes S, dP of the (zero) next slot;
    // they are never used.
    for (int n = 0; n < N; n += kRing) {
      step(n, IC<0>{}, sa, da, sb2, db2);
      if (n + 1 >= N) break;
      step(n + 1, IC<1>{}, sb2, db2, sa, da);
      if (n + 2 >= N) break;
      step(n + 2, IC<2>{}, sa, da, sb2, db2);
      if (n + 3 >= N) break;
      step(n + 3, IC<3>{}, sb2, db2, sa, da);
      if (n + 4 >= N) break;
      step(n + 4, IC<4>{}, sa, da, sb2, db2);
      if (n + 5 >= N) break;
      step(n + 5, IC<5>{}, sb2, db2, sa, da);
    }
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // no LDS-DMA in flight past the stream
  }

  // Write back rows [k0, k0+128) n [kv0, kv1): lane <-> d, v <-> key.  In
  // accumulate mode the 32 old values of a d-block are loaded before any of
  // them is stored (dK and dV are distinct buffers, which the C ABI checks),
  // so the loads share one memory round trip instead of one each (the sum
  // is old + dK * scale in one fused multiply-add).  A block
  // whose 128 keys are all in range (every one but a ragged last) takes a
  // branch-free path: key v of the lane sits a compile-time number of rows
  // past the lane's first key.
  float* __restrict__ gdk = a.dk;
  float* __restrict__ gdv = a.dv;
  const int64_t rs = (int64_t)a.Hkv * D;  // elements between consecutive keys
  const int64_t key0 = k0 + 32 * w + 4 * g;
  const int64_t base = ((b * a.S + key0) * a.Hkv + hk) * D + l32;
  auto koff = [](int v) { return 8 * (v / 4) + (v % 4); };
  if (k0 + 128 <= kv1) {
#pragma unroll
    for (int db = 0; db < ND; ++db) {
      float* pk = gdk + base + 32 * db;
      float* pv = gdv + base + 32 * db;
      float ok[16], ov[16];
      if (a.accumulate) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          ok[v] = pk[koff(v) * rs];
          ov[v] = pv[koff(v) * rs];
        }
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        pk[koff(v) * rs] = a.accumulate ? __builtin_fmaf(dk[db][v], a.scale, ok[v]) : dk[db][v] * a.scale;
        pv[koff(v) * rs] = a.accumulate ? ov[v] + dv[db][v] : dv[db][v];
      }
    }
  } else {
#pragma unroll
    for (int db = 0; db < ND; ++db) {
      float ok[16], ov[16];
      if (a.accumulate) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int64_t idx = base + koff(v) * rs + 32 * db;
          ok[v] = key0 + koff(v) < kv1 ? gdk[idx] : 0.f;
          ov[v] = key0 + koff(v) < kv1 ? gdv[idx] : 0.f;
        }
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        if (key0 + koff(v) < kv1) {
          const int64_t idx = base + koff(v) * rs + 32 * db;
          gdk[idx] = a.accumulate ? __builtin_fmaf(dk[db][v], a.scale, ok[v]) : dk[db][v] * a.scale;
          gdv[idx] = a.accumulate ? ov[v] + dv[db][v] : dv[db][v];
        }
      }
    }
  }
  __syncthreads();  // every wave is past s_tile and the ring before the next tile
  }
  // The last workgroup out resets the queues for the next launch (every
  // other one has taken its last tile before it counts itself out).
  if (tid == 0) {
    __threadfence();
    if (atomicAdd(a.tiles + 8, 1) == (int)gridDim.x - 1) {
      for (int x = 0; x < 9; ++x) atomicExch(a.tiles + x, 0);
    }
  }
}

// --------------------------------------------------------------------- dQ
template <int D>
__global__ __launch_bounds__(256, 1) void bwd_dq_bf16_kernel(ChunkArgs a) {
  using T = XTile<D>;
  constexpr int P = T::P, NK = D / 16, ND = D / 32;
  constexpr int IPWK = (kSB / T::RPI) / 4;  // DMA instructions per wave per tensor per sub-block
  static_assert(IPWK >= 1 && IPWK * 4 * T::RPI == kSB, "sub-block splits over 4 waves");
  constexpr int DMA_PER_SB = 2 * IPWK;
  // One LDS object per ring slot: [K rows | V rows].
  constexpr int SLOT = 2 * kSB * P;
  __shared__ __attribute__((aligned(1024))) uint16_t R0[SLOT], R1[SLOT], R2[SLOT], R3[SLOT], R4[SLOT], R5[SLOT];
  auto slot = [&](auto I) -> uint16_t* {
    constexpr int i = decltype(I)::value;
    if constexpr (i == 0) return R0; else if constexpr (i == 1) return R1; else if constexpr (i == 2) return R2;
    else if constexpr (i == 3) return R3; else if constexpr (i == 4) return R4; else return R5;
  };
  auto slot_rt = [&](int i) -> uint16_t* {
    return i == 0 ? R0 : i == 1 ? R1 : i == 2 ? R2 : i == 3 ? R3 : i == 4 ? R4 : R5;
  };

  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  const GridPos gp = xcd_grouped();  // the query tiles of a head behind one L2
  const int t = gridDim.x - 1 - gp.x;  // longest (latest) query tiles first
  const int h = gp.y;
  const int64_t b = gp.z;
  const int hk = h / (a.Hq / a.Hkv);
  const int64_t c0 = a.c0, c1 = a.c1, s = c1 - c0;
  const int64_t q0 = c0 + (int64_t)t * kDqRows;
  const int64_t r = q0 + 32 * w + l32;
  const bool rvalid = r < c1;
  const int64_t kend = (q0 + kDqRows < c1) ? q0 + kDqRows : c1;
  const int nsub = (int)((kend + kSB - 1) / kSB);
  const int N = (int)(q0 / kSB);  // key sub-blocks every row of the workgroup sees in full
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
  int dmak[IPWK];
#pragma unroll
  for (int x = 0; x < IPWK; ++x) dmak[x] = T::dma(lane, w * IPWK + x, kvstride);
  const uint16_t* kbase = static_cast<const uint16_t*>(a.k) + (b * a.S * a.Hkv + hk) * D;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v) + (b * a.S * a.Hkv + hk) * D;

  bf16x8 qf[NK], df[NK];
  float lse2 = INFINITY, ndl = 0.f;  // a padding row gets P = 0
  if (rvalid) {
    const int64_t off = ((b * s + (r - c0)) * a.Hq + h) * D;
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) + off;
    const uint16_t* drow = static_cast<const uint16_t*>(a.dout) + off;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      qf[kk] = as_bf16x8(ld_global16(qrow + 16 * kk + 8 * g));
      df[kk] = as_bf16x8(ld_global16(drow + 16 * kk + 8 * g));
    }
    lse2 = a.lse2[(b * a.Hq + h) * s + (r - c0)];
    ndl = a.delta[(b * a.Hq + h) * s + (r - c0)];
  } else {
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) qf[kk] = df[kk] = bf16x8{};
  }
  f32x16 dq[ND];
#pragma unroll
  for (int db = 0; db < ND; ++db) dq[db] = f32x16{};
  // -Delta of the lane's row in every element: the initial value of each dP^T
  // accumulator, so the MFMAs produce dP^T - Delta.
  f32x16 ninit;
#pragma unroll
  for (int v = 0; v < 16; ++v) ninit[v] = ndl;

  // DMA of K/V sub-block u (keys [32u, 32u+32)) into a slot; keys past the
  // chunk end load zeros, so every call issues DMA_PER_SB instructions.
  // Sub-blocks are issued in key order, so scalar state walks K and V one
  // sub-block per call.
  const int64_t sbb = (int64_t)kSB * kvstride * 2;  // bytes per sub-block of K or V
  const int krow_bytes = (int)(kvstride * 2);
  uint64_t ka = uniform_u64(reinterpret_cast<uint64_t>(kbase)), va = uniform_u64(reinterpret_cast<uint64_t>(vbase));
  int remk = (int)c1;  // keys [k0, c1) are valid
  auto issue_next = [&](uint16_t* dst) {
    const int n = remk <= 0 ? 0 : (remk < kSB ? remk : kSB);
    const auto rk = uniform_rsrc(ka, n * krow_bytes);
    const auto rv = uniform_rsrc(va, n * krow_bytes);
#pragma unroll
    for (int x = 0; x < IPWK; ++x) {
      lds_dma16(rk, dst + (w * IPWK + x) * 512, dmak[x]);
      lds_dma16(rv, dst + kSB * P + (w * IPWK + x) * 512, dmak[x]);
    }
    ka += sbb;
    va += sbb;
    remk -= kSB;
  };
  auto tr_rd = [&](const uint16_t* X, int hh, int db) {
    return ld_tr(X, tro[db][0] + 16 * hh * P, tro[db][1] + 16 * hh * P);
  };
  // S^T = K Q^T and dP^T - Delta = V dO^T - Delta of one sub-block (lane <-> query).
  auto sdp = [&](const uint16_t* K, f32x16& sv, f32x16& dp) {
    const uint16_t* V = K + kSB * P;
    sv = mfma32(ld_nat(K, nat[0]), qf[0], f32x16{});
    dp = mfma32(ld_nat(V, nat[0]), df[0], ninit);
#pragma unroll
    for (int kk = 1; kk < NK; ++kk) {
      sv = mfma32(ld_nat(K, nat[kk]), qf[kk], sv);
      dp = mfma32(ld_nat(V, nat[kk]), df[kk], dp);
    }
  };

  // Prologue: sub-blocks 0..4 (which also covers every diagonal sub-block
  // when N is 0).
  issue_next(R0);
  issue_next(R1);
  issue_next(R2);
  issue_next(R3);
  issue_next(R4);

  if (N > 0) {
    __builtin_amdgcn_s_waitcnt(waitcnt_vm((kAhead - (kEarlyAq ? 2 : 1)) * DMA_PER_SB));
    __syncthreads();
    f32x16 sa, da, sb2, db2;
    sdp(R0, sa, da);
    bf16x8 opn[4];
    if (kEarlyAq) {
#pragma unroll
      for (int m = 0; m < 4; ++m) opn[m] = ld_nat((m & 1) ? R1 + kSB * P : R1, nat[m >> 1]);
    }
    // Step n in slot I: A(n) reads slot I+1 (natural K, V); B(n) reads slot I
    // (transposed K) and, in its last MFMA slots, A(n+1)'s first natural
    // operands from slot I+2.  At its start sub-blocks n+1 and n+2 have
    // landed; then sub-block n+5 goes to slot I+5 = I-1, free since step n-1.
    auto step = [&](int n, auto sl, f32x16& scur, f32x16& dcur, f32x16& snext, f32x16& dnext) {
      constexpr int I = decltype(sl)::value;
      constexpr int I1 = (I + 1) % kRing, I2 = (I + 2) % kRing, I5 = (I + kAhead) % kRing;
      __builtin_amdgcn_s_waitcnt(waitcnt_vm((kAhead - (kEarlyAq ? 3 : 2)) * DMA_PER_SB));
      __syncthreads();
      issue_next(slot(IC<I5>{}));  // sub-block n + kAhead
      const uint16_t* Kn = slot(IC<I1>{});
      const uint16_t* Vn = Kn + kSB * P;
      const uint16_t* Kc = slot(IC<I>{});
      // A(n): MFMA m (NA of them) is S^T(n+1) (m even) or dP^T(n+1) (m odd),
      // k-step m/2; its operand is read four MFMAs ahead.  The VALU turns the
      // 16 elements of S^T(n), dP^T(n) into dS^T(n), element i beside MFMA
      // i / (16 / NA).
      constexpr int NA = 2 * NK, EPM = 16 / NA;
      auto nat_op = [&](int m) { return ld_nat((m & 1) ? Vn : Kn, nat[m >> 1]); };
      bf16x8 op[NA];
#pragma unroll
      for (int m = 0; m < 4; ++m) op[m] = kEarlyAq ? opn[m] : nat_op(m);
      float pv[16], ds[16];
      bf16x8 dsb[2];
      // B(n): MFMA jj is dQ^T d-block jj % ND for k-half jj / ND; its
      // transposed K operand is read three slots ahead (the first three in
      // the last MFMA slots of A(n)).
      constexpr int NB = 2 * ND;
      auto tr_op = [&](int jj) { return tr_rd(Kc, jj / ND, jj % ND); };
      bf16x8 top[NB];
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if (i % EPM == 0) {
          const int mi = i / EPM;
          if (mi & 1) {
            dnext = mfma32(op[mi], df[mi >> 1], mi == 1 ? ninit : dnext);
          } else {
            snext = mfma32(op[mi], qf[mi >> 1], mi == 0 ? f32x16{} : snext);
          }
          if (mi + 4 < NA) op[mi + 4] = nat_op(mi + 4);
          else if (kEarlyTr && mi + 4 - NA < 3) top[mi + 4 - NA] = tr_op(mi + 4 - NA);
        }
        // Element i's exp, element i-1's dS (no exp result read right away).
        pv[i] = fast_exp2(scur[i] * C - lse2);
        if (i > 0) ds[i - 1] = pv[i - 1] * dcur[i - 1];
        if (i == 8) dsb[0] = pack_bf16x8(ds[0], ds[1], ds[2], ds[3], ds[4], ds[5], ds[6], ds[7]);
        if (i % EPM == EPM - 1) __builtin_amdgcn_sched_barrier(0);
      }
      ds[15] = pv[15] * dcur[15];
      dsb[1] = pack_bf16x8(ds[8], ds[9], ds[10], ds[11], ds[12], ds[13], ds[14], ds[15]);
      if (!kEarlyTr) {
        top[0] = tr_op(0);
        top[1] = tr_op(1);
        top[2] = tr_op(2);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int jj = 0; jj < NB; ++jj) {
        dq[jj % ND] = mfma32(top[jj], dsb[jj / ND], dq[jj % ND]);
        if (jj + 3 < NB) {
          top[jj + 3] = tr_op(jj + 3);
        } else if (kEarlyAq) {  // A(n+1)'s first natural operands, from sub-block n+2
          const uint16_t* K2 = slot(IC<I2>{});
          const int m0 = jj + 3 - NB;
          opn[m0] = ld_nat((m0 & 1) ? K2 + kSB * P : K2, nat[m0 >> 1]);
          if (m0 == 2) opn[3] = ld_nat(K2 + kSB * P, nat[1]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    for (int n = 0; n < N; n += kRing) {
      step(n, IC<0>{}, sa, da, sb2, db2);
      if (n + 1 >= N) break;
      step(n + 1, IC<1>{}, sb2, db2, sa, da);
      if (n + 2 >= N) break;
      step(n + 2, IC<2>{}, sa, da, sb2, db2);
      if (n + 3 >= N) break;
      step(n + 3, IC<3>{}, sb2, db2, sa, da);
      if (n + 4 >= N) break;
      step(n + 4, IC<4>{}, sa, da, sb2, db2);
      if (n + 5 >= N) break;
      step(n + 5, IC<5>{}, sb2, db2, sa, da);
    }
  }

  // Diagonal sub-blocks [N, nsub) (at most five): already in the ring, since
  // the steady loop loaded five ahead and the prologue covers N = 0.
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  __syncthreads();
  for (int u = N; u < nsub; ++u) {
    const uint16_t* K = slot_rt(u % kRing);
    f32x16 sv, dp;
    sdp(K, sv, dp);
    const int rel = (int)(r - (int64_t)u * kSB);  // keys past this row are masked
    float ds[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float p = fast_exp2(sv[v] * C - lse2);
      if (8 * (v / 4) + 4 * g + (v % 4) > rel) p = 0.f;
      ds[v] = p * dp[v];
    }
    bf16x8 dsb[2];
    dsb[0] = pack_bf16x8(ds[0], ds[1], ds[2], ds[3], ds[4], ds[5], ds[6], ds[7]);
    dsb[1] = pack_bf16x8(ds[8], ds[9], ds[10], ds[11], ds[12], ds[13], ds[14], ds[15]);
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
      for (int db = 0; db < ND; ++db) dq[db] = mfma32(tr_rd(K, hh, db), dsb[hh], dq[db]);
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

}  // namespace

hipError_t launch_bwd_pre_bf16(const ChunkArgs& a, hipStream_t stream) {
  if (!a.tiles) return hipErrorInvalidValue;
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

// Workgroups of the persistent dK/dV kernel that one CU holds at once (its
// registers allow one; asked of the runtime once per head size).
template <int D>
int dkdv_groups_per_cu() {
  static const int n = [] {
    int b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, reinterpret_cast<const void*>(&bwd_dkdv_bf16_kernel<D>),
                                                     256, 0) != hipSuccess || b < 1) {
      b = 1;
    }
    return b;
  }();
  return n;
}

hipError_t launch_bwd_dkdv_bf16(const ChunkArgs& a, hipStream_t stream) {
  if (a.kv0 < 0 || a.kv1 > a.c1 || a.kv0 >= a.kv1 || !a.tiles || a.n_cu < 1) return hipErrorInvalidValue;
  if (a.D != 128 && a.D != 64) return hipErrorInvalidValue;
  const int64_t tiles = (a.kv1 - a.kv0 + kKvKeys - 1) / kKvKeys * a.Hkv * a.B;
  if (tiles > 0x7fffffff) return hipErrorInvalidValue;
  // persistent: as many workgroups as the CUs hold at once
  const int64_t slots = (int64_t)a.n_cu * (a.D == 128 ? dkdv_groups_per_cu<128>() : dkdv_groups_per_cu<64>());
  dim3 grid((unsigned)(tiles < slots ? tiles : slots));
  if (a.D == 128) {
    hipLaunchKernelGGL(bwd_dkdv_bf16_kernel<128>, grid, dim3(256), 0, stream, a);
  } else {
    hipLaunchKernelGGL(bwd_dkdv_bf16_kernel<64>, grid, dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dq_bf16(const ChunkArgs& a, hipStream_t stream) {
  const int64_t s = a.c1 - a.c0;
  dim3 grid((unsigned)((s + kDqRows - 1) / kDqRows), (unsigned)a.Hq, (unsigned)a.B);
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
