// Internal launch interface between the C-ABI host code (sppo.cpp) and the
// gfx950 kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

namespace sppo {

// Message returned by sppo_last_error(NULL) on this thread: the failure of
// the last context-free call (or of sppo_create).
void set_thread_error(const std::string& msg);

// Arguments of one chunk's attention kernels.  Chunk-local tensors (q, o,
// dout, dq, lse) hold rows [c0, c1) only; k/v/dk/dv are full-length.
struct ChunkArgs {
  const void* q;       // [B, s, Hq, D]
  const void* k;       // [B, S, Hkv, D]
  const void* v;       // [B, S, Hkv, D]
  void* o;             // [B, s, Hq, D]  (fwd output / bwd input)
  float* lse;          // [B, Hq, s]     (fwd output / bwd input)
  const void* dout;    // [B, s, Hq, D]
  void* dq;            // [B, s, Hq, D]
  float* dk;           // [B, S, Hkv, D] fp32 accumulator
  float* dv;           // [B, S, Hkv, D] fp32 accumulator
  float* delta;        // [B, Hq, s]     workspace: <dO_r, O_r> (fp32 kernels) or its negation (bf16)
  float* lse2;         // [B, Hq, s]     workspace: LSE * log2(e) (bf16 backward)
  int64_t B, S, c0, c1;
  int Hq, Hkv, D;
  float scale;
  int accumulate;      // dk/dv: 0 = overwrite rows [kv0, kv1), 1 = add
  int64_t kv0, kv1;    // dkdv: key rows computed, a sub-range of [0, c1)
  int* tiles;          // bf16 dkdv: tile queues, kTileQueueInts ints, zero between launches
  int n_cu;            // compute units of the device (bf16 dkdv: one workgroup each)
};

// The bf16 dK/dV kernel takes its key tiles from one queue per XCD (a
// counter each, [0, 8)) and counts its finished workgroups ([8]); the last
// one resets all nine, so every launch on a stream starts from zero.
constexpr int kTileQueueInts = 16;

// Each launcher enqueues one kernel on `stream` and returns the launch
// status.  The backward of a chunk is pre (Delta), then dkdv (one launch for
// key rows [kv0, kv1); several launches over disjoint ranges give the same
// result), then dq.
hipError_t launch_fwd_bf16(const ChunkArgs& a, hipStream_t stream);
hipError_t launch_bwd_pre_bf16(const ChunkArgs& a, hipStream_t stream);
hipError_t launch_bwd_dkdv_bf16(const ChunkArgs& a, hipStream_t stream);
hipError_t launch_bwd_dq_bf16(const ChunkArgs& a, hipStream_t stream);
hipError_t launch_fwd_f32(const ChunkArgs& a, hipStream_t stream);
hipError_t launch_bwd_pre_f32(const ChunkArgs& a, hipStream_t stream);
hipError_t launch_bwd_dkdv_f32(const ChunkArgs& a, hipStream_t stream);
hipError_t launch_bwd_dq_f32(const ChunkArgs& a, hipStream_t stream);

// Rounding of finished dK/dV rows: out_k/out_v rows [row0, row0 + rows) of
// every batch entry = dk/dv rows (fp32 [B, S, W], W = Hkv * D, W % 8 == 0),
// as bf16 (round to nearest even) when bf16 != 0, else copied as fp32.
// out_k/out_v have the accumulators' [B, S, W] layout; 16-byte aligned.
struct FinalizeArgs {
  const float* dk;
  const float* dv;
  void* out_k;
  void* out_v;
  int64_t B, S, W, row0, rows;
  int bf16;
};
hipError_t launch_finalize(const FinalizeArgs& a, hipStream_t stream);

// `height` rows of `width` bytes from src (row pitch spitch) to dst (dpitch),
// device to device, as a kernel on `stream`.  Widths, pitches and pointers
// must be multiples of 4 bytes (hipErrorInvalidValue otherwise).
hipError_t launch_copy_rows(void* dst, size_t dpitch, const void* src, size_t spitch, size_t width, size_t height,
                            hipStream_t stream);

// Dense bf16 GEMM (fp32 accumulation), C[M, N] (op)= sum_k A(m, k) B(k, n).
//   tn = 0 (NT): a is [M, K] (row stride lda), b is [N, K] (ldb); K % 64 == 0.
//   tn = 1 (TN): a is stored [K, M], b is stored [K, N]; M % 256 == 0 and
//                N % 256 == 0.
// Rows past M (NT) or K (TN) read as zero; only C[m < M][n < N] is written.
// Every pointer 16-byte aligned, every leading dimension a multiple of 8.
enum GemmEpi {
  kEpiBf16 = 0,     // C bf16 = acc
  kEpiAddBf16 = 1,  // C bf16 = acc + aux (bf16 [M, N], ldaux): residual
  kEpiGelu = 2,     // aux bf16 = acc (pre-activation, kept); C bf16 = gelu(bf16(acc))
  kEpiDGelu = 3,    // C bf16 = acc * gelu'(aux) (aux: the kept pre-activation)
  kEpiAccF32 = 4,   // C fp32 += acc
  kEpiF32 = 5       // C fp32 = acc
};
struct GemmArgs {
  int64_t M, N, K;
  const uint16_t* a;
  int64_t lda;
  const uint16_t* b;
  int64_t ldb;
  void* c;
  int64_t ldc;
  void* aux;
  int64_t ldaux;
  int epi;
  int tn;
};
hipError_t launch_gemm_bf16(const GemmArgs& g, hipStream_t stream);

// LayerNorm over rows of H (H % 8 == 0, H <= 8192), bf16 activations, fp32
// parameters and statistics.  Forward: y, mean, rstd.  Backward: y = dx =
// dres + LN'(dy), and dgamma/dbeta (+)= the column sums (deterministic: rows
// in blocks of rows_per_block, partial sums in part [nblocks, 2H], then
// added in block order).
struct LnArgs {
  int64_t rows;
  int H;
  const uint16_t* x;
  int64_t ldx;
  uint16_t* y;
  int64_t ldy;
  const float* gamma;
  const float* beta;
  float* mean;
  float* rstd;
  float eps;
  const uint16_t* dy;
  int64_t lddy;
  const uint16_t* dres;
  int64_t lddres;
  float* dgamma;
  float* dbeta;
  float* part;
  int rows_per_block;
  int nblocks;
  int accumulate;  // bwd: dgamma/dbeta += (1) or = (0) the column sums
};
hipError_t launch_ln_fwd(const LnArgs& a, hipStream_t stream);
hipError_t launch_ln_bwd(const LnArgs& a, hipStream_t stream);
hipError_t launch_gelu(const uint16_t* x, uint16_t* y, int64_t n, hipStream_t stream);
hipError_t launch_transpose(const uint16_t* in, uint16_t* out, int64_t R, int64_t C, hipStream_t stream);

// Rows t < rows of out [rows, wq + 2 wkv] = [dq[t] | bf16(dk[c + t]) |
// bf16(dv[c + t])] (dq bf16 [rows, wq]; dk, dv fp32 [.., wkv]).
struct PackArgs {
  int64_t rows;
  int wq, wkv;
  const uint16_t* dq;
  const float* dk;
  const float* dv;
  int64_t c;
  uint16_t* out;
};
hipError_t launch_pack_dqkv(const PackArgs& a, hipStream_t stream);

}  // namespace sppo
