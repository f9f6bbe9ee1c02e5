// Internal launch interface between the C-ABI host code (sppo.cpp) and the
// gfx950 kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sppo {

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
  float* delta;        // [B, Hq, s]     workspace: <dO_r, O_r>
  float* lse2;         // [B, Hq, s]     workspace: LSE * log2(e) (bf16 backward)
  int64_t B, S, c0, c1;
  int Hq, Hkv, D;
  float scale;
  int accumulate;      // dk/dv: 0 = overwrite rows [kv0, kv1), 1 = add
  int64_t kv0, kv1;    // dkdv: key rows computed, a sub-range of [0, c1)
};

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

}  // namespace sppo
