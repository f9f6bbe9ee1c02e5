// Device-side helpers shared by the gfx950 attention kernels: vector types,
// the bf16 MFMA wrapper, global->register tile loads, and the swizzled LDS
// tile layout with its natural and transposed operand reads.
//
// MFMA register layout used throughout (v_mfma_f32_32x32x16_bf16, wave64):
//   A[i][k] : lane l holds row i = l%32 and 8 k-values in "k-slots"
//   B[k][j] : lane l holds col j = l%32 and 8 k-values in the same k-slots
//   C[i][j] : lane l holds col j = l%32, rows i = 8*(v/4) + 4*(l/32) + v%4,
//             v = 0..15
// Only consistency between the A and B k-slots matters for a product, so
// each kernel picks the k-slot -> k map that lets it feed one MFMA's C
// registers straight into the next MFMA: for a 16-wide k-block kb, slot e of
// lane-half g = l/32 holds k = 16*kb + 8*(e/4) + 4*g + e%4, which is exactly
// where rows 16*kb.. of a C tile live (v = 8*(kb%2) + e).  A natural-layout
// operand (k contiguous in memory, e.g. the head dim) uses the plain map
// k = 16*kk + 8*g + e instead.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sppo {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) short v4i16;
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& x) { return __builtin_bit_cast(bf16x8, x); }

__device__ __forceinline__ u32x4 ld_global16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

// Round 8 floats to bf16 (round-to-nearest-even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16x8 pack_bf16x8(float x0, float x1, float x2, float x3, float x4,
                                              float x5, float x6, float x7) {
  bf16x8 r;
  r[0] = (__bf16)x0; r[1] = (__bf16)x1; r[2] = (__bf16)x2; r[3] = (__bf16)x3;
  r[4] = (__bf16)x4; r[5] = (__bf16)x5; r[6] = (__bf16)x6; r[7] = (__bf16)x7;
  return r;
}

// Four fp32 values rounded to bf16 as two packed dwords.
__device__ __forceinline__ u32x2 pack_bf16x4(float x0, float x1, float x2, float x3) {
  bf16x2 lo, hi;
  lo.x = (__bf16)x0; lo.y = (__bf16)x1;
  hi.x = (__bf16)x2; hi.y = (__bf16)x3;
  return u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ float xor32(float x) { return __shfl_xor(x, 32); }

// ------------------------------------------------------ global tile loads
// A 4-row x 8-column bf16 block held by one thread as four 16-byte words.
struct Block4x8 {
  u32x4 r[4];
};

// Blocks are loaded through a buffer resource based at the first row of a
// tile: the hardware range check returns zero for every byte offset at or
// past num_records, so rows >= valid_rows read as zero with no per-lane test,
// and the per-lane byte offsets stay the same from tile to tile (only the
// scalar base moves).  Offsets are relative to the tile base, so they fit in
// 32 bits whatever the tensor size.
constexpr int kBufferFlags = 0x00020000;  // dword 3 of a raw gfx9 buffer resource

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint16_t* tile_base, int64_t valid_rows,
                                                            int tile_rows, int64_t row_stride) {
  const int64_t n = valid_rows <= 0 ? 0 : (valid_rows < tile_rows ? valid_rows : tile_rows);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(tile_base), (short)0,
                                           (int)(n * row_stride * (int64_t)sizeof(uint16_t)), kBufferFlags);
}

// Byte offsets of rows 4*rg + x, columns 8*cg.. of a tile with the given row
// stride (elements).
struct Block4x8Offsets {
  int b[4];
};
__device__ __forceinline__ Block4x8Offsets block4x8_offsets(int rg, int cg, int64_t row_stride) {
  Block4x8Offsets o;
#pragma unroll
  for (int x = 0; x < 4; ++x) o.b[x] = (int)(((4 * rg + x) * row_stride + 8 * cg) * (int64_t)sizeof(uint16_t));
  return o;
}

__device__ __forceinline__ void load_block4x8(Block4x8& blk, __amdgpu_buffer_rsrc_t rsrc, const Block4x8Offsets& off) {
#pragma unroll
  for (int x = 0; x < 4; ++x) blk.r[x] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off.b[x], 0, 0);
}

// ---------------------------------------------------------------- LDS tiles
// A bf16 tile [rows][D] in LDS is stored in natural layout (row = key or
// query, column = head dim) with row pitch D + 32 elements, and the 16-byte
// chunk index c of row r stored at c ^ ((r >> 2) & 3).  The gfx950 LDS has 64
// four-byte banks; a ds_read_b128 is served 16 lanes at a time, a
// ds_read_b64 / ds_read_b64_tr_b16 32 lanes at a time, and a ds_write_b128 8
// lanes at a time.  With this layout every group touches 64 distinct banks
// (or fewer, disjoint) for the three access patterns used here:
//   * natural operand reads: 16 consecutive rows, one chunk each -- the
//     pitch puts rows r and r+1 4 chunks apart (mod 16) and the swizzle
//     separates r and r+4;
//   * transposed reads: 4 rows x 4 chunks per 32 lanes, each row's 4 chunks
//     a distinct quarter of the 256-byte bank window;
//   * 4x8-block stores: 8 chunks of one row.
// The swizzle only touches the two low bits of the chunk index, so every
// access is a per-lane base (one per parity of the k-step for natural reads,
// one per 8-row half for transposed reads) plus an immediate offset.
template <int D>
struct LdsTile {
  static constexpr int P = D + 32;
  static constexpr int CG = D / 8;  // 16-byte chunks per row
  static __device__ __forceinline__ int swz(int row) { return (row >> 2) & 3; }
  // Element offset of row 4*rg + x, 16-byte chunk cg.
  static __device__ __forceinline__ int store_off(int rg, int x, int cg) {
    return (4 * rg + x) * P + 8 * (cg ^ (rg & 3));
  }
  // Lane bases of natural operand reads: row l%32, chunk 2*kk + l/32, for
  // even and odd k-steps kk (add rb*P + 32*(kk/2) for row block rb, rb % 32
  // == 0).
  struct Nat {
    int b[2];
  };
  static __device__ __forceinline__ Nat nat_base(int lane) {
    const int l32 = lane & 31, g = lane >> 5, s = swz(l32);
    return Nat{{l32 * P + 8 * (g ^ s), l32 * P + 8 * ((2 + g) ^ s)}};
  }
  // Lane bases of a transposed read of rows k0..k0+7 (b[0]) and
  // k0+8..k0+15 (b[1]); add k0*P (+8*P for b[1]) + x0 with k0 % 16 == 0 and
  // x0 % 32 == 0.  Source lane s = 16q + 4e + a supplies the 8 bytes at row
  // 4*(q/2) + e, column 16*(q%2) + 4*a; ds_read_b64_tr_b16 hands output lane
  // 16q + 4a' + b element b of source lanes 16q + 4e + a', e = 0..3.
  struct Tr {
    int b[2];
  };
  static __device__ __forceinline__ Tr tr_base(int lane) {
    const int q = lane >> 4, e = (lane >> 2) & 3, a = lane & 3;
    const int row = 4 * (q >> 1) + e, c = 2 * (q & 1) + (a >> 1);
    return Tr{{row * P + 8 * (c ^ (q >> 1)) + 4 * (a & 1), row * P + 8 * (c ^ ((q >> 1) + 2)) + 4 * (a & 1)}};
  }
};

template <int D>
__device__ __forceinline__ void store_block_tile(const Block4x8& blk, uint16_t* tile, int rg, int cg) {
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    *reinterpret_cast<u32x4*>(tile + LdsTile<D>::store_off(rg, x, cg)) = blk.r[x];
  }
}

// Natural operand: lane l gets row rb + l%32, columns 16*kk + 8*(l/32) + 0..7.
template <int D>
__device__ __forceinline__ bf16x8 ld_lds_nat(const uint16_t* tile, const typename LdsTile<D>::Nat& nat, int rb,
                                             int kk) {
  return as_bf16x8(*reinterpret_cast<const u32x4*>(tile + nat.b[kk & 1] + rb * LdsTile<D>::P + 32 * (kk >> 1)));
}

__device__ __forceinline__ v4i16 ds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p));
}

// Transposed operand from a natural tile: lane l gets column x0 + l%32 and
// rows k0 + {8*(e/4) + 4*(l/32) + e%4 : e = 0..7}, i.e. the permuted k-slot
// map, so it pairs with an operand taken from C-tile registers.
template <int D>
__device__ __forceinline__ bf16x8 ld_lds_tr(const uint16_t* tile, const typename LdsTile<D>::Tr& tr, int k0, int x0) {
  constexpr int P = LdsTile<D>::P;
  const v4i16 lo = ds_read_tr16(tile + tr.b[0] + k0 * P + x0);
  const v4i16 hi = ds_read_tr16(tile + tr.b[1] + (k0 + 8) * P + x0);
  const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
  const u32x4 r = {l2.x, l2.y, h2.x, h2.y};
  return as_bf16x8(r);
}

}  // namespace sppo
