// Device-side helpers shared by the gfx950 attention kernels: vector types,
// bf16 MFMA wrappers, global->register tile loads and register->LDS stores in
// natural ([row][col]) and transposed ([col][row]) layouts.
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

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& x) { return __builtin_bit_cast(bf16x8, x); }

__device__ __forceinline__ u32x4 ld_global16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

__device__ __forceinline__ bf16x8 ld_lds16(const uint16_t* p) {
  return as_bf16x8(*reinterpret_cast<const u32x4*>(p));
}

// Two 8-byte LDS reads (k-slots 0..3 at p, 4..7 at p+8 elements) of a
// transposed tile: the permuted k-slot map described above.
__device__ __forceinline__ bf16x8 ld_lds_perm(const uint16_t* p) {
  u32x2 lo = *reinterpret_cast<const u32x2*>(p);
  u32x2 hi = *reinterpret_cast<const u32x2*>(p + 8);
  u32x4 r = {lo.x, lo.y, hi.x, hi.y};
  return as_bf16x8(r);
}

// Round 8 floats to bf16 (round-to-nearest-even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16x8 pack_bf16x8(float x0, float x1, float x2, float x3, float x4,
                                              float x5, float x6, float x7) {
  bf16x8 r;
  r[0] = (__bf16)x0; r[1] = (__bf16)x1; r[2] = (__bf16)x2; r[3] = (__bf16)x3;
  r[4] = (__bf16)x4; r[5] = (__bf16)x5; r[6] = (__bf16)x6; r[7] = (__bf16)x7;
  return r;
}

// Pack C-tile values v0..v0+7 of a 32x32 accumulator into one bf16x8 operand
// (k-slot e <- value v0 + e).
__device__ __forceinline__ bf16x8 pack_c8(const f32x16& c, int v0) {
  return pack_bf16x8(c[v0 + 0], c[v0 + 1], c[v0 + 2], c[v0 + 3], c[v0 + 4], c[v0 + 5], c[v0 + 6],
                     c[v0 + 7]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ float xor32(float x) { return __shfl_xor(x, 32); }

// A 4-row x 8-column bf16 block held by one thread: rows r0..r0+3 of a tile,
// columns c0..c0+7, as four 16-byte words.
struct Block4x8 {
  u32x4 r[4];
};

// Load rows [row0, row0+4) x cols [col0, col0+8) of a row-major bf16 matrix
// whose row `x` starts at base + x*row_stride; rows >= row_limit read as 0.
__device__ __forceinline__ void load_block4x8(Block4x8& blk, const uint16_t* base, int64_t row_stride,
                                              int64_t row0, int64_t row_limit, int col0) {
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    const int64_t row = row0 + x;
    if (row < row_limit) {
      blk.r[x] = ld_global16(base + row * row_stride + col0);
    } else {
      blk.r[x] = u32x4{0u, 0u, 0u, 0u};
    }
  }
}

// Store the block in natural layout: lds[(row)*pitch + col].
__device__ __forceinline__ void store_block_nat(const Block4x8& blk, uint16_t* lds, int pitch, int row0,
                                                int col0) {
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    *reinterpret_cast<u32x4*>(lds + (row0 + x) * pitch + col0) = blk.r[x];
  }
}

// Store the block transposed: lds[(col)*pitch + row], 4 consecutive rows of
// one column forming one 8-byte word.
__device__ __forceinline__ void store_block_trans(const Block4x8& blk, uint16_t* lds, int pitch,
                                                  int row0, int col0) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int w = e >> 1;
    uint32_t lo, hi;
    if (e & 1) {
      lo = (blk.r[0][w] >> 16) | (blk.r[1][w] & 0xffff0000u);
      hi = (blk.r[2][w] >> 16) | (blk.r[3][w] & 0xffff0000u);
    } else {
      lo = (blk.r[0][w] & 0xffffu) | (blk.r[1][w] << 16);
      hi = (blk.r[2][w] & 0xffffu) | (blk.r[3][w] << 16);
    }
    *reinterpret_cast<u32x2*>(lds + (col0 + e) * pitch + row0) = u32x2{lo, hi};
  }
}

}  // namespace sppo
