// Device-side helpers shared by the gfx950 attention kernels: vector types,
// the bf16 MFMA wrapper, LDS-DMA tile staging, and the swizzled LDS tile
// layout with its natural and transposed operand reads.
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

#include <type_traits>

namespace sppo {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) short v4i16;
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

template <int I>
using IC = std::integral_constant<int, I>;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& x) { return __builtin_bit_cast(bf16x8, x); }

__device__ __forceinline__ u32x4 ld_global16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

// Eight floats to bf16, rounded to nearest even (v_cvt_pk_bf16_f32).
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

// IEEE maximum (NaN-propagating): fmaxf's maxNum must quiet signalling NaNs
// first, so in IEEE mode it puts a v_max_f32 x, x, x in front of every
// operand it cannot prove canonical (all MFMA results); maximum needs no such
// step, and gfx950 evaluates three operands per v_maximum3_f32.
__device__ __forceinline__ float max3_nc(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}
__device__ __forceinline__ float max_nc(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// Reductions across the two 32-lane halves of a wave (lane l with l^32):
// v_permlane32_swap leaves x and its partner in the two results.
__device__ __forceinline__ float max_xor32(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max_nc(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ------------------------------------------------------ buffer resources
// Tiles are read through a buffer resource based at the tile's first row:
// the hardware range check returns zero for every byte offset at or past
// num_records, so rows >= valid_rows read as zero with no per-lane test, and
// the per-lane byte offsets stay the same from tile to tile (only the scalar
// base moves).  Offsets are relative to the tile base, so they fit in 32 bits
// whatever the tensor size.
constexpr int kBufferFlags = 0x00020000;  // dword 3 of a raw gfx9 buffer resource

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint16_t* tile_base, int64_t valid_rows,
                                                            int tile_rows, int64_t row_stride) {
  const int n = valid_rows <= 0 ? 0 : (valid_rows < tile_rows ? (int)valid_rows : tile_rows);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(tile_base), (short)0,
                                           n * (int)(row_stride * (int64_t)sizeof(uint16_t)), kBufferFlags);
}

// A wave-uniform 64-bit value moved to scalar registers (64-bit products
// are formed by the VALU, so an address computed from uniform values can
// still sit in VGPRs; a scalar copy keeps later updates on the SALU).
__device__ __forceinline__ uint64_t uniform_u64(uint64_t x) {
  return ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(x >> 32)) << 32) |
         (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)x);
}

// Buffer resource over the nbytes bytes at byte address addr, with every
// field made wave-uniform (a buffer instruction takes it in scalar registers).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t uniform_rsrc(uint64_t addr, int nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(uniform_u64(addr)), (short)0,
                                           __builtin_amdgcn_readfirstlane(nbytes), kBufferFlags);
}

// ------------------------------------------------------- XCD grouping
// The dispatcher hands workgroups to the 8 XCDs (each with its own L2)
// round-robin in linear order (x fastest).  xcd_grouped() returns the grid
// position a workgroup works on such that each XCD receives one contiguous
// range of linear positions: the query tiles of one head, which all stream
// the same K/V rows, then run side by side behind one L2.  A grid whose size
// is not a multiple of 8 keeps the identity mapping.
struct GridPos {
  int x, y, z;
};
__device__ __forceinline__ GridPos xcd_grouped() {
  const uint32_t nx = gridDim.x, ny = gridDim.y;
  const uint32_t total = nx * ny * gridDim.z;
  uint32_t n = blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z);
  if (total % 8 == 0) n = (n % 8) * (total / 8) + n / 8;
  return GridPos{(int)(n % nx), (int)((n / nx) % ny), (int)(n / (nx * ny))};
}

// ------------------------------------------------------------- LDS-DMA
// buffer_load ... lds moves 16 (or 4) bytes per lane from a buffer resource
// straight into LDS, lane l's bytes landing at lds + 16 l (4 l): one wave
// instruction fills 1 KiB of LDS with no VGPR staging and no ds_write.  The
// loads are issued from inline asm so that the compiler does not treat them
// as LDS stores it must order (its tracking falls back to waiting for every
// outstanding load); the kernels order them themselves, each with an
// explicit s_waitcnt vmcnt(...) followed by a workgroup barrier before any
// wave reads what another wave loaded.  M0 carries the LDS address; no other
// code in these kernels uses M0.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  // A generic pointer into LDS is the shared aperture (high half) plus the
  // LDS offset (low half); truncating skips the null check of a cast.
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
}
// (clang warns that M0 is a reserved register; it is only reserved for the
// compiler's own M0 uses, and these kernels have none.)
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16(__amdgpu_buffer_rsrc_t rsrc, void* lds, int voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds_addr(lds)), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
__device__ __forceinline__ void lds_dma4(__amdgpu_buffer_rsrc_t rsrc, void* lds, int voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :
               : "s"(lds_addr(lds)), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt immediate that waits for the vector-memory counter to drop to v
// (expcnt and lgkmcnt left at their maxima).
__device__ __forceinline__ constexpr int waitcnt_vm(int v) { return (v & 15) | ((v >> 4) << 14) | 0x0F70; }

// ---------------------------------------------------------------- LDS tiles
// A bf16 tile [rows][D] is stored unpadded (row pitch D elements), its
// 16-byte chunk c of row r at physical chunk c ^ f(r).  The gfx950 LDS has 64
// four-byte banks (256 bytes); a ds_read_b128 is served 16 lanes at a time
// and a ds_read_b64_tr_b16 32 lanes at a time.  f spreads both access
// patterns over all 64 banks:
//   * natural operand reads: 16 consecutive rows, one chunk each -- f is a
//     bijection on the low 4 bits of the row (D = 128: a row is one bank
//     window; D = 64: two rows per window, f bijective per row parity);
//   * transposed reads: 4 consecutive rows x 4 consecutive chunks per 32
//     lanes -- the rows land in 4 different 64-byte quarters.
// Rows are written by LDS-DMA in their physical order (1 KiB per wave
// instruction), so lane l of an instruction fetches the global chunk that
// belongs at physical position l.
template <int D>
struct XTile {
  static constexpr int P = D;         // row pitch, elements
  static constexpr int CG = D / 8;    // 16-byte chunks per row
  static constexpr int RPI = 512 / D; // rows per LDS-DMA wave instruction
  static __device__ __forceinline__ int f(int r) {
    if constexpr (D == 128) {
      return ((r & 3) << 2) | ((r >> 2) & 3);
    } else {
      return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
    }
  }
  // Natural operand read of k-step kk for rows rb + l%32 (rb % 32 == 0):
  // element offset (add rb * P).
  static __device__ __forceinline__ int nat(int lane, int kk) {
    const int l32 = lane & 31, g = lane >> 5;
    return l32 * P + 8 * ((2 * kk + g) ^ f(l32));
  }
  // Transposed read of rows k0 + {0..7} (hi = 0) or k0 + {8..15} (hi = 1),
  // columns 32 db..32 db+31 (add k0 * P, k0 % 16 == 0).  Source lane
  // s = 16q + 4e + a supplies the 8 bytes at row 4(q/2) + e, columns
  // 16(q%2) + 4a of the 16x32 block; ds_read_b64_tr_b16 hands output lane
  // 16q + 4a' + b element b of source lanes 16q + 4e + a', e = 0..3.
  static __device__ __forceinline__ int tr(int lane, int db, int hi) {
    const int q = lane >> 4, e = (lane >> 2) & 3, a = lane & 3;
    const int row = 4 * (q >> 1) + e + 8 * hi;
    const int c = 4 * db + 2 * (q & 1) + (a >> 1);
    return row * P + 8 * (c ^ f(row)) + 4 * (a & 1);
  }
  // Byte offset, relative to the first row of a tile in global memory, of
  // the chunk lane `lane` fetches in LDS-DMA instruction u of the tile.
  static __device__ __forceinline__ int dma(int lane, int u, int64_t row_stride) {
    const int row = RPI * u + lane / CG, p = lane % CG;
    return (int)((row * row_stride + 8 * (p ^ f(row))) * (int64_t)sizeof(uint16_t));
  }
};

__device__ __forceinline__ v4i16 ds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p));
}

// Natural operand: lane l gets row l%32, columns 16 kk + 8 (l/32) + 0..7 of
// the 32-row block at X (offset from XTile::nat).
__device__ __forceinline__ bf16x8 ld_nat(const uint16_t* X, int off) {
  return as_bf16x8(*reinterpret_cast<const u32x4*>(X + off));
}

// Transposed operand from a natural tile: lane l gets column l%32 of the
// 32-column block and rows {8(e/4) + 4(l/32) + e%4 : e = 0..7} of the 16-row
// block, i.e. the permuted k-slot map, so it pairs with an operand taken
// from C-tile registers.  lo/hi: XTile::tr offsets plus the block's row base.
__device__ __forceinline__ bf16x8 ld_tr(const uint16_t* X, int lo, int hi) {
  const v4i16 a = ds_read_tr16(X + lo);
  const v4i16 b = ds_read_tr16(X + hi);
  const u32x2 a2 = __builtin_bit_cast(u32x2, a), b2 = __builtin_bit_cast(u32x2, b);
  return as_bf16x8(u32x4{a2.x, a2.y, b2.x, b2.y});
}

// GELU in its tanh form, x/2 (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3))), and
// its derivative; shared by the GEMM epilogues and the recompute kernel so
// the forward and the backward evaluate the same expression.
__device__ __forceinline__ float gelu_tanh(float x) {
  const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
  return 0.5f * x * (1.f + tanhf(u));
}
__device__ __forceinline__ float gelu_tanh_grad(float x) {
  const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
  const float t = tanhf(u);
  return 0.5f * (1.f + t) + 0.5f * x * (1.f - t * t) * 0.7978845608028654f * (1.f + 3.f * 0.044715f * x * x);
}

}  // namespace sppo
