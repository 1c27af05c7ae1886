// Device-side building blocks for gfx950 (CDNA4): bf16 MFMA, LDS transpose
// reads and tile staging.
//
// MFMA v_mfma_f32_32x32x16_bf16 lane layout (one 64-lane wave):
//   A (32 x 16, M x K): lane l supplies row l%32, k = 8*(l/32) + j, j = 0..7
//   B (16 x 32, K x N): lane l supplies column l%32, k = 8*(l/32) + j
//   C (32 x 32):        lane l holds column l%32, element i holds
//                       row 8*(i/4) + 4*(l/32) + i%4
// Any permutation of k applied to A and B alike leaves the product unchanged;
// the kernels use that to feed the accumulator of one product (C layout) as
// the operand of the next without moving data between lanes.
//
// ds_read_b64_tr_b16: within each group of 16 lanes, lane i receives element
// i%4 of the 8-byte reads of lanes i/4 + 4e (e = 0..3).  If local lane j reads
// row r0 + j/4, columns c0 + 4*(j%4) .. +3 of a row-major tile, lane i gets
// rows r0..r0+3 of column c0 + i: the "transposed" MFMA operand, read
// straight from the row-major tile.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nsp {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x4 lds_read_tr4(const bf16 *p) {
  i16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4 *)p);
  return __builtin_bit_cast(bf16x4, r);
}

__device__ __forceinline__ bf16x8 cat4(bf16x4 a, bf16x4 b) {
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Transposed operand for a 32-wide block of columns [c_blk, c_blk+32) and the
// 16 rows r_base + {4h..4h+3, 8+4h..8+4h+3} of a row-major LDS tile with row
// pitch `ld` elements (h = lane/32).  Lane l receives column c_blk + l%32.
// The row order matches the k order of an accumulator element block
// 8a..8a+7 (see the C layout above), so the result pairs with it in an MFMA.
__device__ __forceinline__ bf16x8 lds_tr_operand(const bf16 *tile, int ld, int r_base, int c_blk,
                                                 int lane) {
  const int h = lane >> 5;
  const int g = lane >> 4;
  const int j = lane & 15;
  const int col = c_blk + 16 * (g & 1) + 4 * (j & 3);
  const int row = r_base + 4 * h + (j >> 2);
  bf16x4 lo = lds_read_tr4(tile + row * ld + col);
  bf16x4 hi = lds_read_tr4(tile + (row + 8) * ld + col);
  return cat4(lo, hi);
}

__device__ __forceinline__ float wave_max_halves(float x) { return fmaxf(x, __shfl_xor(x, 32)); }
__device__ __forceinline__ float wave_sum_halves(float x) { return x + __shfl_xor(x, 32); }

}  // namespace nsp
