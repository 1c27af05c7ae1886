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

// LDS tiles hold rows of D bf16 without padding; the 16-byte chunks of row r
// are permuted by an XOR with swz(r) so that the two read patterns of the
// kernels are free of bank conflicts on the 64 x 4-byte banks of the LDS:
//   * row reads (ds_read_b128, 16 lanes per cycle): 16 lanes read the same
//     logical chunk of 16 consecutive rows -> swz must be a bijection on
//     r mod 16 (D=128: one row per 256-byte bank line), or on (r/2) mod 8 for
//     each row parity (D=64: two rows per bank line);
//   * transpose reads (ds_read_b64_tr_b16, 32 lanes per cycle): rows r..r+3
//     (r a multiple of 4) x the aligned group of 4 chunks {q..q+3} -> the 4
//     rows must land in distinct 64-byte bank groups: swz(r+i) / 4 distinct
//     for i = 0..3 (D=128), or distinct for the two rows of each parity
//     (D=64).
template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

// Element offset of (row r, element column col) in a swizzled [rows][D] tile.
template <int D>
__device__ __forceinline__ int tile_off(int r, int col) {
  return r * D + ((((col >> 3) ^ swz<D>(r))) << 3) + (col & 7);
}

// Transposed operand for a 32-wide block of columns [c_blk, c_blk+32) and the
// 16 rows r_base + {4h..4h+3, 8+4h..8+4h+3} of a swizzled row-major LDS tile
// (h = lane/32).  Lane l receives column c_blk + l%32.  The row order matches
// the k order of an accumulator element block 8a..8a+7 (see the C layout
// above), so the result pairs with it in an MFMA.
template <int D>
__device__ __forceinline__ bf16x8 lds_tr_operand(const bf16 *tile, int r_base, int c_blk, int lane) {
  const int h = lane >> 5;
  const int g = lane >> 4;
  const int j = lane & 15;
  const int col = c_blk + 16 * (g & 1) + 4 * (j & 3);
  const int row = r_base + 4 * h + (j >> 2);
  bf16x4 lo = lds_read_tr4(tile + tile_off<D>(row, col));
  bf16x4 hi = lds_read_tr4(tile + tile_off<D>(row + 8, col));
  return cat4(lo, hi);
}

// Row operand: 8 consecutive elements [col, col+8) of row r of a swizzled tile
// (col a multiple of 8).
template <int D>
__device__ __forceinline__ bf16x8 lds_row8(const bf16 *tile, int r, int col) {
  return *(const bf16x8 *)(tile + tile_off<D>(r, col));
}

// Combine a per-lane value with the one of lane l^32 (the other half of the
// 32-wide MFMA column): v_permlane32_swap hands each lane its partner's value.
__device__ __forceinline__ float wave_max_halves(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float wave_sum_halves(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Buffer resource for raw (unformatted, unswizzled) loads from `base`: every
// byte offset below 2^31 is in range (callers keep offsets within their
// tensors).  Word 3 is the gfx9-family default for raw dword access.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void *base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, 0x7fffffff, 0x00020000);
}

// Direct load of `bytes` (4 or 16) per lane from rsrc + voff into LDS: lane l
// lands at lds + bytes*l.  A buffer (MUBUF) load, not a global (FLAT) one: the
// compiler then still counts LDS reads precisely while such loads are in
// flight (with a FLAT one pending it waits for every outstanding LDS read).
template <int BYTES>
__device__ __forceinline__ void load_lds(__amdgpu_buffer_rsrc_t rs, unsigned voff, void *lds) {
  static_assert(BYTES == 4 || BYTES == 16, "load size");
  auto *dst = (__attribute__((address_space(3))) void *)lds;
  if constexpr (BYTES == 16) __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, dst, 16, voff, 0, 0, 0);
  else __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, dst, 4, voff, 0, 0, 0);
}

// Buffer resource for rows r0.. of a tensor whose last valid row is L-1 (row
// stride `stride` elements, D elements used per row): the range ends with the
// data of row L-1, and is empty when r0 >= L.  An out-of-range buffer load
// returns zeros; with an LDS destination it writes zeros into LDS (checked on
// gfx950), and touches no memory.  Callers read at most kRsrcRows rows from
// r0, so the range is capped there (which keeps it in 32 bits); the
// arithmetic is branch-free scalar code, since a branch near the loads makes
// the compiler wait for every load in flight before the next LDS read.
constexpr int kRsrcRows = 1024;
template <int D>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const bf16 *src, int64_t stride, int r0, int L) {
  const int row_bytes = (int)stride * 2;
  const int bytes = max(0, min(L - r0, kRsrcRows) * row_bytes - (row_bytes - 2 * D));
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16 *>(src + (int64_t)r0 * stride), 0, bytes, 0x00020000);
}

// The same load issued as inline assembly (M0 = LDS base of lane 0; M0 is
// written only here in the kernels that use it).  The compiler does not see
// it, so it never adds waits of its own for LDS reads that it cannot tell
// apart from the load's destination; the caller orders the load against the
// reads of its LDS buffer (s_waitcnt vmcnt + workgroup barrier before reading,
// barrier before refilling).  The "memory" clobber keeps the compiler from
// moving other memory accesses across it.
template <int BYTES>
__device__ __forceinline__ void load_lds_untracked(__amdgpu_buffer_rsrc_t rs, unsigned voff, void *lds) {
  static_assert(BYTES == 4 || BYTES == 16, "load size");
  const unsigned m0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) void *)lds;
  if constexpr (BYTES == 16)
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(m0), "v"(voff), "s"(rs)
                 : "memory");
  else
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                 :
                 : "s"(m0), "v"(voff), "s"(rs)
                 : "memory");
}

// Asynchronous copy of ROWS rows of D bf16 into an unpadded LDS tile
// [ROWS][D], by the NW waves of a workgroup, with direct buffer->LDS loads of
// 16 bytes per lane: each instruction moves 64 lanes x 16 bytes, lane l
// landing at the instruction's LDS base + 16*l (so one instruction fills
// 64/(D/8) consecutive rows).  Rows are r0 .. r0+ROWS-1 of a tensor with row
// stride `stride` elements; rows at or past L arrive as zeros (out-of-range
// loads, see rows_rsrc), so a tile wholly past L costs no memory traffic and
// the loads need no per-tile address arithmetic: each lane's byte offsets
// within a tile are fixed at construction.  `wave` must be wave-uniform.
// Completion: s_waitcnt vmcnt, then a workgroup barrier.
template <int D, int ROWS, int NW = 4>
struct TileLoader {
  static constexpr int LPR = D / 8;             // lanes per row
  static constexpr int RPI = 64 / LPR;          // rows per instruction
  static constexpr int PER_WAVE = ROWS / RPI / NW;
  static_assert(ROWS % (RPI * NW) == 0, "tile rows must split evenly over the waves");
  const bf16 *src;             // tensor base (row 0 of the item/head)
  int64_t stride;              // elements between rows
  unsigned voff[PER_WAVE];     // this lane's byte offset within a tile, per instruction
  int lds_off;                 // this wave's first LDS element within the tile

  // Lane l of instruction k fills LDS slot s = l % LPR of tile row
  // r = (first row of the wave) + l / LPR + k*RPI, so it fetches logical chunk
  // s ^ swz(r) of that row.
  __device__ __forceinline__ TileLoader(const bf16 *src_, int64_t stride_, int wave, int lane)
      : src(src_), stride(stride_) {
    const int row_base = wave * PER_WAVE * RPI + lane / LPR;
    const int slot = lane % LPR;
#pragma unroll
    for (int k = 0; k < PER_WAVE; ++k) {
      const int r = row_base + k * RPI;
      voff[k] = (unsigned)((r * (int)stride + ((slot ^ swz<D>(r)) & (LPR - 1)) * 8) * 2);
    }
    lds_off = wave * PER_WAVE * RPI * D;
  }
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(int r0, int L) const {
    return rows_rsrc<D>(src, stride, r0, L);
  }
  __device__ __forceinline__ bf16 *dst(bf16 *lds, int k) const { return lds + lds_off + k * RPI * D; }
  __device__ __forceinline__ void load(bf16 *lds, int r0, int L) const {
    const __amdgpu_buffer_rsrc_t rs = rsrc(r0, L);
#pragma unroll
    for (int k = 0; k < PER_WAVE; ++k) load_lds<16>(rs, voff[k], dst(lds, k));
  }
  __device__ __forceinline__ void load_untracked(bf16 *lds, int r0, int L) const {
    const __amdgpu_buffer_rsrc_t rs = rsrc(r0, L);
#pragma unroll
    for (int k = 0; k < PER_WAVE; ++k) load_lds_untracked<16>(rs, voff[k], dst(lds, k));
  }
};

// s_waitcnt: at most n buffer->LDS loads of this wave still in flight, no LDS
// operation in flight.  (gfx9 encoding: vmcnt[3:0] and [15:14], expcnt[6:4],
// lgkmcnt[11:8].)
template <int N>
__device__ __forceinline__ void wait_loads_le() {
  static_assert(N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | ((N >> 4) << 14));
}

// Workgroup barrier that leaves the loads of later stages in flight (unlike
// __syncthreads, whose fence waits for every outstanding memory operation).
// The empty asm statements keep the compiler from moving LDS accesses across.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// The value, computed at this point of the instruction stream: an empty
// volatile asm that takes and returns it in a VGPR, which the compiler keeps
// in order with the scheduling fences around it.
__device__ __forceinline__ float pin(float x) {
  asm volatile("" : "+v"(x));
  return x;
}

// The wave index as a scalar (wave-uniform) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Per-XCD unit queues of the persistent passes.  The unit list is in launch
// order and slot b belongs to XCD b % 8, so queue x holds slots x, x + 8,
// x + 16, ... and its head (an int in device memory, zero before the pass)
// counts the slots taken.  A workgroup drains the queue of its own XCD first
// -- keeping the XCD runs of the order, and their L2 reuse, on one XCD --
// then takes what is left in the others: XCDs run at different speeds, and a
// fixed slot-to-XCD map would leave the fast ones idle at the end.  Every
// head only grows, so each workgroup stops after at most n_units + 8
// fetches.  One lane fetches; the slot reaches the workgroup through LDS
// between two barriers (the second also keeps the next unit's tile loads
// from overwriting LDS that a wave still reads).  Returns -1 when every
// queue is empty.
constexpr int kXcdQueues = 8;
// s_getreg operand for HW_REG_XCC_ID (register 20, bits 0..15): the XCD a
// wave runs on
constexpr int kHwRegXccId = 20 | (0 << 6) | ((16 - 1) << 11);

__device__ __forceinline__ int next_queue_slot(int *heads, int n_units, int own, int *s_slot) {
  if (threadIdx.x == 0) {
    int slot = -1;
    for (int t = 0; t < kXcdQueues && slot < 0; ++t) {
      const int x = (own + t) % kXcdQueues;
      const int k = atomicAdd(heads + x, 1);
      if (x + kXcdQueues * k < n_units) slot = x + kXcdQueues * k;
    }
    *s_slot = slot;
  }
  __syncthreads();
  const int slot = *s_slot;
  __syncthreads();
  return slot;
}

// The same over per-XCD queues stored one after another: queue x holds the
// slots off[x] .. off[x+1]-1 (off: kXcdQueues + 1 ints).
__device__ __forceinline__ int next_range_slot(int *heads, const int *off, int own, int *s_slot) {
  if (threadIdx.x == 0) {
    int slot = -1;
    for (int t = 0; t < kXcdQueues && slot < 0; ++t) {
      const int x = (own + t) % kXcdQueues;
      const int b = off[x], e = off[x + 1];
      if (b < e) {
        const int k = atomicAdd(heads + x, 1);
        if (b + k < e) slot = b + k;
      }
    }
    *s_slot = slot;
  }
  __syncthreads();
  const int slot = *s_slot;
  __syncthreads();
  return slot;
}

// Wait for this wave's outstanding global (and LDS) operations.
__device__ __forceinline__ void wait_all_loads() { __builtin_amdgcn_s_waitcnt(0); }

}  // namespace nsp
