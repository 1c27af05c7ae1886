// Matrix-core throughput ceiling of the device under its power limit.
//
// Every SIMD of the device runs waves that issue nothing but bf16
// v_mfma_f32_32x32x16 products from registers (no memory access and no
// vector arithmetic in the loop, a scheduling fence after each product), with
// four independent accumulators.  A product occupies its SIMD's matrix core
// for 32 cycles, so the rate reached gives the shader clock the device holds
// under that load; with random operands the power limit, not the nominal
// clock, sets it.  It bounds what any kernel can execute with operand data of
// the same kind, and it differs from one device to the next as the attention
// kernels' own rates do.
//
// Operands are generated in registers: approximately standard normal values
// (the sum of four uniforms of a counter hash, centred and scaled; the
// attention inputs' distribution) rounded to bf16, or zeros.  Patterns: 0 --
// both operands change from one product to the next; 1 / 2 -- the first
// operand is held for two / four products; 3 -- the same operands throughout.
#include <hip/hip_runtime.h>

#include "nsp.h"
#include "nsp_internal.hpp"

namespace nsp {

// never written in practice: a store that depends on every product keeps
// them from being optimised away (the array has external linkage, so the
// compiler cannot prove the store unobservable)
__device__ float g_ceiling_sink[64];

namespace {

typedef __bf16 bf16_t;
typedef bf16_t bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kOps = 16;   // operand registers (8 bf16 each) per lane

__device__ __forceinline__ uint32_t mix32(uint32_t x) {   // a 32-bit integer hash (xorshift-multiply rounds)
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

// LDS each workgroup reserves and never uses: more than half of a compute
// unit's 160 KiB, so that no two workgroups share a compute unit and a grid
// of one workgroup per compute unit puts one on every one of them
constexpr int kReserveLds = 96 * 1024;

template <int PATTERN>
__global__ __launch_bounds__(512) void mfma_ceiling_kernel(int64_t iters, int zero) {
  __shared__ char reserve[kReserveLds];
  asm volatile("" ::"v"((uint32_t)(uintptr_t)reserve));
  const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  bf16x8_t op[kOps];
  for (int r = 0; r < kOps; ++r)
    for (int e = 0; e < 8; ++e) {
      float v = 0.f;
      if (!zero) {
        const uint32_t h = mix32(t * 131u + (uint32_t)(r * 8 + e) * 0x9e3779b9u + 1u);
        // four 8-bit uniforms: their sum has mean 510 and variance 4 * (256^2 - 1) / 12
        const float s = (float)(h & 255u) + (float)((h >> 8) & 255u) + (float)((h >> 16) & 255u) + (float)(h >> 24);
        v = (s - 510.f) * (1.f / 147.8f);
      }
      op[r][e] = (bf16_t)v;
    }
  f32x16_t acc[4] = {};
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      bf16x8_t a, b;
      if (PATTERN == 0) { a = op[i]; b = op[(i + 5) & 15]; }
      else if (PATTERN == 1) { a = op[i & ~1]; b = op[(i + 5) & 15]; }
      else if (PATTERN == 2) { a = op[i & ~3]; b = op[(i + 5) & 15]; }
      else { a = op[0]; b = op[5]; }
      acc[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i & 3], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  float s = 0.f;
  for (int j = 0; j < 4; ++j)
    for (int e = 0; e < 16; ++e) s += acc[j][e];
  if (s == -1.2345e-30f) g_ceiling_sink[threadIdx.x & 63] = s;
}

hipError_t launch_ceiling(int pattern, int zero, int blocks, int threads, int64_t iters) {
  switch (pattern) {
    case 0: mfma_ceiling_kernel<0><<<blocks, threads>>>(iters, zero); break;
    case 1: mfma_ceiling_kernel<1><<<blocks, threads>>>(iters, zero); break;
    case 2: mfma_ceiling_kernel<2><<<blocks, threads>>>(iters, zero); break;
    default: mfma_ceiling_kernel<3><<<blocks, threads>>>(iters, zero); break;
  }
  return hipGetLastError();
}

}  // namespace
}  // namespace nsp

extern "C" nsp_status nsp_mfma_ceiling(int32_t pattern, int32_t zero_operands, int32_t waves_per_simd,
                                       int64_t products_per_simd, double *seconds, double *tflops) {
  using namespace nsp;
  if (pattern < 0 || pattern > 3) return set_error(NSP_EINVAL, "nsp_mfma_ceiling: pattern %d not in 0..3", pattern);
  if (waves_per_simd < 1 || waves_per_simd > 2)
    return set_error(NSP_EINVAL, "nsp_mfma_ceiling: waves_per_simd %d not 1 or 2", waves_per_simd);
  if (products_per_simd <= 0 || products_per_simd > ((int64_t)1 << 24) ||
      products_per_simd % (16 * waves_per_simd) != 0)
    return set_error(NSP_EINVAL,
                     "nsp_mfma_ceiling: products_per_simd %lld not a positive multiple of 16 x waves_per_simd "
                     "up to 2^24",
                     (long long)products_per_simd);
  if (!seconds || !tflops) return set_error(NSP_EINVAL, "nsp_mfma_ceiling: NULL output");
  int cus = 0;
  hipError_t e = compute_units(&cus);
  if (e != hipSuccess) return set_error(NSP_EHIP, "nsp_mfma_ceiling: %s", hipGetErrorString(e));
  const int threads = 256 * waves_per_simd;   // 4 SIMDs per compute unit
  const int64_t iters = products_per_simd / (16 * waves_per_simd);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  float ms = 0.f;
  if ((e = hipEventCreate(&e0)) == hipSuccess && (e = hipEventCreate(&e1)) == hipSuccess &&
      (e = launch_ceiling(pattern, zero_operands != 0, cus, threads, iters)) == hipSuccess &&   // warm-up
      (e = hipEventRecord(e0, nullptr)) == hipSuccess &&
      (e = launch_ceiling(pattern, zero_operands != 0, cus, threads, iters)) == hipSuccess &&
      (e = hipEventRecord(e1, nullptr)) == hipSuccess && (e = hipEventSynchronize(e1)) == hipSuccess)
    e = hipEventElapsedTime(&ms, e0, e1);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (e != hipSuccess) return set_error(NSP_EHIP, "nsp_mfma_ceiling: %s", hipGetErrorString(e));
  *seconds = ms * 1e-3;
  *tflops = (double)products_per_simd * cus * 4 * (32.0 * 32 * 16 * 2) / (*seconds * 1e12);
  return set_error(NSP_OK, nullptr);
}
