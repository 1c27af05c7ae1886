// Matrix-core throughput ceiling of the chip under its power limit.
//
// Every SIMD of the chip runs a wave that issues nothing but bf16
// v_mfma_f32_32x32x16 products from registers (no memory, no vector
// arithmetic in the loop), four independent accumulators, for about 60 ms
// per launch.  The rate it reaches is the most any kernel can execute with
// the same operand data: the products run at one per 32 cycles per SIMD, so
// the rate gives the shader clock the chip holds under that load.
//
// Operand data: "randn" is bf16 of standard normal values (the distribution
// of the attention inputs of the synthetic workloads), "zero" is all zeros.
// Operand patterns (A and B are the two 16x32 bf16 inputs of a product):
//   0  A and B both change from one product to the next
//   1  A held for two consecutive products
//   2  A held for four
//   3  the same A and B for every product
// Build and run (one GPU):
//   hipcc -O3 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       -o mfma_ceiling paper_2609_22755_amd/probes/mfma_ceiling.hip
//   ./mfma_ceiling
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#define CHECK(x)                                                                   \
  do {                                                                             \
    hipError_t e_ = (x);                                                           \
    if (e_ != hipSuccess) {                                                        \
      fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));               \
      exit(1);                                                                     \
    }                                                                              \
  } while (0)

constexpr int kBlocks = 256;   // one workgroup per CU
constexpr int kRegs = 16;      // operand registers per lane (8 bf16 each)

// src holds kRegs * 8 bf16 per thread of the grid; out one float per thread.
template <int MODE>
__global__ __launch_bounds__(512) void products(const unsigned short *src, float *out, int iters) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  bf16x8 op[kRegs];
  for (int r = 0; r < kRegs; ++r)
    for (int e = 0; e < 8; ++e) op[r][e] = __builtin_bit_cast(bf16, src[(size_t)t * kRegs * 8 + r * 8 + e]);
  f32x16 acc[4] = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      bf16x8 a, b;
      if (MODE == 0) { a = op[i]; b = op[(i + 5) & 15]; }
      else if (MODE == 1) { a = op[i & ~1]; b = op[(i + 5) & 15]; }
      else if (MODE == 2) { a = op[i & ~3]; b = op[(i + 5) & 15]; }
      else { a = op[0]; b = op[5]; }
      acc[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i & 3], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);   // keep the products in this order
    }
  }
  float s = 0.f;
  for (int j = 0; j < 4; ++j)
    for (int e = 0; e < 16; ++e) s += acc[j][e];
  out[t] = s;
}

// bf16 (round to nearest even) of a float
static unsigned short to_bf16(float f) {
  unsigned u;
  std::memcpy(&u, &f, 4);
  u += 0x7fff + ((u >> 16) & 1);
  return (unsigned short)(u >> 16);
}

int main() {
  const int iters = 200000;
  for (int waves = 1; waves <= 2; ++waves) {
    const int threads = 256 * waves;   // 4 or 8 waves: one or two per SIMD
    const size_t nthr = (size_t)kBlocks * threads, n = nthr * kRegs * 8;
    std::vector<unsigned short> randn(n), zero(n, 0);
    unsigned long long x = 0x9e3779b97f4a7c15ull;
    auto uni = [&]() {   // 53-bit uniform in (0, 1) from a 64-bit LCG
      x = x * 6364136223846793005ull + 1442695040888963407ull;
      return ((x >> 11) + 0.5) / 9007199254740992.0;
    };
    for (size_t i = 0; i < n; i += 2) {   // Box-Muller pairs
      const double r = std::sqrt(-2.0 * std::log(uni())), th = 6.283185307179586 * uni();
      randn[i] = to_bf16((float)(r * std::cos(th)));
      randn[i + 1] = to_bf16((float)(r * std::sin(th)));
    }
    unsigned short *d;
    float *o;
    CHECK(hipMalloc(&d, n * 2));
    CHECK(hipMalloc(&o, nthr * 4));
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    for (int data = 0; data < 2; ++data) {
      CHECK(hipMemcpy(d, data ? zero.data() : randn.data(), n * 2, hipMemcpyHostToDevice));
      for (int mode = 0; mode < 4; ++mode) {
        auto launch = [&]() {
          const int it = iters / waves;   // the same products per SIMD at either occupancy
          if (mode == 0) products<0><<<kBlocks, threads>>>(d, o, it);
          else if (mode == 1) products<1><<<kBlocks, threads>>>(d, o, it);
          else if (mode == 2) products<2><<<kBlocks, threads>>>(d, o, it);
          else products<3><<<kBlocks, threads>>>(d, o, it);
          CHECK(hipGetLastError());
        };
        launch();   // warm up: the clock settles under the load
        float best = 1e30f;
        for (int rep = 0; rep < 3; ++rep) {
          CHECK(hipEventRecord(e0));
          launch();
          CHECK(hipEventRecord(e1));
          CHECK(hipEventSynchronize(e1));
          float ms;
          CHECK(hipEventElapsedTime(&ms, e0, e1));
          best = ms < best ? ms : best;
        }
        const double per_simd = (double)(iters / waves) * 16 * waves;   // products per SIMD
        const double flops = per_simd * kBlocks * 4 * 32.0 * 32 * 16 * 2;
        printf("waves/SIMD %d  data %-5s  pattern %d: %7.2f ms  %7.1f TFLOP/s  (%.1f%% of 2516.6)  clock %.3f GHz\n",
               waves, data ? "zero" : "randn", mode, best, flops / (best * 1e9), flops / (best * 1e9) / 25.166,
               per_simd * 32 / (best * 1e6));
        fflush(stdout);
      }
    }
    CHECK(hipFree(d));
    CHECK(hipFree(o));
  }
  return 0;
}
