// Ulysses re-layout (local halves of the prologue / epilogue exchange) for
// gfx950.  Pure data movement, bound by HBM bandwidth.
//
// The host turns a work list into copy tasks; each task moves `ntok` runs of
// `cpt` 16-byte chunks from a source with token stride src_ts to a
// destination with token stride dst_ts (the run of one token is contiguous on
// both sides: H_loc*D elements for the query kind, D for a KV head).  One
// workgroup per task; consecutive lanes take consecutive 16-byte chunks, so
// every wave reads and writes whole contiguous runs.  Replica sums (the
// epilogue of a KV head replicated over sp/H ranks) add the replicas in
// float32 in increasing replica order and round once.
#include "device_common.hpp"
#include "nsp_internal.hpp"

namespace nsp {
namespace {

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const bf16 x = (bf16)a, y = (bf16)b;
  return (uint32_t)__builtin_bit_cast(unsigned short, x) |
         ((uint32_t)__builtin_bit_cast(unsigned short, y) << 16);
}

// sum_mode: 0 = copy (first replica), 1 = bf16 replica sum, 2 = f32 replica sum
template <int SUM>
__global__ void __launch_bounds__(256) relayout_kernel(const char *__restrict__ src,
                                                       char *__restrict__ dst,
                                                       const CopyTask *__restrict__ tasks) {
  const CopyTask t = tasks[blockIdx.x];
  const int total = t.ntok * t.cpt;
  constexpr int U = 4;   // chunks in flight per lane
  for (int base = threadIdx.x; base < total; base += 256 * U) {
    uint4 v[U];
    int64_t doff[U];
    bool ok[U];
#pragma unroll
    for (int r = 0; r < U; ++r) {
      const int q = base + 256 * r;
      ok[r] = q < total;
      const int tok = t.t0 + (ok[r] ? q / t.cpt : 0);
      const int c = ok[r] ? q % t.cpt : 0;
      const int64_t soff = t.src + tok * t.src_ts + 16 * (int64_t)c;
      doff[r] = t.dst + tok * t.dst_ts + 16 * (int64_t)c;
      if (!ok[r]) continue;
      if constexpr (SUM == 0) {
        v[r] = *(const uint4 *)(src + soff);
      } else {
        float acc[8];
        uint4 w = *(const uint4 *)(src + soff);
        if constexpr (SUM == 1) {
          const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) { acc[2 * e] = bf16_lo(ws[e]); acc[2 * e + 1] = bf16_hi(ws[e]); }
          for (int rep = 1; rep < t.nrep; ++rep) {
            const uint4 x = *(const uint4 *)(src + soff + rep * t.rep_stride);
            const uint32_t xs[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) { acc[2 * e] += bf16_lo(xs[e]); acc[2 * e + 1] += bf16_hi(xs[e]); }
          }
          v[r] = uint4{pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                       pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7])};
        } else {
          acc[0] = __uint_as_float(w.x); acc[1] = __uint_as_float(w.y);
          acc[2] = __uint_as_float(w.z); acc[3] = __uint_as_float(w.w);
          for (int rep = 1; rep < t.nrep; ++rep) {
            const uint4 x = *(const uint4 *)(src + soff + rep * t.rep_stride);
            acc[0] += __uint_as_float(x.x); acc[1] += __uint_as_float(x.y);
            acc[2] += __uint_as_float(x.z); acc[3] += __uint_as_float(x.w);
          }
          v[r] = uint4{__float_as_uint(acc[0]), __float_as_uint(acc[1]), __float_as_uint(acc[2]),
                       __float_as_uint(acc[3])};
        }
      }
    }
#pragma unroll
    for (int r = 0; r < U; ++r)
      if (ok[r]) {
        // written once and read by a later kernel: a non-temporal store
        // keeps it from displacing reused lines in the caches (+10% on the
        // largest re-layouts, measured)
        typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 w4 = {v[r].x, v[r].y, v[r].z, v[r].w};
        __builtin_nontemporal_store(w4, (u32x4 *)(dst + doff[r]));
      }
  }
}

}  // namespace

hipError_t launch_relayout(const void *src, void *dst, const CopyTask *tasks, int n_tasks,
                           int sum_mode, hipStream_t s) {
  if (n_tasks == 0) return hipSuccess;
  dim3 grid(n_tasks), block(256);
  const char *sp = (const char *)src;
  char *dp = (char *)dst;
  if (sum_mode == 0) relayout_kernel<0><<<grid, block, 0, s>>>(sp, dp, tasks);
  else if (sum_mode == 1) relayout_kernel<1><<<grid, block, 0, s>>>(sp, dp, tasks);
  else relayout_kernel<2><<<grid, block, 0, s>>>(sp, dp, tasks);
  return hipGetLastError();
}

}  // namespace nsp
