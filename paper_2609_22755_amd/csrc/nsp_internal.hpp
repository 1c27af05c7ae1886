// Internal host/device interface of libnsp: per-item descriptors, work units
// and the kernel launchers.  Not part of the public ABI (include/nsp.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nsp {

// One item of the work list in the attention layout.  Offsets are in
// elements of the respective tensor, 64-bit.
struct ItemDesc {
  int64_t q_off;    // Q / O / dO / dQ block: [L][hq][D]
  int64_t kv_off;   // K / V / dK / dV block: [L][hkv][D]
  int64_t lse_off;  // LSE / Delta block: [hq][L] (float32)
  int64_t q_row0;   // q_off / D: first D-row of the item in Q
  int32_t L;
  int32_t hq;
  int32_t hkv;
  int32_t active;   // 1 if the call computes this item (work-list item mask)
};

// One workgroup of the backward preprocess: tokens [t0, t0 + ntok) of local
// query head `head` of item `item` (only the items a call computes are
// covered).  Consecutive tokens of one head are consecutive entries of the
// LSE / Delta layout.
struct PreBlock {
  int32_t item;
  int32_t head;
  int32_t t0;
  int32_t ntok;     // at most kPreBlockRows
};
constexpr int kPreBlockRows = 512;

// Tile geometry shared by host scheduling and the kernels.
constexpr int kFwdWaves = 8;  // waves per forward / dQ workgroup (two per SIMD)
constexpr int kFwdBM = 32 * kFwdWaves;   // query rows per forward / dQ workgroup
constexpr int kFwdBN = 64;    // keys per inner iteration
constexpr int kBwdBN = 128;   // keys per dK/dV workgroup (4 waves x 32)
constexpr int kBwdBM = 64;    // query rows per dK/dV pipeline step (two 32-row sub-steps)
// Consecutive LPT units placed on one XCD (about the workgroups an XCD runs at once).
constexpr int kXcdGroupFwd = 32;
// dK/dV unit tile field: 128-key tile index, and the flag of a unit that
// takes its query tiles from the item end down to the diagonal.
constexpr int kKvDescending = 1 << 30;
constexpr int kKvTileMask = kKvDescending - 1;
// Key-tile pairs per dK/dV gang (the workgroups one XCD runs at once).
constexpr int kKvGang = 32;

// Work unit: int4 {item, tile, a, b}.
//   forward / dQ : a = local query head, b = local KV head
//   dK / dV      : a = first local query head | (end local query head << 16),
//                  b = local KV head
struct Schedule {
  ItemDesc *items = nullptr;   // device
  int4 *fwd_units = nullptr;   // device, LPT order (forward and dQ)
  int4 *kv_units = nullptr;    // device, dK/dV units, per-XCD queues one after another
  int *kv_qoff = nullptr;      // device, 9 ints: queue x is kv_units[kv_qoff[x] .. kv_qoff[x+1])
  PreBlock *pre_blocks = nullptr; // device, the preprocess workgroups of the items the call computes
  int n_items = 0;
  int n_fwd_units = 0;
  int n_kv_units = 0;
  int n_pre_blocks = 0;
  int64_t q_rows = 0;          // sum_j L_j * hq_j
  int64_t q_elems = 0, kv_elems = 0, lse_elems = 0;
};

struct AttnArgs {
  const void *q, *k, *v;
  const void *o;          // forward: output; backward: input
  void *o_out;
  float *lse;
  const float *lse_in;
  const void *dout;
  void *dq, *dk, *dv;
  float *delta;           // workspace: -Delta = -rowsum(dO * O)
  float *lse2;            // workspace: lse * log2(e)
  int *queue;             // workspace: unit queue heads, one per XCD (zeroed by the preprocess)
  const ItemDesc *items;
  const PreBlock *pre_blocks;
  const int4 *units;
  const int *qoff;        // dK/dV: start of each XCD's queue in `units`, and the end
  int n_items;
  float scale;            // softmax scale
  float scale_log2;       // softmax scale * log2(e)
};

// Re-layout copy task: move ntok runs of `cpt` 16-byte chunks.
// Byte offsets; replica r of the source lies at src + r * rep_stride.
struct CopyTask {
  int64_t dst, src;
  int64_t dst_ts, src_ts;   // bytes between consecutive tokens
  int64_t rep_stride;
  int32_t t0, ntok;
  int32_t cpt, nrep;
};

// Device scratch of the allocation-free backward: a schedule region, 256
// bytes of unit-queue heads, then -Delta and lse*log2(e) (float32, each part
// 256-byte aligned).
constexpr size_t kScratchBytes = size_t(96) << 20;
constexpr size_t kScratchSchedBytes = size_t(8) << 20;
// The address of the current device's scratch (looked up once per device).
hipError_t noalloc_scratch(char **ptr);

// Record a thread-local error message (returned by nsp_last_error) and
// return `status`; also clears it when called with NSP_OK and no format.
int32_t set_error(int32_t status, const char *fmt, ...);

// Compute units of the current device (looked up once per device).
hipError_t compute_units(int *cus);

hipError_t launch_attn_fwd(int head_dim, bool o_f32, const AttnArgs &a, int n_units, hipStream_t s);
hipError_t launch_bwd_preprocess(int head_dim, bool o_f32, const AttnArgs &a, int n_blocks, hipStream_t s);
hipError_t launch_bwd_dq(int head_dim, bool g_f32, const AttnArgs &a, int n_units, hipStream_t s);
hipError_t launch_bwd_dkdv(int head_dim, bool g_f32, const AttnArgs &a, int n_units, hipStream_t s);
hipError_t launch_relayout(const void *src, void *dst, const CopyTask *tasks, int n_tasks,
                           int sum_mode, hipStream_t s);

}  // namespace nsp
