// Inter-level phase streaming over the SP-tree nodes of one GPU's path: the
// three backend phases of every node issued as item-masked calls on a compute
// queue and a communication queue (see nsp_executor_step in include/nsp.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <functional>
#include <vector>

#include "nsp.h"
#include "nsp_internal.hpp"

namespace {

struct EventPool {
  std::vector<hipEvent_t> ev;
  ~EventPool() {
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);   // released once the event completes
  }
  hipError_t make(hipEvent_t *out) {
    hipError_t e = hipEventCreateWithFlags(out, hipEventDisableTiming);
    if (e == hipSuccess) ev.push_back(*out);
    return e;
  }
};

nsp_status hip_fail(hipError_t e, const char *what) {
  return nsp::set_error(NSP_EHIP, "executor: %s: %s", what, hipGetErrorString(e));
}

nsp_status einval(const char *what) { return nsp::set_error(NSP_EINVAL, "nsp_executor_step: %s", what); }

}  // namespace

#define NSP_X_TRY(expr)              \
  do {                               \
    nsp_status _s = (expr);          \
    if (_s != NSP_OK) return _s;     \
  } while (0)
#define NSP_X_HIP(expr)                                         \
  do {                                                          \
    hipError_t _e = (expr);                                     \
    if (_e != hipSuccess) return hip_fail(_e, #expr);           \
  } while (0)

extern "C" nsp_status nsp_executor_step(const nsp_worklist *wl, const int32_t *node_sp, int32_t n_nodes,
                                        int32_t phases, float softmax_scale, const nsp_step_buffers *b,
                                        hipStream_t compute, hipStream_t comm) {
  nsp::set_error(NSP_OK, nullptr);
  if (!wl || !b) return einval("work list or buffers NULL");
  if (wl->item_mask) return einval("the work list must not carry an item mask");
  if (phases <= 0 || (phases & ~(NSP_STEP_FORWARD | NSP_STEP_BACKWARD))) return einval("unknown phases");
  if (wl->n_items > 0 && (!wl->sp || !wl->cu_seqlens)) return einval("sp and cu_seqlens must be non-NULL");
  // the nodes: distinct sp values, in the given issue order or root first
  std::vector<int32_t> order;
  if (node_sp) {
    if (n_nodes < 0) return einval("n_nodes < 0");
    order.assign(node_sp, node_sp + n_nodes);
  } else {
    for (int j = 0; j < wl->n_items; ++j) order.push_back(wl->sp[j]);
    std::sort(order.begin(), order.end(), std::greater<int32_t>());
    order.erase(std::unique(order.begin(), order.end()), order.end());
  }
  {
    std::vector<int32_t> u(order);
    std::sort(u.begin(), u.end());
    if (std::adjacent_find(u.begin(), u.end()) != u.end()) return einval("a node appears twice in node_sp");
    for (int j = 0; j < wl->n_items; ++j)
      if (!std::binary_search(u.begin(), u.end(), wl->sp[j])) return einval("an item's sp is missing from node_sp");
    std::vector<int32_t> s(wl->sp, wl->sp + wl->n_items);
    std::sort(s.begin(), s.end());
    for (int32_t v : u)
      if (!std::binary_search(s.begin(), s.end(), v)) return einval("node_sp names an sp no item has");
  }
  const bool fwd = phases & NSP_STEP_FORWARD, bwd = phases & NSP_STEP_BACKWARD;
  if (fwd && (!b->q_seq || !b->k_seq || !b->v_seq || !b->o_seq || !b->q || !b->k || !b->v || !b->o || !b->lse))
    return einval("a buffer of the forward phases is NULL");
  if (bwd && (!b->do_seq || !b->dq_seq || !b->dk_seq || !b->dv_seq || !b->q || !b->k || !b->v || !b->o ||
              !b->lse || !b->dout || !b->dq || !b->dk || !b->dv))
    return einval("a buffer of the backward phases is NULL");

  const size_t n = order.size();
  std::vector<std::vector<uint8_t>> masks(n, std::vector<uint8_t>(std::max(1, wl->n_items), 0));
  std::vector<nsp_worklist> node(n, *wl);
  for (size_t u = 0; u < n; ++u) {
    for (int j = 0; j < wl->n_items; ++j) masks[u][j] = wl->sp[j] == order[u];
    node[u].item_mask = masks[u].data();
  }
  EventPool pool;

  // one pass (forward or backward) over the nodes
  auto pass = [&](bool forward) -> nsp_status {
    std::vector<hipEvent_t> pro(n), cmp(n);
    for (size_t u = 0; u < n; ++u) {
      NSP_X_HIP(pool.make(&pro[u]));
      NSP_X_HIP(pool.make(&cmp[u]));
    }
    auto prologue = [&](size_t u) -> nsp_status {
      const nsp_worklist *w = &node[u];
      if (forward) {
        NSP_X_TRY(nsp_ulysses_pack(w, NSP_KIND_Q, NSP_BF16, b->q_seq, b->q, comm));
        NSP_X_TRY(nsp_ulysses_pack(w, NSP_KIND_KV, NSP_BF16, b->k_seq, b->k, comm));
        NSP_X_TRY(nsp_ulysses_pack(w, NSP_KIND_KV, NSP_BF16, b->v_seq, b->v, comm));
      } else {
        NSP_X_TRY(nsp_ulysses_pack(w, NSP_KIND_Q, NSP_BF16, b->do_seq, b->dout, comm));
      }
      NSP_X_HIP(hipEventRecord(pro[u], comm));
      return NSP_OK;
    };
    auto epilogue = [&](size_t u) -> nsp_status {
      const nsp_worklist *w = &node[u];
      NSP_X_HIP(hipStreamWaitEvent(comm, cmp[u], 0));
      if (forward) {
        NSP_X_TRY(nsp_ulysses_unpack(w, NSP_KIND_Q, NSP_BF16, NSP_UNPACK_SELECT, b->o, b->o_seq, comm));
      } else {
        NSP_X_TRY(nsp_ulysses_unpack(w, NSP_KIND_Q, NSP_BF16, NSP_UNPACK_SELECT, b->dq, b->dq_seq, comm));
        NSP_X_TRY(nsp_ulysses_unpack(w, NSP_KIND_KV, NSP_BF16, NSP_UNPACK_SUM, b->dk, b->dk_seq, comm));
        NSP_X_TRY(nsp_ulysses_unpack(w, NSP_KIND_KV, NSP_BF16, NSP_UNPACK_SUM, b->dv, b->dv_seq, comm));
      }
      return NSP_OK;
    };
    auto compute_phase = [&](size_t u) -> nsp_status {
      const nsp_worklist *w = &node[u];
      NSP_X_HIP(hipStreamWaitEvent(compute, pro[u], 0));
      if (forward)
        NSP_X_TRY(nsp_varlen_attn_fwd(w, softmax_scale, 1, b->q, b->k, b->v, b->o, NSP_BF16, b->lse, compute));
      else
        NSP_X_TRY(nsp_varlen_attn_bwd(w, softmax_scale, 1, b->q, b->k, b->v, b->o, NSP_BF16, b->dout, b->lse,
                                      b->dq, b->dk, b->dv, NSP_BF16, b->workspace, b->ws_bytes,
                                      compute));
      NSP_X_HIP(hipEventRecord(cmp[u], compute));
      return NSP_OK;
    };
    // comm queue: pro(0), pro(1), epi(0), pro(2), epi(1), ..., epi(n-1);
    // compute queue: cmp(0), cmp(1), ...
    if (n > 0) NSP_X_TRY(prologue(0));
    for (size_t u = 0; u < n; ++u) {
      NSP_X_TRY(compute_phase(u));
      if (u + 1 < n) NSP_X_TRY(prologue(u + 1));
      NSP_X_TRY(epilogue(u));
    }
    return NSP_OK;
  };
  if (fwd) NSP_X_TRY(pass(true));
  if (bwd) NSP_X_TRY(pass(false));
  // the step is complete when `compute` is: it waits for the last epilogue
  if (comm != compute) {
    hipEvent_t done;
    NSP_X_HIP(pool.make(&done));
    NSP_X_HIP(hipEventRecord(done, comm));
    NSP_X_HIP(hipStreamWaitEvent(compute, done, 0));
  }
  return NSP_OK;
}
