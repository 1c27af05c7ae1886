/*
 * nsp.h -- C ABI of libnsp.so: the per-GPU hot path of Nested Sequence
 * Parallelism (NSP) on AMD Instinct MI355X (gfx950).
 *
 * NSP routes each sequence of a packed, variable-length batch to one node of
 * an SP tree (Design, Definition 1); a node at Ulysses degree sp shards its
 * sequences over sp GPUs.  After the Ulysses exchange every GPU holds complete
 * sequences for a subset of heads (Background, Sequence Parallelism), so one
 * GPU's share is a packed work list of items
 *     (L_j tokens, query heads [q_lo, q_hi), KV heads [kv_lo, kv_hi), sp_j)
 * over which it runs causal grouped-query attention locally, forward and
 * backward.  This library provides the compute routines and the local halves
 * of the communication prologue / epilogue of the SP-backend interface the
 * paper describes (Implementation, execution engine; Design, SP-backend
 * phase costs):
 *
 *     nsp_ulysses_pack     sequence-sharded -> head-sharded layout (prologue)
 *     nsp_varlen_attn_fwd  attention forward (compute)
 *     nsp_varlen_attn_bwd  attention backward (compute)
 *     nsp_ulysses_unpack   head-sharded -> sequence-sharded layout (epilogue)
 *
 * Conventions shared by every call
 *   - Every data pointer is DEVICE memory owned by the caller; the nsp_worklist
 *     and its arrays are HOST memory, read during the call only.
 *   - Calls enqueue work on `stream` and return without synchronising.
 *   - Outputs are fully overwritten (the selected items' parts, with an item
 *     mask), never accumulated into.
 *   - All arguments are validated before anything is launched; on any error
 *     nothing is launched and outputs are untouched.  nsp_last_error() then
 *     returns a thread-local message naming the offending argument.
 *   - Element offsets are 64-bit; a tensor may exceed 2^31 elements.
 *   - The library allocates no device memory except an internally owned,
 *     cached copy of each work list's tile schedule (a few KB to a few MB),
 *     keyed by the work list's contents and the device.  The cache is
 *     guarded by a mutex and its entries are reference counted (an entry
 *     evicted while another thread's call still uses it is freed after that
 *     call has enqueued its kernels); calls are reentrant.  Two file-scope
 *     device arrays live with the library on every GPU it runs on: the
 *     scratch of nsp_varlen_attn_bwd_noalloc, and 4096 blocks of 64 bytes of
 *     unit-queue counters for the forward, one block per stream that has run
 *     a forward (calls on one stream run in order and share it; calls on
 *     other streams use other blocks; past 4096 streams a call runs without
 *     one, one workgroup per unit).
 *   - Data pointers must be 16-byte aligned (NSP_EINVAL otherwise).
 *
 * Attention layout ("head layout"): item j's Q, O, dO, dQ block is
 * [L_j][hq_j][D] (token-major, heads, head_dim) at element offset
 * D * sum_{i<j} L_i * hq_i; K, V, dK, dV blocks are [L_j][hkv_j][D] at
 * D * sum_{i<j} L_i * hkv_i; LSE is float32 [hq_j][L_j] at sum_{i<j} hq_i L_i,
 * where hq_j = q_hi - q_lo and hkv_j = kv_hi - kv_lo.
 */
#ifndef NSP_H_
#define NSP_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t nsp_status;
#define NSP_OK 0
#define NSP_EINVAL 1          /* invalid argument (see nsp_last_error) */
#define NSP_EUNSUPPORTED 2    /* valid but not implemented (head_dim, causal=0) */
#define NSP_EHIP 3            /* a HIP runtime call or kernel launch failed */
#define NSP_ENOMEM 4          /* the schedule cache could not allocate */
#define NSP_EWORKSPACE 5      /* workspace missing or smaller than required */
#define NSP_EINFEASIBLE 6     /* no SP-tree plan of the batch meets the token budget */

typedef enum { NSP_BF16 = 0, NSP_F32 = 1 } nsp_dtype;
typedef enum { NSP_KIND_Q = 0, NSP_KIND_KV = 1 } nsp_kind;
typedef enum { NSP_UNPACK_SELECT = 0, NSP_UNPACK_SUM = 1 } nsp_replica;

/*
 * One GPU's packed work list.
 *   n_items      >= 0
 *   cu_seqlens   n_items+1 prefix sums of L_j in the attention layout;
 *                cu_seqlens[0] == 0, non-decreasing (L_j == 0 is a no-op item)
 *   q_heads      n_items x 2: [lo, hi) global query heads of item j on this GPU
 *   kv_heads     n_items x 2: [lo, hi) global KV heads of item j on this GPU;
 *                every local query head h must map to a local KV head,
 *                floor(h * hkv_total / hq_total) in [kv_lo, kv_hi)
 *   sp           n_items Ulysses degrees (power of two); read by pack/unpack
 *                only, may be NULL for the attention calls
 *   hq_total, hkv_total   global head counts, hq_total % hkv_total == 0
 *   head_dim     D; 64 or 128 supported
 *   item_mask    NULL (every item), or n_items bytes: only the items j with
 *                item_mask[j] != 0 are computed / moved by a call.  Offsets
 *                and sizes are still those of the whole work list, and the
 *                other items' parts of every output are left untouched.  An
 *                item's results do not depend on which other items a call
 *                selects (each item is tiled on its own), so a masked call
 *                reproduces the selected items of an unmasked one bit for
 *                bit.  This serves the per-node issue of inter-level phase
 *                streaming and the regeneration of RECOMPUTE items' outputs
 *                (Design, NSP Executor).
 */
typedef struct {
  int32_t n_items;
  const int32_t *cu_seqlens;
  const int32_t *q_heads;
  const int32_t *kv_heads;
  const int32_t *sp;
  int32_t hq_total;
  int32_t hkv_total;
  int32_t head_dim;
  const uint8_t *item_mask;
} nsp_worklist;

/*
 * Causal attention forward over every item (Background, Sequence Packing: no
 * attention across items; Background, Sequence Parallelism: local attention
 * over complete sequences for this GPU's heads).  For item j, local query head
 * i (global h = q_lo + i) and its KV head g = floor(h*hkv_total/hq_total):
 *     S[t,s] = softmax_scale * <Q[t,i,:], K[s,g-kv_lo,:]>, s <= t
 *     lse[t] = log sum_{s<=t} exp(S[t,s])          (natural log, float32)
 *     O[t,i] = sum_{s<=t} exp(S[t,s] - lse[t]) V[s,g-kv_lo]
 *   q, k, v   bf16, attention layout
 *   o         o_dtype (NSP_BF16: the float32 result rounded to nearest even;
 *             NSP_F32: the float32 result), attention layout
 *   lse       float32 [hq_j][L_j] per item (needed by the backward)
 *   causal    must be 1 (0 returns NSP_EUNSUPPORTED)
 * Errors: NSP_EINVAL (work list, null/misaligned pointers), NSP_EUNSUPPORTED
 * (head_dim, causal), NSP_ENOMEM, NSP_EHIP.
 */
nsp_status nsp_varlen_attn_fwd(const nsp_worklist *wl, float softmax_scale, int32_t causal,
                               const void *q, const void *k, const void *v,
                               void *o, nsp_dtype o_dtype, float *lse, hipStream_t stream);

/* Bytes of device workspace nsp_varlen_attn_bwd needs for this work list (0
 * if the work list is invalid): -Delta[t] = -<dO[t], O[t]> and lse*log2(e)
 * (float32, laid out like lse, each part 256-byte aligned) and 256 bytes of
 * unit-queue heads for the persistent passes.  A call uses the workspace
 * from its first kernel to its last, so two calls that run at the same time
 * need two workspaces. */
size_t nsp_varlen_attn_bwd_workspace(const nsp_worklist *wl);

/*
 * Causal attention backward (the analytic gradient of the forward above):
 *     P = exp(S - lse), Delta[t] = <dO[t,i], O[t,i]>,
 *     dP[t,s] = <dO[t,i], V[s,g]>, dS = P * (dP - Delta),
 *     dQ[t,i] = scale * sum_s dS[t,s] K[s,g]
 *     dK[s,g] = scale * sum over local i->g, t of dS[t,s] Q[t,i]
 *     dV[s,g] = sum over local i->g, t of P[t,s] dO[t,i]
 * dK/dV of a KV head are summed over the local query heads that share it
 * only; for a KV head replicated across ranks (hkv_total < sp) they are this
 * rank's partial sums (see nsp_ulysses_unpack NSP_UNPACK_SUM).
 *   q, k, v, dout   bf16, attention layout; o in o_dtype; lse from the forward
 *   dq, dk, dv      grad_dtype (NSP_BF16 rounded to nearest even, or NSP_F32)
 *   workspace       device memory of at least nsp_varlen_attn_bwd_workspace(wl)
 *                   bytes, 256-byte aligned; contents on entry are ignored
 * Deterministic: no atomics on data, every output element written by one
 * lane, so results are bitwise repeatable run to run (dQ is a pass of its own
 * that recomputes S and dP, instead of float32 atomics from the dK/dV pass).
 * Errors: as the forward, plus NSP_EWORKSPACE.
 */
nsp_status nsp_varlen_attn_bwd(const nsp_worklist *wl, float softmax_scale, int32_t causal,
                               const void *q, const void *k, const void *v,
                               const void *o, nsp_dtype o_dtype, const void *dout, const float *lse,
                               void *dq, void *dk, void *dv, nsp_dtype grad_dtype,
                               void *workspace, size_t ws_bytes, hipStream_t stream);

/*
 * Allocation-free variant of nsp_varlen_attn_bwd, for callers that cannot
 * allocate device memory: code being captured into a HIP graph, tight
 * serving loops, harnesses that forbid allocation.  Same arguments, results
 * (bit for bit) and errors as nsp_varlen_attn_bwd, without the workspace:
 * the backward workspace and the work list's unit schedule live in a
 * file-scope device array of NSP_NOALLOC_SCRATCH_BYTES that the library
 * holds on every GPU it runs on until the process ends; the call allocates
 * nothing on the device (the schedule is built on the host, kept in a
 * host-side cache, and copied into the array on `stream` when the array does
 * not already hold it).  Limits: sum_j L_j * hq_j <= NSP_NOALLOC_MAX_ROWS
 * (-Delta and lse*log2(e), float32, in 88 MiB) and a schedule of at most
 * 8 MiB (about 500000 work units); larger work lists return NSP_EWORKSPACE
 * with nothing launched.  Every call on a GPU uses that GPU's one array and
 * leaves its contents behind: calls that overlap in time on one GPU (on
 * different streams, or from different threads without ordering) race and
 * must not be issued.
 */
#define NSP_NOALLOC_SCRATCH_BYTES (96u << 20)
#define NSP_NOALLOC_MAX_ROWS 11534272
nsp_status nsp_varlen_attn_bwd_noalloc(const nsp_worklist *wl, float softmax_scale, int32_t causal,
                                       const void *q, const void *k, const void *v,
                                       const void *o, nsp_dtype o_dtype, const void *dout, const float *lse,
                                       void *dq, void *dk, void *dv, nsp_dtype grad_dtype, hipStream_t stream);

/*
 * Ulysses prologue, local half (Background, Sequence Parallelism): re-lay a
 * sequence-sharded tensor as the head-sharded one the exchange delivers.
 * For kind NSP_KIND_Q the head count is H = hq_total, for NSP_KIND_KV
 * H = hkv_total.  Per item j with n = L_j / sp_j, H_loc = H/sp_j if H >= sp_j
 * else 1, and head(s,h') = s*H_loc + h' (H >= sp_j) or floor(s*H/sp_j):
 *     x_seq  : item j at token offset sum_{i<j} L_i/sp_i, [n][H][D]
 *     x_head : item j at element offset D * sum_{i<j} L_i*H_loc(i), [L_j][H_loc][D]
 *     x_head[j][s*n + t][h'][:] = x_seq[c_j + t][head(s,h')][:]
 * i.e. the sp per-destination chunks laid out where the exchange lands them
 * (with the exchange the identity on one GPU).  Bits are moved unchanged.
 * Requirements: sp_j a power of two, L_j % sp_j == 0, H % sp_j == 0 or
 * sp_j % H == 0, and the work list's head-range width of that kind equals
 * H_loc(j) (so x_head is the attention layout).
 *   dtype   element type of both tensors (NSP_BF16 or NSP_F32)
 */
nsp_status nsp_ulysses_pack(const nsp_worklist *wl, nsp_kind kind, nsp_dtype dtype,
                            const void *x_seq, void *x_head, hipStream_t stream);

/*
 * Ulysses epilogue, local half: the inverse of nsp_ulysses_pack.  For
 * H >= sp_j it is the exact inverse permutation.  For H < sp_j (KV head g is
 * replicated in the blocks s with head(s,0) == g):
 *   NSP_UNPACK_SELECT  x_seq[c_j+t][g] = x_head[j][s_g*n + t][0], s_g = g*sp_j/H
 *   NSP_UNPACK_SUM     x_seq[c_j+t][g] = sum of those replicas in float32, in
 *                      increasing s, rounded once to bf16 (nearest even) for
 *                      NSP_BF16 data -- the replica reduction of dK/dV.
 */
nsp_status nsp_ulysses_unpack(const nsp_worklist *wl, nsp_kind kind, nsp_dtype dtype,
                              nsp_replica replica, const void *x_head, void *x_seq,
                              hipStream_t stream);

/*
 * Tree-level recomputation plan (Design, NSP Executor, Tree-Level
 * Recomputation).  Host-only; no device work.  The SP tree is walked from the
 * root toward the leaves -- on one GPU's path, the nodes in decreasing order
 * of sp_j, every item of a node sharing its sp -- accumulating the bytes of
 * the attention-output slices this GPU would keep for the backward (O in
 * o_dtype plus the float32 LSE: L_j * hq_j * (head_dim * size(o_dtype) + 4)).
 * A node that fits in what is left of `budget_bytes` is marked SAVE whole.
 * The first node that does not fit is split by sample: its items are taken in
 * decreasing order of recomputation cost per saved byte (the attention
 * forward cost 4 * head_dim * hq_j * L_j (L_j + 1) / 2 per byte, i.e. longest
 * first; ties by index) and each one that still fits is saved.  Every item of
 * the nodes below is marked RECOMPUTE.
 *   budget_bytes  >= 0
 *   save          out, n_items bytes: 1 = SAVE, 0 = RECOMPUTE (items with
 *                 L_j = 0 hold nothing and are marked SAVE)
 *   saved_bytes   out (may be NULL): bytes of the SAVE slices
 * The RECOMPUTE items' outputs are regenerated before the backward by
 * nsp_varlen_attn_fwd with item_mask = the complement of `save`.
 * Requires wl->sp.  The work list's item_mask is ignored.
 * Errors: NSP_EINVAL.
 */
nsp_status nsp_recompute_plan(const nsp_worklist *wl, int64_t budget_bytes, nsp_dtype o_dtype, uint8_t *save,
                              int64_t *saved_bytes);

/*
 * The work units the attention calls launch for a work list, in launch
 * order (host only; no device work).  This is the schedule step between the
 * work list and the kernels: it balances items of very different L_j over
 * the compute units (Design, NSP Executor: the per-GPU compute of one SP-tree
 * share; Background: the quadratic cost of long sequences), and it is
 * exposed so that it can be inspected and checked without a GPU.
 *   which = NSP_SCHED_FWD: forward and dQ units, one per (item j, 256-row
 *           query tile m, local query head i): {j, m, i, g}, g = the local KV
 *           head of i.  Work: the keys the tile attends, min(L_j, 256 (m+1)).
 *   which = NSP_SCHED_KV: dK/dV units, one per (item j, local KV head g,
 *           128-key tile n): {j, n | (desc << 30), i0 | (i1 << 16), g},
 *           [i0, i1) the local query heads that use g (empty if none: the
 *           unit writes zeros).  Work: the 64-row query tiles at or past the
 *           key tile's first row, times max(1, i1 - i0); the unit takes them
 *           tile by tile, every query head of a tile in turn, up from its
 *           diagonal, or down from the item end when desc = 1.
 *   Forward/dQ units are generated item by item (m, then i) and sorted
 *   longest work first (stable).  Slot b of that list belongs to XCD b % 8:
 *   a one-shot grid's workgroup b starts there (the hardware deals
 *   workgroups round-robin over the 8 XCDs), and the persistent passes take
 *   slot b from the queue of XCD b % 8, their own XCD's queue first, the
 *   others' once it is empty.  When the longest scheduled item's K and V
 *   slices of one head (4 L_j head_dim bytes) exceed one XCD's L2 (4 MiB),
 *   every full chunk of 8 x 32 units gives XCD x one run of 32 consecutive
 *   units of the sorted order -- run x in even chunks, run 7 - x in odd
 *   ones -- so that units streaming the same K/V tiles share an XCD's L2;
 *   the last, incomplete chunk keeps the sorted order.  Otherwise the
 *   sorted order is launched as it is.
 *   dK/dV units are grouped into gangs per item: for n < nk/2 (nk key tiles)
 *   the pairs (n, nk-1-n) over the item's KV heads in order (g, then n), 32
 *   pairs a gang; a gang lists the 32 units n with desc = 1, then the
 *   partners nk-1-n with desc = 0 in increasing nk-1-n (ties in gang order);
 *   the middle tile of an odd nk goes, per KV head, into gangs of up to 32
 *   such tiles (desc = 0).  The item with the most work may leave its K
 *   first and K last tiles unpaired (K a whole number of gangs): the first
 *   in gangs of up to 32 (desc = 1), the last as gangs of one unit each.
 *   That happens when under 1% of the work is in gangs of at most a tenth
 *   of one compute unit's share of it (then K is the least that puts 2% of
 *   the work in the last tiles), and when a model of the persistent pass
 *   (256 compute units, 32 per XCD, each taking the next unit of its own
 *   queue, then of the others) ends more than 8% past an even split (then K
 *   is the candidate, from there to nk/2, with the earliest modelled end).
 *   Gangs are sorted by decreasing duration (the most steps one workgroup
 *   spends on the gang: a pair, or one unit; stable over items in order)
 *   and each goes, in that order, to the XCD with the least work so far
 *   (lowest index on ties); XCD x's queue is the concatenation of its
 *   gangs, and the queues are laid out one after another (see
 *   nsp_attn_kv_queues).  The persistent dK/dV pass takes its own XCD's
 *   queue first, the others' once it is empty; a one-shot grid (no more
 *   units than compute units) runs slot b in workgroup b.
 *   Items with L_j = 0 or outside wl->item_mask contribute no units.
 *   units     out, capacity x 4 int32 in the order above (may be NULL if
 *             capacity = 0: a size query)
 *   n_units   out: the number of units
 * Errors: NSP_EINVAL (work list, unknown `which`, NULL n_units, units NULL
 * or capacity < n_units other than in a size query; n_units is still set),
 * NSP_EUNSUPPORTED (head_dim).
 */
#define NSP_SCHED_FWD 0
#define NSP_SCHED_KV 1
nsp_status nsp_attn_schedule(const nsp_worklist *wl, int32_t which, int32_t *units, int64_t capacity,
                             int64_t *n_units);

/* The layout of the dK/dV unit queues of nsp_attn_schedule(NSP_SCHED_KV):
 * queue_off (out, 9 int32) such that XCD x's queue is units
 * [queue_off[x], queue_off[x + 1]) and queue_off[8] is the number of units.
 * Host only.  Errors: NSP_EINVAL (work list, NULL queue_off),
 * NSP_EUNSUPPORTED (head_dim). */
nsp_status nsp_attn_kv_queues(const nsp_worklist *wl, int32_t *queue_off);

/*
 * Buffers of one GPU's attention step for nsp_executor_step (all DEVICE
 * memory, bf16 unless noted; layouts as in nsp_ulysses_pack and the attention
 * calls).  Sequence-sharded: q_seq, k_seq, v_seq and do_seq are inputs,
 * o_seq, dq_seq, dk_seq and dv_seq outputs (dk/dv of replicated KV heads are
 * the replica sums).  Head-sharded work buffers: q, k, v, dout are written by
 * the prologues, o, lse (float32) by the forward, dq, dk, dv by the backward;
 * workspace as nsp_varlen_attn_bwd needs it.
 */
typedef struct {
  const void *q_seq, *k_seq, *v_seq, *do_seq;
  void *o_seq, *dq_seq, *dk_seq, *dv_seq;
  void *q, *k, *v, *o, *dout, *dq, *dk, *dv;
  float *lse;
  void *workspace;
  size_t ws_bytes;
} nsp_step_buffers;

#define NSP_STEP_FORWARD 1
#define NSP_STEP_BACKWARD 2

/*
 * Inter-level phase streaming (Design, NSP Executor, Inter-level Phase
 * Streaming).  The SP-tree nodes on this GPU's path -- the items sharing one
 * sp value -- are issued in the order `node_sp` (n_nodes distinct sp values
 * covering every item; NULL = root first, i.e. decreasing sp).  Each node
 * runs the three backend phases, communication prologue (pack), attention
 * compute, communication epilogue (unpack), as item-masked calls: compute on
 * `compute`, prologues and epilogues on `comm`, in the paper's queue
 * discipline -- within a node the phases keep their order across the two
 * queues (events), across nodes each queue follows the issue order, and the
 * comm queue takes the prologue of node u+1 before the epilogue of node u,
 * so that the prologue of u+1 runs during the compute of u and the epilogue
 * of u during the compute of u+1.
 *   phases   NSP_STEP_FORWARD: pack Q, K, V -> forward -> unpack O
 *            NSP_STEP_BACKWARD: pack dO -> backward -> unpack dQ, dK (sum),
 *            dV (sum); needs o and lse from a forward of the same items
 *            (both bits: forward then backward)
 * On return the work is enqueued; `compute` waits for the last epilogue, so
 * the step is complete when `compute` is.  The results are bitwise those of
 * the unmasked calls issued one after another.  `comm` may equal `compute`
 * (serial issue, the same results).  Requires wl->sp; the work list's own
 * item_mask must be NULL.
 * Errors: as the calls it makes; NSP_EINVAL when node_sp is not exactly the
 * set of the items' sp values (each once), or a buffer the phases need is
 * NULL.
 */
nsp_status nsp_executor_step(const nsp_worklist *wl, const int32_t *node_sp, int32_t n_nodes, int32_t phases,
                             float softmax_scale, const nsp_step_buffers *buf, hipStream_t compute,
                             hipStream_t comm);

/*
 * SP-tree routing, the NSP planner (Design, NSP Planner: SP Tree Topology,
 * Routing Objective and Cost Model, Routing Algorithm).  Host-only; no
 * device work.
 *
 * The SP tree over `world` = W = 2^K GPUs has nodes (d, i), 0 <= d <= K,
 * 0 <= i < 2^d; node (d, i) covers ranks [i W/2^d, (i+1) W/2^d) and has SP
 * degree W/2^d (leaves: single GPUs).  A plan maps each sample to one node.
 * Token load: Tok_p = sum over samples j whose node covers GPU p of
 * L_j / degree.  Cost model, with the coefficients the paper profiles
 * offline given here: a sample at a node of degree sp adds, on each GPU of
 * the node, the attention compute of Hq/sp query heads over the whole sample
 * (counted flops 4 D per causal pair forward, 10 D backward, at
 * attn_fwd_flops / attn_bwd_flops per second) and, for sp > 1, the Ulysses
 * all-to-all bytes of its phases (forward prologue Q, K, V; forward epilogue
 * O; backward prologue dO; backward epilogue dQ, dK, dV; L/sp tokens per
 * GPU, K/V/dK/dV counting max(Hkv, sp) heads, (sp-1)/sp of them sent over
 * min(sp-1, links) links of link_bytes per second) plus one a2a_latency per
 * phase per active node.  D_p(pass) = the node phases on p's leaf-to-root
 * path + Tok_p * dense_<pass>_per_token; C_p = D_p(fwd) + D_p(bwd);
 * load = max_p D_p(fwd) + max_p D_p(bwd).
 * Routing (Algorithm 1): samples by non-increasing length (stable); for each
 * of the first `prefix` samples every retained plan is extended to every
 * admissible node (degree <= sp_max dividing L_j and hq_total, dividing or
 * divisible by hkv_total, and, if
 * `monotone`, no larger than the degree of any placed longer sample; root
 * first, then by index), extensions with max_p Tok_p > token_budget are
 * dropped and the `beam` of smallest max_p C_p kept (stable); every retained
 * plan then takes the remaining samples longest first, each on the leaf of
 * least C_p among those within the budget, else on the leaf of least Tok_p
 * (lowest index among ties); the completed plan of least max_p C_p is
 * returned (first among ties).  Every per-node sum is an exact integer, so
 * the result does not depend on summation order.
 *   lengths       n sample lengths (host), 0 <= L_j <= 2^31
 *   node_depth,
 *   node_index    out, n each: the node (d, i) of every sample
 *   gpu_cost      out (may be NULL), world doubles: C_p in seconds
 *   gpu_tokens    out (may be NULL), world doubles: Tok_p
 *   load          out (may be NULL): the iteration proxy in seconds
 * Errors: NSP_EINVAL (parameters; a batch whose exact sums could exceed
 * 2^62), NSP_EINFEASIBLE (no placement of a prefix sample meets the token
 * budget; outputs untouched).
 */
typedef struct {
  int32_t world;                 /* GPUs, a power of two */
  int32_t sp_max;                /* largest SP degree, a power of two <= world */
  int32_t hq_total, hkv_total;   /* model query / KV heads, hq_total % hkv_total == 0 */
  int32_t head_dim, elem_bytes;  /* elem_bytes: bytes per exchanged element */
  double attn_fwd_flops;         /* counted flop/s of one GPU's attention, forward (> 0, may be inf) */
  double attn_bwd_flops;         /* the same, backward */
  double link_bytes;             /* bytes/s of one GPU-GPU link (> 0, may be inf) */
  int32_t links;                 /* links per GPU (>= 1) */
  double a2a_latency;            /* seconds per all-to-all (>= 0) */
  double dense_fwd_per_token;    /* seconds per token of the non-attention work, forward (>= 0) */
  double dense_bwd_per_token;    /* the same, backward */
  double token_budget;           /* B_tok, tokens per GPU (> 0, may be inf) */
  int32_t prefix;                /* k: samples placed by the beam search (>= 0) */
  int32_t beam;                  /* w: partial plans kept (>= 1) */
  int32_t monotone;              /* 1: longer samples never take a smaller SP degree */
} nsp_plan_params;

nsp_status nsp_sp_tree_plan(const nsp_plan_params *prm, const int64_t *lengths, int32_t n, int32_t *node_depth,
                            int32_t *node_index, double *gpu_cost, double *gpu_tokens, double *load);

/*
 * GPU `gpu`'s work list under a plan, in nsp_worklist form: the samples
 * whose node covers the GPU, root first (decreasing degree), then in sample
 * order.  For item m: sample[m] = its sample index; cu_seqlens = prefix sums
 * of L (cu_seqlens[0] = 0; the attention layout, full sequences); sp[m] = the
 * node's degree; with r the GPU's rank within the node, q_heads[2m..2m+1] =
 * [r hq/sp, (r+1) hq/sp) and kv_heads[2m..2m+1] = [r hkv/sp, (r+1) hkv/sp),
 * or the one replicated KV head [floor(r hkv/sp), +1) when sp > hkv.
 * Capacities: n for sample and sp, n + 1 for cu_seqlens, 2n for the heads.
 *   n_items       out: items written
 * Errors: NSP_EINVAL (parameters, a node outside the tree or of a degree the
 * sample cannot run at, more than 2^31 - 1 tokens on the GPU).
 */
nsp_status nsp_sp_tree_worklist(const nsp_plan_params *prm, const int64_t *lengths, int32_t n,
                                const int32_t *node_depth, const int32_t *node_index, int32_t gpu, int32_t *n_items,
                                int32_t *sample, int32_t *cu_seqlens, int32_t *q_heads, int32_t *kv_heads,
                                int32_t *sp);

/*
 * Kernel timing (instrumentation, off by default).  While enabled, every
 * kernel this library launches is bracketed by a pair of hipEvents recorded
 * on the launch's stream, so the measured time is the device time of that
 * kernel alone.  nsp_timing_query waits for the recorded events, folds them
 * into per-kernel totals and returns the launch count and total milliseconds
 * since the last nsp_timing_reset for one kernel name: "attn_fwd",
 * "bwd_preprocess", "bwd_dkdv", "bwd_dq" or "relayout".
 * Errors: NSP_EINVAL (unknown name or NULL outputs), NSP_EHIP.
 */
nsp_status nsp_timing_enable(int32_t enable);
nsp_status nsp_timing_reset(void);
nsp_status nsp_timing_query(const char *kernel, int64_t *launches, double *total_ms);

/*
 * Matrix-core throughput ceiling of the current device (instrumentation; not
 * part of the method).  Every SIMD runs waves_per_simd (1 or 2) waves that
 * issue nothing but bf16 v_mfma_f32_32x32x16 products from registers, four
 * independent accumulators, products_per_simd products per SIMD (a positive
 * multiple of 16 x waves_per_simd, at most 2^24); operands approximately
 * standard normal in bf16, or zeros when zero_operands != 0; pattern 0: both
 * operands change from one product to the next, 1 / 2: the first held for two
 * / four products, 3: the same operands throughout.  One warm-up launch, then
 * one timed launch (hipEvents) on the null stream; waits for it.  seconds
 * (out): the timed launch; tflops (out): its dense bf16 rate.  Under load the
 * device's power limit sets its clock, so with random operands this is the
 * most a kernel can execute with such data, typically well under the nominal
 * peak.
 * Errors: NSP_EINVAL (arguments, NULL outputs), NSP_EHIP.
 */
nsp_status nsp_mfma_ceiling(int32_t pattern, int32_t zero_operands, int32_t waves_per_simd,
                            int64_t products_per_simd, double *seconds, double *tflops);

/* Static description of a status code. */
const char *nsp_status_string(nsp_status status);

/* Thread-local detail of the last error returned on this thread ("" if none). */
const char *nsp_last_error(void);

/* Library version string. */
const char *nsp_version(void);

#ifdef __cplusplus
}
#endif

#endif /* NSP_H_ */
