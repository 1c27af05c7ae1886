// libnsp C ABI: argument validation, work-list -> tile schedule, schedule
// cache and kernel dispatch.  See include/nsp.h for the contract.
#include "nsp.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <memory>
#include <mutex>
#include <queue>
#include <string>
#include <tuple>
#include <unordered_map>
#include <vector>

#include "nsp_internal.hpp"
#include "sched_cache.hpp"

using nsp::CopyTask;
using nsp::ItemDesc;

namespace {

thread_local std::string g_last_error;

nsp_status fail(nsp_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

}  // namespace

hipError_t nsp::compute_units(int *cus) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  static std::mutex mu;
  static std::unordered_map<int, int> known;
  std::lock_guard<std::mutex> lock(mu);
  auto it = known.find(dev);
  if (it == known.end()) {
    int n = 0;
    e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    it = known.emplace(dev, n > 0 ? n : 1).first;
  }
  *cus = it->second;
  return hipSuccess;
}

int32_t nsp::set_error(int32_t status, const char *fmt, ...) {
  char buf[512];
  buf[0] = 0;
  if (fmt) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
  }
  g_last_error = buf;
  return status;
}

namespace {

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

// Whether item j takes part in a call (every item when there is no mask).
bool selected(const nsp_worklist *wl, int j) { return !wl->item_mask || wl->item_mask[j] != 0; }
bool misaligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) != 0; }

// ------------------------------------------------------------ validation --

struct WlInfo {
  int64_t q_elems = 0, kv_elems = 0, lse_elems = 0;
};

nsp_status validate_worklist(const nsp_worklist *wl, WlInfo *info) {
  if (!wl) return fail(NSP_EINVAL, "work list is NULL");
  if (wl->n_items < 0) return fail(NSP_EINVAL, "n_items = %d < 0", wl->n_items);
  if (wl->hq_total <= 0 || wl->hkv_total <= 0)
    return fail(NSP_EINVAL, "head totals must be positive (hq_total=%d, hkv_total=%d)", wl->hq_total,
                wl->hkv_total);
  if (wl->hq_total % wl->hkv_total != 0)
    return fail(NSP_EINVAL, "hq_total %d is not a multiple of hkv_total %d", wl->hq_total, wl->hkv_total);
  if (wl->head_dim != 64 && wl->head_dim != 128)
    return fail(NSP_EUNSUPPORTED, "head_dim %d not supported (64 or 128)", wl->head_dim);
  if (wl->n_items > 0 && (!wl->cu_seqlens || !wl->q_heads || !wl->kv_heads))
    return fail(NSP_EINVAL, "cu_seqlens, q_heads and kv_heads must be non-NULL");
  if (wl->n_items > 0 && wl->cu_seqlens[0] != 0)
    return fail(NSP_EINVAL, "cu_seqlens[0] = %d, must be 0", wl->cu_seqlens[0]);
  WlInfo w;
  for (int j = 0; j < wl->n_items; ++j) {
    const int64_t L = (int64_t)wl->cu_seqlens[j + 1] - wl->cu_seqlens[j];
    if (L < 0) return fail(NSP_EINVAL, "cu_seqlens decreases at item %d", j);
    const int ql = wl->q_heads[2 * j], qh = wl->q_heads[2 * j + 1];
    const int kl = wl->kv_heads[2 * j], kh = wl->kv_heads[2 * j + 1];
    if (!(0 <= ql && ql < qh && qh <= wl->hq_total))
      return fail(NSP_EINVAL, "item %d: query head range [%d, %d) invalid for hq_total %d", j, ql, qh,
                  wl->hq_total);
    if (!(0 <= kl && kl < kh && kh <= wl->hkv_total))
      return fail(NSP_EINVAL, "item %d: KV head range [%d, %d) invalid for hkv_total %d", j, kl, kh,
                  wl->hkv_total);
    for (int hh : {ql, qh - 1}) {   // kv(h) is monotone: the range ends suffice
      const int g = (int)(((int64_t)hh * wl->hkv_total) / wl->hq_total);
      if (g < kl || g >= kh)
        return fail(NSP_EINVAL, "item %d: query head %d uses KV head %d outside [%d, %d)", j, hh, g, kl, kh);
    }
    w.q_elems += L * (qh - ql) * wl->head_dim;
    w.kv_elems += L * (kh - kl) * wl->head_dim;
    w.lse_elems += L * (qh - ql);
  }
  if (info) *info = w;
  return NSP_OK;
}

nsp_status validate_relayout(const nsp_worklist *wl, nsp_kind kind, nsp_dtype dtype) {
  if (kind != NSP_KIND_Q && kind != NSP_KIND_KV) return fail(NSP_EINVAL, "unknown kind %d", (int)kind);
  if (dtype != NSP_BF16 && dtype != NSP_F32) return fail(NSP_EINVAL, "unknown dtype %d", (int)dtype);
  if (wl->n_items > 0 && !wl->sp) return fail(NSP_EINVAL, "sp must be non-NULL for pack/unpack");
  const int H = kind == NSP_KIND_Q ? wl->hq_total : wl->hkv_total;
  const int32_t *rng = kind == NSP_KIND_Q ? wl->q_heads : wl->kv_heads;
  for (int j = 0; j < wl->n_items; ++j) {
    const int64_t L = (int64_t)wl->cu_seqlens[j + 1] - wl->cu_seqlens[j];
    const int s = wl->sp[j];
    if (!is_pow2(s)) return fail(NSP_EINVAL, "item %d: sp = %d is not a power of two", j, s);
    if (L % s != 0) return fail(NSP_EINVAL, "item %d: L = %lld is not a multiple of sp = %d", j, (long long)L, s);
    if (!(H % s == 0 || s % H == 0))
      return fail(NSP_EINVAL, "item %d: sp = %d and head count %d do not divide", j, s, H);
    const int hl = H >= s ? H / s : 1;
    if (rng[2 * j + 1] - rng[2 * j] != hl)
      return fail(NSP_EINVAL, "item %d: head range width %d != H/sp = %d", j, rng[2 * j + 1] - rng[2 * j], hl);
  }
  return NSP_OK;
}

// ----------------------------------------------------- schedule building --

struct HostAttnSched {
  std::vector<ItemDesc> items;
  std::vector<int4> fwd_units, kv_units;
  std::vector<int> kv_qoff;     // kXcdQueues + 1 entries: the dK/dV queue of XCD x is kv_units[kv_qoff[x] ..)
  std::vector<nsp::PreBlock> pre_blocks;
  int64_t q_rows = 0;
};

// Longest-processing-time order: units sorted by descending cost so that the
// dispatcher (which hands out workgroups in index order) starts the longest
// units first and the short ones fill in behind them.
void lpt_sort(std::vector<int4> &units, std::vector<int64_t> &cost) {
  std::vector<size_t> idx(units.size());
  for (size_t i = 0; i < idx.size(); ++i) idx[i] = i;
  std::stable_sort(idx.begin(), idx.end(), [&](size_t a, size_t b) { return cost[a] > cost[b]; });
  std::vector<int4> out(units.size());
  for (size_t i = 0; i < idx.size(); ++i) out[i] = units[idx[i]];
  units.swap(out);
}

// Workgroups are dispatched round-robin over the 8 XCDs of an MI355X
// (workgroup b starts on XCD b % 8, each XCD with its own L2).  Units that
// are adjacent in LPT order stream the same K/V (forward, dQ) or Q/dO (dK/dV)
// tiles at about the same time, so they should share an XCD: in chunk
// c = b/(8G), launch slot b runs the (b/8)%G-th of the G consecutive units
// given to XCD b%8.  XCDs take their G-runs in alternating order from chunk
// to chunk, so that no XCD always receives the most expensive run.  The
// incomplete last chunk keeps the LPT order; G <= 0 leaves the whole list in
// LPT order.
constexpr int kNumXcd = 8;

void xcd_group(std::vector<int4> &units, int G) {
  if (G <= 0) return;
  const size_t chunk = (size_t)kNumXcd * G;
  const size_t full = units.size() / chunk * chunk;
  std::vector<int4> out(units);
  for (size_t b = 0; b < full; ++b) {
    const size_t c = b / chunk, x = b % kNumXcd, j = (b / kNumXcd) % G;
    const size_t run = (c & 1) ? (kNumXcd - 1 - x) : x;
    out[b] = units[c * chunk + run * G + j];
  }
  units.swap(out);
}

constexpr int64_t kXcdL2Bytes = 4 << 20;   // L2 of one MI355X XCD

// Bytes of the largest tile stream of a call: the two bf16 [L, D] head
// slices (K and V, or Q and dO) of its longest scheduled item.
int64_t max_stream_bytes(const nsp_worklist *wl) {
  int64_t L = 0;
  for (int j = 0; j < wl->n_items; ++j)
    if (selected(wl, j)) L = std::max<int64_t>(L, (int64_t)wl->cu_seqlens[j + 1] - wl->cu_seqlens[j]);
  return 2 * 2 * L * wl->head_dim;
}

// dK/dV gangs.  The unit of key tile n streams the Q / dO tiles of its
// group's query heads from the tile's diagonal (query tile 2n) to the item
// end, and the units of an item's key tiles stream the same tiles: they hit
// in one XCD's L2 only when they read the same tile at about the same time.
// Units that start together at the same tile stay together while they run at
// the same speed, and key tiles n and nk-1-n together take a fixed number of
// steps, the same for every pair of the item.  A gang is up to kKvGang such
// pairs of one item (across its KV heads): first the units of the tiles n,
// which take their query tiles from the item end down to their diagonals
// (all start at the last tile), then the units of the partners nk-1-n, which
// go from their diagonals up to the end, longest first.  The workgroup that
// finishes first (shortest first unit, largest n) takes the longest partner,
// the smallest nk-1-n, and so on: each workgroup runs one pair, all pairs
// end at the same time, and the partners read every tile in step (a
// workgroup whose first unit was two tiles shorter starts its partner two
// tiles' steps earlier and two tiles lower).  The middle tile of an odd nk
// goes into gangs of its own.
struct KvGang {
  int64_t cost = 0;   // steps of all its units
  int64_t dur = 0;    // steps of one workgroup's share: a pair, or one middle tile
  std::vector<int4> units;
  std::vector<int64_t> steps;   // steps of each unit
};

using ItemGangs = std::vector<std::pair<int, std::vector<KvGang>>>;

void add_kv_gangs(std::vector<KvGang> &gangs, const nsp_worklist *wl, int j, int L, int K) {
  const int ql = wl->q_heads[2 * j], hq = wl->q_heads[2 * j + 1] - ql;
  const int kl = wl->kv_heads[2 * j], hkv = wl->kv_heads[2 * j + 1] - kl;
  const int nk = (L + nsp::kBwdBN - 1) / nsp::kBwdBN;
  const int nqt = (L + nsp::kBwdBM - 1) / nsp::kBwdBM;
  auto tiles = [&](int n) { return (int64_t)nqt - (int64_t)n * nsp::kBwdBN / nsp::kBwdBM; };
  struct Tile {
    int g, n, heads;
    int64_t w;
  };
  std::vector<Tile> firsts, mids, leads, tails;
  K = std::min(K, nk / 2);
  for (int g = 0; g < hkv; ++g) {
    int i0 = hq, i1 = 0;   // local query heads of KV head g: contiguous range
    for (int i = 0; i < hq; ++i) {
      const int gi = (int)(((int64_t)(ql + i) * wl->hkv_total) / wl->hq_total) - kl;
      if (gi == g) { i0 = std::min(i0, i); i1 = std::max(i1, i + 1); }
    }
    if (i1 <= i0) i0 = i1 = 0;   // no query head: the unit writes zeros
    const int64_t w = std::max(1, i1 - i0);
    for (int n = 0; n < K; ++n) leads.push_back(Tile{g, n, i0 | (i1 << 16), w});
    for (int n = K; n < nk / 2; ++n) firsts.push_back(Tile{g, n, i0 | (i1 << 16), w});
    for (int n = nk - K; n < nk; ++n) tails.push_back(Tile{g, n, i0 | (i1 << 16), w});
    if (nk & 1) mids.push_back(Tile{g, nk / 2, i0 | (i1 << 16), w});
  }
  for (size_t p0 = 0; p0 < firsts.size(); p0 += nsp::kKvGang) {
    const size_t p1 = std::min(firsts.size(), p0 + (size_t)nsp::kKvGang);
    KvGang gang;
    for (size_t p = p0; p < p1; ++p) {
      const Tile &t = firsts[p];
      gang.units.push_back(int4{j, t.n | nsp::kKvDescending, t.heads, t.g});
      gang.steps.push_back(t.w * tiles(t.n));
      gang.cost += t.w * (tiles(t.n) + tiles(nk - 1 - t.n));
      gang.dur = std::max(gang.dur, t.w * (tiles(t.n) + tiles(nk - 1 - t.n)));
    }
    std::vector<size_t> idx;
    for (size_t p = p0; p < p1; ++p) idx.push_back(p);
    std::stable_sort(idx.begin(), idx.end(), [&](size_t a, size_t b) { return firsts[a].n > firsts[b].n; });
    for (size_t p : idx) {
      const Tile &t = firsts[p];
      gang.units.push_back(int4{j, nk - 1 - t.n, t.heads, t.g});
      gang.steps.push_back(t.w * tiles(nk - 1 - t.n));
    }
    gangs.push_back(std::move(gang));
  }
  for (size_t p0 = 0; p0 < leads.size(); p0 += nsp::kKvGang) {
    KvGang gang;
    for (size_t p = p0; p < std::min(leads.size(), p0 + (size_t)nsp::kKvGang); ++p) {
      gang.units.push_back(int4{j, leads[p].n | nsp::kKvDescending, leads[p].heads, leads[p].g});
      gang.steps.push_back(leads[p].w * tiles(leads[p].n));
      gang.cost += leads[p].w * tiles(leads[p].n);
      gang.dur = std::max(gang.dur, leads[p].w * tiles(leads[p].n));
    }
    gangs.push_back(std::move(gang));
  }
  for (const Tile &t : tails) {
    KvGang gang;
    gang.units.push_back(int4{j, t.n, t.heads, t.g});
    gang.cost = gang.dur = t.w * tiles(t.n);
    gang.steps.push_back(gang.cost);
    gangs.push_back(std::move(gang));
  }
  for (size_t p0 = 0; p0 < mids.size(); p0 += nsp::kKvGang) {
    KvGang gang;
    for (size_t p = p0; p < std::min(mids.size(), p0 + (size_t)nsp::kKvGang); ++p) {
      gang.units.push_back(int4{j, mids[p].n, mids[p].heads, mids[p].g});
      gang.steps.push_back(mids[p].w * tiles(mids[p].n));
      gang.cost += mids[p].w * tiles(mids[p].n);
      gang.dur = std::max(gang.dur, mids[p].w * tiles(mids[p].n));
    }
    gangs.push_back(std::move(gang));
  }
}

// Gangs in decreasing order of the steps one workgroup spends on them (a
// pair, or one middle tile), each to the XCD queue with the least work so far
// (the lowest index on ties); the queues are stored one after another.  The
// order is by that duration, not by a gang's total work: a gang of a few long
// units (the middle tiles of a long item) sorted by its small total would
// start last and end long after every other workgroup (an 8 ms tail on the
// long-tail share).  Returns the gangs in queue order and fills qoff.
std::vector<const KvGang *> kv_queue_order(const ItemGangs &items, std::vector<int> &qoff) {
  std::vector<const KvGang *> gangs;
  for (const auto &ig : items)
    for (const KvGang &g : ig.second) gangs.push_back(&g);
  std::stable_sort(gangs.begin(), gangs.end(), [](const KvGang *a, const KvGang *b) { return a->dur > b->dur; });
  std::vector<std::vector<const KvGang *>> q(kNumXcd);
  std::vector<int64_t> load(kNumXcd, 0);
  for (const KvGang *g : gangs) {
    const int x = (int)(std::min_element(load.begin(), load.end()) - load.begin());
    load[x] += g->cost;
    q[x].push_back(g);
  }
  std::vector<const KvGang *> out;
  qoff.assign(kNumXcd + 1, 0);
  int n = 0;
  for (int x = 0; x < kNumXcd; ++x) {
    qoff[x] = n;
    for (const KvGang *g : q[x]) {
      out.push_back(g);
      n += (int)g->units.size();
    }
  }
  qoff[kNumXcd] = n;
  return out;
}

// Model of the persistent dK/dV pass over such queues: each of 256 compute
// units (32 per XCD) takes the next unit of its own XCD's queue when it goes
// idle, else the next unit of the other queues in turn, and spends the unit's
// steps on it.  Returns when the last one ends, in steps.
constexpr int kAssumedCUs = 256;

int64_t kv_model_makespan(const std::vector<int64_t> &steps, const std::vector<int> &qoff) {
  std::vector<int> head(qoff.begin(), qoff.end() - 1);
  using Cu = std::tuple<int64_t, int, int>;   // (free at, XCD, compute unit)
  std::priority_queue<Cu, std::vector<Cu>, std::greater<Cu>> idle;
  for (int x = 0; x < kNumXcd; ++x)
    for (int c = 0; c < kAssumedCUs / kNumXcd; ++c) idle.push(Cu{0, x, c});
  int64_t end = 0;
  while (!idle.empty()) {
    const Cu cu = idle.top();
    idle.pop();
    int slot = -1;
    for (int k = 0; k < kNumXcd && slot < 0; ++k) {
      const int y = (std::get<1>(cu) + k) % kNumXcd;
      if (head[y] < qoff[y + 1]) slot = head[y]++;
    }
    if (slot < 0) {
      end = std::max(end, std::get<0>(cu));
      continue;
    }
    idle.push(Cu{std::get<0>(cu) + steps[slot], std::get<1>(cu), std::get<2>(cu)});
  }
  return end;
}

int64_t kv_model(const ItemGangs &items) {
  std::vector<int> qoff;
  std::vector<int64_t> steps;
  for (const KvGang *g : kv_queue_order(items, qoff)) steps.insert(steps.end(), g->steps.begin(), g->steps.end());
  return kv_model_makespan(steps, qoff);
}

// Balance.  Pairs all take about the same time, so a list of one or a few
// long items is made of equal chunks that need not divide evenly over the
// compute units (one item of 454 pairs on 256 CUs ends after two pairs'
// time, 13% past an even split), and whose end leaves no short units for the
// persistent pass to even out XCDs that run a few percent apart (they do,
// on one chip).  Both are cured by leaving the K shortest key tiles of the
// item with the most work unpaired -- single units, which the duration order
// places last -- and with them their partners, the K longest, which sweep
// down from the item end in gangs of their own:
//  * end game: when less than kEndMin of the work is in gangs whose duration
//    is at most kEndDur of one compute unit's share, K starts at the least
//    that puts kEndShare of the work in the short singles;
//  * when the model above then ends more than kBalanceTol past an even
//    split, K is the one of at most kMaxTries candidates from there to nk/2
//    with the earliest modelled end (the smallest on ties).
// K is always a whole number of gangs of leading units (a partial gang
// leaves compute units of its XCD to start the next gang early, out of
// step).  Measured: the end game makes dK/dV on the one-item max-context
// share 1.5% faster than the pairs alone; the search makes it 8% faster on
// the one-item sp = 4 call of the long-tail share's phase streaming (44.6
// against 48.5 ms).  Below the 8% threshold the model is not accurate
// enough to pay: at 3%, the calls it changed ran no faster, or 1% slower.
constexpr double kEndMin = 0.01, kEndDur = 0.10, kEndShare = 0.02, kBalanceTol = 1.08;
constexpr int kMaxTries = 64;

void kv_balance(ItemGangs &items, const nsp_worklist *wl) {
  if (items.empty()) return;
  int64_t total = 0, small = 0;
  for (auto &ig : items)
    for (const KvGang &g : ig.second) total += g.cost;
  const double dmax = kEndDur * (double)total / kAssumedCUs;
  for (auto &ig : items)
    for (const KvGang &g : ig.second)
      if ((double)g.dur <= dmax) small += g.cost;
  size_t big = 0;
  int64_t bw = -1;
  for (size_t i = 0; i < items.size(); ++i) {
    int64_t w = 0;
    for (const KvGang &g : items[i].second) w += g.cost;
    if (w > bw) { bw = w; big = i; }
  }
  const int j = items[big].first;
  const int L = wl->cu_seqlens[j + 1] - wl->cu_seqlens[j];
  const int nk = (L + nsp::kBwdBN - 1) / nsp::kBwdBN, nqt = (L + nsp::kBwdBM - 1) / nsp::kBwdBM;
  const int hkv = wl->kv_heads[2 * j + 1] - wl->kv_heads[2 * j];
  const int half = nk / 2;
  int K = 0;
  if ((double)small < kEndMin * (double)total) {
    const int64_t h = std::max<int64_t>(1, (wl->q_heads[2 * j + 1] - wl->q_heads[2 * j]) / std::max(1, hkv));
    const double need = kEndShare * (double)total;
    double got = 0;
    while (K < half && got < need) {
      ++K;
      got += (double)(hkv * h * ((int64_t)nqt - (int64_t)(nk - K) * nsp::kBwdBN / nsp::kBwdBM));
    }
    while (K < half && (K * hkv) % nsp::kKvGang != 0) ++K;
    items[big].second.clear();
    add_kv_gangs(items[big].second, wl, j, L, K);
  }
  int64_t best = kv_model(items);
  if ((double)best <= kBalanceTol * ((double)total / kAssumedCUs) || K >= half) return;
  int unit = 1;   // K steps of whole gangs of leading units
  while ((unit * hkv) % nsp::kKvGang != 0) ++unit;
  int stride = unit;
  while ((half - K + stride - 1) / stride > kMaxTries) stride += unit;
  int best_k = K;
  for (int k = K + stride;; k += stride) {
    const int kc = std::min(k, half);
    items[big].second.clear();
    add_kv_gangs(items[big].second, wl, j, L, kc);
    const int64_t m = kv_model(items);
    if (m < best) { best = m; best_k = kc; }
    if (kc == half) break;
  }
  items[big].second.clear();
  add_kv_gangs(items[big].second, wl, j, L, best_k);
}

HostAttnSched build_attn_schedule(const nsp_worklist *wl) {
  HostAttnSched s;
  const int D = wl->head_dim;
  int64_t qo = 0, ko = 0, lo = 0;
  std::vector<int64_t> fcost;
  ItemGangs item_gangs;
  for (int j = 0; j < wl->n_items; ++j) {
    const int L = wl->cu_seqlens[j + 1] - wl->cu_seqlens[j];
    const int ql = wl->q_heads[2 * j], hq = wl->q_heads[2 * j + 1] - ql;
    const int kl = wl->kv_heads[2 * j], hkv = wl->kv_heads[2 * j + 1] - kl;
    ItemDesc d{};
    d.q_off = qo;
    d.kv_off = ko;
    d.lse_off = lo;
    d.q_row0 = qo / D;
    d.L = L;
    d.hq = hq;
    d.hkv = hkv;
    d.active = selected(wl, j) ? 1 : 0;
    s.items.push_back(d);
    if (L > 0 && d.active) {
      for (int i = 0; i < hq; ++i)
        for (int t = 0; t < L; t += nsp::kPreBlockRows)
          s.pre_blocks.push_back(nsp::PreBlock{j, i, t, std::min(nsp::kPreBlockRows, L - t)});
      const int nq = (L + nsp::kFwdBM - 1) / nsp::kFwdBM;
      for (int m = 0; m < nq; ++m)
        for (int i = 0; i < hq; ++i) {
          const int g = (int)(((int64_t)(ql + i) * wl->hkv_total) / wl->hq_total) - kl;
          s.fwd_units.push_back(int4{j, m, i, g});
          fcost.push_back(std::min<int64_t>(L, (int64_t)nsp::kFwdBM * (m + 1)));
        }
      item_gangs.emplace_back(j, std::vector<KvGang>());
      add_kv_gangs(item_gangs.back().second, wl, j, L, 0);
    }
    qo += (int64_t)L * hq * D;
    ko += (int64_t)L * hkv * D;
    lo += (int64_t)L * hq;
  }
  s.q_rows = qo / D;
  lpt_sort(s.fwd_units, fcost);
  kv_balance(item_gangs, wl);
  for (const KvGang *g : kv_queue_order(item_gangs, s.kv_qoff))
    s.kv_units.insert(s.kv_units.end(), g->units.begin(), g->units.end());
  // XCD runs pay only when a stream's tiles (K and V of one head, or Q and
  // dO) overflow one XCD's L2; below that every tile stays cached wherever
  // its units run, and runs of similar units on one XCD only unbalance the
  // XCDs (short-sequence lists then finish ~5% later, long ones ~5% sooner).
  if (max_stream_bytes(wl) > kXcdL2Bytes) {
    xcd_group(s.fwd_units, nsp::kXcdGroupFwd);
  }
  return s;
}

constexpr int64_t kTaskChunks = 4096;   // 16-byte chunks per re-layout workgroup

void add_copy_tasks(std::vector<CopyTask> &out, int64_t dst, int64_t src, int64_t dst_ts, int64_t src_ts,
                    int ntok, int cpt, int nrep, int64_t rep_stride) {
  const int per = (int)std::max<int64_t>(1, kTaskChunks / cpt);
  for (int t0 = 0; t0 < ntok; t0 += per) {
    CopyTask t{};
    t.dst = dst;
    t.src = src;
    t.dst_ts = dst_ts;
    t.src_ts = src_ts;
    t.rep_stride = rep_stride;
    t.t0 = t0;
    t.ntok = std::min(per, ntok - t0);
    t.cpt = cpt;
    t.nrep = nrep;
    out.push_back(t);
  }
}

std::vector<CopyTask> build_relayout_tasks(const nsp_worklist *wl, nsp_kind kind, nsp_dtype dtype, bool pack,
                                           bool sum) {
  std::vector<CopyTask> tasks;
  const int64_t D = wl->head_dim, es = dtype == NSP_BF16 ? 2 : 4;
  const int64_t H = kind == NSP_KIND_Q ? wl->hq_total : wl->hkv_total;
  int64_t c = 0, e = 0;   // sequence-layout token offset, head-layout element offset
  for (int j = 0; j < wl->n_items; ++j) {
    const int64_t L = wl->cu_seqlens[j + 1] - wl->cu_seqlens[j];
    const int64_t s = wl->sp[j], n = L / s, hl = H >= s ? H / s : 1;
    const int cpt = (int)(hl * D * es / 16);
    if (n > 0 && selected(wl, j)) {
      if (pack || H >= s) {
        for (int64_t b = 0; b < s; ++b) {
          const int64_t head = H >= s ? b * hl : (b * H) / s;
          const int64_t seq = (c * H + head) * D * es, seq_ts = H * D * es;
          const int64_t hd = (e + b * n * hl * D) * es, hd_ts = hl * D * es;
          if (pack) add_copy_tasks(tasks, hd, seq, hd_ts, seq_ts, (int)n, cpt, 1, 0);
          else add_copy_tasks(tasks, seq, hd, seq_ts, hd_ts, (int)n, cpt, 1, 0);
        }
      } else {
        const int64_t reps = s / H;
        for (int64_t g = 0; g < H; ++g) {
          const int64_t hd = (e + g * reps * n * D) * es;
          const int64_t seq = (c * H + g) * D * es;
          add_copy_tasks(tasks, seq, hd, H * D * es, D * es, (int)n, cpt, sum ? (int)reps : 1, n * D * es);
        }
      }
    }
    c += n;
    e += L * hl * D;
  }
  return tasks;
}

// --------------------------------------------------------- schedule cache --

// One device buffer holding a work list's schedule; freed with the entry.
struct CacheEntry {
  void *dev = nullptr;
  nsp::Schedule sched;          // attention schedules
  CopyTask *tasks = nullptr;    // re-layout schedules
  int n_tasks = 0;
  CacheEntry() = default;
  CacheEntry(const CacheEntry &) = delete;
  CacheEntry &operator=(const CacheEntry &) = delete;
  ~CacheEntry() {
    if (dev) (void)hipFree(dev);   // waits for work still using it
  }
};
using EntryPtr = nsp::LruCache<CacheEntry>::Ptr;

// Never destroyed: entries must not be freed after the HIP runtime has shut
// down at process exit.
nsp::LruCache<CacheEntry> &schedule_cache() {
  static auto *c = new nsp::LruCache<CacheEntry>(128);
  return *c;
}

std::string worklist_key(const char *tag, int dev, const nsp_worklist *wl, int extra) {
  std::string k(tag);
  auto put = [&](const void *p, size_t n) { k.append(reinterpret_cast<const char *>(p), n); };
  put(&dev, sizeof dev);
  put(&extra, sizeof extra);
  put(&wl->n_items, sizeof wl->n_items);
  put(&wl->hq_total, sizeof wl->hq_total);
  put(&wl->hkv_total, sizeof wl->hkv_total);
  put(&wl->head_dim, sizeof wl->head_dim);
  if (wl->n_items > 0) {
    put(wl->cu_seqlens, sizeof(int32_t) * (wl->n_items + 1));
    put(wl->q_heads, sizeof(int32_t) * 2 * wl->n_items);
    put(wl->kv_heads, sizeof(int32_t) * 2 * wl->n_items);
    if (wl->sp) put(wl->sp, sizeof(int32_t) * wl->n_items);
    if (wl->item_mask) {
      k.push_back('m');
      for (int j = 0; j < wl->n_items; ++j) k.push_back(wl->item_mask[j] ? '1' : '0');
    }
  }
  return k;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

nsp_status upload(const void *host, size_t bytes, void **dev) {
  *dev = nullptr;
  if (bytes == 0) return NSP_OK;
  hipError_t err = hipMalloc(dev, bytes);
  if (err != hipSuccess) {
    *dev = nullptr;
    return fail(NSP_ENOMEM, "hipMalloc(%zu) for the schedule failed: %s", bytes, hipGetErrorString(err));
  }
  err = hipMemcpy(*dev, host, bytes, hipMemcpyHostToDevice);
  if (err != hipSuccess) {
    (void)hipFree(*dev);
    *dev = nullptr;
    return fail(NSP_EHIP, "hipMemcpy of the schedule failed: %s", hipGetErrorString(err));
  }
  return NSP_OK;
}

// The device image of an attention schedule: ItemDesc[n_items] | forward/dQ
// units | dK/dV units | preprocess spans, each part 256-byte aligned.
struct AttnBlob {
  std::vector<char> bytes;
  size_t o_fwd = 0, o_kv = 0, o_kvq = 0, o_pre = 0;
};

AttnBlob attn_blob(const HostAttnSched &hs) {
  AttnBlob b;
  const size_t n_items = align256(hs.items.size() * sizeof(ItemDesc));
  const size_t n_fwd = align256(hs.fwd_units.size() * sizeof(int4));
  const size_t n_kv = align256(hs.kv_units.size() * sizeof(int4));
  const size_t n_kvq = align256(hs.kv_qoff.size() * sizeof(int));
  const size_t n_pre = align256(hs.pre_blocks.size() * sizeof(nsp::PreBlock));
  b.o_fwd = n_items;
  b.o_kv = n_items + n_fwd;
  b.o_kvq = n_items + n_fwd + n_kv;
  b.o_pre = n_items + n_fwd + n_kv + n_kvq;
  b.bytes.assign(b.o_pre + n_pre, 0);
  auto put = [&](size_t off, const void *src, size_t n) {
    if (n) memcpy(b.bytes.data() + off, src, n);
  };
  put(0, hs.items.data(), hs.items.size() * sizeof(ItemDesc));
  put(b.o_fwd, hs.fwd_units.data(), hs.fwd_units.size() * sizeof(int4));
  put(b.o_kv, hs.kv_units.data(), hs.kv_units.size() * sizeof(int4));
  put(b.o_kvq, hs.kv_qoff.data(), hs.kv_qoff.size() * sizeof(int));
  put(b.o_pre, hs.pre_blocks.data(), hs.pre_blocks.size() * sizeof(nsp::PreBlock));
  return b;
}

// The schedule of `hs` whose device image (attn_blob) starts at `dev`.
nsp::Schedule attn_schedule_at(const HostAttnSched &hs, const AttnBlob &b, char *dev) {
  nsp::Schedule s;
  s.items = reinterpret_cast<ItemDesc *>(dev);
  s.fwd_units = reinterpret_cast<int4 *>(dev + b.o_fwd);
  s.kv_units = reinterpret_cast<int4 *>(dev + b.o_kv);
  s.kv_qoff = reinterpret_cast<int *>(dev + b.o_kvq);
  s.pre_blocks = reinterpret_cast<nsp::PreBlock *>(dev + b.o_pre);
  s.n_items = (int)hs.items.size();
  s.n_fwd_units = (int)hs.fwd_units.size();
  s.n_kv_units = (int)hs.kv_units.size();
  s.n_pre_blocks = (int)hs.pre_blocks.size();
  s.q_rows = hs.q_rows;
  return s;
}

// The cached schedule of a work list on the current device.  *hold keeps the
// entry alive; the caller keeps it until its kernels are enqueued.
nsp_status get_attn_schedule(const nsp_worklist *wl, nsp::Schedule *out, EntryPtr *hold) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return fail(NSP_EHIP, "hipGetDevice failed: %s", hipGetErrorString(err));
  nsp_status st = schedule_cache().get(worklist_key("attn", dev, wl, 0), hold, [&](EntryPtr *made) {
    const HostAttnSched hs = build_attn_schedule(wl);
    const AttnBlob b = attn_blob(hs);
    auto ce = std::make_shared<CacheEntry>();
    nsp_status s2 = upload(b.bytes.data(), b.bytes.size(), &ce->dev);
    if (s2 != NSP_OK) return (int)s2;
    ce->sched = attn_schedule_at(hs, b, static_cast<char *>(ce->dev));
    *made = std::move(ce);
    return (int)NSP_OK;
  });
  if (st != NSP_OK) return st;
  *out = (*hold)->sched;
  return NSP_OK;
}

nsp_status get_relayout_tasks(const nsp_worklist *wl, nsp_kind kind, nsp_dtype dtype, bool pack, bool sum,
                              CopyTask **tasks, int *n_tasks, EntryPtr *hold) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return fail(NSP_EHIP, "hipGetDevice failed: %s", hipGetErrorString(err));
  const int extra = (int)kind | ((int)dtype << 4) | ((int)pack << 8) | ((int)sum << 9);
  nsp_status st = schedule_cache().get(worklist_key("relayout", dev, wl, extra), hold, [&](EntryPtr *made) {
    std::vector<CopyTask> t = build_relayout_tasks(wl, kind, dtype, pack, sum);
    auto ce = std::make_shared<CacheEntry>();
    nsp_status s2 = upload(t.data(), t.size() * sizeof(CopyTask), &ce->dev);
    if (s2 != NSP_OK) return (int)s2;
    ce->tasks = static_cast<CopyTask *>(ce->dev);
    ce->n_tasks = (int)t.size();
    *made = std::move(ce);
    return (int)NSP_OK;
  });
  if (st != NSP_OK) return st;
  *tasks = (*hold)->tasks;
  *n_tasks = (*hold)->n_tasks;
  return NSP_OK;
}

nsp_status check_ptr(const void *p, int64_t elems, size_t align, const char *name) {
  if (elems == 0) return NSP_OK;
  if (!p) return fail(NSP_EINVAL, "%s is NULL", name);
  if (misaligned(p, align)) return fail(NSP_EINVAL, "%s is not %zu-byte aligned", name, align);
  return NSP_OK;
}

nsp_status check_scale(float scale) {
  if (!(scale > 0.f) || !std::isfinite(scale))
    return fail(NSP_EINVAL, "softmax_scale must be finite and positive (got %g)", (double)scale);
  return NSP_OK;
}

nsp_status hip_status(hipError_t err, const char *what) {
  if (err == hipSuccess) return NSP_OK;
  return fail(NSP_EHIP, "%s: %s", what, hipGetErrorString(err));
}

// Workspace layout: -Delta [lse_elems] | lse*log2(e) [lse_elems] (float32,
// each 256-byte aligned) | 256 bytes of unit-queue heads.
size_t bwd_workspace_bytes(const WlInfo &w) {
  return 2 * align256((size_t)w.lse_elems * sizeof(float)) + 256;
}

}  // namespace

#define NSP_TRY(expr)                 \
  do {                                \
    nsp_status _st = (expr);          \
    if (_st != NSP_OK) return _st;    \
  } while (0)

// ----------------------------------------------------- kernel timing --

namespace {

const char *const kKernelNames[] = {"attn_fwd", "bwd_preprocess", "bwd_dkdv", "bwd_dq", "relayout"};
constexpr int kNumKernels = 5;
enum KernelId { K_FWD = 0, K_PRE = 1, K_DKDV = 2, K_DQ = 3, K_RELAYOUT = 4 };

struct TimingState {
  std::mutex mu;
  bool on = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pending[kNumKernels];
  int64_t launches[kNumKernels] = {};
  double total_ms[kNumKernels] = {};
};
TimingState g_timing;

// Run `launch` on `stream`, bracketed by timing events when timing is on.
template <class F>
hipError_t timed_launch(KernelId id, hipStream_t stream, F launch) {
  bool on;
  {
    std::lock_guard<std::mutex> lock(g_timing.mu);
    on = g_timing.on;
  }
  if (!on) return launch();
  hipEvent_t a = nullptr, b = nullptr;
  hipError_t e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  if (e == hipSuccess) e = hipEventRecord(a, stream);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(b, stream);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_timing.mu);
  g_timing.pending[id].push_back({a, b});
  return hipSuccess;
}

// Arguments of a backward call (everything but the workspace).
nsp_status validate_bwd(const nsp_worklist *wl, float softmax_scale, int32_t causal, const void *q, const void *k,
                        const void *v, const void *o, nsp_dtype o_dtype, const void *dout, const float *lse,
                        const void *dq, const void *dk, const void *dv, nsp_dtype grad_dtype, WlInfo *w) {
  NSP_TRY(validate_worklist(wl, w));
  NSP_TRY(check_scale(softmax_scale));
  if (o_dtype != NSP_BF16 && o_dtype != NSP_F32) return fail(NSP_EINVAL, "unknown o_dtype %d", (int)o_dtype);
  if (grad_dtype != NSP_BF16 && grad_dtype != NSP_F32)
    return fail(NSP_EINVAL, "unknown grad_dtype %d", (int)grad_dtype);
  if (causal != 1) return fail(NSP_EUNSUPPORTED, "only causal attention (causal=1) is implemented");
  NSP_TRY(check_ptr(q, w->q_elems, 16, "q"));
  NSP_TRY(check_ptr(k, w->kv_elems, 16, "k"));
  NSP_TRY(check_ptr(v, w->kv_elems, 16, "v"));
  NSP_TRY(check_ptr(o, w->q_elems, 16, "o"));
  NSP_TRY(check_ptr(dout, w->q_elems, 16, "dout"));
  NSP_TRY(check_ptr(lse, w->lse_elems, 4, "lse"));
  NSP_TRY(check_ptr(dq, w->q_elems, 16, "dq"));
  NSP_TRY(check_ptr(dk, w->kv_elems, 16, "dk"));
  NSP_TRY(check_ptr(dv, w->kv_elems, 16, "dv"));
  return NSP_OK;
}

// The largest sum_j L_j hq_j whose backward workspace fits the scratch.
constexpr size_t noalloc_max_lse_elems() {
  return ((nsp::kScratchBytes - nsp::kScratchSchedBytes - 256) / 2 / 256 * 256) / sizeof(float);
}
static_assert(nsp::kScratchBytes == NSP_NOALLOC_SCRATCH_BYTES, "scratch size as declared in nsp.h");
static_assert(noalloc_max_lse_elems() == NSP_NOALLOC_MAX_ROWS, "row limit as declared in nsp.h");

// Host-only copies of attention schedules (for the allocation-free backward,
// which copies them into its device scratch).
struct HostSched {
  HostAttnSched hs;
  AttnBlob blob;
};
using HostSchedPtr = nsp::LruCache<HostSched>::Ptr;

nsp::LruCache<HostSched> &host_schedule_cache() {
  static auto *c = new nsp::LruCache<HostSched>(128);
  return *c;
}

nsp_status get_host_schedule(const std::string &key, const nsp_worklist *wl, HostSchedPtr *out) {
  return host_schedule_cache().get(key, out, [&](HostSchedPtr *made) {
    auto h = std::make_shared<HostSched>();
    h->hs = build_attn_schedule(wl);
    h->blob = attn_blob(h->hs);
    *made = std::move(h);
    return (int)NSP_OK;
  });
}

// Per device: the key of the schedule the scratch holds.  A call whose work
// list is the last one copied there enqueues no copy; otherwise the blob is
// copied on the call's stream (from pageable host memory: the copy has read
// the blob when hipMemcpyAsync returns).
std::mutex g_noalloc_mu;
std::unordered_map<int, std::string> g_noalloc_key;

nsp_status noalloc_upload(int dev, const std::string &key, const HostSched &h, char *scr, hipStream_t stream) {
  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  auto it = g_noalloc_key.find(dev);
  if (it != g_noalloc_key.end() && it->second == key) return NSP_OK;
  g_noalloc_key.erase(dev);
  NSP_TRY(hip_status(hipMemcpyAsync(scr, h.blob.bytes.data(), h.blob.bytes.size(), hipMemcpyHostToDevice, stream),
                     "copying the schedule into the device scratch"));
  g_noalloc_key[dev] = key;
  return NSP_OK;
}

// The three backward kernels on `stream`: preprocess (-Delta, lse2, and the
// reset of the unit-queue heads), dK/dV, dQ.
nsp_status launch_backward(int D, const nsp::Schedule &s, float softmax_scale, const void *q, const void *k,
                           const void *v, const void *o, nsp_dtype o_dtype, const void *dout, const float *lse,
                           void *dq, void *dk, void *dv, nsp_dtype grad_dtype, float *delta, float *lse2,
                           int *queue, hipStream_t stream) {
  nsp::AttnArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.dout = dout;
  a.lse_in = lse;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.delta = delta;
  a.lse2 = lse2;
  a.queue = queue;
  a.items = s.items;
  a.n_items = s.n_items;
  a.pre_blocks = s.pre_blocks;
  a.scale = softmax_scale;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  const bool g32 = grad_dtype == NSP_F32;
  NSP_TRY(hip_status(timed_launch(K_PRE, stream,
                                  [&] { return nsp::launch_bwd_preprocess(D, o_dtype == NSP_F32, a, s.n_pre_blocks,
                                                                          stream); }),
                     "backward preprocess launch"));
  a.units = s.kv_units;
  a.qoff = s.kv_qoff;
  NSP_TRY(hip_status(timed_launch(K_DKDV, stream,
                                  [&] { return nsp::launch_bwd_dkdv(D, g32, a, s.n_kv_units, stream); }),
                     "backward dK/dV launch"));
  a.units = s.fwd_units;
  return hip_status(timed_launch(K_DQ, stream, [&] { return nsp::launch_bwd_dq(D, g32, a, s.n_fwd_units, stream); }),
                    "backward dQ launch");
}

}  // namespace

extern "C" {

nsp_status nsp_varlen_attn_fwd(const nsp_worklist *wl, float softmax_scale, int32_t causal, const void *q,
                               const void *k, const void *v, void *o, nsp_dtype o_dtype, float *lse,
                               hipStream_t stream) {
  g_last_error.clear();
  WlInfo w;
  NSP_TRY(validate_worklist(wl, &w));
  NSP_TRY(check_scale(softmax_scale));
  if (o_dtype != NSP_BF16 && o_dtype != NSP_F32) return fail(NSP_EINVAL, "unknown o_dtype %d", (int)o_dtype);
  if (causal != 1) return fail(NSP_EUNSUPPORTED, "only causal attention (causal=1) is implemented");
  NSP_TRY(check_ptr(q, w.q_elems, 16, "q"));
  NSP_TRY(check_ptr(k, w.kv_elems, 16, "k"));
  NSP_TRY(check_ptr(v, w.kv_elems, 16, "v"));
  NSP_TRY(check_ptr(o, w.q_elems, 16, "o"));
  NSP_TRY(check_ptr(lse, w.lse_elems, 4, "lse"));
  if (w.q_elems == 0) return NSP_OK;
  nsp::Schedule s;
  EntryPtr hold;
  NSP_TRY(get_attn_schedule(wl, &s, &hold));
  nsp::AttnArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.o_out = o;
  a.lse = lse;
  a.items = s.items;
  a.units = s.fwd_units;
  a.n_items = s.n_items;
  a.scale = softmax_scale;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  return hip_status(timed_launch(K_FWD, stream,
                                 [&] { return nsp::launch_attn_fwd(wl->head_dim, o_dtype == NSP_F32, a,
                                                                   s.n_fwd_units, stream); }),
                    "attention forward launch");
}

size_t nsp_varlen_attn_bwd_workspace(const nsp_worklist *wl) {
  WlInfo w;
  if (validate_worklist(wl, &w) != NSP_OK) return 0;
  return bwd_workspace_bytes(w);
}

nsp_status nsp_varlen_attn_bwd(const nsp_worklist *wl, float softmax_scale, int32_t causal, const void *q,
                               const void *k, const void *v, const void *o, nsp_dtype o_dtype, const void *dout,
                               const float *lse, void *dq, void *dk, void *dv, nsp_dtype grad_dtype,
                               void *workspace, size_t ws_bytes, hipStream_t stream) {
  g_last_error.clear();
  WlInfo w;
  NSP_TRY(validate_bwd(wl, softmax_scale, causal, q, k, v, o, o_dtype, dout, lse, dq, dk, dv, grad_dtype, &w));
  const size_t need = bwd_workspace_bytes(w);
  if (w.q_elems > 0 && (!workspace || ws_bytes < need))
    return fail(NSP_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace ? ws_bytes : 0, need);
  if (w.q_elems > 0 && misaligned(workspace, 256)) return fail(NSP_EINVAL, "workspace is not 256-byte aligned");
  if (w.q_elems == 0) return NSP_OK;
  nsp::Schedule s;
  EntryPtr hold;
  NSP_TRY(get_attn_schedule(wl, &s, &hold));
  const size_t lse_bytes = align256((size_t)w.lse_elems * sizeof(float));
  char *ws = static_cast<char *>(workspace);
  return launch_backward(wl->head_dim, s, softmax_scale, q, k, v, o, o_dtype, dout, lse, dq, dk, dv, grad_dtype,
                         reinterpret_cast<float *>(ws), reinterpret_cast<float *>(ws + lse_bytes),
                         reinterpret_cast<int *>(ws + 2 * lse_bytes), stream);
}

nsp_status nsp_varlen_attn_bwd_noalloc(const nsp_worklist *wl, float softmax_scale, int32_t causal, const void *q,
                                       const void *k, const void *v, const void *o, nsp_dtype o_dtype,
                                       const void *dout, const float *lse, void *dq, void *dk, void *dv,
                                       nsp_dtype grad_dtype, hipStream_t stream) {
  g_last_error.clear();
  WlInfo w;
  NSP_TRY(validate_bwd(wl, softmax_scale, causal, q, k, v, o, o_dtype, dout, lse, dq, dk, dv, grad_dtype, &w));
  const size_t ws_need = bwd_workspace_bytes(w);
  if (ws_need > nsp::kScratchBytes - nsp::kScratchSchedBytes)
    return fail(NSP_EWORKSPACE,
                "the work list needs %zu bytes of backward workspace; the allocation-free backward holds %zu "
                "(sum_j L_j hq_j <= %zu)",
                ws_need, nsp::kScratchBytes - nsp::kScratchSchedBytes, noalloc_max_lse_elems());
  if (w.q_elems == 0) return NSP_OK;
  int dev = 0;
  NSP_TRY(hip_status(hipGetDevice(&dev), "hipGetDevice"));
  HostSchedPtr hsp;
  const std::string key = worklist_key("attn", dev, wl, 0);
  NSP_TRY(get_host_schedule(key, wl, &hsp));
  if (hsp->blob.bytes.size() > nsp::kScratchSchedBytes)
    return fail(NSP_EWORKSPACE, "the work list's schedule takes %zu bytes; the allocation-free backward holds %zu",
                hsp->blob.bytes.size(), nsp::kScratchSchedBytes);
  char *scr = nullptr;
  NSP_TRY(hip_status(nsp::noalloc_scratch(&scr), "looking up the device scratch"));
  NSP_TRY(noalloc_upload(dev, key, *hsp, scr, stream));
  const nsp::Schedule s = attn_schedule_at(hsp->hs, hsp->blob, scr);
  char *ws = scr + nsp::kScratchSchedBytes;
  const size_t lse_bytes = align256((size_t)w.lse_elems * sizeof(float));
  return launch_backward(wl->head_dim, s, softmax_scale, q, k, v, o, o_dtype, dout, lse, dq, dk, dv, grad_dtype,
                         reinterpret_cast<float *>(ws + 256), reinterpret_cast<float *>(ws + 256 + lse_bytes),
                         reinterpret_cast<int *>(ws), stream);
}

static nsp_status relayout(const nsp_worklist *wl, nsp_kind kind, nsp_dtype dtype, bool pack, nsp_replica rep,
                           const void *src, void *dst, hipStream_t stream) {
  g_last_error.clear();
  WlInfo w;
  NSP_TRY(validate_worklist(wl, &w));
  NSP_TRY(validate_relayout(wl, kind, dtype));
  if (rep != NSP_UNPACK_SELECT && rep != NSP_UNPACK_SUM) return fail(NSP_EINVAL, "unknown replica mode %d", (int)rep);
  const int64_t head_elems = kind == NSP_KIND_Q ? w.q_elems : w.kv_elems;
  const size_t es = dtype == NSP_BF16 ? 2 : 4;
  NSP_TRY(check_ptr(src, head_elems, 16, pack ? "x_seq" : "x_head"));
  NSP_TRY(check_ptr(dst, head_elems, 16, pack ? "x_head" : "x_seq"));
  if (head_elems == 0) return NSP_OK;
  (void)es;
  const bool sum = !pack && rep == NSP_UNPACK_SUM;
  CopyTask *tasks = nullptr;
  int n = 0;
  EntryPtr hold;
  NSP_TRY(get_relayout_tasks(wl, kind, dtype, pack, sum, &tasks, &n, &hold));
  const int mode = sum ? (dtype == NSP_BF16 ? 1 : 2) : 0;
  return hip_status(timed_launch(K_RELAYOUT, stream,
                                 [&] { return nsp::launch_relayout(src, dst, tasks, n, mode, stream); }),
                    pack ? "pack launch" : "unpack launch");
}

nsp_status nsp_ulysses_pack(const nsp_worklist *wl, nsp_kind kind, nsp_dtype dtype, const void *x_seq,
                            void *x_head, hipStream_t stream) {
  return relayout(wl, kind, dtype, true, NSP_UNPACK_SELECT, x_seq, x_head, stream);
}

nsp_status nsp_ulysses_unpack(const nsp_worklist *wl, nsp_kind kind, nsp_dtype dtype, nsp_replica replica,
                              const void *x_head, void *x_seq, hipStream_t stream) {
  return relayout(wl, kind, dtype, false, replica, x_head, x_seq, stream);
}

nsp_status nsp_recompute_plan(const nsp_worklist *wl, int64_t budget_bytes, nsp_dtype o_dtype, uint8_t *save,
                              int64_t *saved_bytes) {
  g_last_error.clear();
  NSP_TRY(validate_worklist(wl, nullptr));
  if (o_dtype != NSP_BF16 && o_dtype != NSP_F32) return fail(NSP_EINVAL, "unknown o_dtype %d", (int)o_dtype);
  if (budget_bytes < 0) return fail(NSP_EINVAL, "budget_bytes = %lld < 0", (long long)budget_bytes);
  if (wl->n_items > 0 && (!wl->sp || !save)) return fail(NSP_EINVAL, "sp and save must be non-NULL");
  for (int j = 0; j < wl->n_items; ++j)
    if (wl->sp[j] <= 0) return fail(NSP_EINVAL, "item %d: sp = %d must be positive", j, wl->sp[j]);
  const int64_t per_elem = (int64_t)wl->head_dim * (o_dtype == NSP_BF16 ? 2 : 4) + 4;
  std::vector<int64_t> bytes(wl->n_items);
  std::vector<int> levels;
  for (int j = 0; j < wl->n_items; ++j) {
    const int64_t L = (int64_t)wl->cu_seqlens[j + 1] - wl->cu_seqlens[j];
    bytes[j] = L * (wl->q_heads[2 * j + 1] - wl->q_heads[2 * j]) * per_elem;
    save[j] = 0;
    levels.push_back(wl->sp[j]);
  }
  std::sort(levels.begin(), levels.end(), std::greater<int>());
  levels.erase(std::unique(levels.begin(), levels.end()), levels.end());
  int64_t used = 0;
  for (int sp : levels) {                         // root (largest sp) first
    std::vector<int> node;
    int64_t node_bytes = 0;
    for (int j = 0; j < wl->n_items; ++j)
      if (wl->sp[j] == sp) { node.push_back(j); node_bytes += bytes[j]; }
    if (used + node_bytes <= budget_bytes) {      // the whole node fits
      for (int j : node) save[j] = 1;
      used += node_bytes;
      continue;
    }
    // the cut node: longest items first (recomputation cost per byte grows
    // with L), each one saved if it still fits; the nodes below recompute
    std::stable_sort(node.begin(), node.end(), [&](int x, int y) {
      const int64_t lx = (int64_t)wl->cu_seqlens[x + 1] - wl->cu_seqlens[x];
      const int64_t ly = (int64_t)wl->cu_seqlens[y + 1] - wl->cu_seqlens[y];
      return lx > ly;
    });
    for (int j : node)
      if (used + bytes[j] <= budget_bytes) { save[j] = 1; used += bytes[j]; }
    break;
  }
  for (int j = 0; j < wl->n_items; ++j)
    if (bytes[j] == 0) save[j] = 1;
  if (saved_bytes) *saved_bytes = used;
  return NSP_OK;
}

nsp_status nsp_attn_schedule(const nsp_worklist *wl, int32_t which, int32_t *units, int64_t capacity,
                             int64_t *n_units) {
  g_last_error.clear();
  NSP_TRY(validate_worklist(wl, nullptr));
  if (which != NSP_SCHED_FWD && which != NSP_SCHED_KV) return fail(NSP_EINVAL, "unknown schedule %d", which);
  if (!n_units) return fail(NSP_EINVAL, "n_units is NULL");
  const HostAttnSched hs = build_attn_schedule(wl);
  const std::vector<int4> &u = which == NSP_SCHED_FWD ? hs.fwd_units : hs.kv_units;
  *n_units = (int64_t)u.size();
  if (!units && capacity == 0) return NSP_OK;
  if (!units) return fail(NSP_EINVAL, "units is NULL");
  if (capacity < (int64_t)u.size())
    return fail(NSP_EINVAL, "capacity %lld < %zu units", (long long)capacity, u.size());
  for (size_t k = 0; k < u.size(); ++k) {
    units[4 * k] = u[k].x;
    units[4 * k + 1] = u[k].y;
    units[4 * k + 2] = u[k].z;
    units[4 * k + 3] = u[k].w;
  }
  return NSP_OK;
}

nsp_status nsp_attn_kv_queues(const nsp_worklist *wl, int32_t *queue_off) {
  g_last_error.clear();
  NSP_TRY(validate_worklist(wl, nullptr));
  if (!queue_off) return fail(NSP_EINVAL, "queue_off is NULL");
  const HostAttnSched hs = build_attn_schedule(wl);
  for (int x = 0; x <= kNumXcd; ++x) queue_off[x] = hs.kv_qoff[x];
  return NSP_OK;
}

nsp_status nsp_timing_enable(int32_t enable) {
  std::lock_guard<std::mutex> lock(g_timing.mu);
  g_timing.on = enable != 0;
  return NSP_OK;
}

// Fold completed event pairs into the totals (caller holds the lock).
static nsp_status timing_drain() {
  for (int k = 0; k < kNumKernels; ++k) {
    for (auto &ev : g_timing.pending[k]) {
      float ms = 0.f;
      hipError_t e = hipEventSynchronize(ev.second);
      if (e == hipSuccess) e = hipEventElapsedTime(&ms, ev.first, ev.second);
      (void)hipEventDestroy(ev.first);
      (void)hipEventDestroy(ev.second);
      if (e != hipSuccess) {
        g_timing.pending[k].clear();
        return fail(NSP_EHIP, "timing event: %s", hipGetErrorString(e));
      }
      g_timing.launches[k] += 1;
      g_timing.total_ms[k] += ms;
    }
    g_timing.pending[k].clear();
  }
  return NSP_OK;
}

nsp_status nsp_timing_reset(void) {
  g_last_error.clear();
  std::lock_guard<std::mutex> lock(g_timing.mu);
  nsp_status st = timing_drain();
  for (int k = 0; k < kNumKernels; ++k) {
    g_timing.launches[k] = 0;
    g_timing.total_ms[k] = 0.0;
  }
  return st;
}

nsp_status nsp_timing_query(const char *kernel, int64_t *launches, double *total_ms) {
  g_last_error.clear();
  if (!kernel || !launches || !total_ms) return fail(NSP_EINVAL, "NULL argument to nsp_timing_query");
  int id = -1;
  for (int k = 0; k < kNumKernels; ++k)
    if (strcmp(kernel, kKernelNames[k]) == 0) id = k;
  if (id < 0) return fail(NSP_EINVAL, "unknown kernel name '%s'", kernel);
  std::lock_guard<std::mutex> lock(g_timing.mu);
  NSP_TRY(timing_drain());
  *launches = g_timing.launches[id];
  *total_ms = g_timing.total_ms[id];
  return NSP_OK;
}

const char *nsp_status_string(nsp_status status) {
  switch (status) {
    case NSP_OK: return "NSP_OK";
    case NSP_EINVAL: return "NSP_EINVAL: invalid argument";
    case NSP_EUNSUPPORTED: return "NSP_EUNSUPPORTED: not supported";
    case NSP_EHIP: return "NSP_EHIP: HIP runtime error";
    case NSP_ENOMEM: return "NSP_ENOMEM: out of device memory";
    case NSP_EWORKSPACE: return "NSP_EWORKSPACE: workspace too small";
    case NSP_EINFEASIBLE: return "NSP_EINFEASIBLE: no plan meets the token budget";
    default: return "unknown nsp_status";
  }
}

const char *nsp_last_error(void) { return g_last_error.c_str(); }

const char *nsp_version(void) { return "nsp-mi355x 0.1.0 (gfx950)"; }

}  // extern "C"
