// Host code of libnsp under AddressSanitizer / UndefinedBehaviorSanitizer:
// work-list validation, the unit schedule, the recompute plan, the SP-tree
// planner and the argument checks of every entry point, on seeded random and
// malformed inputs.  Built with g++ from the library's host sources and
// tests/native/launch_stubs.cpp; run by tests/test_host_sanitizers.py on a
// machine without a GPU.  Prints "host checks ok" and exits 0 on success.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <set>
#include <tuple>
#include <vector>

#include "nsp.h"

#define CHECK(c)                                                            \
  do {                                                                      \
    if (!(c)) {                                                             \
      std::fprintf(stderr, "%s:%d: check failed: %s (%s)\n", __FILE__,      \
                   __LINE__, #c, nsp_last_error());                         \
      std::exit(1);                                                         \
    }                                                                       \
  } while (0)

namespace {

std::mt19937_64 rng(20260);
int uni(int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); }

struct Wl {
  std::vector<int32_t> cu, qh, kvh, sp;
  std::vector<uint8_t> mask;
  nsp_worklist w{};
  void finish(int hq, int hkv, int D, bool with_mask) {
    w.n_items = (int)sp.size();
    w.cu_seqlens = cu.data();
    w.q_heads = qh.data();
    w.kv_heads = kvh.data();
    w.sp = sp.data();
    w.hq_total = hq;
    w.hkv_total = hkv;
    w.head_dim = D;
    w.item_mask = with_mask ? mask.data() : nullptr;
  }
};

// A random valid work list: items of rank r at degree s (the rank's query
// heads and its KV heads, or the one replicated KV head).
Wl random_wl(int hq, int hkv, int D, int n, int maxL, bool with_mask) {
  Wl x;
  x.cu.push_back(0);
  for (int j = 0; j < n; ++j) {
    int s = 1 << uni(0, 3);
    while (hq % s) s >>= 1;
    if (!(hkv % s == 0 || s % hkv == 0)) s = 1;
    int L = uni(0, 9) == 0 ? uni(0, 2) : uni(0, maxL);
    L -= L % s;
    const int r = uni(0, s - 1);
    const int hl = hq / s;
    x.qh.insert(x.qh.end(), {r * hl, (r + 1) * hl});
    if (hkv >= s) {
      const int kl = hkv / s;
      x.kvh.insert(x.kvh.end(), {r * kl, (r + 1) * kl});
    } else {
      const int g = r * hkv / s;
      x.kvh.insert(x.kvh.end(), {g, g + 1});
    }
    x.sp.push_back(s);
    x.cu.push_back(x.cu.back() + L);
    x.mask.push_back((uint8_t)uni(0, 1));
  }
  x.finish(hq, hkv, D, with_mask);
  return x;
}

void check_schedule(const Wl &x) {
  const nsp_worklist &w = x.w;
  for (int which : {NSP_SCHED_FWD, NSP_SCHED_KV}) {
    int64_t n = -1;
    CHECK(nsp_attn_schedule(&w, which, nullptr, 0, &n) == NSP_OK && n >= 0);
    std::vector<int32_t> u(4 * (size_t)n + 4);
    int64_t m = -1;
    CHECK(nsp_attn_schedule(&w, which, u.data(), n, &m) == NSP_OK && m == n);
    if (n > 0) CHECK(nsp_attn_schedule(&w, which, u.data(), n - 1, &m) == NSP_EINVAL);
    // every (item, tile, head) once; tiles and heads in range
    std::set<std::tuple<int, int, int>> seen;
    int64_t want = 0;
    for (int j = 0; j < w.n_items; ++j) {
      const int L = w.cu_seqlens[j + 1] - w.cu_seqlens[j];
      if (L == 0 || (w.item_mask && !w.item_mask[j])) continue;
      const int hq = w.q_heads[2 * j + 1] - w.q_heads[2 * j], hkv = w.kv_heads[2 * j + 1] - w.kv_heads[2 * j];
      want += which == NSP_SCHED_FWD ? (int64_t)hq * ((L + 255) / 256) : (int64_t)hkv * ((L + 127) / 128);
    }
    CHECK(want == n);
    for (int64_t k = 0; k < n; ++k) {
      const int j = u[4 * k], t = u[4 * k + 1], a = u[4 * k + 2], g = u[4 * k + 3];
      CHECK(j >= 0 && j < w.n_items);
      const int L = w.cu_seqlens[j + 1] - w.cu_seqlens[j];
      const int hq = w.q_heads[2 * j + 1] - w.q_heads[2 * j], hkv = w.kv_heads[2 * j + 1] - w.kv_heads[2 * j];
      CHECK(g >= 0 && g < hkv);
      if (which == NSP_SCHED_FWD) {
        CHECK(t >= 0 && 256 * t < L && a >= 0 && a < hq);
        CHECK(seen.insert({j, t, a}).second);
      } else {
        // key tile, and the flag of the units that sweep down from the item end
        const int n = t & ((1 << 30) - 1), nk = (L + 127) / 128;
        CHECK(n >= 0 && n < nk && (a & 0xffff) <= (a >> 16) && (a >> 16) <= hq);
        CHECK(((t >> 30) & 1) == (n < nk / 2 ? 1 : 0));
        CHECK(seen.insert({j, n, g}).second);
      }
    }
    if (which == NSP_SCHED_KV) {
      int32_t off[9];
      CHECK(nsp_attn_kv_queues(&w, off) == NSP_OK);
      CHECK(off[0] == 0 && off[8] == n);
      for (int x = 0; x < 8; ++x) CHECK(off[x] <= off[x + 1]);
      CHECK(nsp_attn_kv_queues(&w, nullptr) == NSP_EINVAL);
    }
  }
}

void check_recompute(const Wl &x) {
  std::vector<uint8_t> save(x.sp.size() + 1, 7);
  for (int64_t budget : {int64_t(0), int64_t(1) << 20, int64_t(1) << 40}) {
    int64_t saved = -1;
    for (nsp_dtype dt : {NSP_BF16, NSP_F32}) {
      CHECK(nsp_recompute_plan(&x.w, budget, dt, save.data(), &saved) == NSP_OK);
      CHECK(saved >= 0 && saved <= budget);
      for (size_t j = 0; j < x.sp.size(); ++j) CHECK(save[j] <= 1);
    }
  }
  CHECK(nsp_recompute_plan(&x.w, -1, NSP_BF16, save.data(), nullptr) == NSP_EINVAL);
  CHECK(nsp_recompute_plan(&x.w, 0, (nsp_dtype)9, save.data(), nullptr) == NSP_EINVAL);
}

void check_malformed(const Wl &good) {
  const uintptr_t kFake = 0x10000;
  const void *F = (const void *)kFake;
  Wl x = good;
  x.finish(good.w.hq_total, good.w.hkv_total, good.w.head_dim, false);
  auto fwd = [&](const nsp_worklist *w) {
    return nsp_varlen_attn_fwd(w, 0.1f, 1, F, F, F, (void *)F, NSP_BF16, (float *)F, nullptr);
  };
  if (x.w.n_items > 1 && x.cu[1] < x.cu[x.w.n_items]) {
    Wl bad = x;
    std::swap(bad.cu[1], bad.cu[bad.w.n_items]);   // decreasing prefix sums
    bad.finish(x.w.hq_total, x.w.hkv_total, x.w.head_dim, false);
    CHECK(fwd(&bad.w) == NSP_EINVAL);
    CHECK(nsp_attn_schedule(&bad.w, NSP_SCHED_FWD, nullptr, 0, nullptr) == NSP_EINVAL);
  }
  if (x.w.n_items > 0) {
    Wl bad = x;
    bad.qh[1] = bad.w.hq_total + 1;                  // head range past hq_total
    bad.finish(x.w.hq_total, x.w.hkv_total, x.w.head_dim, false);
    CHECK(fwd(&bad.w) == NSP_EINVAL);
    Wl bad2 = x;
    bad2.kvh[0] = bad2.kvh[1];                       // empty KV range
    bad2.finish(x.w.hq_total, x.w.hkv_total, x.w.head_dim, false);
    CHECK(fwd(&bad2.w) == NSP_EINVAL);
  }
  Wl d96 = x;
  d96.finish(x.w.hq_total, x.w.hkv_total, 96, false);
  CHECK(fwd(&d96.w) == NSP_EUNSUPPORTED);
  CHECK(nsp_varlen_attn_fwd(&x.w, 0.1f, 0, F, F, F, (void *)F, NSP_BF16, (float *)F, nullptr) ==
        (x.w.n_items ? NSP_EUNSUPPORTED : NSP_EUNSUPPORTED));
  CHECK(nsp_varlen_attn_fwd(&x.w, -1.f, 1, F, F, F, (void *)F, NSP_BF16, (float *)F, nullptr) == NSP_EINVAL);
  // the backward: workspace too small, misaligned, bad dtypes
  const size_t ws = nsp_varlen_attn_bwd_workspace(&x.w);
  CHECK(ws >= 256);
  bool any = false;
  for (int j = 0; j < x.w.n_items; ++j) any |= x.cu[j + 1] > x.cu[j];
  if (any) {
    CHECK(nsp_varlen_attn_bwd(&x.w, 0.1f, 1, F, F, F, F, NSP_BF16, F, (const float *)F, (void *)F, (void *)F,
                              (void *)F, NSP_BF16, (void *)F, ws - 1, nullptr) == NSP_EWORKSPACE);
    CHECK(nsp_varlen_attn_bwd(&x.w, 0.1f, 1, F, F, F, F, NSP_BF16, F, (const float *)F, (void *)F, (void *)F,
                              (void *)F, (nsp_dtype)4, (void *)F, ws, nullptr) == NSP_EINVAL);
    CHECK(nsp_varlen_attn_bwd(&x.w, 0.1f, 1, F, F, F, F, NSP_BF16, F, (const float *)F, (void *)F, (void *)F,
                              (void *)F, NSP_BF16, (void *)(kFake + 16), ws, nullptr) == NSP_EINVAL);
    CHECK(nsp_varlen_attn_bwd(&x.w, 0.1f, 1, F, F, F, F, NSP_BF16, F, (const float *)F, (void *)F, (void *)F,
                              (void *)(kFake + 8), NSP_BF16, (void *)F, ws, nullptr) == NSP_EINVAL);
    CHECK(nsp_varlen_attn_bwd_noalloc(&x.w, 0.1f, 1, F, F, F, F, NSP_BF16, F, (const float *)F, (void *)F,
                                      (void *)F, nullptr, NSP_BF16, nullptr) == NSP_EINVAL);
    // valid arguments: with no device the call stops at its first HIP call
    CHECK(fwd(&x.w) == NSP_EHIP);
    CHECK(nsp_varlen_attn_bwd(&x.w, 0.1f, 1, F, F, F, F, NSP_BF16, F, (const float *)F, (void *)F, (void *)F,
                              (void *)F, NSP_BF16, (void *)F, ws, nullptr) == NSP_EHIP);
    CHECK(nsp_varlen_attn_bwd_noalloc(&x.w, 0.1f, 1, F, F, F, F, NSP_BF16, F, (const float *)F, (void *)F,
                                      (void *)F, (void *)F, NSP_BF16, nullptr) == NSP_EHIP);
  }
  // pack / unpack: sp must divide the length and pair with the head counts
  if (any) {
    CHECK(nsp_ulysses_pack(&x.w, (nsp_kind)3, NSP_BF16, F, (void *)F, nullptr) == NSP_EINVAL);
    CHECK(nsp_ulysses_unpack(&x.w, NSP_KIND_KV, NSP_BF16, (nsp_replica)5, F, (void *)F, nullptr) == NSP_EINVAL);
    CHECK(nsp_ulysses_pack(&x.w, NSP_KIND_Q, NSP_BF16, F, (void *)F, nullptr) == NSP_EHIP);
  }
  // the executor: node lists that do not match the items' degrees
  std::set<int32_t> sps(x.sp.begin(), x.sp.end());
  std::vector<int32_t> nodes(sps.rbegin(), sps.rend());
  nsp_step_buffers b;
  std::memset(&b, 0, sizeof b);
  if (!nodes.empty()) {
    std::vector<int32_t> dup(nodes);
    dup.push_back(nodes[0]);
    CHECK(nsp_executor_step(&x.w, dup.data(), (int32_t)dup.size(), NSP_STEP_FORWARD, 0.1f, &b, nullptr, nullptr) ==
          NSP_EINVAL);
    std::vector<int32_t> extra(nodes);
    extra.push_back(1 << 20);
    CHECK(nsp_executor_step(&x.w, extra.data(), (int32_t)extra.size(), NSP_STEP_FORWARD, 0.1f, &b, nullptr,
                            nullptr) == NSP_EINVAL);
    CHECK(nsp_executor_step(&x.w, nodes.data(), (int32_t)nodes.size(), NSP_STEP_FORWARD, 0.1f, &b, nullptr,
                            nullptr) == NSP_EINVAL);   // NULL buffers
  }
}

void check_planner() {
  for (int it = 0; it < 60; ++it) {
    nsp_plan_params p{};
    p.world = 1 << uni(0, 6);
    p.sp_max = 1 << uni(0, __builtin_ctz(p.world));
    p.hq_total = 32;
    p.hkv_total = uni(0, 1) ? 4 : 8;
    p.head_dim = 128;
    p.elem_bytes = 2;
    p.attn_fwd_flops = 1.2e15;
    p.attn_bwd_flops = 0.9e15;
    p.link_bytes = 153e9;
    p.links = 7;
    p.a2a_latency = 2e-5;
    p.dense_fwd_per_token = 2e-7;
    p.dense_bwd_per_token = 4e-7;
    p.prefix = uni(0, 12);
    p.beam = uni(1, 6);
    p.monotone = uni(0, 1);
    const int n = uni(0, 120);
    std::vector<int64_t> len(n);
    int64_t total = 0;
    for (auto &L : len) {
      L = uni(0, 4) == 0 ? uni(0, 3) : uni(1, 70000);
      total += L;
    }
    p.token_budget = uni(0, 3) == 0 ? 1e30 : 1.5 * (double)total / p.world + 70000;
    std::vector<int32_t> d(n + 1), i(n + 1);
    std::vector<double> cost(p.world), tok(p.world);
    double load = -1;
    const nsp_status st = nsp_sp_tree_plan(&p, len.data(), n, d.data(), i.data(), cost.data(), tok.data(), &load);
    CHECK(st == NSP_OK || st == NSP_EINFEASIBLE);
    if (st != NSP_OK) continue;
    CHECK(load >= 0);
    int64_t seen = 0;
    for (int g = 0; g < p.world; ++g) {
      int32_t m = -1;
      std::vector<int32_t> sample(n + 1), cu(n + 2), qh(2 * n + 2), kvh(2 * n + 2), sp(n + 1);
      CHECK(nsp_sp_tree_worklist(&p, len.data(), n, d.data(), i.data(), g, &m, sample.data(), cu.data(), qh.data(),
                                 kvh.data(), sp.data()) == NSP_OK);
      CHECK(m >= 0 && m <= n && cu[0] == 0);
      for (int k = 0; k < m; ++k) {
        CHECK(sample[k] >= 0 && sample[k] < n && sp[k] >= 1);
        CHECK(cu[k + 1] - cu[k] == len[sample[k]]);
        seen += (int64_t)(qh[2 * k + 1] - qh[2 * k]);
      }
    }
    int64_t want = 0;
    for (int k = 0; k < n; ++k) want += p.hq_total;   // every sample's query heads once over the GPUs
    CHECK(seen == want);
  }
  nsp_plan_params bad{};
  bad.world = 3;
  int32_t d = 0, i = 0;
  int64_t L = 5;
  CHECK(nsp_sp_tree_plan(&bad, &L, 1, &d, &i, nullptr, nullptr, nullptr) == NSP_EINVAL);
}

}  // namespace

int main() {
  int devices = 0;
  if (hipGetDeviceCount(&devices) == hipSuccess && devices > 0) {
    std::printf("host checks need a machine without a GPU; skipped\n");
    return 0;
  }
  for (int it = 0; it < 400; ++it) {
    const int kind = uni(0, 3);
    const int hq = kind == 0 ? 32 : kind == 1 ? 8 : kind == 2 ? 16 : 4;
    const int hkv = kind == 0 ? 4 : kind == 1 ? 2 : kind == 2 ? 16 : 1;
    const int D = uni(0, 1) ? 128 : 64;
    const Wl x = random_wl(hq, hkv, D, uni(0, 30), uni(1, 6000), uni(0, 2) == 0);
    check_schedule(x);
    check_recompute(x);
    check_malformed(x);
  }
  check_planner();
  CHECK(nsp_timing_enable(1) == NSP_OK && nsp_timing_reset() == NSP_OK);
  int64_t launches = -1;
  double ms = -1;
  CHECK(nsp_timing_query("attn_fwd", &launches, &ms) == NSP_OK && launches == 0);
  CHECK(nsp_timing_query("nope", &launches, &ms) == NSP_EINVAL);
  CHECK(nsp_timing_enable(0) == NSP_OK);
  CHECK(std::strlen(nsp_status_string(NSP_EWORKSPACE)) > 0 && std::strlen(nsp_version()) > 0);
  std::printf("host checks ok\n");
  return 0;
}
