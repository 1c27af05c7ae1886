// SP-tree routing, the NSP planner (Design, NSP Planner): host code behind
// nsp_sp_tree_plan and nsp_sp_tree_worklist.
//
// The SP tree (Definition of the SP tree) is a complete binary tree over the
// W = 2^K ranks; node (d, i) covers the aligned ranks [i 2^(K-d),
// (i+1) 2^(K-d)) and has SP degree 2^(K-d).  A plan maps every sample to one
// node.  The planner follows the routing algorithm of the paper (Algorithm 1,
// prefix-completion SP-tree routing): samples by non-increasing length, a
// beam search over the longest k of them that keeps the w token-feasible
// partial plans of smallest critical load max_p C_p, then a greedy
// completion of every surviving plan on the leaves, returning the completed
// plan of smallest critical load.
//
// Cost model (Routing Objective and Cost Model), with the coefficients the
// paper takes from offline profiles given as parameters: per active node and
// pass, a Ulysses prologue, the local attention compute and an epilogue,
// summed over the nodes on a GPU's leaf-to-root path, plus non-attention
// time from the GPU's sharded token count; C_p = D_p(fwd) + D_p(bwd).
// Every per-node sum over samples (flops, bytes) and every token count is an
// exact integer; seconds are formed from them by one fixed expression, so a
// plan's costs do not depend on the order its samples were added.
#pragma clang fp contract(off)

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "nsp.h"
#include "nsp_internal.hpp"

namespace {

using nsp::set_error;

constexpr int kSums = 6;   // fwd flops, bwd flops, fwd prologue / epilogue bytes, bwd prologue / epilogue bytes

struct State {
  std::vector<int64_t> sums;    // per node, kSums exact sums
  std::vector<int32_t> count;   // samples per node
  std::vector<double> nf, nb;   // per active node, its phase seconds (fwd, bwd) per GPU
  std::vector<int64_t> tok;     // per GPU, Tok_p
  std::vector<double> df, db;   // per GPU, D_p(fwd), D_p(bwd)
  std::vector<int32_t> node;    // per sample (input order), node id or -1
  std::vector<int32_t> placed;  // samples placed, in processing order
};

struct Planner {
  const nsp_plan_params &p;
  const int64_t *len;
  int n, K, W, nodes;

  Planner(const nsp_plan_params &prm, const int64_t *lengths, int n_)
      : p(prm), len(lengths), n(n_), K(0), W(prm.world), nodes(0) {
    while ((1 << K) < W) ++K;
    nodes = 2 * W - 1;
  }
  static int id(int d, int i) { return (1 << d) - 1 + i; }
  static int depth_of(int u) {
    int d = 0;
    while ((2 << d) - 1 <= u) ++d;
    return d;
  }
  int degree(int d) const { return W >> d; }

  State empty() const {
    State s;
    s.sums.assign((size_t)nodes * kSums, 0);
    s.count.assign(nodes, 0);
    s.nf.assign(nodes, 0.0);
    s.nb.assign(nodes, 0.0);
    s.tok.assign(W, 0);
    s.df.assign(W, 0.0);
    s.db.assign(W, 0.0);
    s.node.assign(n, -1);
    return s;
  }

  // Per-sample contributions of sample j at a node of degree sp.
  void contrib(int64_t L, int sp, int64_t c[kSums]) const {
    const int64_t D = p.head_dim, hq = p.hq_total, eb = p.elem_bytes;
    const int64_t kvh = std::max<int64_t>(p.hkv_total, sp);
    const int64_t pairs = L * (L + 1) / 2, t = L / sp;
    c[0] = 4 * D * (hq / sp) * pairs;
    c[1] = 10 * D * (hq / sp) * pairs;
    c[2] = t * (hq + 2 * kvh) * D * eb;
    c[3] = t * hq * D * eb;
    c[4] = t * hq * D * eb;
    c[5] = t * (hq + 2 * kvh) * D * eb;
  }

  // Forward / backward seconds of one active node's three phases, per GPU.
  void phase_seconds(int sp, const int64_t *s, double &f, double &b) const {
    const double comp_f = (double)s[0] / p.attn_fwd_flops;
    const double comp_b = (double)s[1] / p.attn_bwd_flops;
    if (sp == 1) {
      f = comp_f;
      b = comp_b;
      return;
    }
    const double bw = (double)std::min(sp - 1, p.links) * p.link_bytes;
    const double frac = (double)(sp - 1) / (double)sp;
    const double prol_f = p.a2a_latency + (double)s[2] * frac / bw;
    const double epil_f = p.a2a_latency + (double)s[3] * frac / bw;
    const double prol_b = p.a2a_latency + (double)s[4] * frac / bw;
    const double epil_b = p.a2a_latency + (double)s[5] * frac / bw;
    f = (prol_f + comp_f) + epil_f;
    b = (prol_b + comp_b) + epil_b;
  }

  // D_p(fwd), D_p(bwd) of GPU g: the phase seconds of the active nodes on
  // its path, added root first, then the non-attention time.
  void gpu_cost(const State &s, int g, double &df, double &db) const {
    double af = 0.0, ab = 0.0;
    for (int d = 0; d <= K; ++d) {
      const int u = id(d, g >> (K - d));
      if (!s.count[u]) continue;
      af += s.nf[u];
      ab += s.nb[u];
    }
    df = af + (double)s.tok[g] * p.dense_fwd_per_token;
    db = ab + (double)s.tok[g] * p.dense_bwd_per_token;
  }

  void add(State &s, int j, int d, int i) const {
    const int u = id(d, i), sp = degree(d);
    int64_t c[kSums];
    contrib(len[j], sp, c);
    for (int q = 0; q < kSums; ++q) s.sums[(size_t)u * kSums + q] += c[q];
    ++s.count[u];
    phase_seconds(sp, &s.sums[(size_t)u * kSums], s.nf[u], s.nb[u]);
    for (int g = i * sp; g < (i + 1) * sp; ++g) {
      s.tok[g] += len[j] / sp;
      gpu_cost(s, g, s.df[g], s.db[g]);
    }
    s.node[j] = u;
    s.placed.push_back(j);
  }

  // Maxima of C_p and Tok_p over the GPUs before g (pre[g]) and from g on
  // (suf[g]): a probe then takes the GPUs outside its node from these.
  struct Extremes {
    std::vector<double> pre_c, suf_c, pre_t, suf_t;
  };
  void extremes(const State &s, Extremes &e) const {
    e.pre_c.assign(W + 1, -INFINITY);
    e.suf_c.assign(W + 1, -INFINITY);
    e.pre_t.assign(W + 1, -INFINITY);
    e.suf_t.assign(W + 1, -INFINITY);
    for (int g = 0; g < W; ++g) {
      e.pre_c[g + 1] = std::max(e.pre_c[g], s.df[g] + s.db[g]);
      e.pre_t[g + 1] = std::max(e.pre_t[g], (double)s.tok[g]);
    }
    for (int g = W - 1; g >= 0; --g) {
      e.suf_c[g] = std::max(e.suf_c[g + 1], s.df[g] + s.db[g]);
      e.suf_t[g] = std::max(e.suf_t[g + 1], (double)s.tok[g]);
    }
  }

  // max_p C_p and max_p Tok_p if sample j went to node (d, i), without
  // changing the state.  The GPUs outside the node come from `e`; for those
  // inside, the path above the node is the same for all of them, so its
  // partial sum is formed once (root first, as in gpu_cost), then the node's
  // new phase seconds and each GPU's own nodes below it are added.
  void probe(const State &s, const Extremes &e, int j, int d, int i, double &max_c, double &max_t) const {
    const int u = id(d, i), sp = degree(d), lo = i * sp, hi = (i + 1) * sp;
    int64_t c[kSums];
    contrib(len[j], sp, c);
    for (int q = 0; q < kSums; ++q) c[q] += s.sums[(size_t)u * kSums + q];
    double fu, bu;
    phase_seconds(sp, c, fu, bu);
    double af = 0.0, ab = 0.0;
    for (int dd = 0; dd < d; ++dd) {
      const int a = id(dd, i >> (d - dd));
      if (!s.count[a]) continue;
      af += s.nf[a];
      ab += s.nb[a];
    }
    af += fu;
    ab += bu;
    max_c = std::max(e.pre_c[lo], e.suf_c[hi]);
    max_t = std::max(e.pre_t[lo], e.suf_t[hi]);
    for (int g = lo; g < hi; ++g) {
      double gf = af, gb = ab;
      for (int dd = d + 1; dd <= K; ++dd) {
        const int a = id(dd, g >> (K - dd));
        if (!s.count[a]) continue;
        gf += s.nf[a];
        gb += s.nb[a];
      }
      const int64_t t = s.tok[g] + len[j] / sp;
      const double df = gf + (double)t * p.dense_fwd_per_token;
      const double db = gb + (double)t * p.dense_bwd_per_token;
      max_c = std::max(max_c, df + db);
      max_t = std::max(max_t, (double)t);
    }
  }

  double max_cost(const State &s) const {
    double m = -INFINITY;
    for (int g = 0; g < W; ++g) m = std::max(m, s.df[g] + s.db[g]);
    return m;
  }

  // The degree cap of the monotone-SP constraint for sample j.
  int cap(const State &s, int j) const {
    int c = p.sp_max;
    if (p.monotone)
      for (int jj : s.placed)
        if (len[jj] > len[j]) c = std::min(c, degree(depth_of(s.node[jj])));
    return c;
  }
};

struct Cand {
  double max_c;
  int parent, d, i;
};

bool pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

// A sample of length L can run at degree sp: the sequence and the query
// heads split evenly, and the KV heads split evenly or are replicated
// evenly.
bool admissible(const nsp_plan_params &p, int64_t L, int sp) {
  return L % sp == 0 && p.hq_total % sp == 0 && (p.hkv_total % sp == 0 || sp % p.hkv_total == 0);
}

nsp_status check_params(const nsp_plan_params *prm) {
  if (!prm) return set_error(NSP_EINVAL, "params is NULL");
  const nsp_plan_params &p = *prm;
  if (!pow2(p.world) || p.world > (1 << 16)) return set_error(NSP_EINVAL, "world %d is not a power of two in [1, 65536]", p.world);
  if (!pow2(p.sp_max) || p.sp_max > p.world) return set_error(NSP_EINVAL, "sp_max %d is not a power of two <= world", p.sp_max);
  if (p.hq_total < 1 || p.hkv_total < 1 || p.hq_total % p.hkv_total)
    return set_error(NSP_EINVAL, "head counts %d / %d", p.hq_total, p.hkv_total);
  if (p.head_dim < 1 || p.elem_bytes < 1) return set_error(NSP_EINVAL, "head_dim / elem_bytes must be positive");
  if (!(p.attn_fwd_flops > 0) || !(p.attn_bwd_flops > 0) || !(p.link_bytes > 0) || p.links < 1)
    return set_error(NSP_EINVAL, "throughputs, link bandwidth and links must be positive");
  if (!(p.a2a_latency >= 0) || !std::isfinite(p.a2a_latency) || !(p.dense_fwd_per_token >= 0) ||
      !std::isfinite(p.dense_fwd_per_token) || !(p.dense_bwd_per_token >= 0) || !std::isfinite(p.dense_bwd_per_token))
    return set_error(NSP_EINVAL, "latency and per-token costs must be finite and >= 0");
  if (!(p.token_budget > 0)) return set_error(NSP_EINVAL, "token_budget must be positive");
  if (p.prefix < 0 || p.beam < 1 || (p.monotone != 0 && p.monotone != 1))
    return set_error(NSP_EINVAL, "prefix >= 0, beam >= 1, monotone 0 or 1");
  return NSP_OK;
}

}  // namespace

extern "C" {

nsp_status nsp_sp_tree_plan(const nsp_plan_params *prm, const int64_t *lengths, int32_t n, int32_t *node_depth,
                            int32_t *node_index, double *gpu_cost, double *gpu_tokens, double *load) {
  set_error(NSP_OK, nullptr);
  const nsp_status st = check_params(prm);
  if (st != NSP_OK) return st;
  if (n < 0 || (n > 0 && (!lengths || !node_depth || !node_index)))
    return set_error(NSP_EINVAL, "n < 0 or a NULL lengths / node_depth / node_index");
  // every exact sum stays below 2^62: the largest is a node's backward flops
  // (at most 10 D Hq sum_j L_j (L_j+1)/2) or its epilogue bytes
  long double flops = 0, bytes = 0;
  for (int j = 0; j < n; ++j) {
    if (lengths[j] < 0 || lengths[j] > (1ll << 31)) return set_error(NSP_EINVAL, "length %lld of sample %d", (long long)lengths[j], j);
    flops += 10.0L * prm->head_dim * prm->hq_total * ((long double)lengths[j] * (lengths[j] + 1) / 2);
    bytes += (long double)lengths[j] * (prm->hq_total + 2.0L * std::max(prm->hkv_total, prm->world)) * prm->head_dim *
             prm->elem_bytes;
  }
  if (flops >= 0x1p62L || bytes >= 0x1p62L) return set_error(NSP_EINVAL, "batch too large for exact cost sums");

  const Planner pl(*prm, lengths, n);
  std::vector<int> order(n);
  for (int j = 0; j < n; ++j) order[j] = j;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return lengths[a] > lengths[b]; });
  const int k = std::min(prm->prefix, n);

  // long-prefix tree search
  std::vector<State> beam{pl.empty()};
  std::vector<Cand> cand;
  Planner::Extremes ext;
  for (int step = 0; step < k; ++step) {
    const int j = order[step];
    cand.clear();
    for (int b = 0; b < (int)beam.size(); ++b) {
      const State &s = beam[b];
      const int cap = pl.cap(s, j);
      pl.extremes(s, ext);
      for (int d = 0; d <= pl.K; ++d) {
        const int sp = pl.degree(d);
        if (sp > cap || !admissible(*prm, lengths[j], sp)) continue;
        for (int i = 0; i < (1 << d); ++i) {
          double mc, mt;
          pl.probe(s, ext, j, d, i, mc, mt);
          if (mt <= prm->token_budget) cand.push_back({mc, b, d, i});
        }
      }
    }
    if (cand.empty())
      return set_error(NSP_EINFEASIBLE, "no placement of sample %d (length %lld) meets the token budget", j,
                       (long long)lengths[j]);
    std::stable_sort(cand.begin(), cand.end(), [](const Cand &a, const Cand &b) { return a.max_c < b.max_c; });
    std::vector<State> next;
    next.reserve(std::min<size_t>(cand.size(), (size_t)prm->beam));
    for (size_t c = 0; c < cand.size() && (int)c < prm->beam; ++c) {
      next.push_back(beam[cand[c].parent]);
      pl.add(next.back(), j, cand[c].d, cand[c].i);
    }
    beam.swap(next);
  }

  // greedy short-tail completion on the leaves (single GPUs)
  int best = -1;
  double best_c = 0;
  for (int b = 0; b < (int)beam.size(); ++b) {
    State &s = beam[b];
    for (int step = k; step < n; ++step) {
      const int j = order[step];
      int u = -1;
      for (int g = 0; g < pl.W; ++g)
        if ((double)s.tok[g] + (double)lengths[j] <= prm->token_budget &&
            (u < 0 || s.df[g] + s.db[g] < s.df[u] + s.db[u]))
          u = g;
      if (u < 0) {
        u = 0;
        for (int g = 1; g < pl.W; ++g)
          if (s.tok[g] < s.tok[u]) u = g;
      }
      pl.add(s, j, pl.K, u);
    }
    const double mc = pl.max_cost(s);
    if (best < 0 || mc < best_c) {
      best = b;
      best_c = mc;
    }
  }
  const State &s = beam[best];
  double mf = -INFINITY, mb = -INFINITY;
  for (int g = 0; g < pl.W; ++g) {
    mf = std::max(mf, s.df[g]);
    mb = std::max(mb, s.db[g]);
    if (gpu_cost) gpu_cost[g] = s.df[g] + s.db[g];
    if (gpu_tokens) gpu_tokens[g] = (double)s.tok[g];
  }
  for (int j = 0; j < n; ++j) {
    const int d = Planner::depth_of(s.node[j]);
    node_depth[j] = d;
    node_index[j] = s.node[j] - ((1 << d) - 1);
  }
  if (load) *load = n ? mf + mb : 0.0;
  return NSP_OK;
}

nsp_status nsp_sp_tree_worklist(const nsp_plan_params *prm, const int64_t *lengths, int32_t n,
                                const int32_t *node_depth, const int32_t *node_index, int32_t gpu, int32_t *n_items,
                                int32_t *sample, int32_t *cu_seqlens, int32_t *q_heads, int32_t *kv_heads,
                                int32_t *sp) {
  set_error(NSP_OK, nullptr);
  const nsp_status st = check_params(prm);
  if (st != NSP_OK) return st;
  if (n < 0 || !n_items || !cu_seqlens || (n > 0 && (!lengths || !node_depth || !node_index || !sample || !q_heads ||
                                                     !kv_heads || !sp)))
    return set_error(NSP_EINVAL, "n < 0 or a NULL argument");
  if (gpu < 0 || gpu >= prm->world) return set_error(NSP_EINVAL, "gpu %d outside [0, %d)", gpu, prm->world);
  int K = 0;
  while ((1 << K) < prm->world) ++K;
  for (int j = 0; j < n; ++j) {
    const int d = node_depth[j], i = node_index[j];
    if (d < 0 || d > K || i < 0 || i >= (1 << d)) return set_error(NSP_EINVAL, "node (%d, %d) of sample %d", d, i, j);
    const int deg = prm->world >> d;
    if (deg > prm->sp_max || lengths[j] < 0 || !admissible(*prm, lengths[j], deg))
      return set_error(NSP_EINVAL, "sample %d (length %lld) cannot run at degree %d", j, (long long)lengths[j], deg);
  }
  int m = 0;
  int64_t cu = 0;
  cu_seqlens[0] = 0;
  for (int d = 0; d <= K; ++d) {             // root first
    const int deg = prm->world >> d;
    for (int j = 0; j < n; ++j) {
      if (node_depth[j] != d || gpu / deg != node_index[j]) continue;
      const int r = gpu - node_index[j] * deg;
      const int hq = prm->hq_total, hkv = prm->hkv_total;
      cu += lengths[j];
      if (cu > INT32_MAX) return set_error(NSP_EINVAL, "work list of GPU %d exceeds 2^31 - 1 tokens", gpu);
      sample[m] = j;
      cu_seqlens[m + 1] = (int32_t)cu;
      q_heads[2 * m] = r * hq / deg;
      q_heads[2 * m + 1] = (r + 1) * hq / deg;
      kv_heads[2 * m] = r * hkv / deg;
      kv_heads[2 * m + 1] = deg <= hkv ? (r + 1) * hkv / deg : r * hkv / deg + 1;
      sp[m] = deg;
      ++m;
    }
  }
  *n_items = m;
  return NSP_OK;
}

}  // extern "C"
