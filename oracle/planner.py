"""SP-tree routing (the NSP Planner), written out step by step (plain Python).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py): never imported by the
product path.

What it follows:
  * Design, NSP Planner, SP Tree Topology (Definition of the SP tree): node
    (d, i), 0 <= d <= K, 0 <= i < 2^d, holds the aligned rank range
    [i 2^(K-d), (i+1) 2^(K-d)); its SP degree is 2^(K-d); leaves are single
    GPUs.
  * Routing Objective and Cost Model: the sharded token load
    Tok_p(a) = sum over samples j whose node covers p of L_j / |R(a(j))|,
    the backend phase costs (prologue, compute, epilogue per pass) summed
    over the active nodes on p's leaf-to-root path, plus the non-attention
    time from the token count, D_p = A_p + O_p per pass; the planner's
    per-GPU scalar C_p = D_p(fwd) + D_p(bwd); the iteration proxy
    Load = max_p D_p(fwd) + max_p D_p(bwd).
  * Routing Algorithm (Algorithm 1, prefix-completion SP-tree routing):
    sort by non-increasing length; beam search over the first k samples,
    keeping the w states of smallest max_p C_p among the token-feasible
    extensions; greedy completion of the tail on the leaf units (least
    loaded feasible unit, else the unit of smallest token load); return the
    completed state of smallest max_p C_p.  Optional monotone-SP constraint:
    a sample never takes a smaller SP degree than a longer one.

Readings where the paper is silent (also listed in the design notes):
  1. The cost model's coefficients come from offline profiles the paper does
     not give.  Here they are parameters: per-GPU attention throughput per
     pass (counted flops: 4 D per causal pair and query head forward, 10 D
     backward), one GPU-GPU link's bandwidth and the links per GPU, a latency
     per all-to-all, and the non-attention seconds per token per pass.
  2. Backend = Ulysses.  A sample at a node of degree sp > 1 holds L/sp
     tokens per GPU; each GPU sends (sp-1)/sp of the tensors of a phase,
     spread over min(sp-1, links) links: forward prologue Q, K, V, forward
     epilogue O, backward prologue dO, backward epilogue dQ, dK, dV.  K, V,
     dK, dV count max(Hkv, sp) heads (KV heads are replicated when
     sp > Hkv).  One all-to-all (one latency) per phase per active node;
     degree 1 nodes communicate nothing.  Attention compute per GPU is the
     counted flops of Hq/sp query heads over the full sample.
  3. All sums over samples are kept as exact integers (flops, bytes, tokens)
     and turned into seconds per node and GPU by one fixed expression, so the
     result does not depend on the order samples were added.
  4. FeasibleNodes(T, S, j): nodes of degree <= sp_max with L_j divisible by
     the degree, Hq divisible by the degree and Hkv divisible by it or
     dividing it (the head split a Ulysses group can run), and (monotone)
     degree <= the degree of every placed strictly longer sample; enumerated
     root first (depth ascending), then by index.
  5. Ties: the beam keeps the first states in generation order among equal
     max_p C_p (stable sort); the tail picks the smallest unit index among
     equals; the returned state is the first in beam order among equals.
  6. "Effective leaf units" for the tail are the leaves (single GPUs): every
     tail sample is at most as long as every prefix sample, so degree 1 is
     always admissible under the monotone constraint.
  7. If no extension of the prefix meets the token budget the planner fails
     (returns None); the tail never fails (its fallback ignores the budget).
  8. Samples of equal length keep their input order (stable sort).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

__all__ = ["PlanParams", "Plan", "node_ranks", "tok_loads", "gpu_costs", "plan", "worklist_for_gpu"]


@dataclass(frozen=True)
class PlanParams:
    world: int                 # W GPUs, a power of two
    sp_max: int                # largest SP degree, a power of two <= world
    hq: int                    # query heads of the model
    hkv: int                   # KV heads
    head_dim: int
    elem_bytes: int = 2
    attn_fwd_flops: float = 1.2e15     # counted flop/s of one GPU's attention, forward
    attn_bwd_flops: float = 9.0e14     # backward
    link_bytes: float = 153e9          # bytes/s of one link
    links: int = 7                     # links per GPU
    a2a_latency: float = 20e-6         # seconds per all-to-all
    dense_fwd_per_token: float = 0.0   # seconds per token of non-attention work, forward
    dense_bwd_per_token: float = 0.0   # backward
    token_budget: float = float("inf") # B_tok, tokens per GPU
    prefix: int = 16                   # k
    beam: int = 8                      # w
    monotone: bool = True


@dataclass
class Plan:
    node: List[Tuple[int, int]]        # per sample (input order): (depth, index)
    cost: List[float]                  # C_p
    tokens: List[float]                # Tok_p
    load: float                        # max_p D_p(fwd) + max_p D_p(bwd)


def _K(world: int) -> int:
    return world.bit_length() - 1


def node_ranks(world: int, d: int, i: int) -> range:
    """R(u) of node u = (d, i) (Definition of the SP tree)."""
    size = world >> d
    return range(i * size, (i + 1) * size)


def tok_loads(prm: PlanParams, lengths: Sequence[int], assign: Sequence[Tuple[int, Tuple[int, int]]]) -> List[float]:
    """Tok_p for a partial assignment [(sample, (d, i)), ...]."""
    tok = [0] * prm.world
    for j, (d, i) in assign:
        R = node_ranks(prm.world, d, i)
        for p in R:
            tok[p] += lengths[j] // len(R)
    return [float(t) for t in tok]


def _node_sums(prm: PlanParams, lengths, assign):
    """Per active node: exact integer sums over its samples of the forward /
    backward counted flops and the bytes each GPU sends per phase."""
    D, hq, hkv, eb = prm.head_dim, prm.hq, prm.hkv, prm.elem_bytes
    sums = {}
    for j, u in assign:
        sp = prm.world >> u[0]
        L = lengths[j]
        pairs = L * (L + 1) // 2
        t = L // sp                                   # tokens per GPU of the node
        kvh = max(hkv, sp)
        s = sums.setdefault(u, [0, 0, 0, 0, 0, 0])
        s[0] += 4 * D * (hq // sp) * pairs            # forward flops per GPU
        s[1] += 10 * D * (hq // sp) * pairs           # backward flops per GPU
        s[2] += t * (hq + 2 * kvh) * D * eb           # forward prologue bytes: Q, K, V
        s[3] += t * hq * D * eb                       # forward epilogue: O
        s[4] += t * hq * D * eb                       # backward prologue: dO
        s[5] += t * (hq + 2 * kvh) * D * eb           # backward epilogue: dQ, dK, dV
    return sums


def _phase_seconds(prm: PlanParams, sp: int, s) -> Tuple[float, float]:
    """(forward, backward) seconds of one active node's three phases on each
    of its GPUs: prologue + compute + epilogue."""
    comp_f = s[0] / prm.attn_fwd_flops
    comp_b = s[1] / prm.attn_bwd_flops
    if sp == 1:
        return comp_f, comp_b
    bw = min(sp - 1, prm.links) * prm.link_bytes
    frac = (sp - 1) / sp
    prol_f = prm.a2a_latency + s[2] * frac / bw
    epil_f = prm.a2a_latency + s[3] * frac / bw
    prol_b = prm.a2a_latency + s[4] * frac / bw
    epil_b = prm.a2a_latency + s[5] * frac / bw
    return (prol_f + comp_f) + epil_f, (prol_b + comp_b) + epil_b


def gpu_costs(prm: PlanParams, lengths, assign) -> Tuple[List[float], List[float], List[float], List[float]]:
    """(C_p, Tok_p, D_p fwd, D_p bwd) of a partial assignment, from scratch."""
    K = _K(prm.world)
    tok = tok_loads(prm, lengths, assign)
    sums = _node_sums(prm, lengths, assign)
    cf, cb, cost = [], [], []
    for p in range(prm.world):
        af = ab = 0.0
        for d in range(K + 1):                        # p's leaf-to-root path, root first
            u = (d, p >> (K - d))
            if u in sums:
                f, b = _phase_seconds(prm, prm.world >> d, sums[u])
                af += f
                ab += b
        df = af + tok[p] * prm.dense_fwd_per_token
        db = ab + tok[p] * prm.dense_bwd_per_token
        cf.append(df)
        cb.append(db)
        cost.append(df + db)
    return cost, tok, cf, cb


def _feasible_nodes(prm: PlanParams, lengths, assign, j) -> List[Tuple[int, int]]:
    K = _K(prm.world)
    cap = prm.sp_max
    if prm.monotone:
        for jj, (d, _) in assign:
            if lengths[jj] > lengths[j]:
                cap = min(cap, prm.world >> d)
    out = []
    for d in range(K + 1):
        sp = prm.world >> d
        if sp > cap or lengths[j] % sp or prm.hq % sp or (prm.hkv % sp and sp % prm.hkv):
            continue
        for i in range(1 << d):
            out.append((d, i))
    return out


def plan(prm: PlanParams, lengths: Sequence[int]) -> Optional[Plan]:
    """Algorithm 1 (prefix-completion SP-tree routing)."""
    lengths = [int(x) for x in lengths]
    order = sorted(range(len(lengths)), key=lambda j: -lengths[j])      # stable
    k = min(prm.prefix, len(order))
    head, rest = order[:k], order[k:]

    # states (a, C, T): a = [(sample, node), ...]
    beam = [([], [0.0] * prm.world, [0.0] * prm.world)]
    for j in head:                                    # long-prefix tree search
        nxt = []
        for a, _, _ in beam:
            for u in _feasible_nodes(prm, lengths, a, j):
                a2 = a + [(j, u)]
                C2, T2, _, _ = gpu_costs(prm, lengths, a2)
                if max(T2) <= prm.token_budget:
                    nxt.append((a2, C2, T2))
        if not nxt:
            return None
        nxt.sort(key=lambda s: max(s[1]))             # stable: generation order among ties
        beam = nxt[:prm.beam]

    K = _K(prm.world)
    done = []
    for a, C, T in beam:                              # greedy short-tail completion
        a = list(a)
        for j in rest:
            best = None
            for i in range(prm.world):                # leaf units (K, i), GPU i
                if T[i] + lengths[j] <= prm.token_budget and (best is None or C[i] < C[best]):
                    best = i
            if best is None:
                best = min(range(prm.world), key=lambda i: (T[i], i))
            a.append((j, (K, best)))
            C, T, _, _ = gpu_costs(prm, lengths, a)
        done.append((a, C, T))
    a, C, T = min(done, key=lambda s: max(s[1]))     # first among ties
    node = [None] * len(lengths)
    for j, u in a:
        node[j] = u
    _, _, cf, cb = gpu_costs(prm, lengths, a)
    return Plan(node=node, cost=C, tokens=T, load=max(cf) + max(cb))


def worklist_for_gpu(prm: PlanParams, lengths, node, p: int):
    """GPU p's items under a plan, root first (decreasing degree, then sample
    order): (sample, L, sp, q_heads [lo, hi), kv_heads [lo, hi)), rank r of p
    within the node holding query heads [r Hq/sp, (r+1) Hq/sp) and KV heads
    [r Hkv/sp, (r+1) Hkv/sp), or the one KV head floor(r Hkv/sp) when
    sp > Hkv."""
    K = _K(prm.world)
    items = []
    for d in range(K + 1):
        for j, (dd, i) in enumerate(node):
            if dd != d or p not in node_ranks(prm.world, d, i):
                continue
            sp = prm.world >> d
            r = p - i * sp
            q = (r * prm.hq // sp, (r + 1) * prm.hq // sp)
            if sp <= prm.hkv:
                kv = (r * prm.hkv // sp, (r + 1) * prm.hkv // sp)
            else:
                kv = (r * prm.hkv // sp, r * prm.hkv // sp + 1)
            items.append((j, lengths[j], sp, q, kv))
    return items
