"""Pins of the SP-tree planner oracle (oracle/planner.py) against things other
than itself: the SP-tree definition (nested aligned rank ranges), exhaustive
search over every plan of tiny batches, the classic LPT list schedule for the
greedy tail, conservation of tokens and of attention work over any plan, a
hand-worked cost example, and head coverage of the per-GPU work lists.

Which mistake each pin catches:
  * ranges      -- wrong rank range of a node (shift, size, off by one);
  * exhaustive  -- beam / prefix bookkeeping: a state dropped, wrong argmin,
                   a feasible node missing from FeasibleNodes, the budget test;
  * lpt         -- tail: wrong unit choice (most instead of least loaded),
                   wrong order of the tail samples;
  * tokens, work -- Tok_p or the compute term missing the 1/sp share, a node
                   counted on GPUs outside its range, a path node skipped;
  * hand-worked -- the communication term (fraction (sp-1)/sp, links, bytes
                   per phase, replicated KV heads, latency per phase);
  * monotone    -- the monotone-SP constraint;
  * worklist    -- query / KV head ranges of a rank within its node.
"""
import itertools
import math
import random

import pytest

from oracle import planner as P


def _prm(**kw):
    base = dict(world=8, sp_max=8, hq=32, hkv=4, head_dim=128)
    base.update(kw)
    return P.PlanParams(**base)


def _batch(rng, n, world=8, lo=7, hi=14):
    # lengths that are multiples of the world size, long-tail-ish
    return [world * int(2 ** rng.uniform(lo, hi)) for _ in range(n)]


def test_sp_tree_ranges_are_nested_and_aligned():
    W = 16
    K = 4
    for d in range(K + 1):
        seen = []
        for i in range(1 << d):
            R = P.node_ranks(W, d, i)
            assert len(R) == W >> d and R.start % len(R) == 0
            seen.extend(R)
            if d:
                parent = P.node_ranks(W, d - 1, i // 2)
                assert set(R) <= set(parent)
        assert sorted(seen) == list(range(W))


def _all_plans(prm, lengths):
    K = prm.world.bit_length() - 1
    nodes = [(d, i) for d in range(K + 1) for i in range(1 << d)]
    for choice in itertools.product(nodes, repeat=len(lengths)):
        ok = True
        for j, (d, _) in enumerate(choice):
            sp = prm.world >> d
            if sp > prm.sp_max or lengths[j] % sp or prm.hq % sp or (prm.hkv % sp and sp % prm.hkv):
                ok = False
            for jj, (dd, _) in enumerate(choice):
                if prm.monotone and lengths[jj] > lengths[j] and (prm.world >> dd) < sp:
                    ok = False
        if ok:
            yield choice


@pytest.mark.parametrize("seed", range(6))
def test_full_beam_equals_exhaustive_search(seed):
    rng = random.Random(seed)
    W = 4
    n = 3 + seed % 2
    lengths = [4 * rng.randint(1, 400) for _ in range(n)]
    mean = sum(lengths) / W
    prm = _prm(world=W, sp_max=W, hq=8, hkv=2, head_dim=64, prefix=n, beam=10 ** 6,
               token_budget=1.3 * mean if seed % 3 == 0 else float("inf"),
               dense_fwd_per_token=1e-7, dense_bwd_per_token=2e-7, monotone=bool(seed % 2))
    best = None
    for choice in _all_plans(prm, lengths):
        assign = list(enumerate(choice))
        C, T, _, _ = P.gpu_costs(prm, lengths, assign)
        if max(T) <= prm.token_budget and (best is None or max(C) < best):
            best = max(C)
    got = P.plan(prm, lengths)
    if best is None:
        assert got is None
    else:
        assert got is not None and max(got.cost) == best


def _lpt(costs, W):
    """Longest-processing-time list scheduling: jobs in the given order, each
    to the machine of least load (lowest index among ties)."""
    load = [0.0] * W
    where = []
    for c in costs:
        m = min(range(W), key=lambda i: (load[i], i))
        where.append(m)
        load[m] += c
    return where, load


@pytest.mark.parametrize("seed", range(4))
def test_tail_is_lpt_on_leaves(seed):
    rng = random.Random(100 + seed)
    W = 8
    lengths = _batch(rng, 40, W)
    prm = _prm(prefix=0, a2a_latency=0.0, link_bytes=math.inf)
    got = P.plan(prm, lengths)
    order = sorted(range(len(lengths)), key=lambda j: -lengths[j])
    D, hq = prm.head_dim, prm.hq
    cost = [4 * D * hq * (L * (L + 1) // 2) / prm.attn_fwd_flops + 10 * D * hq * (L * (L + 1) // 2) / prm.attn_bwd_flops
            for L in lengths]
    where, load = _lpt([cost[j] for j in order], W)
    K = W.bit_length() - 1
    for j, m in zip(order, where):
        assert got.node[j] == (K, m)
    assert max(got.cost) == pytest.approx(max(load), rel=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_tokens_and_attention_work_are_conserved(seed):
    rng = random.Random(200 + seed)
    lengths = _batch(rng, 30)
    prm = _prm(a2a_latency=0.0, link_bytes=math.inf, prefix=8, beam=4)
    got = P.plan(prm, lengths)
    assert sum(got.tokens) == sum(lengths)
    D, hq = prm.head_dim, prm.hq
    total = sum(4 * D * hq * (L * (L + 1) // 2) / prm.attn_fwd_flops + 10 * D * hq * (L * (L + 1) // 2) / prm.attn_bwd_flops
                for L in lengths)
    assert sum(got.cost) == pytest.approx(total, rel=1e-12)


def test_hand_worked_communication_cost():
    # One sample of 1024 tokens at the root of 8 GPUs, Hq 32, Hkv 4, D 128,
    # bf16; attention compute and dense work free; links of 1e9 B/s, 7 per
    # GPU; 1e-5 s per all-to-all.  Each GPU holds 128 tokens.
    #   forward prologue: Q 32 heads + K, V 8 heads each (replicated to the 8
    #     ranks) = 48 heads * 128 tokens * 128 * 2 B = 1,572,864 B, of which
    #     7/8 leave over 7 links: 1,376,256 B / 7e9 B/s = 1.966080e-4 s
    #   forward epilogue: O, 32 heads: 1,048,576 B * 7/8 / 7e9 = 1.31072e-4 s
    #   backward prologue dO: 1.31072e-4 s; backward epilogue dQ, dK, dV:
    #     1.966080e-4 s
    #   plus 4 latencies of 1e-5 s: 6.5536e-4 + 4e-5 = 6.9536e-4 s per GPU.
    prm = _prm(attn_fwd_flops=math.inf, attn_bwd_flops=math.inf, link_bytes=1e9, links=7, a2a_latency=1e-5)
    C, T, cf, cb = P.gpu_costs(prm, [1024], [(0, (0, 0))])
    assert T == [128.0] * 8
    for p in range(8):
        assert cf[p] == pytest.approx(1.966080e-4 + 1.31072e-4 + 2e-5, rel=1e-12)
        assert cb[p] == pytest.approx(1.31072e-4 + 1.966080e-4 + 2e-5, rel=1e-12)
        assert C[p] == pytest.approx(6.9536e-4, rel=1e-12)
    # at degree 2 (node (2, 1) = GPUs 2, 3): K, V keep their 4 heads; 512
    # tokens per GPU; 1/2 leaves over 1 link.
    #   fwd prologue (32 + 8) * 512 * 256 B = 5,242,880 B -> 2,621,440 B / 1e9
    C, T, cf, cb = P.gpu_costs(prm, [1024], [(0, (2, 1))])
    assert T == [0, 0, 512, 512, 0, 0, 0, 0]
    assert cf[2] == pytest.approx(2.62144e-3 + 2.097152e-3 + 2e-5, rel=1e-12)
    assert cf[0] == 0.0


@pytest.mark.parametrize("seed", range(3))
def test_plans_are_monotone_and_within_budget(seed):
    rng = random.Random(300 + seed)
    lengths = _batch(rng, 60)
    prm = _prm(token_budget=1.5 * sum(lengths) / 8, prefix=12, beam=6,
               dense_fwd_per_token=2e-6, dense_bwd_per_token=4e-6)
    got = P.plan(prm, lengths)
    assert got is not None
    sp = [8 >> d for d, _ in got.node]
    for a in range(len(lengths)):
        for b in range(len(lengths)):
            if lengths[a] > lengths[b]:
                assert sp[a] >= sp[b]
    order = sorted(range(len(lengths)), key=lambda j: -lengths[j])
    prefix_tok = P.tok_loads(prm, lengths, [(j, got.node[j]) for j in order[:12]])
    assert max(prefix_tok) <= prm.token_budget


def test_worklist_covers_every_head_once():
    rng = random.Random(7)
    lengths = _batch(rng, 25)
    prm = _prm(prefix=10, beam=4, dense_fwd_per_token=1e-6)
    got = P.plan(prm, lengths)
    seen = {}
    for p in range(8):
        items = P.worklist_for_gpu(prm, lengths, got.node, p)
        sps = [it[2] for it in items]
        assert sps == sorted(sps, reverse=True)          # root first
        for j, L, sp, (qlo, qhi), (klo, khi) in items:
            assert qhi - qlo == prm.hq // sp
            for h in range(qlo, qhi):
                seen[(j, h)] = seen.get((j, h), 0) + 1
                assert klo <= h * prm.hkv // prm.hq < khi  # the GQA map stays local
    assert seen == {(j, h): 1 for j in range(len(lengths)) for h in range(prm.hq)}
