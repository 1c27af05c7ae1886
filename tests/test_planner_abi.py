"""The native SP-tree planner (nsp_sp_tree_plan / nsp_sp_tree_worklist,
host-only) against the planner oracle: the same node for every sample, and
the same C_p, Tok_p and load bit for bit (every cost sum is an exact integer
on both sides and seconds come from one fixed expression), over seeded
batches and a grid of tree sizes, head layouts, budgets, beam settings and
cost coefficients; the per-GPU work lists against the oracle's; and the
documented errors.  No GPU is needed.
"""
import math

import numpy as np
import pytest

from oracle import planner as P
from paper_2609_22755_amd import nsp


def _params(**kw):
    """(binding params, oracle params) with the same values."""
    b = nsp.SpTreeParams(**kw)
    o = P.PlanParams(world=b.world, sp_max=b.sp_max, hq=b.hq_total, hkv=b.hkv_total, head_dim=b.head_dim,
                     elem_bytes=b.elem_bytes, attn_fwd_flops=b.attn_fwd_flops, attn_bwd_flops=b.attn_bwd_flops,
                     link_bytes=b.link_bytes, links=b.links, a2a_latency=b.a2a_latency,
                     dense_fwd_per_token=b.dense_fwd_per_token, dense_bwd_per_token=b.dense_bwd_per_token,
                     token_budget=b.token_budget, prefix=b.prefix, beam=b.beam, monotone=bool(b.monotone))
    return b, o


def _lengths(rng, n, world, sigma=1.3, median=2048):
    """Long-tail lengths (lognormal), rounded to multiples of the world size
    (so that every degree divides them), some not rounded to exercise
    divisibility, a few zeros."""
    L = np.exp(rng.normal(math.log(median), sigma, n)).astype(np.int64) + 1
    L = np.where(rng.random(n) < 0.8, (L // world + 1) * world, L)
    L[rng.random(n) < 0.05] = 0
    return L


CASES = [
    # world, sp_max, hq, hkv, n, budget factor, prefix, beam, monotone, dense, link
    (8, 8, 32, 4, 40, None, 16, 8, 1, (1e-6, 2e-6), 153e9),
    (8, 8, 32, 4, 40, 1.3, 16, 8, 1, (1e-6, 2e-6), 153e9),
    (8, 4, 32, 4, 30, 2.0, 8, 4, 1, (0.0, 0.0), 153e9),
    (8, 8, 32, 4, 30, None, 0, 1, 1, (1e-6, 2e-6), 153e9),
    (8, 8, 32, 8, 25, 1.5, 25, 3, 0, (5e-7, 1e-6), 50e9),
    (16, 16, 32, 4, 40, None, 12, 6, 1, (1e-6, 2e-6), 153e9),
    (16, 8, 16, 16, 35, 1.2, 10, 8, 0, (0.0, 3e-6), math.inf),
    (4, 4, 8, 1, 20, 1.1, 6, 5, 1, (2e-6, 2e-6), 100e9),
    (2, 2, 4, 2, 12, None, 12, 100, 0, (0.0, 0.0), 10e9),
    (1, 1, 32, 4, 10, None, 4, 2, 1, (1e-6, 1e-6), 153e9),
    (8, 8, 12, 6, 24, None, 12, 4, 1, (1e-6, 2e-6), 153e9),   # KV heads split by 2 only
]


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("seed", range(2))
def test_native_plan_matches_oracle(case, seed):
    W, spm, hq, hkv, n, bf, k, w, mono, (df, db), link = CASES[case]
    rng = np.random.default_rng(1000 * case + seed)
    L = _lengths(rng, n, W)
    budget = math.inf if bf is None else bf * max(1.0, L.sum() / W)
    b, o = _params(world=W, sp_max=spm, hq_total=hq, hkv_total=hkv, head_dim=128, token_budget=budget, prefix=k,
                   beam=w, monotone=mono, dense_fwd_per_token=df, dense_bwd_per_token=db, link_bytes=link)
    ref = P.plan(o, L.tolist())
    if ref is None:
        with pytest.raises(nsp.NspError) as e:
            nsp.nsp_sp_tree_plan(b, L)
        assert e.value.status == nsp.NSP_EINFEASIBLE
        return
    d, i, cost, tok, load = nsp.nsp_sp_tree_plan(b, L)
    assert list(zip(d.tolist(), i.tolist())) == ref.node
    assert cost.tolist() == ref.cost
    assert tok.tolist() == ref.tokens
    assert load == ref.load
    for p in range(W):
        wl, sample = nsp.nsp_sp_tree_worklist(b, L, d, i, p)
        items = P.worklist_for_gpu(o, L.tolist(), ref.node, p)
        assert sample.tolist() == [it[0] for it in items]
        assert wl.lengths.tolist() == [it[1] for it in items]
        assert wl.sp.tolist() == [it[2] for it in items]
        assert [tuple(x) for x in wl.q_heads.tolist()] == [it[3] for it in items]
        assert [tuple(x) for x in wl.kv_heads.tolist()] == [it[4] for it in items]
        nsp.nsp_recompute_plan(wl, 0)   # host-side validation of the work list (raises if invalid)


def test_infeasible_budget_is_reported():
    b, o = _params(world=4, sp_max=2, hq_total=8, hkv_total=2, head_dim=64, token_budget=100.0)
    L = np.array([1000, 10], dtype=np.int64)       # the long one holds >= 500 tokens on any GPU
    assert P.plan(o, L.tolist()) is None
    with pytest.raises(nsp.NspError) as e:
        nsp.nsp_sp_tree_plan(b, L)
    assert e.value.status == nsp.NSP_EINFEASIBLE


def test_empty_batch():
    b, _ = _params(world=8, sp_max=8, hq_total=32, hkv_total=4, head_dim=128)
    d, i, cost, tok, load = nsp.nsp_sp_tree_plan(b, np.zeros(0, dtype=np.int64))
    assert d.size == 0 and cost.tolist() == [0.0] * 8 and tok.tolist() == [0.0] * 8 and load == 0.0


@pytest.mark.parametrize("bad", [
    dict(world=6), dict(world=0), dict(sp_max=16), dict(sp_max=3), dict(hq_total=30), dict(hkv_total=0),
    dict(head_dim=0), dict(elem_bytes=0), dict(attn_fwd_flops=0.0), dict(link_bytes=-1.0), dict(links=0),
    dict(a2a_latency=-1e-6), dict(dense_bwd_per_token=math.inf), dict(token_budget=0.0), dict(prefix=-1),
    dict(beam=0), dict(monotone=2),
])
def test_plan_rejects_bad_parameters(bad):
    kw = dict(world=8, sp_max=8, hq_total=32, hkv_total=4, head_dim=128)
    kw.update(bad)
    b = nsp.SpTreeParams(**kw)
    with pytest.raises(nsp.NspError) as e:
        nsp.nsp_sp_tree_plan(b, np.array([64, 32], dtype=np.int64))
    assert e.value.status == nsp.NSP_EINVAL


def test_plan_rejects_bad_lengths():
    b = nsp.SpTreeParams(world=8, sp_max=8, hq_total=32, hkv_total=4, head_dim=128)
    for L in ([-1], [(1 << 31) + 1], [1 << 31] * 4):
        with pytest.raises(nsp.NspError) as e:
            nsp.nsp_sp_tree_plan(b, np.array(L, dtype=np.int64))
        assert e.value.status == nsp.NSP_EINVAL


def test_worklist_rejects_bad_nodes():
    b = nsp.SpTreeParams(world=8, sp_max=4, hq_total=32, hkv_total=4, head_dim=128)
    L = np.array([64, 30], dtype=np.int64)
    for d, i, gpu in (([0, 3], [0, 0], 0),      # degree 8 > sp_max
                      ([1, 4], [0, 0], 0),      # depth 4 outside a 3-level tree
                      ([1, 3], [2, 0], 0),      # index 2 at depth 1
                      ([3, 1], [0, 0], 0),      # 30 tokens cannot run at degree 4
                      ([1, 3], [0, 0], 8)):     # GPU 8 of 8
        with pytest.raises(nsp.NspError) as e:
            nsp.nsp_sp_tree_worklist(b, L, d, i, gpu)
        assert e.value.status == nsp.NSP_EINVAL
