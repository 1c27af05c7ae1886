"""Pins of the tree-level recomputation plan oracle (oracle/recompute.py).

Design, NSP Executor, Tree-Level Recomputation fixes the procedure: walk the
SP tree from the root toward the leaves accumulating saved-slice bytes, SAVE
what the budget admits, split the node where the cut falls by sample (keeping
the costlier samples), RECOMPUTE every lower level.  Pinned by a plan worked
by hand (tests/golden/recompute_plan_small.txt) and by properties any plan of
that shape must have, on random work lists:
  * feasibility: the saved bytes are the sum of the SAVE slices, <= budget;
  * root first: levels above the cut are SAVE whole, levels below RECOMPUTE;
  * the cut node is split greedily: an unsaved item of the cut node would
    not have fitted when it was considered (longest first);
  * budget >= everything saves everything; a zero budget saves nothing but
    empty items.
A walk from the leaves up, a shortest-first split or a slice size without the
LSE fails the hand-worked plan.
"""
import numpy as np
import pytest

from conftest import load_golden
from oracle import recompute as R


def golden():
    g = load_golden("recompute_plan_small.txt")
    ints = {k: [int(x) for x in v] for k, v in g.items()}
    return ints


def test_hand_worked_plan():
    g = golden()
    for b, budget in enumerate(g["budgets"]):
        save, used = R.recompute_plan(g["lengths"], g["sp"], g["hq"], 128, 2, budget)
        assert save == g[f"save_{b}"], (budget, save)
        assert used == g["saved"][b]


def test_slice_bytes_counts_o_and_lse():
    assert R.slice_bytes(10, 3, 128, 2) == 10 * 3 * (256 + 4)
    assert R.slice_bytes(10, 3, 64, 4) == 10 * 3 * (256 + 4)
    assert R.slice_bytes(0, 32, 128, 2) == 0


def random_case(rng):
    n = int(rng.integers(1, 12))
    sp = rng.choice([1, 2, 4, 8], size=n)
    L = (rng.integers(0, 5000, size=n) // sp) * sp
    hq = 32 // sp
    return L.tolist(), sp.tolist(), hq.tolist()


@pytest.mark.parametrize("seed", range(40))
def test_plan_properties(seed):
    rng = np.random.default_rng(seed)
    L, sp, hq = random_case(rng)
    D, ob = 128, 2
    size = [R.slice_bytes(L[j], hq[j], D, ob) for j in range(len(L))]
    total = sum(size)
    for budget in [0, total, total + 7] + [int(x) for x in rng.integers(0, total + 1, size=6)]:
        save, used = R.recompute_plan(L, sp, hq, D, ob, budget)
        assert used == sum(s for s, k in zip(size, save) if k) <= budget
        assert all(save[j] for j in range(len(L)) if size[j] == 0)
        levels = sorted(set(sp), reverse=True)
        full = [all(save[j] or size[j] == 0 for j in range(len(L)) if sp[j] == lv) for lv in levels]
        none = [not any(save[j] and size[j] > 0 for j in range(len(L)) if sp[j] == lv) for lv in levels]
        # root first: a prefix of whole levels, at most one split level, then nothing
        k = 0
        while k < len(levels) and full[k]:
            k += 1
        if k < len(levels):
            cut = levels[k]
            assert all(none[k + 1:]), "a level below the cut was saved"
            # greedy split, longest first: re-walk the cut node
            room = budget - sum(size[j] for j in range(len(L)) if sp[j] > cut)
            for j in sorted([j for j in range(len(L)) if sp[j] == cut], key=lambda j: (-L[j], j)):
                if save[j]:
                    room -= size[j]
                else:
                    assert size[j] > room
        if budget >= total:
            assert all(save)
        if budget == 0:
            assert used == 0
