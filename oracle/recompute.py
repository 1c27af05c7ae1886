"""Tree-level recomputation plan, written out step by step (plain Python).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py): never imported by the
product path.

Design, NSP Executor, Tree-Level Recomputation: the Executor walks the routed
SP tree from the root toward the leaves and adds up the bytes of the
attention-output slices it would keep for the backward; the levels admitted
within the activation-memory budget are marked SAVE, and once the budget is
reached the remaining lower levels are marked RECOMPUTE.  When the budget cut
falls inside a tree node, the node is split by sample and the subset with the
larger recomputation cost is saved.

Readings (the paper gives no formula):
  * One GPU's path through the tree has one node per level, and sp shrinks
    from the root down, so the items of a node are the items sharing one sp
    and "root first" is decreasing sp.
  * The slice kept per item is its attention output O (o_bytes per element)
    plus its float32 log-sum-exp: L * hq * (head_dim * o_bytes + 4) bytes.
  * Splitting the cut node: items in decreasing recomputation cost per saved
    byte -- the forward attention cost 4 * head_dim * hq * L (L + 1) / 2 per
    L * hq * (...) bytes grows with L, so longest first, ties by item index --
    each saved if it still fits.
  * Items of length 0 keep nothing and count as SAVE.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

__all__ = ["slice_bytes", "recompute_plan"]


def slice_bytes(L: int, hq: int, head_dim: int, o_bytes: int) -> int:
    """Bytes of the attention-output slice (O and LSE) one item keeps."""
    return L * hq * (head_dim * o_bytes + 4)


def recompute_plan(lengths: Sequence[int], sp: Sequence[int], hq: Sequence[int], head_dim: int,
                   o_bytes: int, budget: int) -> Tuple[List[int], int]:
    """SAVE (1) / RECOMPUTE (0) per item, and the bytes saved."""
    n = len(lengths)
    size = [slice_bytes(int(lengths[j]), int(hq[j]), head_dim, o_bytes) for j in range(n)]
    save = [0] * n
    used = 0
    for level in sorted(set(int(s) for s in sp), reverse=True):     # root first
        node = [j for j in range(n) if int(sp[j]) == level]
        node_size = sum(size[j] for j in node)
        if used + node_size <= budget:                               # the whole node fits
            for j in node:
                save[j] = 1
            used += node_size
            continue
        # the budget cut falls inside this node: split it by sample
        for j in sorted(node, key=lambda j: (-int(lengths[j]), j)):
            if used + size[j] <= budget:
                save[j] = 1
                used += size[j]
        break                                                        # lower levels recompute
    for j in range(n):
        if size[j] == 0:
            save[j] = 1
    return save, used
