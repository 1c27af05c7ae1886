"""The host schedule step (work list -> attention units, in launch order),
through nsp_attn_schedule, on the CPU.

What pins it, and which mistake each check catches:
  * coverage   -- every (item, tile, head) unit appears exactly once, with
                  the KV head (forward) or query-head range (dK/dV) the GQA
                  map gives: a dropped or duplicated tile, a ragged last tile
                  missed, a masked or empty item scheduled, a wrong head map;
                  compared with units enumerated by brute force;
  * order      -- the launch order is the documented one, rebuilt here from
                  its description: units generated item by item, sorted
                  longest work first (stable), and, when the longest item's
                  K/V head slices exceed 4 MiB, in each full chunk of 8 x 32
                  units XCD x (workgroup slots b % 8 == x) takes one run of
                  32 consecutive sorted units, run x or 7 - x in alternate
                  chunks; a wrong cost, an unstable sort, a wrong slot map or
                  a wrong grouping test fails it;
  * balance    -- on the long-tail and max-context shares, greedy dispatch
                  of that order (each XCD starts its slots in order on the
                  first of its 32 compute units to go idle, one workgroup per
                  unit, time proportional to the unit's work) finishes within
                  1% of a perfect split of the total work.
"""
import ctypes

import numpy as np
import pytest

from paper_2609_22755_amd import nsp
from paper_2609_22755_amd.workloads import make_config, make_worklist

FWD_BM, KV_BN, KV_BM = 256, 128, 64     # query rows per forward unit, keys per dK/dV unit, rows per dK/dV step
NXCD, G, CUS_PER_XCD = 8, 32, 32

CONFIGS = ["tiny", "short_sp1", "nested_2level", "longtail_4level", "maxctx_relayout"]


def _heads(wl, j):
    q0, q1 = (int(x) for x in wl.q_heads[j])
    k0, k1 = (int(x) for x in wl.kv_heads[j])
    return q0, q1, k0, k1


def _active(wl, j):
    return int(wl.lengths[j]) > 0 and (wl.item_mask is None or wl.item_mask[j] != 0)


def fwd_units_brute(wl):
    out = []
    for j in range(len(wl.lengths)):
        if not _active(wl, j):
            continue
        L = int(wl.lengths[j])
        q0, q1, k0, _ = _heads(wl, j)
        for m in range(-(-L // FWD_BM)):
            for i in range(q1 - q0):
                g = (q0 + i) * wl.hkv_total // wl.hq_total - k0
                out.append((j, m, i, g))
    return out


def fwd_cost(wl, u):
    return min(int(wl.lengths[u[0]]), FWD_BM * (u[1] + 1))


def kv_units_brute(wl):
    out = []
    for j in range(len(wl.lengths)):
        if not _active(wl, j):
            continue
        L = int(wl.lengths[j])
        q0, q1, k0, k1 = _heads(wl, j)
        for g in range(k1 - k0):
            mine = [i for i in range(q1 - q0) if (q0 + i) * wl.hkv_total // wl.hq_total - k0 == g]
            i0, i1 = (mine[0], mine[-1] + 1) if mine else (0, 0)
            assert mine == list(range(i0, i1))
            for n in range(-(-L // KV_BN)):
                out.append((j, n, i0 | (i1 << 16), g))
    return out


def kv_cost(wl, u):
    L = int(wl.lengths[u[0]])
    i0, i1 = u[2] & 0xFFFF, u[2] >> 16
    return max(1, i1 - i0) * (-(-L // KV_BM) - u[1] * KV_BN // KV_BM)


def launch_order(wl, units, cost):
    """The documented launch order, rebuilt from its description."""
    srt = sorted(units, key=lambda u: -cost(u))        # stable: generation order among equal work
    longest = max([int(wl.lengths[j]) for j in range(len(wl.lengths)) if _active(wl, j)], default=0)
    if 4 * longest * wl.head_dim <= 4 << 20:            # streams fit one XCD's L2: no XCD runs
        return srt
    out = list(srt)
    chunk = NXCD * G
    for c in range(len(srt) // chunk):
        for b in range(chunk):
            x, t = b % NXCD, b // NXCD
            run = x if c % 2 == 0 else NXCD - 1 - x
            out[c * chunk + b] = srt[c * chunk + run * G + t]
    return out


def random_worklist(seed):
    rng = np.random.default_rng(seed)
    hq, hkv = [(8, 2), (32, 4), (12, 6), (16, 16)][seed % 4]
    D = 64 if seed % 2 else 128
    n = int(rng.integers(1, 12))
    lengths, sps, ranks = [], [], []
    for _ in range(n):
        sp = int(rng.choice([s for s in (1, 2, 4, 8) if hq % s == 0 and (hkv % s == 0 or s % hkv == 0)]))
        lengths.append(sp * int(rng.choice([0, 1, 3, 37, 255, 256, 257, 700, 1500])))
        sps.append(sp)
        ranks.append(int(rng.integers(0, sp)))       # non-zero ranks: head ranges off 0
    wl = make_worklist(lengths, sps, hq, hkv, D, rank=ranks)
    if seed % 3 == 0:
        wl = wl.select(rng.integers(0, 2, size=n).astype(np.uint8))
    return wl


def _worklists():
    for name in CONFIGS:
        yield name, make_config(name).wl
    for seed in range(12):
        yield f"random{seed}", random_worklist(seed)


WLS = dict(_worklists())


@pytest.mark.parametrize("name", list(WLS))
def test_units_cover_every_tile_once(name):
    wl = WLS[name]
    for which, brute in ((nsp.NSP_SCHED_FWD, fwd_units_brute), (nsp.NSP_SCHED_KV, kv_units_brute)):
        got = [tuple(int(x) for x in r) for r in nsp.nsp_attn_schedule(wl, which)]
        want = brute(wl)
        assert len(got) == len(set(got)), f"{name}: a unit is scheduled twice"
        assert sorted(got) == sorted(want), f"{name}: schedule {which} does not cover the tiles"


@pytest.mark.parametrize("name", list(WLS))
def test_launch_order_is_longest_first_with_xcd_runs(name):
    wl = WLS[name]
    for which, brute, cost in ((nsp.NSP_SCHED_FWD, fwd_units_brute, lambda u: fwd_cost(wl, u)),
                               (nsp.NSP_SCHED_KV, kv_units_brute, lambda u: kv_cost(wl, u))):
        got = [tuple(int(x) for x in r) for r in nsp.nsp_attn_schedule(wl, which)]
        assert got == launch_order(wl, brute(wl), cost), f"{name}: schedule {which} is not in launch order"


def dispatch_makespan(costs):
    """Greedy dispatch: XCD x starts slots x, x + 8, ... in order, each on the
    first of its compute units to become idle."""
    end = 0.0
    for x in range(NXCD):
        cu = np.zeros(CUS_PER_XCD)
        for c in costs[x::NXCD]:
            k = int(np.argmin(cu))
            cu[k] += c
        end = max(end, float(cu.max()))
    return end


@pytest.mark.parametrize("name", ["longtail_4level", "maxctx_relayout"])
def test_dispatch_balance(name):
    wl = WLS[name]
    for which, cost in ((nsp.NSP_SCHED_FWD, fwd_cost), (nsp.NSP_SCHED_KV, kv_cost)):
        units = [tuple(int(x) for x in r) for r in nsp.nsp_attn_schedule(wl, which)]
        costs = [cost(wl, u) for u in units]
        ideal = sum(costs) / (NXCD * CUS_PER_XCD)
        assert dispatch_makespan(costs) <= 1.01 * ideal, (name, which)


def test_schedule_errors():
    lib = nsp.load_library()
    wl = WLS["tiny"]
    w = nsp._WL(wl)
    i32p = ctypes.POINTER(ctypes.c_int32)
    n = ctypes.c_int64(-1)
    assert lib.nsp_attn_schedule(w.ref, 2, ctypes.cast(None, i32p), 0, ctypes.byref(n)) == nsp.NSP_EINVAL
    assert lib.nsp_attn_schedule(w.ref, 0, ctypes.cast(None, i32p), 0, None) == nsp.NSP_EINVAL
    assert lib.nsp_attn_schedule(w.ref, 0, ctypes.cast(None, i32p), 0, ctypes.byref(n)) == nsp.NSP_OK
    total = n.value
    assert total == len(fwd_units_brute(wl))
    buf = np.zeros((total, 4), dtype=np.int32)
    n.value = -1
    st = lib.nsp_attn_schedule(w.ref, 0, buf.ctypes.data_as(i32p), total - 1, ctypes.byref(n))
    assert st == nsp.NSP_EINVAL and n.value == total
    assert lib.nsp_attn_schedule(w.ref, 0, ctypes.cast(None, i32p), 5, ctypes.byref(n)) == nsp.NSP_EINVAL
    # the work list is validated like every other entry point's
    bad = make_worklist([64, 32], [1, 1], 8, 2, 64)
    bad.kv_heads = bad.kv_heads.copy()
    bad.kv_heads[0] = (1, 2)                      # query heads 0..3 use KV head 0
    st = lib.nsp_attn_schedule(nsp._WL(bad).ref, 0, ctypes.cast(None, i32p), 0, ctypes.byref(n))
    assert st == nsp.NSP_EINVAL and "uses KV head" in lib.nsp_last_error().decode()
    bad = make_worklist([64, 32], [1, 1], 8, 2, 64)
    bad.head_dim = 96
    st = lib.nsp_attn_schedule(nsp._WL(bad).ref, 1, ctypes.cast(None, i32p), 0, ctypes.byref(n))
    assert st == nsp.NSP_EUNSUPPORTED
