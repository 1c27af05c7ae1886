"""The host schedule step (work list -> attention units, in launch order),
through nsp_attn_schedule, on the CPU.

What pins it, and which mistake each check catches:
  * coverage   -- every (item, tile, head) unit appears exactly once, with
                  the KV head (forward) or query-head range (dK/dV) the GQA
                  map gives: a dropped or duplicated tile, a ragged last tile
                  missed, a masked or empty item scheduled, a wrong head map;
                  compared with units enumerated by brute force;
  * order      -- the launch order is the documented one, rebuilt here from
                  its description.  Forward / dQ: units generated item by
                  item, sorted longest work first (stable), and, when the
                  longest item's K/V head slices exceed 4 MiB, in each full
                  chunk of 8 x 32 units XCD x (slots b % 8 == x) takes one
                  run of 32 consecutive sorted units, run x or 7 - x in
                  alternate chunks.  dK/dV: key-tile pairs (n, nk-1-n) in
                  gangs of 32, the first units sweeping down from the item
                  end, the partners up from their diagonals, longest first;
                  middle tiles in gangs of their own; gangs by decreasing
                  duration, each to the XCD queue with the least work, the
                  queues one after another (nsp_attn_kv_queues); the
                  largest item's shortest tiles unpaired by the end-game
                  rule, and more of them where a model of the persistent
                  pass ends over 8% past an even split.  A wrong cost, an
                  unstable sort, a wrong slot map, pairing, direction,
                  queue assignment or balance search fails it (the
                  item-masked work lists of phase streaming included);
  * balance    -- on the long-tail and max-context shares, the persistent
                  passes' dispatch of that order (each compute unit takes the
                  next slot of its XCD's queue when it goes idle, then the
                  other XCDs' queues; time proportional to the unit's work)
                  finishes within 1% of a perfect split of the total work,
                  and the dK/dV pass of each SP level's item-masked call
                  within 8%.
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


def _kv_heads(wl, j, g):
    q0, q1, k0, _ = _heads(wl, j)
    mine = [i for i in range(q1 - q0) if (q0 + i) * wl.hkv_total // wl.hq_total - k0 == g]
    i0, i1 = (mine[0], mine[-1] + 1) if mine else (0, 0)
    assert mine == list(range(i0, i1))
    return i0 | (i1 << 16)


KV_DESC = 1 << 30


def kv_units_brute(wl):
    """(item, key tile, heads, KV head) of every dK/dV unit, direction flag
    left out."""
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
    return max(1, i1 - i0) * (-(-L // KV_BM) - (u[1] & (KV_DESC - 1)) * KV_BN // KV_BM)


def _item_gangs(wl, j, K):
    """The gangs of item j (duration, total work, units), K tiles at each
    end of the key range left unpaired."""
    L = int(wl.lengths[j])
    nk = -(-L // KV_BN)
    K = min(K, nk // 2)
    _, _, k0, k1 = _heads(wl, j)
    pairs, mids, leads, tails = [], [], [], []
    for g in range(k1 - k0):
        hz = _kv_heads(wl, j, g)
        leads += [(g, n, hz) for n in range(K)]
        pairs += [(g, n, hz) for n in range(K, nk // 2)]
        tails += [(g, n, hz) for n in range(nk - K, nk)]
        if nk % 2:
            mids.append((g, nk // 2, hz))
    cost = lambda n, hz: kv_cost(wl, (j, n, hz, 0))
    gangs = []
    for p0 in range(0, len(pairs), G):
        ps = pairs[p0:p0 + G]
        units = [(j, n | KV_DESC, hz, g) for g, n, hz in ps]
        units += [(j, nk - 1 - n, hz, g) for g, n, hz in sorted(ps, key=lambda t: -t[1])]
        w = [cost(n, hz) + cost(nk - 1 - n, hz) for _, n, hz in ps]
        gangs.append((max(w), sum(w), units))
    for p0 in range(0, len(leads), G):
        ls = leads[p0:p0 + G]
        w = [cost(n, hz) for _, n, hz in ls]
        gangs.append((max(w), sum(w), [(j, n | KV_DESC, hz, g) for g, n, hz in ls]))
    for g, n, hz in tails:
        gangs.append((cost(n, hz), cost(n, hz), [(j, n, hz, g)]))
    for p0 in range(0, len(mids), G):
        ms = mids[p0:p0 + G]
        w = [cost(n, hz) for _, n, hz in ms]
        gangs.append((max(w), sum(w), [(j, n, hz, g) for g, n, hz in ms]))
    return gangs


def _queue_order(items):
    """Gangs by decreasing duration (stable), each to the XCD queue with the
    least work so far (lowest index on ties): the queues, as gang lists."""
    gangs = [g for _, gs in items for g in gs]
    gangs.sort(key=lambda t: -t[0])                   # stable
    queues, load = [[] for _ in range(NXCD)], [0] * NXCD
    for g in gangs:
        x = int(np.argmin(load))                      # lowest index on ties
        load[x] += g[1]
        queues[x].append(g)
    return queues


def _layout(items):
    queues = _queue_order(items)
    units = [u for q in queues for g in q for u in g[2]]
    off = np.cumsum([0] + [sum(len(g[2]) for g in q) for q in queues]).astype(np.int32)
    return units, off


def _model(wl, items):
    units, off = _layout(items)
    return persistent_makespan([kv_cost(wl, u) for u in units], off)


def kv_queues(wl):
    """The documented dK/dV queue layout: (units with direction flags, queue
    offsets)."""
    items = [(j, _item_gangs(wl, j, 0)) for j in range(len(wl.lengths)) if _active(wl, j)]
    if not items:
        return _layout(items)
    total = sum(w for _, gs in items for _, w, _ in gs)
    small = sum(w for _, gs in items for d, w, _ in gs if d <= 0.10 * total / 256)
    work = [sum(w for _, w, _ in gs) for _, gs in items]
    big = int(np.argmax(work))                        # the first on ties
    j = items[big][0]
    L = int(wl.lengths[j])
    nk, nqt = -(-L // KV_BN), -(-L // KV_BM)
    q0, q1, k0, k1 = _heads(wl, j)
    hkv, half = k1 - k0, nk // 2
    K = 0
    if small < 0.01 * total:                          # end game: no short gangs at all
        h = max(1, (q1 - q0) // max(1, hkv))
        got = 0.0
        while K < half and got < 0.02 * total:
            K += 1
            got += hkv * h * (nqt - (nk - K) * KV_BN // KV_BM)
        while K < half and (K * hkv) % G:
            K += 1
        items[big] = (j, _item_gangs(wl, j, K))
    best = _model(wl, items)
    if best > 1.08 * (total / 256) and K < half:     # balance: search K in whole gangs
        unit = 1
        while (unit * hkv) % G:
            unit += 1
        stride = unit
        while (half - K + stride - 1) // stride > 64:
            stride += unit
        best_k, k = K, K + stride
        while True:
            kc = min(k, half)
            items[big] = (j, _item_gangs(wl, j, kc))
            m = _model(wl, items)
            if m < best:
                best, best_k = m, kc
            if kc == half:
                break
            k += stride
        items[big] = (j, _item_gangs(wl, j, best_k))
    return _layout(items)


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
    for name in ("nested_2level", "longtail_4level"):   # the item-masked calls of phase streaming
        wl = make_config(name).wl
        for sp in sorted(set(int(x) for x in wl.sp)):
            yield f"{name}_sp{sp}", wl.select((np.asarray(wl.sp) == sp).astype(np.uint8))
    for seed in range(12):
        yield f"random{seed}", random_worklist(seed)


WLS = dict(_worklists())


@pytest.mark.parametrize("name", list(WLS))
def test_units_cover_every_tile_once(name):
    wl = WLS[name]
    for which, brute in ((nsp.NSP_SCHED_FWD, fwd_units_brute), (nsp.NSP_SCHED_KV, kv_units_brute)):
        got = [tuple(int(x) for x in r) for r in nsp.nsp_attn_schedule(wl, which)]
        if which == nsp.NSP_SCHED_KV:
            # the direction flag: down from the item end exactly for the first
            # half of an item's key tiles (paired or not)
            for j, y, _, _ in got:
                n, nk = y & (KV_DESC - 1), -(-int(wl.lengths[j]) // KV_BN)
                assert bool(y & KV_DESC) == (n < nk // 2), (name, j, n)
            got = [(j, y & (KV_DESC - 1), z, g) for j, y, z, g in got]
        want = brute(wl)
        assert len(got) == len(set(got)), f"{name}: a unit is scheduled twice"
        assert sorted(got) == sorted(want), f"{name}: schedule {which} does not cover the tiles"


@pytest.mark.parametrize("name", list(WLS))
def test_launch_order_is_the_documented_one(name):
    wl = WLS[name]
    got = [tuple(int(x) for x in r) for r in nsp.nsp_attn_schedule(wl, nsp.NSP_SCHED_FWD)]
    want = launch_order(wl, fwd_units_brute(wl), lambda u: fwd_cost(wl, u))
    assert got == want, f"{name}: forward schedule is not in launch order"
    got = [tuple(int(x) for x in r) for r in nsp.nsp_attn_schedule(wl, nsp.NSP_SCHED_KV)]
    want, off = kv_queues(wl)
    assert got == want, f"{name}: dK/dV schedule is not the documented gang layout"
    assert np.array_equal(nsp.nsp_attn_kv_queues(wl), off), f"{name}: dK/dV queue offsets"


def persistent_makespan(costs, off):
    """Persistent dispatch: every compute unit takes the next slot of its XCD's
    queue when it goes idle, then the other XCDs' queues in turn."""
    import heapq
    heads = [int(off[x]) for x in range(NXCD)]
    free = [(0.0, x, c) for x in range(NXCD) for c in range(CUS_PER_XCD)]
    heapq.heapify(free)
    end = 0.0
    while free:
        t, x, c = heapq.heappop(free)
        slot = -1
        for k in range(NXCD):
            y = (x + k) % NXCD
            if heads[y] < off[y + 1]:
                slot = heads[y]
                heads[y] += 1
                break
        if slot < 0:
            end = max(end, t)
            continue
        heapq.heappush(free, (t + costs[slot], x, c))
    return end


@pytest.mark.parametrize("name", ["longtail_4level", "maxctx_relayout"])
def test_dispatch_balance(name):
    wl = WLS[name]
    units = [tuple(int(x) for x in r) for r in nsp.nsp_attn_schedule(wl, nsp.NSP_SCHED_FWD)]
    costs = [fwd_cost(wl, u) for u in units]
    order = [b for x in range(NXCD) for b in range(x, len(costs), NXCD)]   # slot b in XCD b % 8's queue
    off = np.cumsum([0] + [len(range(x, len(costs), NXCD)) for x in range(NXCD)])
    ideal = sum(costs) / (NXCD * CUS_PER_XCD)
    assert persistent_makespan([costs[b] for b in order], off) <= 1.01 * ideal, (name, "forward")
    units = [tuple(int(x) for x in r) for r in nsp.nsp_attn_schedule(wl, nsp.NSP_SCHED_KV)]
    costs = [kv_cost(wl, u) for u in units]
    ideal = sum(costs) / (NXCD * CUS_PER_XCD)
    assert persistent_makespan(costs, nsp.nsp_attn_kv_queues(wl)) <= 1.01 * ideal, (name, "dK/dV")


@pytest.mark.parametrize("sp", [8, 4, 2, 1])
def test_node_balance(sp):
    """The item-masked calls of phase streaming (one SP level of the
    long-tail share each, single items at sp 8, 4 and 2): the modelled dK/dV
    pass ends within 8% of a perfect split (the sp = 4 node's one item of 454
    key-tile pairs on 256 compute units ended 13% past it with all tiles
    paired)."""
    wl = WLS[f"longtail_4level_sp{sp}"]
    units = [tuple(int(x) for x in r) for r in nsp.nsp_attn_schedule(wl, nsp.NSP_SCHED_KV)]
    costs = [kv_cost(wl, u) for u in units]
    assert persistent_makespan(costs, nsp.nsp_attn_kv_queues(wl)) <= 1.08 * sum(costs) / 256, sp


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
