"""Properties of the HIP path that hold exactly (bitwise) or by closed form.

  * run-to-run determinism (the default backward has no atomics);
  * segment isolation: perturbing one packed item leaves every other item's
    outputs bitwise unchanged (Background, Sequence Packing);
  * causality: perturbing token t leaves rows < t of O and LSE bitwise
    unchanged;
  * Ulysses equivalence: the head shards of an item at degree sp, run one
    rank after the other on this GPU, reproduce the sp=1 result bitwise for
    O, LSE and dQ, and the replica-summed dK/dV within tolerance
    (Background, Sequence Parallelism);
  * item order: permuting the work list permutes the outputs bitwise;
  * closed forms: Q = 0 gives running means of V and LSE = ln(t+1);
    a length-1 item gives O = V; V = 1 gives O = 1; sum_s dK = 0 and
    sum_s dV = sum over the group of sum_t dO.
"""
import numpy as np
import pytest

from oracle import attention as OA
from oracle import ulysses as OU
from paper_2609_22755_amd import nsp
from paper_2609_22755_amd.workloads import draw_attention_inputs, small_worklist

from gpu_util import rel_l2, require_gpu, run_attention, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def bits(t):
    import torch
    if t.dtype == torch.bfloat16:
        return nsp.bf16_to_numpy_bits(t)
    return t.detach().cpu().numpy().view(np.uint32)


def all_bits(buf):
    return {k: bits(buf[k]) for k in ("o", "lse", "dq", "dk", "dv")}


SCALE = 1.0 / np.sqrt(128.0)


def test_bitwise_determinism():
    wl = small_worklist([700, 129, 1, 300], 32, 4, 128, sp=[2, 1, 1, 8], rank=[1, 0, 0, 6])
    inp = draw_attention_inputs(wl, 21)
    a = all_bits(run_attention(wl, *inp, SCALE))
    b = all_bits(run_attention(wl, *inp, SCALE))
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def _item_slices(wl):
    D = wl.head_dim
    q = np.concatenate([[0], np.cumsum(wl.lengths.astype(np.int64) * wl.hq * D)])
    kv = np.concatenate([[0], np.cumsum(wl.lengths.astype(np.int64) * wl.hkv * D)])
    ls = np.concatenate([[0], np.cumsum(wl.lengths.astype(np.int64) * wl.hq)])
    return q, kv, ls


def test_segment_isolation():
    wl = small_worklist([300, 257, 190], 8, 2, 128)
    qb, kb, vb, db = draw_attention_inputs(wl, 22)
    base = all_bits(run_attention(wl, qb, kb, vb, db, SCALE))
    qs, ks, ls = _item_slices(wl)
    q2, k2, v2, d2 = (x.copy() for x in (qb, kb, vb, db))
    rng = np.random.default_rng(5)
    for arr, sl in ((q2, qs), (k2, ks), (v2, ks), (d2, qs)):
        arr[sl[1]:sl[2]] = rng.integers(0x3000, 0x4000, sl[2] - sl[1]).astype(np.uint16)
    pert = all_bits(run_attention(wl, q2, k2, v2, d2, SCALE))
    for name, sl in (("o", qs), ("dq", qs), ("lse", ls), ("dk", ks), ("dv", ks)):
        for j in (0, 2):
            assert np.array_equal(base[name][sl[j]:sl[j + 1]], pert[name][sl[j]:sl[j + 1]]), (name, j)
        assert not np.array_equal(base[name][sl[1]:sl[2]], pert[name][sl[1]:sl[2]]), name


def test_causality_prefix_rows_unchanged():
    L, H, D = 600, 4, 128
    wl = small_worklist([L], H, 1, D)
    qb, kb, vb, db = draw_attention_inputs(wl, 23)
    base = all_bits(run_attention(wl, qb, kb, vb, db, SCALE, bwd=False))
    for t in (0, 127, 128, 333):
        q2, k2, v2 = qb.copy(), kb.copy(), vb.copy()
        q2[t * H * D:(t + 1) * H * D] ^= 0x0101
        k2[t * D:(t + 1) * D] ^= 0x0101
        v2[t * D:(t + 1) * D] ^= 0x0101
        pert = all_bits(run_attention(wl, q2, k2, v2, db, SCALE, bwd=False))
        assert np.array_equal(base["o"][:t * H * D], pert["o"][:t * H * D])
        lb, lp = base["lse"].reshape(H, L), pert["lse"].reshape(H, L)
        assert np.array_equal(lb[:, :t], lp[:, :t])
        assert not np.array_equal(base["o"][t * H * D:], pert["o"][t * H * D:])


def test_ulysses_rank_emulation_matches_sp1():
    import torch
    L, Hq, Hkv, D = 520, 32, 4, 128
    full = small_worklist([L], Hq, Hkv, D)
    qb, kb, vb, db = draw_attention_inputs(full, 24)
    ref = run_attention(full, qb, kb, vb, db, SCALE, g_dtype=torch.float32)
    rb = {k: bits(ref[k]) for k in ("o", "lse", "dq")}
    Q, K, V, G = (x.reshape(L, -1, D) for x in (qb, kb, vb, db))
    for sp in (2, 4, 8):
        dk_sum = np.zeros((L, Hkv, D))
        dv_sum = np.zeros((L, Hkv, D))
        for r in range(sp):
            wl = small_worklist([L], Hq, Hkv, D, sp=[sp], rank=[r])
            ql, qh = wl.q_heads[0]
            kl, kh = wl.kv_heads[0]
            sub = [np.ascontiguousarray(X[:, a:b]).reshape(-1) for X, a, b in
                   ((Q, ql, qh), (K, kl, kh), (V, kl, kh), (G, ql, qh))]
            out = run_attention(wl, *sub, SCALE, g_dtype=torch.float32)
            assert np.array_equal(bits(out["o"]), rb["o"].reshape(L, Hq, D)[:, ql:qh].reshape(-1))
            assert np.array_equal(bits(out["dq"]), rb["dq"].reshape(L, Hq, D)[:, ql:qh].reshape(-1))
            assert np.array_equal(bits(out["lse"]), rb["lse"].reshape(Hq, L)[ql:qh].reshape(-1))
            dk_sum[:, kl:kh] += to_np(out["dk"]).reshape(L, kh - kl, D)
            dv_sum[:, kl:kh] += to_np(out["dv"]).reshape(L, kh - kl, D)
        assert rel_l2(dk_sum.reshape(-1), to_np(ref["dk"])) < 1e-5
        assert rel_l2(dv_sum.reshape(-1), to_np(ref["dv"])) < 1e-5


def test_item_order_permutation():
    lens = [300, 64, 1, 513, 129]
    wl = small_worklist(lens, 8, 2, 64)
    qb, kb, vb, db = draw_attention_inputs(wl, 25)
    base = all_bits(run_attention(wl, qb, kb, vb, db, 0.125))
    qs, ks, ls = _item_slices(wl)
    perm = [3, 0, 4, 2, 1]
    wp = small_worklist([lens[p] for p in perm], 8, 2, 64)
    cat = lambda x, sl: np.concatenate([x[sl[p]:sl[p + 1]] for p in perm])
    out = all_bits(run_attention(wp, cat(qb, qs), cat(kb, ks), cat(vb, ks), cat(db, qs), 0.125))
    for name, sl in (("o", qs), ("dq", qs), ("lse", ls), ("dk", ks), ("dv", ks)):
        assert np.array_equal(out[name], cat(base[name], sl)), name


def test_closed_forms():
    import torch
    L, D = 300, 128
    wl = small_worklist([L, 1], 4, 1, D)
    qb, kb, vb, db = draw_attention_inputs(wl, 26)
    # Q = 0: uniform attention over the prefix
    q0 = np.zeros_like(qb)
    out = run_attention(wl, q0, kb, vb, db, SCALE, o_dtype=torch.float32, g_dtype=torch.float32)
    V = OA.bf16_to_f64(vb)
    o = to_np(out["o"])
    Va = V[:L * D].reshape(L, D)
    want = np.cumsum(Va, axis=0) / np.arange(1, L + 1)[:, None]
    assert np.max(np.abs(o[:L * 4 * D].reshape(L, 4, D) - want[:, None, :])) < 1e-5
    lse = to_np(out["lse"])[:4 * L].reshape(4, L)
    assert np.max(np.abs(lse - np.log(np.arange(1, L + 1))[None, :])) < 1e-5
    # a length-1 item: O = V exactly (float32 store)
    o1 = o[L * 4 * D:].reshape(4, D)
    assert np.array_equal(o1, np.repeat(V[L * D:].reshape(1, D), 4, axis=0))
    # V = 1: every O row is 1 up to the bf16 rounding of P
    v1 = np.full_like(vb, 0x3F80)
    out = run_attention(wl, qb, kb, v1, db, SCALE, o_dtype=torch.float32, bwd=False)
    assert np.max(np.abs(to_np(out["o"]) - 1.0)) < 4e-3


def test_gradient_invariants():
    import torch
    L, Hq, Hkv, D = 1000, 8, 2, 128
    wl = small_worklist([L], Hq, Hkv, D)
    qb, kb, vb, db = draw_attention_inputs(wl, 27)
    out = run_attention(wl, qb, kb, vb, db, SCALE, g_dtype=torch.float32)
    dk = to_np(out["dk"]).reshape(L, Hkv, D)
    dv = to_np(out["dv"]).reshape(L, Hkv, D)
    dO = OA.bf16_to_f64(db).reshape(L, Hkv, Hq // Hkv, D)
    # sum over keys of dK vanishes (softmax invariance to a common key shift):
    # rounding noise leaves |sum| far below the L1 mass; a dropped or wrong
    # term leaves it of the same order
    assert np.max(np.abs(dk.sum(axis=0)) / np.abs(dk).sum(axis=0)) < 0.02
    # sum over keys of dV equals the summed upstream gradient of the group
    want = dO.sum(axis=(0, 2))
    assert np.max(np.abs(dv.sum(axis=0) - want) / np.abs(dO).sum(axis=(0, 2))) < 0.02


def test_empty_and_unit_items_interleaved():
    wl = small_worklist([0, 1, 0, 65, 0], 8, 2, 128)
    qb, kb, vb, db = draw_attention_inputs(wl, 28)
    out = run_attention(wl, qb, kb, vb, db, SCALE)
    from gpu_util import oracle_full
    ref = oracle_full(wl, qb, kb, vb, db, SCALE)
    assert rel_l2(to_np(out["o"]), ref["o"]) < 5e-3
    for g in ("dq", "dk", "dv"):
        r = ref[g]
        if np.linalg.norm(r) > 0:
            assert rel_l2(to_np(out[g]), r) < 1e-2


def test_persistent_passes_on_concurrent_streams():
    """Two calls at once on two new streams (each with its own buffers and
    workspace) while the persistent passes run -- more units than compute
    units in all three -- reproduce the default-stream results bit for bit:
    each stream takes its forward counters from its own block, each backward
    its queue heads from its own workspace."""
    import torch
    wl = small_worklist([256] * 80, 32, 4, 128)
    inp = draw_attention_inputs(wl, 31)
    ref = all_bits(run_attention(wl, *inp, SCALE))
    q, k, v, do = (nsp.to_device_bf16(x) for x in inp)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    bufs = [nsp.alloc_like_worklist(wl) for _ in streams]
    torch.cuda.synchronize()
    for rep in range(2):
        for s, b in zip(streams, bufs):
            nsp.nsp_varlen_attn_fwd(wl, q, k, v, b["o"], b["lse"], SCALE, stream=s)
            nsp.nsp_varlen_attn_bwd(wl, q, k, v, b["o"], do, b["lse"], b["dq"], b["dk"], b["dv"], b["ws"], SCALE,
                                    stream=s)
        torch.cuda.synchronize()
        for b in bufs:
            got = all_bits(b)
            for key in ref:
                assert np.array_equal(got[key], ref[key]), (rep, key)
