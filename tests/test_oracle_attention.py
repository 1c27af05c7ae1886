"""Pins of the fp64 attention oracle against things other than itself.

Each check below would fail for a plausible mistake in the oracle:
  * brute force over the whole packed batch with an explicit block-diagonal
    causal mask built by loops: wrong mask (strict/non-strict), leakage
    across items, wrong GQA map, wrong scale, wrong item offsets;
  * torch fp64 SDPA + autograd (an independent library): every term of the
    backward, GQA group sums;
  * central finite differences: every term of the backward;
  * the hand-derived two-token example (tests/golden): signs, Delta, scale;
  * closed forms and invariants: row 0, Q = 0, L = 1, rows of P sum to one,
    sum_s dK = 0, sum_s dV = sum dO, causality under perturbation.
test_planted_mistakes_are_caught plants such mistakes in the oracle (on the
CPU) and checks that at least one pin fails for each.
"""
import numpy as np
import pytest
import torch

from oracle import attention as A
from paper_2609_22755_amd.workloads import draw_attention_inputs, small_worklist

from conftest import load_golden


def f64_inputs(wl, seed):
    return [A.bf16_to_f64(x) for x in draw_attention_inputs(wl, seed)]


def run_oracle(wl, q, k, v, do, scale):
    args = (wl.cu_seqlens, wl.q_heads, wl.kv_heads, wl.hq_total, wl.hkv_total, wl.head_dim, scale)
    o, lse = A.forward(q, k, v, *args)
    dq, dk, dv = A.backward(q, k, v, do, *args)
    return o, lse, dq, dk, dv


# ---------------------------------------------------------------- pins ----

def brute_force_packed(wl, q, k, v, scale):
    """Dense attention over the concatenated batch, mask built by loops.

    Requires every item to hold the same heads (so the batch is one dense
    [T, H, D] tensor).  Returns (o [T, hq, D], lse [T, hq]).
    """
    D, T = wl.head_dim, int(wl.lengths.sum())
    hq, hkv = int(wl.hq[0]), int(wl.hkv[0])
    item_of, pos_of = [], []
    for j, L in enumerate(wl.lengths):
        for p in range(int(L)):
            item_of.append(j)
            pos_of.append(p)
    mask = np.zeros((T, T), dtype=bool)
    for a in range(T):
        for b in range(T):
            mask[a, b] = item_of[a] == item_of[b] and pos_of[b] <= pos_of[a]
    Q, K, V = q.reshape(T, hq, D), k.reshape(T, hkv, D), v.reshape(T, hkv, D)
    o = np.zeros((T, hq, D))
    lse = np.zeros((T, hq))
    q_lo, kv_lo = int(wl.q_heads[0, 0]), int(wl.kv_heads[0, 0])
    for i in range(hq):
        g = ((q_lo + i) * wl.hkv_total) // wl.hq_total - kv_lo
        S = np.full((T, T), -np.inf)
        for a in range(T):
            for b in range(T):
                if mask[a, b]:
                    S[a, b] = scale * float(np.dot(Q[a, i], K[b, g]))
        m = S.max(axis=1, keepdims=True)
        e = np.exp(S - m)
        o[:, i] = (e / e.sum(axis=1, keepdims=True)) @ V[:, g]
        lse[:, i] = (m[:, 0] + np.log(e.sum(axis=1)))
    return o, lse


def lse_to_token_major(wl, lse):
    """[hq_j, L_j] per item -> [T, hq] (all items holding the same heads)."""
    out, off = [], 0
    hq = int(wl.hq[0])
    for L in wl.lengths:
        L = int(L)
        out.append(lse[off:off + hq * L].reshape(hq, L).T)
        off += hq * L
    return np.concatenate(out, axis=0)


def torch_reference(wl, q, k, v, do, scale):
    """Per item: torch fp64 SDPA (causal) with K/V repeated per group + autograd."""
    D = wl.head_dim
    res = {n: [] for n in ("o", "dq", "dk", "dv")}
    qo = ko = 0
    for j, L in enumerate(wl.lengths):
        L, hq, hkv = int(L), int(wl.hq[j]), int(wl.hkv[j])
        q_lo, kv_lo = int(wl.q_heads[j, 0]), int(wl.kv_heads[j, 0])
        Q = torch.tensor(q[qo:qo + L * hq * D].reshape(L, hq, D), requires_grad=True)
        K = torch.tensor(k[ko:ko + L * hkv * D].reshape(L, hkv, D), requires_grad=True)
        V = torch.tensor(v[ko:ko + L * hkv * D].reshape(L, hkv, D), requires_grad=True)
        dO = torch.tensor(do[qo:qo + L * hq * D].reshape(L, hq, D))
        idx = torch.tensor([((q_lo + i) * wl.hkv_total) // wl.hq_total - kv_lo for i in range(hq)])
        Kr, Vr = K[:, idx, :], V[:, idx, :]
        O = torch.nn.functional.scaled_dot_product_attention(
            Q.transpose(0, 1), Kr.transpose(0, 1), Vr.transpose(0, 1), is_causal=True, scale=scale
        ).transpose(0, 1)
        O.backward(dO)
        res["o"].append(O.detach().numpy().reshape(-1))
        res["dq"].append(Q.grad.numpy().reshape(-1))
        res["dk"].append(K.grad.numpy().reshape(-1))
        res["dv"].append(V.grad.numpy().reshape(-1))
        qo += L * hq * D
        ko += L * hkv * D
    return {n: np.concatenate(x) if x else np.zeros(0) for n, x in res.items()}


def rel(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


# --------------------------------------------------------------- tests ----

def check_bruteforce(seed=0):
    wl = small_worklist([1, 5, 9, 3], hq_total=4, hkv_total=2, head_dim=8)
    q, k, v, do = f64_inputs(wl, seed)
    scale = 0.37
    o, lse, *_ = run_oracle(wl, q, k, v, do, scale)
    ob, lb = brute_force_packed(wl, q, k, v, scale)
    return rel(o, ob.reshape(-1)) < 1e-13 and np.max(np.abs(lse_to_token_major(wl, lse) - lb)) < 1e-12


def check_torch(seed=1):
    # mixed degrees and ranks: GQA groups, replicated KV head, head offsets
    wl = small_worklist([17, 33, 8, 1, 40], hq_total=8, hkv_total=2, head_dim=16,
                        sp=[1, 2, 4, 1, 8], rank=[0, 1, 3, 0, 5])
    q, k, v, do = f64_inputs(wl, seed)
    scale = 0.25
    o, lse, dq, dk, dv = run_oracle(wl, q, k, v, do, scale)
    ref = torch_reference(wl, q, k, v, do, scale)
    return all(rel(x, ref[n]) < 1e-12 for x, n in ((o, "o"), (dq, "dq"), (dk, "dk"), (dv, "dv")))


def check_finite_differences(seed=2):
    wl = small_worklist([6, 4], hq_total=4, hkv_total=2, head_dim=4, sp=[1, 2], rank=[0, 1])
    q, k, v, do = f64_inputs(wl, seed)
    scale = 0.6
    args = (wl.cu_seqlens, wl.q_heads, wl.kv_heads, wl.hq_total, wl.hkv_total, wl.head_dim, scale)
    grads = dict(zip(("q", "k", "v"), A.backward(q, k, v, do, *args)))
    rng = np.random.default_rng(seed)
    eps = 1e-6

    def loss(q, k, v):
        return float(np.sum(A.forward(q, k, v, *args)[0] * do))

    ok = True
    for name in ("q", "k", "v"):
        base = {"q": q, "k": k, "v": v}
        for idx in rng.choice(base[name].size, size=12, replace=False):
            plus = {n: x.copy() for n, x in base.items()}
            minus = {n: x.copy() for n, x in base.items()}
            plus[name][idx] += eps
            minus[name][idx] -= eps
            fd = (loss(**plus) - loss(**minus)) / (2 * eps)
            ok &= abs(fd - grads[name][idx]) <= 1e-7 * max(1.0, abs(fd))
    return ok


def check_golden():
    g = load_golden("attention_two_token.txt")
    wl = small_worklist([2], hq_total=1, hkv_total=1, head_dim=2)
    q, k, v, do = (np.array(g[n]) for n in ("q", "k", "v", "do"))
    o, lse, dq, dk, dv = run_oracle(wl, q, k, v, do, 1.0)
    return all(np.allclose(x, g[n], rtol=0, atol=1e-14)
               for x, n in ((o, "o"), (lse, "lse"), (dq, "dq"), (dk, "dk"), (dv, "dv")))


def check_invariants(seed=3):
    wl = small_worklist([1, 23, 64, 7], hq_total=8, hkv_total=2, head_dim=16)
    q, k, v, do = f64_inputs(wl, seed)
    scale = 0.3
    o, lse, dq, dk, dv = run_oracle(wl, q, k, v, do, scale)
    D = wl.head_dim
    ok = True
    qo = ko = lo = 0
    for j, L in enumerate(wl.lengths):
        L, hq, hkv = int(L), int(wl.hq[j]), int(wl.hkv[j])
        Q = q[qo:qo + L * hq * D].reshape(L, hq, D)
        K = k[ko:ko + L * hkv * D].reshape(L, hkv, D)
        V = v[ko:ko + L * hkv * D].reshape(L, hkv, D)
        O = o[qo:qo + L * hq * D].reshape(L, hq, D)
        dO = do[qo:qo + L * hq * D].reshape(L, hq, D)
        dK = dk[ko:ko + L * hkv * D].reshape(L, hkv, D)
        dV = dv[ko:ko + L * hkv * D].reshape(L, hkv, D)
        LSE = lse[lo:lo + hq * L].reshape(hq, L)
        for i in range(hq):
            g = (i * wl.hkv_total) // wl.hq_total
            ok &= np.allclose(O[0, i], V[0, g], rtol=0, atol=1e-14)           # row 0
            ok &= abs(LSE[i, 0] - scale * np.dot(Q[0, i], K[0, g])) < 1e-13   # LSE[0]
        # sum_s dK[s, g] = 0 ; sum_s dV[s, g] = sum over the group of sum_t dO
        ok &= np.max(np.abs(dK.sum(axis=0))) < 1e-10 * max(1.0, np.abs(dK).max())
        grp = hq // hkv
        want = dO.sum(axis=0).reshape(hkv, grp, D).sum(axis=1)
        ok &= np.allclose(dV.sum(axis=0), want, rtol=0, atol=1e-10)
        qo += L * hq * D
        ko += L * hkv * D
        lo += L * hq
    return bool(ok)


def test_bruteforce_packed_mask():
    assert check_bruteforce()


def test_matches_torch_sdpa_autograd():
    assert check_torch()


def test_finite_differences():
    assert check_finite_differences()


def test_golden_two_token():
    assert check_golden()


def test_closed_forms_and_gradient_invariants():
    assert check_invariants()


def test_softmax_rows_sum_to_one_and_causal():
    # V = identity with D = L makes O[t] equal to row t of P.
    L = 24
    wl = small_worklist([L], hq_total=2, hkv_total=1, head_dim=L)
    q, _, _, do = f64_inputs(wl, 4)
    k = A.bf16_to_f64(draw_attention_inputs(wl, 5)[1])
    v = np.eye(L).reshape(-1)
    o, *_ = run_oracle(wl, q, k, v, do, 0.5)
    P = o.reshape(L, 2, L)
    for i in range(2):
        assert np.allclose(P[:, i].sum(axis=1), 1.0, rtol=0, atol=1e-12)
        assert np.all(np.triu(P[:, i], 1) == 0.0)       # exactly zero above the diagonal
        assert np.all(P[:, i][np.tril_indices(L)] > 0.0)


def test_uniform_attention_when_q_zero():
    L = 37
    wl = small_worklist([L], hq_total=4, hkv_total=1, head_dim=8)
    _, k, v, do = f64_inputs(wl, 6)
    q = np.zeros(wl.q_elems())
    o, lse, *_ = run_oracle(wl, q, k, v, do, 0.9)
    V = v.reshape(L, 8)
    want = np.cumsum(V, axis=0) / np.arange(1, L + 1)[:, None]
    assert np.allclose(o.reshape(L, 4, 8), want[:, None, :], rtol=0, atol=1e-13)
    assert np.allclose(lse.reshape(4, L), np.log(np.arange(1, L + 1))[None, :], rtol=0, atol=1e-13)


def test_length_one_items():
    wl = small_worklist([1, 1, 1], hq_total=8, hkv_total=2, head_dim=16)
    q, k, v, do = f64_inputs(wl, 7)
    o, lse, dq, dk, dv = run_oracle(wl, q, k, v, do, 0.25)
    V = v.reshape(3, 2, 16)
    assert np.array_equal(o.reshape(3, 8, 16), np.repeat(V, 4, axis=1))
    assert np.all(dq == 0) and np.all(dk == 0)
    assert np.allclose(dv.reshape(3, 2, 16), do.reshape(3, 2, 4, 16).sum(axis=2), rtol=0, atol=1e-14)


def test_causality_under_perturbation():
    wl = small_worklist([50, 30], hq_total=4, hkv_total=2, head_dim=8)
    q, k, v, do = f64_inputs(wl, 8)
    args = (wl.cu_seqlens, wl.q_heads, wl.kv_heads, 4, 2, 8, 0.4)
    o0, l0 = A.forward(q, k, v, *args)
    t = 20
    for x in (q, k, v):
        x2 = x.copy()
        hh = 4 if x is q else 2
        x2[t * hh * 8:(t + 1) * hh * 8] += 1.5          # token t of item 0
        o1, l1 = A.forward(*(x2 if y is x else y for y in (q, k, v)), *args)
        O0, O1 = o0[:50 * 32].reshape(50, 32), o1[:50 * 32].reshape(50, 32)
        assert np.array_equal(O0[:t], O1[:t])
        assert np.array_equal(l0[:200].reshape(4, 50)[:, :t], l1[:200].reshape(4, 50)[:, :t])
        assert np.array_equal(o0[50 * 32:], o1[50 * 32:])  # item 1 untouched
        assert np.array_equal(l0[200:], l1[200:])
        assert not np.array_equal(O0[t:], O1[t:])


def test_gqa_equals_mha_with_repeated_kv():
    wl = small_worklist([29, 12], hq_total=8, hkv_total=2, head_dim=8)
    q, k, v, do = f64_inputs(wl, 9)
    o, lse, dq, dk, dv = run_oracle(wl, q, k, v, do, 0.3)
    wm = small_worklist([29, 12], hq_total=8, hkv_total=8, head_dim=8)
    rep = lambda x: np.repeat(x.reshape(-1, 2, 8), 4, axis=1).reshape(-1)
    om, lm, dqm, dkm, dvm = run_oracle(wm, q, rep(k), rep(v), do, 0.3)
    assert np.allclose(o, om, rtol=0, atol=1e-14) and np.allclose(dq, dqm, rtol=0, atol=1e-13)
    assert np.allclose(dk, dkm.reshape(-1, 2, 4, 8).sum(axis=2).reshape(-1), rtol=0, atol=1e-12)
    assert np.allclose(dv, dvm.reshape(-1, 2, 4, 8).sum(axis=2).reshape(-1), rtol=0, atol=1e-12)


def test_head_sharded_items_equal_full_heads():
    """Ulysses equivalence: a rank's head subset equals those heads at sp=1."""
    L = 40
    full = small_worklist([L], hq_total=8, hkv_total=2, head_dim=8)
    q, k, v, do = f64_inputs(full, 10)
    o, lse, dq, dk, dv = run_oracle(full, q, k, v, do, 0.35)
    Q, K, V, dO = q.reshape(L, 8, 8), k.reshape(L, 2, 8), v.reshape(L, 2, 8), do.reshape(L, 8, 8)
    for sp in (2, 4, 8):
        for r in range(sp):
            wl = small_worklist([L], 8, 2, 8, sp=[sp], rank=[r])
            ql, qh = wl.q_heads[0]
            kl, kh = wl.kv_heads[0]
            sub = lambda X, a, b: X[:, a:b].reshape(-1)
            os_, ls_, dqs, dks, dvs = run_oracle(wl, sub(Q, ql, qh), sub(K, kl, kh), sub(V, kl, kh),
                                                  sub(dO, ql, qh), 0.35)
            assert np.array_equal(os_, o.reshape(L, 8, 8)[:, ql:qh].reshape(-1))
            assert np.array_equal(dqs, dq.reshape(L, 8, 8)[:, ql:qh].reshape(-1))
            assert np.array_equal(ls_, lse.reshape(8, L)[ql:qh].reshape(-1))
    # the replicated KV head's partial dK/dV summed over the ranks = the sp=1 result
    for sp in (4, 8):
        acc_k = np.zeros((L, 2, 8))
        for r in range(sp):
            wl = small_worklist([L], 8, 2, 8, sp=[sp], rank=[r])
            ql, qh = wl.q_heads[0]
            kl, kh = wl.kv_heads[0]
            _, _, _, dks, _ = run_oracle(wl, Q[:, ql:qh].reshape(-1), K[:, kl:kh].reshape(-1),
                                         V[:, kl:kh].reshape(-1), dO[:, ql:qh].reshape(-1), 0.35)
            acc_k[:, kl:kh] += dks.reshape(L, 1, 8)
        assert np.allclose(acc_k.reshape(-1), dk, rtol=0, atol=1e-12)


def test_row_subsets_match_full():
    """The sampled mode (rows and last key rows) equals the full oracle."""
    L, D = 300, 16
    rng = np.random.default_rng(11)
    q, k, v, do = (rng.standard_normal((L, D)) for _ in range(4))
    o, lse = A.head_forward(q, k, v, 0.2, block=64)
    rows = np.array([0, 1, 63, 64, 150, 299])
    o_r, lse_r = A.head_rows_forward(q, k, v, rows, 0.2)
    assert np.allclose(o_r, o[rows], rtol=0, atol=1e-13) and np.allclose(lse_r, lse[rows], rtol=0, atol=1e-13)
    dq, dk, dv = A.head_backward(q, k, v, do, 0.2, block=64)
    tail = np.arange(L - 40, L)
    dq_t, dk_t, dv_t = A.head_backward(q, k, v, do, 0.2, rows=tail)
    assert np.allclose(dq_t, dq[tail], rtol=0, atol=1e-12)
    assert np.allclose(dk_t[L - 40:], dk[L - 40:], rtol=0, atol=1e-12)
    assert np.allclose(dv_t[L - 40:], dv[L - 40:], rtol=0, atol=1e-12)


def test_empty_item_is_noop():
    wl = small_worklist([0, 5, 0], hq_total=4, hkv_total=2, head_dim=8)
    q, k, v, do = f64_inputs(wl, 12)
    o, lse, dq, dk, dv = run_oracle(wl, q, k, v, do, 0.5)
    w1 = small_worklist([5], 4, 2, 8)
    o1, l1, dq1, dk1, dv1 = run_oracle(w1, q, k, v, do, 0.5)
    for a, b in ((o, o1), (lse, l1), (dq, dq1), (dk, dk1), (dv, dv1)):
        assert np.array_equal(a, b)


# ------------------------------------------------- planted mistakes ----

_ALL_CHECKS = (check_bruteforce, check_torch, check_finite_differences, check_golden, check_invariants)


def _mut_scores_nonstrict(q_rows, k, scale, rows, n_keys):
    s = scale * (q_rows @ k[:n_keys].T)
    s[np.arange(n_keys)[None, :] >= np.asarray(rows)[:, None]] = -np.inf
    s[np.isneginf(s).all(axis=1), 0] = 0.0
    return s


def _mut_scores_noscale(q_rows, k, scale, rows, n_keys):
    s = q_rows @ k[:n_keys].T
    s[np.arange(n_keys)[None, :] > np.asarray(rows)[:, None]] = -np.inf
    return s


def _mut_backward(kind):
    orig = A.head_backward

    def hb(q, k, v, do, scale, rows=None, block=256):
        L, D = q.shape
        rows = np.arange(L) if rows is None else np.asarray(rows)
        dq, dk, dv = np.zeros((rows.size, D)), np.zeros((L, D)), np.zeros((L, D))
        n = L
        o_r, lse_r = A.head_rows_forward(q, k, v, rows, scale)
        s = A._scores(q[rows], k, scale, rows, n)
        p = np.exp(s - lse_r[:, None])
        delta = 0.0 if kind == "no_delta" else np.sum(do[rows] * o_r, axis=1)[:, None]
        dp = do[rows] @ v.T
        ds = p * (dp - delta) if kind != "sign" else p * (delta - dp)
        dq[:] = scale * (ds @ k)
        dk[:] = (1.0 if kind == "dk_noscale" else scale) * (ds.T @ q[rows])
        dv[:] = (ds if kind == "dv_uses_ds" else p).T @ do[rows]
        return dq, dk, dv

    return orig, hb


def _mut_kv_map(h, hq_total, hkv_total):
    return h % hkv_total


@pytest.mark.parametrize("mutation", ["nonstrict_mask", "no_scale", "kv_map", "no_delta", "sign",
                                      "dk_noscale", "dv_uses_ds", "gqa_overwrite"])
def test_planted_mistakes_are_caught(monkeypatch, mutation):
    if mutation == "nonstrict_mask":
        monkeypatch.setattr(A, "_scores", _mut_scores_nonstrict)
    elif mutation == "no_scale":
        monkeypatch.setattr(A, "_scores", _mut_scores_noscale)
    elif mutation == "kv_map":
        monkeypatch.setattr(A, "kv_head_of", _mut_kv_map)
    elif mutation == "gqa_overwrite":
        def backward(q, k, v, do, cu, qh, kvh, hqt, hkvt, D, scale):
            dq = np.zeros_like(q)
            dk = np.zeros_like(k)
            dv = np.zeros_like(v)
            for (L, q_lo, q_hi, kv_lo, kv_hi, qo, ko, lo) in A.item_offsets(cu, qh, kvh, D):
                hq, hkv = q_hi - q_lo, kv_hi - kv_lo
                for i in range(hq):
                    g = A.kv_head_of(q_lo + i, hqt, hkvt) - kv_lo
                    Q = q[qo:qo + L * hq * D].reshape(L, hq, D)
                    K = k[ko:ko + L * hkv * D].reshape(L, hkv, D)
                    V = v[ko:ko + L * hkv * D].reshape(L, hkv, D)
                    dO = do[qo:qo + L * hq * D].reshape(L, hq, D)
                    a, b, c = A.head_backward(Q[:, i], K[:, g], V[:, g], dO[:, i], scale)
                    dq[qo:qo + L * hq * D].reshape(L, hq, D)[:, i] = a
                    dk[ko:ko + L * hkv * D].reshape(L, hkv, D)[:, g] = b   # overwrite, not sum
                    dv[ko:ko + L * hkv * D].reshape(L, hkv, D)[:, g] = c
            return dq, dk, dv
        monkeypatch.setattr(A, "backward", backward)
    else:
        _, hb = _mut_backward(mutation)
        monkeypatch.setattr(A, "head_backward", hb)
    failed = [c.__name__ for c in _ALL_CHECKS if not c()]
    assert failed, f"planted mistake {mutation!r} was caught by no pin"


# ------------------------------------------------------- bf16 widening ----

def _bf16_by_fields(bits):
    """bfloat16 value from its fields: (-1)^s * 2^(e-127) * (1 + m/128) for a
    normal number, (-1)^s * 2^-126 * m/128 for a subnormal one, +-inf for an
    all-ones exponent with a zero fraction (the format's definition; no
    reinterpretation of memory)."""
    out = []
    for b in np.asarray(bits, dtype=np.int64).ravel():
        s, e, m = (b >> 15) & 1, (b >> 7) & 0xFF, b & 0x7F
        sign = -1.0 if s else 1.0
        if e == 0xFF:
            assert m == 0, "no NaN patterns in the pin"
            out.append(sign * np.inf)
        elif e == 0:
            out.append(sign * np.ldexp(m / 128.0, -126))
        else:
            out.append(sign * np.ldexp(1.0 + m / 128.0, int(e) - 127))
    return np.array(out)


def test_bf16_widening_exact_bit_patterns():
    """bf16_to_f64 feeds every other pin with its inputs; it is pinned here
    against values fixed by the bfloat16 format itself."""
    cases = {
        0x3F80: 1.0, 0xBF80: -1.0, 0xC020: -2.5, 0x4049: 3.140625, 0x3E00: 0.125,
        0x0000: 0.0, 0x7F7F: (1.0 + 127 / 128) * 2.0 ** 127,    # largest finite
        0x0080: 2.0 ** -126,                                    # smallest normal
        0x0001: 2.0 ** -133, 0x807F: -(127 / 128) * 2.0 ** -126,  # subnormals
        0x7F80: np.inf, 0xFF80: -np.inf,
    }
    bits = np.array(list(cases), dtype=np.uint16)
    got = A.bf16_to_f64(bits)
    assert got.dtype == np.float64
    assert np.array_equal(got, np.array(list(cases.values())))
    neg_zero = A.bf16_to_f64(np.array([0x8000], dtype=np.uint16))
    assert neg_zero[0] == 0.0 and np.signbit(neg_zero[0])


def test_bf16_widening_matches_field_decoding_and_torch():
    """Every finite bit pattern (both signs) decoded from its fields, and a
    seeded sample widened by torch's own bfloat16 type."""
    allbits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    finite = allbits[((allbits >> 7) & 0xFF) != 0xFF]
    assert np.array_equal(A.bf16_to_f64(finite), _bf16_by_fields(finite))
    rng = np.random.default_rng(11)
    sample = rng.integers(0, 1 << 16, 4096).astype(np.uint16)
    sample = sample[((sample >> 7) & 0xFF) != 0xFF]
    via_torch = torch.from_numpy(sample.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    assert np.array_equal(A.bf16_to_f64(sample), via_torch)


@pytest.mark.parametrize("mistake", ["shift15", "as_half", "drop_sign", "via_f16_bits"])
def test_bf16_widening_planted_mistakes_are_caught(monkeypatch, mistake):
    def wrong(bits):
        b = np.asarray(bits, dtype=np.uint16)
        if mistake == "shift15":
            return (b.astype(np.uint32) << np.uint32(15)).view(np.float32).astype(np.float64)
        if mistake == "as_half":
            return b.view(np.float16).astype(np.float64)
        if mistake == "drop_sign":
            return ((b & np.uint16(0x7FFF)).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
        return (b.astype(np.uint32) << np.uint32(13)).view(np.float32).astype(np.float64)
    monkeypatch.setattr(A, "bf16_to_f64", wrong)
    with pytest.raises(AssertionError):
        test_bf16_widening_exact_bit_patterns()


# ------------------------------------------------- key-row backward ----

def test_key_rows_backward_matches_full_backward():
    """Column-wise key-row gradients from the oracle's own O and LSE equal the
    rows of the full row-blocked backward (the row-block form is pinned above
    against brute force, torch autograd and finite differences)."""
    rng = np.random.default_rng(5)
    for L, D in ((1, 64), (7, 64), (300, 128), (517, 64)):
        q, k, v, do = (rng.standard_normal((L, D)) for _ in range(4))
        scale = 1.0 / np.sqrt(D)
        o, lse = A.head_forward(q, k, v, scale, block=64)
        _, dk, dv = A.head_backward(q, k, v, do, scale, block=64)
        keys = np.unique(np.concatenate([[0, L - 1], rng.integers(0, L, 9)]))
        kk, vv = A.head_key_backward(q, k, v, do, o, lse, keys, scale)
        assert np.allclose(kk, dk[keys], rtol=1e-10, atol=1e-12)
        assert np.allclose(vv, dv[keys], rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("mistake", ["strict", "no_delta", "lse_sign"])
def test_key_rows_backward_planted_mistakes(monkeypatch, mistake):
    real = A.head_key_backward

    def wrong(q, k, v, do, o, lse, keys, scale):
        if mistake == "strict":          # drops the diagonal pair t = s
            keys = np.asarray(keys)
            dk, dv = real(q, k, v, do, o, lse, keys, scale)
            p = np.exp(scale * np.sum(q[keys] * k[keys], axis=1) - np.asarray(lse)[keys])
            ds = p * (np.sum(do[keys] * v[keys], axis=1) - np.sum(do[keys] * o[keys], axis=1))
            return dk - scale * ds[:, None] * q[keys], dv - p[:, None] * do[keys]
        if mistake == "no_delta":
            return real(q, k, v, do, np.zeros_like(o), lse, keys, scale)
        return real(q, k, v, do, o, -np.asarray(lse), keys, scale)
    monkeypatch.setattr(A, "head_key_backward", wrong)
    with pytest.raises(AssertionError):
        test_key_rows_backward_matches_full_backward()
