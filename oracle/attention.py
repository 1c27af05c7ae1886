"""fp64 causal grouped-query attention over a packed variable-length batch.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py): never imported by the
product path.

Definition (the FlashAttention kernels the paper uses, Implementation, are
exact attention; Background, Sequence Packing isolates sequences; Background,
Sequence Parallelism computes attention locally over complete sequences for a
subset of heads).  For item j of length L, local query head i with global
index h = q_lo + i and KV head g = floor(h * Hkv / Hq) (local g - kv_lo),
positions t, s in [0, L):

    S[t, s]   = scale * <Q[t, i, :], K[s, g, :]>          (s <= t; s > t masked)
    LSE[t]    = log sum_{s<=t} exp(S[t, s])               (natural log)
    P[t, s]   = exp(S[t, s] - LSE[t])
    O[t, i]   = sum_{s<=t} P[t, s] V[s, g]

Backward for an upstream gradient dO (analytic):

    Delta[t]  = <dO[t, i], O[t, i]>
    dP[t, s]  = <dO[t, i], V[s, g]>
    dS[t, s]  = P[t, s] (dP[t, s] - Delta[t])
    dQ[t, i]  = scale * sum_s dS[t, s] K[s, g]
    dK[s, g] += scale * sum_t dS[t, s] Q[t, i]     (summed over the local i -> g)
    dV[s, g] += sum_t P[t, s] dO[t, i]             (summed over the local i -> g)

Layout (the attention, i.e. head-sharded, layout): item j's Q/O/dO block is
[L_j, hq_j, D] token-major at element offset D * sum_{i<j} L_i hq_i; K/V/dK/dV
blocks are [L_j, hkv_j, D] at D * sum_{i<j} L_i hkv_i; LSE is [hq_j, L_j] at
sum_{i<j} hq_i L_i.

The computation is row-blocked (one block of query rows at a time, exact,
non-online softmax over the block's full key range) only to bound memory;
there is no other reordering.  Matrix products use numpy (BLAS) in float64.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "bf16_to_f64",
    "item_offsets",
    "kv_head_of",
    "forward",
    "backward",
    "head_forward",
    "head_backward",
    "head_rows_forward",
    "head_key_backward",
]


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def kv_head_of(h: int, hq_total: int, hkv_total: int) -> int:
    """Global KV head shared by global query head h (grouped-query attention)."""
    return (h * hkv_total) // hq_total


def item_offsets(cu_seqlens, q_heads, kv_heads, head_dim):
    """Per item: (L, q_lo, q_hi, kv_lo, kv_hi, q_off, kv_off, lse_off)."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    qh = np.asarray(q_heads, dtype=np.int64).reshape(-1, 2)
    kvh = np.asarray(kv_heads, dtype=np.int64).reshape(-1, 2)
    out, qo, ko, lo = [], 0, 0, 0
    for j in range(len(cu) - 1):
        L = int(cu[j + 1] - cu[j])
        hq = int(qh[j, 1] - qh[j, 0])
        hkv = int(kvh[j, 1] - kvh[j, 0])
        out.append((L, int(qh[j, 0]), int(qh[j, 1]), int(kvh[j, 0]), int(kvh[j, 1]), qo, ko, lo))
        qo += L * hq * head_dim
        ko += L * hkv * head_dim
        lo += L * hq
    return out


def _scores(q_rows, k, scale, rows, n_keys):
    """scale * q_rows @ k[:n_keys].T with keys after each row's position masked."""
    s = scale * (q_rows @ k[:n_keys].T)
    s[np.arange(n_keys)[None, :] > np.asarray(rows)[:, None]] = -np.inf
    return s


def head_rows_forward(q, k, v, rows, scale):
    """O and LSE for the given query rows of one (item, head).

    q: [L, D] (this head), k, v: [L, D] (its KV head); rows: increasing int array.
    """
    rows = np.asarray(rows, dtype=np.int64)
    if rows.size == 0:
        return np.zeros((0, q.shape[1])), np.zeros(0)
    n_keys = int(rows.max()) + 1
    s = _scores(q[rows], k, scale, rows, n_keys)
    m = s.max(axis=1)
    e = np.exp(s - m[:, None])
    l = e.sum(axis=1)
    lse = m + np.log(l)
    p = e / l[:, None]
    return p @ v[:n_keys], lse


def head_forward(q, k, v, scale, block=256):
    """O [L, D] and LSE [L] of one (item, query head)."""
    L = q.shape[0]
    o = np.zeros_like(q)
    lse = np.zeros(L)
    for t0 in range(0, L, block):
        rows = np.arange(t0, min(L, t0 + block))
        o[rows], lse[rows] = head_rows_forward(q, k, v, rows, scale)
    return o, lse


def head_backward(q, k, v, do, scale, rows=None, block=256):
    """Backward of one (item, query head) restricted to the given query rows.

    Returns (dq_rows [len(rows), D], dk [L, D], dv [L, D]) where dk/dv hold the
    contributions of these rows only.  With rows = all rows this is the full
    backward; with rows = [r0, L) the key rows s >= r0 of dk/dv are exact
    (only query rows t >= s attend to key s).
    """
    L, D = q.shape
    rows = np.arange(L) if rows is None else np.asarray(rows, dtype=np.int64)
    dq = np.zeros((rows.size, D))
    dk = np.zeros((L, D))
    dv = np.zeros((L, D))
    for b0 in range(0, rows.size, block):
        r = rows[b0:b0 + block]
        n_keys = int(r.max()) + 1
        o_r, lse_r = head_rows_forward(q, k, v, r, scale)
        s = _scores(q[r], k, scale, r, n_keys)
        p = np.exp(s - lse_r[:, None])
        delta = np.sum(do[r] * o_r, axis=1)
        dp = do[r] @ v[:n_keys].T
        ds = p * (dp - delta[:, None])
        dq[b0:b0 + r.size] = scale * (ds @ k[:n_keys])
        dk[:n_keys] += scale * (ds.T @ q[r])
        dv[:n_keys] += p.T @ do[r]
    return dq, dk, dv


def head_key_backward(q, k, v, do, o, lse, keys, scale):
    """dK and dV at the given key rows of one (item, query head), from given
    per-row LSE and O.

    The same analytic backward as head_backward, taken column-wise: key s is
    reached only by query rows t >= s, so

        P[t, s]  = exp(S[t, s] - LSE[t]),  Delta[t] = <dO[t], O[t]>,
        dK[s]    = scale * sum_{t>=s} P[t, s] (<dO[t], V[s]> - Delta[t]) Q[t],
        dV[s]    = sum_{t>=s} P[t, s] dO[t].

    With the O and LSE of head_forward this is exact; given another
    computation's O and LSE (checked beforehand on rows of their own) it
    gives that computation's key-row gradients without a full forward pass.
    q, k, v, do, o: [L, D]; lse: [L]; keys: int array.  Returns (dk, dv),
    each [len(keys), D].
    """
    keys = np.asarray(keys, dtype=np.int64)
    D = q.shape[1]
    if keys.size == 0:
        return np.zeros((0, D)), np.zeros((0, D))
    t0 = int(keys.min())
    t = np.arange(t0, q.shape[0])
    qt, dot = q[t0:], do[t0:]
    s = scale * (qt @ k[keys].T)
    s[t[:, None] < keys[None, :]] = -np.inf
    p = np.exp(s - np.asarray(lse, dtype=np.float64)[t0:, None])
    delta = np.sum(dot * o[t0:], axis=1)
    ds = p * (dot @ v[keys].T - delta[:, None])
    return scale * (ds.T @ qt), p.T @ dot


def _views(x, off, L, h, D):
    return x[off:off + L * h * D].reshape(L, h, D)


def forward(q, k, v, cu_seqlens, q_heads, kv_heads, hq_total, hkv_total, head_dim, scale):
    """Packed varlen causal GQA forward.  q, k, v: flat float64 (attention layout).

    Returns (o flat float64 like q, lse flat float64 of size sum_j L_j hq_j).
    """
    D = head_dim
    items = item_offsets(cu_seqlens, q_heads, kv_heads, D)
    o = np.zeros_like(q, dtype=np.float64)
    lse = np.zeros(sum(it[0] * (it[2] - it[1]) for it in items))
    for (L, q_lo, q_hi, kv_lo, kv_hi, qo, ko, lo) in items:
        hq, hkv = q_hi - q_lo, kv_hi - kv_lo
        Q, K, V = _views(q, qo, L, hq, D), _views(k, ko, L, hkv, D), _views(v, ko, L, hkv, D)
        O = _views(o, qo, L, hq, D)
        for i in range(hq):
            g = kv_head_of(q_lo + i, hq_total, hkv_total) - kv_lo
            oh, lh = head_forward(Q[:, i], K[:, g], V[:, g], scale)
            O[:, i] = oh
            lse[lo + i * L: lo + (i + 1) * L] = lh
    return o, lse


def backward(q, k, v, do, cu_seqlens, q_heads, kv_heads, hq_total, hkv_total, head_dim, scale):
    """Packed varlen causal GQA backward.  Returns flat float64 (dq, dk, dv)."""
    D = head_dim
    items = item_offsets(cu_seqlens, q_heads, kv_heads, D)
    dq = np.zeros_like(q, dtype=np.float64)
    dk = np.zeros_like(k, dtype=np.float64)
    dv = np.zeros_like(v, dtype=np.float64)
    for (L, q_lo, q_hi, kv_lo, kv_hi, qo, ko, lo) in items:
        hq, hkv = q_hi - q_lo, kv_hi - kv_lo
        Q, K, V = _views(q, qo, L, hq, D), _views(k, ko, L, hkv, D), _views(v, ko, L, hkv, D)
        dO = _views(do, qo, L, hq, D)
        dQ, dK, dV = _views(dq, qo, L, hq, D), _views(dk, ko, L, hkv, D), _views(dv, ko, L, hkv, D)
        for i in range(hq):
            g = kv_head_of(q_lo + i, hq_total, hkv_total) - kv_lo
            a, b, c = head_backward(Q[:, i], K[:, g], V[:, g], dO[:, i], scale)
            dQ[:, i] = a
            dK[:, g] += b
            dV[:, g] += c
    return dq, dk, dv
