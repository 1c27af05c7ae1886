"""Shared helpers of the GPU tests: run the HIP path through the C ABI and
compare with the oracle.  Imported by tests only."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import attention as OA
from paper_2609_22755_amd import nsp

# Tolerances of the attention path (float32 accumulation of bf16 products):
FWD_REL_L2 = 5e-3
FWD_MAX_ABS = 1e-2
GRAD_REL_L2 = 1e-2
LSE_MAX_ABS = 2e-3


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    nsp.load_library()   # raises if the HIP library was not built: no fallback


def rel_l2(x, r):
    x = np.asarray(x, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    return float(np.linalg.norm(x - r) / max(np.linalg.norm(r), 1e-300))


def max_abs(x, r):
    return float(np.max(np.abs(np.asarray(x, np.float64) - np.asarray(r, np.float64)))) if np.size(r) else 0.0


def to_np(t):
    import torch
    if t.dtype == torch.bfloat16:
        return OA.bf16_to_f64(nsp.bf16_to_numpy_bits(t))
    return t.detach().cpu().numpy().astype(np.float64)


def run_attention(wl, qb, kb, vb, dob, scale, o_dtype=None, g_dtype=None, bwd=True):
    """Upload bf16 bit arrays, run fwd (+ bwd) through the C ABI; torch tensors out."""
    import torch
    o_dtype = o_dtype or torch.bfloat16
    g_dtype = g_dtype or torch.bfloat16
    q, k, v, do = (nsp.to_device_bf16(x) for x in (qb, kb, vb, dob))
    buf = nsp.alloc_like_worklist(wl, o_dtype=o_dtype, grad_dtype=g_dtype)
    nsp.nsp_varlen_attn_fwd(wl, q, k, v, buf["o"], buf["lse"], scale)
    if bwd:
        nsp.nsp_varlen_attn_bwd(wl, q, k, v, buf["o"], do, buf["lse"], buf["dq"], buf["dk"], buf["dv"],
                                buf["ws"], scale)
    torch.cuda.synchronize()
    return buf


def oracle_full(wl, qb, kb, vb, dob, scale):
    q, k, v, do = (OA.bf16_to_f64(x) for x in (qb, kb, vb, dob))
    args = (wl.cu_seqlens, wl.q_heads, wl.kv_heads, wl.hq_total, wl.hkv_total, wl.head_dim, scale)
    o, lse = OA.forward(q, k, v, *args)
    dq, dk, dv = OA.backward(q, k, v, do, *args)
    return dict(o=o, lse=lse, dq=dq, dk=dk, dv=dv)


def report(name, **vals):
    print(f"[parity] {name}: " + ", ".join(f"{k}={v:.3e}" for k, v in vals.items()), flush=True)
