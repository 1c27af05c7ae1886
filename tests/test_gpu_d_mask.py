"""Item-masked calls and tree-level recomputation on the HIP path.

Design, NSP Executor: phase streaming issues each tree node's prologue,
compute and epilogue separately, and tree-level recomputation regenerates the
attention outputs of RECOMPUTE nodes before the backward.  Both rest on one
property of the kernels, checked here bit for bit: a call restricted to a set
of items (work-list item mask) reproduces those items' results of the
unrestricted call and leaves every other item's part of the outputs untouched.
"""
import numpy as np
import pytest

from oracle import recompute as R
from paper_2609_22755_amd import nsp
from paper_2609_22755_amd.workloads import draw_attention_inputs, draw_bf16, small_worklist

from gpu_util import require_gpu

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def bits(t):
    import torch
    if t.dtype == torch.bfloat16:
        return nsp.bf16_to_numpy_bits(t)
    return t.detach().cpu().numpy().view(np.uint32)


def spans(wl, per_token):
    """[start, end) element ranges of each item for per-token sizes per_token[j]."""
    n = wl.lengths.astype(np.int64) * per_token
    c = np.concatenate([[0], np.cumsum(n)])
    return [(int(c[j]), int(c[j + 1])) for j in range(wl.n_items)]


def fill_sentinel(buf):
    for k in ("o", "lse", "dq", "dk", "dv"):
        buf[k].fill_(float("nan"))


def wl_mixed():
    return small_worklist([700, 129, 1, 300, 2048, 0, 64], 32, 4, 128, sp=[2, 1, 1, 8, 4, 1, 1],
                          rank=[1, 0, 0, 6, 3, 0, 0])


def wl_long():
    # a 9000-token item: its K/V head slices (4.6 MB) exceed one XCD's L2, so
    # the full call launches its units in XCD runs; the masked call below
    # drops that item and launches the rest in plain longest-first order
    return small_worklist([9000, 700, 129, 300, 1], 32, 4, 128, sp=[1, 2, 1, 8, 1], rank=[0, 1, 0, 6, 0])


@pytest.mark.parametrize("case", ["mixed", "long_item_masked_out"])
def test_masked_forward_and_backward_reproduce_selected_items(case):
    import torch
    if case == "mixed":
        wl, mask = wl_mixed(), np.array([1, 0, 1, 0, 1, 1, 0], dtype=np.uint8)
    else:
        wl, mask = wl_long(), np.array([0, 1, 1, 1, 1], dtype=np.uint8)
        assert 4 * 9000 * wl.head_dim > 4 << 20 >= 4 * 700 * wl.head_dim
    print(f"[mask] case {case}: lengths {wl.lengths.tolist()} mask {mask.tolist()}", flush=True)
    qb, kb, vb, db = draw_attention_inputs(wl, 31)
    q, k, v, do = (nsp.to_device_bf16(x) for x in (qb, kb, vb, db))
    full = nsp.alloc_like_worklist(wl)
    nsp.nsp_varlen_attn_fwd(wl, q, k, v, full["o"], full["lse"], SCALE)
    nsp.nsp_varlen_attn_bwd(wl, q, k, v, full["o"], do, full["lse"], full["dq"], full["dk"], full["dv"],
                            full["ws"], SCALE)
    sub = wl.select(mask)
    part = nsp.alloc_like_worklist(wl)
    fill_sentinel(part)
    nsp.nsp_varlen_attn_fwd(sub, q, k, v, part["o"], part["lse"], SCALE)
    nsp.nsp_varlen_attn_bwd(sub, q, k, v, part["o"], do, part["lse"], part["dq"], part["dk"], part["dv"],
                            part["ws"], SCALE)
    torch.cuda.synchronize()
    D = wl.head_dim
    for name, per_tok in (("o", wl.hq * D), ("dq", wl.hq * D), ("lse", wl.hq), ("dk", wl.hkv * D),
                          ("dv", wl.hkv * D)):
        a, b = bits(full[name]), bits(part[name])
        for j, (s, e) in enumerate(spans(wl, per_tok)):
            if mask[j]:
                assert np.array_equal(a[s:e], b[s:e]), (name, j)
            else:
                got = part[name].flatten()[s:e].float()
                assert bool(torch.isnan(got).all()), (name, j)   # untouched


def test_recompute_regenerates_outputs_bitwise():
    import torch
    wl = wl_mixed()
    qb, kb, vb, db = draw_attention_inputs(wl, 32)
    q, k, v, do = (nsp.to_device_bf16(x) for x in (qb, kb, vb, db))
    buf = nsp.alloc_like_worklist(wl)
    nsp.nsp_varlen_attn_fwd(wl, q, k, v, buf["o"], buf["lse"], SCALE)
    torch.cuda.synchronize()
    o_ref, lse_ref = bits(buf["o"]).copy(), bits(buf["lse"]).copy()
    D = wl.head_dim
    sizes = [R.slice_bytes(int(L), int(h), D, 2) for L, h in zip(wl.lengths, wl.hq)]
    for budget in (0, sum(sizes) // 3, sum(sizes) // 2, sum(sizes)):
        save, _ = nsp.nsp_recompute_plan(wl, budget, nsp.NSP_BF16)
        # the forward keeps only the SAVE slices: drop the others
        for name, per_tok in (("o", wl.hq * D), ("lse", wl.hq)):
            for j, (s, e) in enumerate(spans(wl, per_tok)):
                if not save[j]:
                    buf[name].view(-1)[s:e] = float("nan")
        # before the backward: recompute the RECOMPUTE items only
        rec = (1 - save).astype(np.uint8)
        if rec.any():
            nsp.nsp_varlen_attn_fwd(wl.select(rec), q, k, v, buf["o"], buf["lse"], SCALE)
        torch.cuda.synchronize()
        assert np.array_equal(bits(buf["o"]), o_ref), budget
        assert np.array_equal(bits(buf["lse"]), lse_ref), budget


def test_masked_pack_unpack_move_selected_items_only():
    import torch
    wl = small_worklist([256, 64, 512, 96], 32, 4, 128, sp=[8, 2, 4, 1])
    mask = np.array([0, 1, 1, 0], dtype=np.uint8)
    sub = wl.select(mask)
    rng = np.random.default_rng(9)
    for kind, H, elems in ((nsp.NSP_KIND_Q, 32, wl.q_elems()), (nsp.NSP_KIND_KV, 4, wl.kv_elems())):
        xs = nsp.to_device_bf16(draw_bf16(rng, wl.seq_tokens() * H * 128))
        ref = torch.empty(elems, dtype=torch.bfloat16, device="cuda")
        nsp.nsp_ulysses_pack(wl, kind, xs, ref)
        got = torch.full((elems,), float("nan"), dtype=torch.bfloat16, device="cuda")
        nsp.nsp_ulysses_pack(sub, kind, xs, got)
        back = torch.full_like(xs, float("nan"))
        nsp.nsp_ulysses_unpack(sub, kind, nsp.NSP_UNPACK_SELECT, ref, back)
        torch.cuda.synchronize()
        hl = np.array([H // s if H >= s else 1 for s in wl.sp], dtype=np.int64)
        for j, (s, e) in enumerate(spans(wl, hl * 128)):
            if mask[j]:
                assert np.array_equal(bits(got)[s:e], bits(ref)[s:e]), (kind, j)
            else:
                assert bool(torch.isnan(got[s:e].float()).all()), (kind, j)
        seq_tok = wl.lengths.astype(np.int64) // wl.sp
        c = np.concatenate([[0], np.cumsum(seq_tok)]) * H * 128
        for j in range(wl.n_items):
            s, e = int(c[j]), int(c[j + 1])
            if mask[j]:
                assert np.array_equal(bits(back)[s:e], bits(xs)[s:e]), (kind, j)
            else:
                assert bool(torch.isnan(back[s:e].float()).all()), (kind, j)
