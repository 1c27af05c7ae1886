"""The allocation-free backward (nsp_varlen_attn_bwd_noalloc) against the
workspace backward (nsp_varlen_attn_bwd), through the C ABI.

Both run the same kernels on the same unit schedule, so the gradients must
agree bit for bit.  Calls in a row with different work lists -- a larger one,
then a smaller one, then the first again -- check that each call copies its
own schedule into the device scratch (and that a smaller call leaves no trace
of the larger one in its results); the bf16 and float32 gradient stores and
a float32 O input are covered.
"""
import ctypes

import numpy as np
import pytest

from paper_2609_22755_amd import nsp
from paper_2609_22755_amd.workloads import draw_attention_inputs, small_worklist

from gpu_util import require_gpu

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _bits(t):
    import torch
    if t.dtype == torch.bfloat16:
        return nsp.bf16_to_numpy_bits(t)
    return t.cpu().numpy().view(np.uint32)


def _setup(wl, seed, o_dtype):
    import torch
    qb, kb, vb, db = draw_attention_inputs(wl, seed)
    q, k, v, do = (nsp.to_device_bf16(x) for x in (qb, kb, vb, db))
    o = torch.empty(wl.q_elems(), dtype=o_dtype, device="cuda")
    lse = torch.empty(wl.lse_elems(), dtype=torch.float32, device="cuda")
    nsp.nsp_varlen_attn_fwd(wl, q, k, v, o, lse, SCALE)
    return q, k, v, do, o, lse


def _grads(wl, g_dtype):
    import torch
    return [torch.full((n,), float("nan"), dtype=g_dtype, device="cuda")
            for n in (wl.q_elems(), wl.kv_elems(), wl.kv_elems())]


def _check_pair(name, wl, seed, o_dtype, g_dtype):
    import torch
    q, k, v, do, o, lse = _setup(wl, seed, o_dtype)
    ws = torch.empty(nsp.nsp_varlen_attn_bwd_workspace(wl), dtype=torch.uint8, device="cuda")
    ref = _grads(wl, g_dtype)
    nsp.nsp_varlen_attn_bwd(wl, q, k, v, o, do, lse, *ref, ws, SCALE)
    got = _grads(wl, g_dtype)
    nsp.nsp_varlen_attn_bwd_noalloc(wl, q, k, v, o, do, lse, *got, SCALE)
    torch.cuda.synchronize()
    for n, a, b in zip(("dq", "dk", "dv"), ref, got):
        assert np.array_equal(_bits(a), _bits(b)), (name, n)
    print(f"[noalloc] {name}: bitwise equal ({wl.n_items} items, {wl.lse_elems()} rows)", flush=True)


WL_LARGE = small_worklist([4096, 700, 129, 1, 300, 2048, 0, 64, 1500], 32, 4, 128,
                          sp=[4, 2, 1, 1, 8, 4, 1, 1, 1], rank=[1, 1, 0, 0, 6, 3, 0, 0, 0])
WL_SMALL = small_worklist([200, 64, 33], 32, 4, 128, sp=[1, 8, 2], rank=[0, 5, 1])


def test_noalloc_matches_workspace_backward_twice_smaller_second():
    import torch
    _check_pair("large bf16", WL_LARGE, 61, torch.bfloat16, torch.bfloat16)
    _check_pair("small bf16", WL_SMALL, 62, torch.bfloat16, torch.bfloat16)
    _check_pair("large again, f32 O and grads", WL_LARGE, 63, torch.float32, torch.float32)
    _check_pair("small again, d64", small_worklist([100, 17, 260], 8, 2, 64), 64, torch.bfloat16, torch.bfloat16)


def test_noalloc_matches_workspace_backward_at_full_size():
    """The long-tail share (8388608 rows, within the scratch) through both
    backward entry points: the persistent passes loop over thousands of units
    on the scratch's queue heads and schedule; gradients bit for bit equal."""
    import torch
    from paper_2609_22755_amd.workloads import make_config
    w = make_config("longtail_4level")
    wl = w.wl
    assert wl.lse_elems() <= nsp.NSP_NOALLOC_MAX_ROWS
    g = torch.Generator(device="cuda")
    g.manual_seed(71)

    def draw(n):
        return torch.randn(n, generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)

    q, k, v, do = draw(wl.q_elems()), draw(wl.kv_elems()), draw(wl.kv_elems()), draw(wl.q_elems())
    o = torch.empty(wl.q_elems(), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(wl.lse_elems(), dtype=torch.float32, device="cuda")
    nsp.nsp_varlen_attn_fwd(wl, q, k, v, o, lse, w.softmax_scale)
    ws = torch.empty(nsp.nsp_varlen_attn_bwd_workspace(wl), dtype=torch.uint8, device="cuda")
    ref = _grads(wl, torch.bfloat16)
    nsp.nsp_varlen_attn_bwd(wl, q, k, v, o, do, lse, *ref, ws, w.softmax_scale)
    got = _grads(wl, torch.bfloat16)
    nsp.nsp_varlen_attn_bwd_noalloc(wl, q, k, v, o, do, lse, *got, w.softmax_scale)
    torch.cuda.synchronize()
    for n, a, b in zip(("dq", "dk", "dv"), ref, got):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16)), n
    print(f"[noalloc] longtail_4level: bitwise equal ({wl.n_items} items, {wl.lse_elems()} rows)", flush=True)
    del q, k, v, do, o, lse, ws, ref, got
    torch.cuda.empty_cache()


def test_noalloc_rejects_oversized_worklists_through_the_abi():
    lib = nsp.load_library()
    big = small_worklist([nsp.NSP_NOALLOC_MAX_ROWS // 32 + 1], 32, 4, 128)
    fake = ctypes.c_void_p(1 << 20)
    w = nsp._WL(big, with_sp=False)
    st = lib.nsp_varlen_attn_bwd_noalloc(w.ref, 0.1, 1, fake, fake, fake, fake, 0, fake, fake, fake, fake, fake,
                                         0, None)
    assert st == nsp.NSP_EWORKSPACE, nsp.status_string(st)
    assert b"allocation-free" in lib.nsp_last_error()
