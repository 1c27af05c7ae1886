"""libnsp.so loads, exports every symbol include/nsp.h declares, and rejects
invalid arguments with the documented status before launching anything.

These run without a GPU: validation happens on the host before any HIP call.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2609_22755_amd import nsp
from paper_2609_22755_amd.workloads import make_config, small_worklist

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000   # a 16-byte aligned non-NULL address; never dereferenced on error paths


@pytest.fixture(scope="module")
def lib():
    return nsp.load_library()


def declared_functions():
    src = open(os.path.join(ROOT, "include", "nsp.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(nsp_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    assert set(declared_functions()) == set(nsp.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings_and_version(lib):
    for code in range(6):
        assert nsp.status_string(code).startswith("NSP_")
    assert "gfx950" in nsp.version()


def _fwd(wl, **kw):
    lib = nsp.load_library()
    w = nsp._WL(wl, with_sp=False)
    args = dict(scale=0.125, causal=1, q=FAKE, k=FAKE, v=FAKE, o=FAKE, odt=nsp.NSP_BF16, lse=FAKE)
    args.update(kw)
    st = lib.nsp_varlen_attn_fwd(w.ref, args["scale"], args["causal"], args["q"], args["k"], args["v"],
                                 args["o"], args["odt"], args["lse"], None)
    return st, lib.nsp_last_error().decode()


def _wl(**over):
    wl = small_worklist([64, 33, 0, 7], hq_total=8, hkv_total=2, head_dim=64)
    for k, v in over.items():
        setattr(wl, k, v)
    return wl


@pytest.mark.parametrize("case,status,word", [
    ("neg_items", nsp.NSP_EINVAL, "n_items"),
    ("cu0", nsp.NSP_EINVAL, "cu_seqlens[0]"),
    ("decreasing", nsp.NSP_EINVAL, "decreases"),
    ("empty_heads", nsp.NSP_EINVAL, "query head range"),
    ("q_out_of_range", nsp.NSP_EINVAL, "query head range"),
    ("kv_mismatch", nsp.NSP_EINVAL, "uses KV head"),
    ("bad_totals", nsp.NSP_EINVAL, "multiple"),
    ("head_dim", nsp.NSP_EUNSUPPORTED, "head_dim"),
])
def test_worklist_validation(case, status, word):
    wl = _wl()
    if case == "neg_items":
        c = nsp.CWorkList(n_items=-1, hq_total=8, hkv_total=2, head_dim=64)
        lib = nsp.load_library()
        st = lib.nsp_varlen_attn_fwd(ctypes.byref(c), 0.1, 1, FAKE, FAKE, FAKE, FAKE, 0, FAKE, None)
        assert st == status and word in lib.nsp_last_error().decode()
        return
    if case == "cu0":
        cu = _wl().cu_seqlens.copy()
        cu[0] = 5
        wl = _CustomCu(_wl(), cu)
    elif case == "decreasing":
        cu = _wl().cu_seqlens.copy()
        cu[2] = cu[1] - 1
        wl = _CustomCu(_wl(), cu)
    elif case == "empty_heads":
        wl.q_heads = wl.q_heads.copy()
        wl.q_heads[1] = (3, 3)
    elif case == "q_out_of_range":
        wl.q_heads = wl.q_heads.copy()
        wl.q_heads[1] = (0, 9)
    elif case == "kv_mismatch":
        wl.kv_heads = wl.kv_heads.copy()
        wl.kv_heads[0] = (0, 1)   # query heads 4..7 use KV head 1
    elif case == "bad_totals":
        wl.hkv_total = 3
    elif case == "head_dim":
        wl.head_dim = 96
    st, msg = _fwd(wl)
    assert st == status, msg
    assert word in msg


class _CustomCu:
    """A work list view with explicit cu_seqlens."""

    def __init__(self, wl, cu):
        self.__dict__.update(wl.__dict__)
        self._cu = np.asarray(cu, dtype=np.int32)

    @property
    def cu_seqlens(self):
        return self._cu

    @property
    def n_items(self):
        return len(self._cu) - 1


def test_argument_validation():
    wl = _wl()
    assert _fwd(wl, causal=0)[0] == nsp.NSP_EUNSUPPORTED
    assert _fwd(wl, scale=0.0)[0] == nsp.NSP_EINVAL
    assert _fwd(wl, scale=float("nan"))[0] == nsp.NSP_EINVAL
    assert _fwd(wl, q=None)[0] == nsp.NSP_EINVAL
    assert _fwd(wl, v=FAKE + 8)[0] == nsp.NSP_EINVAL      # misaligned
    assert _fwd(wl, odt=7)[0] == nsp.NSP_EINVAL


def test_empty_worklist_is_a_noop():
    wl = small_worklist([], 8, 2, 64)
    assert _fwd(wl, q=None, k=None, v=None, o=None, lse=None)[0] == nsp.NSP_OK
    wl0 = small_worklist([0, 0], 8, 2, 64)
    assert _fwd(wl0, q=None, k=None, v=None, o=None, lse=None)[0] == nsp.NSP_OK


def test_bwd_workspace_and_errors():
    wl = make_config("tiny").wl
    lib = nsp.load_library()
    ws = nsp.nsp_varlen_attn_bwd_workspace(wl)
    assert ws >= wl.lse_elems() * 4 and ws % 256 == 0
    w = nsp._WL(wl, with_sp=False)

    def bwd(ws_ptr, ws_bytes, gdt=nsp.NSP_BF16, odt=nsp.NSP_BF16):
        return lib.nsp_varlen_attn_bwd(w.ref, 0.125, 1, FAKE, FAKE, FAKE, FAKE, odt, FAKE, FAKE, FAKE, FAKE,
                                       FAKE, gdt, ws_ptr, ws_bytes, None)
    assert bwd(FAKE, ws - 1) == nsp.NSP_EWORKSPACE
    assert bwd(None, ws) == nsp.NSP_EWORKSPACE
    assert bwd(FAKE, ws, odt=5) == nsp.NSP_EINVAL
    assert bwd(FAKE, ws, gdt=3) == nsp.NSP_EINVAL
    assert bwd(FAKE + 16, ws) == nsp.NSP_EINVAL           # workspace not 256-aligned


def test_relayout_validation():
    lib = nsp.load_library()
    base = make_config("tiny").pack_wl

    def pack(wl, kind=nsp.NSP_KIND_Q, dtype=nsp.NSP_BF16):
        return lib.nsp_ulysses_pack(nsp._WL(wl).ref, kind, dtype, FAKE, FAKE, None)

    bad_sp = small_worklist([64, 128], 8, 2, 64, sp=[2, 2])
    bad_sp.sp = np.array([3, 2], dtype=np.int32)
    assert pack(bad_sp) == nsp.NSP_EINVAL
    odd = small_worklist([63], 8, 2, 64, sp=[2])
    assert pack(odd) == nsp.NSP_EINVAL
    width = small_worklist([64], 8, 2, 64, sp=[2])
    width.q_heads = np.array([[0, 8]], dtype=np.int32)
    assert pack(width) == nsp.NSP_EINVAL
    assert pack(base, kind=5) == nsp.NSP_EINVAL
    assert pack(base, dtype=9) == nsp.NSP_EINVAL
    nosp = small_worklist([64], 8, 2, 64, sp=[2])
    assert lib.nsp_ulysses_pack(nsp._WL(nosp, with_sp=False).ref, 0, 0, FAKE, FAKE, None) == nsp.NSP_EINVAL
    assert lib.nsp_ulysses_unpack(nsp._WL(base).ref, 0, 0, 7, FAKE, FAKE, None) == nsp.NSP_EINVAL


# --------------------------------------------------- tree-level recompute --
# nsp_recompute_plan is host-only, so it is checked here against the oracle.

def _plan_wl(L, sp, hq_total=32, hkv_total=4, D=128):
    from paper_2609_22755_amd.workloads import make_worklist
    return make_worklist(L, sp, hq_total, hkv_total, D)


def test_recompute_plan_hand_worked():
    from conftest import load_golden
    g = {k: [int(x) for x in v] for k, v in load_golden("recompute_plan_small.txt").items()}
    wl = _plan_wl(g["lengths"], g["sp"])
    for b, budget in enumerate(g["budgets"]):
        save, used = nsp.nsp_recompute_plan(wl, budget, nsp.NSP_BF16)
        assert save.tolist() == g[f"save_{b}"]
        assert used == g["saved"][b]


@pytest.mark.parametrize("seed", range(25))
def test_recompute_plan_matches_oracle(seed):
    from oracle import recompute as R
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 20))
    sp = rng.choice([1, 2, 4, 8], size=n)
    L = (rng.integers(0, 20000, size=n) // sp) * sp
    wl = _plan_wl(L.tolist(), sp.tolist())
    for odt, ob in ((nsp.NSP_BF16, 2), (nsp.NSP_F32, 4)):
        size = [R.slice_bytes(int(L[j]), int(wl.hq[j]), 128, ob) for j in range(n)]
        for budget in [0, sum(size)] + [int(x) for x in rng.integers(0, sum(size) + 1, size=4)]:
            ref, ref_used = R.recompute_plan(L.tolist(), sp.tolist(), wl.hq.tolist(), 128, ob, budget)
            save, used = nsp.nsp_recompute_plan(wl, budget, odt)
            assert save.tolist() == ref and used == ref_used


def test_recompute_plan_rejects_bad_arguments(lib):
    wl = _plan_wl([64, 32], [2, 1])
    with pytest.raises(nsp.NspError) as e:
        nsp.nsp_recompute_plan(wl, -1)
    assert e.value.status == nsp.NSP_EINVAL
    with pytest.raises(nsp.NspError) as e:
        nsp.nsp_recompute_plan(wl, 10, o_dtype=7)
    assert e.value.status == nsp.NSP_EINVAL


# ------------------------------------------------- phase-streaming executor --

def _exec_status(wl, node_sp=None, phases=3, missing=()):
    import ctypes as C
    lib = nsp.load_library()
    w = nsp._WL(wl)
    b = nsp.CStepBuffers()
    for name, _ in nsp.CStepBuffers._fields_[:-1]:
        setattr(b, name, None if name in missing else FAKE)
    b.ws_bytes = 1 << 20
    order = None if node_sp is None else np.ascontiguousarray(node_sp, dtype=np.int32)
    st = lib.nsp_executor_step(w.ref, None if order is None else order.ctypes.data_as(C.POINTER(C.c_int32)),
                               0 if order is None else int(order.size), phases, 0.125, C.byref(b), None, None)
    return st, lib.nsp_last_error().decode()


def test_executor_rejects_bad_arguments(lib):
    wl = small_worklist([64, 32, 128], hq_total=8, hkv_total=2, head_dim=64, sp=[2, 1, 2])
    for kw in (dict(node_sp=[2]), dict(node_sp=[2, 1, 2]), dict(node_sp=[4, 2, 1]), dict(phases=0),
               dict(phases=4), dict(missing=("o_seq",)), dict(phases=2, missing=("dout",))):
        st, msg = _exec_status(wl, **kw)
        assert st == nsp.NSP_EINVAL and "nsp_executor_step" in msg, (kw, msg)
    st, msg = _exec_status(wl.select([1, 0, 1]))
    assert st == nsp.NSP_EINVAL and "mask" in msg


def test_noalloc_backward_limits_without_a_gpu():
    """The allocation-free backward rejects a work list beyond its scratch
    before any device call; one row under the limit passes that check (it
    then needs a device)."""
    lib = nsp.load_library()
    fake = ctypes.c_void_p(FAKE)

    def call(wl):
        w = nsp._WL(wl, with_sp=False)
        return lib.nsp_varlen_attn_bwd_noalloc(w.ref, 0.1, 1, fake, fake, fake, fake, 0, fake, fake, fake, fake,
                                               fake, 0, None)
    rows = nsp.NSP_NOALLOC_MAX_ROWS
    over = small_worklist([rows // 32 + 1], 32, 4, 128)
    assert call(over) == nsp.NSP_EWORKSPACE
    assert b"allocation-free" in lib.nsp_last_error()
    over_by_one = small_worklist([rows // 4 + 1], 4, 1, 128)
    assert call(over_by_one) == nsp.NSP_EWORKSPACE
    import torch
    if torch.cuda.device_count() == 0:
        # with no device the call stops at its first HIP call, past the size
        # check (never run where a device would execute the fake pointers)
        exact = small_worklist([rows // 4], 4, 1, 128)
        assert exact.lse_elems() == rows
        assert call(exact) == nsp.NSP_EHIP


def test_mfma_ceiling_rejects_bad_arguments(lib):
    """The ceiling measurement checks its arguments before any device call."""
    sec, tf = ctypes.c_double(0.0), ctypes.c_double(0.0)
    for args in ((4, 0, 1, 1 << 16), (-1, 0, 1, 1 << 16), (0, 0, 3, 1 << 16), (0, 0, 0, 1 << 16),
                 (0, 0, 1, 0), (0, 0, 1, 24), (0, 0, 2, 16), (0, 0, 1, (1 << 24) + 16)):
        assert lib.nsp_mfma_ceiling(*args, ctypes.byref(sec), ctypes.byref(tf)) == nsp.NSP_EINVAL, args
    assert lib.nsp_mfma_ceiling(0, 0, 1, 1 << 16, None, ctypes.byref(tf)) == nsp.NSP_EINVAL
    assert b"nsp_mfma_ceiling" in lib.nsp_last_error()
