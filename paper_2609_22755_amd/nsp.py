"""Thin ctypes binding of libnsp.so (include/nsp.h), same names as the C ABI.

Argument marshalling only: every step of the hot path runs in the HIP
kernels of libnsp.so.  Tensors are torch tensors on a ROCm device (torch is
used for device memory and streams only); work lists are
``paper_2609_22755_amd.workloads.WorkList`` objects (host arrays).

The library must have been built (``python -m paper_2609_22755_amd.build``);
loading fails loudly otherwise -- there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libnsp.so")

NSP_OK, NSP_EINVAL, NSP_EUNSUPPORTED, NSP_EHIP, NSP_ENOMEM, NSP_EWORKSPACE, NSP_EINFEASIBLE = range(7)
NSP_BF16, NSP_F32 = 0, 1
NSP_KIND_Q, NSP_KIND_KV = 0, 1
NSP_UNPACK_SELECT, NSP_UNPACK_SUM = 0, 1

EXPORTED = (
    "nsp_varlen_attn_fwd",
    "nsp_varlen_attn_bwd_workspace",
    "nsp_varlen_attn_bwd",
    "nsp_varlen_attn_bwd_noalloc",
    "nsp_ulysses_pack",
    "nsp_ulysses_unpack",
    "nsp_recompute_plan",
    "nsp_attn_schedule",
    "nsp_attn_kv_queues",
    "nsp_executor_step",
    "nsp_sp_tree_plan",
    "nsp_sp_tree_worklist",
    "nsp_status_string",
    "nsp_last_error",
    "nsp_version",
    "nsp_timing_enable",
    "nsp_timing_reset",
    "nsp_timing_query",
    "nsp_mfma_ceiling",
)


class NspError(RuntimeError):
    def __init__(self, status: int, call: str, detail: str):
        self.status = status
        super().__init__(f"{call} failed with status {status}: {detail}")


class CWorkList(ctypes.Structure):
    _fields_ = [
        ("n_items", ctypes.c_int32),
        ("cu_seqlens", ctypes.POINTER(ctypes.c_int32)),
        ("q_heads", ctypes.POINTER(ctypes.c_int32)),
        ("kv_heads", ctypes.POINTER(ctypes.c_int32)),
        ("sp", ctypes.POINTER(ctypes.c_int32)),
        ("hq_total", ctypes.c_int32),
        ("hkv_total", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("item_mask", ctypes.POINTER(ctypes.c_uint8)),
    ]


class CStepBuffers(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "q_seq", "k_seq", "v_seq", "do_seq", "o_seq", "dq_seq", "dk_seq", "dv_seq",
        "q", "k", "v", "o", "dout", "dq", "dk", "dv", "lse", "workspace")] + [("ws_bytes", ctypes.c_size_t)]


NSP_STEP_FORWARD, NSP_STEP_BACKWARD = 1, 2


class CPlanParams(ctypes.Structure):
    _fields_ = [
        ("world", ctypes.c_int32), ("sp_max", ctypes.c_int32),
        ("hq_total", ctypes.c_int32), ("hkv_total", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("elem_bytes", ctypes.c_int32),
        ("attn_fwd_flops", ctypes.c_double), ("attn_bwd_flops", ctypes.c_double),
        ("link_bytes", ctypes.c_double), ("links", ctypes.c_int32),
        ("a2a_latency", ctypes.c_double),
        ("dense_fwd_per_token", ctypes.c_double), ("dense_bwd_per_token", ctypes.c_double),
        ("token_budget", ctypes.c_double),
        ("prefix", ctypes.c_int32), ("beam", ctypes.c_int32), ("monotone", ctypes.c_int32),
    ]


@dataclasses.dataclass
class SpTreeParams:
    """nsp_plan_params (include/nsp.h).  The default rates are this library's
    measured ones on MI355X: attention forward about 1.2 PFLOP/s and backward
    about 0.9 PFLOP/s (counted flops), seven xGMI links of about 153 GB/s."""
    world: int
    sp_max: int
    hq_total: int
    hkv_total: int
    head_dim: int
    elem_bytes: int = 2
    attn_fwd_flops: float = 1.2e15
    attn_bwd_flops: float = 9.0e14
    link_bytes: float = 153e9
    links: int = 7
    a2a_latency: float = 20e-6
    dense_fwd_per_token: float = 0.0
    dense_bwd_per_token: float = 0.0
    token_budget: float = float("inf")
    prefix: int = 16
    beam: int = 8
    monotone: bool = True

    def c(self) -> CPlanParams:
        return CPlanParams(**{f: (int(v) if isinstance(v, bool) else v)
                              for f, v in dataclasses.asdict(self).items()})

_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libnsp.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} not found: build it with `python -m paper_2609_22755_amd.build` "
                          "(there is no non-HIP fallback)")
    lib = ctypes.CDLL(path)
    p, i32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    wl = ctypes.POINTER(CWorkList)
    lib.nsp_varlen_attn_fwd.argtypes = [wl, f32, i32, p, p, p, p, i32, p, p]
    lib.nsp_varlen_attn_fwd.restype = i32
    lib.nsp_varlen_attn_bwd_workspace.argtypes = [wl]
    lib.nsp_varlen_attn_bwd_workspace.restype = sz
    lib.nsp_varlen_attn_bwd.argtypes = [wl, f32, i32, p, p, p, p, i32, p, p, p, p, p, i32, p, sz, p]
    lib.nsp_varlen_attn_bwd.restype = i32
    lib.nsp_varlen_attn_bwd_noalloc.argtypes = [wl, f32, i32, p, p, p, p, i32, p, p, p, p, p, i32, p]
    lib.nsp_varlen_attn_bwd_noalloc.restype = i32
    lib.nsp_ulysses_pack.argtypes = [wl, i32, i32, p, p, p]
    lib.nsp_ulysses_pack.restype = i32
    lib.nsp_ulysses_unpack.argtypes = [wl, i32, i32, i32, p, p, p]
    lib.nsp_ulysses_unpack.restype = i32
    lib.nsp_recompute_plan.argtypes = [wl, ctypes.c_int64, i32, ctypes.POINTER(ctypes.c_uint8),
                                       ctypes.POINTER(ctypes.c_int64)]
    lib.nsp_recompute_plan.restype = i32
    lib.nsp_attn_schedule.argtypes = [wl, i32, ctypes.POINTER(ctypes.c_int32), ctypes.c_int64,
                                      ctypes.POINTER(ctypes.c_int64)]
    lib.nsp_attn_schedule.restype = i32
    lib.nsp_attn_kv_queues.argtypes = [wl, ctypes.POINTER(ctypes.c_int32)]
    lib.nsp_attn_kv_queues.restype = i32
    lib.nsp_executor_step.argtypes = [wl, ctypes.POINTER(ctypes.c_int32), i32, i32, f32,
                                      ctypes.POINTER(CStepBuffers), p, p]
    lib.nsp_executor_step.restype = i32
    pp, i64p = ctypes.POINTER(CPlanParams), ctypes.POINTER(ctypes.c_int64)
    i32p, dp = ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double)
    lib.nsp_sp_tree_plan.argtypes = [pp, i64p, i32, i32p, i32p, dp, dp, dp]
    lib.nsp_sp_tree_plan.restype = i32
    lib.nsp_sp_tree_worklist.argtypes = [pp, i64p, i32, i32p, i32p, i32, i32p, i32p, i32p, i32p, i32p, i32p]
    lib.nsp_sp_tree_worklist.restype = i32
    lib.nsp_status_string.argtypes = [i32]
    lib.nsp_status_string.restype = ctypes.c_char_p
    lib.nsp_last_error.argtypes = []
    lib.nsp_last_error.restype = ctypes.c_char_p
    lib.nsp_version.argtypes = []
    lib.nsp_version.restype = ctypes.c_char_p
    lib.nsp_timing_enable.argtypes = [i32]
    lib.nsp_timing_enable.restype = i32
    lib.nsp_timing_reset.argtypes = []
    lib.nsp_timing_reset.restype = i32
    lib.nsp_timing_query.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_int64),
                                     ctypes.POINTER(ctypes.c_double)]
    lib.nsp_timing_query.restype = i32
    lib.nsp_mfma_ceiling.argtypes = [i32, i32, i32, ctypes.c_int64, ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(ctypes.c_double)]
    lib.nsp_mfma_ceiling.restype = i32
    _lib = lib
    return lib


class _WL:
    """Keeps the int32 arrays behind a CWorkList alive for the call."""

    def __init__(self, wl, with_sp: bool = True):
        self.cu = np.ascontiguousarray(wl.cu_seqlens, dtype=np.int32)
        self.qh = np.ascontiguousarray(wl.q_heads, dtype=np.int32).reshape(-1)
        self.kvh = np.ascontiguousarray(wl.kv_heads, dtype=np.int32).reshape(-1)
        self.sp = np.ascontiguousarray(wl.sp, dtype=np.int32) if with_sp and wl.sp is not None else None
        mask = getattr(wl, "item_mask", None)
        self.mask = None if mask is None else np.ascontiguousarray(np.asarray(mask) != 0, dtype=np.uint8)
        ip = ctypes.POINTER(ctypes.c_int32)
        bp = ctypes.POINTER(ctypes.c_uint8)
        self.c = CWorkList(
            n_items=int(wl.n_items),
            cu_seqlens=self.cu.ctypes.data_as(ip),
            q_heads=self.qh.ctypes.data_as(ip),
            kv_heads=self.kvh.ctypes.data_as(ip),
            sp=self.sp.ctypes.data_as(ip) if self.sp is not None else ip(),
            hq_total=int(wl.hq_total),
            hkv_total=int(wl.hkv_total),
            head_dim=int(wl.head_dim),
            item_mask=self.mask.ctypes.data_as(bp) if self.mask is not None else bp(),
        )

    @property
    def ref(self):
        return ctypes.byref(self.c)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _dtype_code(t, default=NSP_BF16) -> int:
    import torch
    if t is None:
        return default
    if t.dtype == torch.bfloat16:
        return NSP_BF16
    if t.dtype == torch.float32:
        return NSP_F32
    raise TypeError(f"unsupported dtype {t.dtype} (bfloat16 or float32)")


def _check(status: int, call: str):
    if status != NSP_OK:
        lib = load_library()
        raise NspError(status, call, lib.nsp_last_error().decode())


def status_string(status: int) -> str:
    return load_library().nsp_status_string(status).decode()


def version() -> str:
    return load_library().nsp_version().decode()


def nsp_varlen_attn_fwd(wl, q, k, v, o, lse, softmax_scale: float, causal: int = 1, stream=None):
    """Attention forward into o (bf16 or float32) and lse (float32)."""
    lib = load_library()
    w = _WL(wl, with_sp=False)
    st = lib.nsp_varlen_attn_fwd(w.ref, float(softmax_scale), int(causal), _ptr(q), _ptr(k), _ptr(v),
                                 _ptr(o), _dtype_code(o), _ptr(lse), _stream(stream))
    _check(st, "nsp_varlen_attn_fwd")


def nsp_varlen_attn_bwd_workspace(wl) -> int:
    lib = load_library()
    return int(lib.nsp_varlen_attn_bwd_workspace(_WL(wl, with_sp=False).ref))


def nsp_varlen_attn_bwd(wl, q, k, v, o, dout, lse, dq, dk, dv, workspace, softmax_scale: float,
                        causal: int = 1, stream=None):
    """Attention backward into dq, dk, dv (all bf16 or all float32)."""
    lib = load_library()
    w = _WL(wl, with_sp=False)
    gcode = _dtype_code(dq)
    if _dtype_code(dk) != gcode or _dtype_code(dv) != gcode:
        raise TypeError("dq, dk, dv must share one dtype")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.nsp_varlen_attn_bwd(w.ref, float(softmax_scale), int(causal), _ptr(q), _ptr(k), _ptr(v),
                                 _ptr(o), _dtype_code(o), _ptr(dout), _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv),
                                 gcode, _ptr(workspace), ws_bytes, _stream(stream))
    _check(st, "nsp_varlen_attn_bwd")


NSP_NOALLOC_SCRATCH_BYTES = 96 << 20
NSP_NOALLOC_MAX_ROWS = 11534272


def nsp_varlen_attn_bwd_noalloc(wl, q, k, v, o, dout, lse, dq, dk, dv, softmax_scale: float,
                                causal: int = 1, stream=None):
    """Attention backward without a workspace (the library's device scratch):
    allocates nothing on the device.  Calls overlapping in time on one GPU race."""
    lib = load_library()
    w = _WL(wl, with_sp=False)
    gcode = _dtype_code(dq)
    if _dtype_code(dk) != gcode or _dtype_code(dv) != gcode:
        raise TypeError("dq, dk, dv must share one dtype")
    st = lib.nsp_varlen_attn_bwd_noalloc(w.ref, float(softmax_scale), int(causal), _ptr(q), _ptr(k), _ptr(v),
                                         _ptr(o), _dtype_code(o), _ptr(dout), _ptr(lse), _ptr(dq), _ptr(dk),
                                         _ptr(dv), gcode, _stream(stream))
    _check(st, "nsp_varlen_attn_bwd_noalloc")


def nsp_ulysses_pack(wl, kind: int, x_seq, x_head, stream=None):
    lib = load_library()
    st = lib.nsp_ulysses_pack(_WL(wl).ref, int(kind), _dtype_code(x_seq), _ptr(x_seq), _ptr(x_head),
                              _stream(stream))
    _check(st, "nsp_ulysses_pack")


def nsp_ulysses_unpack(wl, kind: int, replica: int, x_head, x_seq, stream=None):
    lib = load_library()
    st = lib.nsp_ulysses_unpack(_WL(wl).ref, int(kind), _dtype_code(x_head), int(replica), _ptr(x_head),
                                _ptr(x_seq), _stream(stream))
    _check(st, "nsp_ulysses_unpack")


def nsp_recompute_plan(wl, budget_bytes: int, o_dtype: int = NSP_BF16):
    """SAVE (1) / RECOMPUTE (0) marks per item and the saved bytes (host only)."""
    lib = load_library()
    w = _WL(wl)
    save = np.zeros(max(1, wl.n_items), dtype=np.uint8)
    saved = ctypes.c_int64(0)
    st = lib.nsp_recompute_plan(w.ref, int(budget_bytes), int(o_dtype),
                                save.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), ctypes.byref(saved))
    _check(st, "nsp_recompute_plan")
    return save[:wl.n_items].copy(), int(saved.value)


NSP_SCHED_FWD, NSP_SCHED_KV = 0, 1


def nsp_attn_schedule(wl, which: int) -> np.ndarray:
    """The attention units in launch order (host only), int32 [n, 4]:
    forward / dQ (which=NSP_SCHED_FWD) rows (item, q tile, local q head, local
    KV head); dK/dV (NSP_SCHED_KV) rows (item, key tile | desc << 30,
    i0 | i1 << 16, local KV head), the per-XCD queues one after another."""
    lib = load_library()
    w = _WL(wl)
    n = ctypes.c_int64(0)
    i32p = ctypes.POINTER(ctypes.c_int32)
    _check(lib.nsp_attn_schedule(w.ref, int(which), ctypes.cast(None, i32p), 0, ctypes.byref(n)),
           "nsp_attn_schedule")
    out = np.zeros((max(1, n.value), 4), dtype=np.int32)
    _check(lib.nsp_attn_schedule(w.ref, int(which), out.ctypes.data_as(i32p), n.value, ctypes.byref(n)),
           "nsp_attn_schedule")
    return out[:n.value].copy()


def nsp_attn_kv_queues(wl) -> np.ndarray:
    """Start of each XCD's dK/dV queue in nsp_attn_schedule(wl, NSP_SCHED_KV),
    and the unit count: int32 [9]."""
    lib = load_library()
    w = _WL(wl)
    out = np.zeros(9, dtype=np.int32)
    _check(lib.nsp_attn_kv_queues(w.ref, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))),
           "nsp_attn_kv_queues")
    return out


def nsp_executor_step(wl, buffers: dict, softmax_scale: float, node_sp=None,
                      phases: int = NSP_STEP_FORWARD | NSP_STEP_BACKWARD, compute=None, comm=None):
    """Phase-streamed attention step over the SP-tree nodes (see include/nsp.h).

    buffers: torch tensors named as the fields of nsp_step_buffers (q_seq ...
    dv_seq, q ... dv, lse, workspace); missing ones are passed as NULL.
    compute/comm: torch streams (default: the current stream for both).
    """
    lib = load_library()
    w = _WL(wl)
    b = CStepBuffers()
    for name, _ in CStepBuffers._fields_[:-1]:
        setattr(b, name, _ptr(buffers.get(name)))
    ws = buffers.get("workspace")
    b.ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    order = None if node_sp is None else np.ascontiguousarray(node_sp, dtype=np.int32)
    optr = order.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)) if order is not None else None
    cs = _stream(compute)
    ms = cs if comm is None else _stream(comm)
    st = lib.nsp_executor_step(w.ref, optr, 0 if order is None else int(order.size), int(phases),
                               float(softmax_scale), ctypes.byref(b), cs, ms)
    _check(st, "nsp_executor_step")


def nsp_sp_tree_plan(params: SpTreeParams, lengths):
    """SP-tree plan of a batch (host only): (node_depth, node_index, C_p,
    Tok_p, load)."""
    lib = load_library()
    L = np.ascontiguousarray(lengths, dtype=np.int64)
    n = int(L.size)
    depth = np.zeros(max(1, n), dtype=np.int32)
    index = np.zeros(max(1, n), dtype=np.int32)
    cost = np.zeros(params.world, dtype=np.float64)
    tok = np.zeros(params.world, dtype=np.float64)
    load = ctypes.c_double(0.0)
    i32p, dp = ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double)
    c = params.c()
    st = lib.nsp_sp_tree_plan(ctypes.byref(c), L.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), n,
                              depth.ctypes.data_as(i32p), index.ctypes.data_as(i32p), cost.ctypes.data_as(dp),
                              tok.ctypes.data_as(dp), ctypes.byref(load))
    _check(st, "nsp_sp_tree_plan")
    return depth[:n].copy(), index[:n].copy(), cost, tok, float(load.value)


def nsp_sp_tree_worklist(params: SpTreeParams, lengths, node_depth, node_index, gpu: int):
    """GPU `gpu`'s work list under a plan: (WorkList, sample index per item)."""
    from .workloads import WorkList
    lib = load_library()
    L = np.ascontiguousarray(lengths, dtype=np.int64)
    n = int(L.size)
    d = np.ascontiguousarray(node_depth, dtype=np.int32)
    i = np.ascontiguousarray(node_index, dtype=np.int32)
    m = ctypes.c_int32(0)
    cap = max(1, n)
    sample = np.zeros(cap, dtype=np.int32)
    cu = np.zeros(cap + 1, dtype=np.int32)
    qh = np.zeros(2 * cap, dtype=np.int32)
    kvh = np.zeros(2 * cap, dtype=np.int32)
    sp = np.zeros(cap, dtype=np.int32)
    ip = ctypes.POINTER(ctypes.c_int32)
    c = params.c()
    st = lib.nsp_sp_tree_worklist(ctypes.byref(c), L.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), n,
                                  d.ctypes.data_as(ip), i.ctypes.data_as(ip), int(gpu), ctypes.byref(m),
                                  sample.ctypes.data_as(ip), cu.ctypes.data_as(ip), qh.ctypes.data_as(ip),
                                  kvh.ctypes.data_as(ip), sp.ctypes.data_as(ip))
    _check(st, "nsp_sp_tree_worklist")
    k = int(m.value)
    wl = WorkList(lengths=np.diff(cu[:k + 1]).astype(np.int64), sp=sp[:k].astype(np.int64),
                  q_heads=qh[:2 * k].reshape(k, 2).astype(np.int64), kv_heads=kvh[:2 * k].reshape(k, 2).astype(np.int64),
                  hq_total=params.hq_total, hkv_total=params.hkv_total, head_dim=params.head_dim)
    return wl, sample[:k].copy()


KERNELS = ("attn_fwd", "bwd_preprocess", "bwd_dkdv", "bwd_dq", "relayout")


def nsp_timing_enable(enable: bool = True):
    _check(load_library().nsp_timing_enable(int(bool(enable))), "nsp_timing_enable")


def nsp_timing_reset():
    _check(load_library().nsp_timing_reset(), "nsp_timing_reset")


def nsp_timing_query(kernel: str):
    """(launches, total_ms) of one kernel since the last reset."""
    n = ctypes.c_int64(0)
    ms = ctypes.c_double(0.0)
    _check(load_library().nsp_timing_query(kernel.encode(), ctypes.byref(n), ctypes.byref(ms)),
           "nsp_timing_query")
    return int(n.value), float(ms.value)


def nsp_mfma_ceiling(pattern: int = 0, zero_operands: bool = False, waves_per_simd: int = 1,
                     products_per_simd: int = 1 << 21):
    """(seconds, TFLOP/s) of the device's matrix cores issuing bf16 products
    only (the power-limited ceiling; see the header).  Synchronous."""
    sec = ctypes.c_double(0.0)
    tf = ctypes.c_double(0.0)
    _check(load_library().nsp_mfma_ceiling(int(pattern), int(bool(zero_operands)), int(waves_per_simd),
                                           int(products_per_simd), ctypes.byref(sec), ctypes.byref(tf)),
           "nsp_mfma_ceiling")
    return float(sec.value), float(tf.value)


# ------------------------------------------------------------ allocation --

def alloc_like_worklist(wl, device="cuda", o_dtype=None, grad_dtype=None):
    """Empty output buffers for a work list: o, lse, dq, dk, dv, workspace."""
    import torch
    o_dtype = o_dtype or torch.bfloat16
    grad_dtype = grad_dtype or torch.bfloat16
    qe, ke, le = wl.q_elems(), wl.kv_elems(), wl.lse_elems()
    ws = nsp_varlen_attn_bwd_workspace(wl)
    return dict(
        o=torch.empty(qe, dtype=o_dtype, device=device),
        lse=torch.empty(le, dtype=torch.float32, device=device),
        dq=torch.empty(qe, dtype=grad_dtype, device=device),
        dk=torch.empty(ke, dtype=grad_dtype, device=device),
        dv=torch.empty(ke, dtype=grad_dtype, device=device),
        ws=torch.empty(max(ws, 256), dtype=torch.uint8, device=device),
    )


def to_device_bf16(bits: np.ndarray, device="cuda"):
    """Upload bf16 bit patterns (uint16) as a torch.bfloat16 tensor."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def bf16_to_numpy_bits(t) -> np.ndarray:
    """Download a torch.bfloat16 tensor as uint16 bit patterns."""
    import torch
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)
