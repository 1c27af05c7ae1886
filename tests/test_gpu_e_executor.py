"""Inter-level phase streaming (Design, NSP Executor): the executor issues
each SP-tree node's prologue, compute and epilogue as item-masked calls on a
compute queue and a communication queue.  Its results must be bitwise those
of the plain calls issued one after another, whatever the issue order and
whether the two queues are distinct streams or one."""
import numpy as np
import pytest

from paper_2609_22755_amd import nsp
from paper_2609_22755_amd.workloads import draw_bf16, small_worklist

from gpu_util import require_gpu

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def bits(t):
    return nsp.bf16_to_numpy_bits(t) if str(t.dtype) == "torch.bfloat16" else t.cpu().numpy().view(np.uint32)


def make_buffers(wl, seed):
    import torch
    rng = np.random.default_rng(seed)
    T, D = wl.seq_tokens(), wl.head_dim
    dev = "cuda"
    b = dict(q_seq=nsp.to_device_bf16(draw_bf16(rng, T * wl.hq_total * D)),
             k_seq=nsp.to_device_bf16(draw_bf16(rng, T * wl.hkv_total * D)),
             v_seq=nsp.to_device_bf16(draw_bf16(rng, T * wl.hkv_total * D)),
             do_seq=nsp.to_device_bf16(draw_bf16(rng, T * wl.hq_total * D)))
    for n in ("o_seq", "dq_seq"):
        b[n] = torch.full((T * wl.hq_total * D,), float("nan"), dtype=torch.bfloat16, device=dev)
    for n in ("dk_seq", "dv_seq"):
        b[n] = torch.full((T * wl.hkv_total * D,), float("nan"), dtype=torch.bfloat16, device=dev)
    for n in ("q", "o", "dout", "dq"):
        b[n] = torch.full((wl.q_elems(),), float("nan"), dtype=torch.bfloat16, device=dev)
    for n in ("k", "v", "dk", "dv"):
        b[n] = torch.full((wl.kv_elems(),), float("nan"), dtype=torch.bfloat16, device=dev)
    b["lse"] = torch.full((wl.lse_elems(),), float("nan"), dtype=torch.float32, device=dev)
    b["workspace"] = torch.empty(max(256, nsp.nsp_varlen_attn_bwd_workspace(wl)), dtype=torch.uint8, device=dev)
    return b


def serial(wl, b):
    Q, KV = nsp.NSP_KIND_Q, nsp.NSP_KIND_KV
    nsp.nsp_ulysses_pack(wl, Q, b["q_seq"], b["q"])
    nsp.nsp_ulysses_pack(wl, KV, b["k_seq"], b["k"])
    nsp.nsp_ulysses_pack(wl, KV, b["v_seq"], b["v"])
    nsp.nsp_varlen_attn_fwd(wl, b["q"], b["k"], b["v"], b["o"], b["lse"], SCALE)
    nsp.nsp_ulysses_unpack(wl, Q, nsp.NSP_UNPACK_SELECT, b["o"], b["o_seq"])
    nsp.nsp_ulysses_pack(wl, Q, b["do_seq"], b["dout"])
    nsp.nsp_varlen_attn_bwd(wl, b["q"], b["k"], b["v"], b["o"], b["dout"], b["lse"], b["dq"], b["dk"], b["dv"],
                            b["workspace"], SCALE)
    nsp.nsp_ulysses_unpack(wl, Q, nsp.NSP_UNPACK_SELECT, b["dq"], b["dq_seq"])
    nsp.nsp_ulysses_unpack(wl, KV, nsp.NSP_UNPACK_SUM, b["dk"], b["dk_seq"])
    nsp.nsp_ulysses_unpack(wl, KV, nsp.NSP_UNPACK_SUM, b["dv"], b["dv_seq"])


OUT = ("o_seq", "dq_seq", "dk_seq", "dv_seq", "q", "k", "v", "o", "lse", "dout", "dq", "dk", "dv")


@pytest.mark.parametrize("order,two_streams", [(None, True), ([1, 2, 8, 4], True), (None, False)])
def test_executor_matches_serial_calls(order, two_streams):
    import torch
    wl = small_worklist([1024, 512, 300, 4096, 96, 64, 2048], 32, 4, 128, sp=[8, 1, 1, 4, 2, 1, 2])
    ref = make_buffers(wl, 5)
    serial(wl, ref)
    got = make_buffers(wl, 5)
    comm = torch.cuda.Stream() if two_streams else None
    nsp.nsp_executor_step(wl, got, SCALE, node_sp=order, comm=comm)
    torch.cuda.synchronize()
    for n in OUT:
        assert np.array_equal(bits(ref[n]), bits(got[n])), n


def test_executor_forward_then_backward_separately():
    import torch
    wl = small_worklist([256, 128, 512], 32, 4, 128, sp=[2, 1, 8])
    ref = make_buffers(wl, 6)
    serial(wl, ref)
    got = make_buffers(wl, 6)
    comm = torch.cuda.Stream()
    nsp.nsp_executor_step(wl, got, SCALE, phases=nsp.NSP_STEP_FORWARD, comm=comm)
    nsp.nsp_executor_step(wl, got, SCALE, phases=nsp.NSP_STEP_BACKWARD, comm=comm)
    torch.cuda.synchronize()
    for n in OUT:
        assert np.array_equal(bits(ref[n]), bits(got[n])), n
