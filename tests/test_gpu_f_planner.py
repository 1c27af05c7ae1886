"""Planner to kernels: a batch is routed onto the SP tree by the native
planner (nsp_sp_tree_plan), GPU p's work list is taken from the plan
(nsp_sp_tree_worklist) -- items at several SP degrees, replicated KV heads
where the degree exceeds the KV head count -- and the attention forward and
backward of that work list on the HIP path match the oracle to the
tolerances of the attention tests; the phase-streamed step of the executor
on such a work list matches the plain calls bit for bit."""
import numpy as np
import pytest

from paper_2609_22755_amd import nsp
from paper_2609_22755_amd.workloads import draw_attention_inputs

from gpu_util import require_gpu
from test_gpu_a_parity import check_against_oracle

pytestmark = pytest.mark.gpu


def _plan():
    # a long-tail batch for 8 GPUs: a few long samples and many short ones
    lengths = np.array([2048, 1536, 1024, 512, 384, 200, 136, 96, 72, 64, 40, 32, 24, 16, 8, 1], dtype=np.int64)
    prm = nsp.SpTreeParams(world=8, sp_max=8, hq_total=8, hkv_total=2, head_dim=64, prefix=6, beam=4,
                           dense_fwd_per_token=2e-7, dense_bwd_per_token=4e-7)
    d, i, _, _, _ = nsp.nsp_sp_tree_plan(prm, lengths)
    return prm, lengths, d, i


@pytest.mark.parametrize("gpu", [0, 3, 6])
def test_planned_worklist_parity(gpu):
    require_gpu()
    prm, lengths, d, i = _plan()
    wl, sample = nsp.nsp_sp_tree_worklist(prm, lengths, d, i, gpu)
    print(f"[plan] gpu {gpu}: items (sample, L, sp, q, kv) "
          f"{[(int(s), int(L), int(p), tuple(q), tuple(k)) for s, L, p, q, k in zip(sample, wl.lengths, wl.sp, wl.q_heads.tolist(), wl.kv_heads.tolist())]}",
          flush=True)
    assert wl.n_items > 0 and len(set(wl.sp.tolist())) >= 2
    check_against_oracle(f"plan_gpu{gpu}", wl, draw_attention_inputs(wl, 500 + gpu), 1.0 / np.sqrt(64))


@pytest.mark.parametrize("gpu", [1, 5])
def test_planned_worklist_through_the_executor(gpu):
    """The phase-streamed step (nsp_executor_step, two queues) on a planned
    work list gives bitwise the results of the plain calls issued one after
    another."""
    import torch
    from test_gpu_e_executor import OUT, SCALE, bits, make_buffers, serial
    require_gpu()
    lengths = np.array([4096, 2048, 1536, 1024, 640, 512, 320, 256, 200, 128, 96, 64, 40, 24], dtype=np.int64)
    prm = nsp.SpTreeParams(world=8, sp_max=8, hq_total=32, hkv_total=4, head_dim=128, prefix=8, beam=4,
                           dense_fwd_per_token=2e-7, dense_bwd_per_token=4e-7)
    d, i, _, _, _ = nsp.nsp_sp_tree_plan(prm, lengths)
    wl, sample = nsp.nsp_sp_tree_worklist(prm, lengths, d, i, gpu)
    print(f"[plan] gpu {gpu}: samples {sample.tolist()} sp {wl.sp.tolist()}", flush=True)
    assert len(set(wl.sp.tolist())) >= 2
    ref = make_buffers(wl, 7 + gpu)
    serial(wl, ref)
    got = make_buffers(wl, 7 + gpu)
    nsp.nsp_executor_step(wl, got, SCALE, comm=torch.cuda.Stream())
    torch.cuda.synchronize()
    for n in OUT:
        assert np.array_equal(bits(ref[n]), bits(got[n])), n
