"""Guard bands around every output of the attention and re-layout calls.

Each output tensor (O, LSE, dQ, dK, dV, the backward workspace, pack and
unpack destinations) is the middle of a larger device buffer whose bytes
before and after it hold a seeded random pattern.  After the calls every
guard byte must still hold its pattern (no write past either end of a
buffer), and the results must equal, bit for bit, those of the same calls on
plain allocations (the kernels do not depend on where a buffer lies).
Ragged lengths put partial tiles at the end of every item, including the
last one, whose tail rows sit next to the trailing guard.
"""
import numpy as np
import pytest

from paper_2609_22755_amd import nsp
from paper_2609_22755_amd.workloads import draw_attention_inputs, draw_bf16, small_worklist

from gpu_util import require_gpu, run_attention

pytestmark = pytest.mark.gpu

GUARD = 64 << 10   # bytes on each side (a multiple of every alignment the calls ask for)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


class Guarded:
    """Device buffers with random guard bytes on both sides of each."""

    def __init__(self, seed):
        self.rng = np.random.default_rng(seed)
        self.bufs = []

    def alloc(self, n, dtype):
        import torch
        nbytes = n * torch.empty((), dtype=dtype).element_size()
        pattern = self.rng.integers(0, 256, nbytes + 2 * GUARD, dtype=np.uint8)
        raw = torch.from_numpy(pattern).cuda()
        self.bufs.append((raw, pattern, nbytes))
        return raw[GUARD:GUARD + nbytes].view(dtype)

    def check(self):
        for raw, pattern, nbytes in self.bufs:
            got = raw.cpu().numpy()
            assert np.array_equal(got[:GUARD], pattern[:GUARD]), "write before the start of a buffer"
            assert np.array_equal(got[GUARD + nbytes:], pattern[GUARD + nbytes:]), "write past the end of a buffer"


CASES = {
    # name: (lengths, sp, ranks, hq_total, hkv_total, head_dim)
    "ragged_d128": ([65, 300, 0, 517, 1, 129], None, None, 8, 2, 128),
    "ragged_d64": ([31, 129, 300, 77], None, None, 8, 2, 64),
    "mixed_sp": ([256, 520, 1000, 77], [1, 2, 4, 1], [0, 1, 2, 0], 32, 4, 128),
}


def _bits(t):
    import torch
    return t.detach().view(torch.int16 if t.element_size() == 2 else torch.int32).cpu().numpy()


@pytest.mark.parametrize("name", sorted(CASES))
@pytest.mark.parametrize("f32", [False, True])
def test_attention_outputs_guarded(name, f32):
    import torch
    lengths, sp, ranks, hq, hkv, D = CASES[name]
    wl = small_worklist(lengths, hq, hkv, D, sp=sp, rank=ranks)
    qb, kb, vb, dob = draw_attention_inputs(wl, 5 + len(name))
    scale = 1.0 / np.sqrt(D)
    dt = torch.float32 if f32 else torch.bfloat16
    want = run_attention(wl, qb, kb, vb, dob, scale, o_dtype=dt, g_dtype=dt)

    g = Guarded(17 + len(name) + int(f32))
    q, k, v, do = (nsp.to_device_bf16(x) for x in (qb, kb, vb, dob))
    qe, ke, le = wl.q_elems(), wl.kv_elems(), wl.lse_elems()
    out = dict(o=g.alloc(qe, dt), lse=g.alloc(le, torch.float32), dq=g.alloc(qe, dt), dk=g.alloc(ke, dt),
               dv=g.alloc(ke, dt))
    ws = g.alloc(max(nsp.nsp_varlen_attn_bwd_workspace(wl), 256), torch.uint8)
    nsp.nsp_varlen_attn_fwd(wl, q, k, v, out["o"], out["lse"], scale)
    nsp.nsp_varlen_attn_bwd(wl, q, k, v, out["o"], do, out["lse"], out["dq"], out["dk"], out["dv"], ws, scale)
    torch.cuda.synchronize()
    g.check()
    for key in ("o", "lse", "dq", "dk", "dv"):
        assert np.array_equal(_bits(out[key]), _bits(want[key])), f"{name}: {key} depends on its placement"


@pytest.mark.parametrize("kind", [nsp.NSP_KIND_Q, nsp.NSP_KIND_KV])
def test_relayout_outputs_guarded(kind):
    import torch
    wl = small_worklist([256, 520, 1000, 384, 8], 32, 4, 128, sp=[1, 2, 4, 8, 8])
    H = wl.hq_total if kind == nsp.NSP_KIND_Q else wl.hkv_total
    n_seq = wl.seq_tokens() * H * wl.head_dim
    n_head = wl.q_elems() if kind == nsp.NSP_KIND_Q else wl.kv_elems()
    x = nsp.to_device_bf16(draw_bf16(np.random.default_rng(3 + kind), n_seq))
    y = nsp.to_device_bf16(draw_bf16(np.random.default_rng(9 + kind), n_head))
    g = Guarded(29 + kind)
    packed = g.alloc(n_head, torch.bfloat16)
    sel = g.alloc(n_seq, torch.bfloat16)
    summed = g.alloc(n_seq, torch.bfloat16)
    nsp.nsp_ulysses_pack(wl, kind, x, packed)
    nsp.nsp_ulysses_unpack(wl, kind, nsp.NSP_UNPACK_SELECT, y, sel)
    nsp.nsp_ulysses_unpack(wl, kind, nsp.NSP_UNPACK_SUM, y, summed)
    torch.cuda.synchronize()
    g.check()
    ref = torch.empty(n_head, dtype=torch.bfloat16, device="cuda")
    nsp.nsp_ulysses_pack(wl, kind, x, ref)
    assert np.array_equal(_bits(packed), _bits(ref))
    for mode, got in ((nsp.NSP_UNPACK_SELECT, sel), (nsp.NSP_UNPACK_SUM, summed)):
        r = torch.empty(n_seq, dtype=torch.bfloat16, device="cuda")
        nsp.nsp_ulysses_unpack(wl, kind, mode, y, r)
        assert np.array_equal(_bits(got), _bits(r))
