"""HIP path vs the fp64 oracle, element by element, through the C ABI.

Sizes are those the oracle finishes in seconds while still spanning several
tiles (256-row query tiles, 64-key forward tiles, 128-key dK/dV units) and
ragged tails.  The "many_units" cases hold several times more dK/dV units
than the chip has compute units, so every persistent dK/dV workgroup runs
several units in turn and takes units from other XCDs' queues.
Bars: attention forward rel-L2 <= 5e-3 and max-abs <= 1e-2 (float32 O; a
bf16 O must equal the float32 O rounded to nearest even, bit for bit);
gradients rel-L2 <= 1e-2; pack/unpack bit-exact.
"""
import numpy as np
import pytest

from oracle import ulysses as OU
from paper_2609_22755_amd import nsp
from paper_2609_22755_amd.workloads import (draw_attention_inputs, draw_bf16, make_config,
                                            small_worklist)

from gpu_util import (FWD_MAX_ABS, FWD_REL_L2, GRAD_REL_L2, LSE_MAX_ABS, max_abs, oracle_full, rel_l2,
                      report, require_gpu, run_attention, to_np)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def rne_f32_to_bf16_bits(x):
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


ATTN_CASES = {
    # name: (lengths, sp, ranks, hq_total, hkv_total, head_dim)
    "ragged_d128": ([1, 2, 63, 64, 65, 127, 128, 129, 200, 333, 0, 517], None, None, 8, 2, 128),
    "ragged_d64": ([1, 31, 64, 100, 129, 256, 300], None, None, 8, 2, 64),
    "mixed_sp_qwen": ([256, 520, 1000, 384, 77], [1, 2, 4, 8, 1], [0, 1, 2, 5, 0], 32, 4, 128),
    "mha_d128": ([130, 255], None, None, 4, 4, 128),
    # 150 items x 4 KV heads = 600 dK/dV units of one 128-key tile each
    "many_units_l128": ([128] * 150, None, None, 32, 4, 128),
    # 60 ragged items up to 800 tokens: ~850 dK/dV units of unequal length
    "many_units_ragged": ([int(x) for x in np.random.default_rng(77).integers(1, 800, 60)], None, None,
                          32, 4, 128),
    # single items, whose dK/dV schedules leave key tiles unpaired: an odd
    # number of key tiles (a middle tile) at sp = 8 with one KV head, and a
    # D = 64 item with two KV heads
    "single_item_odd_tiles": ([1152], [8], [0], 32, 4, 128),
    "single_item_d64": ([2048], None, None, 8, 2, 64),
}


def _case_wl(name):
    lengths, sp, ranks, hq, hkv, D = ATTN_CASES[name]
    return small_worklist(lengths, hq, hkv, D, sp=sp, rank=ranks)


def check_against_oracle(name, wl, inputs, scale):
    import torch
    ref = oracle_full(wl, *inputs, scale)
    g32 = run_attention(wl, *inputs, scale, o_dtype=torch.float32, g_dtype=torch.float32)
    g16 = run_attention(wl, *inputs, scale)
    o32, o16 = to_np(g32["o"]), to_np(g16["o"])
    errs = dict(o_rel=rel_l2(o32, ref["o"]), o_max=max_abs(o32, ref["o"]), o16_rel=rel_l2(o16, ref["o"]),
                o16_max=max_abs(o16, ref["o"]), lse_max=max_abs(to_np(g32["lse"]), ref["lse"]))
    for gname in ("dq", "dk", "dv"):
        errs[gname + "_rel"] = rel_l2(to_np(g16[gname]), ref[gname])
        errs[gname + "32_rel"] = rel_l2(to_np(g32[gname]), ref[gname])
    report(name, **errs)
    assert errs["o_rel"] <= FWD_REL_L2 and errs["o_max"] <= FWD_MAX_ABS
    assert errs["o16_rel"] <= FWD_REL_L2
    assert errs["lse_max"] <= LSE_MAX_ABS
    for gname in ("dq", "dk", "dv"):
        assert errs[gname + "_rel"] <= GRAD_REL_L2 and errs[gname + "32_rel"] <= GRAD_REL_L2
    # the bf16 store is the float32 result rounded to nearest even
    assert np.array_equal(nsp.bf16_to_numpy_bits(g16["o"]),
                          rne_f32_to_bf16_bits(g32["o"].cpu().numpy()))
    assert np.array_equal(g16["lse"].cpu().numpy(), g32["lse"].cpu().numpy())


def test_tiny_config_parity():
    w = make_config("tiny")
    check_against_oracle("tiny", w.wl, w.attention_inputs(), w.softmax_scale)


@pytest.mark.parametrize("name", sorted(ATTN_CASES))
def test_small_case_parity(name):
    wl = _case_wl(name)
    check_against_oracle(name, wl, draw_attention_inputs(wl, 100 + len(name)), 1.0 / np.sqrt(wl.head_dim))


# ------------------------------------------------------------ re-layout --

RELAYOUT_CASES = {
    # name: (lengths, sp, hq_total, hkv_total, head_dim)
    "tiny_sp2": ([64, 128, 256, 512], [2, 2, 2, 2], 8, 2, 64),
    "mixed_qwen": ([256, 520, 1000, 384, 8], [1, 2, 4, 8, 8], 32, 4, 128),
    "replicated_d64": ([64, 0, 32], [8, 4, 2], 16, 2, 64),
}


def _relayout_wl(name):
    lengths, sp, hq, hkv, D = RELAYOUT_CASES[name]
    return small_worklist(lengths, hq, hkv, D, sp=sp)


@pytest.mark.parametrize("name", sorted(RELAYOUT_CASES))
@pytest.mark.parametrize("kind", [nsp.NSP_KIND_Q, nsp.NSP_KIND_KV])
def test_pack_unpack_bit_exact(name, kind):
    import torch
    wl = _relayout_wl(name)
    H = wl.hq_total if kind == nsp.NSP_KIND_Q else wl.hkv_total
    D = wl.head_dim
    n_seq = wl.seq_tokens() * H * D
    x = draw_bf16(np.random.default_rng(7 + kind), n_seq)
    want = OU.pack(x, wl.lengths, wl.sp, H, D)
    xs = nsp.to_device_bf16(x)
    xh = torch.empty(want.size, dtype=torch.bfloat16, device="cuda")
    nsp.nsp_ulysses_pack(wl, kind, xs, xh)
    got = nsp.bf16_to_numpy_bits(xh)
    assert np.array_equal(got, want)
    # unpack: SELECT inverts pack; SUM of replicas against the oracle
    for mode, oname in ((nsp.NSP_UNPACK_SELECT, "select"), (nsp.NSP_UNPACK_SUM, "sum")):
        yh = draw_bf16(np.random.default_rng(11 + kind + mode), want.size)
        ys = torch.empty(n_seq, dtype=torch.bfloat16, device="cuda")
        nsp.nsp_ulysses_unpack(wl, kind, mode, nsp.to_device_bf16(yh), ys)
        assert np.array_equal(nsp.bf16_to_numpy_bits(ys), OU.unpack(yh, wl.lengths, wl.sp, H, D, oname))
    back = torch.empty(n_seq, dtype=torch.bfloat16, device="cuda")
    nsp.nsp_ulysses_unpack(wl, kind, nsp.NSP_UNPACK_SELECT, xh, back)
    assert np.array_equal(nsp.bf16_to_numpy_bits(back), x)


@pytest.mark.parametrize("name", ["mixed_qwen", "replicated_d64"])
def test_pack_unpack_f32(name):
    import torch
    wl = _relayout_wl(name)
    H, D = wl.hkv_total, wl.head_dim
    n_seq = wl.seq_tokens() * H * D
    x = np.random.default_rng(3).standard_normal(n_seq).astype(np.float32)
    want = OU.pack(x, wl.lengths, wl.sp, H, D)
    xh = torch.empty(want.size, dtype=torch.float32, device="cuda")
    nsp.nsp_ulysses_pack(wl, nsp.NSP_KIND_KV, torch.from_numpy(x).cuda(), xh)
    assert np.array_equal(xh.cpu().numpy(), want)
    ys = torch.empty(n_seq, dtype=torch.float32, device="cuda")
    y = np.random.default_rng(4).standard_normal(want.size).astype(np.float32)
    nsp.nsp_ulysses_unpack(wl, nsp.NSP_KIND_KV, nsp.NSP_UNPACK_SUM, torch.from_numpy(y).cuda(), ys)
    assert np.array_equal(ys.cpu().numpy(), OU.unpack(y, wl.lengths, wl.sp, H, D, "sum"))


def test_pack_iota_payload_every_index():
    """Each 16-bit element carries its own index (mod 2^16): any wrong index shows."""
    import torch
    wl = _relayout_wl("mixed_qwen")
    H, D = wl.hq_total, wl.head_dim
    n_seq = wl.seq_tokens() * H * D
    x = (np.arange(n_seq) % 65521).astype(np.uint16)   # prime modulus: no short period
    want = OU.pack(x, wl.lengths, wl.sp, H, D)
    xh = torch.empty(want.size, dtype=torch.bfloat16, device="cuda")
    nsp.nsp_ulysses_pack(wl, nsp.NSP_KIND_Q, nsp.to_device_bf16(x), xh)
    assert np.array_equal(nsp.bf16_to_numpy_bits(xh), want)
