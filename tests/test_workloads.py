"""The seeded generator reproduces the five work lists exactly.

The expected lists were derived independently from the length rule (lognormal
draws, clipping, truncation, the smallest-sp rule) when the configurations
were specified; their flop totals are the algorithmic counts
sum_j 14 * D * hq_j * L_j (L_j + 1) / 2.
"""
import numpy as np

from paper_2609_22755_amd import workloads as W


def test_tiny():
    w = W.make_config("tiny")
    assert w.wl.lengths.tolist() == [64, 128, 256, 512]
    assert w.wl.head_dim == 64 and w.wl.hq_total == 8 and w.wl.hkv_total == 2
    assert w.pack_wl.sp.tolist() == [2, 2, 2, 2]
    assert abs(w.softmax_scale - 0.125) < 1e-15


def test_short_sp1():
    wl = W.make_config("short_sp1").wl
    assert wl.n_items == 24 and int(wl.lengths.max()) == 7470 and int(wl.lengths.sum()) == 65536
    assert np.all(wl.sp == 1)
    assert abs(wl.flops_fwd() + wl.flops_bwd() - 6.91e12) / 6.91e12 < 2e-3


def test_nested_2level():
    wl = W.make_config("nested_2level").wl
    assert wl.lengths.tolist() == [131072, 4765, 2696, 2943, 581, 16384, 5399]
    assert wl.sp.tolist() == [8, 1, 1, 1, 1, 1, 1]
    assert wl.q_heads[0].tolist() == [0, 4] and wl.kv_heads[0].tolist() == [0, 1]
    assert abs(wl.flops_fwd() + wl.flops_bwd() - 7.12e13) / 7.12e13 < 2e-3


def test_longtail_4level():
    wl = W.make_config("longtail_4level").wl
    assert wl.n_items == 26 and wl.seq_tokens() == 262144
    items = set(zip(wl.lengths.tolist(), wl.sp.tolist()))
    assert {(262144, 8), (116320, 4), (61112, 2)} <= items
    for L, s, q, kv in zip(wl.lengths, wl.sp, wl.q_heads, wl.kv_heads):
        assert L % s == 0 and L // s <= 32768
        assert q[1] - q[0] == 32 // s and kv[1] - kv[0] == max(1, 4 // s)
    assert abs(wl.flops_fwd() + wl.flops_bwd() - 4.58e14) / 4.58e14 < 2e-3


def test_maxctx():
    w = W.make_config("maxctx_relayout")
    assert w.wl.lengths.tolist() == [393216] and w.wl.sp.tolist() == [8]
    assert w.wl.seq_tokens() == 49152
    assert w.seq_input


def test_chunked_draw_equals_one_draw():
    a = W.draw_bf16(np.random.default_rng(7), 100003, chunk=4096)
    b = W.f32_to_bf16_bits(np.random.default_rng(7).standard_normal(100003, dtype=np.float32))
    assert np.array_equal(a, b)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -8 + 2 ** -20], dtype=np.float32)
    bits = W.f32_to_bf16_bits(x)
    assert bits.tolist() == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x3F81]
    assert np.array_equal(W.bf16_bits_to_f32(bits)[[0, 3]], np.array([1.0, -2.5], dtype=np.float32))
