"""Pins of the re-layout oracle (pack / unpack) against things other than itself.

  * the hand-written example in tests/golden (sp=2 query kind; replicated KV);
  * an element-by-element loop over the definition on an iota payload
    (every element is its own index, so any wrong index shows);
  * counting: each input element appears once (H >= sp) or sp/H times (H < sp);
  * unpack(pack(x)) = x, SELECT for replicated heads;
  * SUM of identical replicas equals an exact multiple;
  * a planted mistake (shard and head index swapped) is caught.
"""
import numpy as np
import pytest

from oracle import ulysses as U
from paper_2609_22755_amd.workloads import draw_bf16

from conftest import load_golden


def definitional_pack(x_seq, lengths, sp, H, D):
    """Loop over every destination element, straight from the definition."""
    T = sum(L // s for L, s in zip(lengths, sp))
    xs = np.asarray(x_seq).reshape(T, H, D)
    out = []
    c = 0
    for L, s in zip(lengths, sp):
        n = L // s
        hl = H // s if H >= s else 1
        for blk in range(s):
            for t in range(n):
                for hp in range(hl):
                    head = blk * hl + hp if H >= s else (blk * H) // s
                    for d in range(D):
                        out.append(xs[c + t, head, d])
        c += n
    return np.array(out, dtype=xs.dtype)


CASES = [
    ([8, 4, 12], [2, 1, 4], 8, 4),     # H >= sp, mixed degrees
    ([8, 16], [4, 8], 2, 3),           # H < sp: replicated heads
    ([6, 0, 10], [2, 1, 2], 4, 2),     # empty item
    ([32], [8], 32, 2),                # Qwen-like 32 heads at sp=8
]


def iota(n):
    return np.arange(n, dtype=np.int64)


@pytest.mark.parametrize("lengths,sp,H,D", CASES)
def test_pack_matches_definition_on_iota(lengths, sp, H, D):
    T = sum(L // s for L, s in zip(lengths, sp))
    x = iota(T * H * D)
    assert np.array_equal(U.pack(x, lengths, sp, H, D), definitional_pack(x, lengths, sp, H, D))


@pytest.mark.parametrize("lengths,sp,H,D", CASES)
def test_each_element_moved_the_right_number_of_times(lengths, sp, H, D):
    T = sum(L // s for L, s in zip(lengths, sp))
    x = iota(T * H * D)
    counts = np.bincount(U.pack(x, lengths, sp, H, D), minlength=x.size)
    c = 0
    for L, s in zip(lengths, sp):
        n = L // s
        blk = counts[c * H * D:(c + n) * H * D]
        if H >= s:
            assert np.all(blk == 1)
        else:
            per_head = blk.reshape(n, H, D)
            assert np.all(per_head == s // H)
        c += n


@pytest.mark.parametrize("lengths,sp,H,D", CASES)
def test_unpack_inverts_pack(lengths, sp, H, D):
    T = sum(L // s for L, s in zip(lengths, sp))
    x = draw_bf16(np.random.default_rng(3), T * H * D)
    y = U.pack(x, lengths, sp, H, D)
    assert y.dtype == np.uint16
    assert np.array_equal(U.unpack(y, lengths, sp, H, D, "select"), x)


def test_sum_of_identical_replicas_is_exact_multiple():
    lengths, sp, H, D = [16], [8], 2, 4          # 4 replicas per head
    x = draw_bf16(np.random.default_rng(4), 2 * H * D)
    y = U.pack(x, lengths, sp, H, D)
    s = U.unpack(y, lengths, sp, H, D, "sum")
    xf = (x.astype(np.uint32) << 16).view(np.float32)
    sf = (s.astype(np.uint32) << 16).view(np.float32)
    assert np.array_equal(sf, 4.0 * xf)         # x4 is exact in bf16


def test_sum_rounds_the_float32_sum_once():
    # two replicas 1.0 and 2^-8: f32 sum 1.00390625 lies exactly halfway
    # between bf16 neighbours 1.0 and 1.0078125 -> ties-to-even gives 1.0
    one, tiny = 0x3F80, 0x3B80
    y = np.array([one, tiny], dtype=np.uint16)   # L=2, sp=2, H=1, D=1 -> replicas
    s = U.unpack(y, [2], [2], 1, 1, "sum")
    assert s.tolist() == [0x3F80]
    y = np.array([0x3F81, tiny], dtype=np.uint16)  # 1.0078125 + 2^-8: tie -> even 1.015625
    assert U.unpack(y, [2], [2], 1, 1, "sum").tolist() == [0x3F82]
    f = np.array([1.5, 2.25], dtype=np.float32)   # float32 data: plain f32 sum
    assert U.unpack(f, [2], [2], 1, 1, "sum").tolist() == [3.75]


def test_golden_small_example():
    g = load_golden("ulysses_pack_small.txt")
    q_seq = np.array(g["q_seq"], dtype=np.int64)
    assert U.pack(q_seq, [4], [2], 4, 1).tolist() == [int(v) for v in g["q_head"]]
    assert U.unpack(np.array(g["q_head"], dtype=np.int64), [4], [2], 4, 1).tolist() == g["q_seq"]
    kv_seq = np.array(g["kv_seq"], dtype=np.int64)
    assert U.pack(kv_seq, [4], [4], 2, 1).tolist() == [int(v) for v in g["kv_head"]]


def test_planted_index_swap_is_caught(monkeypatch):
    def bad_pack(x_seq, lengths, sp, H, D):
        T = sum(L // s for L, s in zip(lengths, sp))
        xs = np.asarray(x_seq).reshape(T, H, D)
        out, c = [], 0
        for L, s in zip(lengths, sp):
            n = L // s
            hl = H // s
            y = xs[c:c + n].reshape(n, hl, s, D).transpose(2, 0, 1, 3)  # head = h'*sp + s
            out.append(y.reshape(-1))
            c += n
        return np.concatenate(out)

    monkeypatch.setattr(U, "pack", bad_pack)
    lengths, sp, H, D = CASES[0]
    T = sum(L // s for L, s in zip(lengths, sp))
    x = iota(T * H * D)
    assert not np.array_equal(U.pack(x, lengths, sp, H, D), definitional_pack(x, lengths, sp, H, D))


def definitional_unpack_sum(x_head, lengths, sp, H, D):
    """Replica sums by a loop over every destination element (H < sp items
    sum the blocks s with floor(s*H/sp) == g; H >= sp items invert pack)."""
    T = sum(L // s for L, s in zip(lengths, sp))
    out = np.zeros((T, H, D), dtype=np.float64)
    c = e = 0
    for L, s in zip(lengths, sp):
        n = L // s
        hl = H // s if H >= s else 1
        for blk in range(s):
            for t in range(n):
                for hp in range(hl):
                    for d in range(D):
                        v = x_head[e + ((blk * n + t) * hl + hp) * D + d]
                        if H >= s:
                            out[c + t, blk * hl + hp, d] = v
                        else:
                            out[c + t, (blk * H) // s, d] += v
        c += n
        e += L * hl * D
    return out.reshape(-1)


@pytest.mark.parametrize("lengths,sp,H,D", CASES)
def test_sum_of_float64_replicas_matches_definitional_loop(lengths, sp, H, D):
    """float64 reference data (an oracle gradient in the head layout) is
    summed over its replicas in float64, in the order of the definition."""
    E = sum(L * (H // s if H >= s else 1) * D for L, s in zip(lengths, sp))
    x = np.random.default_rng(12).standard_normal(E)
    got = U.unpack(x, lengths, sp, H, D, "sum")
    assert got.dtype == np.float64
    assert np.array_equal(got, definitional_unpack_sum(x, lengths, sp, H, D))
