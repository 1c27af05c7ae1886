"""Seeded synthetic work lists and tensors for the per-GPU NSP hot path.

This module is shared by the HIP path's tests/bench and by the CPU oracle's
tests. It holds none of the method's arithmetic: it only draws sequence
lengths, assigns Ulysses degrees and head ranges, and draws N(0,1) tensors,
rounded to bfloat16 bit patterns (uint16).

Workload shapes stand in for the paper's length traces (Evaluation, datasets:
long-tailed corpora, 94% of samples under 8K tokens, a few beyond 128K) and
for its Qwen3-MoE models (32 query heads, 4 KV heads, head_dim 128).  A
per-GPU share of an SP tree (Design, Definition 1) holds long sequences
head-sharded at degree sp (this GPU keeps Hq/sp query heads and
max(1, Hkv/sp) KV heads over the full length) and short sequences whole at
sp=1.

Generation rules (every step is seeded; numpy PCG64 via default_rng(seed)):
  * lengths: L = clip(rint(lognormal(mu, sigma)), lo, hi), drawn one at a
    time; when adding an item would pass the token target, the last item is
    truncated to the remainder so that the total is exact; items with sp>1
    have L rounded down to a multiple of sp;
  * tensors: after the lengths, Q, K, V, dO are drawn in that order as
    float32 standard normals in buffer order and rounded to bf16 (round to
    nearest even); tensors in the sequence-sharded layout (for pack/unpack)
    are drawn after those.
  * head ranges: this GPU is rank 0 of each item's SP group, i.e. query heads
    [0, Hq/sp) and KV heads [0, max(1, Hkv/sp)).
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import List, Optional, Sequence

import numpy as np

__all__ = [
    "WorkList",
    "Workload",
    "f32_to_bf16_bits",
    "bf16_bits_to_f32",
    "make_config",
    "CONFIG_NAMES",
    "make_worklist",
    "draw_bf16",
]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); return uint16 bits.

    Inputs are finite draws from N(0,1); NaN/Inf handling is not needed.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def draw_bf16(rng: np.random.Generator, n: int, chunk: int = 1 << 24) -> np.ndarray:
    """Draw n float32 standard normals in order and round each to bf16 bits.

    Drawn in chunks to bound peak memory; the values are the same as one
    draw of size n (the generator is consumed sequentially).
    """
    out = np.empty(n, dtype=np.uint16)
    pos = 0
    while pos < n:
        m = min(chunk, n - pos)
        out[pos:pos + m] = f32_to_bf16_bits(rng.standard_normal(m, dtype=np.float32))
        pos += m
    return out


@dataclasses.dataclass
class WorkList:
    """A per-GPU packed work list (attention layout), host arrays.

    lengths[j]  : L_j, tokens of item j in the head-sharded (attention) layout
    sp[j]       : Ulysses degree of item j's SP-tree node
    q_heads[j]  : [lo, hi) global query heads this GPU holds for item j
    kv_heads[j] : [lo, hi) global KV heads this GPU holds for item j
    """

    lengths: np.ndarray
    sp: np.ndarray
    q_heads: np.ndarray
    kv_heads: np.ndarray
    hq_total: int
    hkv_total: int
    head_dim: int
    # optional per-item selection passed to the library calls (None = all items)
    item_mask: Optional[np.ndarray] = None

    def select(self, mask) -> "WorkList":
        """The same work list (same layout) restricted to the items where mask != 0."""
        return dataclasses.replace(self, item_mask=np.asarray(mask, dtype=np.uint8).copy())

    @property
    def n_items(self) -> int:
        return int(self.lengths.shape[0])

    @property
    def cu_seqlens(self) -> np.ndarray:
        cu = np.zeros(self.n_items + 1, dtype=np.int32)
        cu[1:] = np.cumsum(self.lengths, dtype=np.int64).astype(np.int32)
        return cu

    @property
    def hq(self) -> np.ndarray:
        return (self.q_heads[:, 1] - self.q_heads[:, 0]).astype(np.int64)

    @property
    def hkv(self) -> np.ndarray:
        return (self.kv_heads[:, 1] - self.kv_heads[:, 0]).astype(np.int64)

    def q_elems(self) -> int:
        return int(np.sum(self.lengths.astype(np.int64) * self.hq)) * self.head_dim

    def kv_elems(self) -> int:
        return int(np.sum(self.lengths.astype(np.int64) * self.hkv)) * self.head_dim

    def lse_elems(self) -> int:
        return int(np.sum(self.lengths.astype(np.int64) * self.hq))

    def seq_tokens(self) -> int:
        """Tokens of the sequence-sharded layout: sum_j L_j / sp_j."""
        return int(np.sum(self.lengths.astype(np.int64) // self.sp.astype(np.int64)))

    def causal_pairs(self) -> np.ndarray:
        L = self.lengths.astype(np.int64)
        return L * (L + 1) // 2

    def flops_fwd(self) -> float:
        """Algorithmic forward flops: QK^T and PV over causal pairs."""
        return float(np.sum(4.0 * self.head_dim * self.hq * self.causal_pairs()))

    def flops_bwd(self) -> float:
        """Algorithmic backward flops: S recompute, dV, dP, dQ, dK over causal pairs."""
        return float(np.sum(10.0 * self.head_dim * self.hq * self.causal_pairs()))

    def digest(self) -> str:
        h = hashlib.sha256()
        for a in (self.lengths, self.sp, self.q_heads, self.kv_heads):
            h.update(np.ascontiguousarray(a, dtype=np.int64).tobytes())
        h.update(np.array([self.hq_total, self.hkv_total, self.head_dim], dtype=np.int64).tobytes())
        return h.hexdigest()[:16]


def make_worklist(lengths: Sequence[int], sp: Sequence[int], hq_total: int, hkv_total: int,
                  head_dim: int, rank: Optional[Sequence[int]] = None) -> WorkList:
    """Build a work list whose items are rank r (default 0) of their SP group.

    For degree sp, rank r holds query heads [r*Hq/sp, (r+1)*Hq/sp) and KV
    head block [r*Hkv/sp, (r+1)*Hkv/sp) when Hkv >= sp, else the single KV
    head floor(r*Hkv/sp) (replicated across sp/Hkv ranks).
    """
    n = len(lengths)
    lengths = np.asarray(lengths, dtype=np.int64)
    sp = np.asarray(sp, dtype=np.int64)
    rank = np.zeros(n, dtype=np.int64) if rank is None else np.asarray(rank, dtype=np.int64)
    qh = np.zeros((n, 2), dtype=np.int32)
    kvh = np.zeros((n, 2), dtype=np.int32)
    for j in range(n):
        s, r = int(sp[j]), int(rank[j])
        hq_loc = hq_total // s
        qh[j] = (r * hq_loc, (r + 1) * hq_loc)
        if hkv_total >= s:
            hk = hkv_total // s
            kvh[j] = (r * hk, (r + 1) * hk)
        else:
            g = (r * hkv_total) // s
            kvh[j] = (g, g + 1)
    return WorkList(lengths=lengths.astype(np.int32), sp=sp.astype(np.int32), q_heads=qh,
                    kv_heads=kvh, hq_total=hq_total, hkv_total=hkv_total, head_dim=head_dim)


def _draw_lengths(rng, mu, sigma, lo, hi, target, sp_rule=None):
    """Draw item lengths until the per-GPU token target is reached exactly.

    sp_rule(L) -> sp gives an item's Ulysses degree (default: 1). Per-GPU
    tokens of an item are L/sp. The last item is truncated to the remaining
    per-GPU tokens and placed at sp=1.
    """
    lengths, sps, tot = [], [], 0
    while tot < target:
        L = int(np.clip(int(np.rint(rng.lognormal(mu, sigma))), lo, hi))
        s = 1 if sp_rule is None else sp_rule(L)
        L -= L % s
        if tot + L // s > target:
            lengths.append(target - tot)
            sps.append(1)
            break
        lengths.append(L)
        sps.append(s)
        tot += L // s
    return lengths, sps


@dataclasses.dataclass
class Workload:
    """A named configuration: its work list plus how its tensors are drawn."""

    name: str
    description: str
    wl: WorkList
    seed: int
    softmax_scale: float
    # sequence-sharded inputs for pack/unpack (None: no re-layout step)
    pack_wl: Optional[WorkList] = None
    seq_input: bool = False  # True: attention inputs come from pack(seq tensors)

    def rng_after_lengths(self) -> np.random.Generator:
        """The seeded generator positioned right after the length draws."""
        rng = np.random.default_rng(self.seed)
        _replay_length_draws(self.name, rng)
        return rng

    def attention_inputs(self):
        """(q, k, v, dout) bf16 bit arrays in the attention layout.

        Not available for workloads whose attention inputs are produced by
        pack from sequence-sharded tensors (seq_input=True).
        """
        if self.seq_input:
            raise ValueError(f"{self.name}: attention inputs come from pack(seq_inputs())")
        rng = self.rng_after_lengths()
        q = draw_bf16(rng, self.wl.q_elems())
        k = draw_bf16(rng, self.wl.kv_elems())
        v = draw_bf16(rng, self.wl.kv_elems())
        do = draw_bf16(rng, self.wl.q_elems())
        return q, k, v, do

    def seq_inputs(self):
        """(xq, xk, xv, xdo) bf16 bit arrays in the sequence-sharded layout.

        Shapes: [sum_j L_j/sp_j, H, D] with H = Hq for q/dO and Hkv for k/v.
        Drawn after the attention-layout tensors (if the workload has them).
        """
        pw = self.pack_wl
        if pw is None:
            raise ValueError(f"{self.name}: no re-layout step")
        rng = self.rng_after_lengths()
        if not self.seq_input:
            for n in (self.wl.q_elems(), self.wl.kv_elems(), self.wl.kv_elems(), self.wl.q_elems()):
                rng.standard_normal(n, dtype=np.float32)  # skip the attention tensors
        T = pw.seq_tokens()
        D = pw.head_dim
        xq = draw_bf16(rng, T * pw.hq_total * D)
        xk = draw_bf16(rng, T * pw.hkv_total * D)
        xv = draw_bf16(rng, T * pw.hkv_total * D)
        xdo = draw_bf16(rng, T * pw.hq_total * D)
        return xq, xk, xv, xdo


CONFIG_NAMES = ("tiny", "short_sp1", "nested_2level", "longtail_4level", "maxctx_relayout")

_C4_SP_LEVELS = (1, 2, 4, 8)


def _c4_sp_rule(L: int) -> int:
    for s in _C4_SP_LEVELS:
        if L // s <= 32768:
            return s
    return _C4_SP_LEVELS[-1]


def _replay_length_draws(name: str, rng: np.random.Generator):
    """Consume the length draws of a named config from rng; return (lengths, sps)."""
    if name == "tiny":
        return [64, 128, 256, 512], [1, 1, 1, 1]
    if name == "short_sp1":
        return _draw_lengths(rng, np.log(2048.0), 1.0, 128, 32768, 65536)
    if name == "nested_2level":
        L, S = _draw_lengths(rng, np.log(4096.0), 0.8, 256, 16384, 32768)
        return [131072] + L, [8] + S
    if name == "longtail_4level":
        return _draw_lengths(rng, np.log(8192.0), 1.3, 256, 262144, 262144, _c4_sp_rule)
    if name == "maxctx_relayout":
        return [393216], [8]
    raise KeyError(name)


def make_config(name: str) -> Workload:
    """The five configurations, by name (in order):

    tiny             4 sequences {64,128,256,512}, 8 q / 2 KV heads, D=64, sp=1, seed 0;
                     plus pack/unpack of the same lengths at sp=2
    short_sp1        lognormal(ln 2048, 1.0) in [128, 32768], 65536 tokens, sp=1,
                     32 q / 4 KV heads, D=128, seed 1
    nested_2level    one 131072-token sequence at sp=8 (4 q, 1 KV head) plus short
                     sequences lognormal(ln 4096, 0.8) in [256, 16384], 32768 tokens
                     at sp=1 (32/4 heads), D=128, seed 2
    longtail_4level  lognormal(ln 8192, 1.3) in [256, 262144]; sp = smallest of
                     {1,2,4,8} with L/sp <= 32768; 262144 per-GPU tokens, D=128, seed 3
    maxctx_relayout  one 393216-token sequence at sp=8: pack [49152, 32, 128] to the
                     head-sharded layout, attention over 393216 tokens (4 q, 1 KV head),
                     unpack back; D=128, seed 4
    """
    seeds = {n: i for i, n in enumerate(CONFIG_NAMES)}
    if name not in seeds:
        raise KeyError(f"unknown config {name!r}; choose from {CONFIG_NAMES}")
    seed = seeds[name]
    lengths, sps = _replay_length_draws(name, np.random.default_rng(seed))
    if name == "tiny":
        wl = make_worklist(lengths, sps, 8, 2, 64)
        pack_wl = make_worklist(lengths, [2] * 4, 8, 2, 64)
        return Workload(name, "4 seqs {64..512}, 8q/2kv, D=64, sp=1 (+pack/unpack at sp=2)",
                        wl, seed, 1.0 / np.sqrt(64.0), pack_wl=pack_wl)
    wl = make_worklist(lengths, sps, 32, 4, 128)
    scale = 1.0 / np.sqrt(128.0)
    if name == "maxctx_relayout":
        return Workload(name, "1 x 393216 @ sp=8 (4q/1kv), pack -> attention -> unpack",
                        wl, seed, scale, pack_wl=wl, seq_input=True)
    desc = {
        "short_sp1": "lognormal(ln 2048, 1) short items, 65536 tokens, sp=1, 32q/4kv, D=128",
        "nested_2level": "131072 @ sp=8 (4q/1kv) + shorts lognormal(ln 4096, 0.8), 32768 tokens",
        "longtail_4level": "lognormal(ln 8192, 1.3), sp in {1,2,4,8}, 262144 per-GPU tokens",
    }[name]
    return Workload(name, desc, wl, seed, scale)


def small_worklist(lengths: Sequence[int], hq_total: int = 8, hkv_total: int = 2,
                   head_dim: int = 64, sp: Optional[Sequence[int]] = None,
                   rank: Optional[Sequence[int]] = None) -> WorkList:
    """Convenience for tests: items at the given degrees (default sp=1)."""
    sp = [1] * len(lengths) if sp is None else list(sp)
    return make_worklist(list(lengths), sp, hq_total, hkv_total, head_dim, rank)


def draw_attention_inputs(wl: WorkList, seed: int):
    """Q, K, V, dO bf16 bits for an arbitrary work list (test helper)."""
    rng = np.random.default_rng(seed)
    return (draw_bf16(rng, wl.q_elems()), draw_bf16(rng, wl.kv_elems()),
            draw_bf16(rng, wl.kv_elems()), draw_bf16(rng, wl.q_elems()))


def item_lengths_summary(wl: WorkList) -> List[tuple]:
    return [(int(L), int(s), int(q[1] - q[0]), int(k[1] - k[0]))
            for L, s, q, k in zip(wl.lengths, wl.sp, wl.q_heads, wl.kv_heads)]
