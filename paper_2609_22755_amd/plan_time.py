"""Time the native SP-tree planner on long-tail batches (host only).

    python -m paper_2609_22755_amd.plan_time [--repeats R] [--seed S]

Batches follow the paper's evaluation protocol (Evaluation, Setup): 2M
tokens per training batch, sequences longer than the maximum context (192K
or 384K tokens) filtered out.  Lengths are synthetic, lognormal around 8192
tokens with sigma 1.3 (the long-tail mix of this library's other
workloads), rounded up to a multiple of the largest SP degree; the paper's
own length traces are not available.  The planner runs with the default
cost coefficients of SpTreeParams (this library's measured attention rates,
xGMI links) on one 8-GPU node and on 64 GPUs, for a 32-head / 4-KV-head,
head_dim 128 model, with a token budget of 1.25x the mean tokens per GPU, a
beam of 8 and a searched prefix of max(16, GPUs) samples (the paper gives
neither value; at 64 GPUs a 16-sample prefix leaves the plan about 20% out
of balance, a 64-sample one about 2%).
Prints one JSON line per configuration: median / min milliseconds per plan,
the number of samples, the SP degrees used and the plan's load balance
(max / mean of C_p).
"""
from __future__ import annotations

import argparse
import json
import math
import time

import numpy as np

from . import nsp

BATCH_TOKENS = 2 * 1024 * 1024


def long_tail_batch(rng, max_ctx: int, multiple: int, tokens: int = BATCH_TOKENS):
    out, total = [], 0
    while True:
        L = int(math.exp(rng.normal(math.log(8192), 1.3)))
        L = max(multiple, -(-L // multiple) * multiple)
        if L > max_ctx:
            continue
        if total + L > tokens:
            break
        out.append(L)
        total += L
    return np.array(out, dtype=np.int64)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--repeats", type=int, default=20)
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args(argv)
    nsp.load_library()
    configs = [(8, 192 * 1024), (8, 384 * 1024), (64, 192 * 1024), (64, 384 * 1024)]
    for c, (world, max_ctx) in enumerate(configs):
        rng = np.random.default_rng(1000 * args.seed + c)
        L = long_tail_batch(rng, max_ctx, world)
        prm = nsp.SpTreeParams(world=world, sp_max=world, hq_total=32, hkv_total=4, head_dim=128,
                               token_budget=1.25 * L.sum() / world, prefix=max(16, world), beam=8)
        times = []
        for _ in range(args.repeats):
            t0 = time.perf_counter()
            d, i, cost, tok, load = nsp.nsp_sp_tree_plan(prm, L)
            times.append(time.perf_counter() - t0)
        levels = sorted({world >> int(x) for x in d}, reverse=True)
        print(json.dumps({
            "what": "SP-tree plan (native planner), host CPU",
            "world": world, "max_ctx": max_ctx, "samples": int(L.size), "tokens": int(L.sum()),
            "longest": int(L.max()), "prefix": prm.prefix, "beam": prm.beam,
            "ms_median": round(1e3 * float(np.median(times)), 3), "ms_min": round(1e3 * min(times), 3),
            "sp_levels_used": levels, "load_s": round(load, 6),
            "cost_max_over_mean": round(float(cost.max() / cost.mean()), 4),
            "tokens_max_over_budget": round(float(tok.max() / prm.token_budget), 4),
        }), flush=True)

if __name__ == "__main__":
    main()
