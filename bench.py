#!/usr/bin/env python3
"""Benchmark of the per-GPU NSP hot path on one MI355X.

One step = one pass of the whole per-GPU path over one synthetic batch:
  pack Q, K, V (sequence-sharded -> head-sharded) -> attention forward ->
  unpack O -> pack dO -> attention backward -> unpack dQ, dK (replica sum),
  dV (replica sum)
all in libnsp's HIP kernels, inputs resident in HBM.  The reported value is
counted attention flops (fwd + bwd, sum_j 14 * D * hq_j * L_j (L_j + 1) / 2)
per second of step time, in TFLOP/s; the step time includes the re-layout.

After the timed steps it measures this GPU's matrix-core ceiling under its
power limit (nsp_mfma_ceiling: bf16 products only, random operands) and
reports each kernel's executed rate against it (mfma_ceiling,
kernel_roofline.*.frac_of_ceiling): boards differ by several percent in the
clock they hold under load, and that figure does not.

Prints one JSON line.  Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "causal varlen attention fwd+bwd TFLOP/s and % of bf16 MFMA peak, 1 GPU"
PEAK_BF16_TFLOPS = 2516.6     # 256 CU x 2.4 GHz x 4096 dense bf16 flop/clk/CU
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="longtail_4level")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="time budget of the oracle sample")
    ap.add_argument("--no-streaming", action="store_true",
                    help="skip the phase-streamed step (two queues, one launch set per SP-tree node)")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the matrix-core ceiling measurement after the timed steps")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one plain device copy of this size (for HBM counter scaling)")
    return ap.parse_args()


def gpu_inputs(wl, seed, device):
    """Seeded N(0,1) bf16 tensors in the sequence-sharded layout, drawn on the GPU."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    T, D = wl.seq_tokens(), wl.head_dim

    def draw(n):
        return torch.randn(n, generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)

    return dict(q=draw(T * wl.hq_total * D), k=draw(T * wl.hkv_total * D), v=draw(T * wl.hkv_total * D),
                do=draw(T * wl.hq_total * D))


def counter_record(workload, kind="hbm_traffic"):
    """A committed rocprofv3 counter record of a workload -- kind "hbm_traffic"
    (HBM bytes and observed shader clock per kernel, see
    paper_2609_22755_amd/traffic.py) or "mfma_utilization" (matrix-core busy
    share per kernel, see paper_2609_22755_amd/mfma_util.py) -- or None when
    there is none or the kernel sources have changed since the counters were
    taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{kind}_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    h = hashlib.sha256()
    for src in rec["sources"]:
        full = os.path.join(ROOT, src)
        if not os.path.exists(full):
            return None
        h.update(open(full, "rb").read())
    csrc = os.path.join(ROOT, "paper_2609_22755_amd", "csrc")
    if h.hexdigest() != rec["source_sha256"] or sorted(os.listdir(csrc)) != sorted(
            os.path.basename(x) for x in rec["sources"]):
        return None
    return rec


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the counter record (FETCH_SIZE /
    WRITE_SIZE, scaled by a plain-copy calibration), or None."""
    rec = counter_record(workload)
    k = None if rec is None else rec["kernels"].get(kernel)
    return None if k is None else k["hbm_bytes_per_launch"]


def observed_sclk_ghz(workload, kern):
    """Shader clock of the attention kernels in the counter record
    (GRBM_GUI_ACTIVE per XCD over the dispatch time), weighted by this run's
    kernel times, or None."""
    rec = counter_record(workload)
    if rec is None:
        return None
    num = den = 0.0
    for k in ("attn_fwd", "bwd_dkdv", "bwd_dq"):
        ghz = rec["kernels"].get(k, {}).get("sclk_ghz")
        if ghz is None:
            return None
        num += ghz * kern[k]["ms_per_step"]
        den += kern[k]["ms_per_step"]
    return num / den if den else None


def cpu_baseline(wl, scale, budget_s, counted_flops):
    """The fp64 oracle on a bounded sample of the same work list, on the host.

    Sample: passes over the items in order; pass p takes one local query head
    of each item and its query rows [L - 128(p+1), L - 128p) (forward rows +
    their backward), inputs seeded N(0,1) (drawn outside the timed region);
    items and passes are taken until the oracle's own time reaches the budget.
    Flops are the algorithmic count of the rows done: 14 * D * sum_t (t + 1).
    The whole step's oracle time is extrapolated from the sampled rate (the
    step's counted flops over it) and labelled as such.
    """
    from oracle import attention as OA
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    D = wl.head_dim
    flops, rows_done, dt, passes = 0.0, 0, 0.0, 0
    lengths = wl.lengths.tolist()
    inputs = {}
    while dt <= budget_s and any(L > 128 * passes for L in lengths):
        for j, L in enumerate(lengths):
            if dt > budget_s:
                break
            hi = L - 128 * passes
            if hi <= 0:
                continue
            if j not in inputs:
                rng = np.random.default_rng(1000 + j)
                inputs[j] = [rng.standard_normal((L, D), dtype=np.float32).astype(np.float64) for _ in range(4)]
            q, k, v, do = inputs[j]
            rows = np.arange(max(0, hi - 128), hi)
            t0 = time.perf_counter()      # only the oracle's own work is timed
            OA.head_rows_forward(q, k, v, rows, scale)
            OA.head_backward(q, k, v, do, scale, rows=rows)
            dt += time.perf_counter() - t0
            flops += 14.0 * D * float(np.sum(rows + 1))
            rows_done += rows.size
        passes += 1
    rate = flops / dt
    return {"value": rate / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "full_step_s_extrapolated": round(counted_flops / rate, 1),
            "sample": f"fp64 oracle fwd+bwd of one local head per item, {rows_done} query rows in {passes} "
                      f"pass(es) of 128-row blocks from the end of each of the {wl.n_items} items; "
                      f"{flops:.3e} flops in {dt:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU exchange "
              "(RCCL all-to-all) is not part of this build", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2609_22755_amd import nsp
    from paper_2609_22755_amd.workloads import make_config

    dev = "cuda:0"
    torch.cuda.set_device(0)
    lib = nsp.load_library()
    w = make_config(args.workload)
    wl = w.wl
    scale = w.softmax_scale
    print(f"[bench] workload {w.name}: {wl.n_items} items, {wl.seq_tokens()} per-GPU tokens, "
          f"sum L {int(wl.lengths.sum())}", file=sys.stderr, flush=True)

    x = gpu_inputs(wl, w.seed, dev)
    qe, ke = wl.q_elems(), wl.kv_elems()
    bf = torch.bfloat16
    t = dict(q=torch.empty(qe, dtype=bf, device=dev), k=torch.empty(ke, dtype=bf, device=dev),
             v=torch.empty(ke, dtype=bf, device=dev), do=torch.empty(qe, dtype=bf, device=dev))
    buf = nsp.alloc_like_worklist(wl, device=dev)
    out = dict(o=torch.empty_like(x["q"]), dq=torch.empty_like(x["q"]), dk=torch.empty_like(x["k"]),
               dv=torch.empty_like(x["v"]))
    Q, KV = nsp.NSP_KIND_Q, nsp.NSP_KIND_KV
    SEL, SUM = nsp.NSP_UNPACK_SELECT, nsp.NSP_UNPACK_SUM

    def step():
        nsp.nsp_ulysses_pack(wl, Q, x["q"], t["q"])
        nsp.nsp_ulysses_pack(wl, KV, x["k"], t["k"])
        nsp.nsp_ulysses_pack(wl, KV, x["v"], t["v"])
        nsp.nsp_varlen_attn_fwd(wl, t["q"], t["k"], t["v"], buf["o"], buf["lse"], scale)
        nsp.nsp_ulysses_unpack(wl, Q, SEL, buf["o"], out["o"])
        nsp.nsp_ulysses_pack(wl, Q, x["do"], t["do"])
        nsp.nsp_varlen_attn_bwd(wl, t["q"], t["k"], t["v"], buf["o"], t["do"], buf["lse"], buf["dq"],
                                buf["dk"], buf["dv"], buf["ws"], scale)
        nsp.nsp_ulysses_unpack(wl, Q, SEL, buf["dq"], out["dq"])
        nsp.nsp_ulysses_unpack(wl, KV, SUM, buf["dk"], out["dk"])
        nsp.nsp_ulysses_unpack(wl, KV, SUM, buf["dv"], out["dv"])

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        print(f"[bench] warmup step {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)

    nsp.nsp_timing_reset()
    nsp.nsp_timing_enable(True)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ev[0].record()
    for i in range(args.steps):
        step()
        ev[i + 1].record()
    torch.cuda.synchronize()
    nsp.nsp_timing_enable(False)
    ms_per_step = ev[0].elapsed_time(ev[-1]) / args.steps
    per_step = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))
    print(f"[bench] timed {args.steps} steps: {ms_per_step:.3f} ms/step", file=sys.stderr, flush=True)

    kern = {}
    for name in nsp.KERNELS:
        n, ms = nsp.nsp_timing_query(name)
        kern[name] = {"launches": n, "total_ms": ms, "avg_ms": ms / n if n else 0.0,
                      "ms_per_step": ms / args.steps}

    D = wl.head_dim
    pairs_hq = float(np.sum(wl.hq * wl.causal_pairs()))
    flops_fwd, flops_bwd = 4.0 * D * pairs_hq, 10.0 * D * pairs_hq
    flops = flops_fwd + flops_bwd
    value = flops / (ms_per_step * 1e-3) / 1e12
    attn_ms = sum(kern[k]["ms_per_step"] for k in ("attn_fwd", "bwd_preprocess", "bwd_dkdv", "bwd_dq"))
    # algorithmic flops per launch of each attention kernel (MFMA products over causal pairs):
    # forward QK^T + PV = 4 D; dK/dV pass S + dP + dV + dK = 8 D; dQ pass S + dP + dQ = 6 D
    kflops = {"attn_fwd": 4.0 * D * pairs_hq, "bwd_dkdv": 8.0 * D * pairs_hq, "bwd_dq": 6.0 * D * pairs_hq}
    # the share of the counted 14 D that each kernel's products make up: the dQ
    # pass recomputes S and dP (counted in the dK/dV pass), so only its dQ
    # product (2 D) is counted
    kcounted = {"attn_fwd": 4.0 * D * pairs_hq, "bwd_dkdv": 8.0 * D * pairs_hq, "bwd_dq": 2.0 * D * pairs_hq}
    dom = max(kflops, key=lambda k: kern[k]["total_ms"])
    util = counter_record(w.name, "mfma_utilization")
    kernel_roofline = {}
    for k in kflops:
        sec = kern[k]["avg_ms"] * 1e-3
        e = kflops[k] / sec / 1e12 if sec else None
        cnt = kcounted[k] / sec / 1e12 if sec else None
        kernel_roofline[k] = {
            "ms_per_launch": round(kern[k]["avg_ms"], 3),
            "executed_tflops": None if e is None else round(e, 2),
            "frac_executed": None if e is None else round(e / PEAK_BF16_TFLOPS, 4),
            "counted_tflops": None if cnt is None else round(cnt, 2),
            "frac_counted": None if cnt is None else round(cnt / PEAK_BF16_TFLOPS, 4),
            "mfma_busy_counter": (None if util is None or k not in util["kernels"]
                                  else round(util["kernels"][k]["mfma_busy"], 4)),
            "sclk_ghz_counter": (None if util is None or k not in util["kernels"]
                                 else round(util["kernels"][k]["sclk_ghz"], 3)),
        }
    achieved = kflops[dom] / (kern[dom]["avg_ms"] * 1e-3) / 1e12
    # re-layout bytes per step: every element read once and written once (replica sums read sp/H copies)
    seq_q = wl.seq_tokens() * wl.hq_total * D * 2
    seq_kv = wl.seq_tokens() * wl.hkv_total * D * 2
    head_q, head_kv = qe * 2, ke * 2
    relayout_bytes = 4 * (seq_q + head_q) + 4 * (seq_kv + head_kv)
    rl_ms = kern["relayout"]["ms_per_step"]

    res = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "description": w.description, "items": wl.n_items,
                   "per_gpu_tokens": wl.seq_tokens(), "sum_L": int(wl.lengths.sum()),
                   "max_L": int(wl.lengths.max()), "hq_total": wl.hq_total, "hkv_total": wl.hkv_total,
                   "head_dim": D, "worklist_sha": wl.digest(), "counted_flops": flops},
        "ms_per_step_median": round(float(np.median(per_step)), 3),
        "ms_per_step_min": round(per_step[0], 3),
        "pct_of_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "attention_only_tflops": round(flops / (attn_ms * 1e-3) / 1e12, 2) if attn_ms else None,
        "fwd_tflops": round(flops_fwd / (kern["attn_fwd"]["ms_per_step"] * 1e-3) / 1e12, 2),
        "bwd_tflops": round(flops_bwd / ((kern["bwd_preprocess"]["ms_per_step"] + kern["bwd_dkdv"]["ms_per_step"]
                                          + kern["bwd_dq"]["ms_per_step"]) * 1e-3) / 1e12, 2),
        "relayout_gbs": round(relayout_bytes / (rl_ms * 1e-3) / 1e9, 1) if rl_ms else None,
        "kernels_ms_per_step": {k: round(v["ms_per_step"], 4) for k, v in kern.items()},
        "roofline": {"kernel": dom, "bound": "mfma", "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic(w.name, dom)},
        # per attention kernel: algorithmic flops it executes (4 D, 8 D, 6 D per
        # causal pair and head) and its share of the counted 14 D, over its
        # live launch time, against the dense bf16 peak; with the committed
        # counter record (same kernel sources), the share of SIMD cycles its
        # matrix cores were busy and the shader clock it ran at
        "kernel_roofline": kernel_roofline,
    }
    if not args.no_ceiling:
        # this GPU's matrix-core ceiling under its power limit (bf16 products
        # only, approximately normal operands that change every product),
        # measured after the timed steps: what the kernels' executed rates can
        # be held against on this particular board
        csec, ctf = nsp.nsp_mfma_ceiling(0, False, 1, 1 << 21)
        step_exec = sum(kflops.values()) / (ms_per_step * 1e-3) / 1e12
        res["mfma_ceiling"] = {"tflops": round(ctf, 1), "frac_of_peak": round(ctf / PEAK_BF16_TFLOPS, 4),
                               "ms": round(csec * 1e3, 2), "operands": "bf16, approximately normal, new every product",
                               "step_executed_tflops": round(step_exec, 1),
                               "step_frac_of_ceiling": round(step_exec / ctf, 4)}
        for k, r in kernel_roofline.items():
            r["frac_of_ceiling"] = None if r["executed_tflops"] is None else round(r["executed_tflops"] / ctf, 4)
        print(f"[bench] matrix-core ceiling of this GPU: {ctf:.1f} TFLOP/s; the step executes "
              f"{step_exec:.1f} TFLOP/s ({100 * step_exec / ctf:.1f}% of it)", file=sys.stderr, flush=True)
    sclk = observed_sclk_ghz(w.name, kern)
    res["observed_sclk_ghz"] = None if sclk is None else round(sclk, 3)
    # the same peak at the clock the kernels ran at (CUs x sclk x 4096 flop/clk/CU)
    res["pct_of_peak_at_observed_sclk"] = (None if sclk is None else
                                           round(100.0 * value / (256 * 4096 * sclk * 1e9 / 1e12), 2))
    if not args.no_streaming:
        # the same step issued by the phase-streaming executor: per SP-tree node
        # (items sharing an sp), pack -> attention -> unpack as item-masked
        # calls, compute and re-layout on two streams (default priority)
        comm = torch.cuda.Stream()
        ex = dict(q_seq=x["q"], k_seq=x["k"], v_seq=x["v"], do_seq=x["do"], o_seq=out["o"], dq_seq=out["dq"],
                  dk_seq=out["dk"], dv_seq=out["dv"], q=t["q"], k=t["k"], v=t["v"], o=buf["o"], dout=t["do"],
                  dq=buf["dq"], dk=buf["dk"], dv=buf["dv"], lse=buf["lse"], workspace=buf["ws"])
        for _ in range(max(1, args.warmup)):
            nsp.nsp_executor_step(wl, ex, scale, comm=comm)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            nsp.nsp_executor_step(wl, ex, scale, comm=comm)
        e1.record()
        torch.cuda.synchronize()
        st_ms = e0.elapsed_time(e1) / args.steps
        nodes = sorted(set(int(v) for v in wl.sp), reverse=True)
        res["phase_streaming"] = {"ms_per_step": round(st_ms, 3), "tflops": round(flops / (st_ms * 1e-3) / 1e12, 2),
                                  "nodes_sp": nodes, "serial_ms_per_step": round(ms_per_step, 3),
                                  "speedup_vs_serial": round(ms_per_step / st_ms, 4)}
        print(f"[bench] phase-streamed step: {st_ms:.3f} ms ({len(nodes)} nodes)", file=sys.stderr, flush=True)
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20) // 4
        a = torch.empty(n, dtype=torch.float32, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        res["copy_calibration_bytes"] = 2 * n * 4
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host (cpu_baseline)", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(wl, scale, args.cpu_seconds, res["config"]["counted_flops"])
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
