"""Matrix-core utilisation record read by bench.py, from two rocprofv3 counter runs.

    python -m paper_2609_22755_amd.mfma_util WORKLOAD MFMA_DIR LDS_DIR

MFMA_DIR and LDS_DIR are the output directories (-d) of

    rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_VALU_MFMA_COEXEC_CYCLES SQ_BUSY_CU_CYCLES \\
        SQ_WAVE_CYCLES SQ_INSTS_MFMA SQ_INSTS_VALU GRBM_GUI_ACTIVE -f csv -d MFMA_DIR -o run -- \\
        python3 bench.py --workload WORKLOAD --steps 1 --warmup 0 --no-cpu-baseline --no-streaming --no-ceiling

and of the same command with --pmc SQ_LDS_IDX_ACTIVE SQ_LDS_BANK_CONFLICT
SQ_LDS_DATA_FIFO_FULL SQ_INSTS_LDS SQ_WAIT_INST_LDS SQ_WAIT_INST_ANY
SQ_ACTIVE_INST_VALU GRBM_GUI_ACTIVE (each pass within the per-block counter
limits of one rocprofv3 run).

Normalisation (GRBM_GUI_ACTIVE is summed over the XCDs; the SQ counters over
every SIMD or CU of the chip):
  cycles        = GRBM_GUI_ACTIVE / XCDs: shader clocks the dispatch was busy
  sclk          = cycles / dispatch duration
  mfma_busy     = SQ_VALU_MFMA_BUSY_CYCLES / (cycles * CUs * 4): share of SIMD
                  cycles with a matrix product executing (each
                  v_mfma_f32_32x32x16_bf16 holds its SIMD's matrix core for 32
                  cycles, so this equals SQ_INSTS_MFMA * 32 / (cycles * SIMDs))
  frac_of_peak  = mfma_busy * sclk / 2.4 GHz: the executed matrix-core rate
                  against the dense bf16 peak (256 CUs x 4096 flop/clk x 2.4 GHz)
  cu_occupied   = SQ_BUSY_CU_CYCLES / (cycles * CUs): share of CU time with a
                  workgroup resident (ramp, tail and gaps between units excluded)
  waves_per_busy_cu_quad = SQ_WAVE_CYCLES / SQ_BUSY_CU_CYCLES: resident waves
                  per CU over 4 (1 for the 4-wave dK/dV pass, 2 for the
                  8-wave forward and dQ passes)
  lds_active    = SQ_LDS_IDX_ACTIVE / (cycles * CUs)
  wait shares   = SQ_WAIT_INST_LDS, SQ_WAIT_INST_ANY, SQ_ACTIVE_INST_VALU over
                  SQ_WAVE_CYCLES (per-wave cycle counts, same units)
Writes profiles/mfma_utilization_<WORKLOAD>.json (with the sha256 of the
kernel sources, as the HBM traffic record) and prints a table.
"""
from __future__ import annotations

import json
import os
import sys

from paper_2609_22755_amd.traffic import KERNELS, ROOT, num_xcc, per_dispatch, sources_sha

PEAK_SCLK_GHZ = 2.4
MFMA_CYCLES = 32          # v_mfma_f32_32x32x16_bf16 on one SIMD


def kernel_sums(run_dir: str, counters: list[str]) -> dict:
    """{kernel record name: {counter: mean per dispatch, '_ns': mean duration}}."""
    out: dict = {}
    for c in counters:
        rows = per_dispatch(run_dir, c, with_time=True)
        for k, key in KERNELS.items():
            sel = [(v, t) for n, v, t in rows if key in n]
            if not sel:
                continue
            d = out.setdefault(k, {})
            d[c] = sum(v for v, _ in sel) / len(sel)
            d["_ns"] = sum(t for _, t in sel) / len(sel)
            d["_n"] = len(sel)
    return out


def main(argv: list[str], out_dir: str | None = None) -> dict:
    if len(argv) != 4:
        raise SystemExit(__doc__)
    workload, mdir, ldir = argv[1:4]
    m = kernel_sums(mdir, ["SQ_VALU_MFMA_BUSY_CYCLES", "SQ_VALU_MFMA_COEXEC_CYCLES", "SQ_BUSY_CU_CYCLES",
                           "SQ_WAVE_CYCLES", "SQ_INSTS_MFMA", "SQ_INSTS_VALU", "GRBM_GUI_ACTIVE"])
    lrec = kernel_sums(ldir, ["SQ_LDS_IDX_ACTIVE", "SQ_LDS_BANK_CONFLICT", "SQ_INSTS_LDS", "SQ_WAIT_INST_LDS",
                              "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_VALU", "GRBM_GUI_ACTIVE"])
    nx = num_xcc(mdir)
    cus = 32 * nx
    rel, sha = sources_sha()
    rec = {"workload": workload, "source_sha256": sha, "sources": rel, "xcds": nx, "cus": cus,
           "peak_sclk_ghz": PEAK_SCLK_GHZ, "kernels": {}}
    print(f"{'kernel':14s} {'sclk':>6s} {'mfma_busy':>9s} {'frac_peak':>9s} {'mfma*32/SIMDcyc':>15s} "
          f"{'lds_act':>7s} {'valu/mfma':>9s} {'lds/mfma':>8s} {'wait_lds':>8s} {'wait_any':>8s}")
    for k in ("attn_fwd", "bwd_dkdv", "bwd_dq"):
        if k not in m:
            continue
        a = m[k]
        cyc = a["GRBM_GUI_ACTIVE"] / nx
        sclk = cyc / a["_ns"]
        busy = a["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * cus * 4)
        from_insts = a["SQ_INSTS_MFMA"] * MFMA_CYCLES / (cyc * cus * 4)
        r = {"dispatches": a["_n"], "duration_ms": a["_ns"] / 1e6, "sclk_ghz": sclk, "mfma_busy": busy,
             "mfma_busy_from_insts": from_insts,
             "mfma_coexec": a["SQ_VALU_MFMA_COEXEC_CYCLES"] / (cyc * cus * 4),
             "frac_of_peak_executed": busy * sclk / PEAK_SCLK_GHZ,
             "cu_occupied": a["SQ_BUSY_CU_CYCLES"] / (cyc * cus),
             "waves_per_busy_cu_quad": a["SQ_WAVE_CYCLES"] / max(a["SQ_BUSY_CU_CYCLES"], 1.0),
             "valu_insts_per_mfma": a["SQ_INSTS_VALU"] / a["SQ_INSTS_MFMA"]}
        if k in lrec:
            b = lrec[k]
            lcyc = b["GRBM_GUI_ACTIVE"] / nx
            r["lds_active"] = b["SQ_LDS_IDX_ACTIVE"] / (lcyc * cus)
            r["lds_insts_per_mfma"] = b["SQ_INSTS_LDS"] / a["SQ_INSTS_MFMA"]
            r["lds_bank_conflicts_per_inst"] = b["SQ_LDS_BANK_CONFLICT"] / max(b["SQ_INSTS_LDS"], 1.0)
            for c in ("SQ_WAIT_INST_LDS", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_VALU"):
                r[c.lower() + "_share"] = b[c] / a["SQ_WAVE_CYCLES"]
        rec["kernels"][k] = r
        print(f"{k:14s} {sclk:6.3f} {100 * busy:8.1f}% {100 * r['frac_of_peak_executed']:8.1f}% "
              f"{100 * from_insts:14.1f}% {100 * r.get('lds_active', float('nan')):6.1f}% "
              f"{r['valu_insts_per_mfma']:9.2f} {r.get('lds_insts_per_mfma', float('nan')):8.2f} "
              f"{r.get('sq_wait_inst_lds_share', float('nan')):8.3f} {r.get('sq_wait_inst_any_share', float('nan')):8.3f}")
    out = os.path.join(out_dir or os.path.join(ROOT, "profiles"), f"mfma_utilization_{workload}.json")
    with open(out, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(f"wrote {out}")
    return rec


if __name__ == "__main__":
    main(sys.argv)
