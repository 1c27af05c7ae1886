"""HBM traffic record read by bench.py, from two rocprofv3 counter runs.

    python -m paper_2609_22755_amd.traffic WORKLOAD FETCH_DIR WRITE_DIR [COPY_MIB]

FETCH_DIR and WRITE_DIR are the output directories (-d) of

    rocprofv3 --pmc FETCH_SIZE GRBM_GUI_ACTIVE -f csv -d FETCH_DIR -o run -- \\
        python3 bench.py --workload WORKLOAD --steps 1 --warmup 0 \\
        --no-cpu-baseline --no-streaming --no-ceiling --copy-calibration-mib 1024

and of the same command with --pmc WRITE_SIZE (with --steps 1 --warmup 0
the run holds one step).  Both counters are read in KiB per dispatch.  GRBM_GUI_ACTIVE (busy cycles summed over the XCDs), over
the dispatch's duration and the XCD count, gives the shader clock each kernel
ran at.  The run ends with a plain device copy of COPY_MIB MiB
(default 1024, the --copy-calibration-mib of the run; the largest copy kernel
of the run); what the counters report for it, against the
bytes it really reads and writes, gives the factor that turns a counter
reading into bytes.  The record names the kernel sources and their sha256, so
that bench.py reports the traffic only while the kernels are unchanged.

Writes profiles/hbm_traffic_<WORKLOAD>.json and prints a table.
"""
from __future__ import annotations

import collections
import csv
import glob
import hashlib
import json
import os
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")

KERNELS = {  # record name -> substring of the kernel symbol
    "attn_fwd": "attn_fwd_kernel",
    "bwd_preprocess": "bwd_preprocess_kernel",
    "bwd_dkdv": "bwd_dkdv_kernel",
    "bwd_dq": "bwd_dq_kernel",
}
COPY = "copyBuffer"
RELAYOUT = "relayout_kernel"


def per_dispatch(run_dir: str, counter: str, with_time: bool = False) -> list:
    """(kernel name, counter value summed over its rows[, duration in ns]) per
    dispatch, in order."""
    paths = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not paths:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    val = collections.OrderedDict()
    name, dur = {}, {}
    for p in paths:
        with open(p) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] != counter:
                    continue
                d = (p, int(r["Dispatch_Id"]))
                val[d] = val.get(d, 0.0) + float(r["Counter_Value"])
                name[d] = r["Kernel_Name"]
                dur[d] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    if with_time:
        return [(name[d], v, dur[d]) for d, v in val.items()]
    return [(name[d], v) for d, v in val.items()]


def num_xcc(run_dir: str) -> int:
    for p in glob.glob(os.path.join(run_dir, "**", "*agent_info.csv"), recursive=True):
        with open(p) as f:
            for r in csv.DictReader(f):
                if r.get("Agent_Type") == "GPU":
                    return int(r["Num_Xcc"])
    raise SystemExit(f"no GPU agent in {run_dir}")


def kernel_kib(disp: list[tuple[str, float]], key: str) -> float | None:
    vals = [v for n, v in disp if key in n]
    return sum(vals) / len(vals) if vals else None


def sources_sha() -> tuple[list[str], str]:
    srcs = sorted(f for f in os.listdir(CSRC))
    rel = [os.path.join("paper_2609_22755_amd", "csrc", f) for f in srcs]
    h = hashlib.sha256()
    for r in rel:
        h.update(open(os.path.join(ROOT, r), "rb").read())
    return rel, h.hexdigest()


def main(argv: list[str]) -> None:
    if len(argv) not in (4, 5):
        raise SystemExit(__doc__)
    workload, fdir, wdir = argv[1:4]
    copy_bytes = (int(argv[4]) if len(argv) == 5 else 1024) * (1 << 20)
    fd = per_dispatch(fdir, "FETCH_SIZE")
    wd = per_dispatch(wdir, "WRITE_SIZE")
    gd = per_dispatch(fdir, "GRBM_GUI_ACTIVE", with_time=True)
    nx = num_xcc(fdir)
    fcopy = max((v for n, v in fd if COPY in n), default=None)
    wcopy = max((v for n, v in wd if COPY in n), default=None)
    if not fcopy or not wcopy:
        raise SystemExit("no calibration copy found (run bench.py with --copy-calibration-mib)")
    # the copy reads and writes copy_bytes each
    ff = copy_bytes / (fcopy * 1024.0)
    wf = copy_bytes / (wcopy * 1024.0)
    rel, sha = sources_sha()
    rec = {
        "workload": workload,
        "source_sha256": sha,
        "sources": rel,
        "calibration": {"copy_bytes_read": copy_bytes, "copy_bytes_written": copy_bytes,
                        "fetch_factor": round(ff, 4), "write_factor": round(wf, 4)},
        "kernels": {},
    }
    print(f"calibration: copy of {copy_bytes / 2**30:.2f} GiB reads as FETCH {fcopy / 2**20:.3f} GiB "
          f"(x{ff:.3f}), WRITE {wcopy / 2**20:.3f} GiB (x{wf:.3f})")
    print(f"{'kernel':16s} {'FETCH KiB':>16s} {'WRITE KiB':>14s} {'HBM GB/launch':>14s} {'sclk GHz':>9s}")
    for k, key in KERNELS.items():
        f, w = kernel_kib(fd, key), kernel_kib(wd, key)
        if f is None or w is None:
            continue
        b = f * 1024.0 * ff + w * 1024.0 * wf
        g = [(v, t) for n, v, t in gd if key in n and t > 0]
        ghz = sum(v for v, _ in g) / nx / sum(t for _, t in g) if g else None
        rec["kernels"][k] = {"fetch_kib": f, "write_kib": w, "hbm_bytes_per_launch": b, "sclk_ghz": ghz}
        print(f"{k:16s} {f:16,.0f} {w:14,.0f} {b / 1e9:14.1f} {ghz if ghz else float('nan'):9.3f}")
    # the re-layout kernel runs several times per step with different sizes:
    # its bytes are recorded summed over the run's dispatches (one step)
    f_rl = sum(v for n, v in fd if RELAYOUT in n)
    w_rl = sum(v for n, v in wd if RELAYOUT in n)
    n_rl = sum(1 for n, _ in fd if RELAYOUT in n)
    if n_rl:
        b = f_rl * 1024.0 * ff + w_rl * 1024.0 * wf
        rec["relayout_per_step"] = {"dispatches": n_rl, "fetch_kib": f_rl, "write_kib": w_rl, "hbm_bytes": b}
        print(f"{'relayout (step)':16s} {f_rl:16,.0f} {w_rl:14,.0f} {b / 1e9:14.2f}   ({n_rl} dispatches)")
    out = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.json")
    with open(out, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print("wrote", os.path.relpath(out, ROOT))


if __name__ == "__main__":
    main(sys.argv)
