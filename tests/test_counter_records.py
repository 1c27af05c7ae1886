"""The counter-record readers (HBM traffic, matrix-core utilisation) on
synthetic rocprofv3 CSV files: the normalisation the bench line relies on."""
import csv
import os

import pytest

from paper_2609_22755_amd import mfma_util

AGENT = [{"Agent_Type": "CPU", "Num_Xcc": "0"}, {"Agent_Type": "GPU", "Num_Xcc": "8"}]


def _write_run(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_agent_info.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Agent_Type", "Num_Xcc"])
        w.writeheader()
        w.writerows(AGENT)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
                                          "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        w.writerows(rows)


def test_mfma_utilisation_normalisation(tmp_path):
    ns = 100_000_000                     # a 100 ms dispatch
    sclk = 1.75                          # GHz
    cyc = sclk * ns                      # shader cycles per XCD
    busy = 0.6                           # matrix cores busy 60% of the SIMD cycles
    simd_cycles = cyc * 256 * 4
    mfma = busy * simd_cycles / 32       # 32 cycles per 32x32x16 product
    name = "void nsp::(anonymous namespace)::bwd_dkdv_kernel<128, false>(nsp::AttnArgs, int*, int)"
    # every counter split over two rows (the sum is what counts), GRBM over the 8 XCDs
    vals_m = {"SQ_VALU_MFMA_BUSY_CYCLES": busy * simd_cycles, "SQ_VALU_MFMA_COEXEC_CYCLES": 0.1 * simd_cycles,
              "SQ_BUSY_CU_CYCLES": 0.99 * cyc * 256, "SQ_WAVE_CYCLES": 0.99 * cyc * 256,
              "SQ_INSTS_MFMA": mfma, "SQ_INSTS_VALU": 3 * mfma, "GRBM_GUI_ACTIVE": 8 * cyc}
    vals_l = {"SQ_LDS_IDX_ACTIVE": 0.4 * cyc * 256, "SQ_LDS_BANK_CONFLICT": 0.0, "SQ_INSTS_LDS": 1.5 * mfma,
              "SQ_WAIT_INST_LDS": 0.05 * 0.99 * cyc * 256, "SQ_WAIT_INST_ANY": 0.2 * 0.99 * cyc * 256,
              "SQ_ACTIVE_INST_VALU": 0.3 * 0.99 * cyc * 256, "GRBM_GUI_ACTIVE": 8 * cyc}

    def rows(vals):
        return [dict(Dispatch_Id=7, Kernel_Name=name, Counter_Name=c, Counter_Value=v / 2,
                     Start_Timestamp=1000, End_Timestamp=1000 + ns) for c, v in vals.items() for _ in range(2)]

    _write_run(tmp_path / "m", rows(vals_m))
    _write_run(tmp_path / "l", rows(vals_l))
    rec = mfma_util.main(["x", "synthetic", str(tmp_path / "m"), str(tmp_path / "l")], out_dir=str(tmp_path))
    k = rec["kernels"]["bwd_dkdv"]
    assert k["sclk_ghz"] == pytest.approx(sclk)
    assert k["mfma_busy"] == pytest.approx(busy)
    assert k["mfma_busy_from_insts"] == pytest.approx(busy)
    assert k["frac_of_peak_executed"] == pytest.approx(busy * sclk / 2.4)
    assert k["cu_occupied"] == pytest.approx(0.99)
    assert k["waves_per_busy_cu_quad"] == pytest.approx(1.0)
    assert k["lds_active"] == pytest.approx(0.4)
    assert k["lds_insts_per_mfma"] == pytest.approx(1.5)
    assert k["sq_wait_inst_any_share"] == pytest.approx(0.2)
    assert os.path.exists(tmp_path / "mfma_utilization_synthetic.json")
