"""Host-side checks of the rocprofv3 summary helper on small synthetic CSVs."""

import csv
import json

from paper_2607_27744_amd import prof_summary

_FIELDS = ["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value",
           "Start_Timestamp", "End_Timestamp"]


def _write_pass(d, counters, name="void k<true>(int)", start=1000, dur_ns=2_000_000):
    d.mkdir()
    with open(d / "x_counter_collection.csv", "w", newline="") as f:
        w = csv.DictWriter(f, _FIELDS)
        w.writeheader()
        for c, v in counters.items():
            w.writerow({"Kernel_Name": name, "Grid_Size": 256, "Counter_Name": c,
                        "Counter_Value": v, "Start_Timestamp": start,
                        "End_Timestamp": start + dur_ns})
            # another kernel that must not be counted
            w.writerow({"Kernel_Name": "other", "Grid_Size": 256, "Counter_Name": c,
                        "Counter_Value": 1, "Start_Timestamp": 0, "End_Timestamp": 1})
    with open(d / "x_agent_info.csv", "w", newline="") as f:
        w = csv.DictWriter(f, ["Agent_Type", "Cu_Count", "Simd_Per_Cu"])
        w.writeheader()
        w.writerow({"Agent_Type": "CPU", "Cu_Count": 16, "Simd_Per_Cu": 0})
        w.writerow({"Agent_Type": "GPU", "Cu_Count": 256, "Simd_Per_Cu": 4})


def test_sq_derived_figures(tmp_path, capsys):
    # 2 ms at 1.5 GHz on 256 CUs; matrix cores busy half the SIMD cycles.
    cu_cycles = 256 * 3_000_000
    _write_pass(tmp_path / "p1", {"SQ_WAVE_CYCLES": 1000, "SQ_WAIT_ANY": 250,
                                  "SQ_ACTIVE_INST_VALU": 100})
    _write_pass(tmp_path / "p2", {"SQ_BUSY_CU_CYCLES": cu_cycles,
                                  "SQ_VALU_MFMA_BUSY_CYCLES": 2 * cu_cycles})
    prof_summary.sq("k<true>", "synthetic", str(tmp_path / "p1"), str(tmp_path / "p2"))
    rec = json.loads(capsys.readouterr().out)
    assert rec["dispatches"] == 1
    assert rec["duration_ms"] == 2.0
    assert rec["clock_ghz"] == 1.5
    assert rec["mfma_busy"] == 0.5
    assert rec["wave_cycle_shares"] == {"wait_any": 0.25, "active_inst_valu": 0.1}
    assert rec["counters"]["SQ_WAIT_ANY"] == 250
