"""The summariser behind profiles/: on small synthetic rocprofv3 CSVs, the HBM traffic of a
kernel is its FETCH_SIZE and WRITE_SIZE (KiB per dispatch) scaled by what the same counters read
for a device copy of known size; only the optimisation steps' dispatches (before the first
harden) count; the MFMA summary turns GRBM_GUI_ACTIVE, SQ_VALU_MFMA_BUSY_CYCLES and
SQ_INSTS_VALU_MFMA_MOPS_BF16 into the clock, the busy share and the bf16 rate."""
import csv
import json

import pytest

from paper_2604_18556_amd import rocprof_summary as rs

COLS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id",
        "Grid_Size", "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size",
        "Scratch_Size", "VGPR_Count", "Accum_VGPR_Count", "SGPR_Count", "Counter_Name",
        "Counter_Value", "Start_Timestamp", "End_Timestamp"]
BW = "void gsq::(anonymous namespace)::k_backward<8, false, true, false, 0, false>(gsq::ElemArgs)"
CT = "gsq::(anonymous namespace)::k_contract_bf16(unsigned short const*, ...)"
HD = "void gsq::(anonymous namespace)::k_harden<8, 0>(gsq::ElemArgs, int, int, unsigned char*, void*)"
CP = "__amd_rocclr_copyBuffer"


def _counters(path, rows):
    """rows: (dispatch, kernel, counter, value[, start_ns, end_ns])."""
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, COLS)
        w.writeheader()
        for r in rows:
            d, k, c, v = r[:4]
            t0, t1 = (r[4], r[5]) if len(r) > 4 else (0, 1)
            w.writerow({**{c_: 0 for c_ in COLS}, "Dispatch_Id": d, "Kernel_Name": k,
                        "Counter_Name": c, "Counter_Value": v, "Start_Timestamp": t0,
                        "End_Timestamp": t1})


def test_traffic_scales_by_the_copy_and_counts_only_the_steps(tmp_path, capsys):
    copy_bytes = 1 << 30
    cf, cw = tmp_path / "cf.csv", tmp_path / "cw.csv"
    # the copy reads 2^30 bytes; FETCH_SIZE reports half of them, WRITE_SIZE all
    _counters(cf, [(1, CP, "FETCH_SIZE", copy_bytes / 1024 / 2)])
    _counters(cw, [(1, CP, "WRITE_SIZE", copy_bytes / 1024)])
    f, w = tmp_path / "f.csv", tmp_path / "w.csv"
    # two step dispatches of the backward (1000 and 3000 KiB fetched), then a harden and a
    # backward-named dispatch after it that must not count
    _counters(f, [(1, BW, "FETCH_SIZE", 1000.0), (2, BW, "FETCH_SIZE", 3000.0),
                  (3, HD, "FETCH_SIZE", 7.0), (4, BW, "FETCH_SIZE", 1e9)])
    _counters(w, [(1, BW, "WRITE_SIZE", 500.0), (2, BW, "WRITE_SIZE", 1500.0),
                  (3, HD, "WRITE_SIZE", 7.0), (4, BW, "WRITE_SIZE", 1e9)])
    js = tmp_path / "traffic.json"
    rs.main(["traffic", "--fetch", str(f), "--write", str(w), "--copy-fetch", str(cf),
             "--copy-write", str(cw), "--copy-bytes", str(copy_bytes), "--kernel", "backward",
             "--workload", "wl", "--json", str(js), "--cmd", "cmd"])
    rec = json.load(open(js))["backward:wl"]
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    # mean over the two step dispatches: fetch 2000 KiB x 2, write 1000 KiB x 1
    assert rec["fetch_bytes"] == pytest.approx(2000 * 2 * 1024)
    assert rec["write_bytes"] == pytest.approx(1000 * 1024)
    assert rec["bytes_per_launch"] == pytest.approx((4000 + 1000) * 1024)
    assert rec["source"] == "gsq_elem.hip" and len(rec["source_sha256"]) == 64
    assert "traffic" in capsys.readouterr().out


def test_mfma_summary_clock_busy_share_and_rate(tmp_path, capsys):
    agent = tmp_path / "agent.csv"
    with open(agent, "w", newline="") as f:
        w = csv.DictWriter(f, ["Agent_Type", "Num_Xcc", "Simd_Count"])
        w.writeheader()
        w.writerow({"Agent_Type": "CPU", "Num_Xcc": 0, "Simd_Count": 0})
        w.writerow({"Agent_Type": "GPU", "Num_Xcc": 8, "Simd_Count": 1024})
    c = tmp_path / "c.csv"
    t = 1_000_000                       # 1 ms per dispatch
    active = 8 * 1.8e9 * 1e-3           # 8 XCCs at 1.8 GHz for 1 ms
    busy = 0.7 * active / 8 * 1024      # matrix cores busy 70 % of the SIMD cycles
    mops = 1.0e12 / 512                 # 1 TFLOP in the dispatch -> 1 PFLOP/s
    rows = []
    for d in (1, 2, 3):
        for name, v in (("GRBM_GUI_ACTIVE", active), ("SQ_VALU_MFMA_BUSY_CYCLES", busy),
                        ("SQ_INSTS_VALU_MFMA_MOPS_BF16", mops), ("SQ_LDS_BANK_CONFLICT", 0)):
            rows.append((d, CT, name, v, 0, t))
    _counters(c, rows)
    rs.main(["mfma", str(c), "--agent", str(agent), "--cmd", "cmd"])
    line = [l for l in capsys.readouterr().out.splitlines() if l.startswith("contract")][0].split()
    # kernel calls n us clock busy GFLOP TFLOP/s frac frac@clock conflicts
    assert float(line[3]) == pytest.approx(1000.0)
    assert float(line[4]) == pytest.approx(1.8, abs=1e-3)
    assert float(line[5]) == pytest.approx(0.7, abs=1e-3)
    assert float(line[7]) == pytest.approx(1000.0, rel=1e-3)
    assert float(line[8]) == pytest.approx(0.4, abs=1e-3)
    assert float(line[9]) == pytest.approx(0.4 * 2.4 / 1.8, abs=1e-3)
