"""Host-side logic of bench.py: the probe-count replay of the tile lookup's
schedule and the reducers that turn rocprofv3 csv output into the summaries
under profiles/ (checked here on small synthetic csv files, no GPU)."""
import csv
import json
import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from workloads import CONFIGS, make_workload, scaled  # noqa: E402


def literal_probe_count(cfg, w, X):
    """The tile lookup's schedule, position by position: lengths 3 and 2, then
    5 and 4 behind a flagged length-3 suffix, then 7 and 6 behind a flagged
    length-5 suffix, each only where it fits the window."""
    K = min(cfg.max_n, cfg.max_len)
    rows = list(zip(w.fgrams.tolist(), w.lengths.tolist()))
    ends3 = {tuple(r[L - 3:L]) for r, L in rows if L >= 4}
    ends5 = {tuple(r[L - 5:L]) for r, L in rows if L >= 6}
    total = 0
    for b in range(X.shape[0]):
        for t in range(X.shape[1]):
            top = min(K, t + 1)
            if K <= 2:
                total += top >= 2
                continue
            total += (top >= 3) + (top >= 2)
            if K >= 4 and top >= 3 and tuple(X[b, t - 2:t + 1]) in ends3:
                total += (top >= 5) + (top >= 4)
                if K >= 6 and top >= 5 and tuple(X[b, t - 4:t + 1]) in ends5:
                    total += (top >= 7) + (top >= 6)
    return total / X.size


@pytest.mark.parametrize("name,max_n,max_len", [("c3_10m_k5", 5, 5), ("c2_1m", 3, 3),
                                                 ("c3_10m_k5", 7, 7), ("c3_10m_k5", 2, 5),
                                                 ("c3_10m_k5", 6, 5)])
def test_probe_replay_matches_literal_schedule(name, max_n, max_len):
    cfg = scaled(CONFIGS[name], n_fgrams=3000, B=3, T=200, max_n=max_n, max_len=max_len, V=40)
    w = make_workload(cfg)
    got = bench.probes_per_position(cfg, w, w.tokens)
    assert got == pytest.approx(literal_probe_count(cfg, w, w.tokens), abs=1e-12)
    assert 0 < got <= max(min(max_n, max_len) - 1, 1)


def _write_csv(path, fields, rows):
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=fields)
        wr.writeheader()
        for r in rows:
            wr.writerow(r)


def _plan(steps=3):
    P = bench.Plan()
    P.add("pipelined_first_lookup", "k_lookup")
    P.add("pipelined_timed", "k_pipelined", steps)
    for _ in range(steps):
        P.add("serial_timed", "k_lookup")
        P.add("serial_timed", "k_gather")
    P.add("noreuse_timed", "k_pipelined", steps)
    P.add("uniform_timed", "k_gather", steps)
    return P.entries


KNAMES = {"k_lookup": "void scone::(anonymous namespace)::k_lookup<16, 2>(int)",
          "k_pipelined": "void scone::(anonymous namespace)::k_pipelined<16, 2, 4>(int)",
          "k_gather": "void scone::(anonymous namespace)::k_gather_rows<4>(int)",
          "k_insert": "void scone::(anonymous namespace)::k_insert<16>(int)",
          "copy": "__amd_rocclr_copyBuffer", "fill": "void at::native::fill(int)"}


def test_trace_reducer_takes_each_phase_from_its_own_dispatches(tmp_path):
    entries = _plan()
    # a build kernel and a torch kernel first, then the plan's dispatches with
    # durations that encode their phase
    dur = {"pipelined_timed": 1000, "serial_timed": 0, "noreuse_timed": 3000,
           "uniform_timed": 5000, "pipelined_first_lookup": 7}
    rows, did = [], 0
    for name in ("k_insert", "fill"):
        did += 1
        rows.append({"Kernel_Name": KNAMES[name], "Dispatch_Id": did, "Start_Timestamp": 0,
                     "End_Timestamp": 99, "Grid_Size_X": 1, "Workgroup_Size_X": 1,
                     "VGPR_Count": 1, "LDS_Block_Size": 0})
    for phase, kern in entries:
        did += 1
        ns = dur[phase] + (200 if kern == "k_gather" and phase == "serial_timed" else 0) + \
            (100 if kern == "k_lookup" and phase == "serial_timed" else 0)
        rows.append({"Kernel_Name": KNAMES[kern], "Dispatch_Id": did, "Start_Timestamp": 10,
                     "End_Timestamp": 10 + ns, "Grid_Size_X": 64, "Workgroup_Size_X": 256,
                     "VGPR_Count": 12, "LDS_Block_Size": 0})
    trace = tmp_path / "run_kernel_trace.csv"
    _write_csv(trace, list(rows[0].keys()), rows)
    plan = tmp_path / "plan.json"
    json.dump({"config": "c3_10m_k5", "workload": "w", "steps": 3, "warmup": 0,
               "copy_calibration_mib": 0, "entries": entries}, open(plan, "w"))
    out = tmp_path / "trace.md"
    bench.reduce_trace(str(trace), str(plan), None, str(out), "rocprofv3 ... -- python bench.py")
    text = out.read_text()
    assert "pipelined_timed   k_pipelined<16, 2, 4>" in text and "mean      1.00 us" in text
    assert "noreuse_timed" in text and "mean      3.00 us" in text
    assert "uniform_timed" in text and "mean      5.00 us" in text
    assert "serial_timed      k_gather_rows<4>" in text and "mean      0.20 us" in text
    # a csv that disagrees with the plan is refused
    rows[3]["Kernel_Name"] = KNAMES["k_gather"]
    _write_csv(trace, list(rows[0].keys()), rows)
    with pytest.raises(SystemExit):
        bench.reduce_trace(str(trace), str(plan), None, str(out), "")


def test_counter_reducer_calibrates_and_averages_timed_dispatches(tmp_path):
    entries = _plan()
    cfg = CONFIGS["c3_10m_k5"]
    mib = 4
    files = {}
    for ctr, copy_val, per in (("FETCH_SIZE", mib * 1024 / 2, 2.0), ("WRITE_SIZE", mib * 1024, 1.0)):
        rows, did = [], 0
        for phase, kern in entries:
            did += 1
            v = {"pipelined_timed": 500.0, "noreuse_timed": 600.0, "serial_timed": 300.0,
                 "uniform_timed": 700.0, "pipelined_first_lookup": 1.0}[phase]
            if kern == "k_lookup":
                v = 10.0
            rows.append({"Dispatch_Id": did, "Kernel_Name": KNAMES[kern], "Grid_Size": 64,
                         "Counter_Name": ctr, "Counter_Value": v})
        for k in range(5):   # calibration copies (the small copy before them is ignored)
            did += 1
            rows.append({"Dispatch_Id": did, "Kernel_Name": KNAMES["copy"], "Grid_Size": 4096,
                         "Counter_Name": ctr, "Counter_Value": copy_val})
        rows.insert(0, {"Dispatch_Id": 0, "Kernel_Name": KNAMES["copy"], "Grid_Size": 16,
                        "Counter_Name": ctr, "Counter_Value": 3.0})
        files[ctr] = tmp_path / f"{ctr}.csv"
        _write_csv(files[ctr], list(rows[0].keys()), rows)
    plan = tmp_path / "plan.json"
    json.dump({"config": "c3_10m_k5", "workload": "w", "steps": 3, "warmup": 0,
               "copy_calibration_mib": mib, "entries": entries}, open(plan, "w"))
    bench.reduce_counters(str(files["FETCH_SIZE"]), str(files["WRITE_SIZE"]), str(plan),
                          "fetch cmd", "write cmd", str(tmp_path))
    rec = {}
    for key in ("pipelined", "gather"):
        text = (tmp_path / f"{key}_c3_10m_k5_traffic.md").read_text()
        line = [ln for ln in text.splitlines() if ln.startswith("TRAFFIC ")][0]
        rec[key] = json.loads(line[len("TRAFFIC "):])
        assert "include last-level-cache hits" in text.replace("\n", " ")
    # FETCH scaled by 2, WRITE by 1, per launch in bytes
    assert rec["pipelined"]["traffic_bytes_per_launch"] == (500 * 2 + 500) * 1024
    assert rec["pipelined"]["noreuse_traffic_bytes_per_launch"] == (600 * 2 + 600) * 1024
    assert rec["gather"]["traffic_bytes_per_launch"] == (300 * 2 + 300) * 1024
    assert rec["gather"]["uniform_traffic_bytes_per_launch"] == (700 * 2 + 700) * 1024
    assert rec["pipelined"]["source_sha1"] == bench.source_sha(*bench.KERNEL_SOURCES["pipelined"])
    assert cfg.n_tok > 0


def test_kernel_sources_names_the_defining_files_and_their_headers():
    srcs = bench.kernel_sources({"k_lookup<16, 2>", "k_mark<16>"})
    assert {"lookup.hip", "tile_lookup.h", "table_build.hip", "scone_internal.h",
            "runtime.hip"} <= set(srcs)
    assert "gemm_bf16.h" not in srcs and "discover.hip" not in srcs
    assert "gemm_bf16.h" in bench.kernel_sources({"k_gemm<1, 256, 256, 4, 2, false>"})
