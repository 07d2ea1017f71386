"""Host logic of bench.py: the rocprofv3 summaries (kernel table, counter traffic scaled by the
copy calibration, utilisation), the traffic lookup keyed by the kernel sources, the valid-token
counts of the PSABlock workload, and the one-GPU contract."""
import csv
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from workloads import get_config  # noqa: E402

COLS = ["Kernel_Name", "Counter_Name", "Counter_Value"]


def write_counters(path, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=COLS)
        w.writeheader()
        for name, counter, value in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value})


def test_counter_summary_scales_by_the_copy(tmp_path):
    k = "void psa::psa_pair_kernel<128, 128, true, false>(...)"
    write_counters(tmp_path / "f", [("__amd_rocclr_copyBuffer", "FETCH_SIZE", 524288), (k, "FETCH_SIZE", 1000),
                                    (k, "FETCH_SIZE", 3000)])
    write_counters(tmp_path / "w", [("__amd_rocclr_copyBuffer", "WRITE_SIZE", 1048576), (k, "WRITE_SIZE", 10)])
    md = bench.summarise_counters(str(tmp_path / "f"), str(tmp_path / "w"), 1024)
    vals = dict(l.split(": ", 1) for l in md.splitlines() if l.startswith(("traffic_bytes", "source_hash")))
    # fetch: mean 2000 KiB x scale 2, write: 10 KiB x scale 1
    assert float(vals["traffic_bytes_per_launch"]) == (2000 * 2 + 10) * 1024
    assert vals["source_hash"] == bench.source_hash()


def test_recorded_traffic_follows_the_sources(tmp_path, monkeypatch):
    md = tmp_path / "c.md"
    md.write_text("traffic_bytes_per_launch: 123\nsource_hash: %s\n" % bench.source_hash())
    monkeypatch.setattr(bench, "COUNTERS_MD", str(md))
    assert bench.recorded_traffic() == 123.0
    md.write_text("traffic_bytes_per_launch: 123\nsource_hash: 0000\n")
    assert bench.recorded_traffic() is None
    monkeypatch.setattr(bench, "COUNTERS_MD", str(tmp_path / "missing.md"))
    assert bench.recorded_traffic() is None


def test_kernel_table_and_utilisation(tmp_path):
    trace = tmp_path / "t"
    os.makedirs(trace)
    with open(trace / "run_kernel_stats.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs",
                                          "MaxNs"])
        w.writeheader()
        w.writerow({"Name": "void psa::psa_pair_kernel<128, 128, false, false>(x)", "Calls": 2, "TotalDurationNs": 2e8,
                    "AverageNs": 1e8, "Percentage": 100.0, "MinNs": 1e8, "MaxNs": 1e8})
    table = bench.kernel_stats_table(str(trace))
    assert "| psa::psa_pair_kernel<128, 128, false, false> | 2 | 200000.0 | 100000.0 |" in table
    k = "void psa::psa_pair_kernel<128, 128, false, false>(x)"
    cyc = 1.9e8                                   # per XCD: 1.9 GHz over 0.1 s
    write_counters(tmp_path / "sq", [(k, "GRBM_GUI_ACTIVE", 8 * cyc), (k, "SQ_VALU_MFMA_BUSY_CYCLES", 0.5 * cyc * 1024),
                                     (k, "SQ_INSTS_MFMA", 0.5 * cyc * 1024 / 32), (k, "SQ_INSTS_VALU", cyc * 64),
                                     (k, "SQ_ACTIVE_INST_VALU", 0.1 * cyc * 256), (k, "SQ_LDS_BANK_CONFLICT", 0)])
    write_counters(tmp_path / "tcc", [(k, "TCC_HIT_sum", 90), (k, "TCC_MISS_sum", 10)])
    # the plan's pairing kernels share the prefix of the pair engine but are not attention
    write_counters(tmp_path / "sq" / "plan", [("void psa::psa_pairing_kernel(x)", "SQ_INSTS_MFMA", 0),
                                              ("void psa::psa_paircount_kernel(x)", "SQ_INSTS_MFMA", 0)])
    rows = bench.utilisation_rows(str(tmp_path / "sq"), str(tmp_path / "tcc"), str(trace), "x")
    assert len(rows) == 1
    row = rows[0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[2:6] == ["100.00", "1.90", "0.500", "32.0"] and cells[-1] == "0.900"
    # SQ_INSTS_VALU counts the MFMAs: cyc * 64 VALU over cyc * 16 MFMA = 4 per MFMA, 3 others
    assert cells[6] == "3.00"


def test_hbm_and_wait_summaries(tmp_path):
    trace = tmp_path / "t"
    os.makedirs(trace)
    with open(trace / "run_kernel_stats.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs",
                                          "MaxNs"])
        w.writeheader()
        w.writerow({"Name": "void psa::psa_pair_kernel<128, 128, true, false>(x)", "Calls": 1, "TotalDurationNs": 1e7,
                    "AverageNs": 1e7, "Percentage": 100.0, "MinNs": 1e7, "MaxNs": 1e7})
    k = "void psa::psa_pair_kernel<128, 128, true, false>(x)"
    write_counters(tmp_path / "f", [("__amd_rocclr_copyBuffer", "FETCH_SIZE", 524288), (k, "FETCH_SIZE", 1e6)])
    write_counters(tmp_path / "w", [("__amd_rocclr_copyBuffer", "WRITE_SIZE", 1048576), (k, "WRITE_SIZE", 1e4)])
    cfg = get_config("tiny")
    row = bench.hbm_rows(str(tmp_path / "f"), str(tmp_path / "w"), str(trace), cfg, 1024)[0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    rd, wr = 1e6 * 1024 * 2, 1e4 * 1024            # fetch scale 2, write scale 1
    assert cells[0] == "tiny" and cells[2] == "10.00"
    assert float(cells[3]) == round(rd / 1e9, 1) and float(cells[4]) == round(wr / 1e9, 3)
    assert float(cells[5]) == round(4 * 2 * (2 * 1024 * 64) / 1e9, 3)   # Q, K, V, O: 2 B x 2 heads x N x d
    assert float(cells[6]) == round((rd + wr) / 1e-2 / 1e9)
    write_counters(tmp_path / "q", [(k, "GRBM_GUI_ACTIVE", 8 * 1000.0), (k, "SQ_WAVE_CYCLES", 512 * 1000.0),
                                    (k, "SQ_ACTIVE_INST_ANY", 512 * 300.0), (k, "SQ_WAIT_ANY", 512 * 400.0),
                                    (k, "SQ_WAIT_INST_ANY", 512 * 300.0), (k, "SQ_ACTIVE_INST_SCA", 512 * 50.0),
                                    (k, "SQ_ACTIVE_INST_MISC", 512 * 10.0)])
    cells = [c.strip() for c in bench.wait_rows(str(tmp_path / "q"), "x")[0].strip("|").split("|")]
    assert cells[2:] == ["2.00", "0.300", "0.400", "0.300", "0.050", "0.010"]


def test_group_tokens_of_the_psablock_workload():
    cfg = get_config("wan14b_3d")
    cnt = bench.group_tokens(cfg)
    assert cnt.shape == (7 * 6 * 5,) and cnt.sum() == 21 * 45 * 80
    assert set(np.unique(cnt)) == {3 * 8 * 16, 3 * 5 * 16}      # the last PSABlock row holds 5 of 8 rows


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr
