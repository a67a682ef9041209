"""The bench's rocprofv3 converters on synthetic CSV output (no GPU): the
counter scaling by the copy probe, the last dispatch per kernel, the mean of
the timed steps' launches, the source-hashed traffic records, and the L2
summary.  The summaries go to a temporary directory."""
import argparse
import csv
import json
import os

import pytest

import bench as B


def _write_csv(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as fh:
        wr = csv.DictWriter(fh, fieldnames=list(rows[0].keys()))
        wr.writeheader()
        wr.writerows(rows)


def _counters(d, name, per_kernel):
    """counter_collection.csv: per_kernel = {kernel: [values by dispatch]}."""
    rows, disp = [], 0
    for k, vals in per_kernel.items():
        for v in vals:
            disp += 1
            rows.append({"Dispatch_Id": disp, "Kernel_Name": f"void {k}(args)", "Counter_Name": name,
                         "Counter_Value": v})
    _write_csv(os.path.join(d, "x", "p_counter_collection.csv"), rows)


def _args(**kw):
    base = dict(op="step", workload=4, shards=None, steps=20, traffic_cmd="cmd", traffic_from=None,
                trace_from=None, counters_from=None)
    base.update(kw)
    return argparse.Namespace(**base)


@pytest.fixture
def out(tmp_path, monkeypatch):
    d = tmp_path / "profiles"
    monkeypatch.setattr(B, "PROFILES", str(d))
    return d


def test_traffic_scaled_by_the_copy_probe_and_hashed(tmp_path, out):
    gib_kib = (1 << 30) / 1024
    cf, cw = tmp_path / "cf", tmp_path / "cw"
    _counters(cf, "FETCH_SIZE", {"rs::k_probe_copy": [gib_kib / 2, gib_kib / 2]})  # reads half: x2
    _counters(cw, "WRITE_SIZE", {"rs::k_probe_copy": [gib_kib]})                    # x1
    f, w = tmp_path / "f", tmp_path / "w"
    # two steps: the converter takes each kernel's last dispatch
    _counters(f, "FETCH_SIZE", {"rs::k_pool<float, 16, 0, 16>": [1.0, 1000.0],
                                "rs::k_bwd_short<float, float, 16, 0, true>": [5.0, 2000.0],
                                "rs::k_bwd_long<float, 16, 0>": [300.0], "rs::k_bwd_long_finish<x>": [20.0]})
    _counters(w, "WRITE_SIZE", {"rs::k_pool<float, 16, 0, 16>": [7.0, 500.0],
                                "rs::k_bwd_short<float, float, 16, 0, true>": [9.0, 1500.0],
                                "rs::k_bwd_long<float, 16, 0>": [10.0], "rs::k_bwd_long_finish<x>": [4.0]})
    B.traffic_from(_args(traffic_from=[str(f), str(w), str(cf), str(cw)]))
    wl = "200-feat-growing-d64-adam"
    rec = json.load(open(out / f"traffic_{wl}_pool.json"))
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    assert rec["fetch_bytes"] == pytest.approx(1000.0 * 1024 * 2.0)
    assert rec["write_bytes"] == pytest.approx(500.0 * 1024)
    assert rec["kernel_source_hash"] == B.kernel_source_hash("pool")
    # the hot-key backward is its unit sums and their finish together
    rec = json.load(open(out / f"traffic_{wl}_bwd_long.json"))
    assert rec["bytes_per_launch"] == pytest.approx((300.0 + 20.0) * 1024 * 2.0 + (10.0 + 4.0) * 1024)
    md = open(out / f"traffic_{wl}.md").read()
    assert "| `rs::k_bwd_short<float, float, 16, 0, true>` | 4.1 | 1.5 |" in md  # 2000 KiB x2, 1500 KiB
    assert "fetch x2.000, write x1.000" in md


def test_trace_means_the_timed_steps_and_labels_operators(tmp_path, out):
    d = tmp_path / "t"
    rows, disp = [], 0
    for j in range(25):  # 5 warm-up launches of 1 us, then 20 of 10 us
        disp += 1
        dur = 1000 if j < 5 else 10000
        rows.append({"Dispatch_Id": disp, "Kernel_Name": "rs::k_part_dedup(args)", "Start_Timestamp": 0,
                     "End_Timestamp": dur})
    _write_csv(os.path.join(d, "x", "ids_kernel_trace.csv"), rows)
    _write_csv(os.path.join(d, "x", "ids_kernel_stats.csv"),
               [{"Name": "rs::k_part_dedup(args)", "Calls": 25, "AverageNs": 8200, "MinNs": 1000, "MaxNs": 10000,
                 "Percentage": 100.0}])
    B.trace_from(_args(op="ids-partition", shards=8, steps=20, trace_from=str(d)))
    md = open(out / "step_kernels_ids_partition_1M_8shards.md").read()
    assert "# Kernel time per call: ids_partition_1M_8shards" in md
    assert "| `rs::k_part_dedup` | 10.0 | 100.0 |" in md
    assert "--op ids-partition --shards 8 --steps 20" in md


def test_l2_summary_takes_the_last_dispatch(tmp_path, out):
    d = tmp_path / "l2"
    rows = []
    for disp, (h, m, a) in enumerate([(1e6, 1e6, 0.0), (3e6, 1e6, 2e6)], start=1):
        for name, v in (("TCC_HIT_sum", h), ("TCC_MISS_sum", m), ("TCC_ATOMIC_sum", a)):
            rows.append({"Dispatch_Id": disp, "Kernel_Name": "void rs::k_compact<256>(args)", "Counter_Name": name,
                         "Counter_Value": v})
    _write_csv(os.path.join(d, "x", "p_counter_collection.csv"), rows)
    B.counters_from(_args(workload=2, counters_from=str(d)))
    md = open(out / "l2_100-multi-hot-d32-bf16-mean-adagrad.md").read()
    assert "| `rs::k_compact<256>` | 3.0 | 1.0 | 0.75 | 2.00 |" in md


def test_ceilings_summary(tmp_path, out):
    j = tmp_path / "ceil.json"
    j.write_text('noise\n{"ceilings": {"read": {"bytes": 2147483648, "ms": 0.325, "GBps": 6607.6}}, '
                 '"peak_GBps": 8000.0}\n')
    st = tmp_path / "st"
    _write_csv(os.path.join(st, "x", "c_kernel_stats.csv"),
               [{"Name": "rs::k_probe_read(args)", "Calls": 6, "AverageNs": 326000, "MinNs": 320000,
                 "MaxNs": 340000, "Percentage": 50.0},
                {"Name": "at::native::fill(args)", "Calls": 1, "AverageNs": 1000, "MinNs": 1000, "MaxNs": 1000,
                 "Percentage": 1.0}])
    B.ceilings_from(argparse.Namespace(ceilings_from=[str(j), str(st)], traffic_cmd="cmd"))
    md = open(out / "ceilings_mi355x.md").read()
    assert "| read | 2147483648 | 0.325 | 6608 | 82.6 |" in md
    assert "| `rs::k_probe_read` | 6 | 326.00 | 320.00 | 340.00 |" in md and "fill" not in md


def test_kernel_table_joins_time_traffic_and_ceiling(tmp_path, out):
    gib_kib = (1 << 30) / 1024
    cf, cw = tmp_path / "cf", tmp_path / "cw"
    _counters(cf, "FETCH_SIZE", {"rs::k_probe_copy": [gib_kib / 2]})
    _counters(cw, "WRITE_SIZE", {"rs::k_probe_copy": [gib_kib]})
    f, w = tmp_path / "f", tmp_path / "w"
    kern = "rs::k_bwd_short<float, float, 16, 0, true>"
    _counters(f, "FETCH_SIZE", {kern: [1.0, 2e6]})   # 2e6 KiB x2 = 4.096 GB
    _counters(w, "WRITE_SIZE", {kern: [1.0, 1e6]})   # 1.024 GB
    t = tmp_path / "t"
    rows = [{"Dispatch_Id": j + 1, "Kernel_Name": f"void {kern}(args)", "Start_Timestamp": 0,
             "End_Timestamp": 1_000_000} for j in range(3)]  # 1 ms each
    _write_csv(os.path.join(t, "x", "b_kernel_trace.csv"), rows)
    c = tmp_path / "c.json"
    c.write_text('{"ceilings": {"read-modify-write of random 768-byte rows (+ index)": '
                 '{"bytes": 1, "ms": 1, "GBps": 6400.0}}, "peak_GBps": 8000.0}\n')
    B.kernels_from(_args(steps=2, kernels_from=[str(t), str(f), str(w), str(cf), str(cw), str(c)]))
    md = open(out / "kernels_200-feat-growing-d64-adam.md").read()
    # (4.096 + 1.024) GB in 1 ms = 5120 GB/s, 80% of the probe's 6400
    assert f"| `{kern}` | 1000.0 | 4096.0 | 1024.0 | 5120 | read-modify-write of random 768-byte rows (+ index) " \
           f"| 6400 | 80 |" in md
