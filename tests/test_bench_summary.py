"""CPU-only checks of bench.py's profile summary: the gate/up launches are found in a kernel
trace, the counter runs' values are scaled by the calibration copy and split by row count,
and the bytes per launch written into the summary are the ones bench.py reads back."""
import csv
import json
import os

import pytest

import bench

WL = "llama3-8b-b1-c2048"  # batch 1: the timed step selects with select_length_kernel
GATEUP = "void lsv::gemm_kernel<unsigned short, 2, 2>(lsv::GemmArgs)"
NORM = "void lsv::rmsnorm_kernel<unsigned short>(lsv::NormArgs)"
SELECT = "void lsv::select_length_kernel(lsv::SelectArgs)"
COPY = "__amd_rocclr_copyBuffer"


def write_json(d, obj):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "bench.json"), "w") as f:
        f.write("some progress line\n" + json.dumps(obj) + "\n")


def write_csv(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def trace_run(d, warmup, steps, n_roof, rows):
    """A kernel trace: the selections before the timed region, `steps` timed replays (select,
    gate/up 10 us, rmsnorm 5 us), then the roofline steps (a select and n_roof gate/up launches
    of 40 us)."""
    rows_csv, t, i = [], 0, 0

    def k(name, us):
        nonlocal t, i
        rows_csv.append([i, name, t, t + int(us * 1000)])
        t += int(us * 1000) + 1000
        i += 2  # leave a gap so no two launches share consecutive dispatch ids
    for _ in range(3 + 1 + warmup):
        k(SELECT, 5)
    for _ in range(steps):
        k(SELECT, 5)
        k(GATEUP, 10)
        k(NORM, 5)
    k(SELECT, 5)
    for _ in range(n_roof):
        k(GATEUP, 40)
    write_csv(os.path.join(d, "t_kernel_trace.csv"),
              ["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"], rows_csv)
    write_json(d, {"config": {"workload": WL, "batch": 1, "gamma": rows - 1, "context": 2048},
                   "roofline": {"rows": rows, "launches_timed": n_roof, "avg_launch_us": 41.0, "frac": 0.7},
                   "steps": steps, "warmup": warmup, "ms_per_step": 0.03, "value": 300.0,
                   "step": {"hbm_frac": 0.5}})


def counter_run(d, name, gammas, per_rows, values, copy_kib):
    """A counter run: `per_rows` gate/up launches at each gamma's rows (values[gamma], KiB per
    launch), each split over two consecutive dispatches, then the calibration copy."""
    rows_csv, i = [], 0
    for g in gammas:
        for _ in range(per_rows):
            v = values[g]
            rows_csv.append([i, GATEUP, 1024, name, 0.25 * v])
            rows_csv.append([i + 1, GATEUP, 1024, name, 0.75 * v])
            rows_csv.append([i + 2, NORM, 256, name, 1.0])
            i += 4
    rows_csv.append([i, COPY, 1 << 20, name, copy_kib])
    write_csv(os.path.join(d, "c_counter_collection.csv"),
              ["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"], rows_csv)
    rows = [g + 1 for g in gammas]
    write_json(d, {"config": {"workload": WL, "counters_gammas": ",".join(map(str, gammas))},
                   "roofline": {"rows": rows[0], "rows_list": rows, "launches_per_rows": per_rows,
                                "launches_timed": per_rows * len(rows)}})


def test_summary_splits_counters_by_rows_and_scales_by_the_copy(tmp_path, monkeypatch):
    t, f, w = (str(tmp_path / x) for x in ("t", "f", "w"))
    trace_run(t, warmup=2, steps=3, n_roof=4, rows=10)
    gammas = [8, 9, 10]
    fetch = {8: 100000.0, 9: 110000.0, 10: 120000.0}
    write = {8: 50.0, 9: 60.0, 10: 70.0}
    # the copy of 256 MiB reads half its bytes in FETCH_SIZE units and all of them in WRITE_SIZE
    counter_run(f, "FETCH_SIZE", gammas, 4, fetch, (bench.CALIB_BYTES >> 10) / 2)
    counter_run(w, "WRITE_SIZE", gammas, 4, write, bench.CALIB_BYTES >> 10)
    md = bench.summarize(t, f, w)
    # the timed replays: three steps, one gate/up of 10 us and one rmsnorm of 5 us each
    assert "| `gemm_kernel<unsigned short, 2, 2>` | 1 | 10.00 | 10.0 |" in md
    assert "| `rmsnorm_kernel<unsigned short>` | 1 | 5.00 | 5.0 |" in md
    assert "4 (gemm_kernel<unsigned short, 2, 2>); kernel time 40.00 us per launch" in md
    assert "--counters-only 8,9,10 --roofline-steps 2" in md
    expect = {g + 1: (fetch[g] * 2.0 + write[g]) * 1024 for g in gammas}
    for r, v in expect.items():
        assert f"traffic_rows_{r}: {v:.0f}" in md
    assert "| **10** |" in md  # the timed step's row count is marked
    # bench.py reads those figures back while the kernel sources are unchanged, and only then
    prof = tmp_path / "profile.md"
    prof.write_text(md)
    monkeypatch.setattr(bench, "gateup_profile", lambda wl: str(prof))
    for r, v in expect.items():
        assert bench.measured_traffic(WL, r) == pytest.approx(round(v))
    assert bench.measured_traffic(WL, 12) is None
    prof.write_text(md.replace(f"source_hash: {bench.kernel_source_hash()}", "source_hash: 0000000000000000"))
    assert bench.measured_traffic(WL, 10) is None


def test_summary_refuses_counter_runs_without_the_timed_rows(tmp_path):
    t, f, w = (str(tmp_path / x) for x in ("t", "f", "w"))
    trace_run(t, warmup=1, steps=2, n_roof=2, rows=10)
    counter_run(f, "FETCH_SIZE", [4, 5], 2, {4: 1.0, 5: 1.0}, 1.0)
    counter_run(w, "WRITE_SIZE", [4, 5], 2, {4: 1.0, 5: 1.0}, 1.0)
    with pytest.raises(AssertionError, match="rows"):
        bench.summarize(t, f, w)


def test_counter_summary_keeps_the_timed_rows_of_a_multi_gamma_run(tmp_path):
    """A per-kernel counter summary of a run over gammas 8, 9, 10 averages only the verify calls
    (each opened by its embedding kernel) at the kernel-trace run's 10 rows."""
    t, f = str(tmp_path / "t"), str(tmp_path / "f")
    trace_run(t, warmup=1, steps=2, n_roof=2, rows=10)
    embed = "void lsv::embed_kernel<unsigned short>(lsv::EmbedArgs)"
    rows_csv, i = [], 0
    for g in (8, 9, 10):
        for _ in range(2):  # two calls per gamma
            for name, v in ((embed, 1.0), (GATEUP, 1000.0 * g), (NORM, 10.0 * g)):
                rows_csv.append([i, name, 1024, "FETCH_SIZE", v])
                i += 2
    rows_csv.append([i, COPY, 1 << 20, "FETCH_SIZE", bench.CALIB_BYTES >> 10])  # scale 1 KiB per unit
    write_csv(os.path.join(f, "c_counter_collection.csv"),
              ["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"], rows_csv)
    write_json(f, {"config": {"workload": WL, "counters_gammas": "8,9,10"},
                   "roofline": {"rows": 9, "rows_list": [9, 10, 11], "launches_per_rows": 2,
                                "launches_timed": 6}})
    # the trace ran 10 rows = gamma 9, the second of the run's three row counts
    md = bench.summarize_counters(t, [f])
    gu = next(l for l in md.splitlines() if l.startswith("| `gemm_kernel"))
    nm = next(l for l in md.splitlines() if l.startswith("| `rmsnorm_kernel"))
    assert gu.split("|")[2].strip() == "2" and gu.split("|")[3].strip() == f"{9000 * 1024 / 1e6:.2f} MB"
    assert nm.split("|")[3].strip() == f"{90 * 1024 / 1e6:.2f} MB"
    assert "--counters-only 8,9,10 --roofline-steps 2" in md
