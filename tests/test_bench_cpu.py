"""Host logic of bench.py (no GPU): the one-GPU contract, the rocprofv3
summarizers that pick the benchmark's launches out of a trace or a counter
run by kernel name and grid size, and the fingerprint that keeps stored HBM
counters from being reported for work they were not taken on."""

import csv
import os
import subprocess
import sys

import bench
from synthetic_checkpoint.workloads import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
W = "tiny_fsdp2_to_tp2"


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "single MI355X" in r.stderr and r.stdout == ""


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def test_trace_summary_picks_launches_by_name_and_grid(tmp_path):
    grids, recv_bytes = bench._launch_grids(WORKLOADS[W])
    (pack_x, _), _, pack_alg = grids["pack"]
    (unpack_x, _), _, _ = grids["unpack"]
    assert pack_x != unpack_x  # the two launches are told apart by their grids
    name = "wb::wb_tasks_kernel(wb::Task const*, unsigned long const*, char const*, char const*, unsigned int)"
    rows = [(name, pack_x, 1000, 1000 + d) for d in (6000, 8000)]          # pack: 6 and 8 us
    rows += [(name, unpack_x, 5000, 5000 + d) for d in (4000, 5000, 6000)]  # unpack: 4, 5, 6 us
    rows += [(name, 64, 0, 10 ** 6)]                                        # another rank's launch
    rows += [("__amd_rocclr_copyBuffer", 1 << 20, 0, d) for d in (100, 9000, 9500, 10000)]
    path = tmp_path / "trace.csv"
    _write(path, ["Kernel_Name", "Grid_Size_X", "Start_Timestamp", "End_Timestamp"], rows)
    got = bench.summarize_trace(W, str(path))
    assert got["pack"]["launches"] == 2 and got["pack"]["avg_us"] == 7.0
    assert got["pack"]["GB/s_at_avg"] == round(sum(pack_alg) / 7000, 1)
    assert got["unpack"] == {"launches": 3, "avg_us": 5.0, "min_us": 4.0, "max_us": 6.0,
                             "GB/s_at_avg": got["unpack"]["GB/s_at_avg"]}
    assert "unpack_fp8" not in got                         # the tiny rollout has no fp8 tensors
    assert got["device_copy"] == {"launches": 3, "avg_us": 9.5}  # the three timed copies


def test_counter_summary_calibrates_on_the_copy(tmp_path):
    grids, recv_bytes = bench._launch_grids(WORKLOADS[W])
    copy_bytes = min(recv_bytes, 16 << 30)
    (_, unpack_total), _, alg = grids["unpack"]
    name = "wb::wb_tasks_kernel(args)"
    header = ["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"]
    # FETCH_SIZE counts half of what is read, WRITE_SIZE all that is written
    # (as on this part): the summary must scale each back by the copy's reading
    fetch = [("__amd_rocclr_copyBuffer", 4096, "FETCH_SIZE", copy_bytes / 2 / 1024)] * 3
    fetch += [(name, unpack_total, "FETCH_SIZE", alg[0] / 2 / 1024)] * 2
    write = [("__amd_rocclr_copyBuffer", 4096, "WRITE_SIZE", copy_bytes / 1024)] * 3
    write += [(name, unpack_total, "WRITE_SIZE", alg[1] / 1024)] * 2
    _write(tmp_path / "f.csv", header, fetch)
    _write(tmp_path / "w.csv", header, write)
    got = bench.summarize_counters(W, str(tmp_path / "f.csv"), str(tmp_path / "w.csv"))
    assert got["calibration"]["FETCH_SIZE"]["factor"] == 0.5 and got["calibration"]["WRITE_SIZE"]["factor"] == 1.0
    k = got["kernels"]["unpack"]
    assert k["dispatches"] == 2 and k["hbm_read_bytes"] == alg[0] and k["hbm_write_bytes"] == alg[1]
    assert k["hbm_bytes_per_launch"] == k["algorithmic_bytes"] == sum(alg)
    assert got["work_fingerprint"] == bench.work_fingerprint(W)


def test_fingerprint_follows_the_work_tables(monkeypatch):
    base = bench.work_fingerprint(W)
    monkeypatch.setenv("WB_TASK_BYTES", "4096")  # other work items, other grids
    assert bench.work_fingerprint(W) != base
    monkeypatch.delenv("WB_TASK_BYTES")
    assert bench.work_fingerprint(W) == base
    assert bench.work_fingerprint("llama3_8b_fsdp8_to_tp1") != base



def test_trace_summary_reports_launch_resources(tmp_path):
    grids, _ = bench._launch_grids(WORKLOADS[W])
    (unpack_x, _), _, _ = grids["unpack"]
    name = "wb::wb_tasks_kernel(args)"
    header = ["Kernel_Name", "Grid_Size_X", "Start_Timestamp", "End_Timestamp", "Workgroup_Size",
              "Arch_VGPR_Count", "LDS_Block_Size"]
    _write(tmp_path / "t.csv", header, [(name, unpack_x, 0, 5000, 64, 56, 4224)] * 2)
    got = bench.summarize_trace(W, str(tmp_path / "t.csv"))
    assert got["unpack"]["resources"] == {"Workgroup_Size": 64, "Arch_VGPR_Count": 56, "LDS_Block_Size": 4224}


def test_metric_summary_averages_per_launch(tmp_path):
    grids, _ = bench._launch_grids(WORKLOADS[W])
    (_, unpack_total), _, _ = grids["unpack"]
    (_, pack_total), _, _ = grids["pack"]
    name = "wb::wb_tasks_kernel(args)"
    rows = [(name, unpack_total, "MeanOccupancyPerCU", v) for v in (10.0, 12.0)]
    rows += [(name, pack_total, "MeanOccupancyPerCU", 20.0), (name, pack_total, "OtherMetric", 99.0)]
    _write(tmp_path / "m.csv", ["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"], rows)
    got = bench.summarize_metric(W, "MeanOccupancyPerCU", str(tmp_path / "m.csv"))
    assert got["kernels"]["unpack"] == {"dispatches": 2, "mean": 11.0}
    assert got["kernels"]["pack"] == {"dispatches": 1, "mean": 20.0}


def test_run_workload_keeps_the_workload_name():
    """run_workload reports config.workload and looks up stored counters by
    its `name` argument: nothing in its body may bind that name again (a loop
    variable of that name once made the line report the workload as
    "unpack")."""
    import ast

    tree = ast.parse(open(os.path.join(ROOT, "bench.py")).read())
    fn = next(n for n in ast.walk(tree) if isinstance(n, ast.FunctionDef) and n.name == "run_workload")
    assert [a.arg for a in fn.args.args][:2] == ["args", "name"]
    rebound = [n.lineno for n in ast.walk(fn) if isinstance(n, ast.Name) and n.id == "name"
               and isinstance(n.ctx, (ast.Store, ast.Del))]
    assert rebound == []
