"""Host-side logic of bench.py, on the CPU: the one-GPU guard, the HBM-traffic
summary built from rocprofv3 FETCH_SIZE / WRITE_SIZE passes (calibrated by a copy
kernel of known size, stamped with the kernel source's hash) and the split of a
kernel trace into the taus of the bench run.  Inputs are small fabricated CSVs in
rocprofv3's column layout; outputs go to a temporary directory."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

COPY = "__amd_rocclr_copyBuffer"
DQ = "void mala::mala_bwd_dq_kernel<128>(mala::BwdParams)"
DKDV = "void mala::mala_bwd_dkdv_kernel<128>(mala::BwdParams)"
OTHER = "void other_kernel(float*)"


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "4"})])
def test_more_than_one_gpu_exits_with_a_message(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + argv,
                       capture_output=True, text=True, timeout=120,
                       env=dict(os.environ, **env))
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def _write_counters(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                           "Counter_Value"])
        w.writeheader()
        for d, k, v in rows:
            w.writerow(dict(Dispatch_Id=d, Kernel_Name=k, Counter_Name="X", Counter_Value=v))


@pytest.fixture
def sandbox(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "source_sha", lambda path: "stamp-" + os.path.basename(path))
    return tmp_path


def test_traffic_summary_scales_each_counter_by_the_copy_kernel(sandbox):
    fetch, write = sandbox / "fetch.csv", sandbox / "write.csv"
    # the 512 MiB copy reads 256 Ki KiB by FETCH_SIZE (scale 2) and 512 Ki KiB by
    # WRITE_SIZE (scale 1); a dispatch's rows (one per counter instance) are summed
    # first, then dispatches of one kernel are averaged
    _write_counters(fetch, [(1, COPY, 131072.0), (1, COPY, 131072.0),
                            (2, DQ, 60.0), (2, DQ, 40.0), (3, DQ, 300.0),
                            (4, DKDV, 1000.0), (5, OTHER, 7.0)])
    _write_counters(write, [(1, COPY, 524288.0), (2, DQ, 10.0), (3, DQ, 30.0),
                            (4, DKDV, 5.0), (5, OTHER, 3.0)])
    bench.summarize_counters(str(fetch), str(write), "bwd")
    with open(sandbox / "profiles" / "mala_bwd_traffic_128k.json") as fh:
        d = json.load(fh)
    assert d["fetch_scale"] == 2.0 and d["write_scale"] == 1.0
    dq = (200.0 * 2.0 + 20.0 * 1.0) * 1024
    dkdv = (1000.0 * 2.0 + 5.0 * 1.0) * 1024
    assert d["kernels"][DQ]["bytes"] == dq
    assert d["kernels"][DKDV]["bytes"] == dkdv
    assert OTHER not in d["kernels"] and COPY not in d["kernels"]
    assert d["bytes_per_launch"] == dq + dkdv
    assert d["source_sha"] == "stamp-mala_bwd.hip"
    # the bench reads the figure back only while the kernel source is unchanged
    assert bench.traffic_from_profiles("/x/mala_bwd.hip") == dq + dkdv
    assert bench.traffic_from_profiles("/x/changed.hip") is None


def test_traffic_summary_needs_the_copy_kernel(sandbox):
    fetch, write = sandbox / "fetch.csv", sandbox / "write.csv"
    _write_counters(fetch, [(1, DQ, 1.0)])
    _write_counters(write, [(1, DQ, 1.0)])
    with pytest.raises(SystemExit):
        bench.summarize_counters(str(fetch), str(write), "bwd")


def test_trace_summary_splits_the_dispatches_by_tau(sandbox):
    # 15 dispatches of a backward kernel: 6 at tau = 1e-4 (1 ms), 3 at tau = 0
    # (2 ms), 3 at tau = 1 (3 ms), then 3 calls with the statistics (10 ms, left
    # out of the means); a kernel with another count is reported over all calls
    path = sandbox / "trace.csv"
    t, rows = 0, []
    for i, ms in enumerate([1] * 6 + [2] * 3 + [3] * 3 + [10] * 3):
        rows.append(dict(Kernel_Name=DKDV, Start_Timestamp=t, End_Timestamp=t + ms * 10 ** 6))
        t += 20 * 10 ** 6
    rows.append(dict(Kernel_Name=OTHER, Start_Timestamp=t, End_Timestamp=t + 5 * 10 ** 5))
    rows.reverse()   # the summary orders by start time itself
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        w.writerows(rows)
    bench.summarize_trace(str(path))
    text = (sandbox / "profiles" / "kernels_128k_train_and_decode.md").read_text()
    assert "| `%s` | 15 | 1.000 | 2.000 | 3.000 | 51.000 |" % DKDV in text
    assert "| `%s` | 1 | 0.500 (all) | | | 0.500 |" % OTHER in text
