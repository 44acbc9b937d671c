"""Host logic of the benchmark's counter summary (no GPU): HBM bytes of the
gather from two rocprofv3 --pmc runs, calibrated by the run's 1 GiB copy,
averaged over the last --steps gather dispatches, and the per-workload
lookup the bench line takes its `roofline.traffic` from."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

COLS = ["Correlation_Id", "Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
GATHER = "void gmb::(anonymous namespace)::k_gather<HIP_vector_type<unsigned int, 4u>, 16, 4>(int const*)"
COPY = "__amd_rocclr_copyBuffer"


def write_run(d, counter, dispatches, workload="hubs2m", alg=1000.0):
    """A counter_collection CSV with the given (kernel, value) dispatches in
    order, written out of order to check the summary sorts by dispatch id,
    plus the bench line the summary reads the algorithmic bytes from."""
    os.makedirs(d, exist_ok=True)
    rows = [{"Correlation_Id": i + 1, "Dispatch_Id": i + 1, "Kernel_Name": k, "Counter_Name": counter,
             "Counter_Value": v} for i, (k, v) in enumerate(dispatches)]
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=COLS)
        w.writeheader()
        for r in reversed(rows):
            w.writerow(r)
    line = {"config": {"workload": f"{workload}: a graph"}, "roofline": {"alg_bytes_per_launch": alg}}
    with open(os.path.join(d, "bench.json"), "w") as f:
        f.write("some progress output\n" + json.dumps(line) + "\n")


def summarize(fetch_dir, write_dir, steps):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--summarize-pmc", fetch_dir, write_dir,
                        "--steps", str(steps)], capture_output=True, text=True, cwd=ROOT)
    return r


def test_pass_g_dispatches_and_copy_calibration(tmp_path):
    # earlier passes: a short batch (100 KiB) among full ones; pass G: the
    # last three dispatches; the copy reads half of what it moves, as
    # FETCH_SIZE does on gfx950, and writes all of it
    gib_kib = (1 << 30) / 1024
    fetch = [(GATHER, 900.0), (GATHER, 100.0), (COPY, gib_kib / 2), (COPY, 10.0), (GATHER, 500.0),
             (GATHER, 600.0), (GATHER, 700.0)]
    write = [(GATHER, 1800.0), (GATHER, 200.0), (COPY, gib_kib), (COPY, 20.0), (GATHER, 1000.0),
             (GATHER, 1200.0), (GATHER, 1400.0)]
    alg = 1024.0 * (2 * 600.0 + 1200.0)
    write_run(str(tmp_path / "f"), "FETCH_SIZE", fetch, alg=alg)
    write_run(str(tmp_path / "w"), "WRITE_SIZE", write, alg=alg)
    r = summarize(str(tmp_path / "f"), str(tmp_path / "w"), 3)
    assert r.returncode == 0, r.stderr
    t = json.loads(r.stdout)
    assert t["gather_dispatches"] == [3, 3]
    assert t["fetch_kib_per_launch"] == pytest.approx(600.0)
    assert t["write_kib_per_launch"] == pytest.approx(1200.0)
    assert t["fetch_scale"] == pytest.approx(2.0) and t["write_scale"] == pytest.approx(1.0)
    assert t["copy_dispatches"] == [1, 1]   # the small copy is not the calibration copy
    assert t["traffic_bytes_per_launch"] == pytest.approx(1024.0 * (2 * 600.0 + 1200.0))
    assert t["traffic_over_alg"] == pytest.approx(1.0)
    assert t["workload"] == "hubs2m"
    assert len(t["gather_source_sha256_16"]) == 16


def test_fewer_dispatches_than_steps_is_an_error(tmp_path):
    gib_kib = (1 << 30) / 1024
    write_run(str(tmp_path / "f"), "FETCH_SIZE", [(GATHER, 1.0), (COPY, gib_kib)])
    write_run(str(tmp_path / "w"), "WRITE_SIZE", [(GATHER, 1.0), (COPY, gib_kib)])
    r = summarize(str(tmp_path / "f"), str(tmp_path / "w"), 5)
    assert r.returncode != 0 and "fewer than --steps" in (r.stderr + r.stdout)


def test_stored_traffic_is_per_workload():
    import bench
    for w in ("products2m", "hubs2m", "papers111m"):
        path = bench.traffic_file(w)
        t = json.load(open(path))
        assert t.get("workload", "products2m") == w
        v, why = bench.gather_traffic(w)
        if t["gather_source_sha256_16"] == bench._source_digest(bench.GATHER_SOURCE):
            assert v == t["traffic_bytes_per_launch"] and os.path.basename(path) in why
        else:
            assert v is None and "predates" in why
    v, why = bench.gather_traffic("rmat1m")
    assert v is None and "rmat1m" in why
