"""Host-side logic of bench.py (CPU): percentiles, the rocprofv3 counter
readers, the HBM-traffic record and its use, and the one-GPU guard."""

import csv
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_percentiles():
    v = list(range(1, 11))                     # 1..10
    p = bench.percentiles(v)
    assert p == {"median": 5.5, "p10": round(float(np.percentile(v, 10)), 4),
                 "p90": round(float(np.percentile(v, 90)), 4)}
    assert bench.percentiles([2.0]) == {"median": 2.0, "p10": 2.0, "p90": 2.0}


def write_counters(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "p_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], r)))


def test_counter_per_dispatch_sums_rows_then_averages(tmp_path):
    d = str(tmp_path / "c")
    write_counters(d, [(1, "ns::cascade(P)", "FETCH_SIZE", 10), (1, "ns::cascade(P)", "FETCH_SIZE", 5),
                       (2, "ns::cascade(P)", "FETCH_SIZE", 25), (3, "other", "FETCH_SIZE", 1000),
                       (4, "ns::noncascade(P)", "FETCH_SIZE", 999), (2, "ns::cascade(P)", "WRITE_SIZE", 7)])
    assert bench._counter_per_dispatch(d, "cascade", "FETCH_SIZE") == 20.0   # (15 + 25) / 2
    with pytest.raises(ValueError):
        bench._counter_per_dispatch(d, "cascade", "TCC_HIT")
    with pytest.raises(FileNotFoundError):
        bench._counter_per_dispatch(str(tmp_path / "none"), "cascade", "FETCH_SIZE")


def test_record_and_use_traffic(tmp_path, monkeypatch):
    rec_file = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(rec_file))
    d = tmp_path / "t"
    names = bench._workload_names()
    line = {"dtype": "bf16", "config": {"workload": names[4], "kv_split": 8192}, "requested_kv_split": 0}
    os.makedirs(d)
    (d / "fetch.log").write_text("noise\n" + json.dumps(line) + "\n")
    write_counters(str(d / "fetch"), [(1, "cascade_bf16_kernel", "FETCH_SIZE", 1000.0)])
    write_counters(str(d / "write"), [(1, "cascade_bf16_kernel", "WRITE_SIZE", 100.0)])
    gib_kib = (1 << 30) / 1024.0
    write_counters(str(d / "copy_fetch"), [(1, "__amd_rocclr_copyBuffer", "FETCH_SIZE", gib_kib / 2)])
    write_counters(str(d / "copy_write"), [(1, "__amd_rocclr_copyBuffer", "WRITE_SIZE", gib_kib)])
    bench.record_traffic(str(d))
    r = json.loads(rec_file.read_text())["config4"]
    assert r["fetch_factor"] == 2.0 and r["write_factor"] == 1.0
    assert r["hbm_bytes_per_launch"] == (1000 * 2 + 100) * 1024
    assert r["kernel_sha"] == bench.kernel_sha()
    # used only for the same kernel source and launch configuration
    assert bench.measured_traffic(4, 0, 8192) == r["hbm_bytes_per_launch"]
    assert bench.measured_traffic(4, 0, 4096) is None
    assert bench.measured_traffic(4, 4096, 8192) is None
    assert bench.measured_traffic(3, 0, 8192) is None
    r["kernel_sha"] = "0" * 16
    rec_file.write_text(json.dumps({"config4": r}))
    assert bench.measured_traffic(4, 0, 8192) is None


def test_record_traffic_adds_the_split_merge(tmp_path, monkeypatch):
    """With a split context the operation is the attention kernel plus the
    split merge that reads the partial states back: both kernels' counters."""
    rec_file = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(rec_file))
    d = tmp_path / "t"
    names = bench._workload_names()
    line = {"dtype": "bf16", "config": {"workload": names[5], "kv_split": 10944}, "requested_kv_split": 0,
            "roofline": {"splits": 3}}
    os.makedirs(d)
    (d / "fetch.log").write_text(json.dumps(line) + "\n")
    write_counters(str(d / "fetch"), [(1, "cascade_bf16_kernel", "FETCH_SIZE", 1000.0),
                                      (2, "split_merge_kernel<bf16, 1>", "FETCH_SIZE", 300.0)])
    write_counters(str(d / "write"), [(1, "cascade_bf16_kernel", "WRITE_SIZE", 100.0),
                                      (2, "split_merge_kernel<bf16, 1>", "WRITE_SIZE", 40.0)])
    gib_kib = (1 << 30) / 1024.0
    write_counters(str(d / "copy_fetch"), [(1, "__amd_rocclr_copyBuffer", "FETCH_SIZE", gib_kib)])
    write_counters(str(d / "copy_write"), [(1, "__amd_rocclr_copyBuffer", "WRITE_SIZE", gib_kib)])
    bench.record_traffic(str(d))
    r = json.loads(rec_file.read_text())["config5"]
    assert r["hbm_bytes_per_launch"] == (1300 + 140) * 1024


def test_trace_summary_phases(tmp_path):
    d = tmp_path / "kt"
    os.makedirs(d)
    with open(d / "run_kernel_trace.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        t = 0
        for i in range(2 + 3 * 4):              # warmup 2, steps 4: 14 attention calls, durations 1..14 us
            w.writerow({"Kernel_Name": "ns::cascade_bf16_wide_kernel(P)", "Start_Timestamp": t,
                        "End_Timestamp": t + 1000 * (i + 1)})
            w.writerow({"Kernel_Name": "ns::noncascade_bf16_kernel(P)", "Start_Timestamp": t + 1,
                        "End_Timestamp": t + 99999})
            t += 100000
    r = bench.trace_summary(str(d), 2, 4)["cascade_bf16_wide_kernel"]
    assert r == {"dispatches": 14, "all": 7.5, "warmup": 1.5, "cold": 4.5, "warm": 8.5, "backtoback": 12.5}
    assert "noncascade_bf16_kernel" not in bench.trace_summary(str(d), 2, 4)


def test_attention_kernel_name_follows_the_shape():
    k = bench.attention_kernel_name
    assert k({"dtype": "f32", "config": {}}) == "cascade_attention_kernel"
    assert k({"dtype": "bf16", "config": {"row_group": 128}}) == "cascade_bf16_kernel"
    assert k({"dtype": "bf16", "config": {"row_group": 384, "packed": False}}) == "cascade_bf16_wide_kernel"
    assert k({"dtype": "bf16", "config": {"row_group": 384, "packed": True}}) == "cascade_bf16_packed_kernel"


def test_kernel_names_match_whole_identifiers():
    m = bench.kernel_name_matches
    assert m("d2sd::(anonymous namespace)::cascade_bf16_kernel(d2sd::(anonymous namespace)::Params)",
             "cascade_bf16_kernel")
    assert not m("d2sd::(anonymous namespace)::noncascade_bf16_kernel(Params)", "cascade_bf16_kernel")
    assert m("void split_merge_kernel<__bf16, 4>(Params, int)", "split_merge_kernel")
    assert not m("cascade_bf16_kernel_v2", "cascade_bf16_kernel")


def test_kernel_sha_is_stable():
    a, b = bench.kernel_sha(), bench.kernel_sha()
    assert a == b and len(a) == 16 and int(a, 16) >= 0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_parent_arrays_match_oracle_constructions():
    """The benchmark's parent arrays (inputs of the parent-array tree builder)
    are the oracle's canonical, third-level and resample trees."""
    from oracle.tree import build_tree, resample_parents, third_level_parents

    rng = np.random.default_rng(0)
    for _ in range(200):
        B = int(rng.integers(3, 40))
        K = int(rng.integers(0, min(B - 2, 8) + 1))
        p = rng.choice(np.arange(1, B - 1), size=K, replace=False).tolist()
        q = [int(rng.integers(pk + 1, B)) for pk in p]
        assert bench.bench_parent_array(B, p).tolist() == build_tree(B, p).parent
        if K:
            order = np.argsort(p)
            assert bench.bench_parent_array(B, p, q).tolist() == third_level_parents(B, sorted(p), [q[i] for i in order])
        c = int(rng.integers(1, 5))
        assert bench.bench_parent_array(B, [], chains=c).tolist() == resample_parents(B, c)
