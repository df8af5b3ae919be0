"""Host-side checks of bench.py and of the rocprofv3 summary tool (no GPU)."""
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
from paper_2004_09362_amd import profiling  # noqa: E402
from paper_2004_09362_amd.build import source_hash  # noqa: E402


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr


@pytest.mark.parametrize("workload,k,group,schedule,want_P,want_k", [
    ("small_batch", None, "cyclic", "butterfly", [5, 6, 7, 12], [3, 3, 3, 4]),
    ("gradsync", None, "cyclic", "butterfly", [24], [10]),
    ("gradsync", None, "cyclic", "ring", [24], [46]),
    ("gradsync32", 7, "xor", "butterfly", [32], [7]),
    ("prime_sweep", 9, "cyclic", "butterfly", [37], [9]),
    ("large", None, "cyclic", "butterfly", [127], [14]),
    ("prime3", None, "cyclic", "butterfly", [3], [4]),
])
def test_jobs(workload, k, group, schedule, want_P, want_k):
    _, jobs = bench.jobs_for(workload, k, group, schedule)
    assert [j["P"] for j in jobs] == want_P
    assert [j["k"] for j in jobs] == want_k
    desc = bench.describe(workload, jobs, group, schedule)
    assert desc.startswith(workload + ":")
    if schedule == "ring":
        assert "Ring" in desc
    if group == "xor":
        assert "XOR" in desc


def test_jobs_reject_bad_requests():
    with pytest.raises(SystemExit):
        bench.jobs_for("gradsync", None, "xor", "butterfly")     # P = 24 is not a power of two
    with pytest.raises(SystemExit):
        bench.jobs_for("prime_sweep", 13, "cyclic", "butterfly")  # k outside the workload's values
    with pytest.raises(SystemExit):
        bench.jobs_for("gradsync", None, "cyclic", "butterfly", "max")  # gradsync sums only
    _, jobs = bench.jobs_for("prime_sweep", 9, "cyclic", "butterfly", "max")
    assert [(j["P"], j["k"], j["op"]) for j in jobs] == [(37, 9, "max")]


def test_traffic_lookup_checks_the_source_hash(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    h = source_hash("group")
    data = {"gradsync/ring": {"fused_ring_kernel": {"bytes_per_launch": 123, "source_hash": h}},
            "gradsync": {"fused_bo_kernel<P=24>": {"bytes_per_launch": 456, "source_hash": "stale"}}}
    (tmp_path / "profiles" / "traffic.json").write_text(json.dumps(data))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    key = bench.traffic_key("gradsync", "cyclic", "ring")
    assert bench.kernel_source_hash("fused_ring_kernel") == h
    assert bench.traffic_from_profiles(key, "fused_ring_kernel", h) == 123
    assert bench.traffic_from_profiles("gradsync", "fused_bo_kernel<P=24>", source_hash("col")) is None
    assert bench.traffic_from_profiles("gradsync", "missing", h) is None


def test_generated_column_units_instantiate_every_P_once():
    import re

    from paper_2004_09362_amd import build as b

    for kind in b.COL_KINDS:
        ps = []
        for i in range(b.COL_UNITS):
            ps += [int(m) for m in re.findall(r"launch_fused_%s<(\d+)>" % kind, b.col_unit_text(i))]
        assert sorted(ps) == list(range(2, 129)), kind
    # the generated text counts in the column family's source hash
    h = b.source_hash("col")
    old = b.col_unit_text
    try:
        b.col_unit_text = lambda i: old(i) + "\nint changed_unit;"
        assert b.source_hash("col") != h
    finally:
        b.col_unit_text = old


def test_kernel_families_cover_every_source():
    from paper_2004_09362_amd import build as b

    listed = set(b.COMMON) | {f for fam in b.FAMILIES.values() for f in fam}
    have = {os.path.basename(f) for f in b.SOURCES + b.HEADERS if "/csrc/" in f}
    assert have == listed
    assert {b.kernel_families(k)[0] for k in ("step_kernel<k=10>", "fused_lo_kernel<P=12>", "fused_bo_kernel<P=24>",
                                              "fused_mid_kernel<P=37>", "fused_xor_kernel<P=32,R=0>",
                                              "fused_ring_kernel")} == {"step", "lo", "col", "group"}
    assert b.kernel_families("fused_bo_kernel<P=127>+broadcast") == ["col", "bcast"]
    assert b.kernel_families("fused_bo_kernel<P=127>+broadcast_stream") == ["col", "bcast"]
    assert b.source_hash(["col", "bcast"]) != b.source_hash("col")


def test_cpu_baseline_runs_the_oracle_on_a_sample():
    import torch

    for workload, group, schedule in (("gradsync32", "xor", "butterfly"), ("gradsync", "cyclic", "ring")):
        _, jobs = bench.jobs_for(workload, 10 if group == "xor" else None, group, schedule)
        j = dict(jobs[0], n=64 * jobs[0]["P"] + 5)
        x = np.random.default_rng(0).normal(size=(j["P"], j["n"])).astype(np.float32)
        fetchers = bench.sample_fetchers([j], [torch.from_numpy(x)])
        # the sample is the first columns of every block, copied before any step
        xs, cols = fetchers[0]("columns", 3)
        starts = [b * (j["n"] // j["P"]) + min(b, j["n"] % j["P"]) for b in range(j["P"])]
        assert list(cols) == [s + c for s in starts for c in range(3)]
        assert np.array_equal(xs, x[:, cols])
        cb = bench.cpu_baseline([j], fetchers, budget_s=0.05, group=group, schedule=schedule)
        assert cb["kind"] == "oracle" and cb["cores"] == 1 and cb["value"] > 0 and cb["unit"] == "GB/s"
        assert cb["nproc"] >= 1 and isinstance(cb["cpu_model"], str)
    # a batch: whole instances
    _, jobs = bench.jobs_for("small_batch", None)
    j = dict(jobs[0], batch=8)
    x = np.random.default_rng(1).normal(size=(j["P"], j["batch"] * j["n"])).astype(np.float32)
    fetchers = bench.sample_fetchers([j], [torch.from_numpy(x)])
    assert np.array_equal(fetchers[0]("instances", 3), x.reshape(j["P"], 8, j["n"])[:, :3])
    cb = bench.cpu_baseline([j], fetchers, budget_s=0.05)
    assert cb["value"] > 0 and "instances" in cb["sample"]


def test_default_line_is_the_largest_single_gpu_config():
    """With no arguments the line is the large workload (P = 127, n = 2^26),
    k = 14 on the line and k = 10 under extra."""
    args = bench.make_parser().parse_args([])
    assert args.workload == "large" and args.k is None and args.gpus == 1
    _, jobs = bench.jobs_for("large", None)
    assert [(j["P"], j["n"], j["k"]) for j in jobs] == [(127, 1 << 26, 14)]
    assert bench.EXTRA_K["large"] == [10]
    assert bench.describe("large", jobs, "cyclic", "butterfly").startswith("large: P=127, n=67108864")


def test_host_facts():
    f = bench.host_facts()
    assert f["nproc"] >= 1 and f["cpu_model"]


def _write_counters(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, val in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": val})


def test_traffic_tool_scales_by_the_copy(tmp_path, monkeypatch):
    """A counter that reads half of what the copy moved is scaled by 2."""
    t = tmp_path
    _write_counters(t / "cf", "FETCH_SIZE", [("__amd_rocclr_copyBuffer", 512.0)] * 3)
    _write_counters(t / "cw", "WRITE_SIZE", [("__amd_rocclr_copyBuffer", 1024.0)] * 3)
    _write_counters(t / "kf", "FETCH_SIZE", [("void ar::fused_bo_kernel<24, float, 0, true>(ar::ColArgs)", 100.0),
                                             ("void ar::fused_bo_kernel<24, float, 0, true>(ar::ColArgs)", 102.0),
                                             ("void ar::other_kernel()", 9e9)])
    _write_counters(t / "kw", "WRITE_SIZE", [("void ar::fused_bo_kernel<24, float, 0, true>(ar::ColArgs)", 200.0)] * 2)
    monkeypatch.setattr(profiling, "TRAFFIC", str(t / "traffic.json"))
    ent = profiling.main(["traffic", "--key", "w", "--kernel", "fused_bo_kernel<P=24>", "--match", "fused_bo_kernel<24,",
                          "--fetch", str(t / "kf"), "--write", str(t / "kw"), "--copy-fetch", str(t / "cf"),
                          "--copy-write", str(t / "cw"), "--copy-bytes", str(1024 * 1024), "--alg", "409600"])
    assert ent is None
    data = json.loads((t / "traffic.json").read_text())
    e = data["w"]["fused_bo_kernel<P=24>"]
    assert e["fetch_scale"] == 2.0 and e["write_scale"] == 1.0
    assert e["bytes_per_launch"] == int((101.0 * 2 + 200.0) * 1024)
    assert e["launches_counted"] == 2 and e["source_hash"] == source_hash("col")


def test_stats_tool_lists_library_kernels(tmp_path):
    d = tmp_path / "tr"
    d.mkdir()
    with open(d / "run_kernel_stats.csv", "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Name", "Calls", "AverageNs", "MinNs", "MaxNs"])
        w.writeheader()
        w.writerow({"Name": "void ar::(anonymous namespace)::fused_ring_kernel<2, float, 0, true>(ar::ColArgs)",
                    "Calls": 25, "AverageNs": 536120.0, "MinNs": 527850.0, "MaxNs": 546930.0})
        w.writerow({"Name": "__amd_rocclr_fillBufferAligned", "Calls": 3, "AverageNs": 1.0, "MinNs": 1.0,
                    "MaxNs": 1.0})
    out = profiling.stats(str(d))
    assert "`fused_ring_kernel<2, float, 0, true>` | 25 | 536.12 | 527.85 | 546.93 |" in out
    assert "fillBuffer" not in out


def test_source_hash_ignores_comments():
    from paper_2004_09362_amd.build import code_text

    a = "int f(int x) { // add one\n  return x + 1; /* the\n value */ }\n"
    b = "int f(int x) {\n    return x + 1;  }"
    c = "int f(int x) { return x + 2; }"
    assert code_text(a) == code_text(b)
    assert code_text(a) != code_text(c)
