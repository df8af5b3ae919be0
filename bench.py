#!/usr/bin/env python3
"""Throughput of the generalized Allreduce on one MI355X.

Kolmakov & Zhang, "A Generalization of the Allreduce Operation"
(arXiv:2004.09362).  P virtual ranks live on one GPU; one bench step runs
the workload's Allreduce(s) once through the C-ABI library (libar.so).

Metric: effective Allreduce bandwidth = P * n * element bytes / time (summed
over the workload's instances), and the achieved algorithmic HBM bandwidth
of the dominant kernel against the MI355X peak of 8 TB/s.

Workloads (seeded synthetic rank buffers, resident in HBM before timing):
  small_batch            P in {5, 6, 7, 12}, n = 106 fp32 N(0,1) (about the
                         425-byte average message the paper quotes), 65536
                         instances per launch, latency-optimal k = ceil(log2 P)
  gradsync               P = 24, n = 2^24 fp32 N(0,1e-3), k = 10
  prime_sweep            P = 37, n = 2^22 fp32 U(-1,1), --k in 6..12 (default 12),
                         --op sum (default) or max
  large (default)        P = 127, n = 2^26 fp32 N(0,1e-2) (31.75 GiB of rank
                         buffers, the largest shape that fits one GPU), --k 14
                         (default) or 10; without --k the line reports k = 14
                         and carries k = 10, timed on the same buffers, under
                         "extra"
  prime3                 P = 3, n = 1024 int32 U[-1000,1000], --k 2..4 (default 4)
  gradsync32             P = 32, n = 2^24 fp32 N(0,1e-3), --k 5..10 (default 10)
  small_batch127         P = 127, n = 106 fp32 N(0,1), 65536 instances, k = 7
  medium127              P = 127, n = 2304 fp32 N(0,1) (9 KB), 8192 instances,
                         --k 7..14 (default 11)
  medium128              P = 128, n = 2304 fp32 N(0,1) (9 KB), 8192 instances,
                         --k 7..14 (default 14); with --group xor, Recursive
                         Halving at k = 14

--group xor runs the butterfly schedules over the XOR group (power-of-two P:
Recursive Halving at k = 2 log2 P, Recursive Doubling at k = log2 P);
--schedule ring runs the Ring (k = 2(P-1)) on the workload's shape.

Each step uses one of several input sets in turn, so that the sets together
exceed the 256 MB Infinity Cache and every step reads HBM.

Prints ONE JSON line.  Only one GPU is used: --gpus above 1 exits with an error.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective allreduce GB/s (P*n*bytes/s) and achieved HBM GB/s vs peak, 1 GPU"
HBM_PEAK_GBPS = 8000.0
POOL_BYTES = 1 << 30  # rotate input sets until they span at least this much


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def ceil_log2(P):
    return max(0, (P - 1).bit_length())


def jobs_for(name, k_arg, group="cyclic", schedule="butterfly", op=None):
    from paper_2004_09362_amd import synth
    import numpy as np

    w = synth.WORKLOADS[name]
    if op is not None and op not in w["ops"]:
        raise SystemExit("op %s is not one of the %s workload's ops %s" % (op, name, w["ops"]))
    jobs = []
    for P in w["P"]:
        if group == "xor" and P & (P - 1):
            raise SystemExit("the XOR group needs a power-of-two P; the %s workload has P=%d" % (name, P))
        if schedule == "ring":
            k = 2 * (P - 1)
        elif w["ks"] == "lo":
            k = ceil_log2(P)
        else:
            k = k_arg if k_arg is not None else DEFAULT_K[name]
            if k not in w["ks"]:
                raise SystemExit("k=%d is not one of the %s workload's k values %s" % (k, name, w["ks"]))
        jobs.append(dict(P=P, n=w["n"], batch=w["batch"], k=k, op=op or w["ops"][0],
                         dtype=np.dtype(w["dtype"]), dist=w["dist"], seed=w["seed"]))
    return w, jobs


DEFAULT_K = {"gradsync": 10, "prime_sweep": 12, "large": 14, "prime3": 4, "gradsync32": 10, "medium127": 11,
             "medium128": 14}
# Steps of well under a millisecond get more of them, so that the timed
# region spans tens of milliseconds (prime3: about 10 us per step).
DEFAULT_STEPS = {"large": 10, "small_batch": 200, "small_batch127": 100, "medium127": 100, "medium128": 100,
                 "prime3": 1000}
# further k timed on the same buffers when --k is not given
EXTRA_K = {"large": [10]}
DEFAULT_WARMUP = {"large": 2, "small_batch": 20, "small_batch127": 10, "medium127": 10, "medium128": 10,
                  "prime3": 50}

SHAPES = {
    "small_batch": "small_batch: P in {5,6,7,12}, n=106 fp32 N(0,1), 65536 instances per launch",
    "gradsync": "gradsync: P=24, n=16777216 fp32 N(0,1e-3)",
    "prime_sweep": "prime_sweep: P=37, n=4194304 fp32 U(-1,1)",
    "large": "large: P=127, n=67108864 fp32 N(0,1e-2)",
    "prime3": "prime3: P=3, n=1024 int32 U[-1000,1000]",
    "gradsync32": "gradsync32: P=32, n=16777216 fp32 N(0,1e-3)",
    "small_batch127": "small_batch127: P=127, n=106 fp32 N(0,1), 65536 instances per launch",
    "medium127": "medium127: P=127, n=2304 fp32 N(0,1), 8192 instances per launch",
    "medium128": "medium128: P=128, n=2304 fp32 N(0,1), 8192 instances per launch",
}


def describe(workload, jobs, group, schedule):
    ks = sorted({j["k"] for j in jobs})
    if schedule == "ring":
        sched = "Ring k=2(P-1)" if len(ks) > 1 else "Ring k=%d" % ks[0]
    else:
        kk = "k=ceil(log2 P)" if len(ks) > 1 else "k=%d" % ks[0]
        sched = ("XOR group " if group == "xor" else "") + kk
    return "%s, %s, %s" % (SHAPES[workload], sched, jobs[0]["op"])


def kernel_source_hash(kernel):
    from paper_2004_09362_amd.build import kernel_families, source_hash

    return source_hash(kernel_families(kernel))


def traffic_from_profiles(key, kernel, src_hash):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as fh:
            data = json.load(fh)
        ent = data.get(key, {}).get(kernel)
        if not ent or ent.get("source_hash") != src_hash:
            return None
        return ent.get("bytes_per_launch")
    except (OSError, ValueError):
        return None


def traffic_key(workload, group, schedule):
    """Entry of profiles/traffic.json for a workload run with a group and schedule."""
    return workload + ("/xor" if group == "xor" else "") + ("/ring" if schedule == "ring" else "")


def host_facts():
    """Threads this process may use, and the CPU model, from the OS."""
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count() or 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": usable, "cpu_model": model}


def cpu_baseline(jobs, fetchers, budget_s=12.0, group="cyclic", schedule="butterfly"):
    """The CPU oracle (single thread, as it stands) on a bounded sample.

    ``fetchers[i](kind, count)`` copies job i's sample to the host: the first
    ``count`` instances of a batch ([P, count, n]), or the first ``count``
    columns of every block of a single instance (then it returns the [P,
    ncols] values and their column indices).  Only the sample crosses PCIe.
    """
    import numpy as np

    import oracle

    oracle.lib()
    total_bytes, total_t, parts = 0, 0.0, []
    per_job_budget = budget_s / len(jobs)
    for job, fetch in zip(jobs, fetchers):
        P, n, B, k = job["P"], job["n"], job["batch"], job["k"]
        if B > 1:
            # whole instances; repeat the set if it takes less than the budget
            b = 64
            reps = 1
            while True:
                xb = fetch("instances", b)
                t0 = time.perf_counter()
                for _ in range(reps):
                    oracle.allreduce_batched(xb, k, job["op"], group=group, schedule=schedule)
                dt = time.perf_counter() - t0
                if dt >= per_job_budget:
                    break
                if b < B:
                    b = min(B, max(b * 2, int(b * per_job_budget / max(dt, 1e-3))))
                else:
                    reps = max(reps + 1, int(reps * per_job_budget / max(dt, 1e-3)) + 1)
            total_bytes += P * n * b * reps * job["dtype"].itemsize
            parts.append("P=%d: %d of %d instances x%d" % (P, b, B, reps))
        else:
            # sampled columns: the first `c` of every block (at most the prefetched
            # fetch.cmax), the same replay as a full run at those columns; repeated
            # if that takes less than the budget
            c = min(256, fetch.cmax)
            reps = 1
            while True:
                xs, cols = fetch("columns", c)
                t0 = time.perf_counter()
                for _ in range(reps):
                    oracle.allreduce(xs, k, job["op"], n=n, cols=cols, group=group, schedule=schedule)
                dt = time.perf_counter() - t0
                if dt >= per_job_budget:
                    break
                if c < fetch.cmax:
                    c = min(fetch.cmax, max(c * 2, int(c * per_job_budget / max(dt, 1e-3))))
                else:
                    reps = max(reps + 1, int(reps * per_job_budget / max(dt, 1e-3)) + 1)
            b = len(cols)
            total_bytes += P * b * reps * job["dtype"].itemsize
            parts.append("P=%d: %d of %d columns (the first %d of every block) x%d" % (P, b, n, c, reps))
        total_t += dt
    facts = host_facts()
    return {"value": round(total_bytes / total_t / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": "; ".join(parts) + " (single-threaded C replay, %.1f s)" % total_t,
            "nproc": facts["nproc"], "cpu_model": facts["cpu_model"]}


# Columns per block copied to the host for the oracle's sample (at P = 127
# about 1 GB); the oracle replays them as often as its time budget allows.
SAMPLE_COLS_PER_BLOCK = 16384


def sample_fetchers(jobs, tensors):
    """Copy each job's oracle sample to the host now (before any step changes
    the buffers in place) and return one fetch function per job (see
    cpu_baseline).  Batches are copied whole (at most 1.6 GB in the batched
    workloads); single instances only the first SAMPLE_COLS_PER_BLOCK columns
    of every block."""
    import numpy as np
    import torch

    def make(j, X):
        P, n, B = j["P"], j["n"], j["batch"]
        if B > 1:
            host = X.view(P, B, n).cpu().numpy()

            def fetch_inst(kind, count):
                return np.ascontiguousarray(host[:, :count])

            return fetch_inst
        q, m = n // P, n % P
        cmax = max(1, min(q, SAMPLE_COLS_PER_BLOCK))
        starts = np.array([bb * q + min(bb, m) for bb in range(P)], dtype=np.int64)
        cols_all = (starts[:, None] + np.arange(cmax, dtype=np.int64)[None, :])  # [block, c]
        idx = torch.from_numpy(cols_all.reshape(-1)).to(X.device)
        host = X.index_select(1, idx).cpu().numpy().reshape(P, P, cmax)  # [rank, block, c]

        def fetch_cols(kind, count):
            c = min(count, cmax)
            return np.ascontiguousarray(host[:, :, :c].reshape(P, P * c)), cols_all[:, :c].reshape(-1).copy()

        fetch_cols.cmax = cmax
        return fetch_cols

    return [make(j, X) for j, X in zip(jobs, tensors)]


class HipEvent:
    """A timing event of the HIP runtime torch runs on, created with
    hipEventDisableSystemFence: recording it then skips the system-scope
    cache writeback and invalidation that a default event performs, which
    HIP documents as the way to time device work accurately (a default event
    added about 2 us to a 109 us launch here, and slowed the work after it)."""

    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    @classmethod
    def runtime(cls):
        import ctypes

        if cls._hip is None:
            paths = sorted({ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64" in ln})
            if not paths:
                raise RuntimeError("the HIP runtime is not loaded in this process")
            cls._hip = ctypes.CDLL(paths[0])  # the library torch loaded (same handle)
        return cls._hip

    def __init__(self):
        import ctypes

        self._ct = ctypes
        self.h = ctypes.c_void_p()
        e = self.runtime().hipEventCreateWithFlags(ctypes.byref(self.h), ctypes.c_uint(self.DISABLE_SYSTEM_FENCE))
        if e != 0:
            raise RuntimeError("hipEventCreateWithFlags failed (%d)" % e)

    def record(self, stream):
        e = self.runtime().hipEventRecord(self.h, self._ct.c_void_p(stream.cuda_stream))
        if e != 0:
            raise RuntimeError("hipEventRecord failed (%d)" % e)

    def elapsed_time(self, end):
        ms = self._ct.c_float()
        e = self.runtime().hipEventElapsedTime(self._ct.byref(ms), self.h, end.h)
        if e != 0:
            raise RuntimeError("hipEventElapsedTime failed (%d)" % e)
        return ms.value

    def __del__(self):
        if self._hip is not None and self.h:
            self._hip.hipEventDestroy(self.h)


def copy_probe(nbytes, reps):
    """A plain copy kernel of known size: reads and writes nbytes per launch.
    Its FETCH_SIZE / WRITE_SIZE readings calibrate the HBM counters."""
    import torch

    a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    print(json.dumps({"copy_probe_bytes": nbytes, "reps": reps, "ms": round(ms, 5),
                      "GBps": round(2 * nbytes / (ms * 1e-3) / 1e9, 1)}), flush=True)


def make_parser():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default="large",
                    choices=["small_batch", "gradsync", "prime_sweep", "large", "prime3", "gradsync32",
                             "small_batch127", "medium127", "medium128"])
    ap.add_argument("--k", type=int, default=None)
    ap.add_argument("--op", choices=["sum", "max"], default=None,
                    help="the reduction (default: the workload's first; prime_sweep also runs max)")
    ap.add_argument("--group", choices=["cyclic", "xor"], default="cyclic")
    ap.add_argument("--schedule", choices=["butterfly", "ring"], default="butterfly")
    ap.add_argument("--path", choices=["auto", "stepwise", "fused"], default="auto")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="instead: time a plain device-to-device copy of BYTES (counter calibration)")
    return ap


def main():
    args = make_parser().parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the P ranks are virtual ranks held on a single MI355X, and "
              "runs across several GPUs are not part of this library (asked for --gpus %d)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2004_09362_amd import ar, synth

    if args.copy_probe:
        copy_probe(args.copy_probe, args.steps or 10)
        return

    steps = args.steps if args.steps is not None else DEFAULT_STEPS.get(args.workload, 20)
    warmup = args.warmup if args.warmup is not None else DEFAULT_WARMUP.get(args.workload, 5)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.schedule == "ring" and args.group != "cyclic":
        raise SystemExit("the Ring runs over the cyclic group")
    w, jobs = jobs_for(args.workload, args.k, args.group, args.schedule, args.op)
    path = {"auto": ar.AR_PATH_AUTO, "stepwise": ar.AR_PATH_STEPWISE, "fused": ar.AR_PATH_FUSED}[args.path]
    # the large workload without --k: k = 14 on the line, k = 10 under "extra"
    extra_ks = EXTRA_K.get(args.workload, []) if (args.k is None and args.schedule == "butterfly"
                                                 and args.group == "cyclic") else []

    # ---- resident inputs ----
    set_bytes = sum(j["P"] * j["n"] * j["batch"] * j["dtype"].itemsize for j in jobs)
    n_sets = int(max(1, min(steps + warmup, -(-POOL_BYTES // set_bytes))))
    log("workload %s: %d job(s), %d input set(s) of %.1f MB" % (args.workload, len(jobs), n_sets, set_bytes / 1e6))
    sets = []
    for s in range(n_sets):
        per = []
        for j in jobs:
            X = synth.device_ranks(j["seed"] + 7919 * s, j["P"], j["n"] * j["batch"], j["dtype"], j["dist"], dev)
            per.append(X)
        sets.append(per)
    fetchers = None if args.no_cpu_baseline else sample_fetchers(jobs, sets[0])
    ptr_tables = [[[X[i] for i in range(j["P"])] for j, X in zip(jobs, per)] for per in sets]
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    res = measure(args, jobs, path, ptr_tables, n_sets, steps, warmup, stream)
    desc = describe(args.workload, jobs, args.group, args.schedule)
    out = {
        "metric": METRIC, "value": res["value"], "unit": "GB/s", "n_gpus": 1, "steps": steps,
        "warmup": warmup, "ms_per_step": res["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int32" if jobs[0]["dtype"] == np.int32 else "f32",
        "data": "synthetic (seeded; %d rotating input set(s) resident in HBM)" % n_sets,
        "config": {"workload": desc, "P": [j["P"] for j in jobs], "n": jobs[0]["n"], "batch": jobs[0]["batch"],
                   "k": [j["k"] for j in jobs], "op": jobs[0]["op"],
                   "path": res["path"], "group": args.group, "schedule": args.schedule,
                   "parallelism": "1 GPU, P virtual ranks"},
        "hbm_algorithmic_GBps_step": res["hbm_algorithmic_GBps_step"],
        "wall_s_timed": res["wall_s_timed"],
        "roofline": res["roofline"],
        "source_hash": res["source_hash"],
    }
    if extra_ks:
        # the same buffers, timed again with each further k (they hold the
        # previous results by then; the values do not change the traffic)
        out["extra"] = []
        for k in extra_ks:
            _, jobs_k = jobs_for(args.workload, k, args.group, args.schedule, args.op)
            rk = measure(args, jobs_k, path, ptr_tables, n_sets, steps, warmup, stream)
            rk["workload"] = describe(args.workload, jobs_k, args.group, args.schedule)
            rk["k"] = [j["k"] for j in jobs_k]
            out["extra"].append(rk)
    out["box_reference"] = box_reference(sets[0][0], stream)
    if fetchers is not None:
        log("timing the CPU oracle on a sample")
        out["cpu_baseline"] = cpu_baseline(jobs, fetchers, group=args.group, schedule=args.schedule)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


def measure(args, jobs, path, ptr_tables, n_sets, steps, warmup, stream):
    """Time `steps` steps of the jobs' Allreduces (after `warmup` untimed
    ones) and the dominant job's launches; returns the step time, the
    effective bandwidth and the roofline of the dominant kernel."""
    import torch

    from paper_2004_09362_amd import ar

    plans = [ar.Plan(j["P"], j["n"], j["dtype"].name, j["op"], j["k"], path=path, group=args.group,
                     schedule=args.schedule) for j in jobs]

    # the dominant job: the one moving the most algorithmic bytes
    def alg_bytes(j, p):
        st_ = p.stats()
        fused_ = (path == ar.AR_PATH_FUSED) or (path == ar.AR_PATH_AUTO and st_.fused_ok)
        return (st_.hbm_bytes_fused if fused_ else st_.hbm_bytes_stepwise) * j["batch"], fused_, st_
    dom = max(range(len(jobs)), key=lambda jj: alg_bytes(jobs[jj], plans[jj])[0])

    def run_step(s, ev=None):
        for jj, (j, p) in enumerate(zip(jobs, plans)):
            if ev is not None and jj == dom:
                ev[0].record(stream)
            p.batched(ptr_tables[s % n_sets][jj], j["batch"], j["n"], stream)
            if ev is not None and jj == dom:
                ev[1].record(stream)

    for s in range(warmup):
        run_step(s)
    torch.cuda.synchronize()

    # ---- timed region: exactly `steps` steps on the launch stream, between
    # two HIP events and nothing else.  The events carry no system-scope fence
    # (HipEvent) ----
    start, stop = HipEvent(), HipEvent()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for s in range(steps):
        run_step(warmup + s)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = start.elapsed_time(stop)
    # ---- the dominant kernel's launch time.  With one job the region above
    # times it.  With several, a second pass of `steps` steps brackets the
    # dominant job's launch(es) with events in every step; kept out of the
    # region above, whose step time the event packets would raise (by about
    # 11 us in a 270 us step of four launches) ----
    per_launch = len(jobs) > 1
    if per_launch:
        ev = [(HipEvent(), HipEvent()) for _ in range(steps)]
        for s in range(steps):
            run_step(warmup + steps + s, ev[s])
        torch.cuda.synchronize()
        dom_ms = sum(a.elapsed_time(b) for a, b in ev) / steps
    else:
        dom_ms = total_ms / steps

    eff_bytes = sum(j["P"] * j["n"] * j["batch"] * j["dtype"].itemsize for j in jobs)
    ms_per_step = total_ms / steps
    value = eff_bytes / (ms_per_step * 1e-3) / 1e9

    # ---- roofline of the dominant kernel ----
    dj, dp = jobs[dom], plans[dom]
    alg, fused, st = alg_bytes(dj, dp)
    launches = st.fused_launches if fused else st.launches
    bytes_per_launch = alg / launches
    launch_ms = dom_ms / launches
    achieved = bytes_per_launch / (launch_ms * 1e-3) / 1e9
    kname = kernel_name(args, dj, st, fused)
    src_hash = kernel_source_hash(kname)
    roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic_from_profiles(traffic_key(args.workload, args.group, args.schedule), kname, src_hash),
            "kernel": kname, "job_P": dj["P"], "bytes_per_launch": int(bytes_per_launch),
            "launch_ms": round(launch_ms, 5), "launches_per_step": launches,
            "timed_by": ("HIP events around each launch, in a second pass of the same steps" if per_launch
                         else "HIP events around the timed region")}
    step_alg = sum(alg_bytes(j, p)[0] for j, p in zip(jobs, plans))
    return {"value": round(value, 2), "ms_per_step": round(ms_per_step, 5),
            "path": "fused" if fused else "stepwise",
            "hbm_algorithmic_GBps_step": round(step_alg / (ms_per_step * 1e-3) / 1e9, 1),
            "wall_s_timed": round(wall, 4), "roofline": roof, "source_hash": src_hash}


def box_reference(X, stream, reps=3):
    """HBM rates of this GPU on the workload's own rank buffers, for context:
    torch's fill_ (writes only) over all of X and copy_ of one half onto the
    other (one read and one write stream), best of `reps`.  Run after every
    timed step (it overwrites the buffers).  None for sets under 1 GiB, which
    the 256 MB Infinity Cache would flatter."""
    import torch

    nbytes = X.numel() * X.element_size()
    if nbytes < (1 << 30):
        return None
    flat = X.view(-1)
    half = flat.numel() // 2
    a, b = flat[:half], flat[half:2 * half]

    def best(fn, moved):
        fn()
        torch.cuda.synchronize()
        ms = []
        for _ in range(reps):
            e0, e1 = HipEvent(), HipEvent()
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        return round(moved / (min(ms) * 1e-3) / 1e9, 1)

    out = {"fill_GBps": best(lambda: flat.fill_(0), nbytes),
           "copy_GBps": best(lambda: b.copy_(a), 2 * half * X.element_size()),
           "bytes": nbytes,
           "how": "torch fill_ over the rank buffers and copy_ of one half onto the other, after the timed "
                  "steps, best of %d" % reps}
    return out


def kernel_name(args, dj, st, fused):
    """Name of the dominant job's kernel(s) as the profiles list it."""
    if not fused:
        kname = "step_kernel<k=%d>" % dj["k"]
    elif st.fused_flat and args.group != "xor":
        kname = "fused_rot_kernel<P=%d,%s>" % (dj["P"], "ring" if args.schedule == "ring" else "r=%d" % st.r)
    elif args.schedule == "ring":
        kname = "fused_ring_kernel"
    elif args.group == "xor":
        kname = "fused_xor_kernel<P=%d,R=%d>" % (dj["P"], st.r)
    elif st.r == 0:
        kname = "fused_bo_kernel<P=%d>" % dj["P"]
    elif st.r == st.L and dj["P"] <= 16:
        kname = "fused_lo_kernel<P=%d>" % dj["P"]
    else:
        kname = "fused_mid_kernel<P=%d>" % dj["P"]
    if fused and st.fused_launches == 2:
        # the pair: reducing launch, then the broadcast (destination-major on
        # the bench's contiguous, 16-byte aligned rank rows where the plan allows)
        stream = st.fused_bcast_stream and dj["n"] % 4 == 0  # rows of the [P, batch * n] tensor 16-byte aligned
        kname += "+broadcast_stream" if stream else "+broadcast"
    return kname


if __name__ == "__main__":
    main()
