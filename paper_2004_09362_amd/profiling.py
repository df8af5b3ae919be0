"""Summaries of rocprofv3 output for the library's kernels.

  python -m paper_2004_09362_amd.profiling stats DIR
      the kernel-trace statistics of a `rocprofv3 --kernel-trace --stats
      --output-format csv -d DIR -o run` run, as a markdown table (kernels
      of this library only; times in microseconds).

  python -m paper_2004_09362_amd.profiling traffic --key KEY --kernel NAME
          --match SUBSTR [--match SUBSTR2] --fetch DIR --write DIR
          --copy-fetch DIR --copy-write DIR --copy-bytes N --alg BYTES
      HBM bytes per launch of the kernels whose name contains SUBSTR (any of
      the --match strings: a split launch counts its two kernels), from a
      `rocprofv3 --pmc FETCH_SIZE` and a `--pmc WRITE_SIZE` run (counter
      values in KiB per dispatch), each scaled by what the same counter read
      for a plain device copy of N bytes (`bench.py --copy-probe N`), so that
      a counter reading exactly what the copy moved scales by 1.  Stored in
      profiles/traffic.json under KEY and NAME (a kernel name as bench.py
      reports it) with the hash of that kernel family's current sources,
      which bench.py compares before it reports the figure.

Reads rocprofv3's CSV files only; runs nothing on the GPU.
"""
from __future__ import annotations

import argparse
import csv
import json
import os
import sys

from .build import kernel_families, source_hash

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TRAFFIC = os.path.join(ROOT, "profiles", "traffic.json")


def counter_values(d: str, counter: str, match) -> list[float]:
    pats = [match] if isinstance(match, str) else list(match)
    with open(os.path.join(d, "run_counter_collection.csv")) as fh:
        return [float(r["Counter_Value"]) for r in csv.DictReader(fh)
                if any(p in r["Kernel_Name"] for p in pats) and r["Counter_Name"] == counter]


def mean(v: list[float]) -> float:
    if not v:
        raise SystemExit("no matching dispatches")
    return sum(v) / len(v)


def short_name(name: str) -> str:
    name = name.replace("void ", "").replace("ar::", "").replace("(anonymous namespace)::", "")
    return name.split("(")[0]


def stats(d: str) -> str:
    rows = ["| kernel | calls | avg (us) | min (us) | max (us) |", "|---|---|---|---|---|"]
    with open(os.path.join(d, "run_kernel_stats.csv")) as fh:
        for r in csv.DictReader(fh):
            if "ar::" not in r["Name"]:
                continue
            rows.append("| `%s` | %s | %.2f | %.2f | %.2f |" % (short_name(r["Name"]), r["Calls"],
                                                              float(r["AverageNs"]) / 1e3,
                                                              float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3))
    return "\n".join(rows)


def traffic(a) -> dict:
    cf = mean(counter_values(a.copy_fetch, "FETCH_SIZE", "copyBuffer"))
    cw = mean(counter_values(a.copy_write, "WRITE_SIZE", "copyBuffer"))
    kib = a.copy_bytes / 1024.0
    sf, sw = kib / cf, kib / cw
    f = counter_values(a.fetch, "FETCH_SIZE", a.match)
    w = counter_values(a.write, "WRITE_SIZE", a.match)
    b = (mean(f) * sf + mean(w) * sw) * 1024.0
    ent = {"bytes_per_launch": int(round(b)), "fetch_KiB_raw": round(mean(f), 1), "write_KiB_raw": round(mean(w), 1),
           "fetch_scale": round(sf, 4), "write_scale": round(sw, 4), "launches_counted": len(f),
           "algorithmic_bytes_per_launch": a.alg, "ratio_to_algorithmic": round(b / a.alg, 5) if a.alg else None,
           "source_hash": source_hash(kernel_families(a.kernel))}
    data = {}
    if os.path.exists(TRAFFIC):
        with open(TRAFFIC) as fh:
            data = json.load(fh)
    data["_note"] = ("HBM bytes per launch from rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE (separate runs), each "
                     "scaled by its reading for a plain device copy of known size; valid while source_hash "
                     "matches the kernel sources.")
    data.setdefault(a.key, {})[a.kernel] = ent
    with open(TRAFFIC, "w") as fh:
        json.dump(data, fh, indent=1, sort_keys=True)
    return ent


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    t = sub.add_parser("traffic")
    for name in ("--key", "--kernel", "--fetch", "--write", "--copy-fetch", "--copy-write"):
        t.add_argument(name, required=True)
    t.add_argument("--match", action="append", required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--alg", type=int, required=True)
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        print(stats(a.dir))
    else:
        print(json.dumps(traffic(a)))


if __name__ == "__main__":
    sys.exit(main())
