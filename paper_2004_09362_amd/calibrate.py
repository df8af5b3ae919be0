"""Fit the paper's cost model to the step-wise path on this GPU, and check the
step count it chooses.

Kolmakov & Zhang (arXiv:2004.09362) price a k-step schedule with the model
of Sec. 2 -- alpha per step, beta per byte received, gamma per byte
combined -- and choose k (Sec. 8, optimal number of steps) from alpha,
beta, gamma measured on their cluster (Table 2).  On one GPU the step-wise
path has the same structure: each step is a kernel launch (alpha) whose
time grows with the blocks it pulls (beta) and combines (gamma).  This tool

  1. times the step-wise path for every k at a range of message sizes,
  2. fits alpha, beta, gamma by least squares (relative error) to
     tau = k * alpha + B * u * beta + C * u * gamma, with B and C the plan's
     blocks received and combinations per rank and u = 4n / P,
  3. reports, per size, the measured best k, the k chosen by the fitted
     model (ar_model_best_k on the paper's equations, and the plan-exact
     variant), and how much slower the chosen k is than the best.

With --graph the executes are captured into a HIP graph and replayed, which
removes most of the host's per-launch cost from alpha: the step barrier is
then the kernel boundary alone.  --group xor runs the XOR group's plans
(power-of-two P).

The same sweep also fits the library's own model (ar_model_params, which
ar_plan_create_auto uses): a step launch costs step_alpha plus its HBM
bytes over step_bytes_per_s, and the fused path fused_alpha per launch plus
its bytes over fused_bytes_per_s (the fused path is timed at every size
too).  The output reports the fitted values, and per size the k and path
ar_plan_create_auto picks with them and with the library's defaults, and
the regret of each choice against the fastest (path, k) measured.

Usage: python -m paper_2004_09362_amd.calibrate [--P 37] [--reps 20] [--graph]
Prints one JSON object.  Needs a GPU; all timing is of the library's
kernels through its C ABI.
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np
import torch

from . import ar


def ceil_log2(P: int) -> int:
    return max(0, (P - 1).bit_length())


def time_plan_graph(plan: ar.Plan, bufs, reps: int) -> float:
    """Seconds per execute, `reps` executes captured in one graph, best of
    three replays."""
    plan(bufs)  # allocates the plan's scratch outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for _ in range(reps):
                plan(bufs)
    torch.cuda.synchronize()
    best = None
    for _ in range(3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / reps * 1e-3
        best = t if best is None else min(best, t)
    del g
    return best


def time_plan(plan: ar.Plan, bufs, reps: int, stream) -> float:
    """Seconds per execute, averaged over `reps` back-to-back executes."""
    for _ in range(3):
        plan(bufs, stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        plan(bufs, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps * 1e-3


def main(argv=None) -> dict:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--P", type=int, default=37)
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--min-exp", type=int, default=6, help="smallest n is P * 2^min_exp")
    ap.add_argument("--max-exp", type=int, default=17, help="largest n is P * 2^max_exp")
    ap.add_argument("--graph", action="store_true", help="time executes replayed from a HIP graph")
    ap.add_argument("--group", choices=["cyclic", "xor"], default="cyclic")
    args = ap.parse_args(argv)
    P = args.P
    L = ceil_log2(P)
    ks = list(range(L, 2 * L + 1))
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    sizes = [P * (1 << e) for e in range(args.min_exp, args.max_exp + 1)]
    rows = []
    for n in sizes:
        X = torch.randn(P, n, device=dev) * 1e-3
        bufs = [X[i] for i in range(P)]
        for k in ks:
            plan = ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_STEPWISE, group=args.group)
            st = plan.stats()
            t = time_plan_graph(plan, bufs, args.reps) if args.graph else time_plan(plan, bufs, args.reps, stream)
            rows.append(dict(n=n, k=k, t=t, B=st.blocks_pulled_per_rank, C=st.combines_per_rank,
                             launches=st.launches, u=4.0 * n / P, hbm=st.hbm_bytes_algorithmic))
            plan.close()
        del X
        torch.cuda.empty_cache()
        print("[calibrate] n=%d done" % n, file=sys.stderr, flush=True)

    # the fused path at every size (its time does not depend on k)
    fused_rows = []
    for n in sizes:
        X = torch.randn(P, n, device=dev) * 1e-3
        bufs = [X[i] for i in range(P)]
        plan = ar.Plan(P, n, "float32", "sum", 2 * L, path=ar.AR_PATH_FUSED, group=args.group)
        st = plan.stats()
        t = time_plan_graph(plan, bufs, args.reps) if args.graph else time_plan(plan, bufs, args.reps, stream)
        fused_rows.append(dict(n=n, t=t, launches=st.fused_launches, bytes=st.hbm_bytes_fused))
        plan.close()
        del X
        torch.cuda.empty_cache()

    # the library's model: launches * alpha + bytes / bandwidth, least squares on relative error
    def fit2(rows, nl, nb):
        A2 = np.array([[r[nl], r[nb]] for r in rows]) / np.array([[r["t"]] for r in rows])
        c, *_ = np.linalg.lstsq(A2, np.ones(len(rows)), rcond=None)
        a = max(float(c[0]), 0.0)
        inv_bw = max(float(c[1]), 1e-16)
        return a, 1.0 / inv_bw
    for r in rows:
        r["H"] = r["hbm"]
    step_alpha, step_bw = fit2(rows, "launches", "H")
    fused_alpha, fused_bw = fit2(fused_rows, "launches", "bytes")
    lib_fit = dict(step_alpha=step_alpha, step_bytes_per_s=step_bw, fused_alpha=fused_alpha,
                   fused_bytes_per_s=fused_bw)

    # least squares on relative error: (k a + B u b + C u g) / t = 1
    A = np.array([[r["k"], r["B"] * r["u"], r["C"] * r["u"]] for r in rows]) / np.array([[r["t"]] for r in rows])
    coef, *_ = np.linalg.lstsq(A, np.ones(len(rows)), rcond=None)
    alpha, beta, gamma = (max(float(c), 0.0) for c in coef)
    fit_err = [abs((r["k"] * alpha + r["B"] * r["u"] * beta + r["C"] * r["u"] * gamma) / r["t"] - 1) for r in rows]

    per_size = []
    for n in sizes:
        meas = {r["k"]: r["t"] for r in rows if r["n"] == n}
        best = min(meas, key=meas.get)
        k_eq, r_star = ar.ar_model_best_k(P, 4.0 * n, alpha, beta, gamma)
        exact = {}
        for k in ks:
            plan = ar.Plan(P, n, "float32", "sum", k, group=args.group)
            exact[k] = ar.ar_plan_model_time(plan.handle, alpha, beta, gamma)
            plan.close()
        k_exact = min(exact, key=exact.get)
        t_fused = next(r["t"] for r in fused_rows if r["n"] == n)
        best_any = min(min(meas.values()), t_fused)
        auto = {}
        for name, params in (("fitted", lib_fit), ("default", None)):
            h = ar.ar_plan_create_auto(P, n, "float32", "sum", args.group, 1, ar.AR_PATH_AUTO, params)
            sa = ar.ar_plan_stats(h)
            ar.ar_plan_destroy(h)
            hs = ar.ar_plan_create_auto(P, n, "float32", "sum", args.group, 1, ar.AR_PATH_STEPWISE, params)
            ks_ = ar.ar_plan_stats(hs).k
            ar.ar_plan_destroy(hs)
            t_auto = t_fused if sa.exec_path == ar.AR_PATH_FUSED else meas[sa.k]
            auto[name] = dict(k=sa.k, path="fused" if sa.exec_path == ar.AR_PATH_FUSED else "stepwise",
                              regret=round(t_auto / best_any, 4), stepwise_k=ks_,
                              stepwise_regret=round(meas[ks_] / meas[best], 4))
        per_size.append(dict(n=n, bytes=4 * n, measured_best_k=best, measured_us={k: round(v * 1e6, 2) for k, v in meas.items()},
                             fused_us=round(t_fused * 1e6, 2), library_auto=auto,
                             model_k=k_eq, model_k_exact=k_exact, r_closed_form=None if r_star != r_star else round(r_star, 3),
                             regret_model=round(meas[k_eq] / meas[best], 4),
                             regret_model_exact=round(meas[k_exact] / meas[best], 4)))
    out = dict(P=P, path="stepwise", group=args.group, graph=bool(args.graph), library_model_fit=lib_fit,
               alpha_s=alpha, beta_s_per_B=beta, gamma_s_per_B=gamma,
               fit_max_rel_err=round(max(fit_err), 4), fit_mean_rel_err=round(float(np.mean(fit_err)), 4),
               sizes=per_size)
    print(json.dumps(out), flush=True)
    return out


if __name__ == "__main__":
    main()
