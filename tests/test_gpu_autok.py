"""The automatic step count on the GPU (Sec. 8 chooses the number of steps
from the cost model; ar_plan_create_auto / AR_K_AUTO).  For P = 8, 37 and
127 over a sweep of message sizes:

  - the plan the model chose runs bit-exact against the oracle replaying the
    same k (full vectors up to 2^18 elements per rank, sampled columns above);
  - restricted to the step-wise path, where k changes the time, the chosen k
    is within REGRET of the fastest k measured on this GPU;
  - with the path chosen too, the plan is within REGRET of the fastest of
    every (path, k) measured.

REGRET bounds the measured time at the chosen k over the best, as the
step-count calibration reports it for the step-wise path (within 6 % at
most sizes, 14-16 % at the ends of its sweeps); the default parameters are
one fit for every P, hence the margin, and ABS_SLACK_S absorbs launch
jitter on executes of a few microseconds."""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar, synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
REGRET = 1.30
ABS_SLACK_S = 4e-6


def note(msg):
    print("[gpu] " + msg, flush=True)
    sys.stdout.flush()


def time_execute(plan, bufs, reps=20, trials=3):
    """Median over trials of the mean time of `reps` back-to-back executes."""
    for _ in range(3):
        plan(bufs)
    torch.cuda.synchronize()
    out = []
    for _ in range(trials):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            plan(bufs)
        e1.record()
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1) * 1e-3 / reps)
    return sorted(out)[len(out) // 2]


SWEEP = {8: [8 << e for e in (6, 10, 14, 18, 21)],
         37: [37 << e for e in (6, 9, 12, 15, 17)],
         127: [127 << e for e in (4, 7, 10, 13, 14)]}


def sampled_cols(n, P, per_block=48, seed=0):
    q, m = n // P, n % P
    rng = np.random.default_rng(seed)
    cols = []
    for b in range(P):
        off, ln = b * q + min(b, m), q + (1 if b < m else 0)
        pick = set(range(min(8, ln))) | set(range(max(0, ln - 8), ln))
        pick |= set(rng.integers(0, ln, size=min(per_block, ln)).tolist()) if ln else set()
        cols.extend(off + c for c in sorted(pick))
    return np.array(sorted(set(cols)), dtype=np.int64)


@pytest.mark.parametrize("P", [8, 37, 127])
def test_auto_plans_match_the_oracle_and_the_best_measured_k(P):
    L = max(0, (P - 1).bit_length())
    for n in SWEEP[P]:
        X0 = synth.device_ranks(synth.BASE_SEED + 4100 + P, P, n, np.float32, synth.Dist("normal", 0.0, 1.0), DEV)
        # 1. bits of the automatic plan against the oracle at its k
        plan = ar.Plan(P, n, "float32", "sum", "auto")
        st = plan.stats()
        note("auto P=%d n=%d -> k=%d path=%d" % (P, n, st.k, st.exec_path))
        assert L <= st.k <= 2 * L and st.exec_path == ar.AR_PATH_FUSED
        X = X0.clone()
        plan([X[i] for i in range(P)])
        torch.cuda.synchronize()
        if n <= (1 << 18):
            want = oracle.allreduce(X0.cpu().numpy(), st.k, "sum")
            got = X.cpu().numpy()
        else:
            cols = sampled_cols(n, P)
            idx = torch.from_numpy(cols).to(DEV)
            want = oracle.allreduce(X0[:, idx].cpu().numpy(), st.k, "sum", n=n, cols=cols)
            got = X[:, idx].cpu().numpy()
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), (P, n, st.k)
        # 2. timing: every k step-wise, and the fused path
        X = X0.clone()
        bufs = [X[i] for i in range(P)]
        t_step = {}
        for k in range(L, 2 * L + 1):
            p = ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_STEPWISE)
            t_step[k] = time_execute(p, bufs)
            p.close()
        pf = ar.Plan(P, n, "float32", "sum", st.k, path=ar.AR_PATH_FUSED)
        t_fused = time_execute(pf, bufs)
        pf.close()
        ps = ar.Plan(P, n, "float32", "sum", "auto", path=ar.AR_PATH_STEPWISE)
        assert ps.k == st.k and ps.stats().exec_path == ar.AR_PATH_STEPWISE
        best_k = min(t_step, key=t_step.get)
        note("  step-wise us by k: %s; fused %.1f us" % ({k: round(v * 1e6, 1) for k, v in t_step.items()},
                                                          t_fused * 1e6))
        assert t_step[ps.k] <= REGRET * t_step[best_k] + ABS_SLACK_S, (P, n, ps.k, best_k)
        t_auto = time_execute(plan, bufs)
        assert t_auto <= REGRET * min(min(t_step.values()), t_fused) + ABS_SLACK_S, (P, n, t_auto)
        plan.close()
        ps.close()
        del X, X0, bufs
        torch.cuda.empty_cache()
