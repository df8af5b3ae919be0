"""The oracle's pins have teeth: plant plausible mistakes in a copy of the
oracle source (on the CPU, never in the HIP path) and check that the pinned
properties catch every one of them."""
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
from test_oracle_groups import group_root, load_group_golden, relabel, textbook_hybrid_xor, textbook_ring
from test_oracle_pins import golden_root, load_golden, render, rotate

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

# (name, original text, planted mistake)
MUTANTS = [
    ("ceil instead of floor for the operator t^-floor(N/2)",
     "s->f[i] = s->N[i] / 2;", "s->f[i] = (s->N[i] + 1) / 2;"),
    ("received operand first",
     "int32_t id = terms_combine(terms, a[e], b[e]);", "int32_t id = terms_combine(terms, b[e], a[e]);"),
    ("fp32 received operand first in max",
     "for (e = 0; e < len; ++e) d[e] = b[e] > a[e] ? b[e] : a[e];\n      return 0;\n    }\n    case ORC_TERM",
     "for (e = 0; e < len; ++e) d[e] = b[e] >= a[e] ? b[e] : a[e];\n      return 0;\n    }\n    case ORC_TERM"),
    ("receive from x - f in the reduction phase",
     "int32_t y = grp_mul(g, x, f, P);", "int32_t y = grp_mul(g, x, grp_inv(g, f, P), P);"),
    ("one vector of the sent set dropped",
     "for (int32_t v = c; v < N; ++v) {\n          int32_t kept",
     "for (int32_t v = c + 1; v < N; ++v) {\n          int32_t kept"),
    ("distribution refetches held placements",
     "const int32_t lo = s.c[i] > h ? s.c[i] : h;", "const int32_t lo = s.c[i];"),
    ("shift count off by one",
     "s->w = (1 << s->r) < P ? (1 << s->r) : P;", "s->w = (1 << s->r) < P ? (1 << s->r) + (s->r > 0) - (s->r > 1) * 0 : P;"),
    ("distribution pulls from x + f",
     "int32_t y = grp_mul(g, x, grp_inv(g, f, P), P);", "int32_t y = grp_mul(g, x, f, P);"),
    ("XOR inverse taken as the cyclic negation",
     "return g == ORC_GROUP_XOR ? a : mod_p(-(int64_t)a, P);", "return mod_p(-(int64_t)a, P);"),
    ("XOR product taken as addition",
     "return g == ORC_GROUP_XOR ? (a ^ b) : mod_p((int64_t)a + b, P);", "return mod_p((int64_t)a + b, P);"),
    ("ring receives from x + 1",
     "int32_t y = mod_p((int64_t)x - 1, P);", "int32_t y = mod_p((int64_t)x + 1, P);"),
    ("ring combines the wrong placement",
     "int32_t b = mod_p((int64_t)x - to_p, P);", "int32_t b = mod_p((int64_t)x - from_p, P);"),
    ("ring stops one distribution step early",
     "step < 2 * (P - 1) && rc == 0", "step < 2 * (P - 1) - 1 && rc == 0"),
]


def battery(L, golden_dir):
    """Return the list of pinned properties the given oracle build violates."""
    fails = []
    # paper trees
    try:
        for P, k, rule, tree, offs in load_golden(golden_dir):
            t = oracle.Terms(P, k, lib_=L)
            for x in range(P):
                for b in range(P):
                    if t.tree(x, b) != render(rotate(tree, golden_root(P, rule, offs, x, b), P)):
                        raise AssertionError
    except Exception:
        fails.append("golden trees")
    # other groups and schedules: hand-derived trees and textbook formulations
    try:
        for group, sched, P, k, rule, tree, offs in load_group_golden(golden_dir):
            t = oracle.Terms(P, k, lib_=L, group=group, schedule=sched)
            for x in range(P):
                for b in range(P):
                    if t.tree(x, b) != render(relabel(tree, group_root(group, P, rule, offs, x, b), group, P)):
                        raise AssertionError
        for P in (4, 8, 16):
            L2 = max(0, (P - 1).bit_length())
            for k in range(L2, 2 * L2 + 1):
                t, want = oracle.Terms(P, k, lib_=L, group="xor"), textbook_hybrid_xor(P, k)
                assert all(t.tree(x, b) == render(want[x][b]) for x in range(P) for b in range(P))
        for P in (2, 5, 9):
            t, want = oracle.Terms(P, 2 * (P - 1), lib_=L, schedule="ring"), textbook_ring(P)
            assert all(t.tree(x, b) == render(want[x][b]) for x in range(P) for b in range(P))
    except Exception:
        fails.append("groups")
    # exactly-once coverage and cost equations
    try:
        for P in (5, 6, 12, 37):
            L2 = max(0, (P - 1).bit_length())
            for k in range(L2, 2 * L2 + 1):
                t = oracle.Terms(P, k, lib_=L)
                assert t.violations == 0
                for x in range(P):
                    for b in range(P):
                        assert t.ranks(t.ids[x, b]) == set(range(P))
                tr = t.trace
                assert tr.rs_steps + tr.ag_steps == k
        tr = oracle.Terms(37, 7, lib_=L).trace
        assert sum(tr.pulls[:7]) == 212
    except Exception:
        fails.append("coverage / cost")
    # tag brute force and max against the definition
    try:
        for P in (3, 5, 7, 12):
            L2 = max(0, (P - 1).bit_length())
            for k in range(L2, 2 * L2 + 1):
                x = np.stack([np.full(2 * P + 1, 1 << y) for y in range(P)]).astype(np.int32)
                assert np.all(oracle.allreduce(x, k, "sum", lib_=L) == (1 << P) - 1)
        xf = np.zeros((5, 11), np.float32)
        xf[1] = -0.0
        out = oracle.allreduce(xf, 3, "max", lib_=L)
        assert np.array_equal(out.view(np.uint32), oracle.allreduce(xf, 3, "max").view(np.uint32))
    except Exception:
        fails.append("definition")
    return fails


def test_unmodified_oracle_passes_battery(golden_dir):
    assert battery(oracle.lib(), golden_dir) == []


@pytest.mark.parametrize("name,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, golden_dir, name, orig, mut):
    src = open(SRC).read()
    assert src.count(orig) == 1, "mutation anchor must be unique: " + name
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(orig, mut))
    so = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-std=c99", "-O2", "-fPIC", "-shared", "-ffp-contract=off", "-w", "-o", str(so),
                    str(path)], check=True)
    # A mutant may also crash (it can read cells the real schedule never
    # leaves unset), so it runs in a child process; any failure counts.
    code = ("import sys; sys.path[:0] = [%r, %r]; import oracle, test_oracle_mutants as m; "
            "f = m.battery(oracle.load_variant(%r), %r); print(f); sys.exit(3 if f else 0)"
            % (os.path.dirname(os.path.dirname(SRC)), os.path.dirname(__file__), str(so), golden_dir))
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=600)
    assert res.returncode != 0, "planted mistake not caught: " + name
