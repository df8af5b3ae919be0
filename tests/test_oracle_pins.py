"""Pins of the CPU oracle against what the paper and the mathematics fix.

Kolmakov & Zhang, "A Generalization of the Allreduce Operation"
(arXiv:2004.09362).  Each test names the passage it checks.  None of these
tests touches the GPU or the HIP library.
"""
import os

import numpy as np
import pytest

import oracle

ALL_SMALL_P = list(range(1, 41))
LARGE_P = [63, 64, 65, 96, 100, 127, 128]


def ceil_log2(P):
    return max(0, (P - 1).bit_length())


def ks(P):
    L = ceil_log2(P)
    return list(range(L, 2 * L + 1))


def blocks(n, P):
    """Balanced partition: the first n mod P blocks get one extra element."""
    q, m = divmod(n, P)
    lens = [q + (b < m) for b in range(P)]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(int)
    return lens, offs


def block_of_cols(n, P):
    lens, offs = blocks(n, P)
    out = np.empty(n, dtype=int)
    for b in range(P):
        out[offs[b]:offs[b + 1]] = b
    return out


# ---------------------------------------------------------------------------
# Golden trees from the paper's worked examples
# ---------------------------------------------------------------------------

def parse_tree(s):
    pos = 0

    def rec():
        nonlocal pos
        if s[pos] == "(":
            pos += 1
            a = rec()
            assert s[pos] == "+"
            pos += 1
            b = rec()
            assert s[pos] == ")"
            pos += 1
            return (a, b)
        j = pos
        while pos < len(s) and s[pos].isdigit():
            pos += 1
        return int(s[j:pos])

    t = rec()
    assert pos == len(s)
    return t


def rotate(t, root, P):
    if isinstance(t, tuple):
        return (rotate(t[0], root, P), rotate(t[1], root, P))
    return (t + root) % P


def render(t):
    if isinstance(t, tuple):
        return "(%s+%s)" % (render(t[0]), render(t[1]))
    return str(t)


def eval_f32(t, col):
    """Evaluate a tree in float32, one rounding per combination."""
    if isinstance(t, tuple):
        return np.float32(eval_f32(t[0], col) + eval_f32(t[1], col))
    return np.float32(col[t])


def leaves(t):
    if isinstance(t, tuple):
        return leaves(t[0]) + leaves(t[1])
    return [t]


def load_golden(golden_dir):
    cases = []
    with open(os.path.join(golden_dir, "paper_trees.txt")) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            f = line.split()
            P, k, rule, tree = int(f[0]), int(f[1]), f[2], parse_tree(f[3])
            offs = [int(v) for v in f[4:]]
            assert sorted(leaves(tree)) == list(range(P)), "fixture tree must hold every rank once"
            if rule == "table":
                assert len(offs) == P
            cases.append((P, k, rule, tree, offs))
    return cases


def golden_root(P, rule, offs, x, b):
    if rule == "block":
        return b
    if rule == "rank":
        return x
    return (b + offs[(x - b) % P]) % P


def test_golden_fixture_covers_paper_examples(golden_dir):
    got = {(P, k) for P, k, *_ in load_golden(golden_dir)}
    assert {(7, 6), (7, 3), (7, 5), (3, 4), (3, 3), (3, 2)} <= got


def test_trees_match_paper_worked_examples(golden_dir):
    """Sec. 7 even/odd/last-step equations at P=7 (and P=3), Sec. 8 shift,
    Sec. 9 latency-optimal equations: the symbolic replay reproduces the
    hand-derived trees for every rank and block."""
    for P, k, rule, tree, offs in load_golden(golden_dir):
        t = oracle.Terms(P, k)
        assert t.violations == 0
        for x in range(P):
            for b in range(P):
                want = render(rotate(tree, golden_root(P, rule, offs, x, b), P))
                assert t.tree(x, b) == want, (P, k, x, b)


def test_fp32_replay_bits_follow_paper_trees(golden_dir):
    """The value replay rounds exactly as the paper's trees say (float32,
    one rounding per combination), on values whose sum depends on the order."""
    rng = np.random.default_rng(7)
    for P, k, rule, tree, offs in load_golden(golden_dir):
        n = 5 * P + 2  # ragged: P does not divide n
        mant = rng.uniform(-1, 1, size=(P, n))
        expo = rng.integers(-20, 20, size=(P, n))
        x = (mant * np.exp2(expo)).astype(np.float32)
        out = oracle.allreduce(x, k, "sum")
        bcol = block_of_cols(n, P)
        mismatched_if_other_order = 0
        for r in range(P):
            for e in range(n):
                t = rotate(tree, golden_root(P, rule, offs, r, bcol[e]), P)
                want = eval_f32(t, x[:, e])
                assert out[r, e].view(np.uint32) == np.float32(want).view(np.uint32), (P, k, r, e)
                # the left-to-right sum usually differs: the check has teeth
                lin = np.float32(0)
                for y in range(P):
                    lin = np.float32(lin + x[y, e])
                mismatched_if_other_order += int(lin != want)
        if P > 3:
            assert mismatched_if_other_order > 0


# ---------------------------------------------------------------------------
# Exactly-once coverage and the plain definition
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P", ALL_SMALL_P + LARGE_P)
def test_every_output_holds_each_rank_once(P):
    """Sec. 5.4: only co-placed blocks with equal indices combine; the final
    vector is the combination of all P inputs.  Symbolic run: every
    combination joins disjoint rank sets of one block, and every output holds
    all P ranks of its own block."""
    full = set(range(P))
    for k in ks(P):
        t = oracle.Terms(P, k)
        assert t.violations == 0, (P, k)
        for x in range(P):
            for b in range(P):
                node = t.ids[x, b]
                assert t.block(node) == b
                assert t.ranks(node) == full, (P, k, x, b)


@pytest.mark.parametrize("P", range(2, 32))
def test_brute_force_tag_inputs(P):
    """Rank x contributes 1 << x: any missed or doubled term changes the sum
    (definition of Allreduce, Sec. 1)."""
    want = (1 << P) - 1
    for k in ks(P):
        for n in (1, P - 1, P, 2 * P + 3):
            x = np.stack([np.full(n, 1 << y, dtype=np.int64) for y in range(P)]).astype(np.int32)
            out = oracle.allreduce(x, k, "sum")
            assert np.all(out.astype(np.int64) & 0xFFFFFFFF == want), (P, k, n)


@pytest.mark.parametrize("P", list(range(1, 21)) + [37, 64, 127, 128])
def test_int32_and_max_exact_against_definition(P):
    """int32 sums (wrapping modulo 2^32) and max are order-independent, so
    the replay must equal the direct definition exactly."""
    rng = np.random.default_rng(P)
    n = 3 * P + 5
    xi = rng.integers(-2**31, 2**31, size=(P, n), dtype=np.int64).astype(np.int32)
    xf = rng.normal(size=(P, n)).astype(np.float32)
    want_sum = xi.astype(np.int64).sum(axis=0)
    want_sum = ((want_sum + 2**31) % 2**32 - 2**31).astype(np.int32)
    want_max = xi.max(axis=0)
    want_fmax = xf.max(axis=0)
    assert np.array_equal(oracle.direct(xi, "sum"), want_sum)
    assert np.array_equal(oracle.direct(xi, "max"), want_max)
    assert np.array_equal(oracle.direct(xf, "max"), want_fmax)
    for k in (ks(P) if P <= 20 else [ks(P)[0], ks(P)[len(ks(P)) // 2], ks(P)[-1]]):
        assert np.array_equal(oracle.allreduce(xi, k, "sum"), np.broadcast_to(want_sum, (P, n))), k
        assert np.array_equal(oracle.allreduce(xi, k, "max"), np.broadcast_to(want_max, (P, n))), k
        assert np.array_equal(oracle.allreduce(xf, k, "max"), np.broadcast_to(want_fmax, (P, n))), k


@pytest.mark.parametrize("P", [2, 3, 5, 7, 12, 24, 37, 64, 127, 128])
def test_fp32_sum_within_rounding_bound(P):
    """fp32 sums: a tree of depth <= ceil(log2 P) (one level per reduction
    step) is within depth * 2^-24 * sum|V| of the exact sum; the target
    bound is 1e-5 of sum|V| against the fp64 direct sum."""
    rng = np.random.default_rng(100 + P)
    n = 2 * P + 3
    x = rng.normal(size=(P, n)).astype(np.float32)
    s64 = x.astype(np.float64).sum(axis=0)
    assert np.allclose(oracle.direct(x, "sum"), s64, rtol=0, atol=1e-12)
    mag = np.abs(x.astype(np.float64)).sum(axis=0)
    L = ceil_log2(P)
    for k in ks(P):
        out = oracle.allreduce(x, k, "sum").astype(np.float64)
        err = np.abs(out - s64) / mag
        assert err.max() <= 1e-5
        assert err.max() <= 1.01 * L * 2.0**-24 + 1e-12


# ---------------------------------------------------------------------------
# Steps and traffic against the cost equations (Secs. 7-9)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P", range(1, 129))
def test_steps_and_traffic_match_cost_equations(P):
    """Sec. 7 cost: 2*ceil(log P) steps, 2(P-1) blocks sent per rank, P-1
    combinations.  Sec. 8 cost: 2*ceil(log P) - r steps and
    2(P-1) + (2^r - 1)(ceil(log P) - 1) blocks; exact while the 2^r shifted
    schedules do not wrap round the P placements (2^r <= ceil(P/2) + 1),
    fewer otherwise; combinations at most (P-1) + (2^r-1)(2 ceil(log P) - 2).
    Sec. 9 cost: ceil(log P) steps, P ceil(log P) blocks, at most
    P (2 ceil(log P) - 2) combinations."""
    L = ceil_log2(P)
    for k in ks(P):
        r = 2 * L - k
        t = oracle.Terms(P, k)
        tr = t.trace
        assert (tr.rs_steps, tr.ag_steps) == (L, L - r)
        assert tr.rs_steps + tr.ag_steps == k
        ns = k
        pulls = list(tr.pulls[:ns])
        total = sum(pulls)
        combines = sum(tr.combines[:L])
        # every rank receives the same number of blocks (translation invariance)
        for s in range(ns):
            per_rank = {sum(bin(int(w)).count("1") for w in tr.recv_blocks[s][x]) for x in range(P)}
            assert per_rank == {pulls[s]}, (P, k, s)
        # a rank never receives two different vectors of one block in a step
        for s in range(L):
            got = sum(bin(int(w)).count("1") for w in tr.recv_blocks[s][0])
            assert got == pulls[s]
        if P == 1:
            assert total == 0 and combines == 0
            continue
        if r == 0:
            assert total == 2 * (P - 1)
            assert combines == P - 1
        elif r == L:
            assert total == L * P
            assert combines <= P * (2 * L - 2) or P == 2
        else:
            bound = 2 * (P - 1) + (2 ** r - 1) * (L - 1)
            if 2 ** r <= (P + 1) // 2 + 1:
                assert total == bound, (P, k)
            else:
                assert total < bound, (P, k)
            assert combines <= (P - 1) + (2 ** r - 1) * (2 * L - 2)
        # the reduction phase sends f_i + w - 1 blocks per step unless it wraps
        w = min(2 ** r, P)
        N = P
        for i in range(L):
            f = N // 2
            assert pulls[i] == min(P, f + w - 1), (P, k, i)
            N -= f
        # the distribution phase delivers the P - w placements not held
        assert sum(pulls[L:]) == P - w


def test_latency_optimal_p7_combination_count():
    """Sec. 9: at P=7 the primed vectors combine at every step but the last and
    the starred ones at the even step and the last: 7 + 14 + 7 = P(2L-2)."""
    tr = oracle.Terms(7, 3).trace
    assert list(tr.combines[:3]) == [7, 14, 7]


@pytest.mark.parametrize("P", [2, 4, 8, 16, 32, 64, 128])
def test_power_of_two_starred_equals_primed(P):
    """Power-of-two P: every N_i is even, no vector is ever left out, so the
    starred and primed vectors coincide and LO combines once per placement and
    step (P * log P), moving n elements per rank each step as Recursive
    Doubling does (Sec. 8, the closing remark)."""
    L = ceil_log2(P)
    tr = oracle.Terms(P, L).trace
    assert list(tr.combines[:L]) == [P] * L
    assert list(tr.pulls[:L]) == [P] * L


def test_total_bytes_equal_blocks_times_n():
    """Whatever the ragged partition, summed over all ranks the bytes moved
    are (blocks per rank) * n * element size."""
    for P, k in [(7, 5), (24, 10), (37, 8), (37, 7), (12, 4), (127, 10)]:
        n = 10 * P + 3
        lens, _ = blocks(n, P)
        x = np.zeros((P, n), np.int32)
        _, tr = oracle.allreduce(x, k, "sum", trace=True)
        total_elems = 0
        for s in range(tr.rs_steps + tr.ag_steps):
            for r in range(P):
                for b in range(P):
                    if (int(tr.recv_blocks[s][r][b >> 6]) >> (b & 63)) & 1:
                        total_elems += lens[b]
        assert total_elems == sum(tr.pulls[:tr.rs_steps + tr.ag_steps]) * n


def test_distribution_fetches_only_missing_placements():
    """P=37, k=7: 32 shifted schedules wrap round the 37 placements; the
    distribution delivers only the 5 placements not held (212 blocks per rank
    in total, below the Sec. 8 equation's 227, which assumes no wrap)."""
    tr = oracle.Terms(37, 7).trace
    assert list(tr.pulls[:7]) == [37, 37, 36, 33, 32, 32, 5]
    assert sum(tr.pulls[:7]) == 212


# ---------------------------------------------------------------------------
# Special cases
# ---------------------------------------------------------------------------

def test_single_rank_is_identity():
    x = np.arange(10, dtype=np.int32)[None, :]
    assert np.array_equal(oracle.allreduce(x, 0, "sum"), x)
    with pytest.raises(ValueError):
        oracle.allreduce(x, 1, "sum")


def test_two_ranks():
    """P=2: one exchange.  k=1 (latency-optimal) pulls the whole vector once;
    k=2 (bandwidth-optimal) swaps one block each way in each phase
    (Sec. 7: the last step is the only one for P=2)."""
    t1 = oracle.Terms(2, 1)
    assert [t1.tree(x, b) for x in range(2) for b in range(2)] == ["(0+1)", "(0+1)", "(1+0)", "(1+0)"]
    assert list(t1.trace.pulls[:1]) == [2]
    t2 = oracle.Terms(2, 2)
    assert [t2.tree(x, b) for x in range(2) for b in range(2)] == ["(0+1)", "(1+0)", "(0+1)", "(1+0)"]
    assert list(t2.trace.pulls[:2]) == [1, 1]


def test_rejects_out_of_range_k_and_P():
    x = np.zeros((5, 8), np.int32)
    for k in (2, 7):
        with pytest.raises(ValueError):
            oracle.allreduce(x, k, "sum")
    with pytest.raises(ValueError):
        oracle.allreduce(np.zeros((129, 4), np.int32), 14, "sum")


def test_empty_vector():
    x = np.zeros((5, 0), np.float32)
    assert oracle.allreduce(x, 3, "sum").shape == (5, 0)


def test_sampled_columns_equal_full_run():
    """Each column's tree depends only on its block, so replaying a sample of
    columns gives the full run's values at those columns."""
    rng = np.random.default_rng(3)
    for P, k in [(7, 5), (24, 10), (37, 8), (13, 4)]:
        n = 9 * P + 4
        x = rng.normal(size=(P, n)).astype(np.float32)
        full = oracle.allreduce(x, k, "sum")
        cols = np.sort(rng.choice(n, size=n // 3, replace=False))
        part = oracle.allreduce(x[:, cols], k, "sum", n=n, cols=cols)
        assert np.array_equal(part.view(np.uint32), full[:, cols].view(np.uint32))


def test_batched_instances_are_independent():
    rng = np.random.default_rng(4)
    P, n, B, k = 6, 23, 5, 3
    x = rng.normal(size=(P, B, n)).astype(np.float32)
    out = oracle.allreduce_batched(x, k, "sum")
    for j in range(B):
        assert np.array_equal(out[:, j].view(np.uint32), oracle.allreduce(x[:, j], k, "sum").view(np.uint32))
