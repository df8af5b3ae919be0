"""Pins of the oracle's other groups and schedules.

Kolmakov & Zhang (arXiv:2004.09362) show that Ring (Sec. 6, the cyclic
group with the operator t at every step), Recursive Halving (Sec. 7,
closing remark) and Recursive Doubling (Sec. 9, closing remark) are special
cases of the generalized Allreduce, the last two with the group of Table 1b
(t_k(x) = x XOR k, power-of-two P).  These tests pin the oracle's replay of
them to hand-derived trees, to textbook formulations written here
independently of the oracle (in terms of ranks and block indices, not of
placements), and to the plain definition.  None touches the GPU.
"""
import os

import numpy as np
import pytest

import oracle
from test_oracle_pins import blocks, block_of_cols, eval_f32, leaves, parse_tree, render

POW2 = [2, 4, 8, 16, 32, 64, 128]


def ceil_log2(P):
    return max(0, (P - 1).bit_length())


def ks(P):
    L = ceil_log2(P)
    return list(range(L, 2 * L + 1))


def relabel(t, root, group, P):
    if isinstance(t, tuple):
        return (relabel(t[0], root, group, P), relabel(t[1], root, group, P))
    return (t ^ root) if group == "xor" else (t + root) % P


def load_group_golden(golden_dir):
    cases = []
    with open(os.path.join(golden_dir, "group_trees.txt")) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            f = line.split()
            group, sched, P, k, rule, tree = f[0], f[1], int(f[2]), int(f[3]), f[4], parse_tree(f[5])
            offs = [int(v) for v in f[6:]]
            assert sorted(leaves(tree)) == list(range(P)), "fixture tree must hold every rank once"
            if rule == "table":
                assert len(offs) == P
            cases.append((group, sched, P, k, rule, tree, offs))
    return cases


def group_root(group, P, rule, offs, x, b):
    if rule == "block":
        return b
    if rule == "rank":
        return x
    if group == "xor":
        return b ^ offs[x ^ b]
    return (b + offs[(x - b) % P]) % P


# ---------------------------------------------------------------------------
# Textbook formulations (symbolic: a leaf is a rank, a node a pair (own, recv))
# ---------------------------------------------------------------------------

def textbook_hybrid_xor(P, k):
    """Power-of-two P, dimensions taken from the highest bit down.  Reduce-
    scatter by recursive halving over distances P/2 .. w (rank x keeps the
    half of its blocks whose bit d agrees with x), recursive doubling of the
    held 2^r blocks over distances w/2 .. 1, then allgather over distances
    w .. P/2.  r = 2 log P - k, w = 2^r.  Returns trees[x][b]."""
    L = ceil_log2(P)
    r = 2 * L - k
    w = 1 << r
    held = [{b: x for b in range(P)} for x in range(P)]
    d = P // 2
    while d >= 1:
        new = []
        for x in range(P):
            y = x ^ d
            if d >= w:   # halving: keep the half matching x in bit d
                new.append({b: (held[x][b], held[y][b]) for b in held[x] if not ((b ^ x) & d)})
            else:        # doubling: combine everything held
                new.append({b: (held[x][b], held[y][b]) for b in held[x]})
        held = new
        d //= 2
    d = w
    while d < P:
        new = []
        for x in range(P):
            m = dict(held[x])
            for b, v in held[x ^ d].items():
                assert b not in m
                m[b] = v
            new.append(m)
        held = new
        d *= 2
    return held


def textbook_ring(P):
    """Ring: in reduce-scatter step s = 0 .. P-2 rank x passes its partial of
    chunk (x - s) mod P to rank x + 1, which combines its own chunk with it;
    then P - 1 allgather steps pass the finished chunk (x + 1 - s) mod P on."""
    held = [{b: x for b in range(P)} for x in range(P)]
    for s in range(P - 1):
        msgs = [((x + 1) % P, (x - s) % P, held[x][(x - s) % P]) for x in range(P)]
        for y, b, v in msgs:
            held[y][b] = (held[y][b], v)
    for s in range(P - 1):
        msgs = [((x + 1) % P, (x + 1 - s) % P, held[x][(x + 1 - s) % P]) for x in range(P)]
        for y, b, v in msgs:
            held[y][b] = v
    return held


# ---------------------------------------------------------------------------
# Trees
# ---------------------------------------------------------------------------

def test_group_golden_fixture_covers_examples(golden_dir):
    got = {(g, s, P, k) for g, s, P, k, *_ in load_group_golden(golden_dir)}
    assert {("cyclic", "ring", 7, 12), ("xor", "butterfly", 8, 6), ("xor", "butterfly", 8, 3),
            ("xor", "butterfly", 8, 5), ("xor", "butterfly", 8, 4)} <= got


def test_group_trees_match_hand_derived(golden_dir):
    """Sec. 6 ring reduction result at P = 7, 3, 2; the Sec. 7-9 equations
    with the group of Table 1b at P = 8 and 4, every k."""
    for group, sched, P, k, rule, tree, offs in load_group_golden(golden_dir):
        t = oracle.Terms(P, k, group=group, schedule=sched)
        assert t.violations == 0
        for x in range(P):
            for b in range(P):
                want = render(relabel(tree, group_root(group, P, rule, offs, x, b), group, P))
                assert t.tree(x, b) == want, (group, sched, P, k, x, b)


@pytest.mark.parametrize("P", [2, 4, 8, 16, 32])
def test_xor_group_is_textbook_halving_doubling(P):
    """With the group of Table 1b the replay equals Recursive Halving (k = 2 log P),
    Recursive Doubling (k = log P) and their hybrid (Secs. 7-9, closing
    remarks), operand for operand."""
    for k in ks(P):
        want = textbook_hybrid_xor(P, k)
        t = oracle.Terms(P, k, group="xor")
        assert t.violations == 0
        for x in range(P):
            for b in range(P):
                assert t.tree(x, b) == render(want[x][b]), (P, k, x, b)


@pytest.mark.parametrize("P", list(range(1, 21)) + [31, 37])
def test_ring_is_textbook_ring(P):
    """Sec. 6: the cyclic group with the operator t at every step is the Ring
    algorithm, 2(P-1) steps."""
    want = textbook_ring(P)
    t = oracle.Terms(P, 2 * (P - 1), schedule="ring")
    assert t.violations == 0
    for x in range(P):
        for b in range(P):
            assert t.tree(x, b) == render(want[x][b]), (P, x, b)


@pytest.mark.parametrize("P", POW2)
def test_xor_every_output_holds_each_rank_once(P):
    full = set(range(P))
    for k in ks(P):
        t = oracle.Terms(P, k, group="xor")
        assert t.violations == 0
        for x in range(P):
            for b in range(P):
                assert t.block(t.ids[x, b]) == b
                assert t.ranks(t.ids[x, b]) == full


# ---------------------------------------------------------------------------
# Values against the definition
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P", POW2)
def test_xor_tags_int_and_max_exact(P):
    rng = np.random.default_rng(500 + P)
    n = 3 * P + 5
    xi = rng.integers(-2**31, 2**31, size=(P, n), dtype=np.int64).astype(np.int32)
    xf = rng.normal(size=(P, n)).astype(np.float32)
    tags = np.stack([np.full(2 * P + 1, (1 << (y % 31)) + (y // 31), dtype=np.int64) for y in range(P)]).astype(np.int32)
    for k in ks(P):
        for arr, op in ((xi, "sum"), (xi, "max"), (xf, "max"), (tags, "sum")):
            got = oracle.allreduce(arr, k, op, group="xor")
            assert np.array_equal(got, np.broadcast_to(oracle.direct(arr, op).astype(arr.dtype), got.shape)), (P, k, op)


@pytest.mark.parametrize("P", list(range(1, 41)) + [64, 127, 128])
def test_ring_int_and_max_exact(P):
    rng = np.random.default_rng(700 + P)
    n = 2 * P + 3
    xi = rng.integers(-2**31, 2**31, size=(P, n), dtype=np.int64).astype(np.int32)
    xf = rng.normal(size=(P, n)).astype(np.float32)
    for arr, op in ((xi, "sum"), (xi, "max"), (xf, "max")):
        got = oracle.allreduce(arr, 2 * (P - 1), op, schedule="ring")
        assert np.array_equal(got, np.broadcast_to(oracle.direct(arr, op).astype(arr.dtype), got.shape)), (P, op)


@pytest.mark.parametrize("group,schedule,P", [("xor", "butterfly", 8), ("xor", "butterfly", 16),
                                              ("cyclic", "ring", 7), ("cyclic", "ring", 12)])
def test_fp32_bits_follow_textbook_trees(group, schedule, P):
    """float32, one rounding per combination in the textbook tree's order."""
    rng = np.random.default_rng(11 * P)
    n = 3 * P + 2
    x = (rng.uniform(-1, 1, size=(P, n)) * np.exp2(rng.integers(-20, 20, size=(P, n)))).astype(np.float32)
    bcol = block_of_cols(n, P)
    kk = [2 * (P - 1)] if schedule == "ring" else ks(P)
    for k in kk:
        want = textbook_ring(P) if schedule == "ring" else textbook_hybrid_xor(P, k)
        out = oracle.allreduce(x, k, "sum", group=group, schedule=schedule)
        for r in range(P):
            for e in range(n):
                assert out[r, e].view(np.uint32) == np.float32(eval_f32(want[r][bcol[e]], x[:, e])).view(np.uint32)


def test_ring_fp32_within_chain_bound():
    """The ring's chain has depth P - 1: error <= (P-1) 2^-24 sum|V|."""
    P = 37
    rng = np.random.default_rng(9)
    x = rng.normal(size=(P, 2 * P + 1)).astype(np.float32)
    s64 = x.astype(np.float64).sum(axis=0)
    mag = np.abs(x.astype(np.float64)).sum(axis=0)
    out = oracle.allreduce(x, 2 * (P - 1), "sum", schedule="ring").astype(np.float64)
    assert (np.abs(out - s64) / mag).max() <= 1.01 * (P - 1) * 2.0**-24


# ---------------------------------------------------------------------------
# Steps and traffic
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P", POW2)
def test_xor_traffic(P):
    """Group of Table 1b: the shifts s < w = 2^r form a subgroup, so the w
    shifted schedules share every vector while f_i >= w; a reduction step
    then sends and combines max(f_i, w) blocks, and the distribution sends
    f_i at each of its L - r steps.  r = 0 is the Sec. 7 cost (2(P-1) blocks,
    P-1 combinations), r = L Recursive Doubling (P blocks a step)."""
    L = ceil_log2(P)
    for k in ks(P):
        r = 2 * L - k
        w = 1 << r
        t = oracle.Terms(P, k, group="xor")
        tr = t.trace
        assert (tr.rs_steps, tr.ag_steps) == (L, L - r)
        f = [P >> (i + 1) for i in range(L)]
        assert list(tr.pulls[:L]) == [max(fi, w) for fi in f]
        assert list(tr.combines[:L]) == [max(fi, w) for fi in f]
        assert list(tr.pulls[L:k]) == [f[i] for i in reversed(range(L - r))]
        assert list(tr.step_peer[:L]) == f
        if r == 0:
            assert sum(tr.pulls[:k]) == 2 * (P - 1) and sum(tr.combines[:L]) == P - 1
        if r == L:
            assert sum(tr.pulls[:k]) == L * P


@pytest.mark.parametrize("P", range(2, 10))
def test_ring_steps_and_blocks(P):
    """Sec. 6: 2(P-1) steps, one block per rank each (2(P-1) blocks), P-1
    combinations; at reduction step i rank x receives block x - 1 - i, at
    distribution step j block x - j (ranks pass along the ring)."""
    k = 2 * (P - 1)
    _, tr = oracle.allreduce(np.zeros((P, 3 * P), np.int32), k, "sum", schedule="ring", trace=True)
    assert (tr.rs_steps, tr.ag_steps) == (P - 1, P - 1)
    assert list(tr.pulls[:k]) == [1] * k
    for s in range(k):
        for x in range(P):
            b = (x - 1 - s) % P if s < P - 1 else (x - (s - (P - 1))) % P
            mask = [int(tr.recv_blocks[s][x][0]), int(tr.recv_blocks[s][x][1])]
            assert mask == [1 << b, 0], (P, s, x)
    t = oracle.Terms(P, k, schedule="ring")
    assert sum(t.trace.combines[:P - 1]) == P - 1


def test_ring_total_bytes():
    """Ragged partition: the ring moves 2(P-1) blocks per rank, i.e.
    2 (P-1) n elements over all ranks."""
    for P in (3, 5, 7):
        n = 10 * P + 3
        lens, _ = blocks(n, P)
        _, tr = oracle.allreduce(np.zeros((P, n), np.int32), 2 * (P - 1), "sum", schedule="ring", trace=True)
        tot = 0
        for s in range(2 * (P - 1)):
            for x in range(P):
                for b in range(P):
                    if (int(tr.recv_blocks[s][x][b >> 6]) >> (b & 63)) & 1:
                        tot += lens[b]
        assert tot == 2 * (P - 1) * n


# ---------------------------------------------------------------------------
# Special cases and rejections
# ---------------------------------------------------------------------------

def test_single_rank_and_empty():
    x = np.arange(6, dtype=np.int32)[None, :]
    assert np.array_equal(oracle.allreduce(x, 0, "sum", schedule="ring"), x)
    assert oracle.allreduce(np.zeros((4, 0), np.float32), 3, "sum", group="xor").shape == (4, 0)
    assert oracle.allreduce(np.zeros((5, 0), np.float32), 8, "sum", schedule="ring").shape == (5, 0)


def test_xor_two_ranks_equals_cyclic():
    """P = 2: both groups have the one transposition (0 1)."""
    for k in (1, 2):
        a, b = oracle.Terms(2, k), oracle.Terms(2, k, group="xor")
        assert [a.tree(x, c) for x in range(2) for c in range(2)] == [b.tree(x, c) for x in range(2) for c in range(2)]


def test_rejections():
    x6 = np.zeros((6, 8), np.int32)
    with pytest.raises(ValueError):
        oracle.allreduce(x6, 3, "sum", group="xor")          # not a power of two
    with pytest.raises(ValueError):
        oracle.allreduce(x6, 9, "sum", schedule="ring")      # ring needs k = 2(P-1)
    with pytest.raises(ValueError):
        oracle.allreduce(np.zeros((4, 8), np.int32), 6, "sum", group="xor", schedule="ring")
    with pytest.raises(ValueError):
        oracle.allreduce(np.zeros((8, 8), np.int32), 7, "sum", group="xor")  # k outside [L, 2L]


def test_batched_groups():
    rng = np.random.default_rng(5)
    for P, k, g, s in ((8, 4, "xor", "butterfly"), (5, 8, "cyclic", "ring")):
        x = rng.normal(size=(P, 3, 4 * P + 1)).astype(np.float32)
        out = oracle.allreduce_batched(x, k, "sum", group=g, schedule=s)
        for j in range(3):
            want = oracle.allreduce(x[:, j], k, "sum", group=g, schedule=s)
            assert np.array_equal(out[:, j].view(np.uint32), want.view(np.uint32))
