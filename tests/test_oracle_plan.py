"""Pins for the planner oracle (CPU only).

- hand-worked costs, Eq. 3 values, greedy and zig-zag assignments and
  optima (tests/golden/plan_worked_example.txt);
- brute force on tiny inputs: the greedy never beats the optimum, and when
  the capacity does not bind it stays within Graham's LPT bound
  (4/3 - 1/(3M)) * OPT;
- special cases with known answers (n <= M, equal costs, one microbatch);
- I8: each sample at most once, capacity respected.
"""

import math

import numpy as np
import pytest

from oracle.plan import (brute_force, cost_scaled, eq3_cost, greedy_partition, imbalance, members, snake,
                         zigzag_partition)
from conftest import read_golden


def _kv_lists(fields):
    """'K 10 C 15 M 2 lengths 5 9 ...' -> dict of name -> list of ints."""
    out, key = {}, None
    for f in fields:
        if f.lstrip("-").isdigit():
            out[key].append(int(f))
        else:
            key = f
            out[key] = []
    return out


def test_worked_examples():
    seen = set()
    for ln in read_golden("plan_worked_example.txt"):
        f = ln.split()
        seen.add(f[0])
        if f[0] == "cost":
            assert cost_scaled(int(f[1]), int(f[2])) == int(f[3])
        elif f[0] == "eq3":
            L = int(f[1])
            eq = f.index("=")
            lens = [int(x) for x in f[2:eq]]
            assert math.isclose(eq3_cost(lens, L), float(f[eq + 1]), rel_tol=1e-15)
        elif f[0] == "greedy":
            arrow = f.index("->")
            a = _kv_lists(f[1:arrow])
            b = _kv_lists(f[arrow + 1:])
            assign, tok, cst = greedy_partition(a["lengths"], a["K"][0], a["C"][0], a["M"][0])
            assert assign == b["assign"] and tok == b["tokens"] and cst == b["cost"]
        elif f[0] == "zigzag":
            arrow = f.index("->")
            a = _kv_lists(f[1:arrow])
            b = _kv_lists(f[arrow + 1:])
            assign, tok, cst = zigzag_partition(a["lengths"], a["K"][0], a["C"][0], a["M"][0])
            assert assign == b["assign"] and tok == b["tokens"] and cst == b["cost"]
        elif f[0] == "opt":
            eq = f.index("=")
            a = _kv_lists(f[1:eq])
            opt, _ = brute_force(a["lengths"], a["K"][0], a["C"][0], a["M"][0])
            assert opt == int(f[eq + 1])
        elif f[0] == "lex":
            eq = f.index("=")
            a = _kv_lists(f[1:eq])
            _, lex = brute_force(a["lengths"], a["K"][0], a["C"][0], a["M"][0])
            assert lex == (int(f[eq + 1]), -int(f[eq + 2]))
    assert seen == {"cost", "eq3", "greedy", "zigzag", "opt", "lex"}


def _check_plan(lengths, capacity, n_mb, assign, tok, cst, k):
    assert len(assign) == len(lengths)
    for j in range(n_mb):
        mem = [i for i, a in enumerate(assign) if a == j]
        assert sum(lengths[i] for i in mem) == tok[j] <= capacity
        assert sum(cost_scaled(lengths[i], k) for i in mem) == cst[j]


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_bounds(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 8))
    M = int(rng.integers(1, 4))
    K = int(rng.integers(1, 50))
    lengths = [int(x) for x in rng.integers(1, 40, size=n)]
    binding = bool(rng.integers(0, 2))
    C = int(rng.integers(max(lengths), 2 * max(lengths) + 1)) if binding else sum(lengths)
    assign, tok, cst = greedy_partition(lengths, K, C, M)
    _check_plan(lengths, C, M, assign, tok, cst, K)
    opt, lex = brute_force(lengths, K, C, M)
    if -1 not in assign:
        assert opt is not None and max(cst) >= opt
    assert sum(tok) <= lex[0]
    if not binding:
        assert -1 not in assign
        assert max(cst) <= (4 / 3 - 1 / (3 * M)) * opt + 1e-9


def test_greedy_strictly_worse_than_opt_within_bound():
    # Classic LPT example; the ratio approaches Graham's 7/6 for M = 2.
    for K in (10, 1000, 10 ** 6):
        lengths = [3, 3, 2, 2, 2]
        _, _, cst = greedy_partition(lengths, K, 100, 2)
        opt, _ = brute_force(lengths, K, 100, 2)
        assert max(cst) == 7 * K + 17 and opt == 6 * K + 18
        assert opt < max(cst) <= (4 / 3 - 1 / 6) * opt


def test_special_cases():
    # n <= M: one sample per microbatch, max cost = the largest sample's cost.
    lengths = [5, 17, 3]
    a, tok, cst = greedy_partition(lengths, 8, 100, 4)
    assert sorted(a) == [0, 1, 2] and max(cst) == cost_scaled(17, 8) == brute_force(lengths, 8, 100, 4)[0]
    # n = q*M equal lengths: q per microbatch, optimal.
    a, tok, cst = greedy_partition([7] * 12, 5, 1000, 4)
    assert tok == [21] * 4 and cst == [3 * cost_scaled(7, 5)] * 4
    # M = 1: longest first, everything that still fits.
    a, tok, cst = greedy_partition([4, 9, 2, 6], 3, 12, 1)
    assert a == [-1, 0, 0, -1] and tok == [11]
    # Nothing fits.
    a, tok, cst = greedy_partition([13, 20], 3, 12, 2)
    assert a == [-1, -1] and tok == [0, 0]
    # Empty input.
    assert greedy_partition([], 3, 12, 2) == ([], [0, 0], [0, 0])


def test_members_keep_input_order_and_imbalance():
    assign = [1, 0, 1, -1, 0]
    assert members(assign, 3) == [[1, 4], [0, 2], []]
    assert imbalance([2, 4, 6]) == 1.5


def test_snake_order():
    assert [snake(p, 3) for p in range(13)] == [0, 1, 2, 2, 1, 0, 0, 1, 2, 2, 1, 0, 0]
    assert [snake(p, 1) for p in range(4)] == [0, 0, 0, 0]


@pytest.mark.parametrize("seed", range(20))
def test_zigzag_properties(seed):
    """I8 for the zig-zag policy; without a binding capacity the sample at
    sorted position p lands in snake(p); with one microbatch it is the greedy."""
    rng = np.random.default_rng(600 + seed)
    n, m, k = int(rng.integers(0, 30)), int(rng.integers(1, 6)), int(rng.integers(1, 5000))
    lengths = rng.integers(1, 200, size=n).tolist()
    for capacity in (10 ** 9, int(rng.integers(1, 600))):
        assign, tok, cst = zigzag_partition(lengths, k, capacity, m)
        _check_plan(lengths, capacity, m, assign, tok, cst, k)
        if capacity == 10 ** 9:
            order = sorted(range(n), key=lambda i: (-cost_scaled(lengths[i], k), i))
            assert [assign[i] for i in order] == [snake(p, m) for p in range(n)]
        for i, a in enumerate(assign):            # a deferred sample fit in no microbatch then,
            if a < 0:                             # nor after (token counts only grow)
                assert all(t + lengths[i] > capacity for t in tok)
    assert zigzag_partition(lengths, k, 300, 1) == greedy_partition(lengths, k, 300, 1)


def _turns(lengths, k):
    """Samples in the order both policies take them: decreasing cost, ties by lower index."""
    costs = [cost_scaled(int(l), k) for l in lengths]
    return sorted(range(len(lengths)), key=lambda i: (-costs[i], i)), costs


@pytest.mark.parametrize("seed", range(30))
def test_greedy_certificate(seed):
    """Reading R11, checked on the output alone: replaying the assignment in
    the samples' turn order, each placed sample went to a microbatch of
    least accumulated cost among those with room at its turn, the lowest
    index among equals, and each deferred sample fit in none. Random inputs
    with many equal lengths, so the tie rules decide often."""
    rng = np.random.default_rng(500 + seed)
    n, n_mb = int(rng.integers(1, 30)), int(rng.integers(1, 6))
    lengths = [int(x) for x in rng.choice([1, 2, 3, 5, 8, 13], size=n)]
    capacity, k = int(rng.integers(8, 40)), int(rng.choice([1, 10, 4096]))
    assign, tok, cst = greedy_partition(lengths, k, capacity, n_mb)
    order, costs = _turns(lengths, k)
    t, c = [0] * n_mb, [0] * n_mb
    for i in order:
        room = [j for j in range(n_mb) if t[j] + lengths[i] <= capacity]
        if not room:
            assert assign[i] == -1
            continue
        least = min(c[j] for j in room)
        assert assign[i] == min(j for j in room if c[j] == least)
        t[assign[i]] += lengths[i]
        c[assign[i]] += costs[i]
    assert t == tok and c == cst


@pytest.mark.parametrize("seed", range(30))
def test_zigzag_certificate(seed):
    """Reading R11's zig-zag form, checked on the output alone: the sample
    at turn p went to the first microbatch with room along the snake from
    position p (0, 1, ..., M-1, M-1, ..., 0, 0, 1, ...), and a deferred one
    found room in none."""
    rng = np.random.default_rng(600 + seed)
    n, n_mb = int(rng.integers(1, 30)), int(rng.integers(1, 6))
    lengths = [int(x) for x in rng.choice([1, 2, 3, 5, 8, 13], size=n)]
    capacity, k = int(rng.integers(8, 40)), int(rng.choice([1, 10, 4096]))
    assign, tok, cst = zigzag_partition(lengths, k, capacity, n_mb)
    order, costs = _turns(lengths, k)
    walk = [x for x in range(n_mb)] + [x for x in reversed(range(n_mb))]     # one period of the snake
    t = [0] * n_mb
    for p, i in enumerate(order):
        along = [walk[(p + q) % (2 * n_mb)] for q in range(2 * n_mb)]
        room = [j for j in along if t[j] + lengths[i] <= capacity]
        if not room:
            assert assign[i] == -1
            continue
        assert assign[i] == room[0]
        t[assign[i]] += lengths[i]
    assert t == tok
