"""Pins for the allocator oracle (Sec. 3.3, Eq. 1-2), CPU only.

- hand-worked flow-matching solutions and candidate lists
  (tests/golden/allocator_flow_example.txt);
- closed form: with an unlimited budget, G = min(best encoder sum, best
  backbone throughput), and F follows from the closest encoder sum;
- monotonicity: a larger budget never lowers G;
- the candidate rules hold for every listed configuration and no valid one
  is missing.
"""

import itertools

import numpy as np
import pytest

from conftest import read_golden
from oracle.allocate import candidates, divisors, solve


def _modules(words):
    mods, cur = [], None
    for w in words:
        if w in ("enc", "bb"):
            cur = []
            mods.append(cur)
        else:
            t, r = w.split(":")
            cur.append((int(t), int(r)))
    return mods


def test_worked_examples():
    kinds = set()
    for ln in read_golden("allocator_flow_example.txt"):
        head, _, tail = ln.partition("->")
        f = head.split()
        kinds.add(f[0])
        if f[0] == "solve":
            got = solve(_modules(f[3:]), int(f[2]))
            t = tail.split()
            if t == ["NONE"]:
                assert got is None
                continue
            gi = t.index("G")
            assert got == ([int(x) for x in t[:gi]], int(t[gi + 1]), int(t[gi + 3]), int(t[gi + 5]))
        else:
            kv = dict(zip(f[2::2], f[3::2]))
            want = [tuple(int(x) for x in c.split(",")) for c in tail.split()]
            assert candidates(f[1] == "backbone", int(kv["devices"]), int(kv["per_node"]), int(kv["batch"]),
                              int(kv["layers"])) == want
    assert kinds == {"solve", "candidates"}


@pytest.mark.parametrize("seed", range(10))
def test_unlimited_budget_closed_form(seed):
    rng = np.random.default_rng(seed)
    mods = [[(int(rng.integers(1, 50)), int(rng.integers(1, 5))) for _ in range(int(rng.integers(1, 4)))]
            for _ in range(int(rng.integers(2, 4)))]
    choice, g, f, dev = solve(mods, 10 ** 9)
    sums = sorted(set(sum(c) for c in itertools.product(*[[t for t, _ in m] for m in mods[:-1]])))
    best_bb = max(t for t, _ in mods[-1])
    assert g == min(max(sums), best_bb)
    if max(sums) >= best_bb:
        assert f == min(s for s in sums if s >= best_bb) - best_bb
    else:
        assert f == min(t for t, _ in mods[-1] if t >= max(sums)) - max(sums)


def test_budget_monotone():
    rng = np.random.default_rng(4)
    mods = [[(int(rng.integers(1, 80)), int(rng.integers(1, 9))) for _ in range(5)] for _ in range(3)]
    last = -1
    for R in range(0, 30):
        r = solve(mods, R)
        g = -1 if r is None else r[1]
        assert g >= last
        last = g


@pytest.mark.parametrize("backbone", [False, True])
def test_candidate_rules(backbone):
    devices, per_node, batch, layers = 24, 8, 48, 12
    got = candidates(backbone, devices, per_node, batch, layers)
    for dp, tp, pp in got:
        assert batch % dp == 0 and per_node % tp == 0 and layers % pp == 0 and dp * tp * pp <= devices
        assert backbone or pp == 1
    every = [(dp, tp, pp) for dp in range(1, 49) for tp in range(1, 9) for pp in range(1, 13)
             if batch % dp == 0 and per_node % tp == 0 and layers % pp == 0 and dp * tp * pp <= devices
             and (backbone or pp == 1)]
    assert got == sorted(every)
    assert divisors(12) == [1, 2, 3, 4, 6, 12]
