"""Pins for the allocator oracle (Sec. 3.3, Eq. 1-2), CPU only.

- hand-worked flow-matching solutions and candidate lists
  (tests/golden/allocator_flow_example.txt);
- closed form: with an unlimited budget, G = min(best encoder sum, best
  backbone throughput), and F follows from the closest encoder sum;
- monotonicity: a larger budget never lowers G;
- the candidate rules, checked by simulating what each prunes (an even
  batch split, TP groups inside one node, equal pipeline stages, the device
  budget) over every configuration in range, plus hand-worked lists that tell
  the rules apart (a TP degree that fits a node without dividing it, a PP
  degree that fits the budget without dividing the layers, a budget below the
  product of the largest degrees).
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


def _batch_splits_evenly(batch, dp):
    """Deal the global batch's samples to dp replicas round-robin; equal shares?"""
    share = [0] * dp
    for i in range(batch):
        share[i % dp] += 1
    return len(set(share)) == 1


def _tp_groups_stay_in_nodes(tp, per_node, span):
    """TP groups of tp consecutive devices, laid from every multiple of tp
    below ``span``: does any group hold devices of two nodes?"""
    for start in range(0, span, tp):
        if len({d // per_node for d in range(start, start + tp)}) > 1:
            return False
    return True


def _stages_equal(layers, pp):
    """Cut the layers into pp contiguous stages, as evenly as possible; equal?"""
    cuts = [round(k * layers / pp) for k in range(pp + 1)]
    return len({b - a for a, b in zip(cuts, cuts[1:])}) == 1


@pytest.mark.parametrize("backbone", [False, True])
@pytest.mark.parametrize("cluster", [(24, 8, 48, 12), (12, 6, 30, 10), (16, 4, 16, 0), (5, 8, 12, 7)])
def test_candidate_rules_by_simulation(backbone, cluster):
    """Each kept configuration splits the batch evenly, keeps every TP group
    inside one node, cuts the layers into equal stages (if a layer count is
    given) and fits the devices; every configuration in range that is left
    out breaks one of these, checked by simulating the split, the placement
    and the stage cut rather than by the divisibility formulas."""
    devices, per_node, batch, layers = cluster
    got = candidates(backbone, devices, per_node, batch, layers)
    assert got == sorted(set(got))
    span = 2 * per_node * per_node     # every TP alignment against the node size repeats within this span
    ok = set()
    for dp in range(1, batch + 1):
        for tp in range(1, per_node + 1):
            for pp in range(1, (devices if backbone else 1) + 1):
                if (dp * tp * pp <= devices and _batch_splits_evenly(batch, dp)
                        and _tp_groups_stay_in_nodes(tp, per_node, span)
                        and (not backbone or not layers or (pp <= layers and _stages_equal(layers, pp)))):
                    ok.add((dp, tp, pp))
    assert set(got) == ok
    # a TP degree above the node size always straddles nodes
    assert not _tp_groups_stay_in_nodes(per_node + 1, per_node, span)
    assert divisors(12) == [1, 2, 3, 4, 6, 12]
