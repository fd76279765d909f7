"""Heterogeneous parallel allocator oracle (Sec. 3.3, Eq. 1-2). TEST INFRASTRUCTURE ONLY.

The allocator splits a device budget R between the encoder modules and the
backbone and picks one parallelism configuration per module. With tau_i(c)
the throughput and r_i(c) the device count of configuration c of module i:

    T_enc = sum over encoders e of tau_e(c_e),   T_bb = tau_b(c_b)       (Eq. 1)
    lexmax (G, -F)  with  G = min(T_enc, T_bb),  F = |T_enc - T_bb|,
    one configuration per module, sum of r_i(c_i) <= R                    (Eq. 2)

First the candidate configurations are pruned (Sec. 3.3, first step):
encoders use data and tensor parallelism (DP x TP devices), the backbone also
pipeline parallelism (DP x TP x PP devices). The paper prunes three kinds of
configuration; each is read here as one rule:
- the global batch is not divisible by DP: kept iff DP divides it;
- TP and PP degrees that fail to split a module's device budget: a module's
  budget is the device count of its configuration, the product of its
  degrees by construction, so the rule bounds that count by the
  cluster's devices (DP x TP x PP <= devices); where the caller gives the
  backbone's layer count (layers > 0), PP must also divide it, so that every
  pipeline stage holds the same number of layers (a low-efficiency pruning
  the paper does not spell out; layers = 0 leaves it out);
- cross-node tensor parallelism: TP must divide the devices of one node, the
  condition under which TP groups laid over consecutive devices from any
  multiple of TP never straddle a node boundary.

Here the problem is solved by enumerating every combination (the paper
solves the same problem as a MILP). Readings where the paper leaves a
detail open:
- throughputs and device counts are integers, so G and F are exact;
- among combinations with the best (G, F), fewer devices win, then the
  lexicographically smallest choice vector (encoders in order, then the
  backbone);
- candidates are listed in increasing (DP, TP, PP) order.
"""

from __future__ import annotations

import itertools
from typing import List, Sequence, Tuple


def divisors(n: int) -> List[int]:
    return [d for d in range(1, n + 1) if n % d == 0]


def candidates(backbone: bool, devices: int, per_node: int, global_batch: int, layers: int):
    """Pruned (DP, TP, PP) configurations of one module, in increasing order.
    layers = 0: no layer rule for the backbone's PP."""
    out = []
    if not backbone:
        pps = [1]
    elif layers:
        pps = divisors(layers)
    else:
        pps = list(range(1, devices + 1))
    for dp in divisors(global_batch):
        for tp in divisors(per_node):
            for pp in pps:
                if dp * tp * pp <= devices:
                    out.append((dp, tp, pp))
    return sorted(out)


def solve(modules: Sequence[Sequence[Tuple[int, int]]], budget: int):
    """modules: encoders then the backbone, each a list of (tau, r).
    Returns (choice, G, F, devices) or None when nothing fits the budget."""
    enc, bb = modules[:-1], modules[-1]
    best = None
    for choice in itertools.product(*[range(len(m)) for m in modules]):
        cost = sum(modules[i][c][1] for i, c in enumerate(choice))
        if cost > budget:
            continue
        t_enc = sum(enc[i][c][0] for i, c in enumerate(choice[:-1]))
        t_bb = bb[choice[-1]][0]
        g, f = min(t_enc, t_bb), abs(t_enc - t_bb)
        key = (-g, f, cost, choice)
        if best is None or key < best:
            best = key
    if best is None:
        return None
    return list(best[3]), -best[0], best[1], best[2]
