"""Planner oracle: costs, greedy balanced partition, brute force. TEST INFRASTRUCTURE ONLY.

Sec. 3.4 models a packed microbatch's execution time as linear in its valid
tokens (MLP layers) plus quadratic in its longest sequence (attention), and
normalises both by the microbatch capacity L (Eq. 3):

    Cost(B) = (1/L) * sum_{s in B} l(s) + (1/L^2) * l_max(B)^2

The workloads state the cost per sample as l + l^2/K. Its exact integer form
K*l + l^2 (the cost scaled by K) is what the partition adds up; a
microbatch's cost is the sum over its samples.

The greedy balanced partition (longest processing time first, with a
capacity): samples in order of decreasing cost (ties: lower input index
first) each go to the microbatch of least accumulated cost among those whose
token count still has room for them (ties: lower microbatch index); a sample
that fits nowhere is deferred (-1) and stays in the pool for a later plan.
Since K*l + l^2 is strictly increasing in l, decreasing cost is decreasing
length.

The zig-zag policy (a reading: Alg. 1 deals its sorted microbatches to the
data-parallel ranks in a snake order; applied here to samples and
microbatches): samples in the same decreasing-cost order; the sample at
position p of that order goes to microbatch snake(p), where snake runs
0, 1, ..., M-1, M-1, ..., 1, 0, 0, 1, ... (period 2M); if that microbatch has
no room, to the first microbatch with room among snake(p+1), snake(p+2), ...
(2M positions cover every microbatch); deferred (-1) if none has room. The
position advances with every sample, placed or deferred.

Brute force enumerates every assignment for tiny inputs to give the optimal
max-cost partition.

The tie rules of both policies are readings (the paper states none). They
are pinned by hand-worked partitions written from them (with equal lengths,
exact fits and deferrals) and by a check of the output alone: replayed in
the samples' turn order, each placed sample went where the rule sends it
(least cost with room, lowest index among equals; or the first microbatch
with room along the snake) and each deferred one fit nowhere. The
assignment's quality is pinned against brute force and Graham's bound for
LPT.
"""

from __future__ import annotations

import itertools
from typing import List, Sequence


def cost_scaled(length: int, k: int) -> int:
    """Per-sample cost l + l^2/K, scaled by K to an exact integer."""
    return k * length + length * length


def eq3_cost(lengths: Sequence[int], capacity: int) -> float:
    """Eq. 3 for one microbatch with sequence lengths ``lengths`` and capacity L."""
    if not lengths:
        return 0.0
    return sum(lengths) / capacity + (max(lengths) ** 2) / (capacity ** 2)


def greedy_partition(lengths: Sequence[int], k: int, capacity: int, n_mb: int):
    """Returns (assign[n] in [0, n_mb) or -1, mb_tokens[n_mb], mb_cost_scaled[n_mb])."""
    n = len(lengths)
    costs = [cost_scaled(int(l), k) for l in lengths]
    order = sorted(range(n), key=lambda i: (-costs[i], i))
    tokens = [0] * n_mb
    mb_cost = [0] * n_mb
    assign = [-1] * n
    for i in order:
        best = -1
        for j in range(n_mb):
            if tokens[j] + int(lengths[i]) <= capacity:
                if best < 0 or mb_cost[j] < mb_cost[best]:
                    best = j
        if best >= 0:
            assign[i] = best
            tokens[best] += int(lengths[i])
            mb_cost[best] += costs[i]
    return assign, tokens, mb_cost


def snake(p: int, n_mb: int) -> int:
    """Microbatch of snake position p: 0, 1, ..., M-1, M-1, ..., 0, 0, 1, ..."""
    q = p % (2 * n_mb)
    return q if q < n_mb else 2 * n_mb - 1 - q


def zigzag_partition(lengths: Sequence[int], k: int, capacity: int, n_mb: int):
    """The zig-zag policy. Returns (assign, mb_tokens, mb_cost_scaled) like greedy_partition."""
    n = len(lengths)
    costs = [cost_scaled(int(l), k) for l in lengths]
    order = sorted(range(n), key=lambda i: (-costs[i], i))
    tokens = [0] * n_mb
    mb_cost = [0] * n_mb
    assign = [-1] * n
    for p, i in enumerate(order):
        for q in range(2 * n_mb):
            j = snake(p + q, n_mb)
            if tokens[j] + int(lengths[i]) <= capacity:
                assign[i] = j
                tokens[j] += int(lengths[i])
                mb_cost[j] += costs[i]
                break
    return assign, tokens, mb_cost


def members(assign: Sequence[int], n_mb: int) -> List[List[int]]:
    """Sample indices of each microbatch, in input order."""
    out: List[List[int]] = [[] for _ in range(n_mb)]
    for i, j in enumerate(assign):
        if j >= 0:
            out[j].append(i)
    return out


def imbalance(mb_cost: Sequence[int]) -> float:
    """max / mean of the microbatch costs (all microbatches, empty ones included)."""
    mean = sum(mb_cost) / len(mb_cost)
    return (max(mb_cost) / mean) if mean > 0 else 1.0


def brute_force(lengths: Sequence[int], k: int, capacity: int, n_mb: int):
    """Exhaustive search over all (n_mb + 1)^n assignments (value n_mb = deferred).

    Returns (opt_max_cost, lex_best) where opt_max_cost is the least possible
    maximum microbatch cost over assignments that defer nothing and respect
    the capacity (None if there is none), and lex_best = (packed tokens,
    -max cost) maximised lexicographically over all feasible assignments.
    """
    n = len(lengths)
    costs = [cost_scaled(int(l), k) for l in lengths]
    opt = None
    lex = None
    for combo in itertools.product(range(n_mb + 1), repeat=n):
        tok = [0] * n_mb
        cst = [0] * n_mb
        ok = True
        for i, j in enumerate(combo):
            if j < n_mb:
                tok[j] += int(lengths[i])
                cst[j] += costs[i]
                if tok[j] > capacity:
                    ok = False
                    break
        if not ok:
            continue
        mx = max(cst)
        packed = sum(tok)
        if all(j < n_mb for j in combo):
            opt = mx if opt is None else min(opt, mx)
        key = (packed, -mx)
        lex = key if lex is None else max(lex, key)
    return opt, lex
