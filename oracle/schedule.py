"""Dynamic packing scheduler oracle (Alg. 1). TEST INFRASTRUCTURE ONLY.

Sec. 3.4 builds balanced microbatches in two phases (Alg. 1):

1. Best-fit packing. Sequences arrive one at a time. Each goes to the open
   microbatch whose residual capacity is the smallest one that still holds
   it; if there is none, a new microbatch of capacity L is opened for it. A
   microbatch whose residual capacity drops below the shortest sequence
   length is closed (no sequence can fit it any more). The paper finds the
   best fit with a segment tree over residual capacities [0, L]; here it is
   a plain scan over the open microbatches, which is the definition the tree
   computes.

2. Two-dimension load balancing. Each packed microbatch gets the cost of
   Eq. 3, Cost(B) = sum(l)/L + l_max^2/L^2; microbatches with similar costs
   are clustered into buckets; each bucket's microbatches, sorted by
   decreasing cost, are dealt to the N data-parallel ranks in zig-zag order
   (ranks 0..N-1, then N-1..0, and so on).

Readings where the paper leaves a detail open:
- the shortest length is taken over the sequences of the call;
- best-fit ties (equal residuals) go to the microbatch opened first;
- the close check applies to the microbatch that just took the sequence;
- costs are kept exactly as the integer L*sum(l) + l_max^2 = L^2 * Cost(B);
- buckets come from one-dimensional k-means (Lloyd's iteration) on those
  integers with exact rational centroids: K = min(n_buckets, microbatches)
  centroids start at the costs of sorted position floor((2k+1) m / 2K);
  each microbatch joins its nearest centroid (ties: the lower index); an
  empty cluster keeps its centroid; stop when no assignment changes or after
  100 rounds; bucket k is cluster k, in increasing centroid order;
- buckets are dealt from the costliest down; within a bucket, ties in cost
  go to the lower microbatch index; each bucket restarts the zig-zag at
  rank 0 going forward, and the deal stops at the end of the list;
- a microbatch's slot is its position in its rank's dispatch order.
"""

from __future__ import annotations

from fractions import Fraction
from typing import Dict, List, Sequence

KMEANS_ROUNDS = 100


def best_fit_pack(lengths: Sequence[int], capacity: int):
    """Phase 1. Returns (mb_of_seq[n], members[m]) with microbatches numbered
    in the order they are opened and members in arrival order."""
    if not lengths:
        return [], []
    l_min = min(int(x) for x in lengths)
    residual: List[int] = []
    is_open: List[bool] = []
    members: List[List[int]] = []
    mb_of_seq: List[int] = []
    for i, l in enumerate(int(x) for x in lengths):
        best = -1
        for j in range(len(residual)):
            if is_open[j] and residual[j] >= l:
                if best < 0 or residual[j] < residual[best]:
                    best = j
        if best < 0:
            best = len(residual)
            residual.append(capacity)
            is_open.append(True)
            members.append([])
        residual[best] -= l
        members[best].append(i)
        mb_of_seq.append(best)
        if residual[best] < l_min:
            is_open[best] = False
    return mb_of_seq, members


def cost_scaled(mb_lengths: Sequence[int], capacity: int) -> int:
    """Eq. 3 multiplied by L^2: L * sum(l) + l_max^2 (0 for an empty microbatch)."""
    if not mb_lengths:
        return 0
    return capacity * sum(int(x) for x in mb_lengths) + max(int(x) for x in mb_lengths) ** 2


def eq3(mb_lengths: Sequence[int], capacity: int) -> Fraction:
    """Eq. 3 as an exact fraction."""
    return Fraction(cost_scaled(mb_lengths, capacity), capacity * capacity)


def kmeans_buckets(costs: Sequence[int], n_buckets: int) -> List[int]:
    """Bucket of each cost: one-dimensional k-means with exact centroids."""
    m = len(costs)
    if m == 0:
        return []
    k_n = min(n_buckets, m)
    order = sorted(range(m), key=lambda j: (costs[j], j))
    centroid = [Fraction(costs[order[(2 * k + 1) * m // (2 * k_n)]]) for k in range(k_n)]
    assign = [-1] * m
    for _ in range(KMEANS_ROUNDS):
        new = []
        for x in costs:
            dist = [abs(x - c) for c in centroid]
            new.append(min(range(k_n), key=lambda k: (dist[k], k)))
        if new == assign:
            break
        assign = new
        for k in range(k_n):
            pts = [costs[j] for j in range(m) if assign[j] == k]
            if pts:
                centroid[k] = Fraction(sum(pts), len(pts))
    return assign


def zigzag(count: int, n_ranks: int) -> List[int]:
    """Ranks of the first ``count`` items of a list dealt in zig-zag order."""
    out: List[int] = []
    forward = True
    while len(out) < count:
        sweep = range(n_ranks) if forward else range(n_ranks - 1, -1, -1)
        for r in sweep:
            if len(out) == count:
                break
            out.append(r)
        forward = not forward
    return out


def dynamic_packing(lengths: Sequence[int], capacity: int, n_ranks: int, n_buckets: int) -> Dict:
    """Alg. 1 end to end. Per microbatch: tokens, max_len, cost_scaled,
    bucket, rank, slot; per sequence: its microbatch."""
    mb_of_seq, members = best_fit_pack(lengths, capacity)
    m = len(members)
    mb_len = [[int(lengths[i]) for i in mem] for mem in members]
    tokens = [sum(x) for x in mb_len]
    max_len = [max(x) for x in mb_len]
    costs = [cost_scaled(x, capacity) for x in mb_len]
    bucket = kmeans_buckets(costs, n_buckets)
    rank = [-1] * m
    slot = [-1] * m
    next_slot = [0] * n_ranks
    n_b = max(bucket) + 1 if bucket else 0
    for b in range(n_b - 1, -1, -1):
        lst = sorted((j for j in range(m) if bucket[j] == b), key=lambda j: (-costs[j], j))
        for j, r in zip(lst, zigzag(len(lst), n_ranks)):
            rank[j] = r
            slot[j] = next_slot[r]
            next_slot[r] += 1
    return dict(mb_of_seq=mb_of_seq, n_mb=m, mb_tokens=tokens, mb_max_len=max_len,
                mb_cost_scaled=costs, mb_bucket=bucket, mb_rank=rank, mb_slot=slot)


def optimal_bins(lengths: Sequence[int], capacity: int) -> int:
    """Fewest microbatches of capacity L that hold all sequences (brute force,
    tiny inputs only): each sequence in turn tries every open bin and a new one."""
    ls = sorted((int(x) for x in lengths), reverse=True)
    best = [len(ls)]

    def go(i: int, bins: List[int]) -> None:
        if len(bins) >= best[0]:
            return
        if i == len(ls):
            best[0] = len(bins)
            return
        seen = set()
        for b in range(len(bins)):
            if bins[b] + ls[i] <= capacity and bins[b] not in seen:
                seen.add(bins[b])
                bins[b] += ls[i]
                go(i + 1, bins)
                bins[b] -= ls[i]
        bins.append(ls[i])
        go(i + 1, bins)
        bins.pop()

    go(0, [])
    return best[0]
