"""Pins for the dynamic packing scheduler oracle (Alg. 1, Sec. 3.4), CPU only.

- hand-worked best-fit packings (including a tie and a case where first fit
  differs), Eq. 3 values, k-means buckets, zig-zag sequences and one full
  schedule (tests/golden/schedule_worked_example.txt);
- textbook bound: Best Fit never uses more than floor(1.7 * OPT) bins
  (Dosa and Sgall, 2014), with OPT by brute force on tiny inputs;
- closed forms: sequences longer than L/2 each get their own microbatch;
  k equal lengths per microbatch for equal lengths;
- k-means: one bucket for K = 1, well-separated groups split exactly, and
  at the fixed point every cost is nearest to its own centroid;
- zig-zag: every complete forward-and-back sweep of an arithmetic sequence
  gives every rank the same sum; each rank gets floor or ceil of count/N.
"""

from fractions import Fraction

import numpy as np
import pytest

from conftest import read_golden
from oracle.schedule import (best_fit_pack, cost_scaled, dynamic_packing, eq3, kmeans_buckets,
                             optimal_bins, zigzag)


def _fields(words):
    out, key = {}, None
    for w in words:
        if w.lstrip("-").isdigit():
            out[key].append(int(w))
        else:
            key = w
            out[key] = []
    return out


def test_worked_examples():
    seen = set()
    for ln in read_golden("schedule_worked_example.txt"):
        head, _, tail = ln.partition("->")
        kind = head.split()[0]
        seen.add(kind)
        if kind == "eq3":
            f = ln.split("=")[0].split()
            L, lens = int(f[1]), [int(x) for x in f[2:]]
            num, den = ln.split("=")[1].split("/")
            assert cost_scaled(lens, L) == int(num) and L * L == int(den)
            assert eq3(lens, L) == Fraction(int(num), int(den))
            continue
        a, b = _fields(head.split()[1:]), _fields(tail.split())
        if kind == "bestfit":
            L, lens = a["L"][0], a["lengths"]
            mb, members = best_fit_pack(lens, L)
            assert mb == b["mb"]
            assert [sum(lens[i] for i in m) for m in members] == b["tokens"]
            assert [max(lens[i] for i in m) for m in members] == b["max"]
            assert [cost_scaled([lens[i] for i in m], L) for m in members] == b["cost"]
        elif kind == "kmeans":
            assert kmeans_buckets(a["costs"], a["K"][0]) == b["bucket"]
        elif kind == "zigzag":
            assert zigzag(a["count"][0], a["N"][0]) == b["ranks"]
        elif kind == "full":
            r = dynamic_packing(a["lengths"], a["L"][0], a["N"][0], a["K"][0])
            assert r["mb_bucket"] == b["bucket"] and r["mb_rank"] == b["rank"] and r["mb_slot"] == b["slot"]
    assert seen == {"bestfit", "eq3", "kmeans", "zigzag", "full"}


@pytest.mark.parametrize("seed", range(40))
def test_best_fit_within_textbook_bound(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(8, 40))
    n = int(rng.integers(1, 9))
    lens = [int(x) for x in rng.integers(1, L + 1, size=n)]
    mb, members = best_fit_pack(lens, L)
    opt = optimal_bins(lens, L)
    assert opt <= len(members) <= int(1.7 * opt)
    assert sorted(i for m in members for i in m) == list(range(n))
    assert all(sum(lens[i] for i in m) <= L for m in members)
    assert all(mb[i] == j for j, m in enumerate(members) for i in m)


def test_optimal_bins_small_cases():
    assert optimal_bins([5, 5, 5, 5], 10) == 2
    assert optimal_bins([6, 6, 4, 4], 10) == 2
    assert optimal_bins([7, 6, 5], 10) == 3
    assert optimal_bins([3, 3, 3, 3, 3, 3], 9) == 2


def test_long_sequences_each_alone():
    L = 100
    lens = [51, 99, 60, 100, 77]
    mb, members = best_fit_pack(lens, L)
    assert mb == list(range(len(lens)))


@pytest.mark.parametrize("l,L,n", [(3, 10, 10), (7, 64, 40), (1, 5, 12), (8, 8, 3)])
def test_equal_lengths_closed_form(l, L, n):
    mb, members = best_fit_pack([l] * n, L)
    per = L // l
    assert len(members) == -(-n // per)
    assert all(len(m) == per for m in members[:-1])


def test_kmeans_properties():
    assert kmeans_buckets([7, 1, 4], 1) == [0, 0, 0]
    low = list(range(100, 111))
    high = list(range(1000, 1011))
    costs = high[:5] + low + high[5:]
    assert kmeans_buckets(costs, 2) == [1] * 5 + [0] * len(low) + [1] * 6
    rng = np.random.default_rng(3)
    for _ in range(30):
        costs = [int(x) for x in rng.integers(0, 10_000, size=int(rng.integers(1, 40)))]
        K = int(rng.integers(1, 6))
        b = kmeans_buckets(costs, K)
        cents = {}
        for k in set(b):
            pts = [c for c, bb in zip(costs, b) if bb == k]
            cents[k] = Fraction(sum(pts), len(pts))
        # buckets are contiguous in cost order and numbered by increasing centroid
        order = sorted(range(len(costs)), key=lambda j: (costs[j], j))
        assert [b[j] for j in order] == sorted(b[j] for j in order)
        # fixed point of Lloyd's iteration: nothing is closer to another centroid
        for c, k in zip(costs, b):
            assert all(abs(c - cents[k]) <= abs(c - v) for v in cents.values())


@pytest.mark.parametrize("N", [1, 2, 3, 8])
def test_zigzag_balances_complete_sweeps(N):
    count = 2 * N * 3
    costs = list(range(count, 0, -1))
    ranks = zigzag(count, N)
    sums = [sum(c for c, r in zip(costs, ranks) if r == k) for k in range(N)]
    assert len(set(sums)) == 1
    for c in range(0, 3 * N + 2):
        got = np.bincount(zigzag(c, N), minlength=N)
        assert got.max() - got.min() <= 1 and got.sum() == c


def test_dynamic_packing_invariants():
    rng = np.random.default_rng(11)
    for _ in range(20):
        L = int(rng.choice([64, 512, 2048]))
        lens = [int(x) for x in np.clip(rng.lognormal(np.log(L / 6), 0.9, size=200).round(), 1, L)]
        N, K = int(rng.integers(1, 9)), int(rng.integers(1, 5))
        r = dynamic_packing(lens, L, N, K)
        m = r["n_mb"]
        assert sum(r["mb_tokens"]) == sum(lens) and max(r["mb_tokens"]) <= L
        assert all(0 <= x < N for x in r["mb_rank"])
        for k in range(N):
            slots = sorted(s for s, x in zip(r["mb_slot"], r["mb_rank"]) if x == k)
            assert slots == list(range(len(slots)))
        # within a rank, slots run through buckets from the costliest down
        for k in range(N):
            seq = sorted((s, b) for s, b, x in zip(r["mb_slot"], r["mb_bucket"], r["mb_rank"]) if x == k)
            assert [b for _, b in seq] == sorted((b for _, b in seq), reverse=True)
        assert m == len(r["mb_cost_scaled"]) == len(r["mb_bucket"])
