"""The library's dynamic packing scheduler (Alg. 1) against the oracle, CPU
only: the C-ABI call is host code, so these run without a GPU.

Bar: identical integers for every output (microbatch of each sequence,
tokens, longest length, scaled Eq. 3 cost, bucket, rank, slot). Inputs:
seeded lengths shaped like the workloads' samples (lognormal text plus image
blocks), clipped to the capacity, at capacities from 64 to 32768, and edge
cases (one sequence, all equal, all longer than half the capacity, more
buckets or ranks than microbatches).
"""

import numpy as np
import pytest

from oracle.schedule import dynamic_packing

fp = pytest.importorskip("paper_2606_23087_amd.flowpool")

KEYS = ("mb_tokens", "mb_max_len", "mb_cost_scaled", "mb_bucket", "mb_rank", "mb_slot")


def _compare(lengths, L, N, K):
    got = fp.plan_dynamic_packing(lengths, L, N, K)
    want = dynamic_packing([int(x) for x in lengths], L, N, K)
    assert got["n_mb"] == want["n_mb"]
    assert got["mb_of_seq"].tolist() == want["mb_of_seq"]
    for k in KEYS:
        assert got[k].tolist() == want[k], k
    return got


def _lengths(rng, n, L):
    text = np.clip(np.round(rng.lognormal(np.log(400), 0.8, size=n)), 16, 4096)
    imgs = rng.integers(0, 5, size=n) * rng.integers(64, 1281, size=n)
    return np.clip(text + imgs, 1, L).astype(np.int32)


@pytest.mark.parametrize("L", [64, 512, 2048, 8192, 32768])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_matches_oracle(L, seed):
    rng = np.random.default_rng([seed, L])
    n = int(rng.integers(50, 400))
    N, K = int(rng.integers(1, 9)), int(rng.integers(1, 6))
    got = _compare(_lengths(rng, n, L), L, N, K)
    assert got["mb_tokens"].max() <= L


@pytest.mark.parametrize("case", ["one", "equal", "long", "many_buckets", "many_ranks", "empty"])
def test_edge_cases(case):
    L = 100
    lengths = {"one": [37], "equal": [25] * 17, "long": [51, 99, 60, 100, 77], "many_buckets": [10, 90, 45, 55, 3],
               "many_ranks": [30, 30, 30, 30, 30, 30, 30], "empty": []}[case]
    N = 16 if case == "many_ranks" else 2
    K = 50 if case == "many_buckets" else 3
    _compare(np.array(lengths, np.int32), L, N, K)


def test_errors():
    with pytest.raises(fp.FlowPoolError, match="EINVAL"):
        fp.plan_dynamic_packing([5, 0], 10, 1, 1)
    with pytest.raises(fp.FlowPoolError, match="EINVAL"):
        fp.plan_dynamic_packing([5, 11], 10, 1, 1)
    with pytest.raises(fp.FlowPoolError, match="EINVAL"):
        fp.plan_dynamic_packing([5], 10, 0, 1)
    with pytest.raises(fp.FlowPoolError, match="EINVAL"):
        fp.plan_dynamic_packing([5], 10, 1, 0)
    with pytest.raises(fp.FlowPoolError, match="EINVAL"):
        fp.plan_dynamic_packing([5], (1 << 20) + 1, 1, 1)


def test_kmeans_tie_goes_to_the_lower_bucket():
    """An exact k-means tie (reading R21: ties to the lower bucket). At L 33,
    lengths 19, 26 and 32 each fill a microbatch of their own, with scaled
    costs 988, 1534 and 2080; two buckets start at 988 and 2080, and 1534 lies
    exactly between them, so it joins bucket 0, whose centroid then moves to
    1261."""
    got = _compare(np.array([19, 26, 32], np.int32), 33, 2, 2)
    assert got["mb_cost_scaled"].tolist() == [988, 1534, 2080]
    assert got["mb_bucket"].tolist() == [0, 0, 1]
