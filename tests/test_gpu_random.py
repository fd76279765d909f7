"""Randomised GPU parity of pack_microbatch against the oracle's definitional
pack: random hidden sizes and page sizes, contiguous and scattered pools
after random frees, samples with empty, adjacent and trailing images, random
sample subsets in random order, and chunk geometries sized for 1, 2, 5 or
all compute units (so full chunks and both shrinking tail sizes occur).

Each case prints its seed and shape before touching the GPU.
Bar: bit-exact (raw 16-bit copies), cu_seqlens and position ids exact,
rows past the microbatch untouched.
"""

import numpy as np
import pytest

from gpu_common import say, to_dev, to_host
from oracle.pack import definitional_pack
from paper_2606_23087_amd.workloads import SampleSpec
from tagging import tagged_table, tagged_vis

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def _spec(rng, vocab):
    while True:
        t = int(rng.integers(0, 61))
        k = int(rng.integers(0, 7))
        pos = np.sort(rng.integers(0, t + 1, size=k)).astype(np.int32)
        if k and rng.random() < 0.3:
            pos[:] = pos[0]                           # all images adjacent
        ntok = rng.integers(0, 51, size=k).astype(np.int32)
        if t + int(ntok.sum()) > 0:
            return SampleSpec(rng.integers(0, vocab, size=t).astype(np.int32), pos, ntok)


@pytest.mark.parametrize("seed", range(1000))
def test_random_packs(fp, seed):
    rng = np.random.default_rng(9000 + seed)
    hidden = int(rng.choice([8, 16, 24, 64, 104, 200, 512, 1000, 2048, 3584, 5120, 8192]))
    page_tokens = int(rng.integers(1, 70))
    alloc = "scatter" if seed % 2 else "contig"
    pack_cus = int(rng.choice([0, 1, 2, 5]))
    vocab = 97
    n = int(rng.integers(1, 41))
    specs = [_spec(rng, vocab) for _ in range(n)]
    say(f"case random seed={seed} H={hidden} P={page_tokens} alloc={alloc} pack_cus={pack_cus} samples={n}")
    pages = sum(-(-s.n_vis // page_tokens) for s in specs)
    pool = fp.pool_create(hidden=hidden, page_tokens=page_tokens, hbm_pages=2 * pages + 8, vocab=vocab,
                          alloc=alloc, pack_cus=pack_cus)
    try:
        table = tagged_table(vocab, hidden, seed)
        t_dev = to_dev(table)
        vis = [tagged_vis(i, s.n_vis, hidden, seed) for i, s in enumerate(specs)]
        ids = [None] * n
        # Write everything, free a random third, write those again: scattered
        # pools then hand out pages in a different order.
        for i, s in enumerate(specs):
            ids[i] = fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok,
                                          to_dev(vis[i]) if s.n_vis else None)
        redo = [i for i in range(n) if rng.random() < 0.33]
        for i in redo:
            fp.pool_free_sample(pool, ids[i])
        for i in redo[::-1]:
            s = specs[i]
            ids[i] = fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok,
                                          to_dev(vis[i]) if s.n_vis else None)
        torch.cuda.synchronize()
        total = sum(s.length for s in specs)
        out = torch.full((total + 40, hidden), 0x5A5A, dtype=torch.int16, device="cuda")
        cu = torch.full((n + 2,), -1, dtype=torch.int32, device="cuda")
        pos = torch.full((total + 40,), -1, dtype=torch.int32, device="cuda")
        for g in range(3):
            pick = rng.permutation(n)[:int(rng.integers(1, n + 1))].tolist()
            m, mx = fp.pack_microbatch(pool, [ids[i] for i in pick], t_dev, vocab, out, out.shape[0], cu, pos)
            torch.cuda.synchronize()
            want = definitional_pack([specs[i] for i in pick], [vis[i] for i in pick], table)
            assert m == len(want[0]) and mx == want[3], f"group {g}"
            assert np.array_equal(to_host(out[:m]), want[0]), f"group {g}"
            assert cu[:len(pick) + 1].cpu().numpy().tolist() == want[1].tolist(), f"group {g}"
            assert pos[:m].cpu().numpy().tolist() == want[2].tolist(), f"group {g}"
            assert bool((out[m:] == 0x5A5A).all()) and bool((pos[m:] == -1).all()), f"group {g}"
            out.fill_(0x5A5A)
            pos.fill_(-1)
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)
