"""Seeded random interleavings of every pool operation across three streams
(Sec. 3.1 decoupling, Sec. 3.2 tiers): writes with random tier wishes,
frees, packs of random subsets, migrations of random subsets to either tier,
and non-waiting reclaims, each on a random stream, with no host
synchronisation between them. The pool must order them itself.

Every pack is checked after the run against the definitional pack of the
samples it named, with the bytes those samples were written with (migration
moves pages, never bytes). At the end every sample is freed, and after a
waiting reclaim all pages of both tiers are free again.
Bar: bit-exact.
"""

import numpy as np
import pytest

from gpu_common import say, to_dev, to_host
from oracle.pack import definitional_pack
from paper_2606_23087_amd.workloads import SampleSpec
from tagging import tagged_table, tagged_vis

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

H, P, VOCAB = 128, 8, 89
HBM, HOST = 160, 160


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def _spec(rng):
    t = int(rng.integers(1, 25))
    k = int(rng.integers(0, 4))
    pos = np.sort(rng.integers(0, t + 1, size=k)).astype(np.int32)
    ntok = rng.integers(0, 4 * P, size=k).astype(np.int32)
    return SampleSpec(rng.integers(0, VOCAB, size=t).astype(np.int32), pos, ntok)


@pytest.mark.parametrize("seed", range(224))
def test_random_interleavings(fp, seed):
    say(f"case chaos seed={seed}")
    rng = np.random.default_rng(7700 + seed)
    table = tagged_table(VOCAB, H, seed)
    t_dev = to_dev(table)
    pool = fp.pool_create(hidden=H, page_tokens=P, hbm_pages=HBM, host_pages=HOST, vocab=VOCAB, alloc="scatter")
    streams = [torch.cuda.Stream() for _ in range(3)]
    live = {}        # sample id -> (spec, host rows)
    keep = []        # device buffers kept alive until the end
    packs = []       # (items, out, cu, pos)
    counts = dict(write=0, free=0, pack=0, migrate=0, reclaim=0, full=0)
    n_written = 0
    try:
        for step in range(250):
            st = streams[int(rng.integers(0, 3))]
            op = rng.choice(["write", "write", "free", "pack", "pack", "migrate", "reclaim"])
            if op == "write" or not live:
                sp = _spec(rng)
                v = tagged_vis(n_written, sp.n_vis, H, seed)
                n_written += 1
                wish = rng.integers(0, 2, size=-(-sp.n_vis // P)).astype(np.uint8) if sp.n_vis else None
                with torch.cuda.stream(st):                    # the upload is ordered before the write
                    d = to_dev(v) if sp.n_vis else None
                keep.append(d)
                try:
                    sid = fp.pool_write_sample(pool, sp.text_ids, sp.img_pos, sp.img_ntok, d, wish, stream=st)
                except fp.FlowPoolError as e:
                    assert e.code == "ENOMEM", e
                    counts["full"] += 1
                    continue
                live[sid] = (sp, v)
                counts["write"] += 1
            elif op == "free":
                sid = list(live)[int(rng.integers(0, len(live)))]
                fp.pool_free_sample(pool, sid)
                live.pop(sid)
                counts["free"] += 1
            elif op == "pack":
                ids = list(live)
                pick = [ids[int(j)] for j in rng.permutation(len(ids))[:int(rng.integers(1, min(len(ids), 12) + 1))]]
                items = [live[s] for s in pick]
                n = sum(sp.length for sp, _ in items)
                with torch.cuda.stream(st):
                    out = torch.empty((n, H), dtype=torch.int16, device="cuda")
                    cu = torch.empty((len(pick) + 1,), dtype=torch.int32, device="cuda")
                    pos = torch.empty((n,), dtype=torch.int32, device="cuda")
                m, _ = fp.pack_microbatch(pool, pick, t_dev, VOCAB, out, n, cu, pos, stream=st)
                assert m == n
                packs.append((items, out, cu, pos))
                counts["pack"] += 1
            elif op == "migrate":
                ids = list(live)
                pick = [ids[int(j)] for j in rng.permutation(len(ids))[:int(rng.integers(1, min(len(ids), 6) + 1))]]
                tier = int(rng.integers(0, 2))
                try:
                    fp.pool_migrate(pool, pick, tier, stream=st)
                except fp.FlowPoolError as e:
                    assert e.code == "ENOMEM", e
                    counts["full"] += 1
                    continue
                counts["migrate"] += 1
            else:
                fp.pool_reclaim(pool, False)
                counts["reclaim"] += 1
        torch.cuda.synchronize()
        say(f"  {counts}")
        for k, (items, out, cu, pos) in enumerate(packs):
            want = definitional_pack([sp for sp, _ in items], [v for _, v in items], table)
            assert np.array_equal(to_host(out), want[0]), f"pack {k}"
            assert cu.cpu().numpy().tolist() == want[1].tolist(), f"pack {k}"
            assert pos.cpu().numpy().tolist() == want[2].tolist(), f"pack {k}"
        for sid in list(live):
            fp.pool_free_sample(pool, sid)
        torch.cuda.synchronize()
        assert fp.pool_reclaim(pool, True) == 0
        stats = fp.pool_stats(pool)
        assert stats["free_hbm_pages"] == HBM and stats["free_host_pages"] == HOST and stats["n_samples"] == 0
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)
