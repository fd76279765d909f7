"""Tier migration on the GPU against the oracle (Sec. 3.2 HBM/DRAM pool).

- Promotions to HBM and demotions to the host tier give the oracle's page
  lists, the oracle's free stacks afterwards (later writes get the same
  pages), and packs bit-identical to the definitional pack.
- A migration racing a pack queued on another stream: the queued pack reads
  the old pages (kept until it has run), a pack queued after the migration
  waits for its copies.
Bar: bit-exact pages and bytes.
"""

import numpy as np
import pytest

from gpu_common import say, to_dev, to_host
from oracle.pack import definitional_pack
from oracle.pool import OraclePool
from paper_2606_23087_amd.workloads import SampleSpec
from tagging import tagged_table, tagged_vis

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

H, P, VOCAB = 256, 16, 101


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def _spec(rng):
    t = int(rng.integers(1, 30))
    k = int(rng.integers(0, 3))
    pos = np.sort(rng.integers(0, t + 1, size=k)).astype(np.int32)
    ntok = rng.integers(0, 3 * P, size=k).astype(np.int32)
    return SampleSpec(rng.integers(0, VOCAB, size=t).astype(np.int32), pos, ntok)


def test_migration_matches_oracle(fp):
    say("case migration vs oracle")
    rng = np.random.default_rng(21)
    table = tagged_table(VOCAB, H, 21)
    t_dev = to_dev(table)
    hbm, host = 48, 48
    pool = fp.pool_create(hidden=H, page_tokens=P, hbm_pages=hbm, host_pages=host, vocab=VOCAB, alloc="scatter")
    orc = OraclePool(H, P, hbm, host, "scatter", VOCAB)
    s = torch.cuda.Stream()
    specs, vis, gids, oids = [], [], [], []
    keep = []

    def write():
        sp = _spec(rng)
        v = tagged_vis(len(specs), sp.n_vis, H, 21)
        wish = rng.integers(0, 2, size=-(-sp.n_vis // P)).astype(np.uint8)
        d = to_dev(v) if sp.n_vis else None
        torch.cuda.synchronize()
        gids.append(fp.pool_write_sample(pool, sp.text_ids, sp.img_pos, sp.img_ntok, d, wish, stream=s))
        oids.append(orc.write(sp.text_ids, sp.img_pos, sp.img_ntok, v, tier_wish=wish))
        specs.append(sp)
        vis.append(v)
        keep.append(d)

    def check():
        torch.cuda.synchronize()
        for g, o in zip(gids, oids):
            assert fp.pool_sample_pages(pool, g).tolist() == orc.sample_pages(o)
        n = sum(x.length for x in specs)
        out = torch.empty((n, H), dtype=torch.int16, device="cuda")
        fp.pack_microbatch(pool, gids, t_dev, VOCAB, out, n, stream=s)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(out), definitional_pack(specs, vis, table)[0])
        assert np.array_equal(to_host(out), orc.pack(oids, table)[0])

    try:
        for _ in range(8):
            write()
        check()
        for rnd in range(6):
            pick = sorted(set(int(i) for i in rng.integers(0, len(gids), size=3)))
            tier = rnd % 2
            say(f"  step {rnd}: samples {pick} -> tier {tier}")
            need = sum(1 for i in pick for g in orc.sample_pages(oids[i]) if orc.translate(g)[0] != tier)
            if need <= len(orc.stack[tier]):
                want = sum(orc.migrate(oids[i], tier) for i in pick)
                assert want == need
                assert fp.pool_migrate(pool, [gids[i] for i in pick], tier, stream=s) == need
            else:
                with pytest.raises(fp.FlowPoolError, match="ENOMEM"):
                    fp.pool_migrate(pool, [gids[i] for i in pick], tier, stream=s)
            torch.cuda.synchronize()
            fp.pool_reclaim(pool, True)
            check()
            write()
            check()
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)


def test_migration_racing_a_queued_pack(fp):
    say("case migration vs queued pack")
    rng = np.random.default_rng(5)
    table = tagged_table(VOCAB, H, 5)
    t_dev = to_dev(table)
    pool = fp.pool_create(hidden=H, page_tokens=P, hbm_pages=16, host_pages=16, vocab=VOCAB, alloc="scatter")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    try:
        sp = SampleSpec(rng.integers(0, VOCAB, size=20).astype(np.int32), np.array([4, 9], np.int32),
                        np.array([2 * P + 3, P], np.int32))
        v = tagged_vis(0, sp.n_vis, H, 5)
        d = to_dev(v)
        torch.cuda.synchronize()
        sid = fp.pool_write_sample(pool, sp.text_ids, sp.img_pos, sp.img_ntok, d,
                                   np.ones(4, np.uint8), stream=sa)
        torch.cuda.synchronize()
        want = definitional_pack([sp], [v], table)[0]
        a = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        with torch.cuda.stream(sb):
            for _ in range(1000):
                b.copy_(a)
        out1 = torch.empty((sp.length, H), dtype=torch.int16, device="cuda")
        fp.pack_microbatch(pool, [sid], t_dev, VOCAB, out1, sp.length, stream=sb)
        old = fp.pool_sample_pages(pool, sid).tolist()
        assert fp.pool_migrate(pool, [sid], fp.FP_TIER_HBM, stream=sa) == 4
        assert fp.pool_reclaim(pool) == 4, "the old pages wait for the queued pack"
        out2 = torch.empty((sp.length, H), dtype=torch.int16, device="cuda")
        fp.pack_microbatch(pool, [sid], t_dev, VOCAB, out2, sp.length, stream=sb)
        torch.cuda.synchronize()
        assert fp.pool_reclaim(pool) == 0
        new = fp.pool_sample_pages(pool, sid).tolist()
        assert set(new).isdisjoint(old)
        assert all(fp.pool_translate(pool, g)[0] == fp.FP_TIER_HBM for g in new)
        assert np.array_equal(to_host(out1), want)
        assert np.array_equal(to_host(out2), want)
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)


def test_migration_errors_leave_the_pool_unchanged(fp):
    say("case migration errors")
    rng = np.random.default_rng(9)
    pool = fp.pool_create(hidden=H, page_tokens=P, hbm_pages=6, host_pages=6, vocab=VOCAB, alloc="scatter")
    contig = fp.pool_create(hidden=H, page_tokens=P, hbm_pages=6, vocab=VOCAB, alloc="contig")
    try:
        sp = SampleSpec(rng.integers(0, VOCAB, size=5).astype(np.int32), np.array([2], np.int32),
                        np.array([4 * P], np.int32))
        v = to_dev(tagged_vis(0, sp.n_vis, H))
        torch.cuda.synchronize()
        a = fp.pool_write_sample(pool, sp.text_ids, sp.img_pos, sp.img_ntok, v, np.ones(4, np.uint8))
        b = fp.pool_write_sample(pool, sp.text_ids, sp.img_pos, sp.img_ntok, v, np.zeros(4, np.uint8))
        c = fp.pool_write_sample(contig, sp.text_ids, sp.img_pos, sp.img_ntok, v)
        torch.cuda.synchronize()
        before = (fp.pool_sample_pages(pool, a).tolist(), fp.pool_sample_pages(pool, b).tolist(), fp.pool_stats(pool))
        cases = [
            (lambda: fp.pool_migrate(contig, [c], fp.FP_TIER_HOST), "EINVAL"),     # contig pools do not migrate
            (lambda: fp.pool_migrate(pool, [a], 7), "EINVAL"),                     # no such tier
            (lambda: fp.pool_migrate(pool, [a, a], fp.FP_TIER_HBM), "EINVAL"),     # listed twice
            (lambda: fp.pool_migrate(pool, [a, 999], fp.FP_TIER_HBM), "ENOENT"),
            (lambda: fp.pool_migrate(pool, [a], fp.FP_TIER_HBM), "ENOMEM"),         # 4 pages, 2 free in HBM
        ]
        for call, code in cases:
            with pytest.raises(fp.FlowPoolError, match=code):
                call()
        assert (fp.pool_sample_pages(pool, a).tolist(), fp.pool_sample_pages(pool, b).tolist(),
                fp.pool_stats(pool)) == before
        assert fp.pool_migrate(pool, [b], fp.FP_TIER_HBM) == 0                   # already there
        with pytest.raises(fp.FlowPoolError, match="ENOENT"):
            fp.plan_pool_packing(pool, [a, 12345], 1000, 2, 2)
        with pytest.raises(fp.FlowPoolError, match="EINVAL"):
            fp.plan_pool_packing(pool, [a], 10, 2, 2)                            # longer than the capacity
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)
        fp.pool_destroy(contig)
