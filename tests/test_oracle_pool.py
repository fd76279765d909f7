"""Pins for the pool oracle's addressing and allocation (CPU only).

- hand-worked allocation and GVA sequences (tests/golden/allocator_worked_example.txt)
  from the segment arithmetic of Sec. 3.2;
- allocator invariants: pages conserved, no page in two samples, freed pages
  reused, contiguous runs under "contig", all-or-nothing failure;
- every page GVA lies in its tier's region and in this rank's segment, and
  translation finds the frame that holds the row (Sec. 3.2);
- a tier-masked pack split into the HBM part and the DRAM part equals one
  full pack.
"""

import numpy as np
import pytest

from oracle.pool import MASK_HBM, MASK_HOST, OraclePool, PoolError
from paper_2606_23087_amd.workloads import CONFIGS, SampleSpec, churn_ops, gen_samples, scaled
from tagging import tagged_table, tagged_vis
from conftest import read_golden


def _golden_blocks():
    blocks, cur = [], None
    for ln in read_golden("allocator_worked_example.txt"):
        f = ln.split()
        if f[0] == "pool":
            kv = dict(zip(f[2::2], f[3::2]))
            cur = {"alloc": f[1], "kv": kv, "ops": []}
        elif f[0] == "end":
            blocks.append(cur)
        else:
            cur["ops"].append(f)
    return blocks


@pytest.mark.parametrize("block", range(5))
def test_allocator_worked_example(block):
    b = _golden_blocks()[block]
    kv = b["kv"]
    pool = OraclePool(hidden=int(kv["hidden"]), page_tokens=int(kv["page_tokens"]),
                      hbm_pages=int(kv["hbm"]), host_pages=int(kv["host"]), alloc=b["alloc"],
                      gva_start=int(kv["start"], 16), world_size=int(kv["world"]), rank=int(kv["rank"]))
    names = {}
    for op in b["ops"]:
        if op[0] == "free":
            pool.free(names.pop(op[1]))
            continue
        if op[0] == "migrate":
            expect = op[op.index("->") + 1:]
            before = (pool.free_pages(), [list(s) for s in pool.stack], pool.sample_pages(names[op[1]]))
            if expect == ["ENOMEM"]:
                with pytest.raises(PoolError) as e:
                    pool.migrate(names[op[1]], int(op[2]))
                assert e.value.code == "ENOMEM"
                assert (pool.free_pages(), [list(s) for s in pool.stack],
                        pool.sample_pages(names[op[1]])) == before
                continue
            pool.migrate(names[op[1]], int(op[2]))
            assert pool.sample_pages(names[op[1]]) == [int(x, 16) for x in expect]
            assert sum(pool.free_pages()) == sum(before[0])
            continue
        arrow = op.index("->")
        nvis = int(op[3])
        wish = [int(x) for x in op[5:arrow]] if "wish" in op else None
        expect = op[arrow + 1:]
        before = (pool.free_pages(), [list(s) for s in pool.stack])
        if expect == ["ENOMEM"]:
            with pytest.raises(PoolError) as e:
                pool.write([1], [0], [nvis], tier_wish=wish)
            assert e.value.code == "ENOMEM"
            assert (pool.free_pages(), [list(s) for s in pool.stack]) == before
            continue
        sid = pool.write([1], [0], [nvis], tier_wish=wish)
        names[op[1]] = sid
        assert pool.sample_pages(sid) == [int(x, 16) for x in expect]


def test_gva_segments_and_translation():
    """I9: page GVAs lie in [region start, start + ws*max) and in this rank's
    [start + r*max, start + (r+1)*max); translating any row address gives the
    frame and offset that hold the row."""
    H, P = 8, 4
    for ws, rank in [(1, 0), (4, 2), (3, 2)]:
        order = [list(range(9, -1, -1)), [3, 1, 4, 0, 5, 2]]
        pool = OraclePool(hidden=H, page_tokens=P, hbm_pages=10, host_pages=6, alloc="scatter",
                          world_size=ws, rank=rank, frame_order=order)
        mx = [10 * P * 2 * H, 6 * P * 2 * H]
        # Page i of tier t is bound to frame order[t][i] (the permuted page table).
        for t in (0, 1):
            for i, f in enumerate(order[t]):
                assert pool.translate(pool.seg_start[t] + i * pool.pb + 3) == (t, f, 3)
        assert pool.region_start[1] == pool.region_start[0] + ws * mx[0]
        rng = np.random.default_rng(ws)
        for i in range(5):
            n = int(rng.integers(1, 10))
            rows = tagged_vis(i, n, H)
            sid = pool.write([0], [0], [n], rows, tier_wish=rng.integers(0, 2, size=-(-n // P)))
            for v, gva in enumerate(pool.sample_pages(sid)):
                tier = 0 if gva < pool.region_start[1] else 1
                assert pool.region_start[tier] <= gva < pool.region_start[tier] + ws * mx[tier]
                assert pool.region_start[tier] + rank * mx[tier] <= gva < pool.region_start[tier] + (rank + 1) * mx[tier]
                assert (gva - pool.seg_start[tier]) % pool.pb == 0
            for v in range(n):
                gva = pool.sample_pages(sid)[v // P] + (v % P) * pool.rb
                t, frame, off = pool.translate(gva)
                assert np.array_equal(pool.frames[t][frame][off // pool.rb], rows[v])


def test_conservation_and_reuse():
    """I6: allocated + free = total, no page in two samples; LIFO reuse."""
    pool = OraclePool(hidden=8, page_tokens=4, hbm_pages=64, alloc="scatter")
    rng = np.random.default_rng(5)
    live = {}
    for step in range(400):
        if live and rng.integers(0, 2):
            k = list(live)[int(rng.integers(0, len(live)))]
            pool.free(k)
            del live[k]
        else:
            n = int(rng.integers(1, 30))
            try:
                sid = pool.write([0], [0], [n])
            except PoolError as e:
                assert e.code == "ENOMEM"
                continue
            live[sid] = pool.sample_pages(sid)
        pages = [g for v in live.values() for g in v]
        assert len(pages) == len(set(pages))
        assert len(pages) + pool.free_pages()[0] == 64
    # Write A, free A, write B of the same page count: B gets A's pages in order.
    a = pool.write([0], [0], [9])
    pa = pool.sample_pages(a)
    pool.free(a)
    b = pool.write([0], [0], [12])
    assert pool.sample_pages(b) == pa


def test_contig_runs():
    """I7: under "contig" every sample's pages are consecutive GVA pages."""
    pool = OraclePool(hidden=8, page_tokens=4, hbm_pages=256, alloc="contig")
    rng = np.random.default_rng(9)
    live = []
    for step in range(300):
        if live and rng.integers(0, 3) == 0:
            pool.free(live.pop(int(rng.integers(0, len(live)))))
            continue
        try:
            sid = pool.write([0], [0], [int(rng.integers(1, 60))])
        except PoolError:
            continue
        live.append(sid)
        g = pool.sample_pages(sid)
        assert all(g[i + 1] - g[i] == pool.pb for i in range(len(g) - 1))


def test_error_paths():
    pool = OraclePool(hidden=8, page_tokens=4, hbm_pages=4, alloc="contig", vocab=10)
    for bad in [dict(text_ids=[1, 2], img_pos=[3], img_ntok=[1]),        # position > T
                dict(text_ids=[1, 2], img_pos=[2, 1], img_ntok=[1, 1]),  # not sorted
                dict(text_ids=[10], img_pos=[], img_ntok=[]),            # id >= vocab
                dict(text_ids=[], img_pos=[], img_ntok=[]),              # empty sample
                dict(text_ids=[1], img_pos=[0], img_ntok=[-1])]:
        with pytest.raises(PoolError) as e:
            pool.write(**bad)
        assert e.value.code == "EINVAL"
    sid = pool.write([1, 2], [1], [16])
    with pytest.raises(PoolError) as e:
        pool.write([1], [0], [1])
    assert e.value.code == "ENOMEM"
    with pytest.raises(PoolError) as e:
        pool.pack([sid], tagged_table(10, 8), out_rows_cap=17)
    assert e.value.code == "ECAPACITY"
    assert pool.pack([sid], tagged_table(10, 8), out_rows_cap=18)[3] == 18     # exactly full is fine
    pool.free(sid)
    for call in (lambda: pool.free(sid), lambda: pool.pack([sid], None)):
        with pytest.raises(PoolError) as e:
            call()
        assert e.value.code == "ENOENT"


def test_tier_mask_split_equals_full():
    """A pack restricted to HBM-tier (plus text) rows followed by one
    restricted to DRAM-tier rows writes the same bytes as one full pack."""
    cfg = scaled(CONFIGS["tiered"], hidden=16, hbm_pages=400, host_pages=400, vocab=500)
    specs = gen_samples(cfg, 1, count=5)
    table = tagged_table(cfg.vocab, cfg.hidden)
    pool = OraclePool(cfg.hidden, cfg.page_tokens, cfg.hbm_pages, cfg.host_pages, "scatter", cfg.vocab)
    rng = np.random.default_rng(3)
    ids = [pool.write(s.text_ids, s.img_pos, s.img_ntok, tagged_vis(i, s.n_vis, cfg.hidden),
                      tier_wish=rng.integers(0, 2, size=-(-s.n_vis // cfg.page_tokens)))
           for i, s in enumerate(specs)]
    full = pool.pack(ids, table)
    out = np.full_like(full[0], 0x5555)
    a = pool.pack(ids, table, tier_mask=MASK_HBM, out=out)
    host_rows = np.all(out == 0x5555, axis=1)
    assert 0 < host_rows.sum() < len(out)
    b = pool.pack(ids, table, tier_mask=MASK_HOST, out=out)
    assert b[1] is None
    assert np.array_equal(out, full[0]) and np.array_equal(a[1], full[1]) and np.array_equal(a[2], full[2])


def test_tier_masks_on_samples_wholly_on_one_tier():
    """Reading R17 on a case checked by eye: sample A has every page on the
    host tier, sample B every page in HBM (the tier wishes are honoured while
    both tiers have room). The HBM mask writes the text rows of both and B's
    image rows and leaves A's image rows as they were; the host mask writes
    A's image rows only and produces no cu_seqlens or position ids."""
    H, P = 8, 2
    pool = OraclePool(H, P, 8, 8, "scatter", 20)
    table = tagged_table(20, H)
    spec_a = SampleSpec(np.array([3, 4, 5], np.int32), np.array([1], np.int32), np.array([3], np.int32))
    spec_b = SampleSpec(np.array([6, 7], np.int32), np.array([2], np.int32), np.array([4], np.int32))
    a = pool.write(spec_a.text_ids, spec_a.img_pos, spec_a.img_ntok, tagged_vis(0, 3, H), tier_wish=[1, 1])
    b = pool.write(spec_b.text_ids, spec_b.img_pos, spec_b.img_ntok, tagged_vis(1, 4, H), tier_wish=[0, 0])
    assert [pool.translate(g)[0] for g in pool.sample_pages(a)] == [1, 1]
    assert [pool.translate(g)[0] for g in pool.sample_pages(b)] == [0, 0]
    # Packed rows: A = t3, v0..v2, t4, t5; B = t6, t7, v0..v3.
    a_vis = [1, 2, 3]
    full = pool.pack([a, b], table)
    sentinel = 0x5A5A
    out = np.full_like(full[0], sentinel)
    hb = pool.pack([a, b], table, tier_mask=MASK_HBM, out=out)
    untouched = np.all(out == sentinel, axis=1)
    assert np.flatnonzero(untouched).tolist() == a_vis
    assert np.array_equal(out[~untouched], full[0][~untouched])
    assert hb[1].tolist() == [0, 6, 12] and hb[2].tolist() == [0, 1, 2, 3, 4, 5, 0, 1, 2, 3, 4, 5]
    out = np.full_like(full[0], sentinel)
    ho = pool.pack([a, b], table, tier_mask=MASK_HOST, out=out)
    written = ~np.all(out == sentinel, axis=1)
    assert np.flatnonzero(written).tolist() == a_vis
    assert np.array_equal(out[written], full[0][written])
    assert ho[1] is None and ho[2] is None


def test_churn_sequence_is_feasible():
    """The churn op sequence never asks a scatter pool for more pages than it
    has free, and ends at or below the target occupancy."""
    cfg = scaled(CONFIGS["frag70b"], hbm_pages=3000)
    ops = churn_ops(cfg, 0, steps=2000)
    pool = OraclePool(hidden=8, page_tokens=cfg.page_tokens, hbm_pages=cfg.hbm_pages, alloc="scatter")
    keys = {}
    for op in ops:
        if op.kind == "write":
            keys[op.key] = pool.write(op.spec.text_ids, op.spec.img_pos, op.spec.img_ntok)
        else:
            pool.free(keys.pop(op.key))
    assert cfg.hbm_pages - pool.free_pages()[0] <= 0.5 * cfg.hbm_pages
    assert sum(op.kind == "write" for op in ops) > 500


def test_migration_keeps_bytes_and_conserves_pages():
    """Moving samples between tiers changes where their rows live, never the
    packed bytes (consumers read by GVA, Sec. 3.2), and conserves pages."""
    cfg = scaled(CONFIGS["tiered"], hidden=64, hbm_pages=40, host_pages=40, vocab=200)
    rng = np.random.default_rng(8)
    pool = OraclePool(cfg.hidden, 8, cfg.hbm_pages, cfg.host_pages, "scatter", cfg.vocab)
    table = tagged_table(cfg.vocab, cfg.hidden)
    ids, vis = [], []
    for i in range(8):
        nv = int(rng.integers(0, 30))
        v = tagged_vis(i, nv, cfg.hidden)
        wish = [int(x) for x in rng.integers(0, 2, size=-(-nv // 8))]
        ids.append(pool.write(rng.integers(0, cfg.vocab, size=5), [2] if nv else [], [nv] if nv else [], v,
                              tier_wish=wish))
        vis.append(v)
    want = pool.pack(ids, table)[0]
    total = sum(pool.free_pages())
    for _ in range(30):
        sid = ids[int(rng.integers(0, len(ids)))]
        try:
            pool.migrate(sid, int(rng.integers(0, 2)))
        except PoolError as e:
            assert e.code == "ENOMEM"
        assert np.array_equal(pool.pack(ids, table)[0], want)
        assert sum(pool.free_pages()) == total
        pages = [g for i in ids for g in pool.sample_pages(i)]
        assert len(pages) == len(set(pages))
    for sid in ids:
        pool.migrate(sid, 0)
        assert all(pool.translate(g)[0] == 0 for g in pool.sample_pages(sid))
    assert np.array_equal(pool.pack(ids, table)[0], want)


def _held(pool, live):
    """(tier, page index) of every page held by the live samples, from their page lists."""
    return {pool._page_of(g) for sid in live for g in pool.sample_pages(sid)}


@pytest.mark.parametrize("seed", range(6))
def test_contig_first_fit_certificate(seed):
    """Reading R6, contig: every write takes the lowest-index run of free
    pages of its length in the HBM tier, else in the host tier, and fails
    exactly when neither tier has such a run. Checked from the outside on
    random writes and frees: the free pages are those no live sample's page
    list holds, and the run is searched for among them, not in the pool's
    own state."""
    rng = np.random.default_rng(300 + seed)
    n_pages = (40, 24)
    pool = OraclePool(hidden=8, page_tokens=3, hbm_pages=n_pages[0], host_pages=n_pages[1], alloc="contig")
    live = []

    def lowest_run(held, n):
        for t in (0, 1):
            run = 0
            for i in range(n_pages[t]):
                run = 0 if (t, i) in held else run + 1
                if run == n:
                    return [(t, j) for j in range(i - n + 1, i + 1)]
        return None

    for step in range(500):
        if live and rng.integers(0, 3) == 0:
            pool.free(live.pop(int(rng.integers(0, len(live)))))
            continue
        n_vis = int(rng.integers(1, 3 * 20))
        n = -(-n_vis // 3)
        want = lowest_run(_held(pool, live), n)
        try:
            sid = pool.write([1], [0], [n_vis])
        except PoolError as e:
            assert e.code == "ENOMEM" and want is None
            continue
        live.append(sid)
        assert [pool._page_of(g) for g in pool.sample_pages(sid)] == want


@pytest.mark.parametrize("seed", range(6))
def test_scatter_lifo_against_a_timestamp_model(seed):
    """Reading R6, scatter: a page goes to the wished tier, or the other one
    when the wished tier has no free page; within a tier the page taken is
    the one freed most recently (a free gives its last page back first, so
    the first page comes back on top), and a never-used page after all freed
    ones, lowest index first. The model keeps no stacks: each free page of a
    tier carries a rank (a never-used page i: -i; a freed page: a counter
    that grows with every page given back) and a write takes the highest
    rank. Random writes with random tier wishes, frees and migrations."""
    rng = np.random.default_rng(400 + seed)
    n_pages = (30, 30)
    P = 2
    pool = OraclePool(hidden=8, page_tokens=P, hbm_pages=n_pages[0], host_pages=n_pages[1], alloc="scatter")
    rank = [{i: -i for i in range(n_pages[t])} for t in (0, 1)]     # free pages of each tier -> rank
    clock = [0]

    def give_back(pages):                       # pages in a sample's order; the last one is given back first
        for t, i in reversed(pages):
            clock[0] += 1
            rank[t][i] = clock[0]

    def take(t):
        i = max(rank[t], key=rank[t].get)
        del rank[t][i]
        return (t, i)

    live = {}
    for step in range(600):
        op = rng.integers(0, 5)
        if live and op == 0:
            sid = list(live)[int(rng.integers(0, len(live)))]
            pool.free(sid)
            give_back(live.pop(sid))
        elif live and op == 1:
            sid = list(live)[int(rng.integers(0, len(live)))]
            tier = int(rng.integers(0, 2))
            moving = [k for k, p in enumerate(live[sid]) if p[0] != tier]
            try:
                pool.migrate(sid, tier)
            except PoolError as e:
                assert e.code == "ENOMEM" and len(moving) > len(rank[tier])
                continue
            old = [live[sid][k] for k in moving]
            for k in moving:
                live[sid][k] = take(tier)
            give_back(old)
            assert [pool._page_of(g) for g in pool.sample_pages(sid)] == live[sid]
        else:
            n_vis = int(rng.integers(1, 2 * 12))
            n = -(-n_vis // P)
            wish = rng.integers(0, 2, size=n).astype(np.uint8)
            free = [len(rank[0]), len(rank[1])]
            try:
                sid = pool.write([1], [0], [n_vis], tier_wish=wish)
            except PoolError as e:
                assert e.code == "ENOMEM" and n > free[0] + free[1]
                continue
            want = []
            for w in wish.tolist():
                t = w if rank[w] else 1 - w
                want.append(take(t))
            live[sid] = want
            assert [pool._page_of(g) for g in pool.sample_pages(sid)] == want
