"""Tier-masked packs of tiered pools against the oracle, element by element.

A masked pack of a pool with a host tier copies only the rows its mask
selects (text rows and rows on HBM pages for FP_TIER_MASK_HBM, rows on host
pages for FP_TIER_MASK_HOST); each row's tier comes from its page-table
entry. Checked on random pools (page sizes from 1 row, random per-page tier
wishes, samples wholly on one tier, hidden sizes whose chunks resolve one row
per wave or one row per lane, chunk geometries for 1, 2, 5 or all compute
units):
- each masked pack writes exactly the oracle's masked rows and leaves every
  other row as it was (the buffers start filled with a marker);
- cu_seqlens and position ids come with the HBM mask only;
- the two masked packs into one buffer equal one full pack.
Plus one pack of 140,000 one-row pages whose tiers alternate row by row.

Each case prints its seed and shape before touching the GPU.
"""

import numpy as np
import pytest

from gpu_common import say, to_dev, to_host
from oracle.pool import MASK_HBM, MASK_HOST, OraclePool
from paper_2606_23087_amd.workloads import SampleSpec
from tagging import tagged_table, tagged_vis

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

MARK = 0x2222


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def _spec(rng, vocab):
    while True:
        t = int(rng.integers(0, 61))
        k = int(rng.integers(0, 6))
        pos = np.sort(rng.integers(0, t + 1, size=k)).astype(np.int32)
        ntok = rng.integers(0, 90, size=k).astype(np.int32)
        if t + int(ntok.sum()) > 0:
            return SampleSpec(rng.integers(0, vocab, size=t).astype(np.int32), pos, ntok)


def _wish(rng, n_pages):
    kind = rng.random()
    if kind < 0.15:
        return np.zeros(n_pages, np.uint8)               # all on HBM
    if kind < 0.3:
        return np.ones(n_pages, np.uint8)                # all on the host tier
    return (rng.random(n_pages) < 0.5).astype(np.uint8)


def _check_masks(fp, pool, ids, opool, oids, t_dev, table, vocab, hidden, total, n):
    out = torch.full((total + 8, hidden), MARK, dtype=torch.int16, device="cuda")
    cu = torch.full((n + 2,), -1, dtype=torch.int32, device="cuda")
    pos = torch.full((total + 8,), -1, dtype=torch.int32, device="cuda")
    m, _ = fp.pack_microbatch(pool, ids, t_dev, vocab, out, out.shape[0], cu, pos, fp.FP_TIER_MASK_HBM)
    torch.cuda.synchronize()
    want = opool.pack(oids, table, tier_mask=MASK_HBM, out=np.full((total, hidden), MARK, np.uint16))
    assert m == total and np.array_equal(to_host(out[:m]), want[0]), "HBM-masked rows"
    assert bool((out[m:] == MARK).all())
    assert cu[:n + 1].cpu().numpy().tolist() == want[1].tolist()
    assert pos[:m].cpu().numpy().tolist() == want[2].tolist() and bool((pos[m:] == -1).all())
    host = torch.full_like(out, MARK)
    fp.pack_microbatch(pool, ids, None, 0, host, host.shape[0], None, None, fp.FP_TIER_MASK_HOST)
    torch.cuda.synchronize()
    want_h = opool.pack(oids, None, tier_mask=MASK_HOST, out=np.full((total, hidden), MARK, np.uint16))
    assert np.array_equal(to_host(host[:m]), want_h[0]), "host-masked rows"
    assert bool((host[m:] == MARK).all())
    # both masks into one buffer == one full pack
    fp.pack_microbatch(pool, ids, None, 0, out, out.shape[0], None, None, fp.FP_TIER_MASK_HOST)
    full = torch.full_like(out, MARK)
    fp.pack_microbatch(pool, ids, t_dev, vocab, full, full.shape[0], None, None, fp.FP_TIER_MASK_ALL)
    torch.cuda.synchronize()
    assert torch.equal(out, full)
    assert np.array_equal(to_host(full[:m]), opool.pack(oids, table)[0])


@pytest.mark.parametrize("seed", range(440))
def test_random_tier_masks(fp, seed):
    rng = np.random.default_rng(7100 + seed)
    hidden = int(rng.choice([8, 24, 64, 200, 1024, 4096, 5120]))
    page_tokens = int(rng.integers(1, 70))
    pack_cus = int(rng.choice([0, 1, 2, 5]))
    vocab = 89
    n = int(rng.integers(1, 40))
    specs = [_spec(rng, vocab) for _ in range(n)]
    wishes = [_wish(rng, -(-s.n_vis // page_tokens)) for s in specs]
    pages = [int((w == 0).sum()) for w in wishes], [int((w == 1).sum()) for w in wishes]
    hbm, host = sum(pages[0]) + 4, sum(pages[1]) + 4
    say(f"case tier masks seed={seed} H={hidden} P={page_tokens} pack_cus={pack_cus} samples={n} "
        f"pages={hbm}+{host}")
    pool = fp.pool_create(hidden=hidden, page_tokens=page_tokens, hbm_pages=hbm, host_pages=host, vocab=vocab,
                          alloc="scatter", pack_cus=pack_cus)
    try:
        opool = OraclePool(hidden, page_tokens, hbm, host, "scatter", vocab)
        table = tagged_table(vocab, hidden, seed)
        t_dev = to_dev(table)
        ids, oids = [], []
        for i, (s, w) in enumerate(zip(specs, wishes)):
            v = tagged_vis(i, s.n_vis, hidden, seed)
            ids.append(fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, to_dev(v) if s.n_vis else None,
                                            w))
            oids.append(opool.write(s.text_ids, s.img_pos, s.img_ntok, v, tier_wish=w))
            assert fp.pool_sample_pages(pool, ids[-1]).tolist() == opool.sample_pages(oids[-1])
        torch.cuda.synchronize()
        for g in range(2):
            pick = rng.permutation(n)[:int(rng.integers(1, n + 1))].tolist()
            total = sum(specs[i].length for i in pick)
            _check_masks(fp, pool, [ids[i] for i in pick], opool, [oids[i] for i in pick], t_dev, table, vocab,
                         hidden, total, len(pick))
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)


def test_alternating_one_row_pages(fp):
    """140,000 one-row pages alternating between the tiers: every other row
    of the image is copied by each mask."""
    hidden, rows, vocab = 8, 140_000, 11
    say(f"case alternating one-row pages H={hidden} P=1 rows={rows}")
    spec = SampleSpec(np.array([1, 2, 3], np.int32), np.array([1], np.int32), np.array([rows], np.int32))
    wish = (np.arange(rows) % 2).astype(np.uint8)
    pool = fp.pool_create(hidden=hidden, page_tokens=1, hbm_pages=rows // 2 + 2, host_pages=rows // 2 + 2,
                          vocab=vocab, alloc="scatter")
    try:
        opool = OraclePool(hidden, 1, rows // 2 + 2, rows // 2 + 2, "scatter", vocab)
        table = tagged_table(vocab, hidden, 1)
        v = tagged_vis(0, rows, hidden, 1)
        sid = fp.pool_write_sample(pool, spec.text_ids, spec.img_pos, spec.img_ntok, to_dev(v), wish)
        oid = opool.write(spec.text_ids, spec.img_pos, spec.img_ntok, v, tier_wish=wish)
        torch.cuda.synchronize()
        _check_masks(fp, pool, [sid], opool, [oid], to_dev(table), table, vocab, hidden, spec.length, 1)
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)
