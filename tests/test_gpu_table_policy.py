"""Packs whose embedding table takes either load policy, against the oracle's
layout, every word.

The pack reads the chunks that hold embedding-table rows with plain loads
when the table (vocab rows of 2H bytes) is at most 2.5 GiB, and with
non-temporal loads when it is larger; the policy changes timing only. Here a
16 MiB table and a 2.95 GB one (H 8192, 180,000 rows, built on the device by
a pattern generator whose host twin gives the expected words) back the same
kind of microbatches: text stretches at ids spread over the whole table (its
first and last rows included) between images. Every word of every row must
equal the row the oracle's layout names for it (Sec. 3.1 pairing), and the
rows past the microbatch stay untouched. Bar: bit-exact.
"""

import numpy as np
import pytest

from gpu_common import say, to_dev, to_host
from oracle.pack import row_sources
from paper_2606_23087_amd.workloads import TAG_TEXT, SampleSpec
from tagging import tagged_vis

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

H = 8192
BASE_ROWS = 89


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def _base(seed):
    return np.random.default_rng([seed, 0x7AB1E]).integers(0, 1 << 16, size=(BASE_ROWS, H), dtype=np.uint16)


def _table_rows_host(ids, base):
    """Row id of the pattern table: a row of the seeded base chosen by the id,
    with its first four words (TAG_TEXT, lo16(id), hi16(id), 0)."""
    ids = np.asarray(ids, np.int64)
    rows = base[(5 * ids + 3) % BASE_ROWS]
    rows[:, 0] = TAG_TEXT
    rows[:, 1] = ids & 0xFFFF
    rows[:, 2] = (ids >> 16) & 0xFFFF
    rows[:, 3] = 0
    return rows


def _table_dev(vocab, base, block=1 << 14):
    """The same table built on the GPU in blocks (int16 view)."""
    def i16(x):
        return ((x & 0xFFFF) ^ 0x8000) - 0x8000

    b = torch.from_numpy(base.view(np.int16)).to("cuda")
    t = torch.empty((vocab, H), dtype=torch.int16, device="cuda")
    for r0 in range(0, vocab, block):
        r = torch.arange(r0, min(r0 + block, vocab), dtype=torch.int64, device="cuda")
        blk = t[r0:r0 + r.numel()]
        blk.copy_(b[(5 * r + 3) % BASE_ROWS])
        blk[:, 0] = i16(TAG_TEXT)
        blk[:, 1] = i16(r).to(torch.int16)
        blk[:, 2] = i16(r >> 16).to(torch.int16)
        blk[:, 3] = 0
    return t


def _specs(rng, vocab, n):
    specs = []
    for i in range(n):
        t = int(rng.integers(20, 400))
        ids = rng.integers(0, vocab, size=t).astype(np.int32)
        if i == 0:
            ids[0], ids[-1] = 0, vocab - 1
        k = int(rng.integers(0, 4))
        pos = np.sort(rng.integers(0, t + 1, size=k)).astype(np.int32)
        ntok = rng.integers(10, 100, size=k).astype(np.int32)
        specs.append(SampleSpec(ids, pos, ntok))
    return specs


@pytest.mark.parametrize("vocab", [1024, 180_000])
def test_table_load_policy(fp, vocab):
    seed = vocab % 97
    rng = np.random.default_rng(seed)
    policy = "plain" if vocab * 2 * H <= 5 << 29 else "non-temporal"
    say(f"case table load policy: vocab={vocab} H={H} ({vocab * 2 * H / 1e9:.2f} GB table, {policy} loads)")
    base = _base(seed)
    torch.cuda.empty_cache()
    table = _table_dev(vocab, base)
    specs = _specs(rng, vocab, 8)
    P = 32
    pages = sum(-(-s.n_vis // P) for s in specs) + 2
    pool = fp.pool_create(hidden=H, page_tokens=P, hbm_pages=pages, vocab=vocab, alloc="scatter")
    try:
        vis = [tagged_vis(i, s.n_vis, H, seed) for i, s in enumerate(specs)]
        ids = [fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, to_dev(v) if s.n_vis else None)
               for s, v in zip(specs, vis)]
        torch.cuda.synchronize()
        for pick in ([0, 1, 2, 3, 4, 5, 6, 7], [7, 3, 0], [5]):
            sp = [specs[i] for i in pick]
            total = sum(s.length for s in sp)
            out = torch.full((total + 3, H), 0x3C3C, dtype=torch.int16, device="cuda")
            m, _ = fp.pack_microbatch(pool, [ids[i] for i in pick], table, vocab, out, out.shape[0])
            torch.cuda.synchronize()
            assert m == total
            want = np.empty((total, H), np.uint16)
            src = row_sources(sp)
            text = [r for r, (k, _, _) in enumerate(src) if k == "text"]
            want[text] = _table_rows_host([src[r][2] for r in text], base)
            for r, (k, g, x) in enumerate(src):
                if k != "text":
                    want[r] = vis[pick[g]][x]
            got = to_host(out[:total])
            bad = np.nonzero(np.any(got != want, axis=1))[0]
            assert bad.size == 0, f"samples {pick}: {bad.size} rows differ, first {bad[:5]}"
            assert bool((out[total:] == 0x3C3C).all())
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)
        del table
        torch.cuda.empty_cache()
