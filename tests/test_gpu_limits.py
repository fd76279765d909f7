"""GPU parity at the limits pack_microbatch accepts, and refusal one step past
them (Sec. 3.1 consumer pack; the limits are the library's own):

- the largest microbatch: 2^31 - 1024 16-byte vectors (2,097,151 rows at
  H 8192, a 32 GiB output) from a 32 GiB pool, whose one large sample is
  itself the largest write;
- the most samples (1024) and the most images (1024) in one microbatch.

The oracle's layout names the source of every row of the large pack: the
tag words of every row, all cu_seqlens and position ids, sampled whole rows
(both ends, the shrinking tail chunks, random ones), and then every word of
every row, slice by slice, against the rows the generators wrote (the host
twin of the device pattern and the host table) are checked, and the guard
rows past the microbatch must be untouched.
Bar: bit-exact.
"""

import numpy as np
import pytest

from gpu_common import say, to_dev, to_host
from oracle.pack import definitional_pack, row_sources
from paper_2606_23087_amd.workloads import TAG_TEXT, TAG_VIS, SampleSpec
from tagging import PATTERN_BASE_ROWS, pattern_base, pattern_row, pattern_rows_dev, tagged_table, tagged_vis

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

MAX_VECTORS = (1 << 31) - 1024


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def test_largest_microbatch(fp):
    H, P, VOCAB, SEED = 8192, 256, 16, 4
    vpr = 2 * H // 16
    max_rows = MAX_VECTORS // vpr                                # 2,097,151
    n_big = max_rows - 6
    specs = [SampleSpec(np.array([5, 6, 7], np.int32), np.array([2], np.int32), np.array([n_big], np.int32)),
             SampleSpec(np.array([8, 9], np.int32), np.array([1], np.int32), np.array([1], np.int32))]
    assert sum(s.length for s in specs) == max_rows
    pages = sum(-(-s.n_vis // P) for s in specs)
    say(f"case largest microbatch: H={H} P={P} rows={max_rows} pages={pages} "
        f"({pages * P * 2 * H / 2**30:.1f} GiB pool)")
    torch.cuda.empty_cache()
    pool = fp.pool_create(hidden=H, page_tokens=P, hbm_pages=pages + 1, vocab=VOCAB, alloc="scatter")
    try:
        table_np = tagged_table(VOCAB, H, SEED)
        table = to_dev(table_np)
        ids = []
        for g, s in enumerate(specs):
            vis = pattern_rows_dev(g, s.n_vis, H, SEED)
            say(f"  write sample {g}: {s.n_vis} image rows")
            ids.append(fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, vis))
            torch.cuda.synchronize()
            del vis
        torch.cuda.empty_cache()
        guard = 4
        out = torch.full((max_rows + guard, H), 0x5A5A, dtype=torch.int16, device="cuda")
        cu = torch.full((3,), -1, dtype=torch.int32, device="cuda")
        pos = torch.full((max_rows + guard,), -1, dtype=torch.int32, device="cuda")
        say("  pack")
        m, mx = fp.pack_microbatch(pool, ids, table, VOCAB, out, out.shape[0], cu, pos)
        torch.cuda.synchronize()
        assert m == max_rows and mx == specs[0].length
        assert cu.cpu().numpy().tolist() == [0, specs[0].length, max_rows]
        want_pos = np.concatenate([np.arange(s.length, dtype=np.int32) for s in specs])
        assert np.array_equal(pos[:m].cpu().numpy(), want_pos)
        assert bool((pos[m:] == -1).all())
        assert bool((out[m:] == 0x5A5A).all())
        say("  tags of every row")
        src = row_sources(specs)
        text = np.fromiter((k == "text" for k, _, _ in src), bool, m)
        g = np.fromiter((s for _, s, _ in src), np.int64, m)
        x = np.fromiter((v for _, _, v in src), np.int64, m)
        # Text rows carry the table's tags, image rows the generator's
        # (TAG_VIS, sample, lo16 and hi16 of the visual index).
        tags = np.where(text[:, None],
                        np.stack([np.full(m, TAG_TEXT), x & 0xFFFF, x >> 16, np.zeros(m, np.int64)], 1),
                        np.stack([np.full(m, TAG_VIS), g & 0xFFFF, x & 0xFFFF, x >> 16], 1)).astype(np.uint16)
        got = to_host(out[:m, :4].contiguous())
        bad = np.nonzero(np.any(got != tags, axis=1))[0]
        assert bad.size == 0, f"{bad.size} rows with a wrong source, first {bad[:5]}"
        say("  sampled whole rows")
        base = pattern_base(H, SEED)
        rng = np.random.default_rng(SEED)
        picks = sorted(set(list(range(4)) + list(range(m - 4, m)) + list(range(m - 700, m, 37)) +
                           rng.integers(0, m, size=24).tolist()))
        for r in picks:
            kind, g, x = src[r]
            want = table_np[x] if kind == "text" else pattern_row(g, x, H, SEED, base)
            assert np.array_equal(to_host(out[r]), want), f"row {r} ({kind})"
        say("  every word of every row, in slices of 65536 rows")
        g = np.fromiter((s for _, s, _ in src), np.int64, m)
        x = np.fromiter((v for _, _, v in src), np.int64, m)
        for a in range(0, m, 1 << 16):
            b = min(a + (1 << 16), m)
            want = np.empty((b - a, H), np.uint16)
            t = text[a:b]
            want[t] = table_np[x[a:b][t]]
            gv, xv = g[a:b][~t], x[a:b][~t]
            rows = base[(7 * xv + gv) % PATTERN_BASE_ROWS]
            rows[:, 0] = TAG_VIS
            rows[:, 1] = gv & 0xFFFF
            rows[:, 2] = xv & 0xFFFF
            rows[:, 3] = (xv >> 16) & 0xFFFF
            want[~t] = rows
            got = to_host(out[a:b])
            assert np.array_equal(got, want), f"rows {a}..{b}: first differing row " \
                f"{a + int(np.nonzero(np.any(got != want, axis=1))[0][0])}"
        say("  one row more, or one visual row more in a write, is refused")
        extra = fp.pool_write_sample(pool, [3], [], [])
        before = fp.pool_stats(pool)
        with pytest.raises(fp.FlowPoolError) as e:
            fp.pack_microbatch(pool, ids + [extra], table, VOCAB, out, out.shape[0], None, pos)
        assert e.value.code == "EINVAL"
        with pytest.raises(fp.FlowPoolError) as e:
            fp.pool_write_sample(pool, [], [0], [max_rows + 1])
        assert e.value.code == "EINVAL"
        assert fp.pool_stats(pool) == before
        torch.cuda.synchronize()
        assert bool((out[m:] == 0x5A5A).all())
        del out, pos
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)
        torch.cuda.empty_cache()


def test_most_samples_and_images(fp):
    """1024 samples with one image each: the staged run table at its largest
    (about three runs per sample). One sample more, or one image more, is
    refused."""
    H, P, VOCAB, SEED = 64, 4, 50, 6
    rng = np.random.default_rng(SEED)
    specs = []
    for _ in range(1024):
        t = int(rng.integers(0, 4))
        specs.append(SampleSpec(rng.integers(0, VOCAB, size=t).astype(np.int32),
                                np.array([int(rng.integers(0, t + 1))], np.int32),
                                np.array([int(rng.integers(1, 6))], np.int32)))
    specs.append(SampleSpec(np.array([1], np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32)))
    specs.append(SampleSpec(np.array([2], np.int32), np.array([0, 1], np.int32), np.array([2, 1], np.int32)))
    say(f"case most samples and images: H={H} P={P} samples=1024")
    pages = sum(-(-s.n_vis // P) for s in specs)
    pool = fp.pool_create(hidden=H, page_tokens=P, hbm_pages=pages, vocab=VOCAB, alloc="scatter")
    try:
        table = tagged_table(VOCAB, H, SEED)
        t_dev = to_dev(table)
        vis = [tagged_vis(i, s.n_vis, H, SEED) for i, s in enumerate(specs)]
        ids = [fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, to_dev(v) if s.n_vis else None)
               for s, v in zip(specs, vis)]
        torch.cuda.synchronize()
        n = sum(s.length for s in specs)
        out = torch.full((n, H), 0x3333, dtype=torch.int16, device="cuda")
        cu = torch.full((1027,), -1, dtype=torch.int32, device="cuda")
        pos = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        pick = list(range(1024))[::-1]
        m, mx = fp.pack_microbatch(pool, [ids[i] for i in pick], t_dev, VOCAB, out, n, cu, pos)
        torch.cuda.synchronize()
        want = definitional_pack([specs[i] for i in pick], [vis[i] for i in pick], table)
        assert m == len(want[0]) and mx == want[3]
        assert np.array_equal(to_host(out[:m]), want[0])
        assert cu[:1025].cpu().numpy().tolist() == want[1].tolist() and int(cu[1025]) == -1
        assert pos[:m].cpu().numpy().tolist() == want[2].tolist()
        assert bool((out[m:] == 0x3333).all())
        with pytest.raises(fp.FlowPoolError) as e:     # a 1025th sample (text only)
            fp.pack_microbatch(pool, [ids[i] for i in pick] + [ids[1024]], t_dev, VOCAB, out, n, cu, pos)
        assert e.value.code == "EINVAL" and "outside [0, 1024]" in str(e.value)
        with pytest.raises(fp.FlowPoolError) as e:     # 1024 samples holding 1025 images
            fp.pack_microbatch(pool, [ids[i] for i in pick[1:]] + [ids[1025]], t_dev, VOCAB, out, n, cu, pos)
        assert e.value.code == "EINVAL" and "1025 images" in str(e.value)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(out[:m]), want[0])
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)
