"""Pins for the definitional pack and the pool oracle's pack (CPU only).

- a hand-worked microbatch (tests/golden/pack_worked_example.txt);
- invariants that the paper's formulation fixes: cu_seqlens are the prefix
  sums of sample lengths, position ids restart per sample, every written
  token appears exactly once in its sample's slot, and the interleaving puts
  image j after exactly p_j of the sample's text tokens (Sec. 3.1, Sec. 4.1);
- the pool's pack equals the definition whatever the physical placement
  (Sec. 3.1 / Sec. 3.2: the backbone reads by GVA without knowing where the
  bytes are).
"""

import numpy as np
import pytest

from oracle.pack import definitional_pack, row_sources, sample_segments
from oracle.pool import OraclePool
from paper_2606_23087_amd.workloads import CONFIGS, SampleSpec, gen_samples, scaled
from tagging import decode, tagged_table, tagged_vis
from conftest import read_golden

H = 16


def _parse_pack_golden():
    lines = read_golden("pack_worked_example.txt")
    text, images, order, rows, cu, pos = {}, {}, None, None, None, None
    for ln in lines:
        f = ln.split()
        if f[0] == "sample" and f[2] == "text":
            text[f[1]] = [int(x) for x in f[3:]]
        elif f[0] == "sample" and f[2] == "images":
            images[f[1]] = [tuple(int(y) for y in x.split(":")) for x in f[3:]]
        elif f[0] == "order":
            order = f[1:]
        elif f[0] == "rows":
            rows = f[1:]
        elif f[0] == "cu":
            cu = [int(x) for x in f[1:]]
        elif f[0] == "pos":
            pos = [int(x) for x in f[1:]]
    specs = []
    for name in order:
        ims = images[name]
        specs.append(SampleSpec(text_ids=np.array(text[name], dtype=np.int32),
                                img_pos=np.array([p for p, _ in ims], dtype=np.int32),
                                img_ntok=np.array([n for _, n in ims], dtype=np.int32)))
    expect = []
    for r in rows:
        name, what = r.split(":")
        s = order.index(name)
        if what[0] == "t":
            expect.append(("text", int(what[1:])))
        else:
            expect.append(("vis", s, int(what[1:])))
    return specs, expect, cu, pos


def _decode_expected(specs):
    out = []
    for kind, s, x in row_sources(specs):
        out.append(("text", x) if kind == "text" else ("vis", s, x))
    return out


def test_worked_example_definitional():
    specs, expect, cu, pos = _parse_pack_golden()
    table = tagged_table(32, H)
    vis = [tagged_vis(i, s.n_vis, H) for i, s in enumerate(specs)]
    rows, cu_o, pos_o, mx = definitional_pack(specs, vis, table)
    assert decode(rows) == expect
    assert cu_o.tolist() == cu
    assert pos_o.tolist() == pos
    assert mx == max(np.diff(cu))
    assert _decode_expected(specs) == expect


@pytest.mark.parametrize("alloc", ["contig", "scatter"])
def test_worked_example_pool(alloc):
    specs, expect, cu, pos = _parse_pack_golden()
    table = tagged_table(32, H)
    pool = OraclePool(hidden=H, page_tokens=2, hbm_pages=16, alloc=alloc, vocab=32)
    ids = [pool.write(s.text_ids, s.img_pos, s.img_ntok, tagged_vis(i, s.n_vis, H))
           for i, s in enumerate(specs)]
    rows, cu_o, pos_o, n, mx = pool.pack(ids, table)
    assert decode(rows) == expect
    assert cu_o.tolist() == cu and pos_o.tolist() == pos and n == cu[-1]


def _random_specs(rng, n, max_text=40, max_img=4, max_tok=9, vocab=50):
    specs = []
    for _ in range(n):
        t = int(rng.integers(0, max_text + 1))
        k = int(rng.integers(0, max_img + 1))
        ntok = rng.integers(0, max_tok + 1, size=k).astype(np.int32)
        if t + int(ntok.sum()) == 0:
            t = 1
        pos = np.sort(rng.integers(0, t + 1, size=k)).astype(np.int32)
        specs.append(SampleSpec(rng.integers(0, vocab, size=t).astype(np.int32), pos, ntok))
    return specs


@pytest.mark.parametrize("seed", range(20))
def test_invariants_random(seed):
    rng = np.random.default_rng(seed)
    specs = _random_specs(rng, int(rng.integers(1, 8)))
    table = tagged_table(50, H, seed)
    vis = [tagged_vis(i, s.n_vis, H, seed) for i, s in enumerate(specs)]
    rows, cu, pos, mx = definitional_pack(specs, vis, table)
    lens = [s.length for s in specs]
    # I1: cu_seqlens are the prefix sums of the sample lengths.
    assert cu[0] == 0 and np.all(np.diff(cu) == np.array(lens)) and np.all(np.diff(cu) > 0)
    # I2: position ids restart at 0 in every sample.
    for k in range(len(specs)):
        assert pos[cu[k]:cu[k + 1]].tolist() == list(range(lens[k]))
    assert mx == max(lens)
    tags = decode(rows)
    for k, s in enumerate(specs):
        seg = tags[cu[k]:cu[k + 1]]
        # I4: each visual row of the sample exactly once, nothing foreign.
        vis_tags = [t for t in seg if t[0] == "vis"]
        assert all(t[1] == k for t in vis_tags)
        assert [t[2] for t in vis_tags] == list(range(s.n_vis))
        # I3: text rows are the sample's ids in order ...
        assert [t[1] for t in seg if t[0] == "text"] == s.text_ids.tolist()
        # ... and image j starts after exactly p_j of the sample's text tokens.
        first_vis = np.cumsum([0] + s.img_ntok.tolist())
        for j in range(len(s.img_pos)):
            if s.img_ntok[j] == 0:
                continue
            at = [i for i, t in enumerate(seg) if t[0] == "vis" and t[2] == first_vis[j]][0]
            assert sum(1 for t in seg[:at] if t[0] == "text") == s.img_pos[j]
    # Row bytes beyond the tags: text rows equal the table rows, visual rows
    # equal the producer's rows.
    for r, t in zip(rows, tags):
        if t[0] == "text":
            assert np.array_equal(r, table[t[1]])
        else:
            assert np.array_equal(r, vis[t[1]][t[2]])


@pytest.mark.parametrize("seed", range(6))
def test_pool_pack_equals_definition_any_placement(seed):
    """I5: placement independence across allocation policy, frame order,
    tier wishes and a history of writes and frees."""
    rng = np.random.default_rng(100 + seed)
    specs = _random_specs(rng, 6, max_tok=11)
    table = tagged_table(50, H, seed)
    vis = [tagged_vis(i, s.n_vis, H, seed) for i, s in enumerate(specs)]
    want = definitional_pack(specs, vis, table)
    P = 3
    variants = []
    perm = [list(rng.permutation(200)), list(rng.permutation(200))]
    for alloc, host, frame_order, churn in [("contig", 0, None, False), ("scatter", 0, None, True),
                                            ("scatter", 200, perm, True), ("contig", 200, perm, True)]:
        pool = OraclePool(hidden=H, page_tokens=P, hbm_pages=200, host_pages=host, alloc=alloc,
                          vocab=50, frame_order=frame_order)
        if churn:
            junk = [pool.write([0] * 3, [1], [int(rng.integers(1, 12))]) for _ in range(8)]
            for j in rng.permutation(len(junk))[:5]:
                pool.free(junk[j])
        ids = []
        for i, s in enumerate(specs):
            npg = -(-s.n_vis // P)
            wish = rng.integers(0, 2, size=npg) if (alloc == "scatter" and host) else None
            ids.append(pool.write(s.text_ids, s.img_pos, s.img_ntok, vis[i], tier_wish=wish))
        variants.append(pool.pack(ids, table))
    for rows, cu, pos, n, mx in variants:
        assert np.array_equal(rows, want[0])
        assert np.array_equal(cu, want[1]) and np.array_equal(pos, want[2]) and mx == want[3]


def test_segments_cover_sample():
    s = sample_segments(5, [2, 2, 5], [2, 1, 3])
    assert s == [("text", 0, 2), ("vis", 0, 2), ("text", 2, 0), ("vis", 2, 1),
                 ("text", 2, 3), ("vis", 3, 3), ("text", 5, 0)]


def test_tiny_workload_pack():
    """The tiny workload packs under both pool policies to its definition."""
    cfg = CONFIGS["tiny"]
    specs = gen_samples(cfg, 0)
    table = tagged_table(cfg.vocab, cfg.hidden)
    vis = [tagged_vis(i, s.n_vis, cfg.hidden) for i, s in enumerate(specs)]
    want = definitional_pack(specs[:3], vis[:3], table)
    pool = OraclePool(cfg.hidden, cfg.page_tokens, cfg.hbm_pages, alloc="contig", vocab=cfg.vocab)
    ids = [pool.write(s.text_ids, s.img_pos, s.img_ntok, vis[i]) for i, s in enumerate(specs)]
    rows, cu, pos, n, mx = pool.pack(ids[:3], table)
    assert np.array_equal(rows, want[0]) and np.array_equal(cu, want[1])
