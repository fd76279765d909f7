"""GPU parity of the HIP path against the CPU oracle, element by element, on
seeded inputs small enough for the oracle (each microbatch spans many
workgroup tiles and ends in a ragged tail).

Every case prints its name, seed and shape before touching the GPU.
Bar: bit-exact (pure indexing and raw 16-bit copies; integer plan).
"""

import numpy as np
import pytest

from gpu_common import oracle_plan, oracle_pool_for, say, to_dev, to_host
from oracle.pack import definitional_pack
from oracle.pool import MASK_HBM, MASK_HOST
from paper_2606_23087_amd.workloads import (CONFIGS, SampleSpec, gen_samples, scaled, table_np,
                                            visual_rows_np)
from tagging import decode, tagged_table, tagged_vis

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def _inputs(cfg, seed, specs, mode):
    if mode == "tagged":
        table = tagged_table(cfg.vocab, cfg.hidden, seed)
        vis = [tagged_vis(i, s.n_vis, cfg.hidden, seed) for i, s in enumerate(specs)]
    elif mode == "bits":
        table = table_np(cfg, seed, mode="bits")
        vis = [visual_rows_np(cfg, seed, i, s.n_vis, mode="bits") for i, s in enumerate(specs)]
    else:
        table = table_np(cfg, seed)
        vis = [visual_rows_np(cfg, seed, i, s.n_vis) for i, s in enumerate(specs)]
    return table, vis


def _run_case(fp, cfg, seed, specs, mode="tagged", frame_shuffle_seed=0, check_pages=True):
    """Write specs into a GPU pool and the oracle pool, plan both, pack every
    microbatch on the GPU and compare everything with the oracle."""
    from paper_2606_23087_amd.harness import GpuWorkload
    say(f"case {cfg.name} seed={seed} mode={mode} H={cfg.hidden} P={cfg.page_tokens} "
        f"samples={len(specs)} shuffle={frame_shuffle_seed}")
    table, vis = _inputs(cfg, seed, specs, mode)
    w = GpuWorkload(cfg, seed, specs=specs, table=to_dev(table),
                    vis_fn=lambda i, s: to_dev(vis[i]) if s.n_vis else None,
                    frame_shuffle_seed=frame_shuffle_seed)
    try:
        opool, oids = oracle_pool_for(cfg, seed, specs, vis)
        if check_pages:
            for gid, oid in zip(w.ids, oids):
                assert fp.pool_sample_pages(w.pool, gid).tolist() == opool.sample_pages(oid)
        plan = w.plan()
        assign, tok, cst, mem = oracle_plan(cfg, specs)
        assert plan["assign"].tolist() == assign
        assert plan["mb_tokens"].tolist() == tok and plan["mb_cost_scaled"].tolist() == cst
        out, cu, pos = w.alloc_outputs(fill=0x3C3C)
        for j, idx in enumerate(mem):
            gids = [w.ids[i] for i in idx]
            n_tok, mx = w.pack(gids, out, cu, pos)
            torch.cuda.synchronize()
            want = opool.pack([oids[i] for i in idx], table)
            ref = definitional_pack([specs[i] for i in idx], [vis[i] for i in idx], table)
            assert np.array_equal(want[0], ref[0]) and np.array_equal(want[1], ref[1])
            assert n_tok == want[3] and mx == want[4]
            got = to_host(out[:n_tok])
            assert np.array_equal(got, want[0]), f"microbatch {j}: rows differ"
            assert np.array_equal(to_host(out[n_tok:]), np.full((out.shape[0] - n_tok, cfg.hidden), 0x3C3C,
                                                                dtype=np.uint16)), "rows past n_tokens touched"
            assert cu[:len(idx) + 1].cpu().numpy().tolist() == want[1].tolist()
            assert pos[:n_tok].cpu().numpy().tolist() == want[2].tolist()
            out.fill_(0x3C3C)
        return w, opool, oids, table, vis
    except Exception:
        w.close()
        raise


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("mode", ["tagged", "normal"])
def test_tiny_full_pipeline(fp, seed, mode):
    cfg = CONFIGS["tiny"]
    w, *_ = _run_case(fp, cfg, seed, gen_samples(cfg, seed), mode)
    w.close()


# Real hidden sizes, page sizes and sample shapes; fewer samples, small pools
# and a reduced vocabulary so the oracle finishes in seconds.
SMALL = {
    "qwen": dict(hbm_pages=600, vocab=3000, capacity=16384, n_mb=2, count=9),
    "frag70b": dict(hbm_pages=1200, vocab=3000, capacity=16384, n_mb=2, count=5, churn_steps=300),
    "video": dict(hbm_pages=400, vocab=3000, capacity=40000, n_mb=2, count=5),
    "tiered": dict(hbm_pages=150, host_pages=150, vocab=3000, capacity=12000, n_mb=2, count=6),
}


@pytest.mark.parametrize("name", list(SMALL))
@pytest.mark.parametrize("seed", [0, 1])
def test_small_configs(fp, name, seed):
    kw = dict(SMALL[name])
    count = kw.pop("count")
    cfg = scaled(CONFIGS[name], **kw)
    w, opool, oids, table, vis = _run_case(fp, cfg, seed, gen_samples(cfg, seed, count=count),
                                           "tagged" if seed == 0 else "bits")
    w.close()


def test_all_bit_patterns(fp):
    """Every one of the 65536 16-bit patterns (NaN payloads, signed zeros,
    denormals, infinities) is copied unchanged."""
    cfg = scaled(CONFIGS["tiny"], vocab=300, hbm_pages=512, capacity=5000, n_mb=1)
    specs = [SampleSpec(np.arange(10, 200, dtype=np.int32) % 300, np.array([7, 150], np.int32),
                        np.array([256, 300], np.int32))]
    say("case all-bit-patterns")
    table = np.arange(300 * 256, dtype=np.uint32).astype(np.uint16).reshape(300, 256)
    vis = [(np.arange(556 * 256, dtype=np.uint32) * 7 + 3).astype(np.uint16).reshape(556, 256)]
    allpat = np.zeros(1 << 16, bool)
    allpat[vis[0].ravel()] = True
    assert allpat.all()
    from paper_2606_23087_amd.harness import GpuWorkload
    w = GpuWorkload(cfg, 0, specs=specs, table=to_dev(table), vis_fn=lambda i, s: to_dev(vis[i]))
    out, cu, pos = w.alloc_outputs(rows=1000)
    n, _ = w.pack(w.ids, out, cu, pos)
    torch.cuda.synchronize()
    want = definitional_pack(specs, vis, table)
    assert np.array_equal(to_host(out[:n]), want[0])
    w.close()


def test_placement_independence(fp):
    """The same samples packed from pools whose physical frames are bound in
    different orders give identical bytes (Sec. 3.1 / Sec. 3.2: consumers
    read by GVA, unaware of physical placement)."""
    cfg = scaled(CONFIGS["qwen"], hbm_pages=600, vocab=3000, capacity=16384, n_mb=2)
    specs = gen_samples(cfg, 4, count=8)
    for shuffle in (0, 12345):
        w, *_ = _run_case(fp, cfg, 4, specs, "tagged", frame_shuffle_seed=shuffle)
        w.close()


def test_edge_cases(fp):
    """Degenerate samples and microbatches: text only, images only, empty
    images, images at position 0 and at the end, one-row samples, an empty
    microbatch, more than 256 samples in one microbatch, duplicated ids."""
    from paper_2606_23087_amd.harness import GpuWorkload
    say("case edge-cases")
    H = 3584
    cfg = scaled(CONFIGS["qwen"], hbm_pages=400, vocab=500, capacity=4000, n_mb=1)
    rng = np.random.default_rng(7)
    specs = [
        SampleSpec(np.array([5, 6, 7], np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32)),
        SampleSpec(np.zeros(0, np.int32), np.array([0, 0], np.int32), np.array([70, 1], np.int32)),
        SampleSpec(np.array([1, 2], np.int32), np.array([0, 1, 2, 2], np.int32), np.array([0, 64, 0, 65], np.int32)),
        SampleSpec(np.array([9], np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32)),
        SampleSpec(np.zeros(0, np.int32), np.array([0], np.int32), np.array([1], np.int32)),
    ]
    specs += [SampleSpec(rng.integers(0, 500, size=int(rng.integers(1, 4))).astype(np.int32),
                         np.zeros(0, np.int32), np.zeros(0, np.int32)) for _ in range(300)]
    table = tagged_table(500, H)
    vis = [tagged_vis(i, s.n_vis, H) for i, s in enumerate(specs)]
    w = GpuWorkload(cfg, 0, specs=specs, table=to_dev(table),
                    vis_fn=lambda i, s: to_dev(vis[i]) if s.n_vis else None)
    out, cu, pos = w.alloc_outputs(rows=2000, fill=0x1111)
    cu = torch.full((400,), -1, dtype=torch.int32, device="cuda")
    groups = [[0], [1], [2], [3], [4], [0, 1, 2, 3, 4], list(range(len(specs))), [2, 2, 0, 2], []]
    for g in groups:
        say(f"  edge group of {len(g)} samples")
        n, mx = w.pack([w.ids[i] for i in g], out, cu, pos)
        torch.cuda.synchronize()
        want = definitional_pack([specs[i] for i in g], [vis[i] for i in g], table)
        assert n == len(want[0]) and mx == want[3]
        assert np.array_equal(to_host(out[:n]), want[0])
        assert cu[:len(g) + 1].cpu().numpy().tolist() == want[1].tolist()
        assert pos[:n].cpu().numpy().tolist() == want[2].tolist()
        assert bool((out[n:] == 0x1111).all())
        out.fill_(0x1111)
    w.close()


def test_error_paths(fp):
    from paper_2606_23087_amd.harness import GpuWorkload
    say("case error-paths")
    cfg = scaled(CONFIGS["tiny"], hbm_pages=8, capacity=512, n_mb=2)
    specs = gen_samples(cfg, 0, count=1)
    w = GpuWorkload(cfg, 0, specs=specs, mode="tagged")
    pool = w.pool
    out, cu, pos = w.alloc_outputs()
    before = fp.pool_stats(pool)
    bad = [
        (dict(text_ids=[1, 2], img_pos=[3], img_ntok=[1]), "EINVAL"),
        (dict(text_ids=[1, 2], img_pos=[2, 1], img_ntok=[1, 1]), "EINVAL"),
        (dict(text_ids=[1000], img_pos=[], img_ntok=[]), "EINVAL"),
        (dict(text_ids=[], img_pos=[], img_ntok=[]), "EINVAL"),
        (dict(text_ids=[1], img_pos=[0], img_ntok=[8 * 16 + 1]), "ENOMEM"),
    ]
    for kw, code in bad:
        with pytest.raises(fp.FlowPoolError) as e:
            fp.pool_write_sample(pool, **kw)
        assert e.value.code == code
        assert fp.pool_stats(pool) == before
    with pytest.raises(ValueError):               # ordinary host memory never reaches a kernel
        fp.pool_write_sample(pool, [1], [0], [2], torch.zeros((2, cfg.hidden), dtype=torch.int16))
    assert fp.pool_stats(pool) == before
    sid = w.ids[0]
    n = specs[0].length
    with pytest.raises(ValueError):
        fp.pack_microbatch(pool, [sid], w.table, cfg.vocab, torch.empty((n, cfg.hidden), dtype=torch.int16), n)
    with pytest.raises(ValueError):               # a buffer smaller than the call says
        fp.pack_microbatch(pool, [sid], w.table, cfg.vocab, out[:n - 1], n)
    with pytest.raises(ValueError):
        fp.pack_microbatch(pool, [sid], w.table, cfg.vocab, out, n, cu, pos[:n - 1])
    with pytest.raises(ValueError):
        fp.pack_microbatch(pool, [sid], w.table[:cfg.vocab - 1], cfg.vocab, out, n)
    with pytest.raises(fp.FlowPoolError) as e:
        fp.pack_microbatch(pool, [sid], w.table, cfg.vocab, out, n - 1)
    assert e.value.code == "ECAPACITY"
    with pytest.raises(fp.FlowPoolError) as e:
        fp.pack_microbatch(pool, [sid], w.table, cfg.vocab, int(out.data_ptr()) + 2, n)
    assert e.value.code == "EALIGN"
    with pytest.raises(fp.FlowPoolError) as e:
        fp.pack_microbatch(pool, [sid], w.table, cfg.vocab - 1, out, n)
    assert e.value.code == "EINVAL"
    with pytest.raises(fp.FlowPoolError) as e:
        fp.plan_microbatches(pool, [sid, sid], 512, 2, 4096)
    assert e.value.code == "EINVAL"
    fp.pool_free_sample(pool, sid)
    for call in (lambda: fp.pool_free_sample(pool, sid),
                 lambda: fp.pack_microbatch(pool, [sid], w.table, cfg.vocab, out, 512),
                 lambda: fp.plan_microbatches(pool, [sid], 512, 2, 4096)):
        with pytest.raises(fp.FlowPoolError) as e:
            call()
        assert e.value.code == "ENOENT"
    w.close()


def test_write_from_pinned_host_memory(fp):
    """A producer may hand over its embeddings in pinned host memory (mapped
    into the GPU's address space): the write kernel reads them over PCIe and
    the pack is the same as from device memory."""
    say("case pinned-host producer buffer")
    H, P, vocab = 512, 16, 50
    specs = [SampleSpec(np.array([3, 4, 5], np.int32), np.array([1, 3], np.int32), np.array([40, 7], np.int32)),
             SampleSpec(np.zeros(0, np.int32), np.array([0], np.int32), np.array([33], np.int32))]
    table = tagged_table(vocab, H, 3)
    vis = [tagged_vis(i, s.n_vis, H, 3) for i, s in enumerate(specs)]
    pool = fp.pool_create(hidden=H, page_tokens=P, hbm_pages=16, vocab=vocab, alloc="scatter")
    try:
        ids = []
        for s, v in zip(specs, vis):
            hv = torch.from_numpy(v.view(np.int16)).pin_memory()
            ids.append(fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, hv))
            torch.cuda.synchronize()              # hv must outlive the write
        n = sum(s.length for s in specs)
        out = torch.full((n, H), 0x2222, dtype=torch.int16, device="cuda")
        cu = torch.empty((3,), dtype=torch.int32, device="cuda")
        pos = torch.empty((n,), dtype=torch.int32, device="cuda")
        m, _ = fp.pack_microbatch(pool, ids, to_dev(table), vocab, out, n, cu, pos)
        torch.cuda.synchronize()
        want = definitional_pack(specs, vis, table)
        assert m == n and np.array_equal(to_host(out), want[0])
        assert cu.cpu().numpy().tolist() == want[1].tolist() and pos.cpu().numpy().tolist() == want[2].tolist()
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)


def test_tier_mask_split(fp):
    """Host-tier rows read zero-copy over PCIe: a pack with the HBM mask and
    one with the host mask write together what one full pack writes."""
    from paper_2606_23087_amd.harness import GpuWorkload
    cfg = scaled(CONFIGS["tiered"], hbm_pages=150, host_pages=150, vocab=3000, capacity=12000, n_mb=2)
    specs = gen_samples(cfg, 3, count=6)
    w, opool, oids, table, vis = _run_case(fp, cfg, 3, specs, "tagged")
    say("case tier-mask-split")
    plan = w.plan()
    mbs = w.microbatches(plan)
    full, cu, pos = w.alloc_outputs(fill=0)
    part, cu2, pos2 = w.alloc_outputs(fill=0x2222)
    for j, g in enumerate(mbs):
        n, _ = w.pack(g, full, cu, pos)
        n2, _ = w.pack(g, part, cu2, pos2, tier_mask=fp.FP_TIER_MASK_HBM)
        torch.cuda.synchronize()
        gi = [w.ids.index(x) for x in g]
        want_hbm = opool.pack([oids[i] for i in gi], table, tier_mask=MASK_HBM,
                              out=np.full((n, cfg.hidden), 0x2222, np.uint16))
        assert np.array_equal(to_host(part[:n]), want_hbm[0])
        fp.pack_microbatch(w.pool, g, None, 0, part, part.shape[0], None, None, fp.FP_TIER_MASK_HOST)
        torch.cuda.synchronize()
        assert torch.equal(part[:n], full[:n]) and torch.equal(cu, cu2) and torch.equal(pos, pos2)
        part.fill_(0x2222)
    w.close()


def _runs(spec):
    """Maximal stretches of text rows or of image rows of one sample."""
    n, ti, in_image = 0, 0, False
    for p, t in zip(spec.img_pos.tolist(), spec.img_ntok.tolist()):
        if p > ti:
            n, ti, in_image = n + 1, p, False
        if t > 0 and not in_image:
            n, in_image = n + 1, True
    return n + (spec.n_text > ti)


def _head_specs(rng, n, max_img, vocab):
    """n samples of 1..29 text tokens; sample i has i % (max_img + 1) images of 0..40 rows each at
    random placeholder positions (some empty, some at 0 or at the end)."""
    specs = []
    for i in range(n):
        t = int(rng.integers(1, 30))           # a sample holds at least one row
        k = i % (max_img + 1)
        pos = np.sort(rng.integers(0, t + 1, size=k)).astype(np.int32)
        ntok = rng.integers(0, 41, size=k).astype(np.int32)
        specs.append(SampleSpec(rng.integers(0, vocab, size=t).astype(np.int32), pos, ntok))
    return specs


@pytest.mark.parametrize("pack_cus", [0, 1])
@pytest.mark.parametrize("hidden,page_tokens", [(8, 3), (16, 16), (64, 5), (96, 7), (128, 1),
                                                (256, 16), (3584, 64), (8192, 32)])
def test_chunk_head_shapes(fp, hidden, page_tokens, pack_cus):
    """Row resolution at every chunk shape: many rows per chunk (small H,
    one row per lane) down to chunks inside one row (large H); page sizes
    that are not powers of two; 17..32 samples with an inline run table,
    samples with eleven images, empty images and adjacent images (merged
    runs), the 32-sample and 160-run limits of the inline table and
    microbatches just past them (staged table), the 8-sample and 24-run
    limits of the compact kernel arguments and one past each, and 64 or
    more samples. pack_cus=1 sizes the chunk
    geometry for one compute unit, so these small packs also take full
    chunks and both shrinking tail stages; with the device's count they are
    all in the last stage."""
    from paper_2606_23087_amd.harness import GpuWorkload
    say(f"case chunk-head H={hidden} P={page_tokens} pack_cus={pack_cus}")
    vocab = 257
    rng = np.random.default_rng(hidden * 1000 + page_tokens)
    specs = _head_specs(rng, 70, 11, vocab) + _head_specs(rng, 70, 1, vocab)
    n_vis = sum(s.n_vis for s in specs)
    pages = sum(-(-s.n_vis // page_tokens) for s in specs) + 8
    cfg = scaled(CONFIGS["tiny"], hidden=hidden, page_tokens=page_tokens, hbm_pages=pages,
                 vocab=vocab, capacity=n_vis + 4000, n_mb=1)
    table = tagged_table(vocab, hidden)
    vis = [tagged_vis(i, s.n_vis, hidden) for i, s in enumerate(specs)]
    w = GpuWorkload(cfg, 0, specs=specs, table=to_dev(table),
                    vis_fn=lambda i, s: to_dev(vis[i]) if s.n_vis else None, pack_cus=pack_cus)
    try:
        total = sum(s.length for s in specs)
        out, cu, pos = w.alloc_outputs(rows=total + 64, fill=0x4545)
        cu = torch.full((150,), -1, dtype=torch.int32, device="cuda")
        runs = np.cumsum([_runs(s) for s in specs])
        r160 = int(np.searchsorted(runs, 160, side="right"))     # first r160 samples form <= 160 runs
        assert runs[r160 - 1] <= 160 < runs[r160] and r160 < 32
        assert runs[101] - runs[69] <= 160                         # samples 70..101 fit the inline table
        # the compact kernel arguments' limits (8 samples, 24 runs) and one past each
        rn = [_runs(s) for s in specs]
        at24 = next([i, j] for i in range(70) for j in range(i + 1, 70) if rn[i] + rn[j] == 24)
        at25 = next([i, j] for i in range(70) for j in range(i + 1, 70) if rn[i] + rn[j] == 25)
        assert sum(rn[i] for i in range(70, 78)) <= 24
        groups = [list(range(17)), list(range(r160)), list(range(r160 + 1)),
                  list(range(70, 102)), list(range(70, 103)), list(range(70, 134)), list(range(70)),
                  [11, 23, 11, 35, 140 - 1], list(range(70, 78)), list(range(70, 79)), at24, at25, [11]]
        for g in groups:
            say(f"  group of {len(g)} samples, {sum(_runs(specs[i]) for i in g)} runs")
            n, mx = w.pack([w.ids[i] for i in g], out, cu, pos)
            torch.cuda.synchronize()
            want = definitional_pack([specs[i] for i in g], [vis[i] for i in g], table)
            assert n == len(want[0]) and mx == want[3]
            assert np.array_equal(to_host(out[:n]), want[0])
            assert cu[:len(g) + 1].cpu().numpy().tolist() == want[1].tolist()
            assert pos[:n].cpu().numpy().tolist() == want[2].tolist()
            assert bool((out[n:] == 0x4545).all())
            out.fill_(0x4545)
    finally:
        w.close()


def test_zigzag_plan_then_pack(fp):
    """plan_microbatches with the zig-zag policy: the per-sample costs from
    the GPU cost kernel and the assignment equal the oracle's, and the
    microbatches pack bit-exactly."""
    from paper_2606_23087_amd.harness import GpuWorkload
    from oracle.plan import cost_scaled, members, zigzag_partition
    say("case zig-zag plan")
    cfg = scaled(CONFIGS["qwen"], hbm_pages=600, vocab=3000, capacity=6000, n_mb=3)
    specs = gen_samples(cfg, 2, count=9)
    table, vis = _inputs(cfg, 2, specs, "tagged")
    w = GpuWorkload(cfg, 2, specs=specs, table=to_dev(table), vis_fn=lambda i, s: to_dev(vis[i]) if s.n_vis else None)
    try:
        plan = fp.plan_microbatches(w.pool, w.ids, cfg.capacity, cfg.n_mb, cfg.cost_k, policy=fp.FP_PLAN_ZIGZAG)
        lengths = [s.length for s in specs]
        assign, tok, cst = zigzag_partition(lengths, cfg.cost_k, cfg.capacity, cfg.n_mb)
        assert plan["sample_cost_scaled"].tolist() == [cost_scaled(l, cfg.cost_k) for l in lengths]
        assert plan["assign"].tolist() == assign
        assert plan["mb_tokens"].tolist() == tok and plan["mb_cost_scaled"].tolist() == cst
        out, cu, pos = w.alloc_outputs()
        for j, idx in enumerate(members(assign, cfg.n_mb)):
            n, _ = w.pack([w.ids[i] for i in idx], out, cu, pos)
            torch.cuda.synchronize()
            want = definitional_pack([specs[i] for i in idx], [vis[i] for i in idx], table)
            assert n == len(want[0]) and np.array_equal(to_host(out[:n]), want[0]), f"microbatch {j}"
            assert cu[:len(idx) + 1].cpu().numpy().tolist() == want[1].tolist()
            assert pos[:n].cpu().numpy().tolist() == want[2].tolist()
        with pytest.raises(fp.FlowPoolError) as e:
            fp.plan_microbatches(w.pool, w.ids, cfg.capacity, cfg.n_mb, cfg.cost_k, policy=7)
        assert e.value.code == "EINVAL"
    finally:
        w.close()


def test_dynamic_packing_then_pack(fp):
    """Alg. 1 over resident samples (plan_pool_packing) gives the oracle's
    plan, and every microbatch it forms, packed in each rank's dispatch
    order, equals the definitional pack of its samples."""
    from oracle.schedule import dynamic_packing
    from paper_2606_23087_amd.harness import GpuWorkload
    cfg = scaled(CONFIGS["qwen"], hbm_pages=900, vocab=3000, capacity=16384, n_mb=2)
    specs = gen_samples(cfg, 5, count=14)
    say(f"case dynamic-packing samples={len(specs)}")
    table, vis = _inputs(cfg, 5, specs, "tagged")
    w = GpuWorkload(cfg, 5, specs=specs, table=to_dev(table),
                    vis_fn=lambda i, s: to_dev(vis[i]) if s.n_vis else None)
    try:
        L, N, K = 8192 + 2048, 3, 2
        keep = [i for i, s in enumerate(specs) if s.length <= L]
        got = fp.plan_pool_packing(w.pool, [w.ids[i] for i in keep], L, N, K)
        want = dynamic_packing([specs[i].length for i in keep], L, N, K)
        assert got["mb_of_seq"].tolist() == want["mb_of_seq"]
        for key in ("mb_tokens", "mb_max_len", "mb_cost_scaled", "mb_bucket", "mb_rank", "mb_slot"):
            assert got[key].tolist() == want[key], key
        out, cu, pos = w.alloc_outputs(rows=L, fill=0x3C3C)
        for rank in range(N):
            order = sorted((s, j) for j, (r, s) in enumerate(zip(want["mb_rank"], want["mb_slot"])) if r == rank)
            for _, j in order:
                idx = [keep[q] for q, m in enumerate(want["mb_of_seq"]) if m == j]
                n, mx = w.pack([w.ids[i] for i in idx], out, cu, pos)
                torch.cuda.synchronize()
                ref = definitional_pack([specs[i] for i in idx], [vis[i] for i in idx], table)
                assert n == want["mb_tokens"][j] == len(ref[0]) and mx == want["mb_max_len"][j]
                assert np.array_equal(to_host(out[:n]), ref[0])
                assert cu[:len(idx) + 1].cpu().numpy().tolist() == ref[1].tolist()
                assert pos[:n].cpu().numpy().tolist() == ref[2].tolist()
    finally:
        w.close()
