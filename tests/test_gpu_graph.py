"""HIP graph capture of packs: a captured step of pack_microbatch calls,
replayed several times with eager work and host synchronisation between
the replays, gives the eager result every time (bit-exact); calls that
cannot be captured refuse with ESTATE and leave the capture usable."""

import numpy as np
import pytest

from gpu_common import say, to_dev
from paper_2606_23087_amd.workloads import CONFIGS, gen_samples, scaled

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def test_captured_packs_replay_exactly(fp):
    from paper_2606_23087_amd.harness import GpuWorkload
    say("case graph capture of packs")
    cfg = scaled(CONFIGS["qwen"], hbm_pages=600, vocab=3000, capacity=16384, n_mb=3)
    w = GpuWorkload(cfg, 2, specs=gen_samples(cfg, 2, count=9), mode="tagged")
    try:
        mbs = w.microbatches(w.plan())
        eager = [w.alloc_outputs(fill=0x1111) for _ in mbs]
        for mb, (o, c, p) in zip(mbs, eager):
            w.pack(mb, o, c, p)
        torch.cuda.synchronize()
        outs = [w.alloc_outputs(fill=0x2222) for _ in mbs]
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            with torch.cuda.graph(g, stream=side):
                for mb, (o, c, p) in zip(mbs, outs):
                    w.pack(mb, o, c, p)
        torch.cuda.synchronize()
        for rep in range(3):
            for o, c, p in outs:                   # eager work between replays: refill as allocated
                o.fill_(0x1111)
                c.fill_(-1)
                p.fill_(-1)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for (o, c, p), (eo, ec, ep) in zip(outs, eager):
                assert torch.equal(o, eo) and torch.equal(c, ec) and torch.equal(p, ep), f"replay {rep}"
        del g
    finally:
        torch.cuda.synchronize()
        w.close()


@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")     # the refused capture records nothing
def test_uncapturable_calls_refuse(fp):
    from paper_2606_23087_amd.harness import GpuWorkload
    say("case graph capture refusals")
    cfg = scaled(CONFIGS["tiny"], hbm_pages=400, capacity=20000, n_mb=1)
    w = GpuWorkload(cfg, 0, specs=gen_samples(cfg, 0, count=70), mode="tagged")
    try:
        torch.cuda.synchronize()
        fp.pool_reclaim(w.pool, True)                 # every write is now known complete
        out, cu, pos = w.alloc_outputs(rows=20000)
        spec = w.specs[0]
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        errors = []
        with torch.cuda.stream(side):
            with torch.cuda.graph(g, stream=side):
                for call in (lambda: w.pack(w.ids, out, cu, pos),                 # 70 samples: staged headers
                             lambda: w.plan(),
                             lambda: fp.pool_write_sample(w.pool, spec.text_ids, spec.img_pos, spec.img_ntok)):
                    try:
                        call()
                    except fp.FlowPoolError as e:
                        errors.append(e.code)
                w.pack(w.ids[:5], out, cu, pos)                                   # still capturable
        assert errors == ["ESTATE", "ESTATE", "ESTATE"]
        # a sample whose write has not been seen complete cannot be captured
        sid = fp.pool_write_sample(w.pool, spec.text_ids, spec.img_pos, spec.img_ntok)
        torch.cuda.synchronize()
        g2 = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            with torch.cuda.graph(g2, stream=side):
                with pytest.raises(fp.FlowPoolError, match="ESTATE"):
                    w.pack([sid], out, cu, pos)
        del g2
        out.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        ref, rc, rp = w.alloc_outputs(rows=20000, fill=0)
        w.pack(w.ids[:5], ref, rc, rp)
        torch.cuda.synchronize()
        assert torch.equal(out, ref)
        del g
    finally:
        torch.cuda.synchronize()
        w.close()


def test_captured_samples_are_held(fp):
    """A captured pack holds its samples: freeing or migrating one returns
    ESTATE (its page list stays where the graph reads it), replays still
    give the eager result, and after pool_release_captured the samples move
    and free as usual (the graph is not replayed after that)."""
    from paper_2606_23087_amd.harness import GpuWorkload
    say("case captured samples are held")
    cfg = scaled(CONFIGS["tiered"], hbm_pages=400, host_pages=400, vocab=3000, capacity=16384, n_mb=1)
    w = GpuWorkload(cfg, 4, specs=gen_samples(cfg, 4, count=3), mode="tagged")
    try:
        torch.cuda.synchronize()
        fp.pool_reclaim(w.pool, True)
        ids = list(w.ids)
        eager, ec, ep = w.alloc_outputs(fill=0x2222)
        w.pack(ids, eager, ec, ep)
        torch.cuda.synchronize()
        out, cu, pos = w.alloc_outputs(fill=0x2222)
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            with torch.cuda.graph(g, stream=side):
                w.pack(ids, out, cu, pos)
        torch.cuda.synchronize()
        pages_before = [fp.pool_sample_pages(w.pool, s).tolist() for s in ids]
        with pytest.raises(fp.FlowPoolError, match="ESTATE"):
            fp.pool_migrate(w.pool, [ids[0]], fp.FP_TIER_HBM)
        with pytest.raises(fp.FlowPoolError, match="ESTATE"):
            fp.pool_free_sample(w.pool, ids[1])
        assert [fp.pool_sample_pages(w.pool, s).tolist() for s in ids] == pages_before
        for rep in range(2):
            out.fill_(0x2222)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(out, eager) and torch.equal(cu, ec) and torch.equal(pos, ep), f"replay {rep}"
        del g
        with pytest.raises(fp.FlowPoolError, match="EINVAL"):
            fp.pool_release_captured(w.pool, ids + ids)        # each was captured once
        with pytest.raises(fp.FlowPoolError, match="ENOENT"):
            fp.pool_release_captured(w.pool, [10 ** 9])
        fp.pool_release_captured(w.pool, ids[::-1])
        with pytest.raises(fp.FlowPoolError, match="EINVAL"):
            fp.pool_release_captured(w.pool, ids[:1])          # already released
        moved = fp.pool_migrate(w.pool, ids, fp.FP_TIER_HBM)
        assert moved > 0
        torch.cuda.synchronize()
        again, ac, ap = w.alloc_outputs(fill=0x2222)
        w.pack(ids, again, ac, ap)
        torch.cuda.synchronize()
        assert torch.equal(again, eager)
        fp.pool_free_sample(w.pool, ids[1])
    finally:
        torch.cuda.synchronize()
        w.close()
