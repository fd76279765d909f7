"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (same pool, same pack entry point, a non-default stream,
rotating output buffers).

Every sample the plan places is also written, with the same bytes and after
the same churn history, into the oracle pool (its visual rows and the table
rows its text names are copied from the seeded generators to the host); then
for every microbatch:
- the plan (assignment, tokens, cost per microbatch) equals the oracle's;
- every sample's page GVAs equal the oracle pool's;
- cu_seqlens and position ids equal the oracle's, in full;
- the tag words of every packed row name exactly the source the oracle's
  layout gives (sample, visual index or text id);
- every word of every row equals the oracle pool's pack, which resolves each
  row through its own page table.
"""

import numpy as np
import pytest

from gpu_common import oracle_plan, oracle_pool_for, say, to_host
from oracle.pack import row_sources
from paper_2606_23087_amd.workloads import CONFIGS, TAG_TEXT, TAG_VIS

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def _expected_tags(idx, specs_mb):
    src = row_sources(specs_mb)
    tags = np.zeros((len(src), 4), np.uint16)
    pos = np.zeros(len(src), np.int32)
    last, count = -1, 0
    for r, (kind, s, x) in enumerate(src):
        count = count + 1 if s == last else 0
        last = s
        pos[r] = count
        if kind == "text":
            tags[r] = (TAG_TEXT, x & 0xFFFF, x >> 16, 0)
        else:
            g = idx[s]
            tags[r] = (TAG_VIS, g & 0xFFFF, g >> 16, x & 0xFFFF)
    return src, tags, pos


@pytest.mark.parametrize("name", ["qwen", "frag70b", "video", "tiered"])
def test_full_size(fp, name):
    from paper_2606_23087_amd.harness import GpuWorkload, vis_rows
    cfg = CONFIGS[name]
    seed = 0
    say(f"full-size {name}: H={cfg.hidden} P={cfg.page_tokens} C={cfg.capacity} M={cfg.n_mb}")
    w = GpuWorkload(cfg, seed, mode="tagged", log=say)
    try:
        assign, tok, cst, mem = oracle_plan(cfg, w.specs)
        members = {i for m in mem for i in m}            # every planned sample
        say(f"  {len(w.ids)} samples written; replaying in the oracle pool with the rows of the "
            f"{len(members)} planned samples")
        vis_np = [to_host(vis_rows(cfg, seed, i, s.n_vis, "tagged")) if i in members and s.n_vis else None
                  for i, s in enumerate(w.specs)]
        opool, oids = oracle_pool_for(cfg, seed, w.specs, vis_np, with_bytes=True)
        del vis_np
        for gid, oid in zip(w.ids, oids):
            assert fp.pool_sample_pages(w.pool, gid).tolist() == opool.sample_pages(oid)
        text_ids = np.unique(np.concatenate([w.specs[i].text_ids for i in members] + [np.zeros(0, np.int32)]))
        host_table = np.zeros((cfg.vocab, cfg.hidden), np.uint16)     # only the named rows are filled
        if text_ids.size:
            host_table[text_ids] = to_host(w.table[torch.from_numpy(text_ids.astype(np.int64)).cuda()])
        plan = w.plan()
        assert plan["assign"].tolist() == assign
        assert plan["mb_tokens"].tolist() == tok and plan["mb_cost_scaled"].tolist() == cst
        mbs = w.microbatches(plan)
        assert mbs == [[w.ids[i] for i in m] for m in mem]
        stream = torch.cuda.Stream()
        outs = [w.alloc_outputs() for _ in range(4)]
        for j, idx in enumerate(mem):
            out, cu, pos = outs[j % 4]
            n, mx = w.pack([w.ids[i] for i in idx], out, cu, pos, stream=stream)
            stream.synchronize()
            specs_mb = [w.specs[i] for i in idx]
            src, tags, pos_want = _expected_tags(idx, specs_mb)
            lens = [s.length for s in specs_mb]
            assert n == len(src) == sum(lens) and mx == max(lens)
            assert cu[:len(idx) + 1].cpu().numpy().tolist() == [0] + np.cumsum(lens).tolist()
            assert np.array_equal(pos[:n].cpu().numpy(), pos_want)
            got_tags = to_host(out[:n, :4])
            bad = np.nonzero(np.any(got_tags != tags, axis=1))[0]
            assert bad.size == 0, f"microbatch {j}: {bad.size} rows with wrong source, first {bad[:5]}"
            rows_o, cu_o, pos_o, n_o, mx_o = opool.pack([oids[i] for i in idx], host_table)
            assert (n_o, mx_o) == (n, mx)
            got = to_host(out[:n])
            bad = np.nonzero(np.any(got != rows_o, axis=1))[0]
            assert bad.size == 0, f"microbatch {j}: {bad.size} of {n} rows differ from the oracle, first {bad[:5]}"
            assert cu[:len(idx) + 1].cpu().numpy().tolist() == cu_o.tolist()
            assert np.array_equal(pos[:n].cpu().numpy(), pos_o)
            del got, rows_o
        say(f"  {len(mem)} microbatches checked: every word equals the oracle pool's pack")
        if cfg.host_pages:
            say("  tier-mask split at full size")
            full, cu, pos = w.alloc_outputs(fill=0)
            part, cu2, pos2 = w.alloc_outputs(fill=0x2222)
            for g in mbs[:4]:
                n, _ = w.pack(g, full, cu, pos, stream=stream)
                w.pack(g, part, cu2, pos2, tier_mask=fp.FP_TIER_MASK_HBM, stream=stream)
                w.pack(g, part, None, None, tier_mask=fp.FP_TIER_MASK_HOST, stream=stream)
                stream.synchronize()
                assert torch.equal(part[:n], full[:n]) and torch.equal(cu, cu2) and torch.equal(pos, pos2)
    finally:
        w.close()
        torch.cuda.empty_cache()
