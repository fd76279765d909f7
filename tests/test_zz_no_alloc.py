"""pack_microbatch_noalloc, the pack entry point that allocates nothing,
against pack_microbatch (and the oracle's definitional pack), through the C
ABI: bit-exact rows, cu_seqlens and position ids, rows past the microbatch
untouched.

- two calls in a row on one stream, with no synchronisation between them,
  the second with fewer samples: both large enough for the run table to go
  through the device scratch, so the second overwrites the first's table
  there after the first pack has read it;
- a microbatch whose table travels in the kernel arguments (no scratch);
- the device's free memory is the same before and after the calls (once the
  stream has been used: the runtime sets up a stream's queue on its first
  launches).
"""

import numpy as np
import pytest

from gpu_common import say, to_dev, to_host
from oracle.pack import definitional_pack
from paper_2606_23087_amd.workloads import CONFIGS, gen_samples, scaled
from tagging import tagged_table, tagged_vis

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def _outs(rows, hidden, n):
    out = torch.full((rows, hidden), 0x5A5A, dtype=torch.int16, device="cuda")
    cu = torch.full((n + 1,), -1, dtype=torch.int32, device="cuda")
    pos = torch.full((rows,), -1, dtype=torch.int32, device="cuda")
    return out, cu, pos


def test_noalloc_pack_matches_pack(fp):
    cfg = scaled(CONFIGS["tiny"], hbm_pages=2000)
    seed = 5
    specs = gen_samples(cfg, seed, count=48)
    say(f"case no-alloc pack: H={cfg.hidden} P={cfg.page_tokens} samples={len(specs)}")
    pool = fp.pool_create(hidden=cfg.hidden, page_tokens=cfg.page_tokens, hbm_pages=cfg.hbm_pages,
                          vocab=cfg.vocab, alloc="scatter", pack_cus=2)
    try:
        table = tagged_table(cfg.vocab, cfg.hidden, seed)
        t_dev = to_dev(table)
        vis = [tagged_vis(i, s.n_vis, cfg.hidden, seed) for i, s in enumerate(specs)]
        ids = [fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, to_dev(v) if s.n_vis else None)
               for s, v in zip(specs, vis)]
        torch.cuda.synchronize()
        groups = [list(range(0, 44)), list(range(3, 40)), list(range(7, 12))]   # 44 and 37 samples: scratch; 5: arguments
        rows = [sum(specs[i].length for i in g) for g in groups]
        big = max(rows) + 16
        a = [_outs(big, cfg.hidden, len(g)) for g in groups]
        b = [_outs(big, cfg.hidden, len(g)) for g in groups]
        stream = torch.cuda.Stream()
        # The HIP runtime sets up a stream's queue on its first launches (its
        # kernel-argument pool among them): warm the stream up first, so the
        # check below sees only what the calls themselves allocate.
        warm = _outs(big, cfg.hidden, len(groups[0]))
        with torch.cuda.stream(stream):
            for g in groups:
                fp.pack_microbatch_noalloc(pool, [ids[i] for i in g], t_dev, cfg.vocab, warm[0], big, warm[1], warm[2],
                                           stream=stream)
        stream.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        with torch.cuda.stream(stream):
            got = [fp.pack_microbatch_noalloc(pool, [ids[i] for i in g], t_dev, cfg.vocab, o, big, c, p,
                                              stream=stream) for g, (o, c, p) in zip(groups, b)]
        stream.synchronize()
        free1 = torch.cuda.mem_get_info()[0]
        for g, (o, c, p) in zip(groups, a):
            fp.pack_microbatch(pool, [ids[i] for i in g], t_dev, cfg.vocab, o, big, c, p)
        torch.cuda.synchronize()
        for k, (g, n_rows) in enumerate(zip(groups, rows)):
            want = definitional_pack([specs[i] for i in g], [vis[i] for i in g], table)
            assert got[k] == (n_rows, want[3]), f"call {k}"
            (oa, ca, pa), (ob, cb, pb) = a[k], b[k]
            assert torch.equal(ob, oa) and torch.equal(cb, ca) and torch.equal(pb, pa), f"call {k}"
            assert np.array_equal(to_host(ob[:n_rows]), want[0]), f"call {k}"
            assert cb.cpu().numpy().tolist() == want[1].tolist() and pb[:n_rows].cpu().numpy().tolist() == want[2].tolist()
            assert bool((ob[n_rows:] == 0x5A5A).all()) and bool((pb[n_rows:] == -1).all())
        assert free1 == free0, f"device free memory changed by {free0 - free1} bytes"
        # the same two scratch-staged calls again, on the default stream
        for k in (0, 1):
            o, c, p = b[k]
            o.fill_(0x5A5A)
            fp.pack_microbatch_noalloc(pool, [ids[i] for i in groups[k]], t_dev, cfg.vocab, o, big, c, p)
        torch.cuda.synchronize()
        for k in (0, 1):
            assert torch.equal(b[k][0], a[k][0]), f"repeat {k}"
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)
