"""The page walk's two forms in one microbatch, against the oracle.

The image rows of a sample whose pages have consecutive GVAs are translated
from the page number of its first page (the GVA of page k is that of page 0
plus k pages), those of a sample with scattered pages through its page list;
both end in the page-table entry. A scattered pool is driven so that one
sample gets consecutive pages and another gets pages from two freed
samples (checked on the page lists), and a microbatch holding both is packed
at hidden sizes packed in 12 KiB chunks (where the first form is taken) and
in 8 KiB chunks (where every image row reads the page list), with frames
shuffled. Compared with the oracle pool's pack word for word.

Each case prints its shape before touching the GPU.
"""

import numpy as np
import pytest

from gpu_common import say, to_dev, to_host
from oracle.pool import OraclePool
from paper_2606_23087_amd.workloads import SampleSpec
from tagging import tagged_table, tagged_vis

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

MARK = 0x5A5A


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def _consecutive(gvas, page_bytes):
    return all(int(b) - int(a) == page_bytes for a, b in zip(gvas, gvas[1:]))


@pytest.mark.parametrize("hidden", [64, 1024, 3584, 5120])
def test_consecutive_and_scattered_pages_in_one_pack(fp, hidden):
    P, vocab = 8, 50
    say(f"case walk forms H={hidden} P={P}")
    pool = fp.pool_create(hidden=hidden, page_tokens=P, hbm_pages=64, vocab=vocab, alloc="scatter",
                          frame_shuffle_seed=11)
    opool = OraclePool(hidden, P, 64, 0, "scatter", vocab)
    table = tagged_table(vocab, hidden, 3)
    try:
        def spec(n_text, pos, ntok, seed):
            rng = np.random.default_rng(seed)
            return SampleSpec(rng.integers(0, vocab, size=n_text).astype(np.int32),
                              np.array(pos, np.int32), np.array(ntok, np.int32))

        gid, oid, specs = {}, {}, {}

        def write(name, s, index):
            v = tagged_vis(index, s.n_vis, hidden, 3)
            gid[name] = fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, to_dev(v) if s.n_vis else None)
            oid[name] = opool.write(s.text_ids, s.img_pos, s.img_ntok, v)
            specs[name] = s

        write("x", spec(5, [2], [32], 1), 0)           # pages 0-3
        write("y", spec(7, [0, 7], [10, 22], 2), 1)     # pages 4-7
        write("z", spec(3, [3], [32], 3), 2)            # pages 8-11
        for name in ("x", "z"):
            fp.pool_free_sample(pool, gid[name])
            opool.free(oid[name])
        write("b", spec(9, [4, 4, 9], [20, 24, 20], 4), 3)   # 8 pages from the two freed samples
        write("a", spec(6, [1, 6], [17, 23], 5), 4)          # 5 fresh pages
        torch.cuda.synchronize()
        pb = P * 2 * hidden
        pages = {k: fp.pool_sample_pages(pool, gid[k]).tolist() for k in ("a", "b", "y")}
        for k in pages:
            assert pages[k] == opool.sample_pages(oid[k])
        assert _consecutive(pages["a"], pb) and _consecutive(pages["y"], pb)
        assert not _consecutive(pages["b"], pb)
        order = ["a", "b", "y"]
        total = sum(specs[k].length for k in order)
        out = torch.full((total + 4, hidden), MARK, dtype=torch.int16, device="cuda")
        cu = torch.full((len(order) + 1,), -1, dtype=torch.int32, device="cuda")
        pos = torch.full((total + 4,), -1, dtype=torch.int32, device="cuda")
        n, mx = fp.pack_microbatch(pool, [gid[k] for k in order], to_dev(table), vocab, out, out.shape[0], cu, pos)
        torch.cuda.synchronize()
        rows, cu_o, pos_o, n_o, mx_o = opool.pack([oid[k] for k in order], table)
        assert (n, mx) == (n_o, mx_o) == (total, max(specs[k].length for k in order))
        assert np.array_equal(to_host(out[:n]), rows)
        assert bool((out[n:] == MARK).all())
        assert cu.cpu().numpy().tolist() == cu_o.tolist() and pos[:n].cpu().numpy().tolist() == pos_o.tolist()
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)
