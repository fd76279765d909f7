"""Producer and consumer on two streams of one GPU (Sec. 3.1: encoders write
embeddings into the pool while the backbone's packs read it, decoupled).

- A free while a pack of the sample is still queued is deferred: the
  sample's pages are not handed to a new write until the pack has run, so
  the pack reads the freed sample's bytes, not the new ones.
- A pack on another stream than the sample's write waits for that write.
- A producer thread writing and freeing on one stream and a consumer packing
  on another: every pack equals the definitional pack of its samples.
- A stream handed to pool_forget_stream can be destroyed while the samples it
  packed stay resident; their frees then never touch it.

The delays that keep a pack or a write queued come from ordinary copies
enqueued ahead of it on the same stream.
Bar: bit-exact (raw 16-bit copies).
"""

import threading

import numpy as np
import pytest

from gpu_common import say, to_dev, to_host
from oracle.pack import definitional_pack
from paper_2606_23087_amd.workloads import SampleSpec
from tagging import tagged_table, tagged_vis

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


def _busy(stream, ms_hint=20):
    """Queue about ``ms_hint`` ms of plain copies on ``stream``."""
    a = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    with torch.cuda.stream(stream):
        for _ in range(ms_hint * 50):
            b.copy_(a)
    return a, b


def _spec(rng, vocab, n_text, imgs):
    pos = np.sort(rng.integers(0, n_text + 1, size=len(imgs))).astype(np.int32)
    return SampleSpec(rng.integers(0, vocab, size=n_text).astype(np.int32), pos, np.array(imgs, np.int32))


H, P, VOCAB = 512, 16, 97


def _pool(fp, pages):
    return fp.pool_create(hidden=H, page_tokens=P, hbm_pages=pages, vocab=VOCAB, alloc="contig")


def test_free_while_pack_queued_is_deferred(fp):
    say("case deferred-free")
    rng = np.random.default_rng(1)
    table = tagged_table(VOCAB, H, 1)
    t_dev = to_dev(table)
    x = _spec(rng, VOCAB, 40, [3 * P, P + 5])
    y = _spec(rng, VOCAB, 40, [3 * P, P + 5])
    vx, vy = tagged_vis(0, x.n_vis, H, 1), tagged_vis(1, y.n_vis, H, 1)
    pages = -(-x.n_vis // P)
    pool = _pool(fp, pages)                      # room for exactly one of them
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    try:
        dx, dy = to_dev(vx), to_dev(vy)
        torch.cuda.synchronize()
        idx = fp.pool_write_sample(pool, x.text_ids, x.img_pos, x.img_ntok, dx, stream=sa)
        torch.cuda.synchronize()
        out = torch.full((x.length, H), 0x1234, dtype=torch.int16, device="cuda")
        keep = _busy(sb)
        fp.pack_microbatch(pool, [idx], t_dev, VOCAB, out, x.length, stream=sb)
        fp.pool_free_sample(pool, idx)
        assert fp.pool_reclaim(pool) == pages, "the free should wait for the queued pack"
        # Y needs X's pages: the write waits for the pack before taking them.
        idy = fp.pool_write_sample(pool, y.text_ids, y.img_pos, y.img_ntok, dy, stream=sa)
        torch.cuda.synchronize()
        assert fp.pool_reclaim(pool) == 0
        assert np.array_equal(to_host(out), definitional_pack([x], [vx], table)[0])
        out2 = torch.empty((y.length, H), dtype=torch.int16, device="cuda")
        fp.pack_microbatch(pool, [idy], t_dev, VOCAB, out2, y.length, stream=sb)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(out2), definitional_pack([y], [vy], table)[0])
        del keep
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)


def test_pack_waits_for_write_on_other_stream(fp):
    say("case cross-stream write then pack")
    rng = np.random.default_rng(2)
    table = tagged_table(VOCAB, H, 2)
    t_dev = to_dev(table)
    specs = [_spec(rng, VOCAB, 30, [2 * P + 3]), _spec(rng, VOCAB, 10, [P, 7])]
    vis = [tagged_vis(i, s.n_vis, H, 2) for i, s in enumerate(specs)]
    pool = _pool(fp, 64)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    try:
        dev = [to_dev(v) for v in vis]
        torch.cuda.synchronize()
        keep = _busy(sa)
        ids = [fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, d, stream=sa)
               for s, d in zip(specs, dev)]
        n = sum(s.length for s in specs)
        out = torch.full((n, H), 0x1234, dtype=torch.int16, device="cuda")
        cu = torch.full((3,), -1, dtype=torch.int32, device="cuda")
        pos = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        fp.pack_microbatch(pool, ids, t_dev, VOCAB, out, n, cu, pos, stream=sb)
        plan = fp.plan_microbatches(pool, ids, 4096, 1, 4096, stream=sb)
        assert plan["mb_tokens"].tolist() == [n]
        assert plan["sample_cost_scaled"].tolist() == [4096 * s.length + s.length ** 2 for s in specs]
        torch.cuda.synchronize()
        want = definitional_pack(specs, vis, table)
        assert np.array_equal(to_host(out), want[0])
        assert cu.cpu().numpy().tolist() == want[1].tolist()
        assert pos.cpu().numpy().tolist() == want[2].tolist()
        del keep
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)


def test_producer_and_consumer_threads(fp):
    """A producer thread keeps writing samples (stream A) and freeing old ones;
    the consumer packs groups of resident samples (stream B) into fresh
    buffers. Every pack is checked after both finish."""
    say("case producer/consumer threads")
    rng = np.random.default_rng(3)
    table = tagged_table(VOCAB, H, 3)
    t_dev = to_dev(table)
    pool = _pool(fp, 400)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    lock = threading.Lock()
    resident = {}            # id -> (spec, host rows, device rows)
    done = threading.Event()
    errors = []
    n_writes = 150

    def producer():
        prng = np.random.default_rng(30)
        try:
            for i in range(n_writes):
                s = _spec(prng, VOCAB, int(prng.integers(1, 40)),
                          [int(x) for x in prng.integers(0, 3 * P, size=int(prng.integers(0, 3)))])
                v = tagged_vis(i, s.n_vis, H, 3)
                with torch.cuda.stream(sa):      # the upload is ordered before the write
                    d = to_dev(v) if s.n_vis else None
                    sid = fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, d, stream=sa)
                with lock:
                    resident[sid] = (s, v, d)
                    if len(resident) > 12:
                        old = min(resident)
                        fp.pool_free_sample(pool, old)
                        resident.pop(old)
        except Exception as e:  # surfaced by the main thread
            errors.append(e)
        finally:
            done.set()

    t = threading.Thread(target=producer)
    t.start()
    packs = []
    try:
        while not done.is_set() or len(packs) < 20:
            with lock:
                ids = sorted(resident)
                if not ids:
                    continue
                pick = [ids[int(j)] for j in rng.integers(0, len(ids), size=int(rng.integers(1, 5)))]
                items = [resident[i][:2] for i in pick]
                n = sum(sp.length for sp, _ in items)
                out = torch.empty((n, H), dtype=torch.int16, device="cuda")
                fp.pack_microbatch(pool, pick, t_dev, VOCAB, out, n, stream=sb)
            packs.append((items, out))
            if len(packs) >= 400:
                break
        t.join()
        torch.cuda.synchronize()
        assert not errors, errors
        say(f"  {len(packs)} packs checked")
        for items, out in packs:
            want = definitional_pack([sp for sp, _ in items], [v for _, v in items], table)
            assert np.array_equal(to_host(out), want[0])
    finally:
        t.join()
        torch.cuda.synchronize()
        fp.pool_destroy(pool)


def test_two_producers_and_a_planning_consumer(fp):
    """Two producer threads, each on its own stream, write and free samples
    while the consumer plans (zig-zag policy) and packs resident samples on a
    third stream: the pool's lock serialises the calls and its events order
    the streams. Every pack is checked after all threads finish, and all
    pages come back at the end."""
    say("case two producers, planning consumer")
    rng = np.random.default_rng(4)
    table = tagged_table(VOCAB, H, 4)
    t_dev = to_dev(table)
    pool = _pool(fp, 400)
    streams = [torch.cuda.Stream() for _ in range(3)]
    lock = threading.Lock()
    resident = {}            # id -> (spec, host rows, device rows)
    done = [threading.Event(), threading.Event()]
    errors = []

    def producer(k):
        prng = np.random.default_rng(40 + k)
        st = streams[k]
        try:
            for i in range(100):
                s = _spec(prng, VOCAB, int(prng.integers(1, 40)),
                          [int(x) for x in prng.integers(0, 3 * P, size=int(prng.integers(0, 3)))])
                v = tagged_vis(1000 * k + i, s.n_vis, H, 4)
                with torch.cuda.stream(st):
                    d = to_dev(v) if s.n_vis else None
                    sid = fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, d, stream=st)
                with lock:
                    resident[sid] = (s, v, d, k)
                    mine = sorted(x for x, r in resident.items() if r[3] == k)
                    if len(mine) > 8:
                        fp.pool_free_sample(pool, mine[0])
                        resident.pop(mine[0])
        except Exception as e:  # surfaced by the main thread
            errors.append(e)
        finally:
            done[k].set()

    threads = [threading.Thread(target=producer, args=(k,)) for k in range(2)]
    for t in threads:
        t.start()
    packs = []
    try:
        while not all(d.is_set() for d in done) or len(packs) < 20:
            with lock:
                ids = sorted(resident)
                if len(ids) < 2:
                    continue
                plan = fp.plan_microbatches(pool, ids, 200, 2, 64, stream=streams[2], policy=fp.FP_PLAN_ZIGZAG)
                pick = [ids[i] for i in range(len(ids)) if plan["assign"][i] == 0][:6]
                if not pick:
                    continue
                items = [resident[i][:2] for i in pick]
                n = sum(sp.length for sp, _ in items)
                out = torch.empty((n, H), dtype=torch.int16, device="cuda")
                fp.pack_microbatch(pool, pick, t_dev, VOCAB, out, n, stream=streams[2])
            packs.append((items, out))
            if len(packs) >= 300:
                break
        for t in threads:
            t.join()
        torch.cuda.synchronize()
        assert not errors, errors
        say(f"  {len(packs)} packs checked")
        for items, out in packs:
            want = definitional_pack([sp for sp, _ in items], [v for _, v in items], table)
            assert np.array_equal(to_host(out), want[0])
        for sid in list(resident):
            fp.pool_free_sample(pool, sid)
        torch.cuda.synchronize()
        assert fp.pool_reclaim(pool, True) == 0 and fp.pool_stats(pool)["n_samples"] == 0
    finally:
        for t in threads:
            t.join()
        torch.cuda.synchronize()
        fp.pool_destroy(pool)


def test_forget_stream_then_destroy(fp):
    """A stream handed to pool_forget_stream may be destroyed while samples it
    packed stay resident: later frees wait for the event that stood in for
    it (or for nothing, if it was idle) and never touch the dead handle."""
    import ctypes
    import os
    hip = ctypes.CDLL(os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so"))
    hip.hipStreamCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    hip.hipStreamSynchronize.argtypes = [ctypes.c_void_p]
    say("case forget a stream, then destroy it")
    rng = np.random.default_rng(31)
    specs = [_spec(rng, VOCAB, int(rng.integers(5, 40)), [int(x) for x in rng.integers(1, 60, size=2)])
             for _ in range(12)]
    vis = [tagged_vis(i, s.n_vis, H, 31) for i, s in enumerate(specs)]
    table = tagged_table(VOCAB, H, 31)
    t_dev = to_dev(table)
    pool = _pool(fp, 400)
    try:
        ids = [fp.pool_write_sample(pool, s.text_ids, s.img_pos, s.img_ntok, to_dev(v)) for s, v in zip(specs, vis)]
        torch.cuda.synchronize()
        free0 = fp.pool_stats(pool)["free_hbm_pages"]
        rows = sum(s.length for s in specs)
        for case in ("busy", "idle"):
            raw = ctypes.c_void_p()
            assert hip.hipStreamCreate(ctypes.byref(raw)) == 0
            outs = [torch.full((rows, H), 0x5A5A, dtype=torch.int16, device="cuda") for _ in range(2)]
            keep = _busy(torch.cuda.ExternalStream(raw.value), 10) if case == "busy" else None
            fp.pack_microbatch(pool, ids[:6], t_dev, VOCAB, outs[0], rows, None, None, stream=raw.value)
            fp.pack_microbatch(pool, ids[6:], t_dev, VOCAB, outs[1], rows, None, None, stream=raw.value)
            if case == "idle":
                assert hip.hipStreamSynchronize(raw.value) == 0
            fp.pool_forget_stream(pool, raw.value)
            assert hip.hipStreamSynchronize(raw.value) == 0
            assert hip.hipStreamDestroy(raw.value) == 0
            del keep
            for k, g in enumerate((ids[:6], ids[6:])):
                want = definitional_pack([specs[ids.index(x)] for x in g], [vis[ids.index(x)] for x in g], table)[0]
                assert np.array_equal(to_host(outs[k][:len(want)]), want), (case, k)
            if case == "busy":
                continue                       # the samples stay; the idle case packs them again, then frees
            for sid in ids:
                fp.pool_free_sample(pool, sid)
        assert fp.pool_reclaim(pool, True) == 0
        assert fp.pool_stats(pool) == {"free_hbm_pages": free0 + sum(-(-s.n_vis // P) for s in specs),
                                       "free_host_pages": 0, "n_samples": 0}
    finally:
        torch.cuda.synchronize()
        fp.pool_destroy(pool)
