#!/usr/bin/env python3
"""Benchmark of the paged translate-gather-pack on one MI355X.

One step = one pass of the whole hot path over the resident samples of one
workload: the planner (GPU cost kernel + greedy partition into M
microbatches) followed by pack_microbatch of every microbatch (prefix sum,
page walk, visual-row gather, text-table gather, position ids).

Prints ONE JSON line. ``value`` is the whole-step effective bandwidth:
algorithmic bytes of all packs / wall time of the timed steps (inputs already
resident in HBM, planning included). ``roofline`` is for the pack kernel:
algorithmic bytes per launch / mean launch duration, the duration being one
HIP event pair on the pack stream around all pack launches of the timed steps
divided by their number (back-to-back launches, inter-kernel gaps included).
Per-call event pairs are taken in a separate untimed step: recording events
between launches perturbs the stream they time. ``cpu_baseline`` times the CPU
oracle's pool pack on a bounded sample of the same microbatches.

Algorithmic bytes of one pack (each valid row read once and written once):
  2*n_tokens*row_bytes + 4*n_text (ids) + 16*pages (GVA + PTE)
  + 4*n_tokens (position ids) + 4*(n+1) (cu_seqlens) + 48*n (descriptors)
  + 8*images (placeholder pairs)
"""

from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import platform
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E peak
PCIE_PEAK_GBPS = 63.0           # PCIe Gen5 x16, one direction

METRIC = "pack_microbatch effective GB/s and % of HBM peak (hidden 3584 bf16)"


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def seconds_since_start() -> float:
    """Wall seconds since this process started."""
    try:
        import psutil
        return max(0.0, time.time() - psutil.Process().create_time())
    except Exception:                    # no psutil: since this module was loaded
        return time.perf_counter() - _T_LOADED


_T_LOADED = time.perf_counter()


def cpu_model_name() -> str:
    """The host CPU's model string (from /proc/cpuinfo where there is one)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def masked_pack_bytes(cfg, w, mb, spec_of, mask: int) -> int:
    """Algorithmic bytes of a tier-masked pack: the rows it copies, read once
    and written once, plus (HBM mask) the metadata a full pack moves."""
    from paper_2606_23087_amd import flowpool as fp
    specs = [spec_of[x] for x in mb]
    if mask == fp.FP_TIER_MASK_ALL:
        return pack_bytes(cfg, specs)
    _, tier = row_sources(cfg, w, mb, spec_of, tiers=True)
    rows = int((tier == (1 if mask == fp.FP_TIER_MASK_HOST else 0)).sum())
    meta = pack_bytes(cfg, specs) - 2 * sum(x.length for x in specs) * cfg.row_bytes
    return 2 * rows * cfg.row_bytes + (meta if mask & fp.FP_TIER_MASK_HBM else 0)


def pack_bytes(cfg, specs) -> int:
    rb = cfg.row_bytes
    tokens = sum(s.length for s in specs)
    n_text = sum(s.n_text for s in specs)
    pages = sum(-(-s.n_vis // cfg.page_tokens) for s in specs)
    images = sum(len(s.img_ntok) for s in specs)
    n = len(specs)
    return 2 * tokens * rb + 4 * n_text + 16 * pages + 4 * tokens + 4 * (n + 1) + 48 * n + 8 * images


def kernel_source_hash() -> str:
    """Hash of the kernel sources (kernels.hip and the launch-layout header
    fp_internal.h) with comments and whitespace removed, and of the hipcc
    flags they are built with, so that only a change to the code or its
    compilation invalidates recorded counters."""
    from paper_2606_23087_amd.build import HIPCC_FLAGS
    src = ""
    for name in ("kernels.hip", "fp_internal.h"):
        src += open(os.path.join(ROOT, "paper_2606_23087_amd", "csrc", name)).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    src = re.sub(r"\s+", "", src)
    src += " ".join(HIPCC_FLAGS)
    return hashlib.sha256(src.encode()).hexdigest()[:16]


def counter_traffic(workload: str, mask: str = "all"):
    """HBM bytes per pack launch from the committed rocprofv3 counter summary
    of the workload (and tier mask), if it was taken on the current kernel
    source; else None."""
    name = workload if mask == "all" else f"{workload}_{mask}"
    path = os.path.join(ROOT, "profiles", f"pack_{name}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_sha256:\s*([0-9a-f]+)", text)
    t = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m or not t or m.group(1) != kernel_source_hash():
        return None
    return float(t.group(1))


def cpu_baseline(cfg, w, mbs, seed: int, budget_s: float):
    """Time the oracle's pool pack on the samples of the first microbatches."""
    import numpy as np
    import torch

    from oracle.pool import OraclePool
    from paper_2606_23087_amd.harness import vis_rows
    from paper_2606_23087_amd.workloads import page_tier_draws

    take = [mb for mb in mbs if mb][:2]
    index = {sid: i for i, sid in enumerate(w.ids)}
    pool = OraclePool(cfg.hidden, cfg.page_tokens, cfg.hbm_pages, cfg.host_pages, cfg.alloc, cfg.vocab)
    table = w.table.cpu().view(torch.int16).numpy().view(np.uint16)
    oid = {}
    for mb in take:
        for sid in mb:
            i = index[sid]
            s = w.specs[i]
            rows = vis_rows(cfg, seed, i, s.n_vis, "normal").cpu().view(torch.int16).numpy().view(np.uint16) \
                if s.n_vis else np.zeros((0, cfg.hidden), np.uint16)
            wish = page_tier_draws(seed, i, -(-s.n_vis // cfg.page_tokens)) if cfg.tier_split else None
            oid[sid] = pool.write(s.text_ids, s.img_pos, s.img_ntok, rows, tier_wish=wish)
    total_bytes = 0
    t0 = time.perf_counter()
    packs = 0
    while True:
        for mb in take:
            pool.pack([oid[s] for s in mb], table)
            total_bytes += pack_bytes(cfg, [w.specs[index[s]] for s in mb])
            packs += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    return dict(value=round(total_bytes / el / 1e9, 4), unit="GB/s", cores=1, kind="oracle",
                sample=f"{len(take)} of {cfg.n_mb} microbatches of seed {seed} "
                       f"({sum(len(m) for m in take)} samples), packed {packs} times in {el:.1f} s "
                       f"by the single-threaded numpy pool oracle",
                cpu_model=cpu_model_name(),
                os_cpu_count=os.cpu_count(), affinity=len(os.sched_getaffinity(0)))


def host_tier_rows(cfg, w, sid, spec) -> int:
    """Visual rows of a sample that sit on host-tier pages (from the pool's page table)."""
    from paper_2606_23087_amd import flowpool as fp
    rows = 0
    for i, gva in enumerate(fp.pool_sample_pages(w.pool, sid).tolist()):
        tier, _ = fp.pool_translate(w.pool, int(gva))
        if tier == fp.FP_TIER_HOST:
            rows += min(cfg.page_tokens, spec.n_vis - i * cfg.page_tokens)
    return rows


def tier_split(cfg, w, mbs, spec_of, outs, stream, reps: int = 3):
    """Tiered pool: time the HBM-tier part (text rows + rows on HBM pages) and
    the host-tier part (rows on pinned host pages, read over PCIe) as separate
    masked launches, and both masks concurrently on two streams."""
    import torch
    from paper_2606_23087_amd import flowpool as fp
    host_rows = [sum(host_tier_rows(cfg, w, s, spec_of[s]) for s in mb) for mb in mbs]
    tot_rows = [sum(spec_of[s].length for s in mb) for mb in mbs]
    rb = cfg.row_bytes
    second = torch.cuda.Stream()

    def timed(masks_streams):
        ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        gc.collect()
        gc.disable()
        ev[0].record(stream)
        for _ in range(reps):
            for j, mb in enumerate(mbs):
                out, cu, pos = outs[j % len(outs)]
                for mask, st in masks_streams:
                    if st is not stream:
                        st.wait_stream(stream)
                    w.pack(mb, out, cu if mask & 1 else None, pos if mask & 1 else None, tier_mask=mask, stream=st)
                    if st is not stream:
                        stream.wait_stream(st)
        ev[1].record(stream)
        gc.enable()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) * 1e-3 / reps

    t_hbm = timed([(fp.FP_TIER_MASK_HBM, stream)])
    t_host = timed([(fp.FP_TIER_MASK_HOST, stream)])
    t_both = timed([(fp.FP_TIER_MASK_HBM, stream), (fp.FP_TIER_MASK_HOST, second)])
    t_all = timed([(fp.FP_TIER_MASK_ALL, stream)])
    hbm_bytes = 2 * (sum(tot_rows) - sum(host_rows)) * rb
    pcie_bytes = sum(host_rows) * rb
    # Gather ceiling of the HBM-tier part: the same HBM-side rows (text rows
    # and rows on HBM pages) gathered by the plain measurement kernel.
    import numpy as np
    lists = []
    for mb in mbs:
        a, t = row_sources(cfg, w, mb, spec_of, tiers=True)
        lists.append(torch.from_numpy(a[t == 0].view(np.int64)).to("cuda"))
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for rep in range(reps + 1):
        if rep == 1:
            e0.record(stream)
        for j, lst in enumerate(lists):
            fp.fp_gather_rows(lst, lst.numel(), rb, outs[j % len(outs)][0], stream)
    e1.record(stream)
    torch.cuda.synchronize()
    t_gather = e0.elapsed_time(e1) * 1e-3 / reps
    del lists
    return {"host_tier_row_fraction": round(sum(host_rows) / sum(tot_rows), 4),
            "text_row_fraction_of_hbm_part": round(sum(spec_of[x].n_text for mb in mbs for x in mb)
                                                   / (sum(tot_rows) - sum(host_rows)), 4),
            "hbm_tier": {"GBps": round(hbm_bytes / t_hbm / 1e9, 1), "peak": HBM_PEAK_GBPS,
                         "bytes": hbm_bytes, "ms": round(t_hbm * 1e3, 3),
                         "gather_ceiling_GBps": round(hbm_bytes / t_gather / 1e9, 1),
                         "gather_ceiling_ms": round(t_gather * 1e3, 3)},
            "host_tier": {"GBps": round(pcie_bytes / t_host / 1e9, 2), "peak": PCIE_PEAK_GBPS,
                          "bytes_over_pcie": pcie_bytes, "ms": round(t_host * 1e3, 3)},
            "both_masks_two_streams_ms": round(t_both * 1e3, 3),
            "one_full_pack_ms": round(t_all * 1e3, 3)}


def aux_tiered(args) -> dict:
    """The tiered workload (seed 0) beside the headline: the HBM-tier part
    (text rows and rows on HBM pages) and the host-tier part (rows on pinned
    host pages, read over PCIe) of each microbatch as separate masked packs,
    each timed over ``max(3, steps // 2)`` passes after one warm pass, with
    the gather ceiling of the HBM part and a pinned host-to-device copy rate."""
    import torch

    from paper_2606_23087_amd.harness import GpuWorkload
    from paper_2606_23087_amd.workloads import CONFIGS

    cfg = CONFIGS["tiered"]
    w = GpuWorkload(cfg, 0, mode="normal")
    try:
        stream = torch.cuda.Stream()
        plan = w.plan(stream=stream)
        mbs = w.microbatches(plan)
        spec_of = {sid: sp for sid, sp in zip(w.ids, w.specs)}
        outs = [w.alloc_outputs() for _ in range(4)]
        tiers = tier_split(cfg, w, mbs, spec_of, outs, stream, reps=1)          # warm pass
        tiers = tier_split(cfg, w, mbs, spec_of, outs, stream, reps=max(3, args.steps // 2))
        tiers["hbm_tier"]["frac"] = round(tiers["hbm_tier"]["GBps"] / HBM_PEAK_GBPS, 4)
        tiers["host_tier"]["frac_of_pcie"] = round(tiers["host_tier"]["GBps"] / PCIE_PEAK_GBPS, 4)
        tiers["h2d_copy_GBps"] = round(h2d_ceiling(), 1)
        tiers["config"] = {"workload": f"{cfg.name}-h{cfg.hidden}", "seed": 0, "microbatches": len(mbs),
                           "passes": max(3, args.steps // 2)}
        log(f"aux tiered: HBM part {tiers['hbm_tier']['GBps']} GB/s ({tiers['hbm_tier']['frac']}), host part "
            f"{tiers['host_tier']['GBps']} GB/s over PCIe")
        return tiers
    finally:
        w.close()


def row_sources(cfg, w, mb, spec_of, tiers=False):
    """Device address of the source of every row of microbatch ``mb``, in
    pack order (text rows: their table row, with bit 0 set to mark it as one;
    image rows: their row in the physical page, from the pool's page table),
    for the gather ceiling; with ``tiers``, also each row's tier (text rows
    count as HBM)."""
    import numpy as np
    from paper_2606_23087_amd import flowpool as fp
    rb, P = cfg.row_bytes, cfg.page_tokens
    table = np.uint64(w.table.data_ptr())
    addr, tier = [], []
    for sid in mb:
        sp = spec_of[sid]
        phys, ptier = [], []
        for g in fp.pool_sample_pages(w.pool, sid).tolist():
            t, a = fp.pool_translate(w.pool, int(g))
            phys.append(a)
            ptier.append(t)
        phys = np.array(phys, np.uint64)
        v = np.arange(sp.n_vis, dtype=np.uint64)
        vis = phys[(v // np.uint64(P)).astype(np.int64)] + (v % np.uint64(P)) * np.uint64(rb) if sp.n_vis \
            else np.zeros(0, np.uint64)
        vtier = np.array(ptier, np.int8)[(np.arange(sp.n_vis) // P)] if sp.n_vis else np.zeros(0, np.int8)
        text = (table + sp.text_ids.astype(np.uint64) * np.uint64(rb)) | np.uint64(1)   # bit 0: a table row
        ti = vi = 0
        for p_, nt in zip(sp.img_pos.tolist(), sp.img_ntok.tolist()):
            addr += [text[ti:p_], vis[vi:vi + nt]]
            tier += [np.zeros(p_ - ti, np.int8), vtier[vi:vi + nt]]
            ti, vi = p_, vi + nt
        addr.append(text[ti:])
        tier.append(np.zeros(sp.n_text - ti, np.int8))
    a = np.concatenate(addr)
    return (a, np.concatenate(tier)) if tiers else a


def ceilings(cfg, w, mbs, spec_of, outs, stream, passes: int, mask: int = 3):
    """Same-run ceilings for the pack of these microbatches, from the
    library's measurement kernels (the pack's chunk geometry and cache
    policy, nothing else):
    - copy: one plain copy per microbatch, of its rows' bytes, from a 2 GiB
      source walked forward (cache-cold) into the rotating output buffers;
    - gather: each microbatch's rows gathered from the same source addresses
      the pack reads (table rows and page rows), into the same buffers.
    Each is timed like the pack: one event pair around all launches of
    ``passes`` passes over the microbatches. With a tier mask, only the rows
    of that tier (text rows count as HBM)."""
    import numpy as np
    import torch
    from paper_2606_23087_amd import flowpool as fp
    rb = cfg.row_bytes
    src_lists = []
    for mb in mbs:
        a, t = row_sources(cfg, w, mb, spec_of, tiers=True)
        if mask != fp.FP_TIER_MASK_ALL:
            a = a[t == (1 if mask == fp.FP_TIER_MASK_HOST else 0)]
        src_lists.append(torch.from_numpy(a.view(np.int64)).to("cuda"))
    rows = [x.numel() for x in src_lists]
    pool_bytes = max(2 << 30, max(rows) * rb)
    src = torch.empty(pool_bytes, dtype=torch.uint8, device="cuda")
    offs, at = [], 0
    for n in rows:
        if at + n * rb > pool_bytes:
            at = 0
        offs.append(at)
        at += n * rb

    def run(kind: str) -> float:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for rep in range(passes + 1):
            if rep == 1:
                e0.record(stream)
            for j, n in enumerate(rows):
                out = outs[j % len(outs)][0]
                if kind == "copy":
                    fp.fp_copy_bytes(src.data_ptr() + offs[j], out, n * rb, rb, stream)
                else:
                    fp.fp_gather_rows(src_lists[j], n, rb, out, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / (passes * len(rows))

    torch.cuda.synchronize()
    t_copy = run("copy")
    t_gather = run("gather")
    mean_row_bytes = 2 * rb * float(np.mean(rows))
    del src, src_lists
    return {"what": "plain copy and plain gather of the same microbatch rows, library measurement kernels",
            "copy_us": round(t_copy * 1e6, 3), "copy_GBps": round(mean_row_bytes / t_copy / 1e9, 1),
            "gather_us": round(t_gather * 1e6, 3), "gather_GBps": round(mean_row_bytes / t_gather / 1e9, 1)}


def h2d_ceiling(nbytes: int = 1 << 30, iters: int = 5) -> float:
    """Pinned host -> device copy rate of one large copy (the host tier's link)."""
    import torch
    h = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    d.copy_(h, non_blocking=True)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(iters):
        d.copy_(h, non_blocking=True)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / iters
    del h, d
    return nbytes / (ms * 1e-3) / 1e9


SCHED_CAPACITIES = (2048, 4096, 8192, 16384, 32768)


def scheduler_bench(args) -> int:
    """Overhead of the dynamic packing scheduler (Alg. 1) per scheduling call,
    host only: one call packs a window of n_ranks * mb_per_rank * L tokens of
    qwen-workload sample lengths (clipped to L) into microbatches of L tokens,
    buckets them and deals them to n_ranks ranks. The oracle is timed on the
    same call as the CPU baseline and must give the same plan."""
    import statistics

    import numpy as np

    from oracle.schedule import dynamic_packing
    from paper_2606_23087_amd import flowpool as fp
    from paper_2606_23087_amd.workloads import schedule_lengths

    N, K, per = args.sched_ranks, args.sched_buckets, args.sched_mb_per_rank
    rows = []
    for L in SCHED_CAPACITIES:
        lens = schedule_lengths(args.seed, L, N * per * L)
        r = fp.plan_dynamic_packing(lens, L, N, K)
        ts = []
        for _ in range(args.sched_reps):
            t0 = time.perf_counter()
            r = fp.plan_dynamic_packing(lens, L, N, K)
            ts.append(time.perf_counter() - t0)
        t0 = time.perf_counter()
        want = dynamic_packing([int(x) for x in lens], L, N, K)
        t_oracle = time.perf_counter() - t0
        same = (want["mb_of_seq"] == r["mb_of_seq"].tolist() and want["mb_rank"] == r["mb_rank"].tolist()
                and want["mb_slot"] == r["mb_slot"].tolist() and want["mb_bucket"] == r["mb_bucket"].tolist())
        rank_cost = np.zeros(N)
        np.add.at(rank_cost, r["mb_rank"], r["mb_cost_scaled"].astype(float))
        rows.append(dict(L=L, sequences=int(len(lens)), microbatches=int(r["n_mb"]),
                         ms_median=round(statistics.median(ts) * 1e3, 4), ms_min=round(min(ts) * 1e3, 4),
                         oracle_ms=round(t_oracle * 1e3, 2), same_plan_as_oracle=bool(same),
                         fill=round(float(lens.sum()) / (r["n_mb"] * L), 4),
                         rank_cost_max_over_mean=round(float(rank_cost.max() / rank_cost.mean()), 4)))
        log(f"scheduler L={L}: {rows[-1]}")
    print(json.dumps({
        "metric": "dynamic packing scheduler overhead per scheduling call (Alg. 1)",
        "value": rows[-1]["ms_median"], "unit": "ms", "higher_is_better": False,
        "data": "synthetic (qwen-workload sample lengths, clipped to L)",
        "config": {"workload": "alg1-scheduler", "n_ranks": N, "n_buckets": K, "window_tokens": f"{N * per} * L",
                   "capacities": list(SCHED_CAPACITIES), "reps": args.sched_reps, "seed": args.seed},
        "per_capacity": rows,
        "cpu_baseline": {"value": rows[-1]["oracle_ms"], "unit": "ms", "cores": 1, "kind": "oracle",
                         "sample": "the same call at L = 32768, once, single-threaded Python"},
    }), flush=True)
    return 0 if all(x["same_plan_as_oracle"] for x in rows) else 1


def concurrent_bench(args, cfg, w, mbs, spec_of, outs, pack_stream) -> dict:
    """Pack GB/s of the workload's microbatches alone and while a producer
    thread keeps writing new samples on its own stream (and freeing the oldest
    beyond a window of 16), both timed over the same packs. The packs of one
    pass are captured into a HIP graph and replayed, so the consumer needs no
    host work per pack: enqueuing 1280 packs from Python while the producer
    thread holds the interpreter lock would starve the pack stream and time
    the host instead of the GPU."""
    import collections
    import threading

    import numpy as np
    import torch

    from paper_2606_23087_amd import flowpool as fp
    from paper_2606_23087_amd.harness import vis_rows
    from paper_2606_23087_amd.workloads import gen_samples

    pspecs = gen_samples(cfg, args.seed + 1000, count=32)
    pvis = [vis_rows(cfg, args.seed + 1000, i, s.n_vis, "normal") if s.n_vis else None
            for i, s in enumerate(pspecs)]
    prod_stream = torch.cuda.Stream()
    mb_bytes = sum(pack_bytes(cfg, [spec_of[s] for s in mb]) for mb in mbs)
    passes = max(1, args.steps)

    torch.cuda.synchronize()
    fp.pool_reclaim(w.pool, True)                   # the packed samples' writes are known complete
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(pack_stream):
        with torch.cuda.graph(graph, stream=pack_stream):
            for j, mb in enumerate(mbs):
                out, cu, pos = outs[j % len(outs)]
                w.pack(mb, out, cu, pos, stream=pack_stream)
    with torch.cuda.stream(pack_stream):
        graph.replay()
    torch.cuda.synchronize()

    def packs() -> float:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        gc.disable()          # a collector pause between enqueues would be timed as GPU idle
        e0.record(pack_stream)
        with torch.cuda.stream(pack_stream):
            for _ in range(passes):
                graph.replay()
        e1.record(pack_stream)
        gc.enable()
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e-3

    torch.cuda.synchronize()
    gc.collect()
    t_alone = packs()
    gc.collect()            # before the producer starts: a collection holds the interpreter lock
    stop = threading.Event()
    stats = {"writes": 0, "bytes": 0, "error": None}

    def producer():
        window = collections.deque()
        try:
            with torch.cuda.stream(prod_stream):
                i = 0
                while not stop.is_set():
                    s = pspecs[i % len(pspecs)]
                    sid = fp.pool_write_sample(w.pool, s.text_ids, s.img_pos, s.img_ntok, pvis[i % len(pspecs)],
                                               stream=prod_stream)
                    window.append(sid)
                    if len(window) > 16:
                        fp.pool_free_sample(w.pool, window.popleft())
                    stats["writes"] += 1
                    stats["bytes"] += 2 * s.n_vis * cfg.row_bytes + 4 * s.n_text
                    i += 1
            prod_stream.synchronize()
        except Exception as e:  # reported below
            stats["error"] = repr(e)
        finally:
            for sid in window:
                fp.pool_free_sample(w.pool, sid)

    th = threading.Thread(target=producer)
    th.start()
    time.sleep(0.05)
    wall0 = time.perf_counter()
    w0, b0 = stats["writes"], stats["bytes"]
    t_busy = packs()
    wall = time.perf_counter() - wall0
    w1, b1 = stats["writes"], stats["bytes"]
    stop.set()
    th.join()
    torch.cuda.synchronize()
    del graph
    for mb in mbs:                          # the graph is gone: its packs no longer hold their samples
        fp.pool_release_captured(w.pool, mb)
    alone = mb_bytes * passes / t_alone / 1e9
    busy = mb_bytes * passes / t_busy / 1e9
    prod = (b1 - b0) / wall / 1e9
    log(f"concurrent: pack alone {alone:.0f} GB/s, with producer {busy:.0f} GB/s, producer {prod:.0f} GB/s "
        f"({w1 - w0} writes)")
    return {"pack_alone_GBps": round(alone, 1), "pack_with_producer_GBps": round(busy, 1),
            "producer_GBps": round(prod, 1), "producer_writes": w1 - w0,
            "producer_writes_per_s": round((w1 - w0) / wall, 1), "passes": passes,
            "pack_launches": passes * len(mbs), "producer_error": stats["error"],
            "deferred_pages_after": fp.pool_reclaim(w.pool, True)}


def prefetch_bench(args, cfg, w, mbs, spec_of, outs, pack_stream) -> dict:
    """Tiered pool: pack every microbatch reading host-tier pages zero-copy over
    PCIe, then the same packs with each microbatch's host-tier pages first
    promoted into HBM by DMA copies on a copy stream (pool_migrate), the
    migration of microbatch j+1 overlapping the pack of microbatch j, then the
    packs again once everything sits in HBM."""
    import torch

    from paper_2606_23087_amd import flowpool as fp

    mb_bytes = sum(pack_bytes(cfg, [spec_of[s] for s in mb]) for mb in mbs)
    host_rows = 0
    for mb in mbs:
        for sid in mb:
            pages = fp.pool_sample_pages(w.pool, sid)
            n_vis = spec_of[sid].n_vis
            for k, g in enumerate(pages.tolist()):
                if fp.pool_translate(w.pool, g)[0] == fp.FP_TIER_HOST:
                    host_rows += min(cfg.page_tokens, n_vis - k * cfg.page_tokens)
    host_bytes = host_rows * cfg.row_bytes

    def packs() -> float:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        gc.collect()
        gc.disable()          # a collector pause between enqueues would be timed as GPU idle
        e0.record(pack_stream)
        for j, mb in enumerate(mbs):
            out, cu, pos = outs[j % len(outs)]
            w.pack(mb, out, cu, pos, stream=pack_stream)
        e1.record(pack_stream)
        gc.enable()
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e-3

    packs()
    t_zero_copy = packs()
    copy_stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    gc.collect()
    gc.disable()
    t0 = time.perf_counter()
    c0.record(copy_stream)
    p0.record(pack_stream)
    moved = fp.pool_migrate(w.pool, mbs[0], fp.FP_TIER_HBM, stream=copy_stream)
    for j, mb in enumerate(mbs):
        if j + 1 < len(mbs):
            moved += fp.pool_migrate(w.pool, mbs[j + 1], fp.FP_TIER_HBM, stream=copy_stream)
        out, cu, pos = outs[j % len(outs)]
        w.pack(mb, out, cu, pos, stream=pack_stream)
    c1.record(copy_stream)
    p1.record(pack_stream)
    gc.enable()
    torch.cuda.synchronize()
    t_pipe = time.perf_counter() - t0
    t_copy = c0.elapsed_time(c1) * 1e-3
    t_pipe_gpu = p0.elapsed_time(p1) * 1e-3
    fp.pool_reclaim(w.pool, True)
    t_hbm_all = [packs() for _ in range(4)]
    t_hbm = min(t_hbm_all[1:])              # the first pass after the promotion is a warm-up
    log(f"prefetch: zero-copy {t_zero_copy * 1e3:.2f} ms, pipelined {t_pipe_gpu * 1e3:.2f} ms "
        f"(copies {t_copy * 1e3:.2f} ms, {moved} pages), all-HBM passes "
        f"{', '.join(f'{t * 1e3:.3f}' for t in t_hbm_all)} ms")
    return {"microbatches": len(mbs), "pack_bytes": mb_bytes, "host_tier_bytes": host_bytes,
            "zero_copy_ms": round(t_zero_copy * 1e3, 3),
            "zero_copy_GBps": round(mb_bytes / t_zero_copy / 1e9, 1),
            "pipelined_ms": round(t_pipe_gpu * 1e3, 3), "pipelined_wall_ms": round(t_pipe * 1e3, 3),
            "pages_moved": moved, "copy_stream_ms": round(t_copy * 1e3, 3),
            "copy_GBps": round(host_bytes / t_copy / 1e9, 1),
            "all_hbm_ms": round(t_hbm * 1e3, 3), "all_hbm_GBps": round(mb_bytes / t_hbm / 1e9, 1),
            "all_hbm_passes_ms": [round(t * 1e3, 3) for t in t_hbm_all],
            "pcie_peak_GBps": PCIE_PEAK_GBPS}


ALLOC_DEVICES = (64, 128, 256, 512, 1024)


def table_policy_bench(args) -> int:
    """Gathers of random embedding-table rows through the library's gather
    kernel, with the table-row mark (the plain loads the pack uses for chunks
    holding table rows) and without it (the non-temporal loads of page rows),
    over tables of several sizes: 16000 rows of 7168 bytes per launch at
    uniform random ids, 64 launches into 4 rotating buffers, timed like the
    pack (one event pair around all launches of ``--steps`` passes). Plain
    loads let the device's 256 MB memory-side cache keep table rows, which
    pays while a good part of the table fits there."""
    import numpy as np
    import torch

    from paper_2606_23087_amd import flowpool as fp

    rb, rows, launches, passes = 7168, 16000, 64, max(1, args.steps)
    outs = [torch.empty(rows * rb, dtype=torch.uint8, device="cuda") for _ in range(4)]
    stream = torch.cuda.current_stream()
    res = []
    for table_rows in (9362, 37449, 152064, 228096, 304128, 380160, 456192, 600000):
        table = torch.ones(table_rows * rb, dtype=torch.uint8, device="cuda")
        ids = np.random.default_rng(args.seed).integers(0, table_rows, size=(launches, rows))
        addr = table.data_ptr() + ids.astype(np.int64) * rb
        row = {"table_rows": table_rows, "table_MB": round(table_rows * rb / 1e6, 1)}
        for name, mark in (("plain_loads", 1), ("nontemporal_loads", 0)):
            lists = torch.from_numpy(addr | mark).to("cuda")
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            for rep in range(passes + 1):
                if rep == 1:
                    e0.record(stream)
                for j in range(launches):
                    fp.fp_gather_rows(lists[j], rows, rb, outs[j % 4], stream)
            e1.record(stream)
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / (passes * launches)
            row[name] = {"us": round(us, 3), "GBps": round(2 * rows * rb / us / 1e3, 1)}
            del lists
        row["plain_over_nontemporal"] = round(row["nontemporal_loads"]["us"] / row["plain_loads"]["us"], 4)
        log(f"table policy: {row}")
        res.append(row)
        del table
    at = [x for x in res if x["table_rows"] == 152064][0]
    print(json.dumps({
        "metric": "gather of random 7168-byte embedding-table rows, plain vs non-temporal loads",
        "value": at["plain_loads"]["GBps"], "unit": "GB/s", "higher_is_better": True, "n_gpus": 1,
        "data": "synthetic", "config": {"workload": "table-policy", "rows_per_launch": rows, "launches": launches,
                                        "passes": passes, "seed": args.seed},
        "per_table": res}), flush=True)
    return 0


def copy_sizes_bench(args) -> int:
    """The library's plain copy kernel (the pack's chunk geometry and cache
    policy, rows of 7168 bytes) at launch sizes from one qwen microbatch (230
    MB moved) to sixteen, so the copy's steady rate and the fixed cost of a
    launch's ramp and drain can be read apart: about as many bytes per size,
    sources walked forward through 8 GiB, destinations alternating between
    two buffers, one event pair around all launches of a size (after one
    untimed pass)."""
    import torch

    from paper_2606_23087_amd import flowpool as fp

    time.sleep(max(0.0, args.settle - seconds_since_start()))
    rb = 7168
    src = torch.empty(8 << 30, dtype=torch.uint8, device="cuda")
    dst = [torch.empty(4 << 30, dtype=torch.uint8, device="cuda") for _ in range(2)]
    stream = torch.cuda.current_stream()
    res = []
    for mult in (1, 2, 4, 8, 16):
        n = (115 * 1000 * 1000 * mult) // rb * rb          # bytes read (and written) per launch
        launches = max(4, 64 // mult)
        for rep in range(2):
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for j in range(launches):
                off = (j * n) % ((8 << 30) - n)
                fp.fp_copy_bytes(src.data_ptr() + off - off % 256, dst[j % 2], n, rb, stream)
            e1.record(stream)
            torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / launches
        res.append({"moved_MB": round(2 * n / 1e6, 1), "launches": launches, "us_per_launch": round(us, 3),
                    "GBps": round(2 * n / us / 1e3, 1), "frac": round(2 * n / us / 1e3 / HBM_PEAK_GBPS, 4)})
        log(f"copy sizes: {res[-1]}")
    print(json.dumps({
        "metric": "plain copy kernel with the pack's geometry, by launch size", "value": max(r["GBps"] for r in res),
        "unit": "GB/s", "higher_is_better": True, "n_gpus": 1, "data": "synthetic",
        "config": {"workload": "copy-sizes", "row_bytes": rb}, "per_size": res}), flush=True)
    return 0


def allocator_bench(args) -> int:
    """Time of the allocator's flow matching (Eq. 2) on the host for clusters
    of 8-device nodes (global batch 512, a 28-layer backbone, two encoders),
    on synthetic throughput surrogates over the pruned candidates. The
    oracle's enumeration is timed beside it where it finishes in seconds and
    must give the same answer."""
    import statistics

    from oracle.allocate import solve
    from paper_2606_23087_amd import flowpool as fp
    from paper_2606_23087_amd.workloads import allocator_tables

    rows = []
    for dev in ALLOC_DEVICES:
        mods = allocator_tables(args.seed, dev, candidates_fn=fp.alloc_candidates)
        combos = 1
        for m in mods:
            combos *= len(m)
        r = fp.plan_allocation(mods, dev)
        ts = []
        for _ in range(args.sched_reps):
            t0 = time.perf_counter()
            r = fp.plan_allocation(mods, dev)
            ts.append(time.perf_counter() - t0)
        row = dict(devices=dev, configs=[len(m) for m in mods], combinations=combos,
                   ms_median=round(statistics.median(ts) * 1e3, 4), G=r["G"], F=r["F"], devices_used=r["devices"],
                   choice=r["choice"])
        if combos <= 300_000:
            t0 = time.perf_counter()
            want = solve(mods, dev)
            row["oracle_ms"] = round((time.perf_counter() - t0) * 1e3, 1)
            row["same_as_oracle"] = (list(want) == [r["choice"], r["G"], r["F"], r["devices"]])
        rows.append(row)
        log(f"allocator {dev} devices: {row}")
    at256 = [x for x in rows if x["devices"] == 256][0]
    print(json.dumps({
        "metric": "allocator flow matching (Eq. 2) time per solve",
        "value": at256["ms_median"], "unit": "ms", "higher_is_better": False,
        "data": "synthetic throughput surrogates over pruned candidates",
        "config": {"workload": "allocator", "per_node": 8, "global_batch": 512, "layers": 28, "encoders": 2,
                   "reps": args.sched_reps, "seed": args.seed},
        "per_cluster": rows,
        "cpu_baseline": {"value": at256.get("oracle_ms"), "unit": "ms", "cores": 1, "kind": "oracle",
                         "sample": "enumeration of every combination at 256 devices, once"},
    }), flush=True)
    return 0 if all(x.get("same_as_oracle", True) for x in rows) else 1


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen", choices=["tiny", "qwen", "frag70b", "video", "tiered"])
    ap.add_argument("--seed", type=int, default=0, help="seed of the --prefetch, --concurrent, --scheduler "
                    "and --allocator legs")
    ap.add_argument("--seeds", default="0,1,2", help="seeds whose workloads the timed steps cycle through")
    ap.add_argument("--buffers", type=int, default=4, help="rotating output buffers")
    ap.add_argument("--mask", default="all", choices=["all", "hbm", "host"],
                    help="tier mask of the timed packs (tiered pool: time one tier's part alone)")
    ap.add_argument("--settle", type=float, default=3.0,
                    help="seconds after the process started before the warm-up begins (the device clears "
                         "memory freed by an earlier process in the background for a few seconds, which "
                         "takes HBM bandwidth from the packs)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run one plain 1 GiB copy (reference for HBM byte counters)")
    ap.add_argument("--scheduler", action="store_true",
                    help="time the dynamic packing scheduler (Alg. 1) on the host instead of the pack")
    ap.add_argument("--sched-ranks", type=int, default=32)
    ap.add_argument("--sched-buckets", type=int, default=4)
    ap.add_argument("--sched-mb-per-rank", type=int, default=8)
    ap.add_argument("--sched-reps", type=int, default=50)
    ap.add_argument("--allocator", action="store_true",
                    help="time the allocator's flow matching (Eq. 2) on the host instead of the pack")
    ap.add_argument("--prefetch", action="store_true",
                    help="tiered pool: zero-copy packs vs packs after promoting host-tier pages into HBM")
    ap.add_argument("--graph", action="store_true",
                    help="also time one step's packs captured into a HIP graph and replayed")
    ap.add_argument("--table-policy", action="store_true",
                    help="time gathers of random embedding-table rows with the pack's plain loads and with "
                         "non-temporal ones, over tables of several sizes")
    ap.add_argument("--concurrent", action="store_true",
                    help="time the packs alone and under a concurrent producer on another stream")
    ap.add_argument("--copy-sizes", action="store_true",
                    help="time the library's plain copy kernel at launch sizes from 230 MB to 3.7 GB moved")
    ap.add_argument("--no-aux", action="store_true",
                    help="skip the auxiliary legs the headline run adds to its line (the tiered workload's "
                         "two tier parts, and the packs under a concurrent producer)")
    args = ap.parse_args()

    if args.scheduler:
        return scheduler_bench(args)
    if args.allocator:
        return allocator_bench(args)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the pack path is not sharded across GPUs in this library "
              "(run with --gpus 1)", file=sys.stderr)
        return 2

    if args.table_policy:
        return table_policy_bench(args)
    if args.copy_sizes:
        return copy_sizes_bench(args)

    import numpy as np
    import torch

    from paper_2606_23087_amd import flowpool as fp
    from paper_2606_23087_amd.harness import GpuWorkload
    from paper_2606_23087_amd.workloads import CONFIGS

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    cfg = CONFIGS[args.workload]
    seeds = [int(x) for x in str(args.seeds).split(",")] if not (args.prefetch or args.concurrent) else [args.seed]
    log(f"workload {cfg.name}: H={cfg.hidden} P={cfg.page_tokens} C={cfg.capacity} M={cfg.n_mb}, seeds {seeds}")
    works = {}
    table = None          # the seeds' workloads read one embedding table, as the steps of one job do
    for sd in seeds:
        t_setup = time.perf_counter()
        works[sd] = GpuWorkload(cfg, sd, mode="normal", log=log, table=table)
        table = works[sd].table
        log(f"seed {sd}: pool built, {len(works[sd].ids)} samples in {time.perf_counter() - t_setup:.1f} s, "
            f"{fp.pool_stats(works[sd].pool)}")
    s0 = seeds[0]
    w = works[s0]
    spec_of = {sd: {sid: sp for sid, sp in zip(wk.ids, wk.specs)} for sd, wk in works.items()}

    if args.calibrate_copy:
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
        log("calibration copy: 1 GiB read + 1 GiB written")

    pack_stream = torch.cuda.Stream()
    plan_stream = torch.cuda.Stream()
    outs = [w.alloc_outputs() for _ in range(max(1, args.buffers))]
    mask = {"all": fp.FP_TIER_MASK_ALL, "hbm": fp.FP_TIER_MASK_HBM, "host": fp.FP_TIER_MASK_HOST}[args.mask]

    def one_step(sd, events=None, mark=None):
        """Plan seed sd's resident samples, then pack every microbatch on the
        pack stream; `mark` is recorded on the pack stream before the first pack."""
        wk = works[sd]
        plan = wk.plan(stream=plan_stream)
        mbs = wk.microbatches(plan)
        for j, mb in enumerate(mbs):
            out, cu, pos = outs[j % len(outs)]
            if j == 0 and mark is not None:
                mark.record(pack_stream)
            if events is not None:
                events[j][0].record(pack_stream)
            if mask & fp.FP_TIER_MASK_HBM:
                wk.pack(mb, out, cu, pos, tier_mask=mask, stream=pack_stream)
            else:
                wk.pack(mb, out, None, None, tier_mask=mask, stream=pack_stream)
            if events is not None:
                events[j][1].record(pack_stream)
        return plan, mbs

    info = {}
    for sd in seeds:
        plan, mbs = one_step(sd)
        info[sd] = dict(plan=plan, mbs=mbs,
                        mb_bytes=[masked_pack_bytes(cfg, works[sd], mb, spec_of[sd], mask) for mb in mbs],
                        tokens=int(plan["mb_tokens"].sum()), deferred=int((plan["assign"] < 0).sum()))
        info[sd]["step_bytes"] = sum(info[sd]["mb_bytes"])
    torch.cuda.synchronize()
    since_start = seconds_since_start()
    slept = max(0.0, args.settle - since_start)
    if slept > 0:
        log(f"settling {slept:.2f} s ({since_start:.2f} s since the process started)")
        time.sleep(slept)
    for k in range(args.warmup):
        one_step(seeds[k % len(seeds)])
    torch.cuda.synchronize()
    plan, mbs = info[s0]["plan"], info[s0]["mbs"]
    log(f"warmup done: seed {s0}: {len(mbs)} microbatches, {info[s0]['tokens']} tokens, "
        f"{info[s0]['step_bytes'] / 1e6:.1f} MB per step, {info[s0]['deferred']} samples deferred")

    if args.prefetch:
        res = prefetch_bench(args, cfg, w, mbs, spec_of[s0], outs, pack_stream)
        print(json.dumps({
            "metric": "tiered pack: zero-copy host-tier reads vs host-tier pages promoted into HBM first",
            "value": res["pipelined_ms"], "unit": "ms per 16 microbatches (pipelined promote + pack)",
            "higher_is_better": False, "n_gpus": 1, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"{cfg.name}-h{cfg.hidden}-prefetch", "seed": args.seed},
            "prefetch": res}), flush=True)
        w.close()
        return 0

    if args.concurrent:
        res = concurrent_bench(args, cfg, w, mbs, spec_of[s0], outs, pack_stream)
        print(json.dumps({
            "metric": "pack_microbatch GB/s with a concurrent producer writing on another stream",
            "value": res["pack_with_producer_GBps"], "unit": "GB/s", "higher_is_better": True,
            "n_gpus": 1, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"{cfg.name}-h{cfg.hidden}-concurrent", "producer_window": 16,
                       "producer_samples": 32, "seed": args.seed},
            "concurrent": res}), flush=True)
        w.close()
        return 0 if res["producer_error"] is None else 1

    def timed(order):
        """Whole steps for the seeds in `order`, back to back. Returns the wall
        time, the pack-stream time from the first pack to the last, and the
        launches, bytes and tokens. One event pair brackets all pack launches;
        the wall clock brackets everything, planning included."""
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        gc.collect()
        gc.disable()          # no collector pauses between enqueues inside the timed region
        t0 = time.perf_counter()
        for k, sd in enumerate(order):
            one_step(sd, mark=e0 if k == 0 else None)
        e1.record(pack_stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        gc.enable()
        return dict(wall=wall, packs=e0.elapsed_time(e1) * 1e-3, launches=sum(len(info[sd]["mbs"]) for sd in order),
                    bytes=sum(info[sd]["step_bytes"] for sd in order), tokens=sum(info[sd]["tokens"] for sd in order))

    # Timed region: K whole steps, the seeds' workloads in turn.
    order = [seeds[k % len(seeds)] for k in range(args.steps)]
    main_t = timed(order)
    launch_s = main_t["packs"] / main_t["launches"]
    mean_bytes = main_t["bytes"] / main_t["launches"]
    kernel_gbps = mean_bytes / launch_s / 1e9
    value = main_t["bytes"] / main_t["wall"] / 1e9

    # Each seed alone, K steps, measured the same way (outside the timed region).
    per_seed = []
    for sd in seeds:
        t = timed([sd] * args.steps)
        g = t["bytes"] / t["packs"] / 1e9
        per_seed.append({"seed": sd, "samples": len(works[sd].ids), "step_bytes": info[sd]["step_bytes"],
                         "deferred_samples": info[sd]["deferred"],
                         "mean_us": round(t["packs"] / t["launches"] * 1e6, 3), "GBps": round(g, 2),
                         "frac": round(g / HBM_PEAK_GBPS, 4), "step_GBps": round(t["bytes"] / t["wall"] / 1e9, 2)})
        log(f"seed {sd}: {per_seed[-1]}")

    # Per-call spread, from one extra step of the first seed with an event
    # pair around every launch (per-call event records perturb the stream
    # they time: each launch reads about 1.5 us longer than back to back).
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(len(mbs))]
    one_step(s0, events)
    torch.cuda.synchronize()
    durs = np.array([s_.elapsed_time(e_) * 1e-3 for s_, e_ in events])   # seconds

    ceiling = ceilings(cfg, w, mbs, spec_of[s0], outs, pack_stream, args.steps, mask)
    pack_s0 = [x for x in per_seed if x["seed"] == s0][0]
    ceiling["pack_over_gather"] = round(ceiling["gather_us"] / pack_s0["mean_us"], 4)
    ceiling["pack_over_copy"] = round(ceiling["copy_us"] / pack_s0["mean_us"], 4)

    graph_s = None
    graph2_s = None
    if args.graph:
        # One step's packs captured into a HIP graph and replayed: no host
        # work per pack (matters when the packs are small and host-bound).
        # Captured once as one chain of packs, once as two independent chains
        # (forked from the capture stream): packs into distinct buffers do not
        # depend on each other, and two at a time hide each other's launch
        # ramp and drain.
        fp.pool_reclaim(w.pool, True)
        gouts = [w.alloc_outputs() for _ in range(len(mbs))]

        def replay_s(branches: int) -> float:
            side = [torch.cuda.Stream() for _ in range(branches)]
            g = torch.cuda.CUDAGraph()
            with torch.cuda.stream(pack_stream):
                with torch.cuda.graph(g, stream=pack_stream):
                    for st in side:
                        st.wait_stream(pack_stream)
                    for j, (mb, (o, c, q)) in enumerate(zip(mbs, gouts)):
                        w.pack(mb, o, c, q, stream=side[j % branches] if branches > 1 else pack_stream)
                    for st in side:
                        pack_stream.wait_stream(st)
            with torch.cuda.stream(pack_stream):
                g.replay()
            torch.cuda.synchronize()
            g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            g0.record(pack_stream)
            with torch.cuda.stream(pack_stream):
                for _ in range(args.steps):
                    g.replay()
            g1.record(pack_stream)
            torch.cuda.synchronize()
            del g
            for mb in mbs:
                fp.pool_release_captured(w.pool, mb)
            return g0.elapsed_time(g1) * 1e-3 / args.steps

        graph_s = replay_s(1)
        graph2_s = replay_s(2)
        del gouts

    per_call = np.array(info[s0]["mb_bytes"], dtype=np.float64) / durs / 1e9
    traffic = counter_traffic(cfg.name, args.mask)
    fracs = [x["frac"] for x in per_seed]
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle": {"since_start_s": round(since_start, 3), "slept_s": round(slept, 3)},
        "ms_per_step": round(main_t["wall"] / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}-h{cfg.hidden}", "hidden": cfg.hidden, "page_tokens": cfg.page_tokens,
                   "pool_pages": cfg.hbm_pages + cfg.host_pages, "alloc": cfg.alloc, "capacity": cfg.capacity,
                   "n_mb": cfg.n_mb, "cost_k": cfg.cost_k, "samples": len(w.ids),
                   "seeds": seeds, "steps_cycle_seeds": True, "table": f"one embedding table (seed {s0}'s) for all seeds",
                   "parallelism": "none (1 GPU)"},
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBPS, 2),
        "tokens_per_s": round(main_t["tokens"] / main_t["wall"], 1),
        "step_tokens": info[s0]["tokens"],
        "step_bytes": info[s0]["step_bytes"],
        "deferred_samples": info[s0]["deferred"],
        "pack_kernel": {"launches": main_t["launches"], "mean_us": round(launch_s * 1e6, 3),
                        "mean_bytes": round(mean_bytes),
                        "timing": "pack-stream event pair around all launches of the timed steps",
                        "GBps": round(kernel_gbps, 2),
                        "single_call_events_us_p10_p50_p90_max": [round(float(np.percentile(durs, q)) * 1e6, 2)
                                                                   for q in (10, 50, 90, 100)],
                        "single_call_median_GBps": round(float(np.median(per_call)), 2)},
        "roofline": {"bound": "hbm", "achieved": round(kernel_gbps, 2), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(kernel_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": (round(traffic) if traffic else None),
                     "traffic_over_algorithmic": (round(traffic / mean_bytes, 4) if traffic else None)},
        "per_seed": per_seed,
        "median_over_seeds": {"frac": float(np.median(fracs)),
                              "GBps": float(np.median([x["GBps"] for x in per_seed])),
                              "mean_us": float(np.median([x["mean_us"] for x in per_seed]))},
        "ceiling": ceiling,
    }
    if graph_s is not None:
        step_bytes = info[s0]["step_bytes"]
        result["graph_pack_two_chains"] = {"replay_ms": round(graph2_s * 1e3, 4),
                                           "GBps": round(step_bytes / graph2_s / 1e9, 2)}
        result["graph_pack"] = {"packs_per_replay": len(mbs), "replay_ms": round(graph_s * 1e3, 4),
                                "GBps": round(step_bytes / graph_s / 1e9, 2)}
    imb = plan["mb_cost_scaled"].max() / plan["mb_cost_scaled"].mean()
    result["plan"] = {"max_over_mean_cost": round(float(imb), 5),
                      "eq3_max": round(float(max((t / cfg.capacity) + (m / cfg.capacity) ** 2
                                                 for t, m in zip(plan["mb_tokens"], plan["mb_max_len"]))), 5)}
    if args.mask != "all":
        result["config"]["tier_mask"] = args.mask
    if cfg.host_pages and args.mask == "all":
        result["tiers"] = tier_split(cfg, w, mbs, spec_of[s0], outs, pack_stream)
        result["tiers"]["h2d_copy_GBps"] = round(h2d_ceiling(), 1)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle")
        result["cpu_baseline"] = cpu_baseline(cfg, w, mbs, s0, args.cpu_budget)
    else:
        result["cpu_baseline"] = None
    if cfg.name == "qwen" and args.mask == "all" and not args.no_aux:
        # Auxiliary legs, after everything above is measured: the packs of
        # this workload under a concurrent producer, then the tiered
        # workload's two tier parts. An error in one is recorded in the line.
        # The pools stay resident until the end: the device clears freed
        # memory in the background, which would take bandwidth from the legs.
        aux = {}
        try:
            log("aux: packs under a concurrent producer")
            aux["concurrent"] = concurrent_bench(args, cfg, w, mbs, spec_of[s0], outs, pack_stream)
        except Exception as e:                     # noqa: BLE001 - recorded, the headline stands
            aux["concurrent"] = {"error": repr(e)}
        try:
            log("aux: tiered workload, tier parts")
            aux["tiered"] = aux_tiered(args)
        except Exception as e:                     # noqa: BLE001
            aux["tiered"] = {"error": repr(e)}
        result["aux"] = aux
    for wk in works.values():
        wk.close()
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
