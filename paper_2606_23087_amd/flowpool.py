"""ctypes binding of libflowpool (include/flowpool.h). Argument marshalling only.

Every function has the name of the C entry point it calls. Host arrays are
numpy arrays; device buffers are torch tensors or raw integer addresses;
streams are torch streams, raw hipStream_t integers, or None (torch's current
stream). A non-OK status raises ``FlowPoolError`` with the library's message.

The library must have been built (``python -m paper_2606_23087_amd.build`` or
``__graft_entry__.build()``); importing this module without it fails loudly.
"""

from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libflowpool.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run paper_2606_23087_amd/build.py first")

# torch (when installed) ships its own HIP and HSA runtimes. Loading torch
# first lets the library bind to that already-loaded runtime; loaded the
# other way round, the process ends up with two HSA runtimes, and the second
# one to start finds no device.
try:
    import torch  # noqa: F401
except ImportError:
    pass

_lib = C.CDLL(LIB_PATH)
ABI_VERSION = 5   # FP_ABI_VERSION of include/flowpool.h that these bindings follow
if _lib.fp_abi_version() != ABI_VERSION:
    raise ImportError(f"{LIB_PATH} has ABI version {_lib.fp_abi_version()}, the bindings expect {ABI_VERSION}; rebuild it")

FP_OK, FP_EINVAL, FP_ENOMEM, FP_ENOENT, FP_ECAPACITY, FP_EALIGN, FP_EHIP, FP_ESTATE = 0, -1, -2, -3, -4, -5, -6, -7
STATUS_NAMES = {0: "OK", -1: "EINVAL", -2: "ENOMEM", -3: "ENOENT", -4: "ECAPACITY", -5: "EALIGN",
                -6: "EHIP", -7: "ESTATE"}
FP_ALLOC_CONTIG, FP_ALLOC_SCATTER = 0, 1
FP_TIER_HBM, FP_TIER_HOST = 0, 1
FP_TIER_MASK_HBM, FP_TIER_MASK_HOST, FP_TIER_MASK_ALL = 1, 2, 3
FP_PLAN_LPT, FP_PLAN_ZIGZAG = 0, 1
ALLOC_POLICIES = {"contig": FP_ALLOC_CONTIG, "scatter": FP_ALLOC_SCATTER}


class fp_pool_config(C.Structure):
    _fields_ = [
        ("hidden", C.c_int32), ("page_tokens", C.c_int32),
        ("hbm_pages", C.c_int64), ("host_pages", C.c_int64),
        ("alloc_policy", C.c_int32), ("device", C.c_int32),
        ("vocab", C.c_int64), ("gva_start", C.c_uint64),
        ("world_size", C.c_int32), ("rank", C.c_int32),
        ("max_samples", C.c_int64), ("meta_bytes", C.c_int64),
        ("frame_shuffle_seed", C.c_uint64), ("chunk_bytes", C.c_int64),
        ("hbm_backing", C.c_void_p), ("host_backing", C.c_void_p),
        ("pack_cus", C.c_int32), ("reserved", C.c_int32),
    ]


class FlowPoolError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        self.status = status
        self.code = STATUS_NAMES.get(status, str(status))
        super().__init__(f"{where}: {self.code}: {message}")


_P = C.c_void_p
_i32p = C.POINTER(C.c_int32)
_i64p = C.POINTER(C.c_int64)
_u64p = C.POINTER(C.c_uint64)
_u8p = C.POINTER(C.c_uint8)

_SIGS = {
    "fp_abi_version": (C.c_int32, []),
    "fp_last_error": (C.c_char_p, []),
    "fp_config_init": (None, [C.POINTER(fp_pool_config)]),
    "pool_create": (C.c_int32, [C.POINTER(fp_pool_config), C.POINTER(_P)]),
    "pool_destroy": (C.c_int32, [_P]),
    "pool_write_sample": (C.c_int32, [_P, _i32p, C.c_int32, _i32p, _i32p, C.c_int32, _P, _u8p, _P, _u64p]),
    "pool_free_sample": (C.c_int32, [_P, C.c_uint64]),
    "plan_microbatches": (C.c_int32, [_P, _u64p, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                      _i32p, _i32p, _i64p, _i32p, _i64p, _P]),
    "plan_partition": (C.c_int32, [_i32p, _i64p, C.c_int32, C.c_int32, C.c_int32, C.c_int32, _i32p, _i32p, _i64p,
                                   _i32p]),
    "pack_microbatch": (C.c_int32, [_P, _u64p, C.c_int32, _P, C.c_int64, _P, C.c_int64, _P, _P,
                                    _i32p, _i32p, C.c_int32, _P]),
    "pack_microbatch_noalloc": (C.c_int32, [_P, _u64p, C.c_int32, _P, C.c_int64, _P, C.c_int64, _P, _P,
                                    _i32p, _i32p, C.c_int32, _P]),
    "pool_stats": (C.c_int32, [_P, _i64p, _i64p, _i64p]),
    "pool_sample_pages": (C.c_int32, [_P, C.c_uint64, _u64p, C.c_int32, _i32p]),
    "pool_sample_info": (C.c_int32, [_P, C.c_uint64, _i32p, _i32p, _i32p]),
    "pool_translate": (C.c_int32, [_P, C.c_uint64, _i32p, _u64p]),
    "pool_layout": (C.c_int32, [_P, _u64p, _u64p, _i64p]),
    "pool_reclaim": (C.c_int32, [_P, C.c_int32, _i64p]),
    "pool_release_captured": (C.c_int32, [_P, _u64p, C.c_int32]),
    "pool_forget_stream": (C.c_int32, [_P, _P]),
    "fp_copy_bytes": (C.c_int32, [_P, _P, C.c_int64, C.c_int32, _P]),
    "fp_gather_rows": (C.c_int32, [_P, C.c_int32, C.c_int32, _P, _P]),
    "pool_migrate": (C.c_int32, [_P, _u64p, C.c_int32, C.c_int32, _P, _i64p]),
    "alloc_candidates": (C.c_int32, [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32, _i32p, _i32p, _i32p,
                                     C.c_int32, _i32p]),
    "plan_allocation": (C.c_int32, [C.c_int32, _i32p, _i64p, _i64p, C.c_int64, _i32p, _i64p, _i64p, _i64p]),
    "plan_dynamic_packing": (C.c_int32, [_i32p, C.c_int32, C.c_int32, C.c_int32, C.c_int32, _i32p, _i32p,
                                         _i32p, _i32p, _i64p, _i32p, _i32p, _i32p]),
    "plan_pool_packing": (C.c_int32, [_P, _u64p, C.c_int32, C.c_int32, C.c_int32, C.c_int32, _i32p, _i32p,
                                      _i32p, _i32p, _i64p, _i32p, _i32p, _i32p]),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTED = tuple(_SIGS)


def _check(status: int, where: str) -> None:
    if status != FP_OK:
        raise FlowPoolError(status, where, _lib.fp_last_error().decode(errors="replace"))


def _arr(a, dtype, ptype):
    """Contiguous numpy array of ``dtype`` and a ctypes pointer to it (None if a is None)."""
    if a is None:
        return None, None
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ptype)


def _ptr(x) -> Optional[int]:
    """Device address of a torch tensor / integer / None. A tensor must live
    on the GPU or in pinned host memory: the kernels read and write it
    directly, and an ordinary CPU tensor's address would fault them."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not (x.is_cuda or x.is_pinned()):
        raise ValueError("tensor argument must be on the GPU or in pinned host memory")
    return int(x.data_ptr())


# Hidden size of each pool created through these bindings, to check buffer
# sizes before the kernels touch them (pools created elsewhere are not checked).
_HIDDEN = {}
_DEVICE = {}
# Caller-provided tier backings, kept alive while their pool exists.
_BACKING = {}


def _buf(x, nbytes: int, name: str, device: Optional[int] = None) -> Optional[int]:
    """Like ``_ptr``; a tensor must also be contiguous, hold ``nbytes`` and,
    if on a GPU, be on ``device`` (when given)."""
    if x is None or isinstance(x, int):
        return _ptr(x)
    if device is not None and x.is_cuda and x.device.index != device:
        raise ValueError(f"{name} is on cuda:{x.device.index}, the pool on cuda:{device}")
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if x.numel() * x.element_size() < nbytes:
        raise ValueError(f"{name} holds {x.numel() * x.element_size()} bytes, the call needs {nbytes}")
    return _ptr(x)


def _stream(s) -> Optional[int]:
    if s is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


# ------------------------------------------------------------------ entry points

def fp_abi_version() -> int:
    return int(_lib.fp_abi_version())


def fp_last_error() -> str:
    return _lib.fp_last_error().decode(errors="replace")


def pool_create(hidden: int, page_tokens: int, hbm_pages: int, host_pages: int = 0,
                alloc: str = "contig", vocab: int = 0, device: int = 0, gva_start: int = 0,
                max_samples: int = 0, meta_bytes: int = 0, frame_shuffle_seed: int = 0,
                chunk_bytes: int = 0, world_size: int = 1, rank: int = 0, pack_cus: int = 0,
                hbm_backing=None, host_backing=None) -> int:
    """Create a pool. ``hbm_backing`` / ``host_backing``: optional caller-owned
    memory for a tier (a device tensor / a pinned host tensor, or a raw address);
    the bindings keep a tensor alive until ``pool_destroy``."""
    cfg = fp_pool_config()
    _lib.fp_config_init(C.byref(cfg))
    cfg.hidden, cfg.page_tokens = hidden, page_tokens
    cfg.hbm_pages, cfg.host_pages = hbm_pages, host_pages
    cfg.alloc_policy = ALLOC_POLICIES[alloc] if isinstance(alloc, str) else int(alloc)
    cfg.device, cfg.vocab, cfg.gva_start = device, vocab, gva_start
    cfg.world_size, cfg.rank = world_size, rank
    cfg.max_samples, cfg.meta_bytes = max_samples, meta_bytes
    cfg.frame_shuffle_seed, cfg.chunk_bytes = frame_shuffle_seed, chunk_bytes
    cfg.pack_cus = pack_cus
    page_bytes = 2 * hidden * page_tokens
    cfg.hbm_backing = _buf(hbm_backing, max(hbm_pages, 0) * page_bytes, "hbm_backing")
    cfg.host_backing = _buf(host_backing, max(host_pages, 0) * page_bytes, "host_backing")
    out = _P()
    _check(_lib.pool_create(C.byref(cfg), C.byref(out)), "pool_create")
    _HIDDEN[int(out.value)] = hidden
    _DEVICE[int(out.value)] = device
    _BACKING[int(out.value)] = (hbm_backing, host_backing)
    return int(out.value)


def pool_destroy(pool: int) -> None:
    _check(_lib.pool_destroy(pool), "pool_destroy")
    _HIDDEN.pop(pool, None)
    _DEVICE.pop(pool, None)
    _BACKING.pop(pool, None)


def pool_write_sample(pool: int, text_ids, img_pos, img_ntok, vis_emb=None, page_tier_wish=None,
                      stream=None) -> int:
    t, tp = _arr(text_ids, np.int32, _i32p)
    p, pp = _arr(img_pos, np.int32, _i32p)
    v, vp = _arr(img_ntok, np.int32, _i32p)
    w, wp = _arr(page_tier_wish, np.uint8, _u8p)
    sid = C.c_uint64()
    rb = 2 * _HIDDEN.get(pool, 0)
    vis = _buf(vis_emb, int(v.sum(dtype=np.int64)) * rb if v is not None else 0, "vis_emb", _DEVICE.get(pool))
    _check(_lib.pool_write_sample(pool, tp, len(t), pp, vp, len(p), vis, wp, _stream(stream),
                                  C.byref(sid)), "pool_write_sample")
    return int(sid.value)


def pool_free_sample(pool: int, sample_id: int) -> None:
    _check(_lib.pool_free_sample(pool, sample_id), "pool_free_sample")


def pool_reclaim(pool: int, wait: bool = False) -> int:
    """Complete deferred frees whose packs are done (all, after waiting, if ``wait``).
    Returns the pages still deferred."""
    n = C.c_int64()
    _check(_lib.pool_reclaim(pool, 1 if wait else 0, C.byref(n)), "pool_reclaim")
    return int(n.value)


def pool_release_captured(pool: int, sample_ids) -> None:
    """End a captured pack's hold on its samples (once its graph will not be replayed again)."""
    ids, idp = _arr(sample_ids, np.uint64, _u64p)
    _check(_lib.pool_release_captured(pool, idp, len(ids)), "pool_release_captured")


def pool_forget_stream(pool: int, stream) -> None:
    """Before destroying ``stream``: the pool stops remembering it (an event stands in for its queued work)."""
    _check(_lib.pool_forget_stream(pool, _stream(stream)), "pool_forget_stream")


def pool_migrate(pool: int, sample_ids, tier: int, stream=None) -> int:
    """Move the samples' pages into ``tier`` (FP_TIER_HBM / FP_TIER_HOST). Returns pages moved."""
    ids, idp = _arr(sample_ids, np.uint64, _u64p)
    moved = C.c_int64()
    _check(_lib.pool_migrate(pool, idp, len(ids), tier, _stream(stream), C.byref(moved)), "pool_migrate")
    return int(moved.value)


def plan_microbatches(pool: int, sample_ids, capacity: int, n_mb: int, cost_k: int, stream=None,
                      policy: int = FP_PLAN_LPT):
    """Returns dict(assign, mb_tokens, mb_cost_scaled, mb_max_len, sample_cost_scaled)."""
    ids, idp = _arr(sample_ids, np.uint64, _u64p)
    n = len(ids)
    assign = np.empty(n, np.int32)
    tok = np.empty(n_mb, np.int32)
    cst = np.empty(n_mb, np.int64)
    mx = np.empty(n_mb, np.int32)
    sc = np.empty(n, np.int64)
    _check(_lib.plan_microbatches(pool, idp, n, capacity, n_mb, cost_k, policy,
                                  assign.ctypes.data_as(_i32p), tok.ctypes.data_as(_i32p),
                                  cst.ctypes.data_as(_i64p), mx.ctypes.data_as(_i32p),
                                  sc.ctypes.data_as(_i64p), _stream(stream)), "plan_microbatches")
    return dict(assign=assign, mb_tokens=tok, mb_cost_scaled=cst, mb_max_len=mx, sample_cost_scaled=sc)


def plan_partition(lengths, costs_scaled, capacity: int, n_mb: int, policy: int = FP_PLAN_LPT):
    """Host-only partition. Returns dict(assign, mb_tokens, mb_cost_scaled, mb_max_len)."""
    ln, lp = _arr(lengths, np.int32, _i32p)
    cs, cp = _arr(costs_scaled, np.int64, _i64p)
    n = len(ln)
    assign = np.empty(n, np.int32)
    tok = np.empty(n_mb, np.int32)
    cst = np.empty(n_mb, np.int64)
    mx = np.empty(n_mb, np.int32)
    _check(_lib.plan_partition(lp, cp, n, capacity, n_mb, policy, assign.ctypes.data_as(_i32p),
                               tok.ctypes.data_as(_i32p), cst.ctypes.data_as(_i64p),
                               mx.ctypes.data_as(_i32p)), "plan_partition")
    return dict(assign=assign, mb_tokens=tok, mb_cost_scaled=cst, mb_max_len=mx)


def _packing_call(fn, name, head, n, capacity, n_ranks, n_buckets):
    mb_of_seq = np.empty(n, np.int32)
    n_mb = C.c_int32()
    per = [np.empty(max(n, 1), t) for t in (np.int32, np.int32, np.int64, np.int32, np.int32, np.int32)]
    ptrs = [a.ctypes.data_as(_i64p if a.dtype == np.int64 else _i32p) for a in per]
    _check(fn(*head, n, capacity, n_ranks, n_buckets, mb_of_seq.ctypes.data_as(_i32p), C.byref(n_mb), *ptrs),
           name)
    m = n_mb.value
    keys = ("mb_tokens", "mb_max_len", "mb_cost_scaled", "mb_bucket", "mb_rank", "mb_slot")
    out = dict(mb_of_seq=mb_of_seq, n_mb=m)
    out.update({k: a[:m].copy() for k, a in zip(keys, per)})
    return out


def alloc_candidates(backbone: bool, devices: int, per_node: int, global_batch: int, layers: int):
    """Pruned (DP, TP, PP) configurations of one module, as a list of tuples."""
    n = C.c_int32()
    st = _lib.alloc_candidates(int(backbone), devices, per_node, global_batch, layers, None, None, None, 0,
                               C.byref(n))
    if st != FP_OK and n.value <= 0:
        _check(st, "alloc_candidates")
    cap = max(n.value, 1)
    dp, tp, pp = (np.empty(cap, np.int32) for _ in range(3))
    _check(_lib.alloc_candidates(int(backbone), devices, per_node, global_batch, layers,
                                 dp.ctypes.data_as(_i32p), tp.ctypes.data_as(_i32p), pp.ctypes.data_as(_i32p),
                                 cap, C.byref(n)), "alloc_candidates")
    return [(int(a), int(b), int(c)) for a, b, c in zip(dp[:n.value], tp[:n.value], pp[:n.value])]


def plan_allocation(modules, budget: int):
    """modules: encoders then the backbone, each a list of (tau, devices).
    Returns dict(choice, G, F, devices)."""
    nc = np.array([len(m) for m in modules], np.int32)
    tau = np.array([t for m in modules for t, _ in m], np.int64)
    cost = np.array([r for m in modules for _, r in m], np.int64)
    choice = np.empty(len(modules), np.int32)
    g, f, d = C.c_int64(), C.c_int64(), C.c_int64()
    _check(_lib.plan_allocation(len(modules), nc.ctypes.data_as(_i32p), tau.ctypes.data_as(_i64p),
                                cost.ctypes.data_as(_i64p), budget, choice.ctypes.data_as(_i32p),
                                C.byref(g), C.byref(f), C.byref(d)), "plan_allocation")
    return dict(choice=choice.tolist(), G=g.value, F=f.value, devices=d.value)


def plan_dynamic_packing(lengths, capacity: int, n_ranks: int, n_buckets: int):
    """Alg. 1 on host lengths. Returns dict(mb_of_seq, n_mb, mb_tokens, mb_max_len,
    mb_cost_scaled, mb_bucket, mb_rank, mb_slot)."""
    ln, lp = _arr(lengths, np.int32, _i32p)
    return _packing_call(_lib.plan_dynamic_packing, "plan_dynamic_packing", (lp,), len(ln), capacity,
                         n_ranks, n_buckets)


def plan_pool_packing(pool: int, sample_ids, capacity: int, n_ranks: int, n_buckets: int):
    """Alg. 1 on resident samples (their pool lengths); same result as plan_dynamic_packing."""
    ids, idp = _arr(sample_ids, np.uint64, _u64p)
    return _packing_call(_lib.plan_pool_packing, "plan_pool_packing", (pool, idp), len(ids), capacity,
                         n_ranks, n_buckets)


def pack_microbatch(pool: int, sample_ids, embed_table, vocab: int, out_emb, out_rows_cap: int,
                    out_cu_seqlens=None, out_position_ids=None, tier_mask: int = FP_TIER_MASK_ALL,
                    stream=None, _entry=None):
    """Enqueue the pack of ``sample_ids`` into ``out_emb``. Returns (n_tokens, max_seqlen)."""
    if isinstance(sample_ids, (list, tuple)):
        ids = idp = (C.c_uint64 * len(sample_ids))(*sample_ids)   # cheaper per call than a numpy round trip
    else:
        ids, idp = _arr(sample_ids, np.uint64, _u64p)
    n_tok = C.c_int32()
    mx = C.c_int32()
    rb = 2 * _HIDDEN.get(pool, 0)
    cap = max(int(out_rows_cap), 0)
    dev = _DEVICE.get(pool)
    entry = _lib.pack_microbatch if _entry is None else _entry
    _check(entry(pool, idp, len(ids), _buf(embed_table, max(int(vocab), 0) * rb, "embed_table", dev),
                 vocab, _buf(out_emb, cap * rb, "out_emb", dev), out_rows_cap,
                 _buf(out_cu_seqlens, 4 * (len(ids) + 1), "out_cu_seqlens", dev),
                 _buf(out_position_ids, 4 * cap, "out_position_ids", dev), C.byref(n_tok), C.byref(mx),
                 tier_mask, _stream(stream)), entry.__name__)
    return int(n_tok.value), int(mx.value)


def pack_microbatch_noalloc(pool: int, sample_ids, embed_table, vocab: int, out_emb, out_rows_cap: int,
                            out_cu_seqlens=None, out_position_ids=None, tier_mask: int = FP_TIER_MASK_ALL,
                            stream=None):
    """pack_microbatch through the entry point that allocates nothing. Returns (n_tokens, max_seqlen)."""
    return pack_microbatch(pool, sample_ids, embed_table, vocab, out_emb, out_rows_cap, out_cu_seqlens,
                           out_position_ids, tier_mask, stream, _entry=_lib.pack_microbatch_noalloc)


def fp_copy_bytes(src, dst, nbytes: int, row_bytes: int, stream=None) -> None:
    """Measurement aid: plain copy of ``nbytes`` from device ``src`` to ``dst`` with the pack's geometry."""
    _check(_lib.fp_copy_bytes(_buf(src, nbytes, "src", None), _buf(dst, nbytes, "dst", None), nbytes, row_bytes,
                              _stream(stream)), "fp_copy_bytes")


def fp_gather_rows(rows_src, n_rows: int, row_bytes: int, dst, stream=None) -> None:
    """Measurement aid: dst row r = the row at device address rows_src[r] & ~15 (a device int64
    tensor; bit 0 set marks an embedding-table row, read as the pack reads those)."""
    _check(_lib.fp_gather_rows(_buf(rows_src, 8 * n_rows, "rows_src", None), n_rows, row_bytes,
                               _buf(dst, n_rows * row_bytes, "dst", None), _stream(stream)), "fp_gather_rows")


def pool_stats(pool: int):
    a, b, c = C.c_int64(), C.c_int64(), C.c_int64()
    _check(_lib.pool_stats(pool, C.byref(a), C.byref(b), C.byref(c)), "pool_stats")
    return dict(free_hbm_pages=a.value, free_host_pages=b.value, n_samples=c.value)


def pool_sample_pages(pool: int, sample_id: int):
    n = C.c_int32()
    st = _lib.pool_sample_pages(pool, sample_id, None, 0, C.byref(n))
    if st != FP_OK and not (st == FP_EINVAL and n.value > 0):
        _check(st, "pool_sample_pages")
    out = np.empty(max(n.value, 1), np.uint64)
    _check(_lib.pool_sample_pages(pool, sample_id, out.ctypes.data_as(_u64p), len(out), C.byref(n)),
           "pool_sample_pages")
    return out[:n.value]


def pool_sample_info(pool: int, sample_id: int):
    a, b, c = C.c_int32(), C.c_int32(), C.c_int32()
    _check(_lib.pool_sample_info(pool, sample_id, C.byref(a), C.byref(b), C.byref(c)), "pool_sample_info")
    return dict(length=a.value, n_text=b.value, n_vis=c.value)


def pool_translate(pool: int, gva: int):
    t, ph = C.c_int32(), C.c_uint64()
    _check(_lib.pool_translate(pool, gva, C.byref(t), C.byref(ph)), "pool_translate")
    return int(t.value), int(ph.value)


def pool_layout(pool: int):
    rs = (C.c_uint64 * 2)()
    ss = (C.c_uint64 * 2)()
    pb = C.c_int64()
    _check(_lib.pool_layout(pool, rs, ss, C.byref(pb)), "pool_layout")
    return dict(region_start=list(rs), segment_start=list(ss), page_bytes=pb.value)
