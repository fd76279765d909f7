"""Seeded synthetic inputs for the paged translate-gather-pack workloads.

This module only draws inputs: sample shapes (text lengths, image counts,
visual-token counts, placeholder positions), text ids, visual embeddings,
embedding tables, per-page tier draws and the churn op sequence that
fragments a pool. It performs none of the method's arithmetic (no layout,
no page walk, no packing, no cost, no partition), so both the oracle and the
HIP path can be fed from it without sharing code.

The paper's datasets (InfoVQA and an internal e-commerce set, Sec. 4.1) are
not available; these generators stand in for them with the shapes the paper
states (interleaved image/text subsequences up to 8192 tokens, mixed-size
images, Sec. 2 and Sec. 4.1) and the five workload configurations below.

Streams: every workload seed s spawns independent numpy PCG64 streams from
``numpy.random.SeedSequence(s)`` for lengths, images, positions, ids, churn,
tiers, and derives per-sample embedding streams from (s, sample index).
"""

from __future__ import annotations

import dataclasses
import math
from typing import Iterator, List, Optional, Sequence

import numpy as np

# Stream indices inside SeedSequence(seed).spawn(N_STREAMS).
_S_LEN, _S_IMG, _S_POS, _S_IDS, _S_CHURN, _S_TIER = range(6)
_N_STREAMS = 6

# Tag words used by the tagged-rows input mode (NaN bit patterns on purpose,
# so a copy that goes through floating point would corrupt them).
TAG_VIS = 0xFFC1
TAG_TEXT = 0xFFC2


@dataclasses.dataclass(frozen=True)
class WorkloadConfig:
    name: str
    hidden: int                 # H (bf16 elements per row)
    page_tokens: int            # P (rows per page)
    hbm_pages: int
    host_pages: int
    alloc: str                  # "contig" | "scatter"
    vocab: int
    table_std: float
    capacity: int               # C, tokens per microbatch
    n_mb: int                   # M, microbatches per plan
    cost_k: int                 # K of the per-sample cost l + l^2/K
    # sample shape
    img_count: tuple            # (lo, hi) inclusive number of images per sample
    img_tokens: tuple           # (lo, hi, step) visual tokens per image
    text_dist: str              # "uniform" | "lognormal"
    text_params: tuple          # uniform: (lo, hi); lognormal: (median, sigma, lo, hi)
    video_frames: Optional[tuple] = None   # (lo, hi, tokens_per_frame): one segment
    fixed_samples: Optional[int] = None    # exact sample count (else fill to M*C)
    churn_steps: int = 0
    churn_target_occupancy: float = 0.5
    tier_split: bool = False    # per-page Bernoulli(0.5) tier draw

    @property
    def row_bytes(self) -> int:
        return 2 * self.hidden

    @property
    def page_bytes(self) -> int:
        return self.page_tokens * self.row_bytes


CONFIGS = {
    # Tiny correctness case: H 256, 16-token pages, 1024 HBM pages.
    "tiny": WorkloadConfig(
        name="tiny", hidden=256, page_tokens=16, hbm_pages=1024, host_pages=0,
        alloc="contig", vocab=1000, table_std=1.0, capacity=512, n_mb=2,
        cost_k=4096, img_count=(1, 1), img_tokens=(64, 64, 1),
        text_dist="uniform", text_params=(32, 128), fixed_samples=8),
    # Qwen-style VLM backbone, H 3584: the headline bandwidth workload.
    "qwen": WorkloadConfig(
        name="qwen", hidden=3584, page_tokens=64, hbm_pages=32768, host_pages=0,
        alloc="contig", vocab=152064, table_std=0.02, capacity=16384, n_mb=64,
        cost_k=8192, img_count=(1, 4), img_tokens=(256, 1280, 4),
        text_dist="lognormal", text_params=(400.0, 0.8, 16, 4096)),
    # 70B-class backbone, H 8192, 24 GiB pool of 32-token pages fragmented by
    # 10k write/free churn steps.
    "frag70b": WorkloadConfig(
        name="frag70b", hidden=8192, page_tokens=32, hbm_pages=49152, host_pages=0,
        alloc="scatter", vocab=152064, table_std=0.02, capacity=32768, n_mb=16,
        cost_k=4096, img_count=(1, 6), img_tokens=(196, 1024, 1),
        text_dist="lognormal", text_params=(600.0, 1.0, 16, 8192),
        churn_steps=10000),
    # Video-heavy long context, H 5120, 128-token pages.
    "video": WorkloadConfig(
        name="video", hidden=5120, page_tokens=128, hbm_pages=16384, host_pages=0,
        alloc="contig", vocab=128256, table_std=0.02, capacity=65536, n_mb=16,
        cost_k=4096, img_count=(1, 1), img_tokens=(0, 0, 1),
        text_dist="uniform", text_params=(64, 2048), video_frames=(8, 32, 256)),
    # Tiered pool, H 4096: half the pages in HBM, half in pinned host memory.
    "tiered": WorkloadConfig(
        name="tiered", hidden=4096, page_tokens=64, hbm_pages=8192, host_pages=8192,
        alloc="scatter", vocab=152064, table_std=0.02, capacity=16384, n_mb=16,
        cost_k=8192, img_count=(1, 4), img_tokens=(256, 1024, 1),
        text_dist="lognormal", text_params=(512.0, 0.8, 16, 4096), tier_split=True),
}

CONFIG_ORDER = ["tiny", "qwen", "frag70b", "video", "tiered"]


def scaled(cfg: WorkloadConfig, **kw) -> WorkloadConfig:
    """A copy of ``cfg`` with some fields replaced (small parity cases)."""
    return dataclasses.replace(cfg, **kw)


@dataclasses.dataclass
class SampleSpec:
    """One producer sample: text ids plus images at placeholder positions."""
    text_ids: np.ndarray        # int32 [T]
    img_pos: np.ndarray         # int32 [k], nondecreasing, each in [0, T]
    img_ntok: np.ndarray        # int32 [k]

    @property
    def n_text(self) -> int:
        return int(self.text_ids.shape[0])

    @property
    def n_vis(self) -> int:
        return int(self.img_ntok.sum()) if self.img_ntok.size else 0

    @property
    def length(self) -> int:
        return self.n_text + self.n_vis


def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(_N_STREAMS)]


def round_half_up(x: float) -> int:
    return int(math.floor(x + 0.5))


def _draw_text_len(cfg: WorkloadConfig, rng: np.random.Generator) -> int:
    if cfg.text_dist == "uniform":
        lo, hi = cfg.text_params
        return int(rng.integers(lo, hi + 1))
    median, sigma, lo, hi = cfg.text_params
    v = round_half_up(math.exp(rng.normal(math.log(median), sigma)))
    return int(min(max(v, lo), hi))


def _draw_images(cfg: WorkloadConfig, rng: np.random.Generator) -> np.ndarray:
    if cfg.video_frames is not None:
        flo, fhi, per = cfg.video_frames
        return np.array([int(rng.integers(flo, fhi + 1)) * per], dtype=np.int32)
    clo, chi = cfg.img_count
    k = int(rng.integers(clo, chi + 1))
    lo, hi, step = cfg.img_tokens
    nsteps = (hi - lo) // step
    return np.array([lo + step * int(rng.integers(0, nsteps + 1)) for _ in range(k)],
                    dtype=np.int32)


class SampleStream:
    """Draws samples of one workload in a fixed seeded order."""

    def __init__(self, cfg: WorkloadConfig, seed: int, stream_offset: int = 0):
        self.cfg = cfg
        rs = _streams(seed * 1000003 + stream_offset)
        self._len, self._img, self._pos, self._ids = rs[_S_LEN], rs[_S_IMG], rs[_S_POS], rs[_S_IDS]

    def next(self, constant_ids: bool = False) -> SampleSpec:
        cfg = self.cfg
        t = _draw_text_len(cfg, self._len)
        ntok = _draw_images(cfg, self._img)
        pos = np.sort(self._pos.integers(0, t + 1, size=ntok.shape[0])).astype(np.int32)
        if constant_ids:
            ids = np.zeros(t, dtype=np.int32)
        else:
            ids = self._ids.integers(0, cfg.vocab, size=t).astype(np.int32)
        return SampleSpec(text_ids=ids, img_pos=pos, img_ntok=ntok)


def gen_samples(cfg: WorkloadConfig, seed: int, min_tokens: Optional[int] = None,
                count: Optional[int] = None) -> List[SampleSpec]:
    """Samples in write order: ``count`` of them, else ``cfg.fixed_samples``,
    else as many as it takes for their total length to reach ``min_tokens``
    (default M*C: the producer has accumulated enough for one plan)."""
    st = SampleStream(cfg, seed)
    if count is None:
        count = cfg.fixed_samples
    out: List[SampleSpec] = []
    if count is not None:
        return [st.next() for _ in range(count)]
    if min_tokens is None:
        min_tokens = cfg.n_mb * cfg.capacity
    total = 0
    while total < min_tokens:
        s = st.next()
        out.append(s)
        total += s.length
    return out


def schedule_lengths(seed: int, capacity: int, tokens: int, cfg_name: str = "qwen") -> np.ndarray:
    """Sequence lengths for the dynamic packing scheduler: the lengths (text
    plus image rows) of one workload's samples in write order, clipped to the
    capacity, until their sum reaches ``tokens``."""
    st = SampleStream(CONFIGS[cfg_name], seed)
    out: List[int] = []
    total = 0
    while total < tokens:
        length = min(st.next().length, capacity)
        out.append(length)
        total += length
    return np.array(out, dtype=np.int32)


def allocator_tables(seed: int, devices: int, per_node: int = 8, global_batch: int = 512, layers: int = 28,
                     n_encoders: int = 2, candidates_fn=None):
    """Stand-in for the allocator's profiled throughput surrogates: for each
    module (the encoders, then the backbone) a list of (tau, devices) over its
    candidate configurations. tau (integer tokens/s) grows with data
    parallelism, sublinearly with tensor parallelism, and with pipeline
    parallelism less a pipeline bubble, times a seeded +-10 % perturbation.
    ``candidates_fn(backbone, devices, per_node, global_batch, layers)`` lists
    the configurations."""
    rng = np.random.default_rng([seed, 0xA11C])
    mods = []
    for m in range(n_encoders + 1):
        backbone = m == n_encoders
        base = 9000.0 if backbone else 40000.0 / (m + 1)
        out = []
        for dp, tp, pp in candidates_fn(backbone, devices, per_node, global_batch, layers):
            t = base * dp * tp ** 0.82
            if backbone:
                t *= pp ** 0.92 / (1.0 + (pp - 1) / 16.0)
            t *= 1.0 + 0.1 * (2.0 * rng.random() - 1.0)
            out.append((int(round(t)), dp * tp * pp))
        mods.append(out)
    return mods


# ---------------------------------------------------------------- embeddings

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (input generation)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    out = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def _emb_seed(seed: int, sample_index: int) -> list:
    return [int(seed), 0xE3B, int(sample_index)]


def visual_rows_np(cfg: WorkloadConfig, seed: int, sample_index: int, n_vis: int,
                   mode: str = "normal") -> np.ndarray:
    """uint16 [n_vis, H] bf16 bit patterns for one sample's images (concatenated
    in image order). Modes: "normal" N(0,1) -> bf16; "bits" all 65536 patterns
    uniformly; "tagged" = "bits" with the first four words holding
    (TAG_VIS, lo16(sample), hi16(sample), visual index)."""
    rng = np.random.default_rng(_emb_seed(seed, sample_index))
    h = cfg.hidden
    if mode == "normal":
        rows = f32_to_bf16_bits(rng.standard_normal((n_vis, h), dtype=np.float32))
    else:
        rows = rng.integers(0, 1 << 16, size=(n_vis, h), dtype=np.uint16)
    if mode == "tagged":
        assert n_vis < (1 << 16)
        rows[:, 0] = TAG_VIS
        rows[:, 1] = sample_index & 0xFFFF
        rows[:, 2] = (sample_index >> 16) & 0xFFFF
        rows[:, 3] = np.arange(n_vis, dtype=np.uint16)
    return rows


def table_np(cfg: WorkloadConfig, seed: int, mode: str = "normal") -> np.ndarray:
    """uint16 [vocab, H] embedding table. "tagged" rows hold
    (TAG_TEXT, lo16(id), hi16(id), 0) in their first four words."""
    rng = np.random.default_rng([int(seed), 0x7AB])
    if mode == "normal":
        t = f32_to_bf16_bits(rng.normal(0.0, cfg.table_std,
                                        size=(cfg.vocab, cfg.hidden)).astype(np.float32))
    else:
        t = rng.integers(0, 1 << 16, size=(cfg.vocab, cfg.hidden), dtype=np.uint16)
    if mode == "tagged":
        ids = np.arange(cfg.vocab, dtype=np.int64)
        t[:, 0] = TAG_TEXT
        t[:, 1] = (ids & 0xFFFF).astype(np.uint16)
        t[:, 2] = ((ids >> 16) & 0xFFFF).astype(np.uint16)
        t[:, 3] = 0
    return t


def visual_rows_torch(cfg: WorkloadConfig, seed: int, sample_index: int, n_vis: int,
                      device="cuda"):
    """Device-side N(0,1) -> bf16 rows for full-size workloads (torch's own
    generator; the same call returns the same bytes on the same device)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((int(seed) * 0x9E3779B1 + int(sample_index) * 0x85EBCA6B + 0xE3B) & ((1 << 63) - 1))
    x = torch.randn((n_vis, cfg.hidden), generator=g, device=device, dtype=torch.float32)
    return x.to(torch.bfloat16)


def table_torch(cfg: WorkloadConfig, seed: int, device="cuda"):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((int(seed) * 0x27D4EB2F + 0x7AB) & ((1 << 63) - 1))
    t = torch.empty((cfg.vocab, cfg.hidden), device=device, dtype=torch.float32)
    t.normal_(0.0, cfg.table_std, generator=g)
    return t.to(torch.bfloat16)


# ------------------------------------------------------------- tier draws

def page_tier_draws(seed: int, sample_index: int, n_pages: int) -> np.ndarray:
    """Per-page tier wish, Bernoulli(0.5): 0 = HBM, 1 = pinned host."""
    rng = np.random.default_rng([int(seed), 0x71E, int(sample_index)])
    return rng.integers(0, 2, size=n_pages).astype(np.uint8)


# ------------------------------------------------------------- churn

@dataclasses.dataclass
class ChurnOp:
    kind: str                  # "write" | "free"
    key: int                   # churn ordinal of the sample written / freed
    spec: Optional[SampleSpec] = None


def churn_ops(cfg: WorkloadConfig, seed: int, steps: Optional[int] = None,
              total_pages: Optional[int] = None) -> List[ChurnOp]:
    """Write/free op sequence that fragments a pool before measurement.

    Each step flips a fair coin: write a new churn sample (first freeing
    uniformly chosen residents while its page count does not fit in the free
    page count) or free a uniformly chosen resident (a write if none is
    resident). Afterwards residents are freed at random until at most
    ``churn_target_occupancy`` of the pages are in use. Churn samples carry
    constant text ids and no visual payload. The page count a sample needs,
    ceil(visual tokens / P), only keeps the sequence feasible; which pages
    it gets is up to the pool under test.
    """
    if steps is None:
        steps = cfg.churn_steps
    if total_pages is None:
        total_pages = cfg.hbm_pages + cfg.host_pages
    rng = _streams(seed)[_S_CHURN]
    st = SampleStream(cfg, seed, stream_offset=0xC4)
    ops: List[ChurnOp] = []
    resident: List[tuple] = []     # (key, pages)
    free = total_pages
    key = 0
    for _ in range(steps):
        write = bool(rng.integers(0, 2) == 0) or not resident
        if write:
            spec = st.next(constant_ids=True)
            need = -(-spec.n_vis // cfg.page_tokens)
            if need > total_pages:
                continue
            while free < need:
                i = int(rng.integers(0, len(resident)))
                k, pg = resident.pop(i)
                ops.append(ChurnOp("free", k))
                free += pg
            ops.append(ChurnOp("write", key, spec))
            resident.append((key, need))
            free -= need
            key += 1
        else:
            i = int(rng.integers(0, len(resident)))
            k, pg = resident.pop(i)
            ops.append(ChurnOp("free", k))
            free += pg
    limit = int(cfg.churn_target_occupancy * total_pages)
    while resident and (total_pages - free) > limit:
        i = int(rng.integers(0, len(resident)))
        k, pg = resident.pop(i)
        ops.append(ChurnOp("free", k))
        free += pg
    return ops
