"""Pool oracle: GVA regions, page table, allocators, write / free / pack.
TEST INFRASTRUCTURE ONLY.

Follows Sec. 3.2 (unified memory pool):

- every pool location has a 64-bit global virtual address (GVA);
- the GVA space holds two disjoint contiguous regions, HBM first, then DRAM;
  each region spans world_size * max_size bytes from its start, and process i
  owns the half-open segment [start + i*max_size, start + (i+1)*max_size);
- at initialisation each process binds physical memory (possibly less than
  max_size) to its segment and page tables map GVA pages to physical memory
  in HBM or DRAM; translation is a local table lookup;
- producers write a sample's vision embeddings and text tokens into their own
  segment, with metadata that pairs them; the consumer reads microbatches by
  GVA without knowing where the bytes physically are.

Readings where the paper is silent: the DRAM
region starts where the HBM region ends; max_size of a tier is its page count
times the page size; a sample's visual rows (all images, in image order) fill
its own pages densely, the last page possibly partial, and pages are never
shared; text ids are kept as metadata and their rows come from the embedding
table at pack time; allocation is "contig" (lowest-index first-fit run of
consecutive pages in one tier, HBM before DRAM) or "scatter" (per page, a
LIFO free stack per tier that initially pops page 0 first; a per-page tier
wish is honoured unless that tier is full, then the other tier is used);
freeing pushes a sample's pages back last-page-first, so an equal-sized
write right after gets the same pages in the same order; allocation is
all-or-nothing.

The two allocation policies and the free order are readings (the paper
names no allocator). They are pinned by hand-worked sequences written from
them and by properties that state each reading without its algorithm: under
"contig" every write takes the lowest-index run of free pages found among
the pages no live sample's page list holds, and fails exactly when there is
none; under "scatter" a model that ranks the free pages of a tier by when
they were given back (no stacks) picks the same page for every write and
migration. Everything the pack reads through them (GVA -> page-table entry
-> frame) is pinned by placement independence as well: the pack equals the
plain definition whatever frames the allocator picks.

The physical memory here is a dict of numpy page frames per tier,
materialised only when written.
"""

from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

DEFAULT_GVA_START = 0x0000100000000000
TIER_HBM, TIER_HOST = 0, 1
MASK_HBM, MASK_HOST = 1, 2


class PoolError(Exception):
    """Raised with ``code`` in {"EINVAL", "ENOMEM", "ENOENT", "ECAPACITY"}."""

    def __init__(self, code: str, msg: str = ""):
        super().__init__(f"{code}: {msg}")
        self.code = code


class _Sample:
    __slots__ = ("text_ids", "img_pos", "img_ntok", "n_vis", "length", "pages")


class OraclePool:
    def __init__(self, hidden: int, page_tokens: int, hbm_pages: int, host_pages: int = 0,
                 alloc: str = "contig", vocab: Optional[int] = None,
                 gva_start: int = DEFAULT_GVA_START, world_size: int = 1, rank: int = 0,
                 frame_order: Optional[Sequence[Sequence[int]]] = None):
        if alloc not in ("contig", "scatter"):
            raise PoolError("EINVAL", "alloc policy")
        if not (0 <= rank < world_size):
            raise PoolError("EINVAL", "rank")
        self.hidden = hidden
        self.P = page_tokens
        self.rb = 2 * hidden
        self.pb = page_tokens * self.rb
        self.alloc = alloc
        self.vocab = vocab
        self.gva_start = gva_start
        self.n_pages = [int(hbm_pages), int(host_pages)]
        # Sec. 3.2: per tier, region [start, start + world_size*max_size);
        # this rank's segment [start + rank*max_size, start + (rank+1)*max_size).
        self.max_size = [n * self.pb for n in self.n_pages]
        self.region_start = [gva_start, gva_start + world_size * self.max_size[0]]
        self.region_end = [self.region_start[t] + world_size * self.max_size[t] for t in (0, 1)]
        self.seg_start = [self.region_start[t] + rank * self.max_size[t] for t in (0, 1)]
        self.seg_end = [self.seg_start[t] + self.max_size[t] for t in (0, 1)]
        # Page table: page-aligned GVA -> (tier, physical frame). Frames are
        # bound in order unless a frame order (any permutation) is given.
        self.page_table: Dict[int, tuple] = {}
        for t in (0, 1):
            order = list(range(self.n_pages[t])) if frame_order is None else list(frame_order[t])
            assert sorted(order) == list(range(self.n_pages[t]))
            for i in range(self.n_pages[t]):
                self.page_table[self.seg_start[t] + i * self.pb] = (t, order[i])
        self.frames: List[Dict[int, np.ndarray]] = [{}, {}]
        # Allocator state, indexed by page number inside the tier's segment.
        self.used = [[False] * self.n_pages[0], [False] * self.n_pages[1]]
        self.stack = [list(range(self.n_pages[0] - 1, -1, -1)),
                      list(range(self.n_pages[1] - 1, -1, -1))]
        self.samples: Dict[int, _Sample] = {}
        self.next_id = 1

    # ------------------------------------------------------------ addressing
    def page_gva(self, tier: int, index: int) -> int:
        return self.seg_start[tier] + index * self.pb

    def _page_of(self, gva: int):
        for t in (0, 1):
            if self.seg_start[t] <= gva < self.seg_end[t]:
                return t, (gva - self.seg_start[t]) // self.pb
        raise PoolError("EINVAL", f"GVA {gva:#x} outside this rank's segments")

    def translate(self, gva: int):
        """GVA -> (tier, frame, byte offset inside the frame)."""
        base = self.gva_start + ((gva - self.gva_start) // self.pb) * self.pb
        if base not in self.page_table:
            raise PoolError("EINVAL", f"GVA {gva:#x} not mapped")
        tier, frame = self.page_table[base]
        return tier, frame, gva - base

    # ------------------------------------------------------------ allocation
    def _alloc_contig(self, n: int) -> List[int]:
        for t in (0, 1):
            used = self.used[t]
            run = 0
            for i in range(self.n_pages[t]):
                run = 0 if used[i] else run + 1
                if run == n:
                    first = i - n + 1
                    for j in range(first, i + 1):
                        used[j] = True
                    return [self.page_gva(t, j) for j in range(first, i + 1)]
        raise PoolError("ENOMEM", f"no run of {n} free pages")

    def _alloc_scatter(self, n: int, wish: Optional[Sequence[int]]) -> List[int]:
        left = [len(self.stack[0]), len(self.stack[1])]
        tiers = []
        for j in range(n):
            t = int(wish[j]) if wish is not None else TIER_HBM
            if left[t] == 0:
                t = 1 - t
            if left[t] == 0:
                raise PoolError("ENOMEM", f"{n} pages do not fit")
            left[t] -= 1
            tiers.append(t)
        out = []
        for t in tiers:
            i = self.stack[t].pop()
            self.used[t][i] = True
            out.append(self.page_gva(t, i))
        return out

    # ------------------------------------------------------------ producer
    def write(self, text_ids, img_pos, img_ntok, vis_rows: Optional[np.ndarray] = None,
              tier_wish: Optional[Sequence[int]] = None) -> int:
        text_ids = np.asarray(text_ids, dtype=np.int64)
        img_pos = [int(p) for p in img_pos]
        img_ntok = [int(v) for v in img_ntok]
        T = len(text_ids)
        if len(img_pos) != len(img_ntok):
            raise PoolError("EINVAL", "image arrays differ in length")
        for j, p in enumerate(img_pos):
            if p < 0 or p > T or (j and p < img_pos[j - 1]):
                raise PoolError("EINVAL", "placeholder positions")
        if any(v < 0 for v in img_ntok):
            raise PoolError("EINVAL", "negative image token count")
        if self.vocab is not None and T and (text_ids.min() < 0 or text_ids.max() >= self.vocab):
            raise PoolError("EINVAL", "text id outside the vocabulary")
        n_vis = sum(img_ntok)
        if T + n_vis == 0:
            raise PoolError("EINVAL", "empty sample")
        if vis_rows is not None and vis_rows.shape != (n_vis, self.hidden):
            raise PoolError("EINVAL", "visual rows shape")
        n_pages = -(-n_vis // self.P)
        if tier_wish is not None:
            if self.alloc == "contig" or len(tier_wish) != n_pages:
                raise PoolError("EINVAL", "tier wishes")
        pages = self._alloc_contig(n_pages) if self.alloc == "contig" and n_pages \
            else (self._alloc_scatter(n_pages, tier_wish) if n_pages else [])
        s = _Sample()
        s.text_ids = text_ids.astype(np.int32)
        s.img_pos, s.img_ntok, s.n_vis, s.length, s.pages = img_pos, img_ntok, n_vis, T + n_vis, pages
        if vis_rows is not None:
            for v in range(n_vis):
                gva = pages[v // self.P] + (v % self.P) * self.rb
                tier, frame, off = self.translate(gva)
                page = self.frames[tier].get(frame)
                if page is None:
                    page = np.zeros((self.P, self.hidden), dtype=np.uint16)
                    self.frames[tier][frame] = page
                page[off // self.rb] = vis_rows[v]
        sid = self.next_id
        self.next_id += 1
        self.samples[sid] = s
        return sid

    def free(self, sid: int) -> None:
        s = self.samples.pop(sid, None)
        if s is None:
            raise PoolError("ENOENT", f"sample {sid}")
        for gva in reversed(s.pages):
            t, i = self._page_of(gva)
            self.used[t][i] = False
            if self.alloc == "scatter":
                self.stack[t].append(i)

    def migrate(self, sid: int, tier: int) -> int:
        """Move every page of sample ``sid`` that is not in ``tier`` into a
        page of ``tier`` (a tier promotion or demotion, Sec. 3.2: the pool
        spans HBM and DRAM, and data moves between them by the transport the
        pair of tiers calls for). Scatter pools only. The moving pages, in
        visual-row order, each take the next page popped from the tier's
        stack and keep their bytes; the pages they leave go back to their
        stacks last-page-first, as in a free. All-or-nothing. Returns the
        number of pages moved."""
        s = self.samples.get(sid)
        if s is None:
            raise PoolError("ENOENT", f"sample {sid}")
        if self.alloc != "scatter" or tier not in (TIER_HBM, TIER_HOST):
            raise PoolError("EINVAL", "migration needs the scatter policy and a tier")
        moving = [k for k, gva in enumerate(s.pages) if self._page_of(gva)[0] != tier]
        if len(moving) > len(self.stack[tier]):
            raise PoolError("ENOMEM", f"{len(moving)} pages do not fit in tier {tier}")
        old = [s.pages[k] for k in moving]
        pages = list(s.pages)
        for k in moving:
            i = self.stack[tier].pop()
            self.used[tier][i] = True
            new = self.page_gva(tier, i)
            ot, of, _ = self.translate(pages[k])
            nt, nf, _ = self.translate(new)
            if of in self.frames[ot]:
                self.frames[nt][nf] = self.frames[ot][of].copy()
            else:
                self.frames[nt].pop(nf, None)
            pages[k] = new
        for gva in reversed(old):
            t, i = self._page_of(gva)
            self.used[t][i] = False
            self.stack[t].append(i)
        s.pages = pages
        return len(moving)

    # ------------------------------------------------------------ consumer
    def _rows_of(self, s: _Sample):
        """Row sources of one sample, token by token: before text token t come
        the images whose placeholder is t (in image order); images placed at
        T come after the last text token."""
        v = 0
        j = 0
        k = len(s.img_pos)
        for t in range(len(s.text_ids) + 1):
            while j < k and s.img_pos[j] == t:
                for _ in range(s.img_ntok[j]):
                    yield ("vis", v)
                    v += 1
                j += 1
            if t < len(s.text_ids):
                yield ("text", int(s.text_ids[t]))

    def _read_row(self, s: _Sample, v: int) -> np.ndarray:
        gva = s.pages[v // self.P] + (v % self.P) * self.rb
        tier, frame, off = self.translate(gva)
        page = self.frames[tier].get(frame)
        if page is None:
            return np.zeros(self.hidden, dtype=np.uint16)
        return page[off // self.rb]

    def row_tier(self, sid: int, v: int) -> int:
        s = self.samples[sid]
        return self.translate(s.pages[v // self.P])[0]

    def pack(self, ids: Sequence[int], table: Optional[np.ndarray], out_rows_cap: Optional[int] = None,
             tier_mask: int = MASK_HBM | MASK_HOST, out: Optional[np.ndarray] = None):
        """Resolve and copy every row of the microbatch ``ids`` (in order).

        Returns (rows, cu_seqlens, position_ids, n_tokens, max_seqlen). With a
        tier mask, only text rows and HBM-page rows (MASK_HBM) and/or
        DRAM-page rows (MASK_HOST) are written into ``out``; cu_seqlens and
        position ids are produced when MASK_HBM is set, else returned as None.
        """
        recs = []
        for sid in ids:
            if sid not in self.samples:
                raise PoolError("ENOENT", f"sample {sid}")
            recs.append(self.samples[sid])
        total = sum(s.length for s in recs)
        if out_rows_cap is not None and total > out_rows_cap:
            raise PoolError("ECAPACITY", f"{total} rows > {out_rows_cap}")
        if out is None:
            out = np.zeros((total, self.hidden), dtype=np.uint16)
        cu = [0]
        pos = []
        r = 0
        for s in recs:
            local = 0
            for kind, x in self._rows_of(s):
                if kind == "text":
                    if tier_mask & MASK_HBM:
                        out[r] = table[x]
                else:
                    tier = self.translate(s.pages[x // self.P])[0]
                    want = MASK_HBM if tier == TIER_HBM else MASK_HOST
                    if tier_mask & want:
                        out[r] = self._read_row(s, x)
                pos.append(local)
                local += 1
                r += 1
            cu.append(r)
        max_len = max((s.length for s in recs), default=0)
        if tier_mask & MASK_HBM:
            return out, np.array(cu, dtype=np.int32), np.array(pos, dtype=np.int32), total, max_len
        return out, None, None, total, max_len

    # ------------------------------------------------------------ introspection
    def sample_pages(self, sid: int) -> List[int]:
        if sid not in self.samples:
            raise PoolError("ENOENT", f"sample {sid}")
        return list(self.samples[sid].pages)

    def sample_length(self, sid: int) -> int:
        return self.samples[sid].length

    def free_pages(self):
        return [self.used[t].count(False) for t in (0, 1)]
