"""Definitional packed microbatch (no pool, no pages). TEST INFRASTRUCTURE ONLY.

What a packed microbatch is, written out plainly:

- Sec. 3.1: text tokens and vision embeddings of a sample are paired through
  metadata kept with the pool; the backbone consumes whole microbatches.
- Sec. 4.1: a training sequence interleaves the sample's image and text
  subsequences.
- Sec. 3.4: variable-length sequences are packed back to back into one
  fixed-capacity microbatch; the per-sequence boundaries (cu_seqlens) are
  what a varlen attention kernel consumes.

Readings taken where the paper is silent:
an image placeholder at text position p sits before text token p and
consumes no text token; images at equal positions keep their order; a text
row is the embedding-table row of its id; position ids restart at 0 for each
sample; no padding rows are produced.
"""

from __future__ import annotations

from typing import List, Sequence

import numpy as np


def sample_segments(n_text: int, img_pos: Sequence[int], img_ntok: Sequence[int]):
    """The sample's subsequences in order: ("text", first text index, count)
    and ("vis", first visual index, count). Text runs are cut at the sorted
    placeholder positions p_1 <= ... <= p_k: text[0:p_1], image 1,
    text[p_1:p_2], image 2, ..., image k, text[p_k:T]. Visual indices run over
    the sample's images concatenated in image order."""
    k = len(img_pos)
    bounds = [0] + [int(p) for p in img_pos] + [int(n_text)]
    segs = []
    vis_start = 0
    for j in range(k + 1):
        segs.append(("text", bounds[j], bounds[j + 1] - bounds[j]))
        if j < k:
            segs.append(("vis", vis_start, int(img_ntok[j])))
            vis_start += int(img_ntok[j])
    return segs


def definitional_pack(samples, vis_rows: List[np.ndarray], table: np.ndarray):
    """Pack ``samples`` (in the given order) into one microbatch.

    samples[i] has ``text_ids`` (int32 [T]), ``img_pos`` (int32 [k],
    nondecreasing, in [0, T]) and ``img_ntok`` (int32 [k]); vis_rows[i] is a
    uint16 [sum(img_ntok), H] array of the sample's image rows; table is the
    uint16 [vocab, H] embedding table.

    Returns (rows uint16 [N, H], cu_seqlens int32 [n+1], position_ids int32 [N],
    max_seqlen int).
    """
    h = table.shape[1]
    parts = []
    cu = [0]
    pos = []
    max_len = 0
    for s, spec in enumerate(samples):
        sample_parts = []
        for kind, start, count in sample_segments(len(spec.text_ids), spec.img_pos, spec.img_ntok):
            if count == 0:
                continue
            if kind == "text":
                ids = np.asarray(spec.text_ids[start:start + count], dtype=np.int64)
                sample_parts.append(table[ids])
            else:
                sample_parts.append(vis_rows[s][start:start + count])
        length = sum(p.shape[0] for p in sample_parts)
        parts.extend(sample_parts)
        cu.append(cu[-1] + length)
        pos.extend(range(length))
        max_len = max(max_len, length)
    rows = np.concatenate(parts) if parts else np.zeros((0, h), dtype=np.uint16)
    return (rows.astype(np.uint16, copy=False), np.array(cu, dtype=np.int32),
            np.array(pos, dtype=np.int32), max_len)


def row_sources(samples):
    """Symbolic source of every packed row, in order:
    ("text", sample index, token id) or ("vis", sample index, visual index).
    Same layout as ``definitional_pack`` without touching any bytes, so it can
    describe microbatches of any size."""
    out = []
    for s, spec in enumerate(samples):
        for kind, start, count in sample_segments(len(spec.text_ids), spec.img_pos, spec.img_ntok):
            for i in range(start, start + count):
                if kind == "text":
                    out.append(("text", s, int(spec.text_ids[i])))
                else:
                    out.append(("vis", s, i))
    return out
