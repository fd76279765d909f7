"""Tagged-rows inputs: every visual row names its sample and visual index and
every table row names its token id in the first four 16-bit words (NaN bit
patterns, so a copy through floating point would corrupt them); the remaining
words are random bits."""

import numpy as np

from paper_2606_23087_amd.workloads import TAG_TEXT, TAG_VIS


def tagged_table(vocab: int, hidden: int, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng([seed, 0x7A6])
    t = rng.integers(0, 1 << 16, size=(vocab, hidden), dtype=np.uint16)
    ids = np.arange(vocab, dtype=np.int64)
    t[:, 0] = TAG_TEXT
    t[:, 1] = (ids & 0xFFFF).astype(np.uint16)
    t[:, 2] = ((ids >> 16) & 0xFFFF).astype(np.uint16)
    t[:, 3] = 0
    return t


def tagged_vis(sample_index: int, n_vis: int, hidden: int, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng([seed, 0x715, sample_index])
    r = rng.integers(0, 1 << 16, size=(n_vis, hidden), dtype=np.uint16)
    r[:, 0] = TAG_VIS
    r[:, 1] = sample_index & 0xFFFF
    r[:, 2] = (sample_index >> 16) & 0xFFFF
    r[:, 3] = np.arange(n_vis, dtype=np.int64).astype(np.uint16)
    return r


def decode(rows: np.ndarray):
    """Row tags -> [("text", id) | ("vis", sample_index, visual_index_lo16) | ("?",)]."""
    out = []
    for r in rows:
        if r[0] == TAG_TEXT:
            out.append(("text", int(r[1]) | (int(r[2]) << 16)))
        elif r[0] == TAG_VIS:
            out.append(("vis", int(r[1]) | (int(r[2]) << 16), int(r[3])))
        else:
            out.append(("?",))
    return out
