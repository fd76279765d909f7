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


# Rows too many to draw on the host: row r of sample g is a row of a small
# seeded random base (which one depends on r and g) with its first four
# words set to (TAG_VIS, lo16(g), lo16(r), hi16(r)). The device generator and
# the host twin below produce the same bits.
PATTERN_BASE_ROWS = 97


def pattern_base(hidden: int, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng([seed, 0xBA5E])
    return rng.integers(0, 1 << 16, size=(PATTERN_BASE_ROWS, hidden), dtype=np.uint16)


def pattern_row(sample_index: int, r: int, hidden: int, seed: int = 0, base=None) -> np.ndarray:
    base = pattern_base(hidden, seed) if base is None else base
    row = base[(7 * r + sample_index) % PATTERN_BASE_ROWS].copy()
    row[:4] = (TAG_VIS, sample_index & 0xFFFF, r & 0xFFFF, (r >> 16) & 0xFFFF)
    return row


def pattern_rows_dev(sample_index: int, n_rows: int, hidden: int, seed: int = 0, block: int = 1 << 15,
                     device: str = "cuda"):
    """The same rows as ``pattern_row``, built on the GPU in blocks (int16 view)."""
    import torch

    def i16(x):                     # uint16 values (int64 tensor or int) -> int16 bits
        return ((x & 0xFFFF) ^ 0x8000) - 0x8000

    base = torch.from_numpy(pattern_base(hidden, seed).view(np.int16)).to(device)
    out = torch.empty((n_rows, hidden), dtype=torch.int16, device=device)
    for r0 in range(0, n_rows, block):
        r = torch.arange(r0, min(r0 + block, n_rows), dtype=torch.int64, device=device)
        blk = out[r0:r0 + r.numel()]
        blk.copy_(base[(7 * r + sample_index) % PATTERN_BASE_ROWS])
        blk[:, 0] = i16(TAG_VIS)
        blk[:, 1] = i16(sample_index)
        blk[:, 2] = i16(r).to(torch.int16)
        blk[:, 3] = i16(r >> 16).to(torch.int16)
    return out
