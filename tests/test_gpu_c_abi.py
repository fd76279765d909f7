"""The C ABI driven from plain C: `tests/c_abi/pack_driver` (built by
build(), linked only against libflowpool.so and the HIP runtime; no Python,
no torch in that process) writes samples into a pool, plans with
plan_microbatches and packs every microbatch with pack_microbatch (every
odd-numbered one with pack_microbatch_noalloc). Its output must equal the
oracle's plan and definitional pack, bit for bit.

The workload is the tiny configuration's samples plus hand-made edge
samples: text only, image only, adjacent images, an empty image, an image
at each end.
"""

import os
import struct
import subprocess

import numpy as np
import pytest

from gpu_common import say
from oracle.pack import definitional_pack
from oracle.plan import greedy_partition, members
from paper_2606_23087_amd.workloads import CONFIGS, SampleSpec, gen_samples, table_np, visual_rows_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DRIVER = os.path.join(ROOT, "tests", "c_abi", "pack_driver")


def _edge_specs(vocab):
    i32 = lambda x: np.asarray(x, np.int32)
    return [SampleSpec(i32([1, 2, 3]), i32([]), i32([])),                  # text only
            SampleSpec(i32([]), i32([0]), i32([37])),                      # image only
            SampleSpec(i32([5, 6]), i32([1, 1, 1]), i32([3, 5, 7])),       # adjacent images
            SampleSpec(i32([7, 8, 9, 10]), i32([0, 2, 4]), i32([4, 0, 9])),  # empty image, images at both ends
            SampleSpec(i32(list(range(vocab - 5, vocab))), i32([5]), i32([16]))]


def _write_input(path, cfg, specs, table, vis):
    with open(path, "wb") as f:
        f.write(struct.pack("<7i", cfg.hidden, cfg.page_tokens, cfg.vocab, len(specs), cfg.capacity,
                            cfg.n_mb, cfg.cost_k))
        f.write(np.ascontiguousarray(table, "<u2").tobytes())
        for s, v in zip(specs, vis):
            f.write(struct.pack("<2i", len(s.text_ids), len(s.img_ntok)))
            for a in (s.text_ids, s.img_pos, s.img_ntok):
                f.write(np.ascontiguousarray(a, "<i4").tobytes())
            f.write(np.ascontiguousarray(v, "<u2").tobytes())


def _read_output(path, n, hidden):
    buf = open(path, "rb").read()
    off = 0

    def take(dtype, count):
        nonlocal off
        a = np.frombuffer(buf, dtype, count, off)
        off += a.nbytes
        return a

    n_mb = int(take("<i4", 1)[0])
    assign = take("<i4", n).tolist()
    mbs = []
    for _ in range(n_mb):
        n_tok, mx, k = take("<i4", 3).tolist()
        cu = take("<i4", k + 1).tolist()
        pos = take("<i4", n_tok).tolist()
        rows = take("<u2", n_tok * hidden).reshape(n_tok, hidden)
        mbs.append((n_tok, mx, cu, pos, rows))
    assert off == len(buf)
    return assign, mbs


def test_c_driver_matches_oracle(tmp_path):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    assert os.path.exists(DRIVER), "tests/c_abi/pack_driver is not built; run build()"
    cfg = CONFIGS["tiny"]
    seed = 3
    specs = gen_samples(cfg, seed) + _edge_specs(cfg.vocab)
    table = table_np(cfg, seed, mode="bits")
    vis = [visual_rows_np(cfg, seed, i, s.n_vis, mode="bits") for i, s in enumerate(specs)]
    say(f"case C driver: tiny seed={seed}, {len(specs)} samples, H={cfg.hidden}")
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    _write_input(src, cfg, specs, table, vis)
    r = subprocess.run([DRIVER, str(src), str(dst)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assign, mbs = _read_output(dst, len(specs), cfg.hidden)
    want_assign, want_tok, _ = greedy_partition([s.length for s in specs], cfg.cost_k, cfg.capacity, cfg.n_mb)
    assert assign == want_assign
    for j, idx in enumerate(members(want_assign, cfg.n_mb)):
        rows, cu, pos, mx = definitional_pack([specs[i] for i in idx], [vis[i] for i in idx], table)
        n_tok, got_mx, got_cu, got_pos, got_rows = mbs[j]
        assert n_tok == len(rows) == want_tok[j] and got_mx == mx
        assert got_cu == cu.tolist() and got_pos == pos.tolist()
        assert np.array_equal(got_rows, rows)
