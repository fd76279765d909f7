"""The seeded generators produce the workload shapes they claim, repeatably."""

import numpy as np
import pytest

from paper_2606_23087_amd.workloads import (CONFIGS, f32_to_bf16_bits, gen_samples,
                                            page_tier_draws, visual_rows_np)


@pytest.mark.parametrize("name", ["tiny", "qwen", "frag70b", "video", "tiered"])
def test_shapes_and_determinism(name):
    cfg = CONFIGS[name]
    a = gen_samples(cfg, 1)
    b = gen_samples(cfg, 1)
    assert len(a) == len(b)
    for x, y in zip(a, b):
        assert np.array_equal(x.text_ids, y.text_ids) and np.array_equal(x.img_pos, y.img_pos)
        assert np.array_equal(x.img_ntok, y.img_ntok)
    total = sum(s.length for s in a)
    if cfg.fixed_samples:
        assert len(a) == cfg.fixed_samples
    else:
        assert total >= cfg.n_mb * cfg.capacity and total - a[-1].length < cfg.n_mb * cfg.capacity
    for s in a:
        assert np.all(np.diff(s.img_pos) >= 0) and s.img_pos.min() >= 0 and s.img_pos.max() <= s.n_text
        assert s.text_ids.min() >= 0 and s.text_ids.max() < cfg.vocab
        if cfg.video_frames:
            assert len(s.img_ntok) == 1 and s.img_ntok[0] % 256 == 0 and 8 * 256 <= s.img_ntok[0] <= 32 * 256
        else:
            lo, hi, step = cfg.img_tokens
            assert cfg.img_count[0] <= len(s.img_ntok) <= cfg.img_count[1]
            assert np.all((s.img_ntok >= lo) & (s.img_ntok <= hi) & ((s.img_ntok - lo) % step == 0))
    assert gen_samples(cfg, 2, count=3)[0].length != a[0].length or name == "tiny"


def test_qwen_mean_length():
    # 2.5 images x 768 tokens + lognormal(400, 0.8) text (mean ~ 400*e^0.32 ~ 551)
    s = gen_samples(CONFIGS["qwen"], 0)
    m = np.mean([x.length for x in s])
    assert 2200 < m < 2750
    vis = sum(x.n_vis for x in s) / sum(x.length for x in s)
    assert 0.72 < vis < 0.84


def test_bf16_conversion_rne():
    x = np.array([1.0, -2.5, 1.00390625, 1.01171875, 3.4e38, np.nan, 1e-40], dtype=np.float32)
    got = f32_to_bf16_bits(x).tolist()
    assert got[:5] == [0x3F80, 0xC020, 0x3F80, 0x3F82, 0x7F80]
    assert got[5] == 0x7FC0
    assert visual_rows_np(CONFIGS["tiny"], 0, 3, 5).shape == (5, 256)
    t = page_tier_draws(0, 1, 1000)
    assert set(np.unique(t)) == {0, 1} and 400 < t.sum() < 600


def test_pattern_rows_generator_matches_host_twin():
    """The block-wise tensor generator of large inputs and its row-at-a-time
    host twin give the same bits (checked on the CPU, across block edges and
    past 2^16 rows, where the row tag's high word starts to count)."""
    torch = pytest.importorskip("torch")
    from tagging import pattern_base, pattern_row, pattern_rows_dev
    base = pattern_base(24, 5)
    got = pattern_rows_dev(3, 70000, 24, 5, block=4099, device="cpu").numpy().view(np.uint16)
    for r in [0, 1, 4098, 4099, 65535, 65536, 69999] + list(range(96, 200)):
        assert np.array_equal(got[r], pattern_row(3, r, 24, 5, base)), r
    assert got[65536, 3] == 1 and got[65536, 2] == 0
