"""The seeded input generator's length distributions (no GPU)."""
import numpy as np

import sc_inputs as si


def test_lognormal_lengths_match_the_paper_statistics():
    # ln L ~ N(5.717, 0.738^2): 24 % of the sequences above 512 tokens and 95 % at or below 1024 (the
    # length statistics of the paper's dataset, Sec. 5.2)
    raw = si.lognormal_raw(11, 200_000, 5.717, 0.738)
    assert abs(np.mean(raw > 512) - 0.24) < 0.005
    assert abs(np.mean(raw <= 1024) - 0.95) < 0.005
    # median exp(mu)
    assert abs(np.median(raw) / np.exp(5.717) - 1.0) < 0.01


def test_lognormal_config_lengths():
    cfg = si.CONFIGS[6]
    a = si.lengths(cfg.seed, cfg.B, *cfg.len_range, cfg.len_dist)
    b = si.lengths(cfg.seed, cfg.B, *cfg.len_range, cfg.len_dist)
    assert np.array_equal(a, b) and a.dtype == np.int32
    assert a.min() >= 1 and a.max() <= cfg.n
    # rounding and clipping of the raw draws, in that order
    raw = si.lognormal_raw(cfg.seed, cfg.B, cfg.len_dist[1], cfg.len_dist[2])
    assert np.array_equal(a, np.clip(np.rint(raw), 1, cfg.n).astype(np.int32))


def test_uniform_lengths_unchanged_without_a_distribution():
    vl = si.lengths(3, 8, 2048, 4096)
    assert vl.min() >= 2048 and vl.max() <= 4096
    assert np.array_equal(vl, si.randint(3, si.S_LEN, 8, 2048, 4096).astype(np.int32))
