"""Seeded input generation: determinism, bf16 rounding, page tables, and the
length distribution against the paper's trace statistics."""
import json
import os

import numpy as np
import pytest
import torch

import workload
from workload import gen

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "trace_lengths.json")


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100_000).astype(np.float32) * 7,
                        np.array([0.0, -0.0, 1e-40, -1e-40, 3.4e38, np.inf, -np.inf], np.float32),
                        # exact ties between two bf16 values
                        (np.arange(1, 2000, dtype=np.uint32) << 16 | 0x8000).view(np.float32)])
    ours = workload.bf16_bits_from_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = workload.f32_from_bf16_bits(ours)
    assert np.array_equal(back, torch.from_numpy(ours.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_nan_rounds_to_sentinel():
    assert workload.bf16_bits_from_f32(np.array([np.nan], np.float32))[0] == workload.BF16_NAN


def test_same_seed_same_bits():
    a = workload.make_workload("tiny")
    b = workload.make_workload("tiny")
    for f in ("q", "k_new", "v_new", "prefix_k", "prefix_v", "block_tables", "prefix_slots"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f
    c = workload.make_workload("tiny", seed=99)
    assert not np.array_equal(a.q, c.q)


def test_ragged_lengths_follow_trace_statistics():
    g = json.load(open(GOLDEN))
    rng = np.random.default_rng(1234)
    draws = gen.lognormal_prefix_lengths(rng, 400_000, cap=10**9)
    assert abs(np.median(draws) / g["median_tokens"] - 1) < 0.01
    assert abs(np.percentile(draws, 95) / g["p95_tokens"] - 1) < 0.015
    capped = gen.lognormal_prefix_lengths(np.random.default_rng(5), 10_000)
    assert capped.max() <= gen.RAGGED_PREFIX_CAP


@pytest.mark.parametrize("name", ["tiny", "single", "long", "cold"])
def test_block_tables_are_distinct_and_cover(name):
    wl = workload.make_workload(name)
    ps = wl.page_size
    used = []
    for b in range(wl.num_seqs):
        n = (int(wl.prefix_lens[b]) + int(wl.suffix_lens[b]) + ps - 1) // ps
        row = wl.block_tables[b]
        assert (row[:n] >= 0).all() and (row[:n] < wl.num_pages).all()
        assert (row[n:] == -1).all()
        used.append(row[:n])
    used = np.concatenate(used)
    assert np.unique(used).shape[0] == used.shape[0]


def test_ragged_config_shape():
    wl = workload.make_workload("ragged")
    assert wl.num_seqs == 16
    assert (wl.suffix_lens >= 512).all() and (wl.suffix_lens <= 4096).all()
    assert (wl.prefix_lens <= gen.RAGGED_PREFIX_CAP).all()
    used = wl.block_tables[wl.block_tables >= 0]
    assert np.unique(used).shape[0] == used.shape[0] and used.max() < 300_000


def test_single_config_work():
    wl = workload.make_workload("single")
    # 25,000 = 1562 * 16 + 8: the last prefix page is half full.
    assert wl.prefix_lens[0] % wl.page_size == 8
    pairs = 2048 * 25_000 + 2048 * 2049 // 2
    assert wl.visible_pairs() == pairs == 53_298_176
    assert wl.flops() == 4 * 128 * 8 * pairs


def test_long_config_chunks():
    wl = workload.make_workload("long")
    assert len(wl.chunks) == 4
    for c, (pre, suf, tok) in enumerate(wl.chunks):
        assert pre[0] == 105_000 + 2048 * c and suf[0] == 2048
        assert np.array_equal(tok, np.arange(2048 * c, 2048 * (c + 1)))


def test_prefix_slots_follow_block_tables():
    wl = workload.make_workload("tiny")
    t = np.arange(256)
    assert np.array_equal(wl.prefix_slots, wl.block_tables[0, t // 16].astype(np.int64) * 16 + t % 16)
