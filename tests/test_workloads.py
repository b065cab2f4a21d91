"""Seeded input generator: determinism, allocation accounting and routing skew."""

import numpy as np
import pytest

from paper_2505_05799_amd import workloads as W


def test_deterministic():
    a = W.make_block("tiny", seed=0)
    b = W.make_block("tiny", seed=0)
    assert np.array_equal(a.x, b.x) and np.array_equal(a.topk_ids, b.topk_ids)
    assert np.array_equal(a.topk_w, b.topk_w)
    for la, lb in zip(a.linears, b.linears):
        for x, y in zip(la, lb):
            assert np.array_equal(x.codes, y.codes)
    c = W.make_block("tiny", seed=1)
    assert not np.array_equal(a.x, c.x)


def test_prefix_sample_matches_full():
    full = W.make_block("dsv2lite", with_weights=False)
    part = W.make_block("dsv2lite", T=100, with_weights=False)
    assert np.array_equal(full.x[:100], part.x)
    assert np.array_equal(full.topk_ids[:100], part.topk_ids)


@pytest.mark.parametrize("name,bits", [("tiny", 7.63), ("mixtral", 3.26), ("dsv2lite", 4.79),
                                       ("qwen15_uniform", 4.02), ("qwen15_mixed", 4.01),
                                       ("qwen15_w5a5", 4.92), ("qwen2", 5.01)])
def test_avg_weight_bits(name, bits):
    assert abs(W.avg_weight_bits(W.CONFIGS[name]) - bits) < 0.006


def test_w5a5_allocation_counts():
    """The printed W5A5 allocation (Qwen1.5-MoE layer 5): gate/up mostly
    w4a4-g128 with a few per-channel w4a4 rows and one w8a8 row; down split
    between w8a8 and w4a4-g128; the shared expert is row 60."""
    from collections import Counter
    cfg = W.CONFIGS["qwen15_w5a5"]
    rows = [cfg.alloc(e, 0) for e in range(cfg.E)] + [cfg.shared_alloc]
    assert all(r[0] == r[1] for r in rows)
    gu = Counter(r[0].name for r in rows)
    dn = Counter(r[2].name for r in rows)
    assert gu == {"w4a4g128": 51, "w4a4": 9, "w8a8": 1}
    assert dn == {"w8a8": 35, "w4a4g128": 26}
    assert cfg.shared_alloc == (W.W4A4, W.W4A4, W.W8A8)


def test_packed_size_closed_form():
    """Sec. 5.2: group-128 codes with 16-bit scale and zero cost N + 0.25 bits per weight."""
    for s, avg in ((W.W3G128, 3.25), (W.W2G128, 2.25), (W.W4G128, 4.25)):
        q = W.QLinear(s, 256, 1024, None)
        assert q.nbytes_packed * 8 / (256 * 1024) == avg


def test_routing_shape_and_skew():
    cfg = W.CONFIGS["qwen15_uniform"]
    ids, w = W.make_routing(cfg)
    assert ids.shape == (cfg.T, cfg.k) and w.dtype == np.float32
    assert all(len(set(r)) == cfg.k for r in ids.tolist())
    assert np.all(np.diff(w, axis=1) <= 0)          # top-k sorted by probability
    counts = np.bincount(ids.ravel(), minlength=cfg.E)
    assert (counts == 0).sum() >= 20                  # Zipf(1.5): many cold experts
    hot = int(np.argmin(W.expert_ranks(cfg)))          # rank-1 expert
    assert counts[hot] == counts.max()


def test_schemes_cover_configs():
    for name, cfg in W.CONFIGS.items():
        sch = W.schemes_of(cfg)
        assert len(sch) == cfg.E + cfg.n_shared
        for gate, up, down in sch:
            assert gate == up
