"""Seeded workload generator: determinism, shapes, scales and the skewed row counts."""
import numpy as np
import pytest

from oracle import bsr_oracle as O
from paper_2106_08846_amd import workloads as G


def test_draws_are_seeded_and_scaled():
    a = G.draw_normal(G.item_seed(4, 0), (2304, 768), G.W_SIGMA)
    b = G.draw_normal(G.item_seed(4, 0), (2304, 768), G.W_SIGMA)
    assert a.dtype == np.float32 and np.array_equal(a, b)
    assert abs(float(a.std()) - 0.02) < 2e-4 and abs(float(a.mean())) < 2e-4
    c = G.draw_normal(G.item_seed(4, 1), (2304, 768), G.W_SIGMA)
    assert not np.array_equal(a, c)


# Row counts of the capped Zipf(1.2) allocation (shares of the total in proportion to r^-1.2, rows
# over the cap pinned there and the excess re-spread, then largest-remainder rounding), worked
# out independently of the generator.
ZIPF_32x1 = [1024, 467, 287, 203, 156, 125, 104, 88, 77, 68, 60, 54, 49, 45, 42, 39, 36, 33, 31,
             29, 28, 26, 25, 24, 23, 22, 21, 20, 19, 18, 17, 17]
ZIPF_32x32 = [32, 14, 9, 6, 5, 4, 3, 3, 2, 2, 2, 2] + [1] * 18 + [0, 0]


@pytest.mark.parametrize("nrows,cap,total,expect", [(32, 1024, 3277, ZIPF_32x1),
                                                    (32, 32, 102, ZIPF_32x32)])
def test_zipf_counts(nrows, cap, total, expect):
    c = G.zipf_counts(nrows, cap, total)
    assert c.tolist() == expect
    assert c.sum() == total and c.max() <= cap and np.all(np.diff(c) <= 0)


@pytest.mark.parametrize("nrows,cap,total", [(8, 4, 32), (8, 4, 0), (16, 100, 37), (5, 3, 7)])
def test_zipf_counts_invariants(nrows, cap, total):
    c = G.zipf_counts(nrows, cap, total)
    assert c.sum() == total and c.max(initial=0) <= cap and np.all(np.diff(c) <= 0)


def test_zipf_block_mask_row_counts():
    counts = G.zipf_counts(32, 1024, 3277)
    m = G.zipf_block_mask(counts, 1024, 77)
    assert sorted(m.sum(axis=1).tolist(), reverse=True) == counts.tolist()
    assert np.array_equal(m, G.zipf_block_mask(counts, 1024, 77))


def test_workload_shapes():
    w = G.bert_base_attention()
    assert len(w.projections) == 4 and w.X[0].shape == (128, 768)
    assert all(p.W.shape == (768, 768) and (p.R, p.C) == (32, 1) for p in w.projections)
    w = G.fused_qkv(16, 16, 0.2, bf16=True)
    assert w.X[0].shape == (4096, 768) and w.projections[0].W.shape == (2304, 768) and w.bf16
    w = G.bert_large_zipf(32, 32, 102, layers=2, tokens=64)
    assert len(w.projections) == 8 and len(w.X) == 2 and w.projections[5].x_index == 1
    W = w.projections[0].W
    nz = (W.reshape(32, 32, 32, 32) != 0).any(axis=(1, 3))
    assert sorted(nz.sum(axis=1).tolist(), reverse=True) == ZIPF_32x32


@pytest.mark.parametrize("R,C,total", [(32, 1, 3277), (32, 32, 102)])
def test_skewed_workload_total_is_the_pruning_count(R, C, total):
    """The skewed workload's block total is what the caller passes: at density 0.1 it is the
    oracle's pruning count (the generator itself does no pruning arithmetic)."""
    assert O.prune_count(1024, 1024, R, C, 0.1) == total
    w = G.bert_large_zipf(R, C, total, layers=1, tokens=32)
    W = w.projections[0].W
    nz = (W.reshape(1024 // R, R, 1024 // C, C) != 0).any(axis=(1, 3))
    assert int(nz.sum()) == total and w.projections[0].k == total
