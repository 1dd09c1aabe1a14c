"""GPU parity of the pruning variants (bsr_prune_from_dense_ex): the l1 block key and per-row
balanced selection, bit for bit against the CPU oracle."""
import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B
from paper_2106_08846_amd import workloads as G

from .gpu_common import check_spmm, dev, host, log

pytestmark = pytest.mark.gpu


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def check_prune_variant(W, R, C, k, norm, per_row):
    M = B.bsr_prune_from_dense(dev(W), R, C, k=k, norm=norm, per_row=per_row)
    ip, ix, dt = O.prune(W, R, C, k=k, norm=norm, per_row=per_row)
    torch.cuda.synchronize()
    assert M.nnzb == k
    assert np.array_equal(host(M.indptr), ip), "indptr differs"
    assert np.array_equal(host(M.indices)[:k], ix), "indices differ"
    assert np.array_equal(host(M.data)[:k].view(np.uint32), dt.view(np.uint32)), "data differs"
    return M


@pytest.mark.parametrize("R,C", [(32, 1), (1, 1), (16, 16), (1, 32), (4, 4), (32, 32), (3, 5)])
@pytest.mark.parametrize("norm", ["l1", "l2"])
@pytest.mark.parametrize("per_row", [False, True])
def test_prune_variants_bit_exact(device, R, C, norm, per_row):
    g = rng(9000 + 100 * R + C + 7 * per_row + (norm == "l1"))
    N, K = 24 * R, (40 * C if C > 1 else 320)
    W = g.standard_normal((N, K)).astype(np.float32)
    for d in [0.0, 0.05, 0.3, 1.0]:
        k = B.bsr_prune_count(N, K, R, C, d, per_row=per_row)
        assert k == O.prune_count(N, K, R, C, d, per_row=per_row)
        log(f"prune {norm} per_row={per_row} {R}x{C} d={d} k={k}")
        check_prune_variant(W, R, C, k, norm, per_row)


@pytest.mark.parametrize("norm", ["l1", "l2"])
def test_prune_variants_ties_and_specials(device, norm):
    """Many equal keys (integers, duplicated and sign-flipped blocks, zero rows), +-inf and NaN."""
    g = rng(9100)
    W = g.integers(-2, 3, size=(64, 96)).astype(np.float32)
    W[0:8] = 0.0
    W[8:16, 0:16] = -W[16:24, 0:16]
    W[30, 5] = np.inf
    W[40, 70] = -np.inf
    W[50, 33] = np.nan
    for R, C, per_row in [(8, 1, False), (8, 1, True), (4, 4, True), (1, 8, True), (8, 8, False)]:
        Nb, Kb = 64 // R, 96 // C
        for k_row in [0, 1, Kb // 3, Kb]:
            k = Nb * k_row if per_row else min(Nb * Kb, k_row * 5)
            check_prune_variant(W, R, C, k, norm, per_row)


def test_l1_pruned_product_matches_oracle(device):
    """The fused-QKV workload pruned with l1 keys per row, then the product, against the oracle."""
    w = G.fused_qkv(32, 1, 0.1, tokens=256)
    p = w.projections[0]
    N, K = p.W.shape
    k = B.bsr_prune_count(N, K, 32, 1, 0.1, per_row=True)
    M = check_prune_variant(p.W, 32, 1, k, "l1", True)
    Y = B.bsr_spmm(dev(w.X[0]), M, dev(p.bias))
    torch.cuda.synchronize()
    check_spmm(w.X[0], M, p.bias, Y)
