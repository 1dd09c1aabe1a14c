"""The allocation-free prune entry point (bsr_prune_from_dense_noalloc) against
bsr_prune_from_dense, through the C ABI: bit-identical BSR arrays on two calls in a row, the
second on a smaller matrix, so the second runs on a workspace holding the first call's keys."""
import numpy as np
import pytest
import torch

from paper_2106_08846_amd import bsr as B
from paper_2106_08846_amd import workloads as G

pytestmark = pytest.mark.gpu


def _bits(t):
    t = t.contiguous().cpu()
    return t.view(torch.int32).numpy() if t.dtype == torch.float32 else t.numpy()


@pytest.mark.parametrize("shapes", [[(2304, 768, 32, 1, 0.2), (768, 768, 16, 16, 0.1)],
                                    [(1024, 1024, 1, 1, 0.1), (768, 768, 32, 1, 0.05)]])
def test_noalloc_prune_matches_prune(shapes):
    dev = torch.device("cuda:0")
    for n, (N, K, R, C, d) in enumerate(shapes):
        print(f"noalloc prune call {n}: {N}x{K} {R}x{C} d={d}", flush=True)
        W = torch.from_numpy(G.draw_normal(9000 + n, (N, K), 0.02)).to(dev)
        k = B.bsr_prune_count(N, K, R, C, d)
        ref = B.bsr_prune_from_dense(W, R, C, k=k)
        ip = torch.full((N // R + 1,), -7, dtype=torch.int32, device=dev)
        ix = torch.full((k,), -7, dtype=torch.int32, device=dev)
        dt = torch.full((k, R, C), float("nan"), dtype=torch.float32, device=dev)
        got = B.bsr_prune_from_dense_noalloc(W, R, C, k, ip, ix, dt)
        torch.cuda.synchronize()
        assert got.nnzb == ref.nnzb == k
        assert np.array_equal(_bits(ip), _bits(ref.indptr))
        assert np.array_equal(_bits(ix), _bits(ref.indices[:k]))
        assert np.array_equal(_bits(dt), _bits(ref.data[:k]))


def test_noalloc_prune_rejects_too_many_blocks():
    dev = torch.device("cuda:0")
    W = torch.zeros((1024, 1025), dtype=torch.float32, device=dev)
    out = [torch.zeros(1025, dtype=torch.int32, device=dev),
           torch.zeros(4, dtype=torch.int32, device=dev), torch.zeros(4, dtype=torch.float32,
                                                                       device=dev)]
    with pytest.raises(B.BSRError) as e:
        B.bsr_prune_from_dense_noalloc(W, 1, 1, 4, *out)
    assert e.value.status == 6
