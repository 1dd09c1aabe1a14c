"""The persistent form of the flat-stream kernel on the GPU.

A launch with more (token tile, slice) items than the GPU has CUs runs one workgroup per CU, each
walking several items of its product with the next tile's X rows loaded under the current
tile's stream.  A token tile's outputs depend only on its own X rows, the matrix and the slice
count, and both kernel forms sum in the same order, so the rows of a tile computed in a
persistent launch equal, bit for bit, the same rows computed in a launch small enough to give
every item its own workgroup.  Every case also meets the oracle's tolerance on sampled rows, and
planned equals unplanned bit for bit.
"""
import zlib

import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B
from tests.gpu_common import bf16_tensor, check_spmm, dev, host, log

pytestmark = pytest.mark.gpu

CUS = 256


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def upload(ip, ix, dt, N, K, bf16=False) -> B.BSRMatrix:
    if bf16:
        data = dev(np.ascontiguousarray(O.bf16_round(dt).view(np.int16))).view(torch.bfloat16)
    else:
        data = dev(dt)
    return B.BSRMatrix(N, K, dt.shape[1], dt.shape[2], dev(ip.astype(np.int32)),
                       dev(ix.astype(np.int32)), data, dt.shape[0])


def bits(t: torch.Tensor) -> np.ndarray:
    return host(t).view(np.uint32)


def run(X, M, bias, T, N, slices, plan=None):
    Y = torch.full((T, N), 7.0, dtype=torch.float32, device="cuda:0")
    B.SpmmCall(X, M, bias, Y, slices=slices, plan=plan)()
    return Y


CASES = [
    # name, N, K, T, density, bf16, slices
    ("fp32 ragged T", 768, 768, 4096 + 17, 0.1, False, 4),
    ("fp32 dense rows", 2304, 768, 4096, 0.3, False, 3),
    ("bf16", 768, 768, 4096 + 5, 0.1, True, 4),
    ("bf16 K past 1024 (two staging passes)", 768, 1500, 2048 + 31, 0.1, True, 8),
    ("fp32 odd K", 640, 515, 4096, 0.15, False, 4),
    ("256 block-rows", 8192, 256, 4096, 0.2, False, 3),
    ("many slices", 1024, 1024, 2048, 0.1, False, 16),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_persistent_matches_one_item_launch_and_oracle(device, case):
    name, N, K, T, d, bf16, slices = case
    pairs = -(-T // 32) * slices
    assert -(-pairs // 8) * 8 > CUS, "the case must take the persistent form"
    log(f"persistent case {name}: {pairs} items")
    g = rng(zlib.crc32(name.encode()) % 10000)
    W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
    Xh = g.standard_normal((T, K)).astype(np.float32)
    bias = (g.standard_normal(N) * 0.02).astype(np.float32)
    ip, ix, dt = O.prune(W, 32, 1, density=d)
    M = upload(ip, ix, dt, N, K, bf16)
    X = bf16_tensor(Xh) if bf16 else dev(Xh)
    b = dev(bias)
    Y = run(X, M, b, T, N, slices)
    plan = B.bsr_plan_prepare(M)
    Yp = run(X, M, b, T, N, slices, plan)
    torch.cuda.synchronize()
    assert np.array_equal(bits(Y), bits(Yp)), "planned differs from unplanned"
    # A window of 8 tiles (at most CUS items with these slice counts) in a one-item launch:
    # the first tiles, a window in the middle and the last (partial) tile.
    for t0 in (0, 32 * (T // 64), 32 * ((T - 1) // 32)):
        rows = min(256, T - t0)
        assert -(-rows // 32) * slices <= CUS
        Xw = X[t0:t0 + rows].contiguous()
        Yw = run(Xw, M, b, rows, N, slices, plan)
        torch.cuda.synchronize()
        assert np.array_equal(bits(Y[t0:t0 + rows]), bits(Yw)), f"window at token {t0}"
    sample = np.unique(np.concatenate([np.arange(0, T, 61), [T - 1]]))
    check_spmm(Xh, M, bias, Yp, rows=sample, bf16=bf16)


def test_persistent_batched_products_of_different_lengths(device):
    """Two products of different token counts in one persistent launch (each workgroup walks
    its own product's items), planned and unplanned, against one-product launches."""
    g = rng(5)
    mats, Xs, biases, Ts = [], [], [], (3000, 5000)
    for T in Ts:
        W = (g.standard_normal((1024, 768)) * 0.02).astype(np.float32)
        ip, ix, dt = O.prune(W, 32, 1, density=0.1)
        mats.append(upload(ip, ix, dt, 1024, 768))
        Xs.append(g.standard_normal((T, 768)).astype(np.float32))
        biases.append((g.standard_normal(1024) * 0.02).astype(np.float32))
    X = [dev(x) for x in Xs]
    b = [dev(x) for x in biases]
    plans = [B.bsr_plan_prepare(M) for M in mats]
    for use_plans in (None, plans):
        Ys = [torch.empty((T, 1024), device=device) for T in Ts]
        B.SpmmBatchCall([(X[i], mats[i], b[i], Ys[i]) for i in range(2)], slices=2,
                        plans=use_plans)()
        torch.cuda.synchronize()
        for i, T in enumerate(Ts):
            Y1 = run(X[i], mats[i], b[i], T, 1024, 2, plans[i] if use_plans else None)
            torch.cuda.synchronize()
            assert np.array_equal(bits(Ys[i]), bits(Y1))
            check_spmm(Xs[i], mats[i], biases[i], Ys[i], rows=np.arange(0, T, 97))
