"""Paired products in the persistent flat kernel on the GPU.

A planned launch of an even number of products in which products 2i and 2i + 1 share X (the
same tensor, so the same token tiles) and which takes the persistent form runs the two
products of a pair in one set of workgroups: each item covers one X tile of both products, the
second product's block-rows following the first's.  The waves' shares then run across the
boundary between the products, so the partial sums differ from those of the products launched
alone: both must meet the oracle's tolerance, and on integer-valued inputs (where every order
is exact) equal the exact product bit for bit.  Calls of 16 products run as two launches of 8,
each paired; 4 products of 32768 tokens run as two pairs of 128 workgroups each.
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


CASES = [
    # name, [N per product], K, T, density, bf16, arith, slices
    ("BERT-large layer fp32", [1024, 1024, 1024, 1024], 1024, 6144, 0.1, False, B.ARITH_NATIVE,
     1),
    ("two layers fp32 ragged T", [1024] * 8, 1024, 6144 + 13, 0.1, False, B.ARITH_NATIVE, 1),
    ("different N, slices 2", [2304, 768], 768, 8192 + 5, 0.1, False, B.ARITH_NATIVE, 2),
    ("bf16 32-token tiles", [1024, 1024, 768, 768], 768, 9000, 0.05, True, B.ARITH_NATIVE, 1),
    ("bf16 64-token tiles", [1536, 1536], 768, 20000, 0.3, True, B.ARITH_NATIVE, None),
    ("split arithmetic", [1024, 1024, 1024, 1024], 1024, 6144, 0.1, False, B.ARITH_BF16X3, 1),
    # calls of 16 products (two launches), long token counts
    ("fp32 16 products", [1024] * 16, 1024, 6144, 0.1, False, B.ARITH_NATIVE, 1),
    ("fp32 4 products long T", [1024, 768, 1024, 2304], 1024, 32768 + 3, 0.1, False,
     B.ARITH_NATIVE, 1),
    ("bf16 32-token tiles 16 products", [1024, 768, 2304, 768] * 4, 768, 6144 - 7, 0.05, True,
     B.ARITH_NATIVE, 1),
    ("bf16 64-token tiles 16 products", [1536] * 16, 768, 20000, 0.3, True, B.ARITH_NATIVE, None),
    ("split arithmetic 16 products", [1024] * 16, 1024, 6144, 0.1, False, B.ARITH_BF16X3, 1),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_paired_launch_within_tolerance(device, case):
    name, Ns, K, T, d, bf16, arith, slices = case
    log(f"pair case {name}")
    g = rng(zlib.crc32(name.encode()) % 10000)
    Xh = g.standard_normal((T, K)).astype(np.float32)
    X = bf16_tensor(Xh) if bf16 else dev(Xh)
    mats, biases, Ys, plans = [], [], [], []
    for N in Ns:
        W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
        ip, ix, dt = O.prune(W, 32, 1, density=d)
        M = upload(ip, ix, dt, N, K, bf16)
        mats.append(M)
        biases.append((g.standard_normal(N) * 0.02).astype(np.float32))
        Ys.append(torch.full((T, N), 7.0, dtype=torch.float32, device=device))
        plans.append(B.bsr_plan_prepare(M, arith=arith))
    B.SpmmBatchCall([(X, M, dev(b), Y) for M, b, Y in zip(mats, biases, Ys)], slices=slices,
                    plans=plans)()
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, T, 97), [0, 31, 32, T - 33, T - 1]]))
    for M, b, Y, pl in zip(mats, biases, Ys, plans):
        check_spmm(Xh, M, b, Y, rows=rows, bf16=bf16)
        # the same product alone (not paired) meets the same bound on the same rows
        Y1 = torch.empty_like(Y)
        B.SpmmCall(X, M, dev(b), Y1, slices=slices, plan=pl)()
        torch.cuda.synchronize()
        check_spmm(Xh, M, b, Y1, rows=rows, bf16=bf16)


INT_CASES = [
    # name, [N per product], T
    ("pairs", [1024, 768, 1024, 1024], 8192 + 9),
    ("16 products", [1024, 768, 1024, 1024] * 4, 6144 + 9),
]


@pytest.mark.parametrize("case", INT_CASES, ids=[c[0] for c in INT_CASES])
@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_paired_launch_integers_exact(device, bf16, case):
    """Integer-valued inputs: every summation order is exact, so the paired launch equals the
    exact product bit for bit, and equals the products launched alone."""
    g = rng(77)
    _, Ns, T = case
    K = 768
    Xh = g.integers(-8, 9, (T, K)).astype(np.float32)
    X = bf16_tensor(Xh) if bf16 else dev(Xh)
    mats, exact, Ys, biases = [], [], [], []
    for N in Ns:
        W = g.integers(-8, 9, (N, K)).astype(np.float32)
        bias = g.integers(-8, 9, N).astype(np.float32)
        ip, ix, dt = O.prune(W, 32, 1, density=0.1)
        mats.append(upload(ip, ix, dt, N, K, bf16))
        biases.append(dev(bias))
        exact.append((ip, ix, dt, N, bias))
        Ys.append(torch.empty((T, N), dtype=torch.float32, device=device))
    plans = [B.bsr_plan_prepare(M) for M in mats]
    B.SpmmBatchCall([(X, M, b, Y) for M, b, Y in zip(mats, biases, Ys)], plans=plans)()
    torch.cuda.synchronize()
    sample = np.arange(0, T, 5)
    for (ip, ix, dt, N, bias), M, b, Y, pl in zip(exact, mats, biases, Ys, plans):
        ref = O.spmm_loop(Xh[sample], ip, ix, dt, N, bias).astype(np.float32)
        assert np.array_equal(bits(Y)[sample], ref.view(np.uint32))
        Y1 = torch.empty_like(Y)
        B.SpmmCall(X, M, b, Y1, plan=pl)()
        torch.cuda.synchronize()
        assert np.array_equal(bits(Y), bits(Y1))
