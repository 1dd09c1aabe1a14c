"""Per-matrix plans (bsr_plan_prepare, bsr_spmm_batched_planned) on the GPU.

A product with a plan must give the same Y, bit for bit, as the same call without one (the plan
only changes where the operands are read from), and both must meet the oracle's tolerance.  The
BSR arrays are built by the oracle and uploaded, so the check does not rest on the GPU's own
pruning; the plan's unit row pointer is compared with the per-row unit counts of the oracle's
indptr.
"""
import ctypes
import zlib

import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B
from paper_2106_08846_amd import workloads as G
from tests.gpu_common import bf16_tensor, check_spmm, dev, host, log

pytestmark = pytest.mark.gpu


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def upload(ip, ix, dt, N, K, bf16=False) -> B.BSRMatrix:
    """Oracle BSR arrays as a device matrix (bf16: the data rounded to bf16 by the oracle)."""
    nnzb, R, C = dt.shape
    if bf16:
        bits = O.bf16_round(dt).view(np.int16)
        data = dev(np.ascontiguousarray(bits)).view(torch.bfloat16)
    else:
        data = dev(dt)
    return B.BSRMatrix(N, K, R, C, dev(ip.astype(np.int32)), dev(ix.astype(np.int32)), data,
                       nnzb)


def unit_ptr(ip, kb):
    n = np.diff(ip.astype(np.int64))
    return np.concatenate([[0], np.cumsum((n + kb - 1) // kb)]).astype(np.int32)


def bits(t: torch.Tensor) -> np.ndarray:
    return host(t).view(np.uint32)


def run_pair(X, M, bias, T, N, slices=None, pitch=0):
    """(Y without a plan, Y with a plan, the plan); Y pitched by `pitch` extra columns."""
    def out():
        big = torch.full((T, N + pitch), 7.0, dtype=torch.float32, device="cuda:0")
        return big, big[:, :N]
    b0, Y0 = out()
    b1, Y1 = out()
    B.SpmmCall(X, M, bias, Y0, slices=slices)()
    plan = B.bsr_plan_prepare(M)
    B.SpmmCall(X, M, bias, Y1, slices=slices, plan=plan)()
    torch.cuda.synchronize()
    if pitch:
        assert torch.all(b0[:, N:] == 7.0) and torch.all(b1[:, N:] == 7.0)
    return Y0, Y1, plan


CASES = [
    # name, N, K, R, T, density, bf16, slices
    ("c1 768x768 d0.2 T128", 768, 768, 32, 128, 0.2, False, None),
    ("768x768 d0.1 T128 bf16", 768, 768, 32, 128, 0.1, True, None),
    ("fused QKV d0.05 T4096", 2304, 768, 32, 4096, 0.05, False, None),
    ("fused QKV d0.4 T4096", 2304, 768, 32, 4096, 0.4, False, None),
    ("fused QKV d0.05 T4096 bf16", 2304, 768, 32, 4096, 0.05, True, None),
    ("fused QKV d0.4 T4096 bf16", 2304, 768, 32, 4096, 0.4, True, None),
    ("ragged T=1", 768, 768, 32, 1, 0.1, False, None),
    ("ragged T=33", 768, 768, 32, 33, 0.1, False, None),
    ("ragged T=100 bf16", 768, 768, 32, 100, 0.1, True, None),
    ("slices 1", 768, 768, 32, 96, 0.3, False, 1),
    ("slices 5", 768, 768, 32, 96, 0.3, False, 5),
    ("slices 24", 768, 768, 32, 64, 0.3, False, 24),
    ("256 block-rows (LDS row pointers)", 8192, 256, 32, 64, 0.2, False, None),
    ("256 block-rows bf16", 8192, 256, 32, 64, 0.2, True, 3),
    ("odd K", 640, 515, 32, 70, 0.15, False, None),
    ("odd K bf16", 640, 515, 32, 70, 0.15, True, None),
    ("density 1", 256, 192, 32, 40, 1.0, False, None),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_plan_is_bit_identical_and_within_tolerance(device, case):
    name, N, K, R, T, d, bf16, slices = case
    log(f"plan case {name}")
    g = rng(zlib.crc32(name.encode()) % 10000)
    W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
    Xh = g.standard_normal((T, K)).astype(np.float32)
    bias = (g.standard_normal(N) * 0.02).astype(np.float32)
    ip, ix, dt = O.prune(W, R, 1, density=d)
    M = upload(ip, ix, dt, N, K, bf16)
    X = bf16_tensor(Xh) if bf16 else dev(Xh)
    Y0, Y1, plan = run_pair(X, M, dev(bias), T, N, slices)
    assert np.array_equal(host(plan.uptr()), unit_ptr(ip, plan.unit_blocks))
    assert np.array_equal(bits(Y0), bits(Y1)), "planned product differs from unplanned"
    rows = None if T <= 256 else np.sort(rng(7).choice(T, 96, replace=False))
    check_spmm(Xh, M, bias, Y1, rows=rows, bf16=bf16)


def test_plan_skewed_rows_and_empty_rows(device):
    """Zipf-skewed rows (one layer of the BERT-large workload, 6144 tokens) and a matrix whose
    block-rows are mostly empty, several slice counts: planned equals unplanned bit for bit."""
    w = G.bert_large_zipf(32, 1, B.bsr_prune_count(1024, 1024, 32, 1, 0.1), layers=1)
    p = w.projections[0]
    ip, ix, dt = O.prune(p.W, 32, 1, k=p.k)
    M = upload(ip, ix, dt, 1024, 1024)
    X = dev(w.X[0])
    for slices in (None, 1, 3):
        Y0, Y1, _ = run_pair(X, M, dev(p.bias), 6144, 1024, slices)
        assert np.array_equal(bits(Y0), bits(Y1)), f"slices={slices}"
    check_spmm(w.X[0], M, p.bias, Y1, rows=np.arange(0, 6144, 97))
    g = rng(11)
    W = (g.standard_normal((1024, 256)) * 0.02).astype(np.float32)
    W[: 1024 - 96] = 0.0                       # only the last three block-rows have weight
    ip, ix, dt = O.prune(W, 32, 1, k=40)       # 40 blocks: all in the last rows
    M = upload(ip, ix, dt, 1024, 256)
    Xh = g.standard_normal((50, 256)).astype(np.float32)
    Y0, Y1, _ = run_pair(dev(Xh), M, None, 50, 1024, pitch=3)
    assert np.array_equal(bits(Y0), bits(Y1))
    check_spmm(Xh, M, None, Y1)


def test_plan_zero_blocks(device):
    ip = np.zeros(25, dtype=np.int32)
    M = upload(ip, np.zeros(0, np.int32), np.zeros((0, 32, 1), np.float32), 768, 768)
    bias = rng(3).standard_normal(768).astype(np.float32)
    X = dev(rng(4).standard_normal((40, 768)).astype(np.float32))
    Y0, Y1, _ = run_pair(X, M, dev(bias), 40, 768)
    assert np.array_equal(bits(Y1), np.broadcast_to(bias, (40, 768)).view(np.uint32))
    assert np.array_equal(bits(Y0), bits(Y1))


@pytest.mark.parametrize("bf16", [False, True])
def test_plan_integer_inputs_exact(device, bf16):
    """Integer-valued inputs: every summation order is exact, so planned, unplanned and the
    exact product agree bit for bit."""
    g = rng(21 + bf16)
    N, K, T = 1536, 768, 200
    W = g.integers(-8, 9, (N, K)).astype(np.float32)
    Xh = g.integers(-8, 9, (T, K)).astype(np.float32)
    bias = g.integers(-8, 9, N).astype(np.float32)
    ip, ix, dt = O.prune(W, 32, 1, density=0.15)
    M = upload(ip, ix, dt, N, K, bf16)
    X = bf16_tensor(Xh) if bf16 else dev(Xh)
    Y0, Y1, _ = run_pair(X, M, dev(bias), T, N)
    exact = O.spmm_loop(Xh, ip, ix, dt, N, bias).astype(np.float32)
    assert np.array_equal(bits(Y1), exact.view(np.uint32))
    assert np.array_equal(bits(Y0), bits(Y1))


def test_plan_batched_qkvo(device):
    """The BERT-base Q/K/V/O step in one launch, with and without plans, bit for bit; a call
    mixing planned and unplanned products (two launches) meets the oracle's tolerance."""
    w = G.bert_base_attention()
    X = dev(w.X[0])
    mats, biases = [], []
    for p in w.projections:
        ip, ix, dt = O.prune(p.W, 32, 1, density=p.density)
        mats.append(upload(ip, ix, dt, 768, 768))
        biases.append(dev(p.bias))
    plans = [B.bsr_plan_prepare(M) for M in mats]
    Ys = [[torch.empty((128, 768), device=device) for _ in range(4)] for _ in range(3)]
    B.SpmmBatchCall([(X, M, b, Y) for M, b, Y in zip(mats, biases, Ys[0])])()
    B.SpmmBatchCall([(X, M, b, Y) for M, b, Y in zip(mats, biases, Ys[1])], plans=plans)()
    B.SpmmBatchCall([(X, M, b, Y) for M, b, Y in zip(mats, biases, Ys[2])],
                    plans=[plans[0], None, plans[2], None])()
    torch.cuda.synchronize()
    for i in range(4):
        assert np.array_equal(bits(Ys[0][i]), bits(Ys[1][i]))
        check_spmm(w.X[0], mats[i], w.projections[i].bias, Ys[1][i])
    # A mixed call launches its planned and unplanned products separately, each launch with the
    # automatic slice count of its own products, so its sums may be ordered differently from
    # the single launch above: it is held to the oracle's tolerance.
    for i in range(4):
        check_spmm(w.X[0], mats[i], w.projections[i].bias, Ys[2][i])


def test_plan_rejected_for_another_matrix(device):
    g = rng(31)
    W1 = (g.standard_normal((256, 256)) * 0.02).astype(np.float32)
    W2 = (g.standard_normal((256, 256)) * 0.02).astype(np.float32)
    M1 = upload(*O.prune(W1, 32, 1, density=0.2), 256, 256)
    M2 = upload(*O.prune(W2, 32, 1, density=0.2), 256, 256)
    plan = B.bsr_plan_prepare(M1)
    X = dev(g.standard_normal((8, 256)).astype(np.float32))
    Y = torch.zeros((8, 256), device=device)
    lib = B.library()
    m2 = M2.struct()
    item = B.bsr_spmm_item_t(X.data_ptr(), 0, 8, 256, ctypes.pointer(m2), None, Y.data_ptr(), 256)
    arr = (ctypes.POINTER(B.bsr_plan_t) * 1)(ctypes.pointer(plan.struct))
    assert lib.bsr_spmm_batched_planned(ctypes.byref(item), arr, 1, None, None) == 3
    small = torch.empty(B.bsr_plan_bytes(M1) - 256, dtype=torch.uint8, device=device)
    with pytest.raises(B.BSRError) as e:
        B.bsr_plan_prepare(M1, mem=small)
    assert e.value.status == 6
    torch.cuda.synchronize()
    assert not Y.any()
