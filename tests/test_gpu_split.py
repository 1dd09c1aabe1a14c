"""Split-arithmetic plans (BSR_ARITH_BF16X3) on the GPU.

A plan of split arithmetic stores every fp32 weight of a 32x1 matrix as three bf16 pieces and
the planned product forms each product x * w from the six leading cross terms of the pieces of
x and w on the bf16 matrix cores.  The terms left out are below 2^-20 |x w|, so the product is
held to the same bound as fp32 arithmetic: |Y - Y64| <= 1e-5 sum |x||w| + 1e-6 against the fp64
oracle.  The BSR arrays are built by the oracle and uploaded, as in the native plan tests.
"""
import zlib

import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B
from paper_2106_08846_amd import workloads as G
from tests.gpu_common import check_spmm, dev, host, log
from tests.test_gpu_plan import bits, rng, unit_ptr, upload

pytestmark = pytest.mark.gpu

SPLIT = B.ARITH_BF16X3


def run_split(X, M, bias, T, N, slices=None, pitch=0):
    """(Y with a split plan, the plan); Y pitched by `pitch` extra columns, which must stay."""
    big = torch.full((T, N + pitch), 7.0, dtype=torch.float32, device="cuda:0")
    Y = big[:, :N]
    plan = B.bsr_plan_prepare(M, arith=SPLIT)
    assert plan.arith == SPLIT and plan.unit_blocks == 16
    B.SpmmCall(X, M, bias, Y, slices=slices, plan=plan)()
    torch.cuda.synchronize()
    if pitch:
        assert torch.all(big[:, N:] == 7.0)
    return Y, plan


CASES = [
    # name, N, K, T, density, slices
    ("c1 768x768 d0.2 T128", 768, 768, 128, 0.2, None),
    ("c2 768x768 d0.1 T128", 768, 768, 128, 0.1, None),
    ("fused QKV d0.05 T4096", 2304, 768, 4096, 0.05, None),
    ("fused QKV d0.1 T4096", 2304, 768, 4096, 0.1, None),
    ("fused QKV d0.2 T4096", 2304, 768, 4096, 0.2, None),
    ("fused QKV d0.4 T4096", 2304, 768, 4096, 0.4, None),
    ("ragged T=1", 768, 768, 1, 0.1, None),
    ("ragged T=33", 768, 768, 33, 0.1, None),
    ("ragged T=100", 768, 768, 100, 0.3, None),
    ("slices 1", 768, 768, 96, 0.3, 1),
    ("slices 5", 768, 768, 96, 0.3, 5),
    ("slices 24", 768, 768, 64, 0.3, 24),
    ("256 block-rows (LDS row pointers)", 8192, 256, 64, 0.2, None),
    ("odd K", 640, 515, 70, 0.15, None),
    ("K 1024 (widest fp32 tile here)", 1024, 1024, 200, 0.1, None),
    ("density 1", 256, 192, 40, 1.0, None),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_split_within_tolerance(device, case):
    name, N, K, T, d, slices = case
    log(f"split case {name}")
    g = rng(zlib.crc32(name.encode()) % 10000)
    W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
    Xh = g.standard_normal((T, K)).astype(np.float32)
    bias = (g.standard_normal(N) * 0.02).astype(np.float32)
    ip, ix, dt = O.prune(W, 32, 1, density=d)
    M = upload(ip, ix, dt, N, K)
    Y, plan = run_split(dev(Xh), M, dev(bias), T, N, slices, pitch=3)
    assert np.array_equal(host(plan.uptr()), unit_ptr(ip, 16))
    rows = None if T <= 256 else np.sort(rng(7).choice(T, 96, replace=False))
    worst = check_spmm(Xh, M, bias, Y, rows=rows)
    log(f"  worst err/bound {worst:.3g}")


def test_split_bert_large_layer(device):
    """One layer of the BERT-large workload (Zipf-skewed rows, 6144 tokens) at several slice
    counts; the persistent launch (more token tiles than CUs) is the one the stack runs."""
    w = G.bert_large_zipf(32, 1, B.bsr_prune_count(1024, 1024, 32, 1, 0.1), layers=1)
    for i in (0, 3):
        p = w.projections[i]
        ip, ix, dt = O.prune(p.W, 32, 1, k=p.k)
        M = upload(ip, ix, dt, 1024, 1024)
        for slices in (None, 1, 3):
            Y, _ = run_split(dev(w.X[0]), M, dev(p.bias), 6144, 1024, slices)
            check_spmm(w.X[0], M, p.bias, Y, rows=np.arange(i, 6144, 61))


def test_split_pieces_are_exact(device):
    """The plan's three weight planes: piece 0 is w with its low 16 bits cleared, piece 1 the
    same of the remainder, piece 2 the rest, and the three sum to w exactly (for |w| >= 2^-103;
    below it within 2^-126); the pad blocks of every row's last unit are zero."""
    g = rng(41)
    N, K = 256, 320
    W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
    W[3, :] *= 1e30                                 # large and tiny magnitudes
    W[40, :] *= 1e-30
    ip, ix, dt = O.prune(W, 32, 1, density=0.3)
    M = upload(ip, ix, dt, N, K)
    plan = B.bsr_plan_prepare(M, arith=SPLIT)
    torch.cuda.synchronize()
    s = plan.struct
    mem = host(plan.mem)
    units = int(host(plan.uptr())[-1])
    vals = mem[s.val_offset:s.val_offset + units * 3072].view(np.uint16).reshape(units, 3, 64, 8)
    uptr = host(plan.uptr())
    for r in range(N // 32):
        b0, b1 = int(ip[r]), int(ip[r + 1])
        for u in range(int(uptr[r]), int(uptr[r + 1])):
            for lane in range(64):
                h, f = lane // 32, lane % 32
                for e in range(8):
                    p = b0 + 16 * (u - int(uptr[r])) + 8 * h + e
                    w = np.float32(dt[p, f, 0]) if p < b1 else np.float32(0.0)
                    pcs = vals[u, :, lane, e].astype(np.uint32) << 16
                    w0, w1, w2 = pcs.view(np.float32)
                    wb = np.array([w], np.float32).view(np.uint32)[0]
                    assert pcs[0] == (wb & 0xFFFF0000)
                    rem = np.float32(w - w0)
                    assert pcs[1] == (np.array([rem], np.float32).view(np.uint32)[0] & 0xFFFF0000)
                    # The pieces are exact while the last one is a normal number (|w| >=
                    # 2^-103); below that its low bits fall under 2^-126 and are dropped.
                    err = abs(float(w0) + float(w1) + float(w2) - float(w))
                    assert err == 0.0 if abs(float(w)) >= 2.0 ** -103 else err < 2.0 ** -126


def test_split_zero_blocks_and_integers(device):
    """k = 0 gives Y = bias bit for bit; integer-valued inputs below 256 in magnitude are their
    own first piece, so the split product is exact and equals the exact sum bit for bit."""
    ip = np.zeros(25, dtype=np.int32)
    M = upload(ip, np.zeros(0, np.int32), np.zeros((0, 32, 1), np.float32), 768, 768)
    bias = rng(3).standard_normal(768).astype(np.float32)
    X = dev(rng(4).standard_normal((40, 768)).astype(np.float32))
    Y, _ = run_split(X, M, dev(bias), 40, 768)
    assert np.array_equal(bits(Y), np.broadcast_to(bias, (40, 768)).view(np.uint32))
    g = rng(22)
    N, K, T = 1536, 768, 200
    W = g.integers(-200, 201, (N, K)).astype(np.float32)
    Xh = g.integers(-200, 201, (T, K)).astype(np.float32)
    bias = g.integers(-8, 9, N).astype(np.float32)
    ip, ix, dt = O.prune(W, 32, 1, density=0.15)   # row sums stay below 2^24
    M = upload(ip, ix, dt, N, K)
    Y, _ = run_split(dev(Xh), M, dev(bias), T, N)
    exact = O.spmm_loop(Xh, ip, ix, dt, N, bias)
    assert np.max(np.abs(exact)) < 2 ** 24
    assert np.array_equal(bits(Y), exact.astype(np.float32).view(np.uint32))


def test_split_nan_propagates(device):
    """A NaN in X reaches exactly the outputs whose rows hold a block on its column."""
    g = rng(51)
    N, K, T = 512, 256, 40
    W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
    ip, ix, dt = O.prune(W, 32, 1, density=0.2)
    M = upload(ip, ix, dt, N, K)
    Xh = g.standard_normal((T, K)).astype(np.float32)
    col = int(ix[0])
    Xh[5, col] = np.nan
    Y, _ = run_split(dev(Xh), M, None, T, N)
    Yh = host(Y)
    hit = np.zeros(N, bool)
    for r in range(N // 32):
        if col in set(ix[ip[r]:ip[r + 1]].tolist()):
            hit[32 * r:32 * r + 32] = True
    assert np.all(np.isnan(Yh[5, hit]))
    assert np.all(np.isfinite(Yh[5, ~hit]))
    keep = np.ones(T, bool)
    keep[5] = False
    Xc = Xh.copy()
    Xc[5, col] = 0.0
    check_spmm(Xc[keep], M, None, Y[torch.from_numpy(keep).to(Y.device)])


def test_split_batched_with_native_plans(device):
    """The BERT-base Q/K/V/O step: split plans in one launch, equal to the same products one at
    a time (same launch shape per product); a call mixing split and native plans runs them in
    separate launches, each within the oracle's tolerance."""
    w = G.bert_base_attention()
    X = dev(w.X[0])
    mats, biases = [], []
    for p in w.projections:
        ip, ix, dt = O.prune(p.W, 32, 1, density=p.density)
        mats.append(upload(ip, ix, dt, 768, 768))
        biases.append(dev(p.bias))
    split = [B.bsr_plan_prepare(M, arith=SPLIT) for M in mats]
    native = [B.bsr_plan_prepare(M, arith=B.ARITH_NATIVE) for M in mats]
    Ys = [[torch.empty((128, 768), device=device) for _ in range(4)] for _ in range(2)]
    B.SpmmBatchCall([(X, M, b, Y) for M, b, Y in zip(mats, biases, Ys[0])], plans=split,
                    slices=4)()
    B.SpmmBatchCall([(X, M, b, Y) for M, b, Y in zip(mats, biases, Ys[1])],
                    plans=[split[0], native[1], split[2], native[3]])()
    one = [torch.empty((128, 768), device=device) for _ in range(4)]
    for i in range(4):
        B.SpmmCall(X, mats[i], biases[i], one[i], slices=4, plan=split[i])()
    torch.cuda.synchronize()
    for i in range(4):
        assert np.array_equal(bits(Ys[0][i]), bits(one[i]))
        check_spmm(w.X[0], mats[i], w.projections[i].bias, Ys[0][i])
        check_spmm(w.X[0], mats[i], w.projections[i].bias, Ys[1][i])
