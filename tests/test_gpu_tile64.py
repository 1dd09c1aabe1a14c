"""64-token tiles of bf16 32x1 products on the GPU.

bf16 32x1 products whose block-rows hold at least 128 stored blocks on average (and at least 32
tiles of 64 tokens) run on tiles of 64 tokens: each unit's weights feed the matrix-core
instructions of two 32-token halves, and rows cut by wave boundaries are combined one half at a
time.  Planned and unplanned products take the same tiles, so they must agree bit for bit, and
both must meet the oracle's tolerance.  The cases below sit above the row-length threshold
(densities of 0.3 and more at 768 input columns) and cover tiles that end inside either half,
slice counts, rows cut across many waves, integer inputs and a launch with more items than CUs.
"""
import zlib

import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from tests.gpu_common import bf16_tensor, check_spmm, dev, host, log
from tests.test_gpu_plan import bits, rng, run_pair, unit_ptr, upload

pytestmark = pytest.mark.gpu

CASES = [
    # name, N, K, T, density, slices
    ("T2048 exact tiles", 1536, 768, 2048, 0.3, None),
    ("T2080 last tile one half", 1536, 768, 2080, 0.3, None),
    ("T2100 last tile inside the second half", 1536, 768, 2100, 0.3, None),
    ("fused QKV d0.4 T4096 slices 1", 2304, 768, 4096, 0.4, 1),
    ("fused QKV d0.4 T4096 slices 3", 2304, 768, 4096, 0.4, 3),
    ("fused QKV d0.4 T4096 slices 7", 2304, 768, 4096, 0.4, 7),
    ("four rows cut across many waves", 128, 768, 2048, 0.95, 1),
    ("odd K", 640, 515, 2200, 0.5, None),
    ("persistent T20000", 768, 768, 20000, 0.3, None),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_tile64_planned_equals_unplanned_and_oracle(device, case):
    name, N, K, T, d, slices = case
    log(f"tile64 case {name}")
    g = rng(zlib.crc32(name.encode()) % 10000)
    W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
    Xh = g.standard_normal((T, K)).astype(np.float32)
    bias = (g.standard_normal(N) * 0.02).astype(np.float32)
    ip, ix, dt = O.prune(W, 32, 1, density=d)
    assert len(ix) >= 128 * (N // 32), "the case must sit above the 64-token row threshold"
    M = upload(ip, ix, dt, N, K, bf16=True)
    Y0, Y1, plan = run_pair(bf16_tensor(Xh), M, dev(bias), T, N, slices, pitch=2)
    assert np.array_equal(host(plan.uptr()), unit_ptr(ip, plan.unit_blocks))
    assert np.array_equal(bits(Y0), bits(Y1)), "planned product differs from unplanned"
    # rows in both halves of the first and the last tile, and a sample in between
    last = (T - 1) // 64 * 64
    edge = np.array([0, 31, 32, 63, last, min(last + 31, T - 1), min(last + 32, T - 1), T - 1])
    rows = np.unique(np.concatenate([edge, rng(7).choice(T, 64, replace=False)]))
    check_spmm(Xh, M, bias, Y1, rows=rows, bf16=True)


def test_tile64_integer_inputs_exact(device):
    """Integer-valued inputs: planned, unplanned and the exact product agree bit for bit."""
    g = rng(61)
    N, K, T = 1024, 768, 2112
    W = g.integers(-8, 9, (N, K)).astype(np.float32)
    Xh = g.integers(-8, 9, (T, K)).astype(np.float32)
    bias = g.integers(-8, 9, N).astype(np.float32)
    ip, ix, dt = O.prune(W, 32, 1, density=0.3)
    M = upload(ip, ix, dt, N, K, bf16=True)
    Y0, Y1, _ = run_pair(bf16_tensor(Xh), M, dev(bias), T, N)
    exact = O.spmm_loop(Xh, ip, ix, dt, N, bias).astype(np.float32)
    assert np.array_equal(bits(Y1), exact.view(np.uint32))
    assert np.array_equal(bits(Y0), bits(Y1))
