"""GPU parity of the matrix-core kernels across input widths K whose X-tile pitch falls in every
case of the pitch rule (odd and even K for 32x1; every residue class mod 32 that changes the
16x1 padding; square blocks with K an odd multiple of the block width), on the single-tile
kernel and, for wide inputs, the column-chunked one; fp32 and bf16.  Checked against the
oracle's fp64 product within |Y - Y64| <= 1e-5 * sum|x||w| + 1e-6 (bf16: on the bf16-rounded
inputs).
"""
import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B

from .gpu_common import bf16_tensor, dev, log
from .test_gpu_shapes import check_product, upload

pytestmark = pytest.mark.gpu

LINEAR_K = [1, 2, 3, 30, 31, 33, 62, 63, 65, 95, 97, 769, 1023, 3071, 3073]
SQUARE_K = {16: [16, 48, 80, 784, 1040, 3088], 32: [32, 96, 800, 1056, 3104]}


def run(seed, N, K, T, R, C, density, bf16):
    g = np.random.Generator(np.random.PCG64(seed))
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32)
    ip, ix, dt = O.prune(W, R, C, density=density)
    dtq = O.bf16_round(dt) if bf16 else dt
    log(f"pitch {R}x{C} K={K} T={T} bf16={bf16} nnzb={len(ix)}")
    Y = B.bsr_spmm_ex(bf16_tensor(X) if bf16 else dev(X), upload(ip, ix, dtq, N, K, bf16),
                      dev(b), kernel=B.KERNEL_TILED)
    torch.cuda.synchronize()
    check_product(X, ip, ix, O.bf16_to_f32(dtq) if bf16 else dt, N, K, b, Y, bf16)


@pytest.mark.parametrize("R", [32, 16])
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("K", LINEAR_K)
def test_linear_blocks_every_pitch(device, R, bf16, K):
    run(12000 + K + R + bf16, 2 * R, K, 45, R, 1, 0.3, bf16)


@pytest.mark.parametrize("R", [16, 32])
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_square_blocks_every_pitch(device, R, bf16):
    for K in SQUARE_K[R]:
        run(12500 + K + R + bf16, 2 * R, K, 45, R, R, 0.5, bf16)
