"""GPU parity for the larger block shapes and the FFN layer shapes.

bsr_reblock must reproduce the oracle's reblock bit for bit (indptr, indices, data), on BSR
arrays the oracle built and uploaded.  A matrix pruned with a large block (64 x 64, 1 x 64 ..
1 x 384, 64 x 1, 128 x 1) and re-blocked to a divisor shape with a fast kernel must give the
oracle's product of the original matrix within |Y - Y64| <= 1e-5 * sum|x||w| + 1e-6.  The
BERT FFN layers (3072 x 768 and 768 x 3072) run through the automatic kernel choice.
"""
import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B

from .gpu_common import ABS_TOL, REL_TOL, bf16_tensor, dev, host, log

pytestmark = pytest.mark.gpu

RESHAPES = [((64, 64), (32, 32)), ((64, 64), (16, 16)), ((64, 64), (8, 8)),
            ((1, 64), (1, 32)), ((1, 128), (1, 32)), ((1, 256), (1, 32)), ((1, 384), (1, 32)),
            ((64, 1), (32, 1)), ((128, 1), (32, 1)), ((32, 32), (32, 1)), ((32, 32), (1, 32)),
            ((4, 4), (1, 4)), ((8, 8), (8, 8)), ((2, 6), (1, 3))]


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def upload(ip, ix, dt, N, K, bf16=False) -> B.BSRMatrix:
    """Oracle-built BSR arrays as a device matrix (bf16: dt holds the bf16 bit patterns)."""
    nnzb, R, C = dt.shape
    if bf16:
        data = dev(np.ascontiguousarray(dt).view(np.int16)).view(torch.bfloat16)
    else:
        data = dev(dt)
    return B.BSRMatrix(N, K, R, C, dev(ip.astype(np.int32)), dev(ix.astype(np.int32)), data,
                       nnzb)


def data_bits(M: B.BSRMatrix) -> np.ndarray:
    d = M.data[:M.nnzb].contiguous()
    if d.dtype == torch.bfloat16:
        return host(d.view(torch.int16)).view(np.uint16)
    return host(d).view(np.uint32)


def check_product(X, ip, ix, dt, N, K, bias, Y, bf16=False):
    """Y against the oracle's fp64 product of the ORIGINAL (coarse-block) matrix."""
    Xh = O.bf16_roundtrip(X) if bf16 else X
    Wm = O.to_dense(ip, ix, dt, N, K)
    Y64 = O.spmm_masked_dense(Xh, Wm, bias)
    bound = O.spmm_tolerance(O.tolerance_scale(Xh, Wm), REL_TOL, ABS_TOL)
    Yg = host(Y).astype(np.float64)
    assert np.all(np.isfinite(Yg)), "non-finite output"
    err = np.abs(Yg - Y64)
    worst = float(np.max(err / bound)) if err.size else 0.0
    assert np.all(err <= bound), f"tolerance exceeded: worst err/bound = {worst:.3f}"


@pytest.mark.parametrize("coarse,fine", RESHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_reblock_bit_exact(device, coarse, fine, bf16):
    (R, C), (R2, C2) = coarse, fine
    g = rng(9000 + 7 * R + C + 3 * R2 + C2 + bf16)
    N, K = 768, 768
    W = g.standard_normal((N, K)).astype(np.float32)
    for density in [0.0, 0.07, 1.0]:
        ip, ix, dt = O.prune(W, R, C, density=density)
        if bf16:
            dt = O.bf16_round(dt)
        log(f"reblock {R}x{C} -> {R2}x{C2} bf16={bf16} density={density} nnzb={len(ix)}")
        M2 = B.bsr_reblock(upload(ip, ix, dt, N, K, bf16), R2, C2)
        torch.cuda.synchronize()
        ip2, ix2, dt2 = O.reblock(ip, ix, dt, R2, C2)
        assert (M2.R, M2.C, M2.nnzb) == (R2, C2, len(ix2))
        assert np.array_equal(host(M2.indptr), ip2), "indptr differs"
        assert np.array_equal(host(M2.indices)[:M2.nnzb], ix2), "indices differ"
        want = dt2.view(np.uint16) if bf16 else dt2.view(np.uint32)
        assert np.array_equal(data_bits(M2).reshape(want.shape), want), "data bits differ"


def test_reblock_rows_without_blocks(device):
    """Block-rows with no stored block stay empty at every fine row."""
    g = rng(9100)
    N, K, R, C = 512, 256, 64, 64
    W = g.standard_normal((N, K)).astype(np.float32)
    W[64:192] *= 1e-3          # block-rows 1 and 2 lose every block at this density
    ip, ix, dt = O.prune(W, R, C, density=0.5)
    assert ip[1] == ip[3]
    M2 = B.bsr_reblock(upload(ip, ix, dt, N, K), 16, 32)
    torch.cuda.synchronize()
    ip2, ix2, dt2 = O.reblock(ip, ix, dt, 16, 32)
    assert np.array_equal(host(M2.indptr), ip2)
    assert np.array_equal(host(M2.indices)[:M2.nnzb], ix2)
    assert np.array_equal(host(M2.data)[:M2.nnzb].view(np.uint32), dt2.view(np.uint32))


@pytest.mark.parametrize("coarse,fine", [((64, 64), (32, 32)), ((64, 64), (16, 16)),
                                         ((1, 64), (1, 32)), ((1, 128), (1, 32)),
                                         ((1, 384), (1, 32)), ((64, 1), (32, 1)),
                                         ((128, 1), (32, 1))],
                         ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_large_block_product(device, coarse, fine, bf16):
    """A large-block matrix re-blocked on the device, then the automatic product, against the
    oracle's product of the large-block matrix; T ragged (77 tokens: two full 32-token tiles and
    a tail of 13)."""
    (R, C), (R2, C2) = coarse, fine
    g = rng(9200 + 7 * R + C + bf16)
    N, K, T = 768, 768, 77
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32)
    for density in [0.05, 0.4]:
        ip, ix, dt = O.prune(W, R, C, density=density)
        dtq = O.bf16_round(dt) if bf16 else dt
        M2 = B.bsr_reblock(upload(ip, ix, dtq, N, K, bf16), R2, C2)
        Xd = bf16_tensor(X) if bf16 else dev(X)
        log(f"large block {R}x{C} via {R2}x{C2} bf16={bf16} density={density}")
        Y = B.bsr_spmm(Xd, M2, dev(b))
        torch.cuda.synchronize()
        check_product(X, ip, ix, O.bf16_to_f32(dtq) if bf16 else dt, N, K, b, Y, bf16)


FFN = [(3072, 768), (768, 3072)]   # BERT-base intermediate (W1) and output (W2), [out][in]


@pytest.mark.parametrize("NK", FFN, ids=["w1_3072x768", "w2_768x3072"])
@pytest.mark.parametrize("R,C", [(32, 1), (16, 1), (1, 32), (32, 32), (16, 16), (8, 8), (1, 4)])
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_ffn_shapes(device, NK, R, C, bf16):
    N, K = NK
    g = rng(9300 + N + 7 * R + C + bf16)
    T = 70
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32)
    ip, ix, dt = O.prune(W, R, C, density=0.1)
    dtq = O.bf16_round(dt) if bf16 else dt
    log(f"ffn {N}x{K} {R}x{C} bf16={bf16}")
    Y = B.bsr_spmm(bf16_tensor(X) if bf16 else dev(X), upload(ip, ix, dtq, N, K, bf16), dev(b))
    torch.cuda.synchronize()
    check_product(X, ip, ix, O.bf16_to_f32(dtq) if bf16 else dt, N, K, b, Y, bf16)
