"""GPU parity of the column-chunked kernels, which run when a 32-token X tile is too wide for
LDS (the BERT FFN output layer, K = 3072, and wider): the matrix-core one for the tiled block
shapes (32x1, 16x1, 32x32, 16x16) and the vector-ALU one for the others (1x1 .. 1x32, 2x1 ..
8x1, 2x2 .. 8x8); fp32 and bf16.  Every product is checked against the oracle's fp64 product
within |Y - Y64| <= 1e-5 * sum|x||w| + 1e-6 (bf16: on the bf16-rounded inputs), on integers
bit for bit, and two calls must agree bit for bit.  Inputs are built by the oracle and uploaded.
"""
import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B

from .gpu_common import bf16_tensor, dev, host, log
from .test_gpu_shapes import check_product, upload

pytestmark = pytest.mark.gpu

SHAPES = [(32, 1), (16, 1), (32, 32), (16, 16)]


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def case(seed, N, K, T, R, C, density, bf16, slices=0, bias=True, kernel=None):
    g = rng(seed)
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32) if bias else None
    ip, ix, dt = O.prune(W, R, C, density=density)
    dtq = O.bf16_round(dt) if bf16 else dt
    M = upload(ip, ix, dtq, N, K, bf16)
    Xd = bf16_tensor(X) if bf16 else dev(X)
    log(f"kchunk {N}x{K} {R}x{C} T={T} d={density} bf16={bf16} slices={slices} nnzb={len(ix)}")
    Y = B.bsr_spmm_ex(Xd, M, dev(b) if bias else None,
                      kernel=B.KERNEL_TILED if kernel is None else kernel, slices=slices)
    torch.cuda.synchronize()
    check_product(X, ip, ix, O.bf16_to_f32(dtq) if bf16 else dt, N, K, b, Y, bf16)
    return X, M, b, Y


@pytest.mark.parametrize("R,C", SHAPES)
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_kchunk_densities(device, R, C, bf16):
    """K = 4096 (three or more chunks in fp32, two or three in bf16), ragged T = 45."""
    for d in [0.0, 0.02, 0.3]:
        case(9400 + R + C + bf16, 256, 4096, 45, R, C, d, bf16)


@pytest.mark.parametrize("R,C", SHAPES)
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_kchunk_full_density(device, R, C, bf16):
    case(9450 + R + C + bf16, 128, 2560, 33, R, C, 1.0, bf16)


@pytest.mark.parametrize("R,C", SHAPES)
@pytest.mark.parametrize("slices", [1, 3])
def test_kchunk_two_rows_per_wave(device, R, C, slices):
    """64 block-rows (or more) in one or three slices: waves own two rows each, and slices of
    unequal row counts."""
    N = 64 * R
    case(9500 + R + C + slices, N, 3072, 70, R, C, 0.05, False, slices=slices)


@pytest.mark.parametrize("slices", [3, 4, 5, 8, 12, 24])
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_kchunk_wave_groups(device, slices, bf16):
    """24 block-rows in `slices` slices of 8 .. 1 rows: groups of 2 .. 16 waves split each row
    (and some waves stay idle), with their partial tiles added at the end."""
    case(9550 + slices + bf16, 768, 3072, 77, 32, 1, 0.1, bf16, slices=slices)
    case(9560 + slices + bf16, 768, 3072, 77, 32, 32, 0.1, bf16, slices=slices)


@pytest.mark.parametrize("T", [1, 31, 32, 33, 97])
def test_kchunk_ragged_tokens(device, T):
    case(9600 + T, 768, 3072, T, 32, 1, 0.1, False)
    case(9650 + T, 768, 3072, T, 32, 1, 0.1, True)


@pytest.mark.parametrize("R,C", [(32, 1), (32, 32)])
def test_kchunk_skewed_rows(device, R, C):
    """Rows with no blocks, rows with every block, and rows whose blocks sit in one chunk."""
    g = rng(9700 + R + C)
    N, K, T = 512, 4096, 40
    Nb, Kb = N // R, K // C
    W = g.standard_normal((N, K)).astype(np.float32)
    mask = np.zeros((Nb, Kb), dtype=bool)
    mask[1, :] = True                       # every block
    mask[2, : Kb // 8] = True               # first chunk only
    mask[3, -Kb // 8:] = True               # last chunk only
    mask[5, ::97] = True                    # sparse, spread
    mask[Nb - 1, Kb // 2] = True            # one block in the middle
    ip, ix, dt = O.build_bsr(W, R, C, mask)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32)
    Y = B.bsr_spmm_ex(dev(X), upload(ip, ix, dt, N, K), dev(b), kernel=B.KERNEL_TILED)
    torch.cuda.synchronize()
    check_product(X, ip, ix, dt, N, K, b, Y)


@pytest.mark.parametrize("R,C", SHAPES)
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_kchunk_integers_bit_exact_and_repeatable(device, R, C, bf16):
    """Integer inputs: every partial sum is exact, so the result equals the exact product."""
    g = rng(9800 + R + C + bf16)
    N, K, T = 256, 3072, 50
    W = g.integers(-8, 9, size=(N, K)).astype(np.float32)
    X = g.integers(-8, 9, size=(T, K)).astype(np.float32)
    b = g.integers(-8, 9, size=N).astype(np.float32)
    ip, ix, dt = O.prune(W, R, C, density=0.25)
    M = upload(ip, ix, O.bf16_round(dt) if bf16 else dt, N, K, bf16)
    Xd = bf16_tensor(X) if bf16 else dev(X)
    Y1 = B.bsr_spmm_ex(Xd, M, dev(b), kernel=B.KERNEL_TILED)
    Y2 = B.bsr_spmm(Xd, M, dev(b))
    torch.cuda.synchronize()
    assert torch.equal(Y1, Y2)
    Y64 = X.astype(np.float64) @ O.to_dense(ip, ix, dt, N, K).T.astype(np.float64) + b
    assert np.array_equal(host(Y1).astype(np.float64), Y64)


def test_kchunk_without_bias_and_batched(device):
    """No bias; and the same products through one bsr_spmm_batched call (one launch)."""
    X1, M1, _, Y1 = case(9900, 768, 3072, 64, 32, 1, 0.1, False, bias=False)
    X2, M2, b2, Y2 = case(9901, 384, 3072, 64, 32, 1, 0.2, False)
    Ya = torch.empty_like(Y1)
    Yb = torch.empty_like(Y2)
    B.bsr_spmm_batched([(dev(X1), M1, None, Ya), (dev(X2), M2, dev(b2), Yb)])
    torch.cuda.synchronize()
    assert torch.equal(Ya, Y1) and torch.equal(Yb, Y2)


def test_ffn_w2_full_size_sampled_rows(device):
    """BERT-base FFN output layer at 4096 tokens, 32x1 at density 0.1, fp32 and bf16: the
    oracle recomputes a sample of token rows (first, last, and 62 spread in between)."""
    g = rng(9950)
    N, K, T = 768, 3072, 4096
    W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = (g.standard_normal(N) * 0.02).astype(np.float32)
    ip, ix, dt = O.prune(W, 32, 1, density=0.1)
    rows = np.unique(np.concatenate([[0, T - 1], g.integers(0, T, 62)]))
    for bf16 in (False, True):
        dtq = O.bf16_round(dt) if bf16 else dt
        Y = B.bsr_spmm(bf16_tensor(X) if bf16 else dev(X), upload(ip, ix, dtq, N, K, bf16),
                       dev(b))
        torch.cuda.synchronize()
        Ys = Y[torch.from_numpy(rows).to(Y.device)]
        check_product(X[rows], ip, ix, O.bf16_to_f32(dtq) if bf16 else dt, N, K, b, Ys, bf16)


VALU_SHAPES = [(1, 1), (1, 2), (1, 4), (1, 8), (1, 16), (1, 32), (2, 1), (4, 1), (8, 1),
               (2, 2), (4, 4), (8, 8)]


@pytest.mark.parametrize("R,C,bf16", [(R, C, bf) for R, C in VALU_SHAPES for bf in (False, True)
                                      if not (bf and (R, C) == (1, 1))])
def test_vchunk_shapes(device, R, C, bf16):
    """Vector-ALU shapes with K = 3072 (three chunks in fp32), ragged T = 45, through the
    automatic choice and through the forced vector-ALU kernel (bf16 1x1 blocks have no tile
    kernel)."""
    for d in [0.02, 0.3]:
        case(9900 + 10 * R + C + bf16, 256, 3072, 45, R, C, d, bf16, kernel=B.KERNEL_AUTO)
    case(9950 + 10 * R + C + bf16, 256, 3072, 45, R, C, 0.1, bf16, kernel=B.KERNEL_VALU,
         slices=1)


@pytest.mark.parametrize("R,C", [(1, 1), (1, 32), (8, 8), (4, 1)])
def test_vchunk_rows_per_wave_and_slices(device, R, C):
    """Slices holding the most rows a wave may own (slices forced to 1 is raised to that
    minimum), skewed rows, and rows whose blocks sit in one chunk."""
    g = rng(9960 + R + C)
    N, K, T = 1024, 4096, 70
    Nb, Kb = N // R, K // C
    W = g.standard_normal((N, K)).astype(np.float32)
    mask = g.random((Nb, Kb)) < 0.05
    mask[1, :] = True
    mask[2, :] = False
    mask[3, : Kb // 8] = True
    mask[4, -Kb // 8:] = True
    ip, ix, dt = O.build_bsr(W, R, C, mask)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32)
    for slices in (1, 0):
        Y = B.bsr_spmm_ex(dev(X), upload(ip, ix, dt, N, K), dev(b), kernel=B.KERNEL_VALU,
                          slices=slices)
        torch.cuda.synchronize()
        check_product(X, ip, ix, dt, N, K, b, Y)


@pytest.mark.parametrize("R,C", [(1, 32), (8, 8)])
def test_vchunk_integers_bit_exact(device, R, C):
    g = rng(9970 + R + C)
    N, K, T = 256, 3072, 40
    W = g.integers(-8, 9, size=(N, K)).astype(np.float32)
    X = g.integers(-8, 9, size=(T, K)).astype(np.float32)
    b = g.integers(-8, 9, size=N).astype(np.float32)
    ip, ix, dt = O.prune(W, R, C, density=0.25)
    M = upload(ip, ix, dt, N, K)
    Y1 = B.bsr_spmm(dev(X), M, dev(b))
    Y2 = B.bsr_spmm(dev(X), M, dev(b))
    torch.cuda.synchronize()
    assert torch.equal(Y1, Y2)
    Y64 = X.astype(np.float64) @ O.to_dense(ip, ix, dt, N, K).T.astype(np.float64) + b
    assert np.array_equal(host(Y1).astype(np.float64), Y64)



@pytest.mark.parametrize("R,C,bf16,kernel", [(32, 1, False, 2), (32, 1, True, 2),
                                             (16, 16, False, 2), (1, 32, False, 3),
                                             (8, 8, True, 3), (16, 16, True, 2)])
def test_chunked_pitched_inputs_and_outputs(device, R, C, bf16, kernel):
    """X a column window of a wider matrix (row pitch K + 5, odd) and Y a window of a wider
    output: the chunked kernels read and write through both pitches and leave the columns past
    the window alone.  bf16 square tiles load X in dwords, so an odd bf16 pitch is refused by
    the forced matrix-core kernel, and the automatic choice takes the generic kernel."""
    g = rng(9990 + R + C + bf16)
    N, K, T = 256, 3072, 37
    W = g.standard_normal((N, K)).astype(np.float32)
    Xbig = g.standard_normal((T, K + 5)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32)
    ip, ix, dt = O.prune(W, R, C, density=0.1)
    dtq = O.bf16_round(dt) if bf16 else dt
    M = upload(ip, ix, dtq, N, K, bf16)
    Xd = (bf16_tensor(Xbig) if bf16 else dev(Xbig))[:, :K]
    Ybig = torch.full((T, N + 3), float("nan"), device="cuda:0")
    Y = Ybig[:, :N]
    log(f"pitched {R}x{C} bf16={bf16} kernel={kernel}")
    if bf16 and C > 1 and kernel == B.KERNEL_TILED:
        with pytest.raises(B.BSRError, match="UNSUPPORTED"):
            B.bsr_spmm_ex(Xd, M, dev(b), Y=Y, kernel=kernel)
        kernel = B.KERNEL_AUTO
    B.bsr_spmm_ex(Xd, M, dev(b), Y=Y, kernel=kernel)
    torch.cuda.synchronize()
    check_product(np.ascontiguousarray(Xbig[:, :K]), ip, ix, O.bf16_to_f32(dtq) if bf16 else dt,
                  N, K, b, Y, bf16)
    assert torch.isnan(Ybig[:, N:]).all(), "wrote past the output window"
