"""GPU parity of the vector-ALU tile kernel (BSR_KERNEL_VALU) against the CPU oracle.

It serves the block shapes without a matrix-core kernel: 1 x C (C = 1 .. 32), 2x1 .. 8x1 and
2x2 .. 8x8.  Products must satisfy |Y - Y64| <= 1e-5 * sum|x||w| + 1e-6 per element (bf16:
against the oracle on bf16-rounded inputs) and be bit-exact on integer-valued inputs.
"""
import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B
from paper_2106_08846_amd import workloads as G

from .gpu_common import bf16_tensor, check_spmm, dev, host, log, oracle_bsr, prune_on_gpu

pytestmark = pytest.mark.gpu

VALU_SHAPES = [(1, 1), (1, 2), (1, 4), (1, 8), (1, 16), (1, 32), (2, 1), (4, 1), (8, 1),
               (2, 2), (4, 4), (8, 8)]
VALU_BF16_SHAPES = [s for s in VALU_SHAPES if s != (1, 1)]


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


@pytest.mark.parametrize("R,C", VALU_SHAPES)
@pytest.mark.parametrize("slices", [0, 1, 3])
def test_valu_densities_and_slices(device, R, C, slices):
    g = rng(8000 + 100 * R + C + slices)
    N, K, T = 256, 384, 100
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32)
    for density in [0.0, 0.05, 0.3, 1.0]:
        k = B.bsr_prune_count(N, K, R, C, density)
        log(f"valu {R}x{C} slices={slices} density={density} k={k}")
        M = prune_on_gpu(W, R, C, k)
        Y = B.bsr_spmm_ex(dev(X), M, dev(b), kernel=B.KERNEL_VALU, slices=slices)
        torch.cuda.synchronize()
        check_spmm(X, M, b, Y)


@pytest.mark.parametrize("R,C", VALU_BF16_SHAPES)
def test_valu_bf16(device, R, C):
    g = rng(8100 + 100 * R + C)
    N, K, T = 256, 384, 75
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32)
    for density in [0.1, 0.5]:
        M = prune_on_gpu(W, R, C, B.bsr_prune_count(N, K, R, C, density)).to_bf16()
        for slices in [0, 2]:
            log(f"valu bf16 {R}x{C} density={density} slices={slices}")
            Y = B.bsr_spmm_ex(bf16_tensor(X), M, dev(b), kernel=B.KERNEL_VALU, slices=slices)
            torch.cuda.synchronize()
            check_spmm(X, M, b, Y, bf16=True)


@pytest.mark.parametrize("T", [1, 2, 31, 33, 64, 65, 129])
@pytest.mark.parametrize("R,C", [(1, 1), (1, 32), (8, 1), (4, 4), (8, 8)])
def test_valu_ragged_tokens(device, T, R, C):
    g = rng(8200 + T * 10 + R + C)
    W = g.standard_normal((128, 256)).astype(np.float32)
    X = g.standard_normal((T, 256)).astype(np.float32)
    b = g.standard_normal(128).astype(np.float32)
    M = prune_on_gpu(W, R, C, B.bsr_prune_count(128, 256, R, C, 0.3))
    Y = B.bsr_spmm_ex(dev(X), M, dev(b), kernel=B.KERNEL_VALU)
    torch.cuda.synchronize()
    check_spmm(X, M, b, Y)


@pytest.mark.parametrize("R,K", [(1, 767), (1, 770), (2, 770), (8, 771), (4, 1022)])
def test_valu_odd_widths(device, R, K):
    """K odd or not a multiple of 4 (row pitches of every parity), C = 1."""
    g = rng(8300 + R + K)
    N, T = 64, 40
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    M = prune_on_gpu(W, R, 1, B.bsr_prune_count(N, K, R, 1, 0.2))
    Y = B.bsr_spmm_ex(dev(X), M, None, kernel=B.KERNEL_VALU)
    torch.cuda.synchronize()
    check_spmm(X, M, None, Y)


@pytest.mark.parametrize("R,C", [(1, 1), (1, 4), (1, 32), (4, 4), (8, 1), (8, 8)])
def test_valu_pitched_and_unaligned(device, R, C):
    g = rng(8400 + R + C)
    N, K, T = 128, 256, 45
    W = g.standard_normal((N, K)).astype(np.float32)
    Xbig = g.standard_normal((T, K + 3)).astype(np.float32)
    M = prune_on_gpu(W, R, C, B.bsr_prune_count(N, K, R, C, 0.25))
    Xd = dev(Xbig)[:, 1:K + 1]          # ldx = K + 3, base not 16-byte aligned
    Ybig = torch.zeros((T, N + 5), device="cuda:0")
    Y = Ybig[:, 2:N + 2]
    B.bsr_spmm_ex(Xd, M, None, Y=Y, kernel=B.KERNEL_VALU)
    torch.cuda.synchronize()
    check_spmm(np.ascontiguousarray(Xbig[:, 1:K + 1]), M, None, Y)
    assert not host(Ybig)[:, :2].any() and not host(Ybig)[:, N + 2:].any()


@pytest.mark.parametrize("R,C", VALU_SHAPES)
def test_valu_integers_bit_exact(device, R, C):
    """Integer inputs (|x|, |w| <= 8): every order is exact, so the vector-ALU kernel, the
    generic kernel and the exact product agree bit for bit (fp32, and bf16 where supported)."""
    g = rng(8500 + R * 100 + C)
    W = g.integers(-8, 9, size=(256, 192)).astype(np.float32)
    X = g.integers(-8, 9, size=(70, 192)).astype(np.float32)
    b = g.integers(-8, 9, size=256).astype(np.float32)
    k = B.bsr_prune_count(256, 192, R, C, 0.4)
    M = prune_on_gpu(W, R, C, k)
    ip, ix, dt = O.prune(W, R, C, k=k)
    exact = (X.astype(np.int64) @ O.to_dense(ip, ix, dt, 256, 192).astype(np.int64).T
             + b.astype(np.int64)).astype(np.float32)
    Yv = B.bsr_spmm_ex(dev(X), M, dev(b), kernel=B.KERNEL_VALU, slices=5)
    Yg = B.bsr_spmm_ex(dev(X), M, dev(b), kernel=B.KERNEL_GENERIC)
    torch.cuda.synchronize()
    assert np.array_equal(host(Yv), exact)
    assert torch.equal(Yv, Yg)
    if (R, C) != (1, 1):
        Yb = B.bsr_spmm_ex(bf16_tensor(X), M.to_bf16(), dev(b), kernel=B.KERNEL_VALU)
        torch.cuda.synchronize()
        assert np.array_equal(host(Yb), exact)


@pytest.mark.parametrize("R,C", [(1, 1), (1, 32), (8, 1), (8, 8)])
def test_valu_skewed_rows(device, R, C):
    """Block-rows with Zipf-skewed block counts (one full row), several slice counts."""
    g = rng(8600 + R + C)
    N, K = 512, 512
    Nb, Kb = N // R, K // C
    k = max(1, (Nb * Kb) // 8)
    counts = G.zipf_counts(Nb, Kb, k)
    mask = G.zipf_block_mask(counts, Kb, int(g.integers(1 << 30)))
    W = G.apply_block_mask(g.standard_normal((N, K)).astype(np.float32), R, C, mask)
    X = g.standard_normal((77, K)).astype(np.float32)
    M = prune_on_gpu(W, R, C, k)
    for slices in [1, 2, 5, 0]:
        Y = B.bsr_spmm_ex(dev(X), M, None, kernel=B.KERNEL_VALU, slices=slices)
        torch.cuda.synchronize()
        check_spmm(X, M, None, Y)


def test_valu_infinite_inputs_stay_local(device):
    """An infinite X element reaches only the outputs whose stored blocks read its column:
    skipped (masked) chunk slots must not multiply it by a zero weight."""
    g = rng(8700)
    N, K, T = 64, 128, 33
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    X[:, 5] = np.inf
    M = prune_on_gpu(W, 1, 1, B.bsr_prune_count(N, K, 1, 1, 0.1))
    Y = host(B.bsr_spmm_ex(dev(X), M, None, kernel=B.KERNEL_VALU))
    ip, ix, dt = oracle_bsr(M)
    reads5 = np.array([5 in ix[ip[i]:ip[i + 1]] for i in range(N)])
    assert reads5.any() and (~reads5).any()
    Y64 = O.spmm_loop(X, ip, ix, dt, N)
    assert np.all(np.isinf(Y64[:, reads5]))
    assert np.array_equal(Y[:, reads5], Y64[:, reads5].astype(np.float32))
    Xf = X.copy()
    Xf[:, 5] = 0.0
    bound = O.spmm_tolerance(O.tolerance_scale(Xf, O.to_dense(ip, ix, dt, N, K)))
    err = np.abs(Y[:, ~reads5].astype(np.float64) - Y64[:, ~reads5])
    assert np.all(np.isfinite(Y[:, ~reads5])) and np.all(err <= bound[:, ~reads5])


def test_valu_deterministic(device):
    w = G.block_sweep(1, 1)
    p = w.projections[0]
    M = prune_on_gpu(p.W, 1, 1, B.bsr_prune_count(768, 768, 1, 1, p.density))
    X = dev(w.X[0])
    b = dev(p.bias)
    Y0 = B.bsr_spmm_ex(X, M, b, kernel=B.KERNEL_VALU)
    for _ in range(3):
        Y1 = B.bsr_spmm_ex(X, M, b, kernel=B.KERNEL_VALU)
        torch.cuda.synchronize()
        assert torch.equal(Y0.view(torch.int32), Y1.view(torch.int32))


def test_valu_forced_on_other_shapes(device):
    """Forcing the vector-ALU kernel on a shape it lacks is BSR_ERR_UNSUPPORTED (9)."""
    X = dev(rng(8800).standard_normal((4, 96)).astype(np.float32))
    for R, C in [(3, 3), (32, 1), (16, 16)]:
        M = prune_on_gpu(rng(8801).standard_normal((96, 96)).astype(np.float32), R, C, 10)
        with pytest.raises(B.BSRError) as e:
            B.bsr_spmm_ex(X, M, kernel=B.KERNEL_VALU)
        assert e.value.status == 9


def test_valu_auto_is_used_for_sweep_shapes(device):
    """bsr_spmm (automatic choice) on a sweep shape equals the forced vector-ALU call."""
    for R, C in [(1, 1), (8, 1), (1, 32), (4, 4), (8, 8)]:
        w = G.block_sweep(R, C)
        p = w.projections[0]
        M = prune_on_gpu(p.W, R, C, B.bsr_prune_count(768, 768, R, C, p.density))
        X, b = dev(w.X[0]), dev(p.bias)
        Ya = B.bsr_spmm(X, M, b)
        Yv = B.bsr_spmm_ex(X, M, b, kernel=B.KERNEL_VALU)
        torch.cuda.synchronize()
        assert torch.equal(Ya.view(torch.int32), Yv.view(torch.int32))
        check_spmm(w.X[0], M, p.bias, Ya)


def test_valu_batched_mixed(device):
    """A batch of vector-ALU products of several shapes (and a tiled one): every product
    equals its single call and the oracle."""
    g = rng(8900)
    prods, singles, cases = [], [], []
    for R, C, T in [(1, 1, 50), (1, 1, 128), (4, 4, 33), (8, 8, 64), (32, 1, 40), (1, 32, 1)]:
        N, K = 128, 256
        W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
        X = g.standard_normal((T, K)).astype(np.float32)
        b = (g.standard_normal(N) * 0.02).astype(np.float32)
        M = prune_on_gpu(W, R, C, B.bsr_prune_count(N, K, R, C, 0.2))
        prods.append((dev(X), M, dev(b), None))
        cases.append((X, M, b))
    Ys = B.bsr_spmm_batched(prods, slices=4)
    for Xd, M, bd, _ in prods:
        singles.append(B.bsr_spmm_ex(Xd, M, bd, slices=4))
    torch.cuda.synchronize()
    for (X, M, b), Y, Y1 in zip(cases, Ys, singles):
        assert torch.equal(Y.view(torch.int32), Y1.view(torch.int32))
        check_spmm(X, M, b, Y)


@pytest.mark.parametrize("R,C", [(1, 1), (1, 32), (4, 4)])
def test_valu_graph_replay(device, R, C):
    """The vector-ALU product captured in a HIP graph replays bit-identically to the eager call,
    with eager work between replays."""
    w = G.block_sweep(R, C)
    p = w.projections[0]
    M = prune_on_gpu(p.W, R, C, B.bsr_prune_count(768, 768, R, C, p.density))
    Y = torch.empty((128, 768), device=device)
    run = B.SpmmCall(dev(w.X[0]), M, dev(p.bias), Y, kernel=B.KERNEL_VALU)
    ref = run().clone()
    torch.cuda.synchronize()
    check_spmm(w.X[0], M, p.bias, ref)
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        run()
    for rep in range(3):
        Y.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y.view(torch.int32), ref.view(torch.int32)), f"replay {rep}"
