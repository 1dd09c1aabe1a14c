"""GPU parity: libbsr (through its C ABI) against the CPU oracle on the same seeded inputs.

Pruning, to_dense and the bf16 cast must match bit for bit; products must satisfy
|Y - Y64| <= 1e-5 * sum|x||w| + 1e-6 per element (bf16: against the oracle on bf16-rounded
inputs), and be bit-exact on integer-valued inputs where every summation order is exact.
"""
import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B
from paper_2106_08846_amd import workloads as G

from .gpu_common import (bf16_tensor, check_prune, check_spmm, dev, host, log, oracle_bsr,
                         prune_on_gpu)

pytestmark = pytest.mark.gpu


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


# ----------------------------------------------------------------------------- the workloads


def test_single_768_32x1(device):
    w = G.single_768()
    p = w.projections[0]
    k = B.bsr_prune_count(768, 768, p.R, p.C, p.density)
    log(f"single_768: k={k}")
    M = prune_on_gpu(p.W, p.R, p.C, k)
    check_prune(p.W, p.R, p.C, M, k)
    Y = B.bsr_spmm(dev(w.X[0]), M, dev(p.bias))
    torch.cuda.synchronize()
    check_spmm(w.X[0], M, p.bias, Y)


def test_bert_base_qkvo(device):
    w = G.bert_base_attention()
    X = dev(w.X[0])
    for p in w.projections:
        k = B.bsr_prune_count(768, 768, p.R, p.C, p.density)
        log(f"bert_base {p.name}: k={k}")
        M = prune_on_gpu(p.W, p.R, p.C, k)
        check_prune(p.W, p.R, p.C, M, k)
        Y = B.bsr_spmm(X, M, dev(p.bias))
        torch.cuda.synchronize()
        check_spmm(w.X[0], M, p.bias, Y)


@pytest.mark.parametrize("R,C", G.SHAPES_SWEEP)
def test_block_sweep(device, R, C):
    w = G.block_sweep(R, C)
    p = w.projections[0]
    k = B.bsr_prune_count(768, 768, R, C, p.density)
    log(f"sweep {R}x{C}: k={k}")
    M = prune_on_gpu(p.W, R, C, k)
    check_prune(p.W, R, C, M, k)
    D = B.bsr_to_dense(M)
    Y = B.bsr_spmm(dev(w.X[0]), M, dev(p.bias))
    torch.cuda.synchronize()
    ip, ix, dt = O.prune(p.W, R, C, k=k)
    assert np.array_equal(host(D).view(np.uint32),
                          O.to_dense(ip, ix, dt, 768, 768).view(np.uint32))
    check_spmm(w.X[0], M, p.bias, Y)


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("R,C", [(32, 1), (16, 16)])
@pytest.mark.parametrize("density", G.QKV_DENSITIES)
def test_fused_qkv(device, R, C, density, bf16):
    w = G.fused_qkv(R, C, density, bf16=bf16)
    p = w.projections[0]
    k = B.bsr_prune_count(2304, 768, R, C, density)
    log(f"fused_qkv {R}x{C} d={density} bf16={bf16}: k={k}")
    M = prune_on_gpu(p.W, R, C, k)
    check_prune(p.W, R, C, M, k)
    if bf16:
        M = M.to_bf16()
        X = bf16_tensor(w.X[0])
    else:
        X = dev(w.X[0])
    Y = B.bsr_spmm(X, M, dev(p.bias))
    torch.cuda.synchronize()
    check_spmm(w.X[0], M, p.bias, Y, bf16=bf16)


@pytest.mark.parametrize("R,C", [(32, 1), (32, 32)])
def test_bert_large_zipf(device, R, C):
    """All 96 projections on the GPU in the benchmark's launch configuration: pruned on the GPU
    (every one checked bit for bit against the oracle's prune, with its Zipf row counts), then
    12 batched launches of 8 products with per-matrix plans where the block shape has them (the
    persistent flat kernel for 32x1, products that share X paired in its workgroups); every
    product meets the oracle's tolerance on every one of its 6144 x 1024 outputs.  One-product
    launches of the first launch's products meet it too; unpaired square blocks equal them bit for bit (paired
    products sum in another order: tests/test_gpu_pair.py checks those on integer inputs)."""
    w = G.bert_large_zipf(R, C, B.bsr_prune_count(1024, 1024, R, C, 0.1))
    Xs = [dev(x) for x in w.X]
    planned = (R, C) == (32, 1)
    projs = w.projections
    for g0 in range(0, len(projs), 8):
        group = projs[g0:g0 + 8]
        mats, plans, biases, Ys = [], [], [], []
        for p in group:
            M = prune_on_gpu(p.W, R, C, p.k)
            check_prune(p.W, R, C, M, p.k)
            counts = np.diff(host(M.indptr))
            assert sorted(counts.tolist(), reverse=True) == w.notes["row_counts_by_rank"]
            mats.append(M)
            plans.append(B.bsr_plan_prepare(M) if planned else None)
            biases.append(dev(p.bias))
            Ys.append(torch.empty((w.tokens, 1024), device=device))
        log(f"bert_large {R}x{C}: launch of products {g0}..{g0 + len(group) - 1}")
        B.SpmmBatchCall([(Xs[p.x_index], M, b, Y) for p, M, b, Y in zip(group, mats, biases, Ys)],
                        plans=plans if planned else None)()
        torch.cuda.synchronize()
        for p, M, Y in zip(group, mats, Ys):
            check_spmm(w.X[p.x_index], M, p.bias, Y)
        if g0 == 0:
            for p, M, b, Y in zip(group, mats, biases, Ys):
                Y1 = B.bsr_spmm(Xs[p.x_index], M, b)
                torch.cuda.synchronize()
                check_spmm(w.X[p.x_index], M, p.bias, Y1)
                if not planned:
                    assert np.array_equal(host(Y).view(np.uint32), host(Y1).view(np.uint32))


# ----------------------------------------------------------------------------- edge cases


def test_k_zero_gives_bias(device):
    W = rng(1).standard_normal((64, 96)).astype(np.float32)
    M = prune_on_gpu(W, 32, 1, 0)
    assert host(M.indptr).tolist() == [0, 0, 0]
    X = rng(2).standard_normal((5, 96)).astype(np.float32)
    b = rng(3).standard_normal(64).astype(np.float32)
    Y = B.bsr_spmm(dev(X), M, dev(b))
    assert np.array_equal(host(Y), np.broadcast_to(b, (5, 64)))
    Y0 = B.bsr_spmm(dev(X), M, None)
    assert not host(Y0).any()


def test_density_one_equals_dense(device):
    g = rng(4)
    W = g.standard_normal((128, 64)).astype(np.float32)
    X = g.standard_normal((33, 64)).astype(np.float32)
    b = g.standard_normal(128).astype(np.float32)
    for R, C in [(32, 1), (16, 16), (1, 1)]:
        M = prune_on_gpu(W, R, C, (128 // R) * (64 // C))
        assert np.array_equal(host(B.bsr_to_dense(M)), W)
        Y = B.bsr_spmm(dev(X), M, dev(b))
        torch.cuda.synchronize()
        check_spmm(X, M, b, Y)


@pytest.mark.parametrize("T", [1, 2, 15, 17, 31, 33, 63, 65, 127, 129, 200])
@pytest.mark.parametrize("R,C", [(32, 1), (16, 1), (32, 32), (16, 16), (8, 8), (1, 1), (1, 32),
                                 (4, 4)])
def test_ragged_token_counts(device, T, R, C):
    g = rng(T * 100 + R + C)
    W = g.standard_normal((256, 128)).astype(np.float32)
    X = g.standard_normal((T, 128)).astype(np.float32)
    b = g.standard_normal(256).astype(np.float32)
    k = B.bsr_prune_count(256, 128, R, C, 0.3)
    M = prune_on_gpu(W, R, C, k)
    Y = B.bsr_spmm(dev(X), M, dev(b))
    torch.cuda.synchronize()
    check_spmm(X, M, b, Y)


def test_leading_dimensions(device):
    g = rng(6)
    Wbig = g.standard_normal((96, 80)).astype(np.float32)
    W = Wbig[:, :64]
    Xbig = g.standard_normal((21, 100)).astype(np.float32)
    X = Xbig[:, :64]
    Wd = dev(Wbig)[:, :64]
    M = B.bsr_prune_from_dense(Wd, 32, 1, k=40)
    check_prune(np.ascontiguousarray(W), 32, 1, M, 40)
    Ybig = torch.full((21, 130), 7.0, device="cuda:0")
    Y = Ybig[:, :96]
    B.bsr_spmm(dev(Xbig)[:, :64], M, None, Y=Y)
    torch.cuda.synchronize()
    check_spmm(np.ascontiguousarray(X), M, None, Y)
    assert np.all(host(Ybig)[:, 96:] == 7.0)


def test_single_block_row_and_full_row(device):
    g = rng(7)
    W = g.standard_normal((32, 256)).astype(np.float32)   # R = N: one block-row
    X = g.standard_normal((50, 256)).astype(np.float32)
    M = prune_on_gpu(W, 32, 1, 256)                      # every block of the row kept
    Y = B.bsr_spmm(dev(X), M, None)
    torch.cuda.synchronize()
    check_spmm(X, M, None, Y)
    M = prune_on_gpu(W, 32, 32, 3)
    Y = B.bsr_spmm(dev(X), M, None)
    torch.cuda.synchronize()
    check_spmm(X, M, None, Y)


@pytest.mark.parametrize("R,C", [(32, 1), (16, 16), (32, 32), (1, 1), (8, 1), (4, 4)])
def test_integer_inputs_bit_exact(device, R, C):
    """|x|, |w| <= 8 integers: every partial sum is an integer below 2^24, so any summation
    order gives the exact result; fp32 and bf16 paths must match the exact product."""
    g = rng(8 + R * C)
    W = g.integers(-8, 9, size=(256, 192)).astype(np.float32)
    X = g.integers(-8, 9, size=(70, 192)).astype(np.float32)
    b = g.integers(-8, 9, size=256).astype(np.float32)
    k = B.bsr_prune_count(256, 192, R, C, 0.4)
    M = prune_on_gpu(W, R, C, k)
    ip, ix, dt = O.prune(W, R, C, k=k)
    exact = (X.astype(np.int64) @ O.to_dense(ip, ix, dt, 256, 192).astype(np.int64).T
             + b.astype(np.int64)).astype(np.float32)
    Y = B.bsr_spmm(dev(X), M, dev(b))
    assert np.array_equal(host(Y), exact)
    Yb = B.bsr_spmm(bf16_tensor(X), M.to_bf16(), dev(b))
    assert np.array_equal(host(Yb), exact)


def test_ties_and_zero_blocks(device):
    W = np.zeros((64, 64), dtype=np.float32)
    W[0:16, 16:32] = 1.0
    W[16:32, 48:64] = -1.0          # same key as the block above
    W[32:48, 0:16] = 0.5
    for k in [1, 2, 3, 5, 16]:
        M = prune_on_gpu(W, 16, 16, k)
        check_prune(W, 16, 16, M, k)
    W = np.zeros((32, 32), dtype=np.float32)   # all keys zero: lowest ids first
    M = prune_on_gpu(W, 1, 1, 100)
    check_prune(W, 1, 1, M, 100)


def test_nonfinite_weights_prune(device):
    W = rng(9).standard_normal((64, 64)).astype(np.float32)
    W[3, 5] = np.inf
    W[40, 7] = np.nan
    W[10, 60] = -np.inf
    for R, C in [(32, 1), (8, 8), (1, 1)]:
        k = B.bsr_prune_count(64, 64, R, C, 0.1)
        M = prune_on_gpu(W, R, C, k)
        ip, ix, dt = O.prune(W, R, C, k=k)
        assert np.array_equal(host(M.indptr), ip)
        assert np.array_equal(host(M.indices)[:k], ix)
        assert np.array_equal(host(M.data)[:k].view(np.uint32), dt.view(np.uint32))


def test_cast_bit_exact(device):
    g = rng(10)
    u = g.integers(0, 1 << 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    special = np.array([0, 0x80000000, 0x7F800000, 0xFF800000, 0x7F7FFFFF, 0x7F7F8000,
                        0x7F7F7FFF, 0x3F808000, 0x3F818000, 0x3F808001, 0x00000001, 0x00018000,
                        0x7FC00000, 0x7F800001, 0xFFFFFFFF], dtype=np.uint32)
    u = np.concatenate([special, u])
    x = u.view(np.float32)
    got = host(B.bsr_cast_f32_bf16(dev(x)).view(torch.int16)).view(np.uint16)
    ref = O.bf16_round(x)
    nan = np.isnan(x)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.all(np.isnan(O.bf16_to_f32(got[nan])))
    assert np.array_equal(got[nan], ref[nan])


def test_deterministic(device):
    w = G.fused_qkv(32, 1, 0.2)
    p = w.projections[0]
    M = prune_on_gpu(p.W, 32, 1, B.bsr_prune_count(2304, 768, 32, 1, 0.2))
    X = dev(w.X[0])
    Y1 = B.bsr_spmm(X, M, dev(p.bias))
    Y2 = B.bsr_spmm(X, M, dev(p.bias))
    torch.cuda.synchronize()
    assert torch.equal(Y1.view(torch.int32), Y2.view(torch.int32))


def test_stream_ordering(device):
    """Work enqueued on a side stream is ordered on that stream."""
    w = G.single_768()
    p = w.projections[0]
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        Wd, Xd, bd = dev(p.W), dev(w.X[0]), dev(p.bias)
        M = B.bsr_prune_from_dense(Wd, 32, 1, density=0.2, stream=s)
        Y = B.bsr_spmm(Xd, M, bd, stream=s)
    s.synchronize()
    check_spmm(w.X[0], M, p.bias, Y)


# ------------------------------------------------------------------ kernel choice and shapes

TILED_SHAPES = [(32, 1), (16, 1), (32, 32), (16, 16)]


def _skewed_weight(g, N, K, R, C, k):
    """W whose nonzero blocks follow a Zipf-like row skew with k blocks in all."""
    Nb, Kb = N // R, K // C
    counts = G.zipf_counts(Nb, Kb, k)
    mask = G.zipf_block_mask(counts, Kb, int(g.integers(1 << 30)))
    return G.apply_block_mask(g.standard_normal((N, K)).astype(np.float32), R, C, mask)


@pytest.mark.parametrize("R,C", TILED_SHAPES)
@pytest.mark.parametrize("slices", [1, 2, 3, 7, 0])
def test_tiled_kernel_slices(device, R, C, slices):
    g = rng(1000 + R * 10 + C + slices)
    N, K, T = 256, 384, 100
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32)
    for density in [0.0, 0.05, 0.3, 1.0]:
        k = B.bsr_prune_count(N, K, R, C, density)
        M = prune_on_gpu(W, R, C, k)
        Y = B.bsr_spmm_ex(dev(X), M, dev(b), kernel=B.KERNEL_TILED, slices=slices)
        torch.cuda.synchronize()
        check_spmm(X, M, b, Y)


@pytest.mark.parametrize("R,C", TILED_SHAPES)
def test_tiled_kernel_skewed_rows(device, R, C):
    g = rng(2000 + R + C)
    N, K = 512, 512
    Nb, Kb = N // R, K // C
    k = max(1, (Nb * Kb) // 8)
    W = _skewed_weight(g, N, K, R, C, k)
    X = g.standard_normal((77, K)).astype(np.float32)
    M = prune_on_gpu(W, R, C, k)
    for slices in [1, 2, 5]:
        Y = B.bsr_spmm_ex(dev(X), M, None, kernel=B.KERNEL_TILED, slices=slices)
        torch.cuda.synchronize()
        check_spmm(X, M, None, Y)


@pytest.mark.parametrize("R,C", TILED_SHAPES)
def test_tiled_unaligned_and_pitched(device, R, C):
    """Odd row pitches (no float4 staging) and offsets into larger buffers."""
    g = rng(3000 + R + C)
    N, K, T = 128, 256, 45
    W = g.standard_normal((N, K)).astype(np.float32)
    Xbig = g.standard_normal((T, K + 3)).astype(np.float32)
    k = B.bsr_prune_count(N, K, R, C, 0.25)
    M = prune_on_gpu(W, R, C, k)
    Xd = dev(Xbig)[:, 1:K + 1]          # ldx = K + 3, base not 16-byte aligned
    Ybig = torch.zeros((T, N + 5), device="cuda:0")
    Y = Ybig[:, 2:N + 2]
    B.bsr_spmm_ex(Xd, M, None, Y=Y, kernel=B.KERNEL_TILED)
    torch.cuda.synchronize()
    check_spmm(np.ascontiguousarray(Xbig[:, 1:K + 1]), M, None, Y)
    assert not host(Ybig)[:, :2].any() and not host(Ybig)[:, N + 2:].any()


def test_tiled_odd_width_r_by_1(device):
    """K not a multiple of 4 for R x 1 blocks (scalar staging path)."""
    g = rng(4000)
    N, K, T = 96, 770, 40
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    for R in (32, 16):
        M = prune_on_gpu(W, R, 1, B.bsr_prune_count(N, K, R, 1, 0.2))
        Y = B.bsr_spmm_ex(dev(X), M, None, kernel=B.KERNEL_TILED)
        torch.cuda.synchronize()
        check_spmm(X, M, None, Y)


@pytest.mark.parametrize("R,C", TILED_SHAPES)
def test_kernels_agree_bitwise_on_integers(device, R, C):
    g = rng(5000 + R + C)
    W = g.integers(-8, 9, size=(256, 256)).astype(np.float32)
    X = g.integers(-8, 9, size=(67, 256)).astype(np.float32)
    b = g.integers(-8, 9, size=256).astype(np.float32)
    M = prune_on_gpu(W, R, C, B.bsr_prune_count(256, 256, R, C, 0.35))
    Yg = B.bsr_spmm_ex(dev(X), M, dev(b), kernel=B.KERNEL_GENERIC)
    Yt = B.bsr_spmm_ex(dev(X), M, dev(b), kernel=B.KERNEL_TILED, slices=3)
    torch.cuda.synchronize()
    assert torch.equal(Yg, Yt)


def _bf16_bsr(W, R, C, k):
    return prune_on_gpu(W, R, C, k).to_bf16()


@pytest.mark.parametrize("R,C", TILED_SHAPES)
@pytest.mark.parametrize("slices", [1, 3, 0])
def test_tiled_bf16_slices(device, R, C, slices):
    """bf16 X and blocks on the tiled kernels (native bf16 MFMA for square blocks, widened
    operands for R x 1), against the oracle on the bf16-rounded inputs."""
    g = rng(7100 + R * 10 + C + slices)
    N, K, T = 256, 384, 100
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    b = g.standard_normal(N).astype(np.float32)
    Xb = bf16_tensor(X)
    for density in [0.0, 0.05, 0.3, 1.0]:
        k = B.bsr_prune_count(N, K, R, C, density)
        M = _bf16_bsr(W, R, C, k)
        Y = B.bsr_spmm_ex(Xb, M, dev(b), kernel=B.KERNEL_TILED, slices=slices)
        torch.cuda.synchronize()
        check_spmm(X, M, b, Y, bf16=True)


@pytest.mark.parametrize("R,C", TILED_SHAPES)
def test_tiled_bf16_skewed_rows_ragged_tokens(device, R, C):
    g = rng(7200 + R + C)
    N, K = 512, 512
    Nb, Kb = N // R, K // C
    k = max(1, (Nb * Kb) // 8)
    W = _skewed_weight(g, N, K, R, C, k)
    M = _bf16_bsr(W, R, C, k)
    for T in (1, 31, 33, 77):
        X = g.standard_normal((T, K)).astype(np.float32)
        for slices in [1, 5]:
            Y = B.bsr_spmm_ex(bf16_tensor(X), M, None, kernel=B.KERNEL_TILED, slices=slices)
            torch.cuda.synchronize()
            check_spmm(X, M, None, Y, bf16=True)


@pytest.mark.parametrize("R,C", TILED_SHAPES)
def test_tiled_bf16_pitched(device, R, C):
    """bf16 X with an even row pitch inside a larger buffer; Y pitched."""
    g = rng(7300 + R + C)
    N, K, T = 128, 256, 45
    W = g.standard_normal((N, K)).astype(np.float32)
    Xbig = g.standard_normal((T, K + 6)).astype(np.float32)
    M = _bf16_bsr(W, R, C, B.bsr_prune_count(N, K, R, C, 0.25))
    Xd = bf16_tensor(Xbig)[:, 2:K + 2]          # ldx = K + 6, 4-byte aligned start
    Ybig = torch.zeros((T, N + 5), device="cuda:0")
    Y = Ybig[:, 2:N + 2]
    B.bsr_spmm_ex(Xd, M, None, Y=Y, kernel=B.KERNEL_TILED)
    torch.cuda.synchronize()
    check_spmm(np.ascontiguousarray(Xbig[:, 2:K + 2]), M, None, Y, bf16=True)
    assert not host(Ybig)[:, :2].any() and not host(Ybig)[:, N + 2:].any()


def test_tiled_bf16_odd_width_and_odd_pitch(device):
    """R x 1 bf16 with odd K and odd row pitch runs tiled; a square bf16 product on an odd pitch
    is refused by the forced tiled kernel and computed by the automatic choice."""
    g = rng(7400)
    N, K, T = 96, 771, 40
    W = g.standard_normal((N, K)).astype(np.float32)
    X = g.standard_normal((T, K)).astype(np.float32)
    for R in (32, 16):
        M = _bf16_bsr(W, R, 1, B.bsr_prune_count(N, K, R, 1, 0.2))
        Y = B.bsr_spmm_ex(bf16_tensor(X), M, None, kernel=B.KERNEL_TILED)
        torch.cuda.synchronize()
        check_spmm(X, M, None, Y, bf16=True)
    K2 = 256
    W2 = g.standard_normal((64, K2)).astype(np.float32)
    Xbig = g.standard_normal((T, K2 + 1)).astype(np.float32)
    M2 = _bf16_bsr(W2, 16, 16, B.bsr_prune_count(64, K2, 16, 16, 0.3))
    Xd = bf16_tensor(Xbig)[:, :K2]              # ldx = K2 + 1 (odd)
    with pytest.raises(B.BSRError) as e:
        B.bsr_spmm_ex(Xd, M2, None, kernel=B.KERNEL_TILED)
    assert e.value.status == 9
    Y = B.bsr_spmm_ex(Xd, M2, None)
    torch.cuda.synchronize()
    check_spmm(np.ascontiguousarray(Xbig[:, :K2]), M2, None, Y, bf16=True)


@pytest.mark.parametrize("R,C", TILED_SHAPES)
def test_kernels_agree_bitwise_on_integers_bf16(device, R, C):
    g = rng(7500 + R + C)
    W = g.integers(-8, 9, size=(256, 256)).astype(np.float32)
    X = g.integers(-8, 9, size=(67, 256)).astype(np.float32)
    b = g.integers(-8, 9, size=256).astype(np.float32)
    M = _bf16_bsr(W, R, C, B.bsr_prune_count(256, 256, R, C, 0.35))
    Xb = bf16_tensor(X)
    Yg = B.bsr_spmm_ex(Xb, M, dev(b), kernel=B.KERNEL_GENERIC)
    Yt = B.bsr_spmm_ex(Xb, M, dev(b), kernel=B.KERNEL_TILED, slices=3)
    torch.cuda.synchronize()
    assert torch.equal(Yg, Yt)
    Y64 = X.astype(np.float64) @ O.to_dense(*oracle_bsr(M), 256, 256).T.astype(np.float64) + b
    assert np.array_equal(host(Yt).astype(np.float64), Y64)


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("density", [0.55, 0.9])
def test_16x16_four_block_units_bit_exact(device, bf16, density):
    """16x16 rows averaging 8 or more blocks run four-block units (partial units at most row
    ends); on integers they must equal the generic kernel and the exact product bit for bit."""
    g = rng(7600 + int(density * 100) + bf16)
    W = g.integers(-8, 9, size=(256, 256)).astype(np.float32)
    X = g.integers(-8, 9, size=(75, 256)).astype(np.float32)
    b = g.integers(-8, 9, size=256).astype(np.float32)
    k = B.bsr_prune_count(256, 256, 16, 16, density)
    assert k >= 8 * 16
    M = _bf16_bsr(W, 16, 16, k) if bf16 else prune_on_gpu(W, 16, 16, k)
    Xd = bf16_tensor(X) if bf16 else dev(X)
    Yg = B.bsr_spmm_ex(Xd, M, dev(b), kernel=B.KERNEL_GENERIC)
    for slices in (0, 1, 5):
        Yt = B.bsr_spmm_ex(Xd, M, dev(b), kernel=B.KERNEL_TILED, slices=slices)
        torch.cuda.synchronize()
        assert torch.equal(Yg, Yt)
    Y64 = X.astype(np.float64) @ O.to_dense(*oracle_bsr(M), 256, 256).T.astype(np.float64) + b
    assert np.array_equal(host(Yt).astype(np.float64), Y64)


@pytest.mark.parametrize("R,C", TILED_SHAPES)
def test_generic_kernel_on_tiled_shapes(device, R, C):
    w = G.block_sweep(R, C)
    p = w.projections[0]
    M = prune_on_gpu(p.W, R, C, B.bsr_prune_count(768, 768, R, C, p.density))
    Y = B.bsr_spmm_ex(dev(w.X[0]), M, dev(p.bias), kernel=B.KERNEL_GENERIC)
    torch.cuda.synchronize()
    check_spmm(w.X[0], M, p.bias, Y)


def test_forced_tiled_unsupported_shape(device):
    W = rng(6000).standard_normal((64, 64)).astype(np.float32)
    M = prune_on_gpu(W, 8, 8, 10)
    X = dev(rng(6001).standard_normal((4, 64)).astype(np.float32))
    with pytest.raises(B.BSRError) as e:
        B.bsr_spmm_ex(X, M, kernel=B.KERNEL_TILED)
    assert e.value.status == 9


def test_tiled_deterministic_and_repeatable(device):
    w = G.bert_large_zipf(32, 1, B.bsr_prune_count(1024, 1024, 32, 1, 0.1), layers=1)
    p = w.projections[0]
    M = prune_on_gpu(p.W, 32, 1, p.k)
    X = dev(w.X[0])
    Y1 = B.bsr_spmm(X, M, dev(p.bias))
    Y2 = B.bsr_spmm(X, M, dev(p.bias))
    torch.cuda.synchronize()
    assert torch.equal(Y1.view(torch.int32), Y2.view(torch.int32))


# ------------------------------------------------------------------ prepared calls and graphs


@pytest.mark.parametrize("R,C,kernel,bf16", [(32, 1, B.KERNEL_AUTO, False),
                                             (16, 16, B.KERNEL_AUTO, False),
                                             (8, 8, B.KERNEL_AUTO, False),
                                             (32, 1, B.KERNEL_GENERIC, True)])
def test_graph_replay_matches_eager(device, R, C, kernel, bf16):
    """A captured step replays bit-identically to the eager call, replay after replay."""
    log(f"graph replay R={R} C={C} kernel={kernel} bf16={bf16}")
    w = G.bert_base_attention(R, C, 0.1, tokens=96)
    calls, eager = [], []
    Xd = dev(w.X[0])
    Xin = B.bsr_cast_f32_bf16(Xd) if bf16 else Xd
    for p in w.projections:
        k = B.bsr_prune_count(768, 768, R, C, p.density)
        M = prune_on_gpu(p.W, R, C, k)
        if bf16:
            M = M.to_bf16()
        Y = torch.empty((96, 768), dtype=torch.float32, device=device)
        run = B.SpmmCall(Xin, M, dev(p.bias), Y, kernel=kernel)
        eager.append(run().clone())
        calls.append(run)
    torch.cuda.synchronize()
    check_spmm(w.X[0], calls[0]._keep[0][1], w.projections[0].bias, eager[0], bf16=bf16)
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for run in calls:
            run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for run in calls:
            run()
    for rep in range(3):
        for run in calls:
            run.Y.fill_(float("nan"))     # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for run, ref in zip(calls, eager):
            assert torch.equal(run.Y.view(torch.int32), ref.view(torch.int32)), f"replay {rep}"


def test_prepared_call_matches_bsr_spmm(device):
    w = G.single_768()
    p = w.projections[0]
    k = B.bsr_prune_count(768, 768, 32, 1, p.density)
    M = prune_on_gpu(p.W, 32, 1, k)
    X, b = dev(w.X[0]), dev(p.bias)
    Y = torch.empty((128, 768), dtype=torch.float32, device=device)
    run = B.SpmmCall(X, M, b, Y, slices=5)
    Yp = run().clone()
    Ys = B.bsr_spmm_ex(X, M, b, slices=5)
    torch.cuda.synchronize()
    assert torch.equal(Yp.view(torch.int32), Ys.view(torch.int32))
    with pytest.raises(ValueError):
        B.SpmmCall(X, M, b, torch.empty((127, 768), dtype=torch.float32, device=device))


@pytest.mark.parametrize("kernel", [B.KERNEL_TILED, B.KERNEL_GENERIC])
def test_timed_call_records_kernel_events(device, kernel):
    w = G.single_768()
    p = w.projections[0]
    k = B.bsr_prune_count(768, 768, 32, 1, p.density)
    M = prune_on_gpu(p.W, 32, 1, k)
    X, b = dev(w.X[0]), dev(p.bias)
    run = B.SpmmCall(X, M, b, torch.empty((128, 768), dtype=torch.float32, device=device),
                     kernel=kernel)
    ref = run().clone()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    e1.record()
    run.Y.fill_(float("nan"))
    run.timed(e0, e1)
    torch.cuda.synchronize()
    assert torch.equal(run.Y.view(torch.int32), ref.view(torch.int32))
    ms = e0.elapsed_time(e1)
    assert 0.0 < ms < 100.0



# --------------------------------------------------------------------------- batched products


def test_batched_equals_single_calls(device):
    """One launch for Q, K, V, O gives each product bit for bit what a single call gives."""
    w = G.bert_base_attention()
    X = dev(w.X[0])
    prods, singles = [], []
    for p in w.projections:
        k = B.bsr_prune_count(768, 768, 32, 1, p.density)
        M = prune_on_gpu(p.W, 32, 1, k)
        b = dev(p.bias)
        prods.append((X, M, b, None))
        singles.append(B.bsr_spmm_ex(X, M, b, slices=6))
    Ys = B.bsr_spmm_batched(prods, slices=6)
    torch.cuda.synchronize()
    for (X_, M, b, _), Y, Y1, p in zip(prods, Ys, singles, w.projections):
        assert torch.equal(Y.view(torch.int32), Y1.view(torch.int32))
        check_spmm(w.X[0], M, p.bias, Y)


def test_batched_auto_slices_mixed_shapes(device):
    """A batch mixing tiled shapes, a generic shape, bf16, empty products and more than one
    launch's worth of products; every product checked against the oracle."""
    g = rng(7001)
    cases = []
    for i, (R, C, T, bf16) in enumerate([(32, 1, 200, False), (16, 16, 64, False),
                                          (8, 8, 33, False), (32, 1, 0, False),
                                          (32, 32, 96, False), (16, 1, 40, False),
                                          (32, 1, 128, True)] + [(32, 1, 7 + 9 * j, False)
                                                                 for j in range(9)]):
        N, K = 256, 192
        W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
        X = g.standard_normal((T, K)).astype(np.float32)
        b = (g.standard_normal(N) * 0.02).astype(np.float32)
        k = B.bsr_prune_count(N, K, R, C, 0.3)
        M = prune_on_gpu(W, R, C, k)
        Xd = dev(X)
        if bf16:
            M = M.to_bf16()
            Xd = B.bsr_cast_f32_bf16(Xd)
        cases.append((X, M, b, bf16, (Xd, M, dev(b), None)))
    log(f"batched mixed: {len(cases)} products")
    Ys = B.bsr_spmm_batched([c[4] for c in cases])
    torch.cuda.synchronize()
    for (X, M, b, bf16, _), Y in zip(cases, Ys):
        if X.shape[0]:
            check_spmm(X, M, b, Y, bf16=bf16)
        else:
            assert Y.shape[0] == 0


def test_batched_timed_events(device):
    w = G.bert_base_attention()
    X = dev(w.X[0])
    prods = []
    for p in w.projections:
        M = prune_on_gpu(p.W, 32, 1, B.bsr_prune_count(768, 768, 32, 1, p.density))
        prods.append((X, M, dev(p.bias), torch.empty((128, 768), device=device)))
    run = B.SpmmBatchCall(prods)
    ref = [y.clone() for y in run()]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    e1.record()
    run.timed(e0, e1)
    torch.cuda.synchronize()
    for y, r in zip(run.Y, ref):
        assert torch.equal(y.view(torch.int32), r.view(torch.int32))
    assert 0.0 < e0.elapsed_time(e1) < 100.0
