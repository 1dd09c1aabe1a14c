"""GPU parity of the attention kernel and of the BERT attention block built on the BSR products
(Q/K/V products -> scaled dot-product attention -> O product), against the CPU oracles."""
import numpy as np
import pytest
import torch

from oracle import attention_oracle as A
from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B
from paper_2106_08846_amd import workloads as G

from .gpu_common import check_prune, check_spmm, dev, host, log, oracle_bsr, prune_on_gpu

pytestmark = pytest.mark.gpu


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def check_attention(Q, K, V, ctx_gpu, batch, seq, heads):
    ctx64 = A.attention(Q, K, V, batch, seq, heads, 64)
    bound = A.attention_error_bound(Q, K, V, batch, seq, heads, 64)
    got = host(ctx_gpu).astype(np.float64)
    err = np.abs(got - ctx64)
    assert np.all(np.isfinite(got))
    worst = float(np.max(err / (bound + 1e-30)))
    assert np.all(err <= bound), f"attention outside the bound: worst err/bound {worst:.3g}"
    return worst


@pytest.mark.parametrize("batch,seq,heads,sd", [(1, 128, 12, 1.0), (2, 77, 3, 1.0), (1, 1, 1, 1.0),
                                                (1, 33, 2, 4.0), (3, 64, 4, 0.3), (1, 200, 1, 2.0),
                                                (8, 512, 2, 1.0), (1, 65, 1, 8.0),
                                                (1, 256, 3, 1.0), (2, 300, 2, 2.0),
                                                (1, 1000, 1, 1.0), (4, 257, 2, 0.5),
                                                (1, 384, 12, 4.0),
                                                # vector kernel, 32-query tiles; key split
                                                # with an idle round
                                                (24, 64, 12, 1.0), (8, 200, 12, 2.0),
                                                (1, 150, 2, 1.0),
                                                # matrix-core kernel, key halves on two waves
                                                (8, 512, 6, 1.0), (16, 256, 12, 1.0),
                                                (8, 300, 12, 2.0), (3, 1000, 12, 0.5),
                                                (24, 130, 12, 4.0),
                                                # four query tiles per workgroup (>= 2048 tiles)
                                                (48, 128, 12, 1.0), (36, 200, 12, 2.0)])
def test_attention_matches_oracle(device, batch, seq, heads, sd):
    g = rng(9500 + batch * 1000 + seq + heads)
    T, W = batch * seq, heads * 64
    Q, K, V = [(g.standard_normal((T, W)) * sd).astype(np.float32) for _ in range(3)]
    log(f"attention batch={batch} seq={seq} heads={heads} sd={sd}")
    ctx = B.bsr_attention(dev(Q), dev(K), dev(V), batch, seq, heads)
    torch.cuda.synchronize()
    check_attention(Q, K, V, ctx, batch, seq, heads)


def test_attention_on_a_fused_qkv_output(device):
    """Q, K, V as column views of one [T, 3*768] buffer (row pitch 2304), output pitched too."""
    g = rng(9600)
    batch, seq, heads = 2, 96, 12
    T = batch * seq
    QKV = (g.standard_normal((T, 3 * 768)) * 0.5).astype(np.float32)
    d = dev(QKV)
    Obig = torch.full((T, 800), 3.0, device=device)
    B.bsr_attention(d[:, :768], d[:, 768:1536], d[:, 1536:], batch, seq, heads, O=Obig[:, :768])
    torch.cuda.synchronize()
    check_attention(QKV[:, :768], QKV[:, 768:1536], QKV[:, 1536:], Obig[:, :768], batch, seq,
                    heads)
    assert torch.all(Obig[:, 768:] == 3.0)


def test_attention_deterministic(device):
    g = rng(9700)
    Q, K, V = [dev((g.standard_normal((256, 128))).astype(np.float32)) for _ in range(3)]
    a = B.bsr_attention(Q, K, V, 2, 128, 2)
    for _ in range(3):
        b = B.bsr_attention(Q, K, V, 2, 128, 2)
        torch.cuda.synchronize()
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_attention_unsupported_inputs(device):
    lib = B.library()
    x = torch.zeros((64, 128), device=device)
    p = x.data_ptr()
    assert lib.bsr_attention(p, 128, p, 128, p, 128, p + 1024, 128, 1, 64, 4, 32, 0.1, None) == 9
    assert lib.bsr_attention(p + 4, 128, p, 128, p, 128, p, 128, 1, 64, 2, 64, 0.1, None) == 9
    assert lib.bsr_attention(p, 130, p, 128, p, 128, p, 128, 1, 64, 2, 64, 0.1, None) == 9


def _block(R, C, density, batch, seq, kernel=None):
    w = G.bert_base_attention(R, C, density, tokens=batch * seq)
    mats, biases = [], []
    for prj in w.projections:
        k = B.bsr_prune_count(768, 768, R, C, prj.density)
        mats.append(prune_on_gpu(prj.W, R, C, k))
        biases.append(dev(prj.bias))
    X = dev(w.X[0])
    call = B.AttentionBlockCall(X, mats[0], biases[0], mats[1], biases[1], mats[2], biases[2],
                                mats[3], biases[3], batch, seq, 12, kernel=kernel)
    return w, mats, call


@pytest.mark.parametrize("R,C,density,batch,seq", [(32, 1, 0.1, 1, 128), (16, 16, 0.2, 2, 64),
                                                   (1, 32, 0.1, 1, 128), (32, 32, 0.1, 3, 50)])
def test_attention_block_stage_by_stage(device, R, C, density, batch, seq):
    """Each stage of the block against its oracle, on the GPU's own inputs to that stage."""
    w, mats, call = _block(R, C, density, batch, seq)
    Y = call()
    torch.cuda.synchronize()
    X = w.X[0]
    for M, prj, out in zip(mats[:3], w.projections[:3], (call.Q, call.K, call.V)):
        check_spmm(X, M, prj.bias, out)
    Qh, Kh, Vh = host(call.Q), host(call.K), host(call.V)
    check_attention(Qh, Kh, Vh, call.ctx, batch, seq, 12)
    check_spmm(host(call.ctx), mats[3], w.projections[3].bias, Y)


@pytest.mark.parametrize("R,C,density,batch,seq", [(32, 1, 0.1, 1, 128), (16, 16, 0.2, 2, 64),
                                                   (32, 1, 0.1, 2, 256)])
def test_attention_block_end_to_end(device, R, C, density, batch, seq):
    """The block's output Y against the fp64 oracle's whole block (attention_block) run from X
    and the pruned weights, with a bound propagated through the stages:
      * Q, K, V: the product bound dP = 1e-5 S + 1e-6 (A12);
      * ctx: the kernel's own rounding at its inputs (attention_error_bound at the GPU's Q, K,
        V), plus the effect of the inputs' error: the scores move by at most
        D = max_j scale sum_d (dQ |k_jd| + |q_d| dK_jd + dQ dK_jd), so the softmax weights move
        by a factor within exp(+-2D), and ctx by (e^{2D} - 1) sum_j p_j |v_jd| +
        e^{2D} sum_j p_j dV_jd;
      * Y: the product bound at the GPU's ctx plus dctx |Wo|^T."""
    w, mats, call = _block(R, C, density, batch, seq)
    Y = call()
    torch.cuda.synchronize()
    X = w.X[0].astype(np.float64)
    for M, prj in zip(mats, w.projections):
        check_prune(prj.W, R, C, M, M.nnzb)
    Wd = [O.to_dense(*oracle_bsr(M), 768, 768) for M in mats]
    bs = [prj.bias for prj in w.projections]
    Q64, K64, V64, ctx64, Y64 = A.attention_block(X, Wd[0], bs[0], Wd[1], bs[1], Wd[2], bs[2],
                                                  Wd[3], bs[3], batch, seq, 12)
    dQ, dK, dV = (1e-5 * O.tolerance_scale(X, Wm) + 1e-6 for Wm in Wd[:3])
    Qg, Kg, Vg, ctxg = (host(t).astype(np.float64) for t in (call.Q, call.K, call.V, call.ctx))
    dctx = A.attention_error_bound(Qg, Kg, Vg, batch, seq, 12, 64)
    scale = 64 ** -0.5
    for b in range(batch):
        rows = slice(b * seq, (b + 1) * seq)
        for h in range(12):
            cols = slice(h * 64, (h + 1) * 64)
            q, k, v = Q64[rows, cols], K64[rows, cols], V64[rows, cols]
            s = scale * (q @ k.T)
            p = np.exp(s - s.max(axis=1, keepdims=True))
            p /= p.sum(axis=1, keepdims=True)
            D = scale * (dQ[rows, cols] @ np.abs(k).T + np.abs(q) @ dK[rows, cols].T
                         + dQ[rows, cols] @ dK[rows, cols].T)
            f = np.exp(2 * D.max(axis=1, keepdims=True))
            dctx[rows, cols] += (f - 1) * (p @ np.abs(v)) + f * (p @ dV[rows, cols])
    bound = 1e-5 * O.tolerance_scale(ctxg, Wd[3]) + 1e-6 + dctx @ np.abs(Wd[3]).T
    err = np.abs(host(Y).astype(np.float64) - Y64)
    log(f"end to end {R}x{C} {batch}x{seq}: worst err/bound {np.max(err / bound):.3g}")
    assert np.all(np.isfinite(host(Y)))
    assert np.all(err <= bound)


def test_attention_block_graph_replay(device):
    """The block captured in a HIP graph replays bit-identically to the eager call."""
    w, mats, call = _block(32, 1, 0.1, 1, 128)
    ref = call().clone()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        call()
    for rep in range(3):
        call.Y.fill_(float("nan"))
        call.ctx.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(call.Y.view(torch.int32), ref.view(torch.int32)), f"replay {rep}"


def test_attention_block_plans_bit_identical(device):
    """The block with per-matrix plans (the default for 32x1 weights) gives the same Y, bit for
    bit, as the block without them; shapes without plans run unplanned."""
    w, mats, call = _block(32, 1, 0.1, 2, 128)
    assert all(p is not None for p in call.plans)
    X = dev(w.X[0])
    biases = [dev(prj.bias) for prj in w.projections]
    plain = B.AttentionBlockCall(X, mats[0], biases[0], mats[1], biases[1], mats[2], biases[2],
                                 mats[3], biases[3], 2, 128, 12, plans=False)
    assert all(p is None for p in plain.plans)
    Y1, Y0 = call(), plain()
    torch.cuda.synchronize()
    for a, b in ((call.Q, plain.Q), (call.K, plain.K), (call.V, plain.V), (Y1, Y0)):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    _, _, sq = _block(16, 16, 0.2, 1, 64)
    assert all(p is None for p in sq.plans)
