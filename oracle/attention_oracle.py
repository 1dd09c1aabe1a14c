"""Plain CPU oracle for the synthetic BERT attention block built around the BSR products.

TEST INFRASTRUCTURE ONLY.  The test suite, the smoke check and the benchmark's CPU-baseline leg
may import this module; the library's product path never does.  It shares no code with the GPU
kernels and imports nothing from the library package.

The paper prunes the attention weights of BERT (Sec. 2.3; Sec. 1 names attention weights as the
pruned parameters) and times end-to-end inference (Table 1).  The block computed here is the
attention layer those weights belong to, with the pruned projections as BSR products:

    Q = X Wq^T + bq,  K = X Wk^T + bk,  V = X Wv^T + bv        (three BSR products, Sec. 2.2)
    ctx[b, s, head h] = sum_j softmax_j(scale * <Q[b,s,h], K[b,j,h]>) V[b,j,h]
    Y = ctx Wo^T + bo                                           (a fourth BSR product)

with the standard scaled dot-product attention of the Transformer that BERT uses (the paper
cites it for the attention kernels): scale = 1/sqrt(head_dim), no mask (every token attends to
every token of its sequence).  Rows are tokens t = b * seq + s; head h owns columns
h * head_dim .. (h + 1) * head_dim - 1 of Q, K, V and ctx.  Everything is fp64.
"""

from __future__ import annotations

import math

import numpy as np

U32 = 2.0 ** -24   # unit roundoff of fp32


def attention(Q, K, V, batch: int, seq: int, heads: int, head_dim: int,
              scale: float | None = None) -> np.ndarray:
    """ctx = softmax(scale * Q_bh K_bh^T) V_bh for every sequence b and head h, in fp64.

    The softmax subtracts each row's maximum before exponentiating (the value is unchanged; it
    only keeps exp finite).
    """
    if scale is None:
        scale = 1.0 / math.sqrt(head_dim)
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    T = batch * seq
    width = heads * head_dim
    if Q.shape[0] != T or Q.shape[1] < width or K.shape[0] != T or V.shape[0] != T:
        raise ValueError("Q, K, V must be (batch * seq) x (heads * head_dim)")
    ctx = np.zeros((T, width), dtype=np.float64)
    for b in range(batch):
        rows = slice(b * seq, (b + 1) * seq)
        for h in range(heads):
            cols = slice(h * head_dim, (h + 1) * head_dim)
            s = scale * (Q[rows, cols] @ K[rows, cols].T)          # [query, key]
            s = s - s.max(axis=1, keepdims=True)
            e = np.exp(s)
            p = e / e.sum(axis=1, keepdims=True)
            ctx[rows, cols] = p @ V[rows, cols]
    return ctx


def attention_error_bound(Q, K, V, batch: int, seq: int, heads: int, head_dim: int,
                          scale: float | None = None) -> np.ndarray:
    """First-order bound on |ctx_fp32 - ctx_fp64| for an fp32 kernel given the same fp32 inputs.

    Scores s_j = scale * sum_d q_d k_jd carry an error <= (head_dim + 2) u sigma_j, with
    sigma_j = scale * sum_d |q_d k_jd| and u = 2^-24.  Each weight e_j = exp(s_j - m) then has
    a relative error eps_j <= (head_dim + 2) u sigma_j + u |s_j - m| + 4u (the exponential to
    within a few ulp; the shift m cancels in the ratio).  Perturbing the weights of
    ctx = sum_j e_j v_j / sum_j e_j by factors (1 + eps_j) moves it by at most
    2 max_j eps_j * sum_j p_j |v_j|; summing seq terms in fp32 adds (seq + 2) u per sum, twice.
    Returns, per element, 2 max_j eps_j * A + 2 (seq + 2) u * A + u |ctx|, with
    A = sum_j p_j |v_jd|.
    """
    if scale is None:
        scale = 1.0 / math.sqrt(head_dim)
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    T = batch * seq
    width = heads * head_dim
    bound = np.zeros((T, width), dtype=np.float64)
    for b in range(batch):
        rows = slice(b * seq, (b + 1) * seq)
        for h in range(heads):
            cols = slice(h * head_dim, (h + 1) * head_dim)
            q, k, v = Q[rows, cols], K[rows, cols], V[rows, cols]
            s = scale * (q @ k.T)
            sigma = scale * (np.abs(q) @ np.abs(k).T)
            m = s.max(axis=1, keepdims=True)
            p = np.exp(s - m)
            p = p / p.sum(axis=1, keepdims=True)
            eps = (head_dim + 2) * U32 * sigma + U32 * np.abs(s - m) + 4 * U32
            A = p @ np.abs(v)
            ctx = p @ v
            bound[rows, cols] = (2 * eps.max(axis=1, keepdims=True) * A
                                 + 2 * (seq + 2) * U32 * A + U32 * np.abs(ctx))
    return bound


def attention_block(X, Wq, bq, Wk, bk, Wv, bv, Wo, bo, batch: int, seq: int, heads: int):
    """The whole block in fp64 from dense (already masked) weights: returns (Q, K, V, ctx, Y).

    W* are N x K row-major [out][in] (zeros where blocks were pruned); biases may be None.
    """
    X = np.asarray(X, dtype=np.float64)

    def lin(W, b):
        y = X @ np.asarray(W, dtype=np.float64).T
        return y if b is None else y + np.asarray(b, dtype=np.float64)

    Q, K, V = lin(Wq, bq), lin(Wk, bk), lin(Wv, bv)
    head_dim = Q.shape[1] // heads
    ctx = attention(Q, K, V, batch, seq, heads, head_dim)
    Y = ctx @ np.asarray(Wo, dtype=np.float64).T
    if bo is not None:
        Y = Y + np.asarray(bo, dtype=np.float64)
    return Q, K, V, ctx, Y
