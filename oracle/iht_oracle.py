"""Plain CPU oracle for the iterative projection (iterative hard thresholding) of Eq. 2.

TEST INFRASTRUCTURE ONLY.  The test suite may import this module; the library's path never
does.  It shares no code with the GPU kernels and imports nothing from the library package.

Sec. 2.1 states pruning as a constrained problem (Eq. 2): minimise a loss f0(w) subject to a
bound tau on the structured norm of Eq. 3.  With p = 0 and blocks as the groups, the bound caps
the number of nonzero blocks at k = tau, and the constraint set is "at most k nonzero blocks".
The one-shot prune (bsr_oracle.prune) is the Euclidean projection onto that set.  The paper
minimises its training loss; with no data here, the loss is a quadratic stand-in (a reading of
the paper): the reconstruction error of the layer's output on calibration activations X
(T x K),

    f(W) = 1/(2T) || X W^T - X W0^T ||_F^2 = 1/2 tr((W - W0) H (W - W0)^T),   H = X^T X / T,

whose gradient is (W - W0) H.  Projected gradient descent on Eq. 2 (iterative hard
thresholding) takes, from W_0 = P_k(W0),

    W_{t+1} = P_k(W_t - eta (W_t - W0) H),

with P_k the projection that keeps the k blocks of largest l2 norm (ties to the lower row-major
block id, as in the one-shot prune) and zeroes the rest.  For a constant step eta <= 1 / lambda_max
(H), f never increases along the iterates.

Everything here is fp64.  update_f32 spells out, operation by operation, the fp32 arithmetic of
the GPU's update step (V = W - eta (G - C0), each operation rounded to fp32, no fused
multiply-add), for a bit-exact comparison of that one kernel.
"""

from __future__ import annotations

import numpy as np

from oracle import bsr_oracle as O


def gram(X: np.ndarray) -> np.ndarray:
    """H = X^T X / T in fp64 (the Hessian of the reconstruction loss)."""
    X = np.asarray(X, dtype=np.float64)
    return X.T @ X / X.shape[0]


def objective(W: np.ndarray, W0: np.ndarray, H: np.ndarray) -> float:
    """f(W) = 1/2 tr((W - W0) H (W - W0)^T)."""
    E = np.asarray(W, dtype=np.float64) - np.asarray(W0, dtype=np.float64)
    return 0.5 * float(np.sum((E @ H) * E))


def gradient(W: np.ndarray, W0: np.ndarray, H: np.ndarray) -> np.ndarray:
    """grad f(W) = (W - W0) H (N x K)."""
    return (np.asarray(W, dtype=np.float64) - np.asarray(W0, dtype=np.float64)) @ H


def block_keys64(V: np.ndarray, R: int, C: int) -> np.ndarray:
    """Squared l2 norm of every block of an fp64 matrix, row-major block order, summed
    sequentially (row r outer, column c inner) from +0.0."""
    V = np.asarray(V, dtype=np.float64)
    N, K = V.shape
    Nb, Kb = O.check_shape(N, K, R, C)
    b = V.reshape(Nb, R, Kb, C)
    key = np.zeros((Nb, Kb), dtype=np.float64)
    for r in range(R):
        for c in range(C):
            key = key + b[:, r, :, c] * b[:, r, :, c]
    return key.reshape(-1)


def project(V: np.ndarray, R: int, C: int, k: int) -> np.ndarray:
    """P_k(V): V with all but its k blocks of largest l2 norm set to zero (ties to the lower
    block id), fp64."""
    V = np.asarray(V, dtype=np.float64)
    N, K = V.shape
    Nb, Kb = O.check_shape(N, K, R, C)
    keep = O.select_topk(block_keys64(V, R, C), int(k)).reshape(Nb, Kb)
    mask = np.repeat(np.repeat(keep, R, axis=0), C, axis=1)
    return np.where(mask, V, 0.0)


def iht(W0: np.ndarray, H: np.ndarray, R: int, C: int, k: int, eta: float, iters: int,
        W_start: np.ndarray | None = None) -> list[np.ndarray]:
    """The iterates [W_0, W_1, ..., W_iters] of projected gradient descent on Eq. 2 with the
    quadratic loss above; W_0 = P_k(W0) unless W_start is given (then W_0 = P_k(W_start))."""
    W0 = np.asarray(W0, dtype=np.float64)
    W = project(W0 if W_start is None else W_start, R, C, k)
    out = [W]
    for _ in range(iters):
        W = project(W - eta * gradient(W, W0, H), R, C, k)
        out.append(W)
    return out


def update_f32(W: np.ndarray, G: np.ndarray, C0: np.ndarray, eta: float) -> np.ndarray:
    """The GPU update step in its own fp32 arithmetic: V[n, j] = W[n, j] - eta * (G[j, n] -
    C0[j, n]), where G = H W^T and C0 = H W0^T are K x N (the products' outputs).  Each of the
    subtraction, the product and the final subtraction is rounded to fp32."""
    W = np.asarray(W, dtype=np.float32)
    d = np.asarray(G, dtype=np.float32).T - np.asarray(C0, dtype=np.float32).T
    m = np.float32(eta) * d
    return W - m
