"""Pins of the IHT oracle (oracle/iht_oracle.py) to facts that do not come from its own code.

* Hand-worked examples (tests/golden/iht_examples.json): two iterations in exact decimals, one
  below the step bound (monotone convergence), one above it (the kept entry switches), and a
  block-norm decision with 1x2 blocks.
* With H = I and eta = 1 every iterate is the one-shot projection of W0, which must equal the
  pinned one-shot prune (bsr_oracle.prune).
* With k = all blocks there is no constraint, and the iterates of gradient descent on the
  quadratic have the closed form W_t - W0 = (W_start - W0)(I - eta H)^t (a matrix power).
* The gradient is the derivative of the objective (central differences), and the objective with
  H = gram(X) is the output reconstruction error 1/(2T)||X W^T - X W0^T||^2 computed directly.
* For eta <= 1 / lambda_max(H) the objective never increases along the iterates.
* update_f32 matches fp64 within fp32 rounding, and is exact on small integers.
"""
import json
import os

import numpy as np
import pytest

from oracle import bsr_oracle as O
from oracle import iht_oracle as I

HERE = os.path.dirname(os.path.abspath(__file__))


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def test_hand_examples():
    with open(os.path.join(HERE, "golden", "iht_examples.json")) as f:
        ex = json.load(f)["examples"]
    for e in ex:
        W0, H = np.array(e["W0"]), np.array(e["H"])
        tr = I.iht(W0, H, e["R"], e["C"], e["k"], e["eta"], e["iters"])
        assert len(tr) == len(e["iterates"])
        for W, want in zip(tr, e["iterates"]):
            np.testing.assert_allclose(W, np.array(want), rtol=0, atol=1e-12, err_msg=e["name"])
        fs = [I.objective(W, W0, H) for W in tr]
        np.testing.assert_allclose(fs, e["objective"], rtol=1e-12, err_msg=e["name"])


@pytest.mark.parametrize("R,C", [(32, 1), (1, 32), (4, 4), (1, 1)])
def test_identity_hessian_unit_step_is_one_shot_prune(R, C):
    g = rng(R * 100 + C)
    W0 = g.standard_normal((64, 96)).astype(np.float32)
    k = O.prune_count(64, 96, R, C, 0.2)
    tr = I.iht(W0, np.eye(96), R, C, k, 1.0, 3)
    want = O.to_dense(*O.prune(W0, R, C, k=k), 64, 96)
    for W in tr:
        assert np.array_equal(W, want)
    # Equal block norms everywhere: the one-shot prune keeps the lowest block ids.
    Wt = np.ones((64, 96), dtype=np.float32)
    want = O.to_dense(*O.prune(Wt, R, C, k=k), 64, 96)
    assert np.array_equal(I.iht(Wt, np.eye(96), R, C, k, 1.0, 1)[-1], want)


def test_unconstrained_closed_form():
    g = rng(2)
    N, K = 8, 12
    W0 = g.standard_normal((N, K))
    Ws = g.standard_normal((N, K))
    X = g.standard_normal((40, K))
    H = I.gram(X)
    eta = 0.5 / np.linalg.eigvalsh(H)[-1]
    nb = N * K
    tr = I.iht(W0, H, 1, 1, nb, eta, 6, W_start=Ws)
    M = np.eye(K) - eta * H
    for t, W in enumerate(tr):
        want = W0 + (Ws - W0) @ np.linalg.matrix_power(M, t)
        np.testing.assert_allclose(W, want, rtol=1e-10, atol=1e-12)


def test_gradient_is_derivative_of_objective():
    g = rng(3)
    N, K = 5, 7
    W0, W = g.standard_normal((N, K)), g.standard_normal((N, K))
    H = I.gram(g.standard_normal((30, K)))
    G = I.gradient(W, W0, H)
    h = 1e-6
    for i in range(N):
        for j in range(K):
            E = np.zeros((N, K))
            E[i, j] = h
            fd = (I.objective(W + E, W0, H) - I.objective(W - E, W0, H)) / (2 * h)
            assert abs(fd - G[i, j]) <= 1e-6 * max(1.0, abs(G[i, j]))


def test_objective_is_reconstruction_error():
    g = rng(4)
    T, N, K = 50, 6, 9
    X, W0, W = g.standard_normal((T, K)), g.standard_normal((N, K)), g.standard_normal((N, K))
    direct = 0.5 / T * float(np.sum((X @ W.T - X @ W0.T) ** 2))
    assert abs(I.objective(W, W0, I.gram(X)) - direct) <= 1e-12 * direct


@pytest.mark.parametrize("R,C,density", [(32, 1, 0.1), (4, 4, 0.25), (1, 1, 0.3), (1, 32, 0.2)])
def test_objective_never_increases_below_the_step_bound(R, C, density):
    g = rng(R * 7 + C)
    N, K, T = 64, 64, 256
    W0 = g.standard_normal((N, K))
    X = g.standard_normal((T, K)) * np.linspace(0.2, 2.0, K)   # uneven input scales
    X[:, 1:] += 0.5 * X[:, :-1]                                   # correlated inputs
    H = I.gram(X)
    eta = 1.0 / np.linalg.eigvalsh(H)[-1]
    k = O.prune_count(N, K, R, C, density)
    tr = I.iht(W0, H, R, C, k, eta, 15)
    fs = [I.objective(W, W0, H) for W in tr]
    for a, b in zip(fs, fs[1:]):
        assert b <= a * (1 + 1e-12)
    assert fs[-1] < fs[0]          # the iteration improves on the one-shot prune here
    for W in tr:                    # every iterate is feasible: at most k nonzero blocks
        assert np.count_nonzero(I.block_keys64(W, R, C)) <= k


def test_update_f32_rounding():
    g = rng(6)
    N, K = 16, 24
    W = g.standard_normal((N, K)).astype(np.float32)
    G = g.standard_normal((K, N)).astype(np.float32)
    C0 = g.standard_normal((K, N)).astype(np.float32)
    eta = 0.37
    V = I.update_f32(W, G, C0, eta)
    assert V.dtype == np.float32
    V64 = W.astype(np.float64) - np.float64(np.float32(eta)) * (G.T.astype(np.float64) - C0.T)
    err = np.abs(V.astype(np.float64) - V64)
    bound = 2.0 ** -23 * (np.abs(W) + 3 * abs(eta) * (np.abs(G.T) + np.abs(C0.T)))
    assert np.all(err <= bound)
    Wi = g.integers(-8, 9, (N, K)).astype(np.float32)
    Gi = g.integers(-8, 9, (K, N)).astype(np.float32)
    Ci = g.integers(-8, 9, (K, N)).astype(np.float32)
    assert np.array_equal(I.update_f32(Wi, Gi, Ci, 0.5), Wi - 0.5 * (Gi.T - Ci.T))
