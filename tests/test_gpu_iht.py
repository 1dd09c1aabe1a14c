"""The iterative projection for Eq. 2 (bsr_iht_update and the bsr_iht driver) on the GPU.

* The update kernel equals the oracle's fp32 spelling of it (update_f32) bit for bit, pitched
  and in place.
* Every step of a GPU run: its update V_t meets a bound derived from the products' tolerance
  against the fp64 update of the same iterate, and the next iterate is the oracle's prune of the
  GPU's own V_t, bit for bit (the keep decisions are taken on the same fp32 values).
* Whole runs: the kept blocks of every GPU iterate equal those of the fp64 oracle's iterates, and
  the loss never rises for eta = 1 / lambda_max(H); with H = I and eta = 1 every iterate is the
  one-shot prune.
H is the oracle's Gram matrix of seeded synthetic calibration activations, rounded to fp32.
"""
import zlib

import numpy as np
import pytest
import torch

from oracle import bsr_oracle as O
from oracle import iht_oracle as I
from paper_2106_08846_amd import bsr as B
from tests.gpu_common import dev, host, log

pytestmark = pytest.mark.gpu


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def bits(a) -> np.ndarray:
    return np.ascontiguousarray(host(a) if isinstance(a, torch.Tensor) else a).view(np.uint32)


def dense_of(M: B.BSRMatrix) -> np.ndarray:
    return host(B.bsr_to_dense(M))


def problem(name, N, K, T=512):
    g = rng(zlib.crc32(name.encode()) % 10000)
    W0 = (g.standard_normal((N, K)) * 0.05).astype(np.float32)
    X = g.standard_normal((T, K)) * np.linspace(0.3, 1.5, K)
    X[:, 1:] += 0.6 * X[:, :-1]
    H = I.gram(X).astype(np.float32)
    eta = float(np.float32(1.0 / np.linalg.eigvalsh(H.astype(np.float64))[-1]))
    return W0, H, eta


@pytest.mark.parametrize("N,K,pitch,inplace", [(37, 100, 0, False), (256, 768, 3, False),
                                               (768, 768, 0, True), (1, 1, 0, False)])
def test_update_bit_exact(device, N, K, pitch, inplace):
    g = rng(N * 1000 + K)
    W = g.standard_normal((N, K)).astype(np.float32)
    G = g.standard_normal((K, N)).astype(np.float32)
    C0 = g.standard_normal((K, N)).astype(np.float32)
    eta = 0.173
    want = I.update_f32(W, G, C0, eta)

    def pitched(a):
        big = torch.full((a.shape[0], a.shape[1] + pitch), 9.0, device=device)
        big[:, :a.shape[1]] = dev(a)
        return big, big[:, :a.shape[1]]
    _, Wd = pitched(W)
    gb, Gd = pitched(G)
    cb, Cd = pitched(C0)
    if inplace:
        V = B.bsr_iht_update(Wd, Gd, Cd, eta, V=Wd)
    else:
        vb, Vd = pitched(np.zeros((N, K), np.float32))
        V = B.bsr_iht_update(Wd, Gd, Cd, eta, V=Vd)
    torch.cuda.synchronize()
    assert np.array_equal(bits(V), want.view(np.uint32))
    if pitch:
        assert torch.all(gb[:, N:] == 9.0) and torch.all(cb[:, N:] == 9.0)
        assert torch.all(vb[:, K:] == 9.0)


CASES = [
    # name, N, K, R, C, density, iters
    ("32x1", 256, 256, 32, 1, 0.1, 8),
    ("1x32", 256, 256, 1, 32, 0.2, 6),
    ("16x16", 256, 256, 16, 16, 0.25, 6),
    ("4x4", 128, 192, 4, 4, 0.2, 6),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_iht_steps_and_trajectory(device, case):
    name, N, K, R, C, d, iters = case
    log(f"iht case {name}")
    W0, H, eta = problem(name, N, K)
    k = O.prune_count(N, K, R, C, d)
    M, hist = B.bsr_iht(dev(W0), dev(H), R, C, k, eta, iters, trace=True)
    torch.cuda.synchronize()
    Wg = [host(Wt) for _, Wt in hist] + [dense_of(M)]
    # The first iterate is the one-shot prune of W0.
    assert np.array_equal(Wg[0], O.to_dense(*O.prune(W0, R, C, k=k), N, K))
    H64, W064 = H.astype(np.float64), W0.astype(np.float64)
    Hs = np.abs(H64)
    for t, (Vt, _) in enumerate(hist):
        V = host(Vt)
        Wt = Wg[t].astype(np.float64)
        G64 = H64 @ Wt.T                                   # K x N
        C64 = H64 @ W064.T
        V64 = Wt - eta * (G64 - C64).T
        SG = Hs @ np.abs(Wt).T
        SC = Hs @ np.abs(W064).T
        bound = (eta * (1e-5 * (SG + SC) + 2e-6)).T + 2.0 ** -22 * (
            np.abs(Wt) + eta * (np.abs(G64) + np.abs(C64)).T)
        err = np.abs(V.astype(np.float64) - V64)
        assert np.all(err <= bound), f"step {t}: worst err/bound {np.max(err / bound):.3f}"
        # The next iterate: the oracle's prune of this very V, bit for bit.
        assert np.array_equal(bits(Wg[t + 1]), bits(O.to_dense(*O.prune(V, R, C, k=k), N, K)))
    # The whole run against the fp64 oracle: the same kept blocks at every step, and a loss
    # that never rises.
    ref = I.iht(W064, H64, R, C, k, eta, iters)
    fs = []
    for t, (Wt, Wr) in enumerate(zip(Wg, ref)):
        kg = I.block_keys64(Wt, R, C) > 0
        kr = I.block_keys64(Wr, R, C) > 0
        assert np.array_equal(kg, kr), f"kept blocks differ at step {t}"
        fs.append(I.objective(Wt, W064, H64))
    for a, b in zip(fs, fs[1:]):
        assert b <= a * (1 + 1e-5)
    assert fs[-1] < fs[0]


def test_iht_identity_hessian_is_one_shot_prune(device):
    g = rng(77)
    N, K, R, C = 128, 256, 32, 1
    W0 = g.standard_normal((N, K)).astype(np.float32)
    k = O.prune_count(N, K, R, C, 0.15)
    M, hist = B.bsr_iht(dev(W0), torch.eye(K, device=device), R, C, k, 1.0, 3, trace=True)
    want = O.to_dense(*O.prune(W0, R, C, k=k), N, K)
    for V, Wt in hist:
        assert np.array_equal(bits(Wt), want.view(np.uint32))
    assert np.array_equal(bits(dense_of(M)), want.view(np.uint32))
