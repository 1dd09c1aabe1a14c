"""The global top-k selection on both sides of its register-resident limit.

Weights with at most 32768 blocks are selected with every key held in the registers of one
workgroup (32 keys per thread, thread order = block-id order); larger ones stream the keys from
memory.  Both must give the oracle's BSR arrays bit for bit, in particular where keys tie (the
lower block id wins, Sec. 2.1 Eq. 2 read with ties broken by id), where every key shares its
leading bytes, and for non-finite weights.  Sizes sit at the limit (32767, 32768 and 32769
blocks) and k runs from 1 to nb.
"""
import numpy as np
import pytest

from paper_2106_08846_amd import bsr as B

from .gpu_common import check_prune, log, prune_on_gpu

pytestmark = pytest.mark.gpu

LIMIT = 1024 * 32


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


SHAPES = [
    # N, K, R, C  (nb = N/R * K/C)
    (1024, 1024, 32, 1),    # 32768 blocks: the register limit exactly
    (1, 32767, 1, 1),       # one below, a partial last thread
    (3, 10923, 1, 1),       # 32769 blocks: one above, streamed
    (96, 768, 32, 1),       # 2304 blocks: most threads empty
]


def weights(kind: str, N: int, K: int, seed: int) -> np.ndarray:
    g = rng(seed)
    if kind == "normal":
        return (g.standard_normal((N, K)) * 0.02).astype(np.float32)
    if kind == "ties":     # few distinct values: many equal keys
        return g.integers(-2, 3, (N, K)).astype(np.float32)
    if kind == "narrow":   # keys in [1, 1 + 2^-20): identical leading bytes
        return (1.0 + g.random((N, K)) * 2.0 ** -21).astype(np.float32)
    W = (g.standard_normal((N, K)) * 0.02).astype(np.float32)   # non-finite
    flat = W.reshape(-1)
    idx = g.choice(flat.size, 12, replace=False)
    flat[idx[:4]] = np.nan
    flat[idx[4:8]] = np.inf
    flat[idx[8:]] = -np.inf
    return W


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{s[0]}x{s[1]}_{s[2]}x{s[3]}" for s in SHAPES])
@pytest.mark.parametrize("kind", ["normal", "ties", "narrow", "nonfinite"])
def test_select_bit_exact(device, shape, kind):
    N, K, R, C = shape
    nb = (N // R) * (K // C)
    W = weights(kind, N, K, seed=nb % 1000 + len(kind))
    for k in sorted({1, 7, nb // 10, nb // 2, nb - 1, nb}):
        log(f"select {kind} {N}x{K} {R}x{C} nb={nb} ({'registers' if nb <= LIMIT else 'streamed'}) k={k}")
        M = prune_on_gpu(W, R, C, k)
        check_prune(W, R, C, M, k)


def test_select_all_keys_equal(device):
    """Every key equal (no radix pass is needed): the k lowest ids are kept."""
    W = np.full((1024, 1024), 0.5, dtype=np.float32)
    for k in (1, 1000, LIMIT):
        M = prune_on_gpu(W, 32, 1, k)
        check_prune(W, 32, 1, M, k)
