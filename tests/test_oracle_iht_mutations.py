"""The IHT oracle's pins have teeth: each plausible mistake planted in the oracle (monkeypatched
for one test, on the CPU) fails some pin of tests/test_oracle_iht.py."""
import numpy as np
import pytest

from oracle import bsr_oracle as O
from oracle import iht_oracle as I
import tests.test_oracle_iht as P

_orig = {name: getattr(I, name) for name in ("gradient", "objective", "gram", "project",
                                              "block_keys64", "iht", "update_f32")}


def _gradient_without_w0(W, W0, H):
    return np.asarray(W, dtype=np.float64) @ H


def _gradient_sign(W, W0, H):
    return -_orig["gradient"](W, W0, H)


def _objective_without_half(W, W0, H):
    return 2.0 * _orig["objective"](W, W0, H)


def _gram_without_mean(X):
    X = np.asarray(X, dtype=np.float64)
    return X.T @ X


def _keys_l1(V, R, C):
    V = np.abs(np.asarray(V, dtype=np.float64))
    N, K = V.shape
    return V.reshape(N // R, R, K // C, C).sum(axis=(1, 3)).ravel()


def _project_keeps_smallest(V, R, C, k):
    V = np.asarray(V, dtype=np.float64)
    N, K = V.shape
    key = _orig["block_keys64"](V, R, C)
    order = np.lexsort((np.arange(key.size), key))
    keep = np.zeros(key.size, dtype=bool)
    keep[order[:int(k)]] = True
    keep = keep.reshape(N // R, K // C)
    return np.where(np.repeat(np.repeat(keep, R, 0), C, 1), V, 0.0)


def _project_ties_to_higher_id(V, R, C, k):
    V = np.asarray(V, dtype=np.float64)
    N, K = V.shape
    key = _orig["block_keys64"](V, R, C)
    ids = np.arange(key.size)
    order = np.lexsort((-ids, -key))
    keep = np.zeros(key.size, dtype=bool)
    keep[order[:int(k)]] = True
    keep = keep.reshape(N // R, K // C)
    return np.where(np.repeat(np.repeat(keep, R, 0), C, 1), V, 0.0)


def _iht_unprojected_start(W0, H, R, C, k, eta, iters, W_start=None):
    W0 = np.asarray(W0, dtype=np.float64)
    W = W0 if W_start is None else np.asarray(W_start, dtype=np.float64)
    out = [W]
    for _ in range(iters):
        W = I.project(W - eta * I.gradient(W, W0, H), R, C, k)
        out.append(W)
    return out


def _update_f32_in_fp64(W, G, C0, eta):
    d = np.asarray(G, dtype=np.float64).T - np.asarray(C0, dtype=np.float64).T
    return (np.asarray(W, dtype=np.float64) - eta * d).astype(np.float32) * np.float32(1.0 + 2**-20)


MUTANTS = {
    "gradient without W0": ("gradient", _gradient_without_w0),
    "gradient sign": ("gradient", _gradient_sign),
    "objective without 1/2": ("objective", _objective_without_half),
    "gram without 1/T": ("gram", _gram_without_mean),
    "l1 block keys": ("block_keys64", _keys_l1),
    "projection keeps the smallest blocks": ("project", _project_keeps_smallest),
    "projection ties to the higher id": ("project", _project_ties_to_higher_id),
    "first iterate not projected": ("iht", _iht_unprojected_start),
    "update rounding off": ("update_f32", _update_f32_in_fp64),
}


def _all_pins():
    P.test_hand_examples()
    for R, C in [(32, 1), (1, 32), (4, 4), (1, 1)]:
        P.test_identity_hessian_unit_step_is_one_shot_prune(R, C)
    P.test_unconstrained_closed_form()
    P.test_gradient_is_derivative_of_objective()
    P.test_objective_is_reconstruction_error()
    for R, C, d in [(32, 1, 0.1), (4, 4, 0.25), (1, 1, 0.3), (1, 32, 0.2)]:
        P.test_objective_never_increases_below_the_step_bound(R, C, d)
    P.test_update_f32_rounding()


def test_pins_pass_unmutated():
    _all_pins()


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_planted_mistake_is_caught(mutant, monkeypatch):
    name, fn = MUTANTS[mutant]
    monkeypatch.setattr(I, name, fn)
    with pytest.raises(AssertionError):
        _all_pins()
