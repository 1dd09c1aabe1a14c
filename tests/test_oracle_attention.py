"""Pins for the attention oracle: closed forms, invariances, torch's fp64 attention and a
40-digit reference; planted mistakes in the oracle must trip them."""
import json
import math
import os
from fractions import Fraction

import mpmath
import numpy as np
import pytest
import torch

from oracle import attention_oracle as A
from oracle import bsr_oracle as O


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def qkv(seed, batch, seq, heads, d, sd=1.0):
    g = rng(seed)
    T, W = batch * seq, heads * d
    return [(g.standard_normal((T, W)) * sd).astype(np.float32) for _ in range(3)]


def pin_uniform_keys_give_the_mean():
    """Equal keys within a sequence and head: every weight is 1/seq, ctx is the mean of V."""
    Q, K, V = qkv(1, 2, 5, 3, 4)
    for b in range(2):
        K[b * 5:(b + 1) * 5] = K[b * 5]
    ctx = A.attention(Q, K, V, 2, 5, 3, 4)
    for b in range(2):
        for c in range(12):
            mean = sum(Fraction(float(V[b * 5 + j, c])) for j in range(5)) / 5
            for s in range(5):
                assert abs(ctx[b * 5 + s, c] - float(mean)) <= 1e-15 * (1 + abs(float(mean)))


def pin_single_token_is_v():
    Q, K, V = qkv(2, 3, 1, 2, 8)
    assert np.array_equal(A.attention(Q, K, V, 3, 1, 2, 8), V.astype(np.float64))


def pin_key_shift_invariance():
    """Adding one vector c to every key of a (sequence, head) adds <q, c> to a whole row of
    scores, which the softmax ignores."""
    Q, K, V = qkv(3, 2, 6, 2, 4)
    K2 = K.astype(np.float64).copy()
    c = rng(4).standard_normal(4)
    K2[0:6, 4:8] += c
    K2[6:12, 0:4] -= 2 * c
    a = A.attention(Q, K, V, 2, 6, 2, 4)
    b = A.attention(Q, K2, V, 2, 6, 2, 4)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-13)


def pin_key_permutation_invariance():
    Q, K, V = qkv(5, 1, 9, 2, 4)
    perm = rng(6).permutation(9)
    a = A.attention(Q, K, V, 1, 9, 2, 4)
    b = A.attention(Q, K[perm], V[perm], 1, 9, 2, 4)
    assert np.allclose(a, b, rtol=1e-13, atol=1e-14)


def pin_matches_torch_sdpa_fp64():
    batch, seq, heads, d = 2, 13, 3, 8
    Q, K, V = qkv(7, batch, seq, heads, d, sd=2.0)

    def split(x):
        return torch.from_numpy(x.astype(np.float64)).reshape(batch, seq, heads, d).transpose(1, 2)

    ref = torch.nn.functional.scaled_dot_product_attention(split(Q), split(K), split(V))
    ref = ref.transpose(1, 2).reshape(batch * seq, heads * d).numpy()
    assert np.allclose(A.attention(Q, K, V, batch, seq, heads, d), ref, rtol=1e-12, atol=1e-13)


def pin_matches_40_digit_reference():
    Q, K, V = qkv(8, 1, 5, 2, 4, sd=3.0)
    mpmath.mp.dps = 40
    ctx = A.attention(Q, K, V, 1, 5, 2, 4)
    for h in range(2):
        cols = range(4 * h, 4 * h + 4)
        for s in range(5):
            sc = [mpmath.mpf(0.5) * mpmath.fsum(mpmath.mpf(float(Q[s, c])) * mpmath.mpf(float(K[j, c]))
                                               for c in cols) for j in range(5)]
            e = [mpmath.exp(x) for x in sc]
            z = mpmath.fsum(e)
            for c in cols:
                exact = mpmath.fsum(e[j] * mpmath.mpf(float(V[j, c])) for j in range(5)) / z
                assert abs(ctx[s, c] - float(exact)) <= 1e-14 * (1 + abs(float(exact)))


def pin_fp32_computation_is_within_the_bound():
    """An fp32 evaluation (numpy float32 throughout) lies within attention_error_bound."""
    for seed, (batch, seq, heads, d, sd) in enumerate([(1, 128, 4, 64, 0.3), (2, 77, 2, 64, 1.0),
                                                      (1, 512, 1, 64, 0.2), (1, 33, 3, 32, 3.0)]):
        Q, K, V = qkv(20 + seed, batch, seq, heads, d, sd)
        ctx64 = A.attention(Q, K, V, batch, seq, heads, d)
        bound = A.attention_error_bound(Q, K, V, batch, seq, heads, d)
        scale = np.float32(1.0 / math.sqrt(d))
        for b in range(batch):
            r = slice(b * seq, (b + 1) * seq)
            for h in range(heads):
                c = slice(h * d, (h + 1) * d)
                s = (Q[r, c] @ K[r, c].T) * scale
                e = np.exp(s - s.max(axis=1, keepdims=True))
                ctx32 = (e @ V[r, c]) / e.sum(axis=1, keepdims=True)
                assert ctx32.dtype == np.float32
                assert np.all(np.abs(ctx32 - ctx64[r, c]) <= bound[r, c])


def pin_bound_hand_worked():
    """attention_error_bound on a case worked by hand (tests/golden/hand_examples.json)."""
    with open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")) as f:
        ex = json.load(f)["attention_examples"][0]
    Q, K, V = (np.array(ex[n], dtype=np.float32) for n in ("Q", "K", "V"))
    args = (ex["batch"], ex["seq"], ex["heads"], ex["head_dim"], ex["scale"])
    ctx = A.attention(Q, K, V, *args)
    assert np.allclose(ctx, np.array(ex["ctx"]), rtol=1e-15, atol=0)
    bound = A.attention_error_bound(Q, K, V, *args)
    want = np.array(ex["bound_in_units_of_2^-24"], dtype=np.float64) * 2.0 ** -24
    assert np.allclose(bound, want, rtol=1e-12, atol=0)


def pin_bound_is_not_loose():
    """The bound is a first-order worst case, but not a loose one: on the same four fp32
    evaluations as above, the largest error reaches at least 1/500 of it (measured: 0.011, 0.0067,
    0.0019 and 0.011 of the bound).  A bound ten times too large fails here."""
    worst = 0.0
    for seed, (batch, seq, heads, d, sd) in enumerate([(1, 128, 4, 64, 0.3), (2, 77, 2, 64, 1.0),
                                                      (1, 512, 1, 64, 0.2), (1, 33, 3, 32, 3.0)]):
        Q, K, V = qkv(20 + seed, batch, seq, heads, d, sd)
        ctx64 = A.attention(Q, K, V, batch, seq, heads, d)
        bound = A.attention_error_bound(Q, K, V, batch, seq, heads, d)
        scale = np.float32(1.0 / math.sqrt(d))
        for b in range(batch):
            r = slice(b * seq, (b + 1) * seq)
            for h in range(heads):
                c = slice(h * d, (h + 1) * d)
                s = (Q[r, c] @ K[r, c].T) * scale
                e = np.exp(s - s.max(axis=1, keepdims=True))
                ctx32 = (e @ V[r, c]) / e.sum(axis=1, keepdims=True)
                worst = max(worst, float((np.abs(ctx32 - ctx64[r, c]) / bound[r, c]).max()))
    assert worst >= 2e-3, worst


def pin_block_composes_the_products():
    g = rng(30)
    batch, seq, heads, d = 1, 8, 2, 4
    X = g.standard_normal((batch * seq, 8)).astype(np.float32)
    Ws = [g.standard_normal((8, 8)).astype(np.float32) for _ in range(4)]
    bs = [g.standard_normal(8).astype(np.float32) for _ in range(4)]
    Q, K, V, ctx, Y = A.attention_block(X, Ws[0], bs[0], Ws[1], bs[1], Ws[2], bs[2], Ws[3], bs[3],
                                        batch, seq, heads)
    assert np.allclose(Q, O.spmm_masked_dense(X, Ws[0], bs[0]), rtol=1e-15, atol=0)
    assert np.allclose(ctx, A.attention(Q, K, V, batch, seq, heads, d), rtol=1e-15, atol=0)
    assert np.allclose(Y, O.spmm_masked_dense(ctx, Ws[3], bs[3]), rtol=1e-14, atol=1e-15)


PINS = [pin_uniform_keys_give_the_mean, pin_single_token_is_v, pin_key_shift_invariance,
        pin_key_permutation_invariance, pin_matches_torch_sdpa_fp64,
        pin_matches_40_digit_reference, pin_fp32_computation_is_within_the_bound,
        pin_bound_hand_worked, pin_bound_is_not_loose, pin_block_composes_the_products]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_attention_pin(pin):
    pin()


# ---------------------------------------------------------------------- planted mistakes


def _make(variant):
    orig = A.__dict__["_orig_attention"]

    def f(Q, K, V, batch, seq, heads, head_dim, scale=None):
        if scale is None:
            scale = 1.0 / math.sqrt(head_dim)
        if variant == "no scale":
            return orig(Q, K, V, batch, seq, heads, head_dim, 1.0)
        if variant == "scale by 1/d":
            return orig(Q, K, V, batch, seq, heads, head_dim, 1.0 / head_dim)
        Q = np.asarray(Q, np.float64)
        K = np.asarray(K, np.float64)
        V = np.asarray(V, np.float64)
        ctx = np.zeros((batch * seq, heads * head_dim))
        for b in range(batch):
            r = slice(b * seq, (b + 1) * seq)
            for h in range(heads):
                c = slice(h * head_dim, (h + 1) * head_dim)
                ck = slice(((h + 1) % heads) * head_dim, ((h + 1) % heads + 1) * head_dim)
                s = scale * (Q[r, c] @ K[r, ck if variant == "keys of the next head" else c].T)
                axis = 0 if variant == "softmax over queries" else 1
                e = np.exp(s - s.max(axis=axis, keepdims=True))
                p = e / e.sum(axis=axis, keepdims=True)
                ctx[r, c] = (p.T if variant == "weights transposed" else p) @ V[r, c]
        return ctx
    return f


@pytest.mark.parametrize("variant", ["no scale", "scale by 1/d", "keys of the next head",
                                     "softmax over queries", "weights transposed"])
def test_planted_attention_mistake_is_caught(variant, monkeypatch):
    monkeypatch.setitem(A.__dict__, "_orig_attention", A.attention)
    monkeypatch.setattr(A, "attention", _make(variant))
    caught = []
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches: {variant}"


def _bound_mutant(variant):
    """attention_error_bound with one plausible mistake planted."""
    orig = A.__dict__["_orig_attention_error_bound"]
    u = 2.0 ** -24

    def f(Q, K, V, batch, seq, heads, head_dim, scale=None):
        if variant == "bound 100 times too large":
            return 100.0 * orig(Q, K, V, batch, seq, heads, head_dim, scale)
        if scale is None:
            scale = 1.0 / math.sqrt(head_dim)
        Q, K, V = (np.asarray(x, dtype=np.float64) for x in (Q, K, V))
        out = np.zeros((batch * seq, heads * head_dim))
        for b in range(batch):
            r = slice(b * seq, (b + 1) * seq)
            for h in range(heads):
                c = slice(h * head_dim, (h + 1) * head_dim)
                s = scale * (Q[r, c] @ K[r, c].T)
                sigma = scale * (np.abs(Q[r, c]) @ np.abs(K[r, c]).T)
                m = s.max(axis=1, keepdims=True)
                p = np.exp(s - m)
                p = p / p.sum(axis=1, keepdims=True)
                width = 1 if variant == "score error without the head-width factor" else head_dim
                eps = (width + 2) * u * sigma + u * np.abs(s - m) + 4 * u
                Aabs = p @ np.abs(V[r, c])
                seq_term = 0.0 if variant == "sequence-sum term dropped" else 2 * (seq + 2) * u * Aabs
                out[r, c] = 2 * eps.max(axis=1, keepdims=True) * Aabs + seq_term + u * np.abs(p @ V[r, c])
        return out
    return f


@pytest.mark.parametrize("variant", ["bound 100 times too large", "sequence-sum term dropped",
                                     "score error without the head-width factor"])
def test_planted_bound_mistake_is_caught(variant, monkeypatch):
    monkeypatch.setitem(A.__dict__, "_orig_attention_error_bound", A.attention_error_bound)
    monkeypatch.setattr(A, "attention_error_bound", _bound_mutant(variant))
    caught = []
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches: {variant}"
