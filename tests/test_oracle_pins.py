"""Pins for the CPU oracle: closed forms, brute force, exact arithmetic and library routines.

Each check ties the oracle to something other than itself: hand-worked examples, exact rational
arithmetic, brute-force enumeration of subsets, SciPy's BSR type and torch's bf16 conversion.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import bsr_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


# ------------------------------------------------------------------------- hand-worked examples


def _golden():
    with open(os.path.join(GOLDEN, "hand_examples.json")) as f:
        return json.load(f)["examples"]


@pytest.mark.parametrize("ex", _golden(), ids=lambda e: e["name"])
def test_hand_examples(ex):
    W = np.array(ex["W"], dtype=np.float32)
    R, C = ex["R"], ex["C"]
    norm, per_row = ex.get("norm", "l2"), ex.get("per_row", False)
    assert O.block_keys(W, R, C, norm).tolist() == ex["keys"]
    assert O.prune_count(W.shape[0], W.shape[1], R, C, ex["density"], per_row=per_row) == ex["k"]
    indptr, indices, data = O.prune(W, R, C, density=ex["density"], norm=norm, per_row=per_row)
    assert indptr.tolist() == ex["indptr"]
    assert indices.tolist() == ex["indices"]
    assert data.tolist() == ex["data"]
    X = np.array(ex["X"], dtype=np.float32)
    b = np.array(ex["bias"], dtype=np.float32)
    Y = O.spmm_loop(X, indptr, indices, data, W.shape[0], b)
    assert Y.tolist() == ex["Y"]
    if "S" in ex:
        # The acceptance bound of every floating-point product check, worked by hand.
        S = O.tolerance_scale(X, O.to_dense(indptr, indices, data, W.shape[0], W.shape[1]))
        assert S.tolist() == ex["S"]
        bound = O.spmm_tolerance(S)
        assert np.allclose(bound, np.array(ex["bound"]), rtol=1e-12, atol=0)


# ------------------------------------------------------------------------------ pruning count


@pytest.mark.parametrize("N,K,R,C,d,k", [
    (768, 768, 32, 1, 0.2, 3686),      # 0.2 * 18432 = 3686.4
    (768, 768, 32, 1, 0.1, 1843),      # 1843.2
    (768, 768, 1, 1, 0.1, 58982),      # 58982.4
    (768, 768, 8, 1, 0.1, 7373),       # 7372.8
    (768, 768, 16, 1, 0.1, 3686),
    (768, 768, 1, 32, 0.1, 1843),
    (768, 768, 4, 4, 0.1, 3686),
    (768, 768, 8, 8, 0.1, 922),        # 921.6
    (768, 768, 16, 16, 0.1, 230),      # 230.4
    (768, 768, 32, 32, 0.1, 58),       # 57.6
    (2304, 768, 32, 1, 0.05, 2765),    # 2764.8
    (2304, 768, 32, 1, 0.4, 22118),    # 22118.4
    (2304, 768, 16, 16, 0.05, 346),    # 345.6
    (2304, 768, 16, 16, 0.4, 2765),    # 2764.8
    (1024, 1024, 32, 1, 0.1, 3277),    # 3276.8
    (1024, 1024, 32, 32, 0.1, 102),    # 102.4
    (64, 64, 32, 32, 0.5, 2),          # 0.5 * 4 = 2 exactly
    (64, 64, 16, 16, 0.5 / 16, 1),     # 0.5 exactly -> rounds half up
    (64, 64, 32, 32, 0.0, 0),
    (64, 64, 32, 32, 1.0, 4),
])
def test_prune_count_closed_form(N, K, R, C, d, k):
    assert O.prune_count(N, K, R, C, d) == k


@pytest.mark.parametrize("args", [(768, 768, 7, 1, 0.1), (768, 768, 32, 5, 0.1),
                                  (64, 64, 8, 8, -0.1), (64, 64, 8, 8, 1.5),
                                  (64, 64, 8, 8, float("nan")), (64, 64, 0, 8, 0.1)])
def test_prune_count_rejects(args):
    with pytest.raises(ValueError):
        O.prune_count(*args)


# -------------------------------------------------------------------------------------- keys


def test_keys_unit_blocks_are_exact_squares():
    W = rng(1).standard_normal((16, 24)).astype(np.float32)
    key = O.block_keys(W, 1, 1)
    assert np.array_equal(key, (W.astype(np.float64) ** 2).ravel())


def test_keys_integer_entries_are_exact():
    W = rng(2).integers(-1000, 1000, size=(32, 64)).astype(np.float32)
    for R, C in [(32, 1), (1, 32), (4, 4), (8, 8), (16, 16), (32, 32)]:
        key = O.block_keys(W, R, C)
        Wi = W.astype(np.int64)
        Nb, Kb = 32 // R, 64 // C
        exact = [int((Wi[i * R:(i + 1) * R, j * C:(j + 1) * C] ** 2).sum())
                 for i in range(Nb) for j in range(Kb)]
        assert key.tolist() == [float(e) for e in exact]


def test_keys_constant_half():
    W = np.full((64, 64), 0.5, dtype=np.float32)
    for R, C in [(32, 1), (4, 4), (32, 32)]:
        assert np.all(O.block_keys(W, R, C) == R * C / 4)


def test_keys_within_fsum_bound():
    """Sequential fp64 sum is within gamma_n of the correctly rounded sum (fsum)."""
    W = rng(3).standard_normal((64, 64)).astype(np.float32)
    for R, C in [(32, 1), (32, 32), (16, 16)]:
        key = O.block_keys(W, R, C)
        Kb = 64 // C
        n = R * C
        gamma = n * 2.0 ** -53 / (1 - n * 2.0 ** -53)
        for b, kv in enumerate(key):
            i, j = divmod(b, Kb)
            blk = W[i * R:(i + 1) * R, j * C:(j + 1) * C].astype(np.float64).ravel()
            ref = math.fsum(float(x) * float(x) for x in blk)
            assert abs(kv - ref) <= gamma * ref


def test_keys_sequential_order_matters_at_the_last_bit():
    """A block whose pairwise sum rounds differently from the sequential (r, c) sum."""
    W = np.zeros((1, 4), dtype=np.float32)
    W[0] = [1.0, 2.0 ** -27, 2.0 ** -27, 2.0 ** -27]
    # sequential: ((1 + 2^-54) + 2^-54) + 2^-54 rounds to 1 at every step
    assert O.block_keys(W, 1, 4)[0] == 1.0
    W[0] = [2.0 ** -27, 2.0 ** -27, 2.0 ** -27, 1.0]
    # sequential: 3 * 2^-54 is exact, then 1 + 3 * 2^-54 rounds up to 1 + 2^-52
    assert O.block_keys(W, 1, 4)[0] == 1.0 + 2.0 ** -52
    # 32 elements: 1 then 31 tiny squares; every sequential step rounds back to 1, whereas an
    # 8-way pairwise sum would first gather the tiny squares and end above 1.
    W32 = np.full((1, 32), 2.0 ** -27, dtype=np.float32)
    W32[0, 0] = 1.0
    assert O.block_keys(W32, 1, 32)[0] == 1.0
    # r outer, c inner: rows are finished one at a time.  Block [[e, e, e], [1, 0, 0]] gives
    # 3 e^2 + 1 -> 1 + 2^-52 in that order, but 1 (every step rounds back) in column order.
    B = np.zeros((2, 3), dtype=np.float32)
    B[0, :] = 2.0 ** -27
    B[1, 0] = 1.0
    assert O.block_keys(B, 2, 3)[0] == 1.0 + 2.0 ** -52


def test_keys_nonfinite():
    W = np.ones((2, 4), dtype=np.float32)
    W[0, 1] = np.inf
    W[1, 2] = np.nan
    key = O.block_keys(W, 1, 2)
    assert key[0] == np.inf and key[1] == 2.0 and key[2] == 2.0 and np.isnan(key[3])


# --------------------------------------------------------------------------------- selection


def _brute_force_mask(key, k):
    """Block b is kept iff fewer than k blocks beat it; NaN beats +inf; ties: lower id wins."""
    def beats(a, b):
        ka, kb = key[a], key[b]
        ra = math.inf if math.isnan(ka) else ka
        rb = math.inf if math.isnan(kb) else kb
        na, nbn = math.isnan(ka), math.isnan(kb)
        if na != nbn:
            return na
        if ra != rb:
            return ra > rb
        return a < b
    nb = len(key)
    return np.array([sum(beats(o, b) for o in range(nb) if o != b) < k for b in range(nb)])


@pytest.mark.parametrize("seed", range(6))
def test_select_matches_brute_force(seed):
    g = rng(100 + seed)
    nb = int(g.integers(1, 60))
    # few distinct values -> many ties; a couple of infinities and NaNs on some seeds
    key = g.integers(0, 6, size=nb).astype(np.float64) * 0.25
    if seed % 2:
        key[g.integers(0, nb)] = np.inf
        key[g.integers(0, nb)] = np.nan
    for k in sorted({0, 1, nb // 3, nb // 2, nb - 1, nb} - {-1}):
        m = O.select_topk(key, k)
        assert m.sum() == k
        assert np.array_equal(m, _brute_force_mask(key, k))


def test_select_exchange_invariant():
    g = rng(7)
    key = g.standard_normal(5000) ** 2
    key[::7] = key[3]          # many exact ties
    k = 1234
    m = O.select_topk(key, k)
    kept, dropped = np.nonzero(m)[0], np.nonzero(~m)[0]
    worst_kept = min(kept, key=lambda b: (key[b], -b))
    best_dropped = max(dropped, key=lambda b: (key[b], -b))
    assert (key[worst_kept], -worst_kept) > (key[best_dropped], -best_dropped)


def test_select_ties_all_zero_keeps_lowest_ids():
    for k in [0, 1, 5, 16]:
        m = O.select_topk(np.zeros(16), k)
        assert np.nonzero(m)[0].tolist() == list(range(k))


def test_select_duplicate_and_sign_flipped_blocks():
    g = rng(8)
    W = g.standard_normal((32, 32)).astype(np.float32)
    # block (0,1) := -block(0,0), block (1,1) := block(0,0): three equal keys
    W[0:16, 16:32] = -W[0:16, 0:16]
    W[16:32, 16:32] = W[0:16, 0:16]
    W[16:32, 0:16] *= 0.01
    key = O.block_keys(W, 16, 16)
    assert key[0] == key[1] == key[3]
    assert O.select_topk(key, 1).nonzero()[0].tolist() == [0]
    assert O.select_topk(key, 2).nonzero()[0].tolist() == [0, 1]
    assert O.select_topk(key, 3).nonzero()[0].tolist() == [0, 1, 3]


@pytest.mark.parametrize("R,C,k", [(32, 32, 1), (32, 32, 2), (32, 32, 3), (16, 16, 3),
                                   (16, 16, 5), (32, 16, 4)])
def test_select_is_the_projection_for_eq2(R, C, k):
    """Kept set minimises ||W - W*M||_F^2 over all k-subsets (exact rational arithmetic)."""
    W = rng(9 + R + C + k).standard_normal((64, 64)).astype(np.float32)
    Nb, Kb = 64 // R, 64 // C
    energy = []
    for i in range(Nb):
        for j in range(Kb):
            blk = W[i * R:(i + 1) * R, j * C:(j + 1) * C].ravel()
            energy.append(sum(Fraction(float(x)) ** 2 for x in blk))
    total = sum(energy)
    best = min(total - sum(energy[b] for b in sub)
               for sub in itertools.combinations(range(Nb * Kb), k))
    indptr, indices, data = O.prune(W, R, C, k=k)
    kept_ids = [i * Kb + int(indices[p]) for i in range(Nb)
                for p in range(indptr[i], indptr[i + 1])]
    assert total - sum(energy[b] for b in kept_ids) == best


def test_select_nan_ranks_above_inf():
    key = np.array([1.0, np.inf, np.nan, 2.0])
    assert O.select_topk(key, 1).nonzero()[0].tolist() == [2]
    assert O.select_topk(key, 2).nonzero()[0].tolist() == [1, 2]


# ---------------------------------------------------------------- l1 keys (p = 1 of Eq. 1, 2)


def test_l1_keys_unit_blocks_are_exact_magnitudes():
    W = rng(11).standard_normal((16, 24)).astype(np.float32)
    assert np.array_equal(O.block_keys(W, 1, 1, "l1"), np.abs(W.astype(np.float64)).ravel())


def test_l1_keys_integer_entries_are_exact():
    W = rng(12).integers(-1000, 1000, size=(32, 64)).astype(np.float32)
    Wi = np.abs(W.astype(np.int64))
    for R, C in [(32, 1), (1, 32), (4, 4), (8, 8), (32, 32)]:
        Nb, Kb = 32 // R, 64 // C
        exact = [int(Wi[i * R:(i + 1) * R, j * C:(j + 1) * C].sum())
                 for i in range(Nb) for j in range(Kb)]
        assert O.block_keys(W, R, C, "l1").tolist() == [float(e) for e in exact]


def test_l1_keys_sign_blind_constant():
    W = np.full((64, 64), -0.5, dtype=np.float32)
    W[::2] = 0.5
    for R, C in [(32, 1), (4, 4), (32, 32)]:
        assert np.all(O.block_keys(W, R, C, "l1") == R * C / 2)


def test_l1_keys_within_fsum_bound():
    W = rng(13).standard_normal((64, 64)).astype(np.float32)
    for R, C in [(32, 1), (32, 32), (16, 16)]:
        key = O.block_keys(W, R, C, "l1")
        Kb, n = 64 // C, R * C
        gamma = n * 2.0 ** -53 / (1 - n * 2.0 ** -53)
        for b, kv in enumerate(key):
            i, j = divmod(b, Kb)
            ref = math.fsum(abs(float(x)) for x in W[i * R:(i + 1) * R, j * C:(j + 1) * C].ravel())
            assert abs(kv - ref) <= gamma * ref


def test_l1_keys_sequential_order_matters_at_the_last_bit():
    # 1 + 2^-53 is a tie that rounds to even (1); a pairwise sum would first add the two tiny
    # terms exactly (2^-52) and end at 1 + 2^-52.
    W = np.array([[1.0, 2.0 ** -53, -(2.0 ** -53)]], dtype=np.float32)
    assert O.block_keys(W, 1, 3, "l1")[0] == 1.0
    W = np.array([[2.0 ** -53, -(2.0 ** -53), 1.0]], dtype=np.float32)
    assert O.block_keys(W, 1, 3, "l1")[0] == 1.0 + 2.0 ** -52


def test_l1_keys_nonfinite():
    W = np.ones((2, 4), dtype=np.float32)
    W[0, 1] = -np.inf
    W[1, 2] = np.nan
    key = O.block_keys(W, 1, 2, "l1")
    assert key[0] == np.inf and key[1] == 2.0 and key[2] == 2.0 and np.isnan(key[3])


@pytest.mark.parametrize("R,C,k", [(16, 16, 3), (32, 16, 4), (8, 32, 5)])
def test_l1_selection_keeps_the_largest_l1_mass(R, C, k):
    """The kept set has the largest total l1 norm of all k-subsets (exact rationals)."""
    W = rng(14 + R + C + k).standard_normal((64, 64)).astype(np.float32)
    Nb, Kb = 64 // R, 64 // C
    mass = [sum(abs(Fraction(float(x))) for x in W[i * R:(i + 1) * R, j * C:(j + 1) * C].ravel())
            for i in range(Nb) for j in range(Kb)]
    best = max(sum(mass[b] for b in sub) for sub in itertools.combinations(range(Nb * Kb), k))
    indptr, indices, _ = O.prune(W, R, C, k=k, norm="l1")
    kept = [i * Kb + int(indices[p]) for i in range(Nb) for p in range(indptr[i], indptr[i + 1])]
    assert len(kept) == k and sum(mass[b] for b in kept) == best


def test_block_keys_rejects_other_norms():
    with pytest.raises(ValueError):
        O.block_keys(np.ones((4, 4), np.float32), 2, 2, "l0")


# ------------------------------------------------------------------ per-row balanced selection


@pytest.mark.parametrize("N,K,R,C,d,k", [
    (768, 768, 32, 1, 0.1, 24 * 77),     # k_row = floor(76.8 + 0.5) = 77
    (768, 768, 1, 1, 0.2, 768 * 154),    # floor(153.6 + 0.5) = 154
    (2304, 768, 16, 16, 0.05, 144 * 2),  # floor(2.4 + 0.5) = 2
    (64, 64, 8, 8, 0.0, 0), (64, 64, 8, 8, 1.0, 64),
    (96, 40, 3, 5, 0.4, 32 * 3),         # floor(3.2 + 0.5) = 3
])
def test_per_row_count_closed_form(N, K, R, C, d, k):
    assert O.prune_count(N, K, R, C, d, per_row=True) == k


@pytest.mark.parametrize("seed", range(5))
def test_per_row_matches_brute_force(seed):
    """In every row, a block is kept iff fewer than k_row blocks of that row beat it."""
    g = rng(200 + seed)
    Nb, Kb = int(g.integers(1, 7)), int(g.integers(1, 12))
    key = g.integers(0, 5, size=Nb * Kb).astype(np.float64) * 0.5
    if seed % 2:
        key[g.integers(0, Nb * Kb)] = np.inf
        key[g.integers(0, Nb * Kb)] = np.nan
    for k_row in sorted({0, 1, Kb // 2, Kb}):
        m = O.select_topk_rows(key, Nb, Kb, k_row).reshape(Nb, Kb)
        for i in range(Nb):
            row = key[i * Kb:(i + 1) * Kb]
            assert np.array_equal(m[i], _brute_force_mask(row, k_row))


@pytest.mark.parametrize("norm", ["l2", "l1"])
def test_per_row_keeps_equal_counts_and_is_the_row_projection(norm):
    """Every row keeps k_row blocks; for l2 the kept set minimises ||W - W*M||_F^2 over all
    masks with k_row blocks in each row (exact rationals, all combinations)."""
    W = rng(15).standard_normal((48, 64)).astype(np.float32)
    R, C, k_row = 16, 16, 2
    Nb, Kb = 3, 4
    indptr, indices, data = O.prune(W, R, C, k=Nb * k_row, norm=norm, per_row=True)
    assert np.diff(indptr).tolist() == [k_row] * Nb
    if norm == "l2":
        energy = [[sum(Fraction(float(x)) ** 2 for x in W[i * R:(i + 1) * R, j * C:(j + 1) * C].ravel())
                   for j in range(Kb)] for i in range(Nb)]
        best = sum(min(sum(energy[i]) - sum(energy[i][j] for j in sub)
                       for sub in itertools.combinations(range(Kb), k_row)) for i in range(Nb))
        got = sum(sum(energy[i]) - sum(energy[i][int(j)] for j in indices[indptr[i]:indptr[i + 1]])
                  for i in range(Nb))
        assert got == best


def test_per_row_ties_keep_lowest_columns():
    key = np.zeros(12)
    m = O.select_topk_rows(key, 3, 4, 2).reshape(3, 4)
    assert all(np.nonzero(m[i])[0].tolist() == [0, 1] for i in range(3))


def test_per_row_rejects_uneven_k():
    W = np.ones((64, 64), np.float32)
    with pytest.raises(ValueError):
        O.prune(W, 32, 32, k=3, per_row=True)


# ----------------------------------------------------------------------------------- reblock


@pytest.mark.parametrize("R,C,R2,C2", [(64, 64, 32, 32), (1, 128, 1, 32), (128, 1, 32, 1),
                                       (32, 32, 16, 16), (8, 8, 8, 1), (4, 4, 1, 1),
                                       (64, 64, 64, 64)])
def test_reblock_is_the_same_matrix(R, C, R2, C2):
    """The refined matrix expands to the same dense matrix bit for bit, its pattern is the
    original one refined, and SciPy's conversion to the smaller block size agrees."""
    import scipy.sparse as sp
    g = rng(40 + R + C + R2)
    N, K = 4 * R, 3 * C if C > 1 else 96
    W = g.standard_normal((N, K)).astype(np.float32)
    W[0, 0] = -0.0
    ip, ix, dt = O.prune(W, R, C, density=0.4)
    ip2, ix2, dt2 = O.reblock(ip, ix, dt, R2, C2)
    D = O.to_dense(ip, ix, dt, N, K)
    assert np.array_equal(O.to_dense(ip2, ix2, dt2, N, K).view(np.uint32), D.view(np.uint32))
    a, b = R // R2, C // C2
    assert ip2[-1] == len(ix) * a * b and np.all(np.diff(ip2) >= 0)
    for i2 in range(len(ip2) - 1):
        row = ix2[ip2[i2]:ip2[i2 + 1]]
        assert np.all(np.diff(row) > 0)
        i = i2 // a
        assert sorted(set(row // b)) == sorted(ix[ip[i]:ip[i + 1]].tolist())
    ref = sp.bsr_matrix((dt, ix, ip), shape=(N, K)).tobsr(blocksize=(R2, C2))
    ref.sort_indices()
    got = sp.bsr_matrix((dt2, ix2, ip2), shape=(N, K))
    assert np.array_equal(got.toarray(), ref.toarray())


def test_reblock_hand_case():
    """A 2x4 block [[1,2,3,4],[5,6,7,8]] at block-column 1 of a 2x8 matrix, cut into 1x2 pieces:
    rows 0 and 1 each hold two pieces, at block-columns 2 and 3."""
    ip, ix, dt = (np.array([0, 1]), np.array([1]),
                  np.array([[[1, 2, 3, 4], [5, 6, 7, 8]]], dtype=np.float32))
    ip2, ix2, dt2 = O.reblock(ip, ix, dt, 1, 2)
    assert ip2.tolist() == [0, 2, 4]
    assert ix2.tolist() == [2, 3, 2, 3]
    assert dt2.tolist() == [[[1, 2]], [[3, 4]], [[5, 6]], [[7, 8]]]


def test_reblock_rejects_non_divisors():
    with pytest.raises(ValueError):
        O.reblock(np.array([0, 0]), np.zeros(0, np.int32), np.zeros((0, 4, 4), np.float32), 3, 4)


# --------------------------------------------------------------------- BSR build and to_dense


@pytest.mark.parametrize("R,C,d", [(32, 1, 0.2), (1, 32, 0.1), (4, 4, 0.3), (16, 16, 0.5),
                                   (1, 1, 0.1), (64, 8, 0.5), (8, 8, 1.0), (8, 8, 0.0)])
def test_bsr_matches_scipy_and_round_trips(R, C, d):
    import scipy.sparse as sp
    W = rng(11).standard_normal((128, 64)).astype(np.float32)
    indptr, indices, data = O.prune(W, R, C, density=d)
    k = O.prune_count(128, 64, R, C, d)
    assert indptr[0] == 0 and indptr[-1] == k == len(indices) == data.shape[0]
    assert np.all(np.diff(indptr) >= 0)
    for i in range(128 // R):
        row = indices[indptr[i]:indptr[i + 1]]
        assert np.all(np.diff(row) > 0)
    D = O.to_dense(indptr, indices, data, 128, 64)
    mask = O.select_topk(O.block_keys(W, R, C), k).reshape(128 // R, 64 // C)
    M = np.repeat(np.repeat(mask, R, axis=0), C, axis=1)
    assert np.array_equal(D.view(np.uint32), np.where(M, W, np.float32(0)).view(np.uint32))
    if d == 1.0:
        assert np.array_equal(D, W)
    ref = sp.bsr_matrix((data, indices, indptr), shape=(128, 64)).toarray()
    assert np.array_equal(ref, D)
    if k:
        # SciPy's own dense -> BSR conversion of the masked matrix finds the same structure.
        S = sp.bsr_matrix(D, blocksize=(R, C))
        S.sort_indices()
        assert np.array_equal(S.indptr, indptr) and np.array_equal(S.indices, indices)
        assert np.array_equal(S.data, data)


def test_build_bit_copies_special_values():
    W = np.ones((4, 4), dtype=np.float32)
    W[0, 0] = -0.0
    W[1, 1] = np.float32(1e-45)           # subnormal
    W[2, 2] = np.inf
    indptr, indices, data = O.prune(W, 2, 2, density=1.0)
    D = O.to_dense(indptr, indices, data, 4, 4)
    assert np.array_equal(D.view(np.uint32), W.view(np.uint32))


# ---------------------------------------------------------------------------------- products


def _exact_product(X, W_masked, b):
    T, K = X.shape
    N = W_masked.shape[0]
    out = []
    for t in range(T):
        row = []
        for n in range(N):
            s = Fraction(float(b[n])) if b is not None else Fraction(0)
            for kk in range(K):
                w = W_masked[n, kk]
                if w != 0:
                    s += Fraction(float(X[t, kk])) * Fraction(float(w))
            row.append(s)
        out.append(row)
    return out


@pytest.mark.parametrize("R,C", [(32, 1), (16, 16), (1, 32), (4, 4)])
def test_spmm_against_exact_rationals(R, C):
    g = rng(20 + R)
    W = g.standard_normal((64, 64)).astype(np.float32)
    X = g.standard_normal((4, 64)).astype(np.float32)
    b = g.standard_normal(64).astype(np.float32)
    indptr, indices, data = O.prune(W, R, C, density=0.3)
    Wm = O.to_dense(indptr, indices, data, 64, 64)
    exact = _exact_product(X, Wm, b)
    Y = O.spmm_loop(X, indptr, indices, data, 64, b)
    S = O.tolerance_scale(X, Wm) + np.abs(b)[None, :]
    gamma = 65 * 2.0 ** -53 / (1 - 65 * 2.0 ** -53)
    for t in range(4):
        for n in range(64):
            assert abs(Fraction(float(Y[t, n])) - exact[t][n]) <= Fraction(gamma * S[t, n])


@pytest.mark.parametrize("R,C,d", [(32, 1, 0.1), (1, 1, 0.2), (8, 8, 0.5), (32, 32, 0.25)])
def test_spmm_routes_agree_and_match_scipy(R, C, d):
    import scipy.sparse as sp
    g = rng(30)
    W = (g.standard_normal((256, 128)) * 0.02).astype(np.float32)
    X = g.standard_normal((48, 128)).astype(np.float32)
    b = (g.standard_normal(256) * 0.02).astype(np.float32)
    indptr, indices, data = O.prune(W, R, C, density=d)
    Wm = O.to_dense(indptr, indices, data, 256, 128)
    Y1 = O.spmm_loop(X, indptr, indices, data, 256, b)
    Y2 = O.spmm_masked_dense(X, Wm, b)
    S = O.tolerance_scale(X, Wm)
    assert np.all(np.abs(Y1 - Y2) <= 1e-12 * S + 1e-15)
    A = sp.bsr_matrix((data.astype(np.float64), indices, indptr), shape=(256, 128))
    Y3 = (A @ X.astype(np.float64).T).T + b.astype(np.float64)[None, :]
    assert np.all(np.abs(Y1 - Y3) <= 1e-12 * S + 1e-15)


def test_spmm_density_one_is_dense_gemm():
    g = rng(31)
    W = g.standard_normal((64, 96)).astype(np.float32)
    X = g.standard_normal((5, 96)).astype(np.float32)
    b = g.standard_normal(64).astype(np.float32)
    indptr, indices, data = O.prune(W, 16, 8, density=1.0)
    Y = O.spmm_loop(X, indptr, indices, data, 64, b)
    ref = X.astype(np.float64) @ W.astype(np.float64).T + b
    S = np.abs(X.astype(np.float64)) @ np.abs(W.astype(np.float64)).T
    assert np.all(np.abs(Y - ref) <= 1e-13 * S)


def test_spmm_special_cases():
    g = rng(32)
    W = g.standard_normal((64, 64)).astype(np.float32)
    b = g.standard_normal(64).astype(np.float32)
    # k = 0: Y == bias exactly (and zero without bias)
    indptr, indices, data = O.prune(W, 32, 1, k=0)
    X = g.standard_normal((3, 64)).astype(np.float32)
    assert np.array_equal(O.spmm_loop(X, indptr, indices, data, 64, b),
                          np.broadcast_to(b.astype(np.float64), (3, 64)))
    assert not O.spmm_loop(X, indptr, indices, data, 64).any()
    # one-hot token rows pick out a column of the masked weight
    indptr, indices, data = O.prune(W, 32, 1, density=0.25)
    Wm = O.to_dense(indptr, indices, data, 64, 64)
    E = np.eye(64, dtype=np.float32)[[0, 5, 63]]
    Y = O.spmm_loop(E, indptr, indices, data, 64, b)
    for r, col in enumerate([0, 5, 63]):
        assert np.array_equal(Y[r], Wm[:, col].astype(np.float64) + b)
    # identity weight stored as its diagonal 16x16 blocks: Y == X + b
    I = np.eye(64, dtype=np.float32)
    indptr, indices, data = O.prune(I, 16, 16, k=4)
    assert indices.tolist() == [0, 1, 2, 3]
    assert np.array_equal(O.spmm_loop(X, indptr, indices, data, 64, b),
                          X.astype(np.float64) + b)


def test_spmm_integer_inputs_exact():
    g = rng(33)
    W = g.integers(-8, 9, size=(96, 64)).astype(np.float32)
    X = g.integers(-8, 9, size=(7, 64)).astype(np.float32)
    b = g.integers(-8, 9, size=96).astype(np.float32)
    indptr, indices, data = O.prune(W, 32, 1, density=0.5)
    Wm = O.to_dense(indptr, indices, data, 96, 64).astype(np.int64)
    exact = X.astype(np.int64) @ Wm.T + b.astype(np.int64)
    assert np.array_equal(O.spmm_loop(X, indptr, indices, data, 96, b), exact.astype(np.float64))


# ------------------------------------------------------------------------------------ bf16


def _torch_bf16_bits(x):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_bf16_hand_cases():
    cases = [
        (1.0, 0x3F80),
        (1.0 + 2.0 ** -8, 0x3F80),              # tie between 0x3F80 (even) and 0x3F81
        (1.0 + 3 * 2.0 ** -8, 0x3F82),          # tie between 0x3F81 and 0x3F82 (even)
        (1.0 + 2.0 ** -8 + 2.0 ** -20, 0x3F81),  # just above the tie
        (-2.0, 0xC000),
        (0.0, 0x0000),
        (-0.0, 0x8000),
        (float(np.finfo(np.float32).max), 0x7F80),  # past halfway to 2^128 -> inf
        (float("inf"), 0x7F80),
        (float("-inf"), 0xFF80),
    ]
    x = np.array([c[0] for c in cases], dtype=np.float32)
    assert O.bf16_round(x).tolist() == [c[1] for c in cases]
    nan = O.bf16_round(np.array([np.nan], dtype=np.float32))
    assert np.isnan(O.bf16_to_f32(nan))[0]


def test_bf16_matches_torch_on_every_upper_half():
    hi = np.arange(1 << 16, dtype=np.uint32) << np.uint32(16)
    for low in [0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x4321, 0xC0DE]:
        u = hi | np.uint32(low)
        x = u.view(np.float32)
        ours = O.bf16_round(x)
        ref = _torch_bf16_bits(x)
        finite = ~np.isnan(x)
        assert np.array_equal(ours[finite], ref[finite])
        assert np.all(np.isnan(O.bf16_to_f32(ours[~finite])))


def test_bf16_matches_torch_random():
    u = rng(40).integers(0, 1 << 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    x = u.view(np.float32)
    finite = ~np.isnan(x)
    assert np.array_equal(O.bf16_round(x)[finite], _torch_bf16_bits(x)[finite])


# --------------------------------------------------------------------------- the C oracle twin


def test_c_oracle_keys_equal_numpy_keys():
    from oracle import cpu_oracle
    W = (rng(50).standard_normal((256, 192)) * 0.02).astype(np.float32)
    for R, C in [(32, 1), (1, 32), (1, 1), (16, 16), (32, 32), (4, 4)]:
        assert np.array_equal(cpu_oracle.block_keys(W, R, C), O.block_keys(W, R, C))


@pytest.mark.parametrize("R,C", [(32, 1), (1, 1), (16, 16), (1, 32), (8, 8)])
def test_c_oracle_spmm_matches_numpy(R, C):
    from oracle import cpu_oracle
    g = rng(51)
    W = (g.standard_normal((256, 192)) * 0.02).astype(np.float32)
    X = g.standard_normal((40, 192)).astype(np.float32)
    b = (g.standard_normal(256) * 0.02).astype(np.float32)
    indptr, indices, data = O.prune(W, R, C, density=0.2)
    Yc = cpu_oracle.spmm(X, indptr, indices, data, 256, b)
    Yn = O.spmm_loop(X, indptr, indices, data, 256, b)
    S = O.tolerance_scale(X, O.to_dense(indptr, indices, data, 256, 192))
    assert np.all(np.abs(Yc - Yn) <= 1e-12 * S + 1e-15)
    W2 = g.integers(-8, 9, size=(256, 192)).astype(np.float32)
    X2 = g.integers(-8, 9, size=(9, 192)).astype(np.float32)
    ip, ix, dt = O.prune(W2, R, C, density=0.3)
    assert np.array_equal(cpu_oracle.spmm(X2, ip, ix, dt, 256), O.spmm_loop(X2, ip, ix, dt, 256))
