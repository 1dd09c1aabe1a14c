"""The oracle's pins have teeth: each plausible mistake planted in the oracle fails some pin.

Mistakes are planted only in the CPU oracle (monkeypatched for one test), never in GPU code.
"""
import math

import numpy as np
import pytest

from oracle import bsr_oracle as O
import tests.test_oracle_pins as P


def _ties_to_higher_id(key, k):
    key = np.asarray(key, dtype=np.float64)
    bits = O._rank_bits(key)
    ids = np.arange(key.size)
    order = np.lexsort((-ids, ~bits))
    m = np.zeros(key.size, dtype=bool)
    m[order[:k]] = True
    return m


def _nan_ranks_lowest(key, k):
    key = np.nan_to_num(np.asarray(key, dtype=np.float64), nan=-1.0)
    ids = np.arange(key.size)
    order = np.lexsort((ids, -key))
    m = np.zeros(key.size, dtype=bool)
    m[order[:k]] = True
    return m


def _l1_keys(W, R, C, norm="l2"):
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    return np.abs(W.astype(np.float64)).reshape(N // R, R, K // C, C).sum(axis=(1, 3)).ravel()


def _pairwise_keys(W, R, C, norm="l2"):
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    x = W.astype(np.float64).reshape(N // R, R, K // C, C)
    t = x * x if norm == "l2" else np.abs(x)
    return np.sum(t, axis=(1, 3)).ravel()


def _column_major_block_order(W, R, C, norm="l2"):
    key = O.__dict__["_orig_block_keys"](W, R, C, norm)
    N, K = np.asarray(W).shape
    return key.reshape(N // R, K // C).T.ravel()


def _l1_as_squares(W, R, C, norm="l2"):
    return O.__dict__["_orig_block_keys"](W, R, C, "l2")


def _l1_signed_sum(W, R, C, norm="l2"):
    if norm == "l2":
        return O.__dict__["_orig_block_keys"](W, R, C, "l2")
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    x = W.astype(np.float64).reshape(N // R, R, K // C, C)
    key = np.zeros((N // R, K // C))
    for r in range(R):
        for c in range(C):
            key = key + x[:, r, :, c]
    return key.ravel()


def _reblock_pieces_column_major(indptr, indices, data, R2, C2):
    """Pieces of each stored block listed column-major (s outer) inside a fine row."""
    ip2, ix2, dt2 = O.__dict__["_orig_reblock"](indptr, indices, data, R2, C2)
    C = np.asarray(data).shape[2]
    b = C // C2
    if b > 1:
        for i2 in range(len(ip2) - 1):
            a0, a1 = ip2[i2], ip2[i2 + 1]
            n = (a1 - a0) // b
            order = np.arange(a1 - a0).reshape(n, b).T.ravel()
            ix2[a0:a1] = ix2[a0:a1][order]
            dt2[a0:a1] = dt2[a0:a1][order]
    return ip2, ix2, dt2


def _reblock_rows_swapped(indptr, indices, data, R2, C2):
    """Sub-rows of a block taken bottom-up."""
    d = np.asarray(data)[:, ::-1, :].copy()
    return O.__dict__["_orig_reblock"](indptr, indices, d, R2, C2)


def _round_half_even(N, K, R, C, d, per_row=False):
    Nb, Kb = O.check_shape(N, K, R, C)
    if not (0.0 <= d <= 1.0):
        raise ValueError
    return Nb * round(d * Kb) if per_row else round(d * Nb * Kb)


def _truncating_count(N, K, R, C, d, per_row=False):
    Nb, Kb = O.check_shape(N, K, R, C)
    if not (0.0 <= d <= 1.0):
        raise ValueError
    return Nb * int(d * Kb) if per_row else int(d * Nb * Kb)


def _per_row_count_from_global(N, K, R, C, d, per_row=False):
    return O.__dict__["_orig_prune_count"](N, K, R, C, d)


def _rows_ties_to_higher_column(key, Nb, Kb, k_row):
    key = np.asarray(key, dtype=np.float64).reshape(Nb, Kb)
    m = np.zeros((Nb, Kb), dtype=bool)
    for i in range(Nb):
        order = np.lexsort((-np.arange(Kb), ~O._rank_bits(key[i])))
        m[i, order[:k_row]] = True
    return m.ravel()


def _rows_as_global_topk(key, Nb, Kb, k_row):
    return O.select_topk(key, Nb * k_row)


def _spmm_untransposed(X, indptr, indices, data, N, bias=None):
    X64 = np.asarray(X, dtype=np.float64)
    d64 = np.asarray(data, dtype=np.float64)
    R, C = d64.shape[1:]
    Y = np.zeros((X64.shape[0], N))
    if bias is not None:
        Y += np.asarray(bias, np.float64)
    for i in range(N // R):
        for p in range(indptr[i], indptr[i + 1]):
            j = indices[p]
            blk = d64[p] if R == C else d64[p].reshape(C, R)
            Y[:, i * R:(i + 1) * R] += X64[:, j * C:(j + 1) * C] @ blk
    return Y


def _spmm_no_bias(X, indptr, indices, data, N, bias=None):
    return O.__dict__["_orig_spmm_loop"](X, indptr, indices, data, N, None)


def _spmm_off_by_one_row(X, indptr, indices, data, N, bias=None):
    X64 = np.asarray(X, dtype=np.float64)
    d64 = np.asarray(data, dtype=np.float64)
    R, C = d64.shape[1:]
    Y = np.zeros((X64.shape[0], N))
    if bias is not None:
        Y += np.asarray(bias, np.float64)
    Nb = N // R
    for i in range(Nb):
        hi = indptr[i + 1] - 1 if indptr[i + 1] > indptr[i] + 1 else indptr[i + 1]
        for p in range(indptr[i], hi):
            j = indices[p]
            Y[:, i * R:(i + 1) * R] += X64[:, j * C:(j + 1) * C] @ d64[p].T
    return Y


def _bf16_truncate(x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _bf16_ties_away(x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + np.uint64(0x8000)) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(x)
    r[nan] = ((u[nan] >> np.uint64(16)) | np.uint64(0x40)).astype(np.uint16)
    return r


def _to_dense_transposed_blocks(indptr, indices, data, N, K):
    data = np.asarray(data)
    R, C = data.shape[1:]
    out = np.zeros((N, K), dtype=data.dtype)
    for i in range(N // R):
        for p in range(indptr[i], indptr[i + 1]):
            j = indices[p]
            out[i * R:(i + 1) * R, j * C:(j + 1) * C] = data[p][::-1]
    return out


def _build_desc_indices(W, R, C, mask):
    indptr, indices, data = O.__dict__["_orig_build_bsr"](W, R, C, mask)
    for i in range(len(indptr) - 1):
        a, b = indptr[i], indptr[i + 1]
        indices[a:b] = indices[a:b][::-1]
        data[a:b] = data[a:b][::-1]
    return indptr, indices, data


def _scale_signed(X, W_masked):
    return np.asarray(X, dtype=np.float64) @ np.asarray(W_masked, np.float64).T


def _scale_abs_x_only(X, W_masked):
    return np.abs(np.asarray(X, dtype=np.float64)) @ np.asarray(W_masked, np.float64).T


def _scale_abs_w_only(X, W_masked):
    return np.asarray(X, dtype=np.float64) @ np.abs(np.asarray(W_masked, np.float64)).T


def _tolerance_rel_abs_swapped(S, rel=1e-5, abs_=1e-6):
    return abs_ * S + rel


def _tolerance_ten_times_loose(S, rel=1e-5, abs_=1e-6):
    return 10 * rel * S + abs_


MUTANTS = {
    "ties go to the higher id": ("select_topk", _ties_to_higher_id),
    "NaN keys rank lowest": ("select_topk", _nan_ranks_lowest),
    "l1 block key": ("block_keys", _l1_keys),
    "pairwise-summed key": ("block_keys", _pairwise_keys),
    "column-major block ids": ("block_keys", _column_major_block_order),
    "l1 key sums squares": ("block_keys", _l1_as_squares),
    "l1 key sums signed values": ("block_keys", _l1_signed_sum),
    "k rounds half to even": ("prune_count", _round_half_even),
    "k truncates": ("prune_count", _truncating_count),
    "per-row count is the global count": ("prune_count", _per_row_count_from_global),
    "per-row ties go to the higher column": ("select_topk_rows", _rows_ties_to_higher_column),
    "per-row selection is a global top-k": ("select_topk_rows", _rows_as_global_topk),
    "block not transposed in the product": ("spmm_loop", _spmm_untransposed),
    "bias dropped": ("spmm_loop", _spmm_no_bias),
    "last block of each row skipped": ("spmm_loop", _spmm_off_by_one_row),
    "bf16 truncates": ("bf16_round", _bf16_truncate),
    "bf16 ties away from zero": ("bf16_round", _bf16_ties_away),
    "block rows flipped in to_dense": ("to_dense", _to_dense_transposed_blocks),
    "indices descending in a row": ("build_bsr", _build_desc_indices),
    "reblock lists pieces column-major": ("reblock", _reblock_pieces_column_major),
    "reblock takes sub-rows bottom-up": ("reblock", _reblock_rows_swapped),
    "tolerance scale without abs": ("tolerance_scale", _scale_signed),
    "tolerance scale with |X| only": ("tolerance_scale", _scale_abs_x_only),
    "tolerance scale with |W| only": ("tolerance_scale", _scale_abs_w_only),
    "tolerance rel and abs swapped": ("spmm_tolerance", _tolerance_rel_abs_swapped),
    "tolerance ten times loose": ("spmm_tolerance", _tolerance_ten_times_loose),
}


def _all_pins():
    """(name, callable) for every pin of the oracle, with its parametrisations expanded."""
    calls = []
    for ex in P._golden():
        calls.append(("hand", lambda ex=ex: P.test_hand_examples(ex)))
    calls += [
        ("count", lambda: [P.test_prune_count_closed_form(768, 768, 32, 1, 0.2, 3686),
                           P.test_prune_count_closed_form(64, 64, 16, 16, 0.5 / 16, 1),
                           P.test_prune_count_closed_form(2304, 768, 32, 1, 0.4, 22118)]),
        ("keys-int", P.test_keys_integer_entries_are_exact),
        ("keys-seq", P.test_keys_sequential_order_matters_at_the_last_bit),
        ("keys-nonfinite", P.test_keys_nonfinite),
        ("l1-unit", P.test_l1_keys_unit_blocks_are_exact_magnitudes),
        ("l1-int", P.test_l1_keys_integer_entries_are_exact),
        ("l1-const", P.test_l1_keys_sign_blind_constant),
        ("l1-seq", P.test_l1_keys_sequential_order_matters_at_the_last_bit),
        ("l1-mass", lambda: P.test_l1_selection_keeps_the_largest_l1_mass(16, 16, 3)),
        ("row-count", lambda: [P.test_per_row_count_closed_form(768, 768, 32, 1, 0.1, 24 * 77),
                               P.test_per_row_count_closed_form(96, 40, 3, 5, 0.4, 96)]),
        ("row-brute", lambda: [P.test_per_row_matches_brute_force(s) for s in range(5)]),
        ("row-projection", lambda: P.test_per_row_keeps_equal_counts_and_is_the_row_projection("l2")),
        ("row-ties", P.test_per_row_ties_keep_lowest_columns),
        ("select-brute", lambda: [P.test_select_matches_brute_force(s) for s in range(6)]),
        ("select-zero", P.test_select_ties_all_zero_keeps_lowest_ids),
        ("select-dup", P.test_select_duplicate_and_sign_flipped_blocks),
        ("select-nan", P.test_select_nan_ranks_above_inf),
        ("projection", lambda: P.test_select_is_the_projection_for_eq2(16, 16, 3)),
        ("scipy", lambda: [P.test_bsr_matches_scipy_and_round_trips(R, C, d)
                           for R, C, d in [(32, 1, 0.2), (4, 4, 0.3), (16, 16, 0.5)]]),
        ("exact-product", lambda: [P.test_spmm_against_exact_rationals(R, C)
                                   for R, C in [(32, 1), (16, 16)]]),
        ("product-special", P.test_spmm_special_cases),
        ("product-int", P.test_spmm_integer_inputs_exact),
        ("bf16-hand", P.test_bf16_hand_cases),
        ("bf16-torch", P.test_bf16_matches_torch_random),
        ("reblock", lambda: [P.test_reblock_is_the_same_matrix(*a) for a in
                             [(64, 64, 32, 32), (1, 128, 1, 32), (128, 1, 32, 1)]]),
        ("reblock-hand", P.test_reblock_hand_case),
    ]
    return calls


@pytest.mark.parametrize("mutant", list(MUTANTS), ids=list(MUTANTS))
def test_planted_mistake_is_caught(mutant, monkeypatch):
    name, fn = MUTANTS[mutant]
    monkeypatch.setitem(O.__dict__, "_orig_" + name, getattr(O, name))
    monkeypatch.setattr(O, name, fn)
    caught = []
    for pin, call in _all_pins():
        try:
            call()
        except (AssertionError, ValueError, IndexError):
            caught.append(pin)
    assert caught, f"no pin catches the planted mistake: {mutant}"
