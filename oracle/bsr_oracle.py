"""Plain CPU oracle for block-magnitude pruning and block-sparse-row (BSR) products.

TEST INFRASTRUCTURE ONLY.  The test suite, the smoke check and the CPU-baseline timing leg of the
benchmark may import this module; the library's product path never does.  It shares no code,
tables or helpers with the GPU kernels, and it imports nothing from the library package.

What is computed, and which passage of the paper defines it:

* Blocks and their norm -- Sec. 2.1, Eq. 3: the structured norm of a weight matrix is a sum over
  its N blocks of a per-block norm.  The default per-block norm is the l2 group norm (the
  group-lasso definition that Sec. 2.1 keeps in its source as a commented-out draft); its key is
  the squared l2 norm, which orders blocks exactly as the norm does.  The l1 block norm (Eq. 1
  and Eq. 2 allow p in {0, 1}; Table 1's header names l1) is the alternative key: the sum of
  absolute values over the block.
* Selection -- Sec. 2.1, Eq. 2: the constrained form with tolerance tau on the number of nonzero
  groups.  With tau = k blocks, the Euclidean projection of W onto that set keeps the k blocks of
  largest key.  Ties go to the lower row-major block id, which makes the result unique.  The
  per-row balanced form applies the same constraint to every block-row separately (tau = k_row
  blocks in each row), so every block-row keeps the same number of blocks.
* Storage -- Sec. 2.2, second bullet: BSR as data values, indices and indptr, following SciPy.
* Product -- Sec. 2.2, first and second bullets: only stored blocks are multiplied with the input
  tensor.  The operation is Y = X W^T + b with W the pruned weight (BERT projections, Sec. 2.3).

Conventions (the paper leaves these open; the readings are listed with the design notes):
* W is N x K, row-major [out][in]; a block R x C covers R output rows and C input columns.
  Block (i, j) covers W[iR:(i+1)R, jC:(j+1)C]; its id is i*Kb + j with Kb = K/C.
* k = floor(density * nb + 0.5), computed in fp64, clamped to [0, nb].
* Keys are fp64, summed sequentially with r outer and c inner from +0.0 (l2: x*x, l1: |x|, both
  exact in fp64).  A NaN key ranks above +inf.
* Per-row balanced selection keeps k_row = floor(density * Kb + 0.5) blocks in every row.
* Products accumulate in fp64.  bf16 inputs are rounded to nearest, ties to even.
"""

from __future__ import annotations

import math

import numpy as np

# ---------------------------------------------------------------------------------------------
# Block partition and pruning count (Sec. 2.1, Eq. 2 and Eq. 3)
# ---------------------------------------------------------------------------------------------


def check_shape(N: int, K: int, R: int, C: int) -> tuple[int, int]:
    """Validate a block shape against a weight shape; return (Nb, Kb).

    Eq. 3 partitions the weight matrix into whole blocks, so R must divide N and C must divide K.
    """
    if R <= 0 or C <= 0 or N < 0 or K < 0:
        raise ValueError("block and matrix sizes must be positive")
    if N % R or K % C:
        raise ValueError(f"block {R}x{C} does not tile a {N}x{K} matrix")
    return N // R, K // C


def prune_count(N: int, K: int, R: int, C: int, density: float, per_row: bool = False) -> int:
    """Number of blocks kept at a block density: floor(density * nb + 0.5), in [0, nb].

    Eq. 2 bounds the count of nonzero groups by tau; density d names tau = round(d * nb)
    with halves rounded up.  With per_row, the bound applies to every block-row: each keeps
    floor(density * Kb + 0.5) of its Kb blocks, and the total is Nb times that.
    """
    Nb, Kb = check_shape(N, K, R, C)
    d = float(density)
    if not (0.0 <= d <= 1.0):  # also rejects NaN
        raise ValueError("density must lie in [0, 1]")
    if per_row:
        k_row = max(0, min(Kb, math.floor(d * Kb + 0.5)))
        return Nb * k_row
    nb = Nb * Kb
    k = math.floor(d * nb + 0.5)
    return max(0, min(nb, k))


def block_keys(W: np.ndarray, R: int, C: int, norm: str = "l2") -> np.ndarray:
    """Key of every block, fp64, in row-major block-id order (Eq. 3).

    norm "l2": the squared l2 norm (sum of x*x), the key of the l2 group norm.
    norm "l1": the l1 norm (sum of |x|), the p = 1 case of Eq. 1 and Eq. 2.
    The sum runs sequentially over the block's elements, row r outer and column c inner, starting
    from +0.0.  It is vectorised across blocks only, so the rounding of each key is that of the
    plain sequential loop.  Both terms are exact in fp64 (a product of two fp32 values has at
    most 48 significant bits), so only the additions round.
    """
    if norm not in ("l2", "l1"):
        raise ValueError("norm must be 'l2' or 'l1'")
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    Nb, Kb = check_shape(N, K, R, C)
    blocks = W.astype(np.float64).reshape(Nb, R, Kb, C)
    key = np.zeros((Nb, Kb), dtype=np.float64)
    for r in range(R):
        for c in range(C):
            x = blocks[:, r, :, c]
            key = key + (x * x if norm == "l2" else np.abs(x))
    return key.reshape(-1)


def _rank_bits(key: np.ndarray) -> np.ndarray:
    """Order-preserving uint64 image of non-negative fp64 keys; every NaN maps above +inf."""
    bits = np.ascontiguousarray(key, dtype=np.float64).view(np.uint64).copy()
    bits[np.isnan(key)] = np.uint64(0x7FF8000000000000)
    return bits


def select_topk(key: np.ndarray, k: int) -> np.ndarray:
    """Boolean mask of the k blocks that come first in the order (key descending, id ascending).

    This is the projection for Eq. 2 with a block-count constraint.  Keys are sums of squares, so
    they are >= +0.0 or NaN, and their IEEE bit patterns sort like their values.
    """
    key = np.asarray(key, dtype=np.float64)
    nb = key.size
    if not (0 <= k <= nb):
        raise ValueError("k must lie in [0, nb]")
    bits = _rank_bits(key)
    ids = np.arange(nb, dtype=np.int64)
    # np.lexsort sorts by the last key first: descending bits, then ascending id.
    order = np.lexsort((ids, ~bits))
    mask = np.zeros(nb, dtype=bool)
    mask[order[:k]] = True
    return mask


def select_topk_rows(key: np.ndarray, Nb: int, Kb: int, k_row: int) -> np.ndarray:
    """Boolean mask keeping, in every block-row, the k_row blocks that come first in the order
    (key descending, id ascending) among that row's blocks.

    This is Eq. 2 with the block-count constraint tau = k_row imposed on each block-row
    separately; the rows do not compete with each other.
    """
    key = np.asarray(key, dtype=np.float64).reshape(Nb, Kb)
    if not (0 <= k_row <= Kb):
        raise ValueError("k_row must lie in [0, Kb]")
    mask = np.zeros((Nb, Kb), dtype=bool)
    for i in range(Nb):
        bits = _rank_bits(key[i])
        cols = np.arange(Kb, dtype=np.int64)
        order = np.lexsort((cols, ~bits))
        mask[i, order[:k_row]] = True
    return mask.reshape(-1)


def build_bsr(W: np.ndarray, R: int, C: int, mask: np.ndarray):
    """BSR arrays (indptr int32[Nb+1], indices int32[k], data float32[k, R, C]) of W under mask.

    Sec. 2.2 stores a block-sparse matrix as data, indices and indptr in SciPy's layout: the
    blocks of block-row i are data[indptr[i]:indptr[i+1]], in ascending column order, and
    indices holds their block-column numbers.  Block values are exact copies of W's bits.
    """
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    Nb, Kb = check_shape(N, K, R, C)
    mask = np.asarray(mask, dtype=bool).reshape(Nb, Kb)
    indptr = np.zeros(Nb + 1, dtype=np.int32)
    indices: list[int] = []
    blocks: list[np.ndarray] = []
    for i in range(Nb):
        for j in range(Kb):
            if mask[i, j]:
                indices.append(j)
                blocks.append(W[i * R:(i + 1) * R, j * C:(j + 1) * C])
        indptr[i + 1] = len(indices)
    data = (np.stack(blocks).astype(np.float32) if blocks
            else np.zeros((0, R, C), dtype=np.float32))
    return indptr, np.asarray(indices, dtype=np.int32), data


def prune(W: np.ndarray, R: int, C: int, density: float | None = None, k: int | None = None,
          norm: str = "l2", per_row: bool = False):
    """Dense W -> BSR keeping the top-k blocks by block norm (Eq. 2 and Eq. 3).

    Give exactly one of density and k.  norm is "l2" or "l1" (block_keys).  With per_row, k is
    the total over all block-rows and must be a multiple of Nb; every row keeps k / Nb blocks.
    Returns (indptr, indices, data).
    """
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    Nb, Kb = check_shape(N, K, R, C)
    if (density is None) == (k is None):
        raise ValueError("give exactly one of density and k")
    if k is None:
        k = prune_count(N, K, R, C, density, per_row=per_row)
    key = block_keys(W, R, C, norm)
    if per_row:
        if Nb == 0 or int(k) % Nb:
            raise ValueError("per-row selection needs k to be a multiple of Nb")
        mask = select_topk_rows(key, Nb, Kb, int(k) // Nb)
    else:
        mask = select_topk(key, int(k))
    return build_bsr(W, R, C, mask)


def reblock(indptr, indices, data, R2: int, C2: int):
    """The same matrix in finer blocks R2 x C2 (R2 | R, C2 | C): every stored R x C block is cut
    into (R/R2) x (C/C2) stored blocks.  Values are bit copies; the stored pattern is the
    original one refined (a zero R2 x C2 piece of a stored block stays stored).

    Sec. 2.2 stores a matrix as data/indices/indptr for one block shape; this is SciPy's
    conversion of a BSR matrix to a smaller block size, written out: fine block-row i * a + r
    (a = R/R2, r < a) holds, for each stored block p of block-row i in column order, the pieces
    s < b = C/C2 with block-column indices[p] * b + s.
    """
    data = np.asarray(data)
    R, C = data.shape[1], data.shape[2]
    if R2 <= 0 or C2 <= 0 or R % R2 or C % C2:
        raise ValueError("the new block shape must divide the old one")
    a, b = R // R2, C // C2
    indptr = np.asarray(indptr, dtype=np.int64)
    Nb = indptr.size - 1
    new_ptr = [0]
    new_idx: list[int] = []
    new_data: list[np.ndarray] = []
    for i in range(Nb):
        for r in range(a):
            for p in range(indptr[i], indptr[i + 1]):
                for s_ in range(b):
                    new_idx.append(int(indices[p]) * b + s_)
                    new_data.append(data[p, r * R2:(r + 1) * R2, s_ * C2:(s_ + 1) * C2])
            new_ptr.append(len(new_idx))
    out = (np.stack(new_data) if new_data else np.zeros((0, R2, C2), dtype=data.dtype))
    return (np.asarray(new_ptr, dtype=np.int32), np.asarray(new_idx, dtype=np.int32),
            out.astype(data.dtype))


def to_dense(indptr, indices, data, N: int, K: int) -> np.ndarray:
    """Expand BSR arrays to a dense N x K matrix; positions outside stored blocks are +0.0."""
    data = np.asarray(data)
    if data.ndim != 3:
        raise ValueError("data must be [nnzb, R, C]")
    R, C = data.shape[1], data.shape[2]
    Nb, Kb = check_shape(N, K, R, C)
    out = np.zeros((N, K), dtype=data.dtype)
    for i in range(Nb):
        for p in range(int(indptr[i]), int(indptr[i + 1])):
            j = int(indices[p])
            out[i * R:(i + 1) * R, j * C:(j + 1) * C] = data[p]
    return out


# ---------------------------------------------------------------------------------------------
# Products (Sec. 2.2): two independent routes, both fp64
# ---------------------------------------------------------------------------------------------


def spmm_loop(X: np.ndarray, indptr, indices, data, N: int, bias=None) -> np.ndarray:
    """Y = X W^T + b by walking the stored blocks only (fp64).

    For block-row i and each stored block p with block-column j:
    Y[:, iR:(i+1)R] += X[:, jC:(j+1)C] @ data[p]^T.  Vectorised over tokens only.
    """
    X64 = np.asarray(X, dtype=np.float64)
    T, K = X64.shape
    data64 = np.asarray(data, dtype=np.float64)
    R, C = data64.shape[1], data64.shape[2]
    Nb, _ = check_shape(N, K, R, C)
    Y = np.zeros((T, N), dtype=np.float64)
    if bias is not None:
        Y += np.asarray(bias, dtype=np.float64)[None, :]
    for i in range(Nb):
        acc = Y[:, i * R:(i + 1) * R]
        for p in range(int(indptr[i]), int(indptr[i + 1])):
            j = int(indices[p])
            acc += X64[:, j * C:(j + 1) * C] @ data64[p].T
    return Y


def spmm_masked_dense(X: np.ndarray, W_masked: np.ndarray, bias=None) -> np.ndarray:
    """Y = X (W masked)^T + b with a dense fp64 matrix product (the plain definition)."""
    Y = np.asarray(X, dtype=np.float64) @ np.asarray(W_masked, dtype=np.float64).T
    if bias is not None:
        Y = Y + np.asarray(bias, dtype=np.float64)[None, :]
    return Y


def tolerance_scale(X: np.ndarray, W_masked: np.ndarray) -> np.ndarray:
    """S[t, n] = sum_k |X[t, k]| * |W_masked[n, k]| in fp64: the scale of the fp32 error bound."""
    return np.abs(np.asarray(X, dtype=np.float64)) @ np.abs(np.asarray(W_masked, np.float64)).T


def spmm_tolerance(S: np.ndarray, rel: float = 1e-5, abs_: float = 1e-6) -> np.ndarray:
    """Per-element acceptance bound |Y_gpu - Y64| <= rel * S + abs for fp32 accumulation."""
    return rel * S + abs_


# ---------------------------------------------------------------------------------------------
# bf16 rounding (input precision of the bf16 configurations)
# ---------------------------------------------------------------------------------------------


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even.

    Written from the definition: the two bf16 neighbours of x are its truncation toward zero and
    the next bf16 away from zero; pick the nearer (fp64 distances are exact here), and on a tie
    the one with an even last mantissa bit.  Past the largest finite bf16 the upper neighbour is
    taken at the value 2**128, so halfway and beyond round to infinity.  NaN stays NaN (quiet).
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    sign = u & np.uint64(0x80000000)
    mag = u & np.uint64(0x7FFFFFFF)
    lo = mag & np.uint64(0xFFFF0000)
    hi = lo + np.uint64(0x10000)
    # NaN and infinite inputs give meaningless distances here; they are replaced below.
    with np.errstate(invalid="ignore"):
        v = np.abs(x.astype(np.float64))
        v_lo = (lo.astype(np.uint32)).view(np.float32).astype(np.float64)
        hi_is_inf = hi >= np.uint64(0x7F800000)
        v_hi = np.where(hi_is_inf, 2.0 ** 128,
                        (np.minimum(hi, np.uint64(0x7F7F0000)).astype(np.uint32))
                        .view(np.float32).astype(np.float64))
        d_lo = v - v_lo
        d_hi = v_hi - v
    lo_even = ((lo >> np.uint64(16)) & np.uint64(1)) == 0
    take_hi = (d_hi < d_lo) | ((d_hi == d_lo) & ~lo_even)
    out_mag = np.where(take_hi, hi, lo)
    out = ((sign | out_mag) >> np.uint64(16)).astype(np.uint16)
    is_inf = mag == np.uint64(0x7F800000)
    out = np.where(is_inf, ((sign | mag) >> np.uint64(16)).astype(np.uint16), out)
    is_nan = mag > np.uint64(0x7F800000)
    nan_bits = (((sign | mag) >> np.uint64(16)) | np.uint64(0x0040)).astype(np.uint16)
    out = np.where(is_nan, nan_bits, out)
    return out.astype(np.uint16)


def bf16_to_f32(h: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> the fp32 values they denote (exact)."""
    h = np.ascontiguousarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_roundtrip(x: np.ndarray) -> np.ndarray:
    """x rounded to bf16 and widened back to fp32."""
    return bf16_to_f32(bf16_round(x))
