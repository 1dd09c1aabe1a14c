"""Helpers for the GPU parity tests: run libbsr on the device, compare with the CPU oracle."""
from __future__ import annotations

import numpy as np
import torch

from oracle import bsr_oracle as O
from paper_2106_08846_amd import bsr as B

REL_TOL = 1e-5
ABS_TOL = 1e-6


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").numpy()


def log(msg: str) -> None:
    print(msg, flush=True)


def check_prune(W: np.ndarray, R: int, C: int, M: B.BSRMatrix, k: int) -> None:
    """indptr, indices and data of the GPU result equal the oracle's, bit for bit."""
    ip, ix, dt = O.prune(W, R, C, k=k)
    assert M.nnzb == k
    g_ip = host(M.indptr)
    g_ix = host(M.indices)[:k]
    g_dt = host(M.data)[:k]
    assert np.array_equal(g_ip, ip), "indptr differs"
    assert np.array_equal(g_ix, ix), "indices differ"
    assert np.array_equal(g_dt.view(np.uint32), dt.view(np.uint32)), "data bits differ"


def oracle_bsr(M: B.BSRMatrix):
    """The GPU BSR arrays copied to the host (fp32 data, or bf16 widened exactly to fp32)."""
    ip = host(M.indptr)
    ix = host(M.indices)[:M.nnzb]
    d = M.data[:M.nnzb]
    if d.dtype == torch.bfloat16:
        dt = O.bf16_to_f32(host(d.contiguous().view(torch.int16)).view(np.uint16))
    else:
        dt = host(d)
    return ip, ix, dt.reshape(M.nnzb, M.R, M.C)


def check_spmm(X: np.ndarray, M: B.BSRMatrix, bias: np.ndarray | None, Y: torch.Tensor,
               rows: np.ndarray | None = None, bf16: bool = False) -> float:
    """|Y - Y64| <= 1e-5 * S + 1e-6 elementwise, Y64 from the fp64 oracle on the same inputs.

    For bf16, X and the BSR data are the bf16-rounded values (rounded by the oracle's own
    bf16_round for X; the data comes back from the device and is widened exactly).  `rows`
    restricts the comparison to a sample of token rows.  Returns the worst ratio err / bound.
    """
    ip, ix, dt = oracle_bsr(M)
    Xh = O.bf16_roundtrip(X) if bf16 else X
    if rows is not None:
        Xh = Xh[rows]
    Wm = O.to_dense(ip, ix, dt, M.n_rows, M.n_cols)
    Y64 = O.spmm_masked_dense(Xh, Wm, bias)
    S = O.tolerance_scale(Xh, Wm)
    Yg = host(Y)
    if rows is not None:
        Yg = Yg[rows]
    bound = O.spmm_tolerance(S, REL_TOL, ABS_TOL)
    err = np.abs(Yg.astype(np.float64) - Y64)
    assert np.all(np.isfinite(Yg)), "non-finite output"
    worst = float(np.max(err / bound)) if err.size else 0.0
    assert np.all(err <= bound), f"tolerance exceeded: worst err/bound = {worst:.3f}"
    return worst


def prune_on_gpu(W: np.ndarray, R: int, C: int, k: int) -> B.BSRMatrix:
    """W pruned to its k largest R x C blocks on the GPU, checked bit for bit against the
    oracle's prune before it is returned, so that every product test whose oracle input is
    built from the device's BSR arrays (oracle_bsr) multiplies the matrix the paper's pruning
    defines."""
    M = B.bsr_prune_from_dense(dev(W), R, C, k=k)
    check_prune(W, R, C, M, k)
    return M


def bf16_tensor(x: np.ndarray) -> torch.Tensor:
    """Device bf16 tensor of x rounded by libbsr's cast kernel."""
    return B.bsr_cast_f32_bf16(dev(np.ascontiguousarray(x, dtype=np.float32)))
