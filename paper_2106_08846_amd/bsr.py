"""Thin Python binding of libbsr's C ABI (ctypes).

Argument marshalling only: torch tensors supply device memory and the current HIP stream; every
computation runs in libbsr's kernels.  The functions carry the C entry points' names.  Loading
fails loudly when libbsr.so has not been built -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(_HERE, "libbsr.so")

BSR_F32, BSR_BF16 = 0, 1
STATUS = {0: "BSR_OK", 1: "BSR_ERR_NULL", 2: "BSR_ERR_SHAPE", 3: "BSR_ERR_ARG",
          4: "BSR_ERR_DTYPE", 5: "BSR_ERR_CAPACITY", 6: "BSR_ERR_WORKSPACE", 7: "BSR_ERR_HIP",
          8: "BSR_ERR_ARCH", 9: "BSR_ERR_UNSUPPORTED"}

# The C ABI's exported entry points (the tests check this list against include/libbsr.h).
EXPORTS = ["bsr_prune_count", "bsr_prune_count_ex", "bsr_prune_workspace_bytes",
           "bsr_prune_from_dense", "bsr_prune_from_dense_noalloc", "bsr_prune_from_dense_ex",
           "bsr_spmm", "bsr_spmm_ex",
           "bsr_spmm_batched", "bsr_plan_bytes", "bsr_plan_bytes_ex", "bsr_plan_prepare",
           "bsr_plan_prepare_ex", "bsr_spmm_batched_planned", "bsr_attention", "bsr_reblock",
           "bsr_to_dense",
           "bsr_cast_f32_bf16", "bsr_iht_update",
           "bsr_status_str", "bsr_last_hip_error"]
NORM_L2, NORM_L1 = 0, 1
SELECT_GLOBAL, SELECT_PER_ROW = 0, 1
KERNEL_AUTO, KERNEL_GENERIC, KERNEL_TILED, KERNEL_VALU = 0, 1, 2, 3
ARITH_AUTO, ARITH_NATIVE, ARITH_BF16X3 = 0, 1, 2


class BSRError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        name = STATUS.get(status, str(status))
        msg = f"{where}: {name} ({_lib().bsr_status_str(status).decode()})"
        if detail:
            msg += f": {detail}"
        super().__init__(msg)


class bsr_spmm_options_t(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32), ("slices", ctypes.c_int32),
                ("start_event", ctypes.c_void_p), ("stop_event", ctypes.c_void_p)]


class bsr_prune_options_t(ctypes.Structure):
    _fields_ = [("norm", ctypes.c_int32), ("select", ctypes.c_int32)]


class bsr_matrix_t(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int64), ("n_cols", ctypes.c_int64),
                ("R", ctypes.c_int32), ("C", ctypes.c_int32), ("nnzb", ctypes.c_int64),
                ("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p),
                ("data", ctypes.c_void_p), ("dtype", ctypes.c_int)]


class bsr_spmm_item_t(ctypes.Structure):
    _fields_ = [("X", ctypes.c_void_p), ("x_dtype", ctypes.c_int), ("T", ctypes.c_int64),
                ("ldx", ctypes.c_int64), ("W", ctypes.POINTER(bsr_matrix_t)),
                ("bias", ctypes.c_void_p), ("Y", ctypes.c_void_p), ("ldy", ctypes.c_int64)]


class bsr_plan_t(ctypes.Structure):
    _fields_ = [("mem", ctypes.c_void_p), ("bytes", ctypes.c_size_t),
                ("n_rows", ctypes.c_int64), ("n_cols", ctypes.c_int64), ("nnzb", ctypes.c_int64),
                ("R", ctypes.c_int32), ("C", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p),
                ("data", ctypes.c_void_p), ("unit_blocks", ctypes.c_int32),
                ("max_units", ctypes.c_int64), ("uptr_offset", ctypes.c_int64),
                ("col_offset", ctypes.c_int64), ("val_offset", ctypes.c_int64),
                ("arith", ctypes.c_int32)]


_LIB = None


def _lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIBRARY):
            raise RuntimeError(f"libbsr is not built ({LIBRARY} missing); "
                               "run paper_2106_08846_amd/build.py")
        lib = ctypes.CDLL(LIBRARY)
        i64, i32, p, sz = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t
        st = ctypes.c_int
        lib.bsr_prune_count.argtypes = [i64, i64, i32, i32, ctypes.c_double,
                                        ctypes.POINTER(i64)]
        lib.bsr_prune_count.restype = st
        lib.bsr_prune_count_ex.argtypes = [i64, i64, i32, i32, ctypes.c_double,
                                           ctypes.POINTER(bsr_prune_options_t),
                                           ctypes.POINTER(i64)]
        lib.bsr_prune_count_ex.restype = st
        lib.bsr_prune_from_dense_ex.argtypes = [p, i64, i64, i64, i32, i32, i64, p, p, p, i64,
                                                p, sz, ctypes.POINTER(bsr_prune_options_t), p]
        lib.bsr_prune_from_dense_ex.restype = st
        lib.bsr_prune_workspace_bytes.argtypes = [i64, i64, i32, i32]
        lib.bsr_prune_workspace_bytes.restype = sz
        lib.bsr_prune_from_dense.argtypes = [p, i64, i64, i64, i32, i32, i64, p, p, p, i64, p,
                                             sz, p]
        lib.bsr_prune_from_dense.restype = st
        lib.bsr_prune_from_dense_noalloc.argtypes = [p, i64, i64, i64, i32, i32, i64, p, p, p,
                                                     i64, p]
        lib.bsr_prune_from_dense_noalloc.restype = st
        lib.bsr_spmm.argtypes = [p, ctypes.c_int, i64, i64, ctypes.POINTER(bsr_matrix_t), p, p,
                                 i64, p]
        lib.bsr_spmm.restype = st
        lib.bsr_spmm_ex.argtypes = [p, ctypes.c_int, i64, i64, ctypes.POINTER(bsr_matrix_t), p,
                                    p, i64, ctypes.POINTER(bsr_spmm_options_t), p]
        lib.bsr_spmm_ex.restype = st
        lib.bsr_spmm_batched.argtypes = [ctypes.POINTER(bsr_spmm_item_t), i32,
                                         ctypes.POINTER(bsr_spmm_options_t), p]
        lib.bsr_spmm_batched.restype = st
        lib.bsr_plan_bytes.argtypes = [ctypes.POINTER(bsr_matrix_t), ctypes.POINTER(sz)]
        lib.bsr_plan_bytes.restype = st
        lib.bsr_plan_prepare.argtypes = [ctypes.POINTER(bsr_matrix_t), p, sz,
                                         ctypes.POINTER(bsr_plan_t), p]
        lib.bsr_plan_prepare.restype = st
        lib.bsr_plan_bytes_ex.argtypes = [ctypes.POINTER(bsr_matrix_t), i32, ctypes.POINTER(sz)]
        lib.bsr_plan_bytes_ex.restype = st
        lib.bsr_plan_prepare_ex.argtypes = [ctypes.POINTER(bsr_matrix_t), i32, p, sz,
                                            ctypes.POINTER(bsr_plan_t), p]
        lib.bsr_plan_prepare_ex.restype = st
        lib.bsr_spmm_batched_planned.argtypes = [ctypes.POINTER(bsr_spmm_item_t),
                                                 ctypes.POINTER(ctypes.POINTER(bsr_plan_t)), i32,
                                                 ctypes.POINTER(bsr_spmm_options_t), p]
        lib.bsr_spmm_batched_planned.restype = st
        lib.bsr_to_dense.argtypes = [ctypes.POINTER(bsr_matrix_t), p, i64, p]
        lib.bsr_to_dense.restype = st
        lib.bsr_attention.argtypes = [p, i64, p, i64, p, i64, p, i64, i32, i32, i32, i32,
                                      ctypes.c_float, p]
        lib.bsr_attention.restype = st
        lib.bsr_reblock.argtypes = [ctypes.POINTER(bsr_matrix_t), i32, i32, p, p, p, p]
        lib.bsr_reblock.restype = st
        lib.bsr_cast_f32_bf16.argtypes = [p, p, i64, p]
        lib.bsr_cast_f32_bf16.restype = st
        lib.bsr_iht_update.argtypes = [p, i64, p, i64, p, i64, ctypes.c_float, i64, i64, p, i64,
                                       p]
        lib.bsr_iht_update.restype = st
        lib.bsr_status_str.argtypes = [ctypes.c_int]
        lib.bsr_status_str.restype = ctypes.c_char_p
        lib.bsr_last_hip_error.argtypes = []
        lib.bsr_last_hip_error.restype = ctypes.c_char_p
        _LIB = lib
    return _LIB


def library() -> ctypes.CDLL:
    """The loaded libbsr (raises if it has not been built)."""
    return _lib()


def _check(status: int, where: str) -> None:
    if status != 0:
        detail = _lib().bsr_last_hip_error().decode() if status == 7 else ""
        raise BSRError(status, where, detail)


# torch's current stream as a raw handle, without building a torch.cuda.Stream object (that
# costs about 3 us per call, more than a kernel launch's host time here).
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_cur_device = getattr(torch._C, "_cuda_getDevice", None)


def _stream(stream) -> int | None:
    if stream is None:
        if _raw_stream is not None and _cur_device is not None:
            return _raw_stream(_cur_device())
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _require_cuda(t: torch.Tensor, name: str, dtype=None) -> None:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")


def _pitch(t: torch.Tensor, name: str) -> int:
    """Row pitch (elements) of a 2-D tensor whose rows are contiguous."""
    if t.dim() == 2 and t.numel() == 0:
        return max(t.shape[1], 1)          # an empty tensor's strides carry no layout
    if t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError(f"{name} must be 2-D with unit column stride")
    return t.stride(0) if t.shape[0] > 1 else max(t.shape[1], 1)


@dataclass
class BSRMatrix:
    """A BSR matrix whose arrays live in torch device tensors (Sec. 2.2 layout)."""
    n_rows: int
    n_cols: int
    R: int
    C: int
    indptr: torch.Tensor      # int32 [N/R + 1]
    indices: torch.Tensor     # int32 [>= nnzb]
    data: torch.Tensor        # float32 or bfloat16 [>= nnzb, R, C]
    nnzb: int

    @property
    def dtype(self) -> int:
        return BSR_BF16 if self.data.dtype == torch.bfloat16 else BSR_F32

    def check(self) -> None:
        """Raise unless the tensors hold the arrays the descriptor names (the C side cannot see
        a tensor's size): indptr int32 with at least N/R + 1 entries, indices int32 with at
        least nnzb, data [>= nnzb, R, C] float32 or bfloat16, each contiguous on a GPU."""
        if self.R <= 0 or self.C <= 0 or self.n_rows % self.R or self.n_cols % self.C:
            raise ValueError(f"block {self.R}x{self.C} does not tile {self.n_rows}x{self.n_cols}")
        nb_rows = self.n_rows // self.R
        for t, n, dt, need in ((self.indptr, "indptr", torch.int32, nb_rows + 1),
                               (self.indices, "indices", torch.int32, self.nnzb)):
            if not isinstance(t, torch.Tensor) or t.dtype != dt or not t.is_contiguous():
                raise ValueError(f"{n} must be a contiguous {dt} tensor")
            if t.numel() < need:
                raise ValueError(f"{n} holds {t.numel()} entries, the matrix needs {need}")
        d = self.data
        if (not isinstance(d, torch.Tensor) or d.dtype not in (torch.float32, torch.bfloat16)
                or d.dim() != 3 or tuple(d.shape[1:]) != (self.R, self.C)
                or not d.is_contiguous()):
            raise ValueError(f"data must be a contiguous [nnzb, {self.R}, {self.C}] float32 or "
                             "bfloat16 tensor")
        if d.shape[0] < self.nnzb:
            raise ValueError(f"data holds {d.shape[0]} blocks, the matrix has {self.nnzb}")
        for t, n in ((self.indptr, "indptr"), (self.indices, "indices"), (d, "data")):
            _require_cuda(t, n)

    def struct(self) -> bsr_matrix_t:
        self.check()
        return bsr_matrix_t(self.n_rows, self.n_cols, self.R, self.C, self.nnzb,
                            _ptr(self.indptr), _ptr(self.indices), _ptr(self.data), self.dtype)

    def to_bf16(self, stream=None) -> "BSRMatrix":
        """Copy with data rounded to bf16 by bsr_cast_f32_bf16 (indices shared)."""
        data = bsr_cast_f32_bf16(self.data[: self.nnzb], stream=stream)
        return BSRMatrix(self.n_rows, self.n_cols, self.R, self.C, self.indptr, self.indices,
                         data, self.nnzb)


def _prune_opts(norm: str, per_row: bool) -> bsr_prune_options_t:
    if norm not in ("l2", "l1"):
        raise ValueError("norm must be 'l2' or 'l1'")
    return bsr_prune_options_t(NORM_L1 if norm == "l1" else NORM_L2,
                               SELECT_PER_ROW if per_row else SELECT_GLOBAL)


def bsr_prune_count(N: int, K: int, R: int, C: int, density: float, per_row: bool = False) -> int:
    k = ctypes.c_int64(0)
    if per_row:
        opts = _prune_opts("l2", True)
        _check(_lib().bsr_prune_count_ex(N, K, R, C, float(density), ctypes.byref(opts),
                                         ctypes.byref(k)), "bsr_prune_count_ex")
    else:
        _check(_lib().bsr_prune_count(N, K, R, C, float(density), ctypes.byref(k)),
               "bsr_prune_count")
    return k.value


def bsr_prune_workspace_bytes(N: int, K: int, R: int, C: int) -> int:
    return int(_lib().bsr_prune_workspace_bytes(N, K, R, C))


def bsr_prune_from_dense(W: torch.Tensor, R: int, C: int, k: int | None = None,
                         density: float | None = None, workspace: torch.Tensor | None = None,
                         stream=None, norm: str = "l2", per_row: bool = False) -> BSRMatrix:
    """Prune dense fp32 W (device, [N, K]) to BSR with R x C blocks, keeping k blocks.

    norm "l2" (default) or "l1" selects the block key; per_row keeps k / Nb blocks in every
    block-row (bsr_prune_from_dense_ex); the defaults call bsr_prune_from_dense."""
    _require_cuda(W, "W", torch.float32)
    N, K = W.shape
    ldw = _pitch(W, "W")
    if (k is None) == (density is None):
        raise ValueError("give exactly one of k and density")
    opts = _prune_opts(norm, per_row)
    if k is None:
        k = bsr_prune_count(N, K, R, C, density, per_row=per_row)
    dev = W.device
    Nb = N // R if R > 0 and N % R == 0 else 0
    indptr = torch.empty(Nb + 1, dtype=torch.int32, device=dev)
    indices = torch.empty(max(k, 1), dtype=torch.int32, device=dev)
    data = torch.empty((max(k, 1), R, C), dtype=torch.float32, device=dev)
    ws_bytes = bsr_prune_workspace_bytes(N, K, R, C)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    ws_len = workspace.numel() * workspace.element_size()
    if norm == "l2" and not per_row:
        _check(_lib().bsr_prune_from_dense(_ptr(W), N, K, ldw, R, C, k, _ptr(indptr),
                                           _ptr(indices), _ptr(data), max(k, 1), _ptr(workspace),
                                           ws_len, _stream(stream)),
               "bsr_prune_from_dense")
    else:
        _check(_lib().bsr_prune_from_dense_ex(_ptr(W), N, K, ldw, R, C, k, _ptr(indptr),
                                              _ptr(indices), _ptr(data), max(k, 1),
                                              _ptr(workspace), ws_len, ctypes.byref(opts),
                                              _stream(stream)),
               "bsr_prune_from_dense_ex")
    return BSRMatrix(N, K, R, C, indptr, indices, data, k)


NOALLOC_MAX_BLOCKS = 1 << 20


def bsr_prune_from_dense_noalloc(W: torch.Tensor, R: int, C: int, k: int, indptr: torch.Tensor,
                                 indices: torch.Tensor, data: torch.Tensor,
                                 stream=None) -> BSRMatrix:
    """bsr_prune_from_dense_noalloc into caller-allocated outputs (the library allocates
    nothing: its workspace is a fixed array, at most NOALLOC_MAX_BLOCKS blocks)."""
    _require_cuda(W, "W", torch.float32)
    N, K = W.shape
    ldw = _pitch(W, "W")
    Nb = N // R if R > 0 and N % R == 0 else 0
    if indptr.numel() < Nb + 1 or indices.numel() < k or data.numel() < k * R * C:
        raise ValueError("output tensors are smaller than k blocks need")
    for t, n, dt in ((indptr, "indptr", torch.int32), (indices, "indices", torch.int32),
                     (data, "data", torch.float32)):
        _require_cuda(t, n, dt)
        if not t.is_contiguous():
            raise ValueError(f"{n} must be contiguous")
    cap = min(indices.numel(), data.numel() // max(R * C, 1))
    _check(_lib().bsr_prune_from_dense_noalloc(_ptr(W), N, K, ldw, R, C, k, _ptr(indptr),
                                               _ptr(indices), _ptr(data), cap, _stream(stream)),
           "bsr_prune_from_dense_noalloc")
    return BSRMatrix(N, K, R, C, indptr, indices, data.view(-1)[: max(cap, 1) * R * C]
                     .view(max(cap, 1), R, C), k)


def bsr_spmm(X: torch.Tensor, W: BSRMatrix, bias: torch.Tensor | None = None,
             Y: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Y = X W^T + bias with W in BSR (fp32 or bf16 inputs; fp32 accumulate and output)."""
    return bsr_spmm_ex(X, W, bias, Y, None, None, stream)


def bsr_spmm_ex(X: torch.Tensor, W: BSRMatrix, bias: torch.Tensor | None = None,
                Y: torch.Tensor | None = None, kernel: int | None = None,
                slices: int | None = None, stream=None) -> torch.Tensor:
    """bsr_spmm with an explicit kernel (KERNEL_*) and slice count; None = automatic."""
    if Y is None and isinstance(X, torch.Tensor) and X.dim() == 2:
        Y = torch.empty((X.shape[0], W.n_rows), dtype=torch.float32, device=X.device)
    _check_call(X, W, bias, Y)
    x_dtype = BSR_BF16 if X.dtype == torch.bfloat16 else BSR_F32
    T = X.shape[0]
    ldx = _pitch(X, "X")
    ldy = _pitch(Y, "Y")
    m = W.struct()
    if kernel is None and slices is None:
        _check(_lib().bsr_spmm(_ptr(X), x_dtype, T, ldx, ctypes.byref(m), _ptr(bias), _ptr(Y),
                               ldy, _stream(stream)), "bsr_spmm")
    else:
        opts = bsr_spmm_options_t(kernel or 0, slices or 0, None, None)
        _check(_lib().bsr_spmm_ex(_ptr(X), x_dtype, T, ldx, ctypes.byref(m), _ptr(bias),
                                  _ptr(Y), ldy, ctypes.byref(opts), _stream(stream)),
               "bsr_spmm_ex")
    return Y


def _check_call(X: torch.Tensor, W: BSRMatrix, bias: torch.Tensor | None,
                Y: torch.Tensor) -> None:
    """Shapes before anything reaches the library: X is [T, K] and Y [T, N] with K, N the
    matrix's, so every row the kernels read or write lies inside its tensor; then devices."""
    if not isinstance(X, torch.Tensor) or X.dim() != 2 or X.shape[1] != W.n_cols:
        raise ValueError(f"X must be [T, {W.n_cols}]")
    if not isinstance(Y, torch.Tensor) or tuple(Y.shape) != (X.shape[0], W.n_rows):
        raise ValueError(f"Y must be [{X.shape[0]}, {W.n_rows}]")
    if bias is not None and (not isinstance(bias, torch.Tensor) or bias.dim() != 1
                             or bias.numel() != W.n_rows or not bias.is_contiguous()):
        raise ValueError("bias must be a contiguous [N] float32 tensor")
    W.check()
    _require_cuda(X, "X")
    if X.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("X must be float32 or bfloat16")
    if bias is not None:
        _require_cuda(bias, "bias", torch.float32)
    _require_cuda(Y, "Y", torch.float32)


class BSRPlan:
    """A per-matrix product plan (bsr_plan_prepare) in a torch device buffer: the matrix's unit
    row pointer and its units' columns and weights packed in the order the matrix cores read
    them.  It stays valid while the matrix's arrays are unchanged."""

    def __init__(self, W: BSRMatrix, mem: torch.Tensor, plan: bsr_plan_t):
        self.W = W
        self.mem = mem
        self.struct = plan

    @property
    def unit_blocks(self) -> int:
        return self.struct.unit_blocks

    @property
    def arith(self) -> int:
        """The plan's arithmetic: ARITH_NATIVE or ARITH_BF16X3."""
        return self.struct.arith

    def uptr(self) -> torch.Tensor:
        """The unit row pointer (a view into the plan's memory)."""
        nb = self.W.n_rows // self.W.R + 1
        off = self.struct.uptr_offset
        return self.mem[off:off + 4 * nb].view(torch.int32)


def bsr_plan_bytes(W: BSRMatrix, arith: int = ARITH_AUTO) -> int:
    """Device bytes of W's plan of the given arithmetic (bsr_plan_bytes_ex; raises BSRError
    BSR_ERR_UNSUPPORTED for shapes without one)."""
    n = ctypes.c_size_t(0)
    m = W.struct()
    _check(_lib().bsr_plan_bytes_ex(ctypes.byref(m), int(arith), ctypes.byref(n)),
           "bsr_plan_bytes_ex")
    return int(n.value)


def bsr_plan_prepare(W: BSRMatrix, mem: torch.Tensor | None = None, stream=None,
                     arith: int = ARITH_AUTO) -> BSRPlan:
    """Prepare W's plan of the given arithmetic (bsr_plan_prepare_ex) in `mem` (a uint8
    device tensor of at least bsr_plan_bytes(W, arith) bytes, allocated here when None)."""
    nbytes = bsr_plan_bytes(W, arith)
    if mem is None:
        mem = torch.empty(nbytes, dtype=torch.uint8, device=W.indptr.device)
    _require_cuda(mem, "mem", torch.uint8)
    if not mem.is_contiguous():
        raise ValueError("mem must be contiguous")
    plan = bsr_plan_t()
    m = W.struct()
    _check(_lib().bsr_plan_prepare_ex(ctypes.byref(m), int(arith), _ptr(mem), mem.numel(),
                                      ctypes.byref(plan), _stream(stream)),
           "bsr_plan_prepare_ex")
    return BSRPlan(W, mem, plan)


class SpmmBatchCall:
    """A bsr_spmm_batched call with its arguments marshalled once.

    `products` is a list of (X, W, bias, Y) tuples; `plans` (optional) a list of the same
    length whose entries are BSRPlan objects or None, making it a bsr_spmm_batched_planned
    call.  Calling the object re-issues the same C call on the given stream, or on torch's
    current stream, which is what a serving loop or a HIP graph capture needs: the per-call
    host cost is one foreign call.  The tensors stay referenced by the object.
    """

    def __init__(self, products, kernel: int | None = None, slices: int | None = None,
                 plans=None):
        self._keep = list(products)
        self._mats = []
        items = (bsr_spmm_item_t * max(len(products), 1))()
        for i, (X, W, bias, Y) in enumerate(products):
            _check_call(X, W, bias, Y)
            m = W.struct()
            self._mats.append(m)
            items[i] = bsr_spmm_item_t(_ptr(X), BSR_BF16 if X.dtype == torch.bfloat16 else BSR_F32,
                                       X.shape[0], _pitch(X, "X"), ctypes.pointer(m), _ptr(bias),
                                       _ptr(Y), _pitch(Y, "Y"))
        self._items = items
        self._opts = bsr_spmm_options_t(kernel or 0, slices or 0, None, None)
        self._timed_opts = bsr_spmm_options_t(kernel or 0, slices or 0, None, None)
        self._n = len(products)
        self.Y = [p[3] for p in products]
        self._plans = None
        if plans is not None:
            if len(plans) != len(products):
                raise ValueError("give one plan (or None) per product")
            self._keep_plans = list(plans)
            arr = (ctypes.POINTER(bsr_plan_t) * max(len(plans), 1))()
            for i, (pl, (X, W, bias, Y)) in enumerate(zip(plans, products)):
                if pl is not None:
                    if pl.W is not W:
                        raise ValueError("a plan must be prepared for its product's matrix")
                    arr[i] = ctypes.pointer(pl.struct)
            self._plans = arr
            fn = _lib().bsr_spmm_batched_planned
            plans_arr = arr
            self._fn = lambda items, n, opts, st: fn(items, plans_arr, n, opts, st)
            self._name = "bsr_spmm_batched_planned"
        else:
            self._fn = _lib().bsr_spmm_batched
            self._name = "bsr_spmm_batched"

    def __call__(self, stream=None):
        st = self._fn(self._items, self._n, ctypes.byref(self._opts), _stream(stream))
        if st != 0:
            _check(st, self._name)
        return self.Y

    def timed(self, start: torch.cuda.Event, stop: torch.cuda.Event, stream=None):
        """Issue the call with `start`/`stop` recorded at the start of its first kernel and the
        end of its last one.

        Both events must be timing events that have been recorded once (torch creates the
        underlying HIP event lazily); afterwards start.elapsed_time(stop) is the device time of
        the call's kernels in ms.
        """
        if not start.cuda_event or not stop.cuda_event:
            raise ValueError("record both events once before passing them")
        self._timed_opts.start_event = start.cuda_event
        self._timed_opts.stop_event = stop.cuda_event
        st = self._fn(self._items, self._n, ctypes.byref(self._timed_opts), _stream(stream))
        if st != 0:
            _check(st, self._name)
        return self.Y


class SpmmCall(SpmmBatchCall):
    """A single prepared product (a batch of one): bsr_spmm_ex with arguments marshalled once."""

    def __init__(self, X: torch.Tensor, W: BSRMatrix, bias: torch.Tensor | None,
                 Y: torch.Tensor, kernel: int | None = None, slices: int | None = None,
                 plan: "BSRPlan | None" = None):
        super().__init__([(X, W, bias, Y)], kernel, slices,
                         plans=None if plan is None else [plan])
        self.Y = Y

    def __call__(self, stream=None) -> torch.Tensor:
        super().__call__(stream)
        return self.Y

    def timed(self, start, stop, stream=None) -> torch.Tensor:
        super().timed(start, stop, stream)
        return self.Y


def bsr_spmm_batched(products, kernel: int | None = None, slices: int | None = None,
                     stream=None, plans=None) -> list:
    """Several products Y_i = X_i W_i^T + bias_i in as few launches as possible.

    `products` is a list of (X, W, bias, Y) with Y allocated by the caller (Y may be None to
    allocate it); `plans` optionally one BSRPlan (or None) per product
    (bsr_spmm_batched_planned).  Returns the list of Y tensors.
    """
    full = []
    for X, W, bias, Y in products:
        if Y is None:
            Y = torch.empty((X.shape[0], W.n_rows), dtype=torch.float32, device=X.device)
        full.append((X, W, bias, Y))
    return SpmmBatchCall(full, kernel, slices, plans=plans)(stream)


def bsr_to_dense(W: BSRMatrix, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Dense fp32 [N, K] expansion of an fp32 BSR matrix."""
    if out is None:
        out = torch.empty((W.n_rows, W.n_cols), dtype=torch.float32, device=W.indptr.device)
    if not isinstance(out, torch.Tensor) or tuple(out.shape) != (W.n_rows, W.n_cols):
        raise ValueError(f"out must be [{W.n_rows}, {W.n_cols}]")
    _require_cuda(out, "out", torch.float32)
    m = W.struct()
    _check(_lib().bsr_to_dense(ctypes.byref(m), _ptr(out), _pitch(out, "out"), _stream(stream)),
           "bsr_to_dense")
    return out


def bsr_iht_update(W: torch.Tensor, G: torch.Tensor, C0: torch.Tensor, eta: float,
                   V: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """V = W - eta (G - C0)^T (bsr_iht_update): W [N, K], G and C0 [K, N], fp32 on the device;
    V may be W itself (in place)."""
    for t, name in ((W, "W"), (G, "G"), (C0, "C0")):
        _require_cuda(t, name, torch.float32)
    if W.dim() != 2:
        raise ValueError("W must be [N, K]")
    N, K = W.shape
    if tuple(G.shape) != (K, N) or tuple(C0.shape) != (K, N):
        raise ValueError(f"G and C0 must be [{K}, {N}]")
    if V is None:
        V = torch.empty((N, K), dtype=torch.float32, device=W.device)
    _require_cuda(V, "V", torch.float32)
    if tuple(V.shape) != (N, K):
        raise ValueError(f"V must be [{N}, {K}]")
    _check(_lib().bsr_iht_update(_ptr(W), _pitch(W, "W"), _ptr(G), _pitch(G, "G"), _ptr(C0),
                                 _pitch(C0, "C0"), float(eta), N, K, _ptr(V), _pitch(V, "V"),
                                 _stream(stream)), "bsr_iht_update")
    return V


def bsr_iht(W0: torch.Tensor, H: torch.Tensor, R: int, C: int, k: int, eta: float, iters: int,
            stream=None, trace: bool = False):
    """Iterative projection for Eq. 2 (Sec. 2.1) on the quadratic loss
    f(W) = 1/2 tr((W - W0) H (W - W0)^T): W_0 = P_k(W0), W_{t+1} = P_k(W_t - eta (W_t - W0) H),
    P_k the block prune keeping k blocks of R x C.  W0: [N, K] fp32; H: [K, K] fp32, symmetric
    (for the reconstruction loss, X^T X / T of calibration activations X).

    Each step runs on the library: G = H W_t^T (bsr_spmm with the BSR iterate), the dense
    iterate (bsr_to_dense), the update (bsr_iht_update, in place) and the prune; C0 = H W0^T is
    one bsr_spmm with W0 stored with all its blocks.  Returns the BSR iterate W_iters; with
    trace, also the list of (V_t, W_t) dense pairs of every step (W_t the iterate the step
    started from, V_t its update before the projection)."""
    _require_cuda(W0, "W0", torch.float32)
    _require_cuda(H, "H", torch.float32)
    if W0.dim() != 2:
        raise ValueError("W0 must be [N, K]")
    N, K = W0.shape
    if tuple(H.shape) != (K, K):
        raise ValueError(f"H must be [{K}, {K}]")
    if R <= 0 or C <= 0 or N % R or K % C:
        raise ValueError("the block shape must divide W0")
    if iters < 0:
        raise ValueError("iters must be >= 0")
    dev = W0.device
    full = bsr_prune_from_dense(W0, R, C, k=(N // R) * (K // C), stream=stream)
    C0 = bsr_spmm(H, full, None, torch.empty((K, N), dtype=torch.float32, device=dev), stream)
    del full
    M = bsr_prune_from_dense(W0, R, C, k=k, stream=stream)
    G = torch.empty((K, N), dtype=torch.float32, device=dev)
    hist = []
    for _ in range(iters):
        bsr_spmm(H, M, None, G, stream)
        Wt = bsr_to_dense(M, stream=stream)
        V = bsr_iht_update(Wt, G, C0, eta, V=Wt.clone() if trace else Wt, stream=stream)
        if trace:
            hist.append((V, Wt))
        M = bsr_prune_from_dense(V, R, C, k=k, stream=stream)
    return (M, hist) if trace else M


def bsr_reblock(W: BSRMatrix, R2: int, C2: int, stream=None) -> BSRMatrix:
    """The same matrix with finer R2 x C2 blocks (R2 | R, C2 | C), in new device tensors."""
    if R2 <= 0 or C2 <= 0 or W.R % R2 or W.C % C2:
        pieces, nb2 = 1, 1
    else:
        pieces, nb2 = (W.R // R2) * (W.C // C2), W.n_rows // R2
    n2 = W.nnzb * pieces
    dev = W.indptr.device
    indptr = torch.empty(nb2 + 1, dtype=torch.int32, device=dev)
    indices = torch.empty(max(n2, 1), dtype=torch.int32, device=dev)
    data = torch.empty((max(n2, 1), max(R2, 1), max(C2, 1)), dtype=W.data.dtype, device=dev)
    m = W.struct()
    _check(_lib().bsr_reblock(ctypes.byref(m), R2, C2, _ptr(indptr), _ptr(indices), _ptr(data),
                              _stream(stream)), "bsr_reblock")
    return BSRMatrix(W.n_rows, W.n_cols, R2, C2, indptr, indices, data, n2)


def _check_attention_shapes(Q, K, V, O, batch: int, seq: int, heads: int, head_dim: int):
    """Every tensor has batch * seq rows and at least heads * head_dim columns (the kernel
    reads and writes exactly that much of each)."""
    for t, n in ((Q, "Q"), (K, "K"), (V, "V"), (O, "O")):
        if (not isinstance(t, torch.Tensor) or t.dim() != 2 or t.shape[0] != batch * seq
                or t.shape[1] < heads * head_dim):
            raise ValueError(f"{n} must be [{batch * seq}, >= {heads * head_dim}]")


def bsr_attention(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, batch: int, seq: int,
                  heads: int, O: torch.Tensor | None = None, scale: float | None = None,
                  stream=None) -> torch.Tensor:
    """Scaled dot-product attention per (sequence, head) of [batch*seq, heads*64] fp32 tensors
    (row pitch from the tensors' strides); returns O."""
    head_dim = 64
    if O is None and isinstance(Q, torch.Tensor):
        O = torch.empty((batch * seq, heads * head_dim), dtype=torch.float32, device=Q.device)
    _check_attention_shapes(Q, K, V, O, batch, seq, heads, head_dim)
    for t, n in ((Q, "Q"), (K, "K"), (V, "V"), (O, "O")):
        _require_cuda(t, n, torch.float32)
    if scale is None:
        scale = head_dim ** -0.5
    _check(_lib().bsr_attention(_ptr(Q), _pitch(Q, "Q"), _ptr(K), _pitch(K, "K"), _ptr(V),
                                _pitch(V, "V"), _ptr(O), _pitch(O, "O"), batch, seq, heads,
                                head_dim, float(scale), _stream(stream)),
           "bsr_attention")
    return O


def _plan_or_none(W: "BSRMatrix") -> "BSRPlan | None":
    """W's native plan, or None for a block shape or dtype without plans."""
    try:
        return bsr_plan_prepare(W)
    except BSRError as e:
        if e.status == 9:   # BSR_ERR_UNSUPPORTED
            return None
        raise


class AttentionBlockCall:
    """The BERT attention block on pruned weights, prepared once and re-issued:
    Q, K, V = three BSR products of X (one bsr_spmm_batched launch), ctx = bsr_attention,
    Y = the O BSR product of ctx.  Buffers are allocated here, on construction; with
    `plans` (the default) every weight whose block shape has per-matrix plans gets its native
    plan here too (same Y, bit for bit, as without; the kernel choice `kernel` must then be
    automatic)."""

    def __init__(self, X: torch.Tensor, Wq: "BSRMatrix", bq, Wk: "BSRMatrix", bk,
                 Wv: "BSRMatrix", bv, Wo: "BSRMatrix", bo, batch: int, seq: int, heads: int,
                 kernel: int | None = None, plans: bool = True):
        T = batch * seq
        dev = X.device
        self.batch, self.seq, self.heads = batch, seq, heads
        self.Q = torch.empty((T, Wq.n_rows), dtype=torch.float32, device=dev)
        self.K = torch.empty((T, Wk.n_rows), dtype=torch.float32, device=dev)
        self.V = torch.empty((T, Wv.n_rows), dtype=torch.float32, device=dev)
        self.ctx = torch.empty((T, heads * 64), dtype=torch.float32, device=dev)
        self.Y = torch.empty((T, Wo.n_rows), dtype=torch.float32, device=dev)
        use = plans and not kernel
        self.plans = [_plan_or_none(W) if use else None for W in (Wq, Wk, Wv, Wo)]
        qkv_plans = self.plans[:3] if any(p is not None for p in self.plans[:3]) else None
        self.qkv = SpmmBatchCall([(X, Wq, bq, self.Q), (X, Wk, bk, self.K), (X, Wv, bv, self.V)],
                                 kernel=kernel, plans=qkv_plans)
        self.out = SpmmCall(self.ctx, Wo, bo, self.Y, kernel=kernel, plan=self.plans[3])
        bsr_attention(self.Q, self.K, self.V, batch, seq, heads, O=self.ctx)   # checks once
        lib = _lib()
        args = (_ptr(self.Q), _pitch(self.Q, "Q"), _ptr(self.K), _pitch(self.K, "K"),
                _ptr(self.V), _pitch(self.V, "V"), _ptr(self.ctx), _pitch(self.ctx, "O"),
                batch, seq, heads, 64, ctypes.c_float(64 ** -0.5))
        self._attn = lambda st: lib.bsr_attention(*args, st)

    def attention(self, stream=None) -> torch.Tensor:
        st = self._attn(_stream(stream))
        if st != 0:
            _check(st, "bsr_attention")
        return self.ctx

    def __call__(self, stream=None) -> torch.Tensor:
        st = _stream(stream)
        self.qkv(st)
        self.attention(st)
        return self.out(st)


def bsr_cast_f32_bf16(src: torch.Tensor, dst: torch.Tensor | None = None,
                      stream=None) -> torch.Tensor:
    """Round a contiguous fp32 tensor to bf16 (nearest, ties to even); returns a bf16 tensor."""
    _require_cuda(src, "src", torch.float32)
    if not src.is_contiguous():
        raise ValueError("src must be contiguous")
    if dst is None:
        dst = torch.empty(src.shape, dtype=torch.bfloat16, device=src.device)
    _require_cuda(dst, "dst", torch.bfloat16)
    if dst.numel() != src.numel() or not dst.is_contiguous():
        raise ValueError("dst must be contiguous with src's element count")
    _check(_lib().bsr_cast_f32_bf16(_ptr(src), _ptr(dst), src.numel(), _stream(stream)),
           "bsr_cast_f32_bf16")
    return dst
