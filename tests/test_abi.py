"""C-ABI checks that need no GPU: exports, host-only entry points and every validation error.

Each error case is built so that validation rejects it before any HIP call, so these run on a
machine without a GPU.  (Fake device pointers are never dereferenced.)
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import bsr_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "libbsr.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2106_08846_amd import bsr as libbsr
    return libbsr.library()


@pytest.fixture(scope="module")
def L():
    from paper_2106_08846_amd import bsr as libbsr
    return libbsr


def declared_symbols():
    text = open(HEADER).read()
    return re.findall(r"LIBBSR_API\s+[\w\s\*]+?\b(bsr_\w+)\s*\(", text)


def test_header_declares_the_binding_exports(L):
    assert sorted(declared_symbols()) == sorted(L.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    names = declared_symbols()
    assert names
    for name in names:
        assert getattr(lib, name) is not None


def test_only_the_abi_is_exported():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only",
                          os.path.join(ROOT, "paper_2106_08846_amd", "libbsr.so")],
                         capture_output=True, text=True, check=True).stdout
    text_syms = sorted(l.split()[-1] for l in out.splitlines() if " T " in l)
    assert text_syms == sorted(declared_symbols())


def test_status_strings(lib):
    for s in range(10):
        assert lib.bsr_status_str(s)
    assert lib.bsr_status_str(0) == b"ok"
    assert lib.bsr_status_str(123) == b"unknown status"


@pytest.mark.parametrize("N,K,R,C,d", [(768, 768, 32, 1, 0.2), (768, 768, 1, 1, 0.1),
                                       (2304, 768, 16, 16, 0.05), (1024, 1024, 32, 32, 0.1),
                                       (64, 64, 16, 16, 0.5 / 16), (64, 64, 8, 8, 0.0),
                                       (64, 64, 8, 8, 1.0), (96, 40, 3, 5, 0.37)])
def test_prune_count_matches_oracle(L, N, K, R, C, d):
    assert L.bsr_prune_count(N, K, R, C, d) == O.prune_count(N, K, R, C, d)


@pytest.mark.parametrize("args,status", [((768, 768, 7, 1, 0.1), 2), ((768, 768, 32, 5, 0.1), 2),
                                         ((0, 768, 32, 1, 0.1), 2), ((64, 64, 8, 8, -0.1), 3),
                                         ((64, 64, 8, 8, 1.5), 3),
                                         ((64, 64, 8, 8, float("nan")), 3)])
def test_prune_count_errors(lib, args, status):
    k = ctypes.c_int64(-1)
    assert lib.bsr_prune_count(*args, ctypes.byref(k)) == status
    assert k.value == -1
    assert lib.bsr_prune_count(64, 64, 8, 8, ctypes.c_double(0.5), None) == 1


def test_prune_workspace_bytes(lib):
    nb = 18432
    expect = ((nb * 8 + 255) // 256 * 256 + nb * 4 + 255) // 256 * 256
    assert lib.bsr_prune_workspace_bytes(768, 768, 32, 1) == expect
    assert lib.bsr_prune_workspace_bytes(768, 768, 7, 1) == 0


FAKE = 0x10000  # never dereferenced: every call below fails validation first
FAKE_Y = 0x20000  # an output address whose range stays clear of FAKE's inputs


def _prune(lib, W=FAKE, N=64, K=64, ldw=64, R=8, C=8, k=6, indptr=FAKE, indices=FAKE,
           data=FAKE, cap=6, ws=FAKE, ws_bytes=1 << 20):
    return lib.bsr_prune_from_dense(W, N, K, ldw, R, C, k, indptr, indices, data, cap, ws,
                                    ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    ({"W": None}, 1), ({"indptr": None}, 1), ({"indices": None}, 1), ({"data": None}, 1),
    ({"R": 7}, 2), ({"C": 3}, 2), ({"ldw": 63}, 2), ({"N": 0}, 2),
    ({"k": -1}, 3), ({"k": 65}, 3),
    ({"cap": 5}, 5),
    ({"ws": None}, 6), ({"ws_bytes": 100}, 6),
])
def test_prune_errors(lib, kw, status):
    assert _prune(lib, **kw) == status


def _matrix(L, N=64, K=64, R=8, C=8, nnzb=6, indptr=FAKE, indices=FAKE, data=FAKE, dtype=0):
    return L.bsr_matrix_t(N, K, R, C, nnzb, indptr, indices, data, dtype)


def _spmm(L, lib, m=None, X=FAKE, x_dtype=0, T=4, ldx=64, Y=FAKE_Y, ldy=64):
    m = m if m is not None else _matrix(L)
    return lib.bsr_spmm(X, x_dtype, T, ldx, ctypes.byref(m), None, Y, ldy, None)


@pytest.mark.parametrize("kw,mkw,status", [
    ({"X": None}, {}, 1), ({"Y": None}, {}, 1),
    ({}, {"indptr": None}, 1), ({}, {"indices": None}, 1), ({}, {"data": None}, 1),
    ({}, {"R": 7}, 2), ({}, {"C": 3}, 2), ({"ldx": 63}, {}, 2), ({"ldy": 63}, {}, 2),
    ({"T": -1}, {}, 2),
    ({}, {"nnzb": -1}, 3), ({}, {"nnzb": 65}, 3), ({"x_dtype": 2}, {}, 3), ({}, {"dtype": 5}, 3),
    ({"x_dtype": 1}, {}, 4), ({}, {"dtype": 1}, 4),
])
def test_spmm_errors(L, lib, kw, mkw, status):
    assert _spmm(L, lib, m=_matrix(L, **mkw), **kw) == status


@pytest.mark.parametrize("where", ["X", "bias", "indptr", "indices", "data"])
def test_spmm_output_overlapping_an_input(L, lib, where):
    """Y's byte range (T x ldy fp32 = 4 x 64 x 4 bytes from 0x100000) overlapping an input is
    BSR_ERR_ARG."""
    Y = 0x100000
    inside, outside = Y + 1000, Y + 4096
    ptrs = {"X": outside, "bias": outside, "indptr": 0x200000, "indices": 0x300000,
            "data": 0x400000}
    ptrs[where] = inside
    m = _matrix(L, indptr=ptrs["indptr"], indices=ptrs["indices"], data=ptrs["data"])
    assert lib.bsr_spmm(ptrs["X"], 0, 4, 64, ctypes.byref(m), ptrs["bias"], Y, 64, None) == 3


def test_spmm_null_matrix(lib):
    assert lib.bsr_spmm(FAKE, 0, 4, 64, None, None, FAKE, 64, None) == 1


def test_spmm_zero_tokens_is_a_noop(L, lib):
    # T = 0 returns before touching the device, even with NULL X and Y.
    assert _spmm(L, lib, X=None, Y=None, T=0) == 0


@pytest.mark.parametrize("mkw,ldo,out,status", [
    ({}, 64, None, 1), ({"dtype": 1}, 64, FAKE, 4), ({}, 63, FAKE, 2), ({"R": 5}, 64, FAKE, 2),
])
def test_to_dense_errors(L, lib, mkw, ldo, out, status):
    m = _matrix(L, **mkw)
    assert lib.bsr_to_dense(ctypes.byref(m), out, ldo, None) == status


@pytest.mark.parametrize("mkw,R2,C2,outs,status", [
    ({}, 4, 4, (None, FAKE, FAKE), 1), ({}, 4, 4, (FAKE, None, FAKE), 1),
    ({}, 4, 4, (FAKE, FAKE, None), 1), ({"indptr": None}, 4, 4, (FAKE, FAKE, FAKE), 1),
    ({}, 3, 4, (FAKE, FAKE, FAKE), 2), ({}, 4, 0, (FAKE, FAKE, FAKE), 2),
    ({}, 16, 8, (FAKE, FAKE, FAKE), 2), ({}, -8, 8, (FAKE, FAKE, FAKE), 2),
    ({"R": 7}, 1, 1, (FAKE, FAKE, FAKE), 2), ({"nnzb": 65}, 4, 4, (FAKE, FAKE, FAKE), 3),
    ({"dtype": 3}, 4, 4, (FAKE, FAKE, FAKE), 3),
    ({"N": 1 << 20, "K": 1 << 20, "R": 64, "C": 64}, 1, 1, (FAKE, FAKE, FAKE), 9),
    ({}, 4, 4, (FAKE, 0x200000, 0x300000), 3),          # indptr_out over W's indptr (FAKE)
    ({}, 4, 4, (0x200000, 0x200000 + 8, 0x300000), 3),  # indices_out inside indptr_out
])
def test_reblock_errors(L, lib, mkw, R2, C2, outs, status):
    m = _matrix(L, **mkw)
    assert lib.bsr_reblock(ctypes.byref(m), R2, C2, *outs, None) == status


def test_cast_errors(lib):
    assert lib.bsr_cast_f32_bf16(FAKE, FAKE, -1, None) == 2
    assert lib.bsr_cast_f32_bf16(None, FAKE, 4, None) == 1
    assert lib.bsr_cast_f32_bf16(FAKE, None, 4, None) == 1
    assert lib.bsr_cast_f32_bf16(None, None, 0, None) == 0


def test_iht_update_errors(lib):
    f = ctypes.c_float
    a = 1 << 20   # three disjoint fake device ranges
    W, G, C0, V = FAKE, FAKE + a, FAKE + 2 * a, FAKE + 3 * a
    ok = dict(W=W, ldw=8, G=G, ldg=4, C0=C0, ldc=4, eta=0.5, N=4, K=8, V=V, ldv=8)

    def call(**kw):
        d = dict(ok, **kw)
        return lib.bsr_iht_update(d["W"], d["ldw"], d["G"], d["ldg"], d["C0"], d["ldc"],
                                  f(d["eta"]), d["N"], d["K"], d["V"], d["ldv"], None)
    assert call(N=-1) == 2 and call(K=-1) == 2
    assert call(ldw=7) == 2 and call(ldv=7) == 2 and call(ldg=3) == 2 and call(ldc=3) == 2
    assert call(eta=float("nan")) == 3 and call(eta=float("inf")) == 3
    assert call(W=None) == 1 and call(G=None) == 1 and call(C0=None) == 1 and call(V=None) == 1
    assert call(V=G) == 3 and call(V=C0 + 16) == 3          # V overlaps G or C0
    assert call(V=W + 4) == 3                                # overlaps W without being W
    assert call(V=W, ldv=9) == 3                             # in place with another pitch
    assert call(N=0) == 0 and call(K=0) == 0                 # empty: no device needed
    assert call(K=65535 * 64 + 1, ldw=65535 * 64 + 1, ldv=65535 * 64 + 1) == 9


def test_python_binding_rejects_cpu_tensors(L):
    import torch
    with pytest.raises(TypeError):
        L.bsr_cast_f32_bf16(torch.zeros(4))


@pytest.mark.parametrize("kernel,slices,start,stop", [
    (4, 0, None, None), (-1, 0, None, None), (0, -1, None, None),
    (0, 0, FAKE, None), (0, 0, None, FAKE),
])
def test_spmm_ex_option_errors(L, lib, kernel, slices, start, stop):
    m = _matrix(L)
    opts = L.bsr_spmm_options_t(kernel, slices, start, stop)
    assert lib.bsr_spmm_ex(FAKE, 0, 4, 64, ctypes.byref(m), None, FAKE, 64, ctypes.byref(opts),
                           None) == 3



def _item(L, m, X=FAKE, x_dtype=0, T=4, ldx=64, Y=FAKE_Y, ldy=64):
    return L.bsr_spmm_item_t(X, x_dtype, T, ldx, ctypes.pointer(m), None, Y, ldy)


def test_spmm_batched_errors(L, lib):
    m = _matrix(L)
    bad = _matrix(L, R=7)
    items = (L.bsr_spmm_item_t * 3)(_item(L, m), _item(L, bad), _item(L, m))
    assert lib.bsr_spmm_batched(items, 3, None, None) == 2      # second item: R does not divide N
    assert lib.bsr_spmm_batched(items, -1, None, None) == 3
    assert lib.bsr_spmm_batched(None, 2, None, None) == 1
    assert lib.bsr_spmm_batched(None, 0, None, None) == 0
    empty = (L.bsr_spmm_item_t * 2)(_item(L, m, X=None, Y=None, T=0), _item(L, m, T=0))
    assert lib.bsr_spmm_batched(empty, 2, None, None) == 0     # nothing to launch
    one_event = L.bsr_spmm_options_t(0, 0, FAKE, None)
    assert lib.bsr_spmm_batched(empty, 2, ctypes.byref(one_event), None) == 3


# ------------------------------------------------------------------ pruning variants (_ex calls)


@pytest.mark.parametrize("N,K,R,C,d", [(768, 768, 32, 1, 0.1), (768, 768, 1, 1, 0.2),
                                       (2304, 768, 16, 16, 0.05), (96, 40, 3, 5, 0.4),
                                       (64, 64, 8, 8, 0.0), (64, 64, 8, 8, 1.0)])
@pytest.mark.parametrize("per_row", [False, True])
def test_prune_count_ex_matches_oracle(L, N, K, R, C, d, per_row):
    assert L.bsr_prune_count(N, K, R, C, d, per_row=per_row) == O.prune_count(
        N, K, R, C, d, per_row=per_row)


def test_prune_count_ex_errors(L, lib):
    k = ctypes.c_int64(-1)
    for norm, sel in [(2, 0), (-1, 0), (0, 2), (0, -1)]:
        opts = L.bsr_prune_options_t(norm, sel)
        assert lib.bsr_prune_count_ex(64, 64, 8, 8, ctypes.c_double(0.5), ctypes.byref(opts),
                                      ctypes.byref(k)) == 3
    opts = L.bsr_prune_options_t(1, 1)
    assert lib.bsr_prune_count_ex(64, 64, 7, 8, ctypes.c_double(0.5), ctypes.byref(opts),
                                  ctypes.byref(k)) == 2
    assert lib.bsr_prune_count_ex(64, 64, 8, 8, ctypes.c_double(1.5), ctypes.byref(opts),
                                  ctypes.byref(k)) == 3
    assert lib.bsr_prune_count_ex(64, 64, 8, 8, ctypes.c_double(0.5), ctypes.byref(opts),
                                  None) == 1
    assert k.value == -1
    assert lib.bsr_prune_count_ex(64, 64, 8, 8, ctypes.c_double(0.5), None, ctypes.byref(k)) == 0
    assert k.value == 32


def _prune_ex(L, lib, norm=0, sel=0, k=6, **kw):
    opts = L.bsr_prune_options_t(norm, sel)
    a = dict(W=FAKE, N=64, K=64, ldw=64, R=8, C=8, indptr=FAKE, indices=FAKE, data=FAKE, cap=64,
             ws=FAKE, ws_bytes=1 << 20)
    a.update(kw)
    return lib.bsr_prune_from_dense_ex(a["W"], a["N"], a["K"], a["ldw"], a["R"], a["C"], k,
                                       a["indptr"], a["indices"], a["data"], a["cap"], a["ws"],
                                       a["ws_bytes"], ctypes.byref(opts), None)


@pytest.mark.parametrize("norm,sel,k,kw,status", [
    (2, 0, 6, {}, 3), (0, 5, 6, {}, 3),          # unknown norm / selection
    (0, 1, 6, {}, 3), (1, 1, 9, {}, 3),          # per-row k not a multiple of Nb = 8
    (0, 1, 8, {"W": None}, 1), (1, 0, 6, {"R": 7}, 2), (0, 1, 72, {}, 3),
    (1, 1, 16, {"cap": 15}, 5), (1, 1, 16, {"ws": None}, 6),
])
def test_prune_ex_errors(L, lib, norm, sel, k, kw, status):
    assert _prune_ex(L, lib, norm, sel, k, **kw) == status


@pytest.mark.parametrize("args,status", [
    # (Q, ldq, K, ldk, V, ldv, O, ldo, batch, seq, heads, head_dim, scale)
    ((None, 128, FAKE, 128, FAKE, 128, FAKE, 128, 1, 4, 2, 64, 0.1), 1),
    ((FAKE, 128, FAKE, 128, FAKE, 128, None, 128, 1, 4, 2, 64, 0.1), 1),
    ((FAKE, 127, FAKE, 128, FAKE, 128, FAKE, 128, 1, 4, 2, 64, 0.1), 2),
    ((FAKE, 128, FAKE, 128, FAKE, 128, FAKE, 100, 1, 4, 2, 64, 0.1), 2),
    ((FAKE, 128, FAKE, 128, FAKE, 128, FAKE, 128, -1, 4, 2, 64, 0.1), 2),
    ((FAKE, 128, FAKE, 128, FAKE, 128, FAKE, 128, 1, 4, 0, 64, 0.1), 2),
    ((FAKE, 128, FAKE, 128, FAKE, 128, FAKE, 128, 1, 4, 2, 64, float("inf")), 3),
    ((FAKE, 128, FAKE, 128, FAKE, 128, FAKE, 128, 1, 4, 4, 32, 0.1), 9),
    ((FAKE + 4, 128, FAKE, 128, FAKE, 128, FAKE, 128, 1, 4, 2, 64, 0.1), 9),
    ((FAKE, 130, FAKE, 128, FAKE, 128, FAKE, 128, 1, 4, 2, 64, 0.1), 9),
    ((None, 128, None, 128, None, 128, None, 128, 0, 4, 2, 64, 0.1), 0),   # no-op
    ((None, 128, None, 128, None, 128, None, 128, 3, 0, 2, 64, 0.1), 0),   # no-op
])
def test_attention_errors(lib, args, status):
    assert lib.bsr_attention(*args, None) == status


# ------------------------------------------- binding: tensor sizes checked before any C call


def _cpu_matrix(L, N=64, K=64, R=8, C=8, nnzb=6, indptr_n=None, indices_n=None, data_n=None,
                data_shape=None):
    import torch
    ip = torch.zeros(indptr_n if indptr_n is not None else N // R + 1, dtype=torch.int32)
    ix = torch.zeros(indices_n if indices_n is not None else nnzb, dtype=torch.int32)
    dshape = data_shape or (data_n if data_n is not None else nnzb, R, C)
    return L.BSRMatrix(N, K, R, C, ip, ix, torch.zeros(dshape), nnzb)


@pytest.mark.parametrize("case", ["x_narrow", "x_column_view", "y_short", "y_narrow",
                                  "bias_short", "indptr_short", "indices_short", "data_short",
                                  "data_block_shape"])
def test_binding_rejects_wrong_sizes(L, case):
    """Each case would read or write past a tensor if it reached the library; the binding
    raises ValueError first (with CPU tensors, so nothing could be enqueued: the device check
    comes after the size checks)."""
    import torch
    W = _cpu_matrix(L)
    X = torch.zeros(4, 64)
    Y = torch.zeros(4, 64)
    bias = None
    if case == "x_narrow":
        X = torch.zeros(4, 63)
    elif case == "x_column_view":
        X = torch.zeros(4, 128)[:, 65:]
    elif case == "y_short":
        Y = torch.zeros(3, 64)
    elif case == "y_narrow":
        Y = torch.zeros(4, 128)[:, 70:]
    elif case == "bias_short":
        bias = torch.zeros(63)
    elif case == "indptr_short":
        W = _cpu_matrix(L, indptr_n=8)
    elif case == "indices_short":
        W = _cpu_matrix(L, indices_n=5)
    elif case == "data_short":
        W = _cpu_matrix(L, data_n=5)
    elif case == "data_block_shape":
        W = _cpu_matrix(L, data_shape=(6, 8, 4))
    with pytest.raises(ValueError):
        L.bsr_spmm(X, W, bias, Y)
    with pytest.raises(ValueError):
        L.SpmmBatchCall([(X, W, bias, Y)])


def test_binding_accepts_right_sizes_then_requires_the_gpu(L):
    import torch
    W = _cpu_matrix(L)
    with pytest.raises(TypeError):   # sizes pass; CPU tensors are then refused
        L.bsr_spmm(torch.zeros(4, 64), W, torch.zeros(64), torch.zeros(4, 64))


def test_binding_to_dense_and_attention_sizes(L):
    import torch
    W = _cpu_matrix(L)
    with pytest.raises(ValueError):
        L.bsr_to_dense(W, out=torch.zeros(63, 64))
    with pytest.raises(ValueError):
        L.bsr_to_dense(W, out=torch.zeros(64, 128)[:, 70:])
    batch, seq, heads = 2, 3, 2
    ok = torch.zeros(batch * seq, heads * 64)
    for bad in (torch.zeros(batch * seq - 1, heads * 64), torch.zeros(batch * seq, 127)):
        for i in range(4):
            args = [ok, ok, ok, ok]
            args[i] = bad
            with pytest.raises(ValueError):
                L.bsr_attention(args[0], args[1], args[2], batch, seq, heads, O=args[3])
    with pytest.raises(TypeError):
        L.bsr_attention(ok, ok, ok, batch, seq, heads, O=torch.zeros(batch * seq, heads * 64))


def test_spmm_batched_rejects_aliasing_between_products(L, lib):
    m = _matrix(L)
    Y0, Y1 = 0x20000, 0x30000           # each Y spans (4 - 1) * 64 + 64 floats = 1 KiB
    chained = (L.bsr_spmm_item_t * 2)(_item(L, m, Y=Y0), _item(L, m, X=Y0 + 64, Y=Y1))
    assert lib.bsr_spmm_batched(chained, 2, None, None) == 3     # product 1 reads product 0's Y
    same_y = (L.bsr_spmm_item_t * 2)(_item(L, m, Y=Y0), _item(L, m, Y=Y0 + 512))
    assert lib.bsr_spmm_batched(same_y, 2, None, None) == 3      # the two outputs overlap
    ws = _matrix(L, data=Y1 + 16)
    into_w = (L.bsr_spmm_item_t * 2)(_item(L, m, Y=Y1), _item(L, ws, Y=Y0))
    assert lib.bsr_spmm_batched(into_w, 2, None, None) == 3      # Y1 covers the other's data
    shared_x = (L.bsr_spmm_item_t * 2)(_item(L, m, Y=Y0), _item(L, m, Y=Y1))
    assert lib.bsr_spmm_batched(shared_x, 2, None, None) not in (1, 2, 3)  # valid: past checks


def test_prune_noalloc_validation(lib):
    """The allocation-free prune checks its arguments like bsr_prune_from_dense and refuses a
    matrix with more blocks than its fixed workspace holds, before touching a device."""
    def call(N=64, K=64, R=8, C=8, k=6, cap=6, W=FAKE, indptr=FAKE, indices=FAKE, data=FAKE):
        return lib.bsr_prune_from_dense_noalloc(W, N, K, K, R, C, k, indptr, indices, data, cap,
                                                None)
    assert call(W=None) == 1
    assert call(R=7) == 2
    assert call(k=65) == 3
    assert call(cap=5) == 5
    big = 1 << 20                                # N * K blocks of 1 x 1: one past the maximum
    assert call(N=1024, K=1025, R=1, C=1, k=10, cap=10) == 6
    assert call(N=1024, K=1025, R=1, C=1, k=10, cap=10, W=None) == 1   # other errors first
    assert call(N=1024, K=1024, R=1, C=1, k=10, cap=10) not in (1, 2, 3, 5, 6)  # fits: past checks
    assert big == 1024 * 1024


def test_plan_validation(L, lib):
    """Plan sizes and preparation are checked on the host before any device work."""
    n = ctypes.c_size_t(0)
    assert lib.bsr_plan_bytes(None, ctypes.byref(n)) == 1
    m = _matrix(L, N=768, K=768, R=32, C=1, nnzb=100)
    assert lib.bsr_plan_bytes(ctypes.byref(m), ctypes.byref(n)) == 0
    units = -(-100 // 8) + 24                       # ceil(nnzb / 8) + block-rows
    assert n.value >= 25 * 4 + units * (32 + 1024)
    mb = _matrix(L, N=768, K=768, R=32, C=1, nnzb=100, dtype=1)
    nb16 = ctypes.c_size_t(0)
    assert lib.bsr_plan_bytes(ctypes.byref(mb), ctypes.byref(nb16)) == 0
    assert nb16.value >= 25 * 4 + (-(-100 // 16) + 24) * (64 + 1024)
    sq = _matrix(L, N=64, K=64, R=16, C=16, nnzb=4)
    assert lib.bsr_plan_bytes(ctypes.byref(sq), ctypes.byref(n)) == 9   # no plan for 16x16
    assert lib.bsr_plan_bytes(ctypes.byref(_matrix(L, R=7)), ctypes.byref(n)) == 2
    plan = L.bsr_plan_t()
    need = lib.bsr_plan_bytes(ctypes.byref(m), ctypes.byref(n)) or n.value
    assert lib.bsr_plan_prepare(ctypes.byref(m), None, need, ctypes.byref(plan), None) == 1
    assert lib.bsr_plan_prepare(ctypes.byref(m), 0x900000, need, None, None) == 1
    assert lib.bsr_plan_prepare(ctypes.byref(m), 0x900000, need - 1, ctypes.byref(plan),
                                None) == 6
    # plan memory overlapping the matrix's data (FAKE is its base)
    assert lib.bsr_plan_prepare(ctypes.byref(m), FAKE - 64, need, ctypes.byref(plan), None) == 3
    # a planned call whose plan describes another matrix, or NULL memory
    other = _matrix(L, N=768, K=768, R=32, C=1, nnzb=100, indices=FAKE + 8)
    plan2 = L.bsr_plan_t(0x900000, need, 768, 768, 100, 32, 1, 0, FAKE, FAKE, FAKE, 8, units,
                         0, 256, 256 + 256 * ((units * 32 + 255) // 256), L.ARITH_NATIVE)
    arr = (ctypes.POINTER(L.bsr_plan_t) * 1)(ctypes.pointer(plan2))
    it = _item(L, other, ldx=768, ldy=768)
    assert lib.bsr_spmm_batched_planned(ctypes.byref(it), arr, 1, None, None) == 3
    plan2.mem = None
    it = _item(L, m, ldx=768, ldy=768)
    assert lib.bsr_spmm_batched_planned(ctypes.byref(it), arr, 1, None, None) == 1
    # a plan struct whose recorded arithmetic names none, or whose layout is not that arithmetic's
    plan2.mem = 0x900000
    for bad in (L.ARITH_AUTO, 7, -1):
        plan2.arith = bad
        assert lib.bsr_spmm_batched_planned(ctypes.byref(it), arr, 1, None, None) == 3
    plan2.arith = L.ARITH_BF16X3                     # the fp32 layout is not the split one
    assert lib.bsr_spmm_batched_planned(ctypes.byref(it), arr, 1, None, None) == 3


def test_plan_arith_validation(L, lib):
    """Plan arithmetic: the split layout's size, and the shapes, dtypes and values refused."""
    n = ctypes.c_size_t(0)
    m = _matrix(L, N=768, K=768, R=32, C=1, nnzb=100)
    assert lib.bsr_plan_bytes_ex(None, L.ARITH_BF16X3, ctypes.byref(n)) == 1
    assert lib.bsr_plan_bytes_ex(ctypes.byref(m), L.ARITH_BF16X3, ctypes.byref(n)) == 0
    units = -(-100 // 16) + 24                      # 16-block units
    assert n.value >= 25 * 4 + units * (32 + 3 * 1024)
    native = ctypes.c_size_t(0)
    assert lib.bsr_plan_bytes_ex(ctypes.byref(m), L.ARITH_NATIVE, ctypes.byref(native)) == 0
    auto = ctypes.c_size_t(0)
    assert lib.bsr_plan_bytes(ctypes.byref(m), ctypes.byref(auto)) == 0
    assert auto.value == native.value               # AUTO is NATIVE
    for bad in (3, -1, 1 << 20):
        assert lib.bsr_plan_bytes_ex(ctypes.byref(m), bad, ctypes.byref(n)) == 3
    mb = _matrix(L, N=768, K=768, R=32, C=1, nnzb=100, dtype=1)
    assert lib.bsr_plan_bytes_ex(ctypes.byref(mb), L.ARITH_BF16X3, ctypes.byref(n)) == 9
    assert lib.bsr_plan_bytes_ex(ctypes.byref(mb), L.ARITH_NATIVE, ctypes.byref(n)) == 0
    # the split plan's 16-bit column offsets reach 4 * 16383 bytes
    wide = _matrix(L, N=64, K=16384, R=32, C=1, nnzb=10)
    assert lib.bsr_plan_bytes_ex(ctypes.byref(wide), L.ARITH_BF16X3, ctypes.byref(n)) == 9
    ok = _matrix(L, N=64, K=16383, R=32, C=1, nnzb=10)
    assert lib.bsr_plan_bytes_ex(ctypes.byref(ok), L.ARITH_BF16X3, ctypes.byref(n)) == 0
    plan = L.bsr_plan_t()
    assert lib.bsr_plan_prepare_ex(ctypes.byref(mb), L.ARITH_BF16X3, 0x900000, 1 << 20,
                                   ctypes.byref(plan), None) == 9
    assert lib.bsr_plan_prepare_ex(ctypes.byref(m), 9, 0x900000, 1 << 20, ctypes.byref(plan),
                                   None) == 3
