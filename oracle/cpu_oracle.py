"""ctypes loader for the plain C oracle (cpu_oracle.c).

TEST INFRASTRUCTURE ONLY: used by the tests and by the CPU-baseline timing leg of the benchmark.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "cpu_oracle.c")
LIBRARY = os.path.join(_HERE, "libcpu_oracle.so")


def build(verbose: bool = False) -> str:
    """Compile cpu_oracle.c into libcpu_oracle.so with gcc (plain -O2, OpenMP, no fast-math)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
           "-std=c11", "-Wall", "-Wextra", SOURCE, "-o", LIBRARY + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIBRARY + ".tmp", LIBRARY)
    return LIBRARY


_lib = None


def load() -> ctypes.CDLL:
    """Load libcpu_oracle.so, building it first if it is absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            build()
        lib = ctypes.CDLL(LIBRARY)
        i64, i32, p = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        lib.oracle_num_threads.restype = ctypes.c_int
        lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
        lib.oracle_block_keys.argtypes = [p, i64, i64, i64, i32, i32, p]
        lib.oracle_spmm.argtypes = [p, i64, i64, i64, p, p, p, i32, i32, i64, p, p]
        _lib = lib
    return _lib


def num_threads() -> int:
    return int(load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    load().oracle_set_num_threads(int(n))


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def block_keys(W: np.ndarray, R: int, C: int) -> np.ndarray:
    W = np.ascontiguousarray(W, dtype=np.float32)
    N, K = W.shape
    key = np.empty((N // R) * (K // C), dtype=np.float64)
    load().oracle_block_keys(_ptr(W), N, K, K, R, C, _ptr(key))
    return key


def spmm(X: np.ndarray, indptr, indices, data, N: int, bias=None) -> np.ndarray:
    """fp64 Y = X W^T + b over the stored blocks (plain loops, OpenMP over tokens)."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    T, K = X.shape
    indptr = np.ascontiguousarray(indptr, dtype=np.int32)
    indices = np.ascontiguousarray(indices, dtype=np.int32)
    data = np.ascontiguousarray(data, dtype=np.float32)
    R, C = data.shape[1], data.shape[2]
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    Y = np.empty((T, N), dtype=np.float64)
    load().oracle_spmm(_ptr(X), T, K, K, _ptr(indptr), _ptr(indices), _ptr(data), R, C, N,
                       _ptr(b), _ptr(Y))
    return Y
