"""CPU oracle for batched Monotonic Alignment Search.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``; never by the product package, which
must fail loudly rather than fall back to this code.

The arithmetic lives in ``mas_oracle.c`` (plain C99, Algorithm 1 of the
Super-MAS paper with the readings listed in its header).  This module only
compiles it with gcc and marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mas_oracle.c")
_LIB = os.path.join(_HERE, "libmas_oracle.so")

ITEM_OK, ITEM_EMPTY, ITEM_INFEASIBLE, ITEM_OUT_OF_RANGE = 0, 1, 2, 3

# Strict IEEE evaluation: no contraction into FMA, no fast-math, SSE2 scalar
# float arithmetic (x86-64 default), no flush-to-zero.
CFLAGS = ["-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]


def build(force: bool = True) -> str:
    """Compile the oracle into ``oracle/libmas_oracle.so`` with gcc."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32 = ctypes.c_int32
        lib.oracle_mas_batch_neg.argtypes = [P, i32, i32, i32, P, P, ctypes.c_float, P, P, P]
        lib.oracle_mas_batch_neg.restype = ctypes.c_int
        lib.oracle_durations.argtypes = [P, i32, i32, i32, P]
        lib.oracle_durations.restype = None
        lib.oracle_expand_text.argtypes = [P, P, i32, i32, i32, i32, i32, P]
        lib.oracle_expand_text.restype = ctypes.c_int
        lib.oracle_gauss_loglik_cells.argtypes = [P, P, P, i32, i32, i32, i32, P, ctypes.c_int64, P]
        lib.oracle_gauss_loglik_cells.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def mas(value: np.ndarray, t_x, t_y, *, neg: float = -np.inf):
    """Run the oracle on a batch.

    value: float32 [B, T, S] (C-contiguous); t_x, t_y: int [B].
    Returns (path u8 [B,T,S], score f32 [B], status i32 [B]).
    """
    value = np.ascontiguousarray(value, dtype=np.float32)
    if value.ndim != 3:
        raise ValueError("value must be [B, T, S]")
    B, T, S = value.shape
    tx = np.ascontiguousarray(t_x, dtype=np.int32).reshape(B)
    ty = np.ascontiguousarray(t_y, dtype=np.int32).reshape(B)
    path = np.empty((B, T, S), dtype=np.uint8)
    score = np.empty(B, dtype=np.float32)
    status = np.empty(B, dtype=np.int32)
    rc = _load().oracle_mas_batch_neg(_ptr(value), B, T, S, _ptr(tx), _ptr(ty), float(neg),
                                      _ptr(path), _ptr(score), _ptr(status))
    if rc != 0:
        raise MemoryError("oracle allocation failed")
    return path, score, status


def durations(path: np.ndarray) -> np.ndarray:
    """Row sums of each item's path slab: int32 [B, T]."""
    path = np.ascontiguousarray(path, dtype=np.uint8)
    B, T, S = path.shape
    dur = np.empty((B, T), dtype=np.int32)
    _load().oracle_durations(_ptr(path), B, T, S, _ptr(dur))
    return dur


def row_start(path: np.ndarray, t_x, t_y) -> np.ndarray:
    """First speech column of every text row on each item's path, plus t_y.

    int32 [B, T+1]; entries past t_x are t_y, and invalid items are all 0.
    Derived from the path only (test helper, not part of the method).
    """
    B, T, S = path.shape
    out = np.zeros((B, T + 1), dtype=np.int32)
    for b in range(B):
        tx, ty = int(t_x[b]), int(t_y[b])
        if not (0 < tx <= ty and tx <= T and ty <= S):
            continue
        rows = path[b, :tx, :ty]
        first = rows.argmax(axis=1)
        out[b, :tx] = first
        out[b, tx:] = ty
    return out


def expand_text(path: np.ndarray, h: np.ndarray) -> np.ndarray:
    """Aligned text grid: out[b, j] = the row of h[b] that column j of the
    path selects (zeros where no row does).  path u8 [B, T, S]; h [B, T, C]
    of any fixed-width element type.  Returns [B, S, C] of h's dtype."""
    path = np.ascontiguousarray(path, dtype=np.uint8)
    h = np.ascontiguousarray(h)
    B, T, S = path.shape
    if h.ndim != 3 or h.shape[:2] != (B, T):
        raise ValueError("h must be [B, T, C] with the path's B and T")
    C = h.shape[2]
    out = np.empty((B, S, C), dtype=h.dtype)
    if _load().oracle_expand_text(_ptr(path), _ptr(h), B, T, S, C, h.dtype.itemsize, _ptr(out)) != 0:
        raise ValueError("a path column holds more than one 1")
    return out


def gauss_loglik(mu: np.ndarray, log_sigma: np.ndarray | None, z: np.ndarray, cells: np.ndarray | None = None):
    """log N(z_j; mu_i, sigma_i) summed over channels, in float64.

    mu, log_sigma: f32 [B, T, D] (log_sigma None: unit variance); z: f32
    [B, S, D].  With cells None returns every cell, float64 [B, T, S];
    otherwise cells is int [n, 3] of (b, i, j) and the result is float64 [n].
    """
    mu = np.ascontiguousarray(mu, dtype=np.float32)
    z = np.ascontiguousarray(z, dtype=np.float32)
    ls = None if log_sigma is None else np.ascontiguousarray(log_sigma, dtype=np.float32)
    B, T, D = mu.shape
    S = z.shape[1]
    if z.shape != (B, S, D) or (ls is not None and ls.shape != mu.shape):
        raise ValueError("mu, log_sigma [B, T, D] and z [B, S, D] must agree")
    full = cells is None
    if full:
        b, i, j = np.meshgrid(np.arange(B), np.arange(T), np.arange(S), indexing="ij")
        cells = np.stack([b.ravel(), i.ravel(), j.ravel()], axis=1)
    cells = np.ascontiguousarray(cells, dtype=np.int32).reshape(-1, 3)
    out = np.empty(len(cells), dtype=np.float64)
    if _load().oracle_gauss_loglik_cells(_ptr(mu), _ptr(ls), _ptr(z), B, T, S, D, _ptr(cells), len(cells),
                                         _ptr(out)) != 0:
        raise ValueError("a cell lies outside [B, T, S]")
    return out.reshape(B, T, S) if full else out
