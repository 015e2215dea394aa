"""TEST INFRASTRUCTURE -- CPU oracle of the GF(2) affine-map learner.

ctypes wrapper over ``oracle/f2_oracle.c`` (plain single-threaded C written
from the paper: streaming elimination of Sec. 2.2, encode by reduction of
Sec. 2.3).  Only the tests, the smoke check and the benchmark's CPU-baseline
leg use it; the GPU library never imports, links or calls it.

The oracle lays out its outputs with its own rule (basis capacity
(n+1)(fw+2) words, n+1 pivot entries, 2(n+1) map words per context, packed in
context order) and exposes per-context results as numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# F2ORACLE_LIB may name another build of f2_oracle.c (the sanitizer build of the CPU tests)
_SO = os.environ.get("F2ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "f2_oracle.c")
_lib = None

CTX_CONTRADICTION, CTX_BAD_SEGMENT, CTX_BAD_WIDTH, CTX_BAD_OUTPUT = 1, 2, 4, 8
Q_OUT_OF_SPAN, Q_CTX_CONTRADICTORY, Q_BAD_CTX = 1, 2, 4
MAX_N = 4095


def build() -> str:
    subprocess.run(["gcc", "-O2", "-fPIC", "-shared", "-o", _SO, _SRC], check=True)
    return _SO


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        L.oracle_fit_context.argtypes = [P, i64, ctypes.c_int, P, P, P, P, P]
        L.oracle_fit_context.restype = ctypes.c_int
        L.oracle_reduce_query.argtypes = [P, P, ctypes.c_int, ctypes.c_int, P, P, P]
        L.oracle_reduce_query.restype = ctypes.c_int
        L.oracle_fit_batch.argtypes = [P, i64, P, P, i32, P, i64, P, i64, P, i64, P, P, P, P, P, P, P]
        L.oracle_fit_batch.restype = None
        L.oracle_encode_batch.argtypes = [i32, P, P, P, P, P, P, P, P, P, i32, i64, P, P]
        L.oracle_encode_batch.restype = None
        _lib = L
    return _lib


def _p(a):
    return ctypes.c_void_p(a.ctypes.data)


def feature_words(n):
    return (np.asarray(n, dtype=np.int64) + 64) // 64


def layout(n_bits):
    """Oracle-side output offsets: (basis_off, piv_off, map_off), each int64 [C+1]."""
    n = np.asarray(n_bits, np.int64)
    d = n + 1
    W = feature_words(n) + 2
    offs = []
    for per in (d * W, d, 2 * d):
        o = np.zeros(len(n) + 1, np.int64)
        np.cumsum(per, out=o[1:])
        offs.append(o)
    return tuple(offs)


class FitResult:
    def __init__(self, n_bits, basis_off, piv_off, map_off, basis, pivots, maps, rank, flags, n_contra,
                 first_contra):
        self.n_bits = n_bits
        self.basis_off, self.piv_off, self.map_off = basis_off, piv_off, map_off
        self.basis, self.pivots, self.maps = basis, pivots, maps
        self.rank, self.flags, self.n_contra, self.first_contra = rank, flags, n_contra, first_contra

    def context(self, c):
        """(pivots[rank], basis[rank, fw+2], map[n+1, 2]) of context c."""
        n = int(self.n_bits[c])
        W = int(feature_words(n)) + 2
        r = int(self.rank[c])
        piv = self.pivots[self.piv_off[c]:self.piv_off[c] + r]
        B = self.basis[self.basis_off[c]:self.basis_off[c] + r * W].reshape(r, W)
        M = self.maps[self.map_off[c]:self.map_off[c] + 2 * (n + 1)].reshape(n + 1, 2)
        return piv, B, M


def fit_batch(rows, row_off, n_bits) -> FitResult:
    """Fit every context; rows uint64 [*], row_off int64 [C+1] (words), n_bits int32 [C]."""
    L = lib()
    rows = np.ascontiguousarray(rows, np.uint64)
    row_off = np.ascontiguousarray(row_off, np.int64)
    n_bits = np.ascontiguousarray(n_bits, np.int32)
    C = len(n_bits)
    nb = np.clip(n_bits, 0, MAX_N)
    basis_off, piv_off, map_off = layout(nb)
    basis = np.zeros(max(int(basis_off[-1]), 1), np.uint64)
    pivots = np.full(max(int(piv_off[-1]), 1), -1, np.int32)
    maps = np.zeros(max(int(map_off[-1]), 1), np.uint64)
    rank = np.zeros(C, np.int32)
    flags = np.zeros(C, np.uint32)
    n_contra = np.zeros(C, np.int32)
    first = np.full(C, -1, np.int64)
    L.oracle_fit_batch(_p(rows), rows.size, _p(row_off), _p(n_bits), C, _p(basis_off), int(basis_off[-1]),
                       _p(piv_off), int(piv_off[-1]), _p(map_off), int(map_off[-1]), _p(basis), _p(pivots),
                       _p(maps), _p(rank), _p(flags), _p(n_contra), _p(first))
    return FitResult(n_bits, basis_off, piv_off, map_off, basis, pivots, maps, rank, flags, n_contra, first)


def fit_context(rows_2d, n):
    """Fit one context from rows [m, fw+2]; returns (rank, pivots, basis [rank, W], map [n+1, 2], n_contra, first)."""
    L = lib()
    W = int(feature_words(n)) + 2
    rows_2d = np.ascontiguousarray(np.asarray(rows_2d, np.uint64).reshape(-1, W))
    m = rows_2d.shape[0]
    basis = np.zeros((n + 1) * W, np.uint64)
    piv = np.zeros(n + 1, np.int32)
    M = np.zeros(2 * (n + 1), np.uint64)
    nc = np.zeros(1, np.int32)
    fc = np.zeros(1, np.int64)
    r = L.oracle_fit_context(_p(rows_2d), m, n, _p(basis), _p(piv), _p(M), _p(nc), _p(fc))
    return r, piv[:r].copy(), basis[:r * W].reshape(r, W).copy(), M.reshape(n + 1, 2), int(nc[0]), int(fc[0])


def reduce_query(pivots, basis_2d, n, q_words):
    """Reduce an explicit feature vector (fw words incl. the constant bit as given): (in_span, acc[2], residual[fw])."""
    L = lib()
    fw = int(feature_words(n))
    piv = np.ascontiguousarray(pivots, np.int32)
    B = np.ascontiguousarray(basis_2d, np.uint64).reshape(-1)
    q = np.ascontiguousarray(q_words, np.uint64).reshape(fw)
    acc = np.zeros(2, np.uint64)
    res = np.zeros(fw, np.uint64)
    if B.size == 0:
        B = np.zeros(1, np.uint64)
    if piv.size == 0:
        piv = np.zeros(1, np.int32)
    ok = L.oracle_reduce_query(_p(B), _p(piv), len(pivots), n, _p(q), _p(acc), _p(res))
    return bool(ok), acc, res


def encode_batch(fit: FitResult, ctx_id, x, stride):
    """Encode queries against a FitResult: returns (words uint64 [Q, 2], qflags uint8 [Q])."""
    L = lib()
    ctx_id = np.ascontiguousarray(ctx_id, np.int32)
    x = np.ascontiguousarray(x, np.uint64)
    Q = len(ctx_id)
    words = np.zeros(2 * max(Q, 1), np.uint64)
    qf = np.zeros(max(Q, 1), np.uint8)
    if Q:
        L.oracle_encode_batch(len(fit.n_bits), _p(fit.n_bits), _p(fit.basis_off), _p(fit.piv_off), _p(fit.basis),
                              _p(fit.pivots), _p(fit.rank), _p(fit.flags), _p(ctx_id), _p(x), stride, Q,
                              _p(words), _p(qf))
    return words[:2 * Q].reshape(Q, 2), qf[:Q]
