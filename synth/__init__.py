"""Seeded synthetic workloads for the GF(2) affine-map learner.

Thin ctypes wrapper over ``synth/gen.c``.  The module draws data only (widths,
row counts, planted maps, feature vectors, queries); it holds no elimination or
encoding step, so it can feed both the CPU oracle and the GPU library.

Workload recipes (seed ``0xF2A50000 + k`` for recipe k):

* ``1``: one context, 32 drawn input bits plus one reserved bit, 200 rows;
  1,000 queries of which 10% set the reserved bit (out of span).
* ``2``: 4,096 contexts, 16..96 drawn bits plus one reserved bit,
  rows = 2(active+1), 5% of contexts carry one contradictory row;
  1M queries, uniform contexts, 2% out of span.
* ``3``: 80,000 contexts, widths 8+Geometric(1/33) <= 256, lognormal row
  counts (median 30, sigma 1.5, clipped to [1, 4000]), x from a random
  subspace of dimension ceil(0.7 n), 1% contradictory contexts.
* ``4``: 64 contexts of width 4,095, 8,192 uniform rows each.
* ``5``: queries only: Zipf(1.1) contexts of recipe 3, 1% out of span.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libf2synth.so")
_SRC = os.path.join(_HERE, "gen.c")
_lib = None

SEED_BASE = 0xF2A50000
DEFAULT_CTX = {1: 1, 2: 4096, 3: 80000, 4: 64}


def build() -> str:
    """Compile the generator library in place."""
    subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", _SO, _SRC, "-lm"], check=True)
    return _SO


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        L.syn_shapes.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_int32, P, P, P]
        L.syn_rows.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_int32, P, P, P, P, P, P]
        L.syn_queries.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_int32, P, P, P, P, ctypes.c_int64,
                                  ctypes.c_int32, ctypes.c_double, ctypes.c_double, P, P, P]
        for f in (L.syn_shapes, L.syn_rows, L.syn_queries):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def feature_words(n):
    return (np.asarray(n, dtype=np.int64) + 64) // 64


class FitWorkload:
    """Packed training rows of a batch of contexts (all arrays are numpy, host memory)."""

    def __init__(self, recipe, seed, n_bits, m_rows, contra, row_off, rows, contra_row):
        self.recipe = recipe
        self.seed = seed
        self.n_bits = n_bits          # int32 [C]
        self.m_rows = m_rows          # int64 [C]
        self.contra = contra          # uint8 [C], 1 = contradiction injected
        self.row_off = row_off        # int64 [C+1], uint64-word offsets
        self.rows = rows              # uint64 [row_off[-1]]
        self.contra_row = contra_row  # int64 [C], injected row index or -1

    @property
    def num_ctx(self):
        return int(self.n_bits.shape[0])

    @property
    def total_rows(self):
        return int(self.m_rows.sum())

    def row_words(self):
        return feature_words(self.n_bits) + 2


def fit_workload(recipe: int, num_ctx: int | None = None, seed: int | None = None) -> FitWorkload:
    """Training rows for recipe 1-4 (recipe 5 reuses recipe 3's contexts)."""
    base = 3 if recipe == 5 else recipe
    if num_ctx is None:
        num_ctx = DEFAULT_CTX[base]
    if seed is None:
        seed = SEED_BASE + recipe
    L = lib()
    n_bits = np.zeros(num_ctx, np.int32)
    m_rows = np.zeros(num_ctx, np.int64)
    contra = np.zeros(num_ctx, np.uint8)
    if L.syn_shapes(base, seed, num_ctx, _p(n_bits), _p(m_rows), _p(contra)) != 0:
        raise ValueError("bad recipe")
    W = feature_words(n_bits) + 2
    row_off = np.zeros(num_ctx + 1, np.int64)
    np.cumsum(m_rows * W, out=row_off[1:])
    rows = np.zeros(int(row_off[-1]), np.uint64)
    contra_row = np.full(num_ctx, -1, np.int64)
    rc = L.syn_rows(base, seed, num_ctx, _p(n_bits), _p(m_rows), _p(contra), _p(row_off), _p(rows), _p(contra_row))
    if rc != 0:
        raise RuntimeError(f"syn_rows failed ({rc})")
    return FitWorkload(recipe, seed, n_bits, m_rows, contra, row_off, rows, contra_row)


def custom_workload(n_bits, m_rows, rows_list):
    """Pack caller-given rows (list of uint64 arrays of shape [m, fw+2]) into a FitWorkload."""
    n_bits = np.asarray(n_bits, np.int32)
    m_rows = np.asarray(m_rows, np.int64)
    W = feature_words(n_bits) + 2
    row_off = np.zeros(len(n_bits) + 1, np.int64)
    np.cumsum(m_rows * W, out=row_off[1:])
    rows = np.zeros(int(row_off[-1]), np.uint64)
    for c, r in enumerate(rows_list):
        r = np.asarray(r, np.uint64).reshape(-1)
        rows[row_off[c]:row_off[c + 1]] = r
    return FitWorkload(0, 0, n_bits, m_rows, np.zeros(len(n_bits), np.uint8), row_off, rows,
                       np.full(len(n_bits), -1, np.int64))


def queries(wl: FitWorkload, num_queries: int, stride: int, out_frac: float, zipf_s: float = 0.0,
            seed: int | None = None):
    """Query stream over the contexts of ``wl``: returns (ctx_id int32, x uint64 [Q*stride], planted_out uint8)."""
    base = 3 if wl.recipe in (3, 5) else wl.recipe
    if seed is None:
        seed = wl.seed
    L = lib()
    ctx_id = np.zeros(num_queries, np.int32)
    x = np.zeros(num_queries * stride, np.uint64)
    planted = np.zeros(num_queries, np.uint8)
    rc = L.syn_queries(base, seed, wl.num_ctx, _p(wl.n_bits), _p(wl.m_rows), _p(wl.row_off), _p(wl.rows),
                       num_queries, stride, out_frac, zipf_s, _p(ctx_id), _p(x), _p(planted))
    if rc != 0:
        raise RuntimeError(f"syn_queries failed ({rc})")
    return ctx_id, x, planted


# query-stream parameters of each recipe: (num_queries, stride words, out-of-span fraction, zipf exponent)
QUERY_RECIPE = {1: (1000, 1, 0.10, 0.0), 2: (1_000_000, 2, 0.02, 0.0), 5: (100_000_000, 4, 0.01, 1.1)}
