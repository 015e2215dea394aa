"""TEST INFRASTRUCTURE -- CPU oracle of interleaved-stream ingestion.

Plain Python, one row at a time; only the tests and the benchmark's CPU-baseline
leg use it.

group_rows -- the observations of a corpus arrive as one stream in which the
    rows of many contexts are mixed (Sec. 3 gathers them across CUBINs); the
    streaming elimination of Sec. 2.2 takes each context's rows in stream order,
    because which row of a dependent set is kept depends on that order.  Each
    row is appended, trimmed to its context's row width (fw + 2 words), to its
    context's list; rows of a context id out of range, of a width outside
    [0, MAX_N], or whose row width exceeds the stride are dropped.  The output
    is the concatenation of the lists in context order with the word offsets
    of each context (the fit's row_off).
"""
from __future__ import annotations

import numpy as np

MAX_N = 4095


def group_rows(ctx_id, rows, stride: int, n_bits):
    """Returns (rows_out uint64 [words], row_off int64 [C + 1], dropped)."""
    ctx_id = np.asarray(ctx_id, np.int64).reshape(-1)
    rows = np.asarray(rows, np.uint64).reshape(-1, stride) if len(ctx_id) else np.zeros((0, stride), np.uint64)
    n_bits = [int(n) for n in np.asarray(n_bits).reshape(-1)]
    C = len(n_bits)
    lists = [[] for _ in range(C)]
    dropped = 0
    for r in range(len(ctx_id)):
        c = int(ctx_id[r])
        if c < 0 or c >= C or n_bits[c] < 0 or n_bits[c] > MAX_N:
            dropped += 1
            continue
        W = (n_bits[c] + 64) // 64 + 2
        if W > stride:
            dropped += 1
            continue
        lists[c].append(rows[r, :W])
    row_off = np.zeros(C + 1, np.int64)
    parts = []
    for c in range(C):
        W = (n_bits[c] + 64) // 64 + 2 if 0 <= n_bits[c] <= MAX_N else 0
        row_off[c + 1] = row_off[c] + len(lists[c]) * W
        parts.extend(lists[c])
    out = np.concatenate(parts) if parts else np.zeros(0, np.uint64)
    return out.astype(np.uint64), row_off, dropped
