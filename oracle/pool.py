"""TEST INFRASTRUCTURE -- CPU oracle of basis pooling.

The paper trains every exact (f, m, s) group on its own, then tests whether
groups with the same (f, m) can share one map: their bases are combined and
eliminated; a single map serves them all when the combined system has no
contradiction and every member learned the same output bits, else each keeps
its own (Sec. 2.1, the paragraph after Eq. 1; the same elimination merges
shard bases, Sec. 2.2).

pool_bases follows that description: for each pool, the basis rows of its
members (in member order, each member's rows in its stored order) form one
row stream that the core oracle fits; the pool is shared when that fit has no
contradiction, every member is a valid consistent context of the same width,
and the members' output masks are equal.  Only the tests, the smoke check and
the benchmark's CPU-baseline leg use it.
"""
from __future__ import annotations

import numpy as np

import oracle

POOL_SHARED, POOL_CONTRADICTION, POOL_WIDTH_MISMATCH, POOL_MASK_MISMATCH, POOL_BAD_MEMBER = 1, 2, 4, 8, 16


class PoolResult:
    def __init__(self, fit, flags, row_off, rows):
        self.fit, self.flags, self.row_off, self.rows = fit, flags, row_off, rows


def pool_bases(ref: "oracle.FitResult", pool_off, members, pooled_n, out_mask=None) -> PoolResult:
    """ref: fitted member contexts; pool p = members[pool_off[p]:pool_off[p+1]];
    pooled_n[p]: the width of pool p; out_mask: uint64 [C*2] or None (all equal)."""
    pool_off = np.asarray(pool_off, np.int64)
    members = np.asarray(members, np.int64)
    P = len(pool_off) - 1
    C = len(ref.n_bits)
    flags = np.zeros(P, np.uint32)
    seg = []
    for p in range(P):
        n = int(pooled_n[p])
        W = int(oracle.feature_words(n)) + 2
        mem = members[pool_off[p]:pool_off[p + 1]]
        bad = any(c < 0 or c >= C for c in mem)
        if not bad:
            bad = any(int(ref.flags[c]) != 0 for c in mem)   # malformed or contradictory member
        width_bad = (not bad) and any(int(ref.n_bits[c]) != n for c in mem)
        mask_bad = False
        if out_mask is not None and len(mem) and not bad:
            m0 = (int(out_mask[2 * mem[0]]), int(out_mask[2 * mem[0] + 1]))
            mask_bad = any((int(out_mask[2 * c]), int(out_mask[2 * c + 1])) != m0 for c in mem)
        rows = []
        if not bad and not width_bad:
            for c in mem:
                _, B, _ = ref.context(int(c))
                rows.extend(B.reshape(-1).tolist())
        seg.append(np.array(rows, np.uint64).reshape(-1) if rows else np.zeros(0, np.uint64))
        flags[p] = (POOL_BAD_MEMBER if bad else 0) | (POOL_WIDTH_MISMATCH if width_bad else 0) | \
                   (POOL_MASK_MISMATCH if mask_bad else 0)
    row_off = np.zeros(P + 1, np.int64)
    row_off[1:] = np.cumsum([len(s) for s in seg])
    rows = np.concatenate(seg) if P and row_off[-1] else np.zeros(0, np.uint64)
    fit = oracle.fit_batch(rows if rows.size else np.zeros(1, np.uint64), row_off, np.asarray(pooled_n, np.int32))
    for p in range(P):
        if fit.flags[p] & oracle.CTX_CONTRADICTION:
            flags[p] |= POOL_CONTRADICTION
        if flags[p] == 0:
            flags[p] = POOL_SHARED
    return PoolResult(fit, flags, row_off, rows)
