"""GPU parity of basis pooling (f2_pool_bases) against the pooling oracle
(oracle/pool.py): pooled bases, pivots, maps, parity rows, ranks and flags bit
for bit, and the per-pool flags."""
import numpy as np
import pytest

import oracle
from oracle import pool as PL
import parity
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def f2(require_gpu):
    from paper_2608_20532_amd import f2gpu
    return f2gpu


def _pool_and_compare(f2, wl, pool_off, members, pooled_n, out_mask=None):
    import torch
    ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    model = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    parity.compare_fit(model, ref)
    exp = PL.pool_bases(ref, pool_off, members, pooled_n, out_mask)
    mem = np.asarray(members, np.int32)
    pooled, flags = f2.pool(model, parity.to_dev(np.asarray(pool_off, np.int64)),
                            parity.to_dev(mem if mem.size else np.zeros(1, np.int32))[:len(mem)],
                            np.asarray(pooled_n, np.int32),
                            parity.to_dev(np.asarray(out_mask, np.uint64)) if out_mask is not None else None)
    torch.cuda.synchronize()
    got = parity.host(flags, np.uint32)[:len(pooled_n)]
    assert np.array_equal(got, exp.flags), (got, exp.flags)
    # fitted pools (rows present) match the oracle's fit of the concatenated bases
    parity.compare_fit(pooled, exp.fit)
    return exp


def test_pool_shards_of_recipe3_contexts(f2):
    """Each of 3000 recipe-3 contexts split into 3 shard contexts (stream order kept); the
    shard bases pooled back equal the fit of the whole context."""
    wl0 = synth.fit_workload(3, num_ctx=3000)
    n_bits, rows_list = [], []
    for c in range(wl0.num_ctx):
        n = int(wl0.n_bits[c]); W = (n + 64) // 64 + 2
        rows = wl0.rows[wl0.row_off[c]:wl0.row_off[c + 1]].reshape(-1, W)
        for part in np.array_split(rows, 3):
            n_bits.append(n)
            rows_list.append(part)
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    C0 = wl0.num_ctx
    pool_off = np.arange(0, 3 * C0 + 1, 3, dtype=np.int64)
    exp = _pool_and_compare(f2, wl, pool_off, np.arange(3 * C0), wl0.n_bits)
    whole = oracle.fit_batch(wl0.rows, wl0.row_off, wl0.n_bits)
    consistent = (whole.flags == 0)
    # members of a contradictory context may be contradictory themselves: compare where all is consistent
    ok = consistent & (exp.flags == PL.POOL_SHARED)
    assert ok.sum() > 0.95 * C0
    assert np.array_equal(exp.fit.rank[ok], whole.rank[ok])


def test_pool_shared_and_contradictory_maps_all_widths(f2):
    rng = np.random.default_rng(7)
    n_bits, rows_list, pool_off, members, pooled_n = [], [], [0], [], []
    c = 0
    for n in (3, 40, 63, 64, 100, 190, 300, 520, 700):
        fw = (n + 64) // 64
        Wm = rng.integers(0, 2 ** 63, size=(n + 1, 2), dtype=np.uint64)
        for variant in range(2):   # variant 1: one member uses a different map on one coordinate
            start = c
            for k in range(3):
                m = int(rng.integers(5, 2 * n + 10))
                X = rng.integers(0, 2 ** 63, size=(m, fw), dtype=np.uint64)
                X[:, fw - 1] &= np.uint64((1 << ((n % 64))) - 1) if n % 64 else np.uint64(0)
                X[:, n // 64] |= np.uint64(1) << np.uint64(n % 64)        # the constant
                if k:   # later members see only a subspace: clear a band of coordinates
                    X[:, 0] &= np.uint64(0xFFFFFFFF00000000) if k == 1 else np.uint64(0x00000000FFFFFFFF) | (np.uint64(1) << np.uint64(n % 64) if n < 64 else np.uint64(0))
                Wk = Wm.copy()
                if variant == 1 and k == 2:
                    Wk[1, 0] ^= np.uint64(1)
                Y = np.zeros((m, 2), np.uint64)
                bits = np.unpackbits(X.view(np.uint8), axis=1, bitorder="little")[:, :n + 1].astype(bool)
                for h in range(2):
                    Y[:, h] = np.bitwise_xor.reduce(np.where(bits, Wk[:, h][None, :], np.uint64(0)), axis=1)
                rows = np.concatenate([X, Y], axis=1)
                n_bits.append(n)
                rows_list.append(rows)
                c += 1
            members.extend(range(start, c))
            pool_off.append(len(members))
            pooled_n.append(n)
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    exp = _pool_and_compare(f2, wl, pool_off, members, pooled_n)
    assert (exp.flags == PL.POOL_SHARED).sum() >= 8 and (exp.flags & PL.POOL_CONTRADICTION).any()


def test_pool_flags_masks_bad_members_and_overflow(f2):
    rng = np.random.default_rng(9)
    wl0 = synth.fit_workload(2, num_ctx=12)
    n_bits = wl0.n_bits.copy()
    # pools: width or mask mismatch, out-of-range id, contradictory member, empty pool, self pool
    import torch
    ref0 = oracle.fit_batch(wl0.rows, wl0.row_off, wl0.n_bits)
    cc = int(np.nonzero(ref0.flags == oracle.CTX_CONTRADICTION)[0][0]) if (ref0.flags == oracle.CTX_CONTRADICTION).any() else None
    good = [c for c in range(12) if ref0.flags[c] == 0]
    a, b = good[0], good[1]
    mask = np.tile(np.array([ALLW, ALLW], np.uint64), 12)
    mask[2 * b] = np.uint64(5)
    pools = [[a, b], [a, a], [a, 99], [a], [], [b]]
    pooled_n = [int(n_bits[a]), int(n_bits[a]), int(n_bits[a]), int(n_bits[a]), 7, int(n_bits[b])]
    if cc is not None:
        pools.append([cc])
        pooled_n.append(int(n_bits[cc]))
    pool_off = np.cumsum([0] + [len(p) for p in pools])
    members = [m for p in pools for m in p]
    exp = _pool_and_compare(f2, wl0, pool_off, members, pooled_n, mask)
    assert exp.flags[2] == PL.POOL_BAD_MEMBER and exp.flags[4] == PL.POOL_SHARED
    # one context in many pools: past the row buffer (which holds every member basis
    # once) every pool is flagged and fitted from no rows
    big = max(good, key=lambda c: int(n_bits[c]))
    pool_off = np.arange(0, 25, 4, dtype=np.int64)
    members = np.array([big] * 24, np.int32)
    W = (int(n_bits[big]) + 64) // 64 + 2
    model = parity.gpu_fit(f2, wl0.rows, wl0.row_off, wl0.n_bits)
    pooled, flags = f2.pool(model, parity.to_dev(pool_off), parity.to_dev(members), np.array([int(n_bits[big])] * 6, np.int32))
    torch.cuda.synchronize()
    got = parity.host(flags, np.uint32)[:6]
    need = 24 * int(ref0.rank[big]) * W
    assert need > int(model.basis_off_host[-1])
    assert (got == PL.POOL_BAD_MEMBER).all() and (parity.host(pooled.rank, np.int32)[:6] == 0).all()


def test_pool_many_members_per_pool(f2):
    """Pools of 70 to 150 members (more than the 64 members the copy takes at a time),
    each the shards of one long recipe-3 context, against the pooling oracle."""
    wl0 = synth.fit_workload(3, num_ctx=20000)
    long_ctx = [c for c in range(wl0.num_ctx) if wl0.m_rows[c] >= 300][:24]
    assert len(long_ctx) == 24
    rng = np.random.default_rng(13)
    n_bits, rows_list, pool_off, pooled_n = [], [], [0], []
    for c in long_ctx:
        n = int(wl0.n_bits[c]); W = (n + 64) // 64 + 2
        rows = wl0.rows[wl0.row_off[c]:wl0.row_off[c + 1]].reshape(-1, W)
        k = int(rng.integers(70, 151))
        for part in np.array_split(rows, k):
            n_bits.append(n)
            rows_list.append(part)
        pool_off.append(pool_off[-1] + k)
        pooled_n.append(n)
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    exp = _pool_and_compare(f2, wl, np.asarray(pool_off, np.int64), np.arange(wl.num_ctx), pooled_n)
    assert (exp.flags != PL.POOL_BAD_MEMBER).sum() > 12


def test_pool_more_than_a_thousand_offset_blocks(f2):
    """270,000 pools (the row-offset scan runs over 1,055 blocks of 256 pools, more than
    one chunk of 1,024), each the two halves of a small consistent context: every pool
    is shared and its fit equals the oracle's fit of the whole context."""
    import torch
    rng = np.random.default_rng(17)
    P, n, m = 270_000, 12, 4
    X = rng.integers(0, 1 << n, size=(P, m), dtype=np.uint64) | (np.uint64(1) << np.uint64(n))
    Wm = rng.integers(0, 2 ** 63, size=(P, n + 1, 2), dtype=np.uint64)
    Y = np.zeros((P, m, 2), np.uint64)
    for b in range(n + 1):  # y = W phi over GF(2): consistent, no contradiction
        sel = ((X >> np.uint64(b)) & np.uint64(1)).astype(bool)
        Y ^= np.where(sel[:, :, None], Wm[:, b][:, None, :], np.uint64(0))
    rows = np.ascontiguousarray(np.concatenate([X[:, :, None], Y], axis=2)).reshape(-1)  # P contexts of m rows
    W = 3                                                                # words per row (n < 63)
    # the members: each context's two halves, consecutive segments of the same rows
    model = parity.gpu_fit(f2, rows, np.arange(2 * P + 1, dtype=np.int64) * (m // 2) * W, np.full(2 * P, n, np.int32))
    pooled, flags = f2.pool(model, parity.to_dev(np.arange(0, 2 * P + 1, 2, dtype=np.int64)),
                            parity.to_dev(np.arange(2 * P, dtype=np.int32)), np.full(P, n, np.int32))
    torch.cuda.synchronize()
    assert (parity.host(flags, np.uint32)[:P] == PL.POOL_SHARED).all()
    parity.compare_fit(pooled, oracle.fit_batch(rows, np.arange(P + 1, dtype=np.int64) * m * W, np.full(P, n, np.int32)))


ALLW = 2 ** 64 - 1
