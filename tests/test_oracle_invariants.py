"""Oracle invariants on seeded workloads shaped like the benchmark recipes.

* planted recovery: full-rank contexts recover the planted [W | b] exactly; on
  rank-deficient ones every basis pair satisfies r_k W = z_k (App. C basis-pair
  invariant) and the canonical map agrees with W on the span;
* flag <=> injected contradiction, with the injected row reported first;
* every training row is reproduced by the fitted map (Eq. 9);
* the basis is fully reduced and rank <= min(m, n+1);
* consistent contexts give the same result in any row order (uniqueness of
  the reduced basis);
* resume: fitting [basis of a prefix ++ remaining rows] equals the full fit
  (Sec. 2.2, merging of retained rows);
* generated queries: unsupported exactly when built outside the span, and the
  word of an in-span combination equals the XOR of the combined outputs.
"""
import numpy as np
import pytest

import oracle
import synth


def ints(words):
    return [int(w) for w in words]


def gf2_apply(Wbits, feat_bits):
    """XOR of the rows of W selected by the set bits (plain definition of Eq. 2)"""
    y = np.zeros(2, np.uint64)
    for j in np.nonzero(feat_bits)[0]:
        y ^= Wbits[j]
    return y


def unpack_bits(words, nbits):
    out = np.zeros(nbits, np.uint8)
    for i in range(nbits):
        out[i] = (int(words[i // 64]) >> (i % 64)) & 1
    return out


def planted_rows(rng, n, m, sub_dim=None):
    d = n + 1
    fw = (n + 64) // 64
    Wp = rng.integers(0, 2 ** 63, size=(d, 2), dtype=np.uint64) ^ (rng.integers(0, 2, size=(d, 2), dtype=np.uint64) << np.uint64(63))
    if sub_dim is not None:
        U = rng.integers(0, 2, size=(sub_dim, n), dtype=np.uint8)
    rows = np.zeros((m, fw + 2), np.uint64)
    feats = np.zeros((m, d), np.uint8)
    for i in range(m):
        if sub_dim is None:
            x = rng.integers(0, 2, size=n, dtype=np.uint8)
        else:
            s = rng.integers(0, 2, size=sub_dim, dtype=np.uint8)
            x = (s @ U) % 2 if sub_dim else np.zeros(n, np.uint8)
        f = np.concatenate([x, [1]]).astype(np.uint8)
        feats[i] = f
        for b in np.nonzero(f)[0]:
            rows[i, b // 64] |= np.uint64(1) << np.uint64(b % 64)
        rows[i, fw:] = gf2_apply(Wp, f)
    return rows, feats, Wp


@pytest.mark.parametrize("n", [0, 1, 7, 33, 63, 64, 100, 200])
def test_planted_full_rank_recovery(n):
    rng = np.random.default_rng(n)
    d = n + 1
    rows, feats, Wp = planted_rows(rng, n, 3 * d + 8)
    r, piv, B, M, nc, fc = oracle.fit_context(rows, n)
    assert r == d and nc == 0 and fc == -1
    assert np.array_equal(M, Wp)


@pytest.mark.parametrize("n,k", [(10, 4), (40, 28), (130, 91)])
def test_planted_rank_deficient(n, k):
    rng = np.random.default_rng(100 + n)
    rows, feats, Wp = planted_rows(rng, n, 2 * n, sub_dim=k)
    r, piv, B, M, nc, fc = oracle.fit_context(rows, n)
    assert r <= k + 1 and nc == 0
    fw = (n + 64) // 64
    for i in range(r):
        rb = unpack_bits(B[i, :fw], n + 1)
        assert np.array_equal(gf2_apply(Wp, rb), B[i, fw:])          # r_k W = z_k
        assert np.array_equal(gf2_apply(M, rb), B[i, fw:])           # canonical map agrees on the basis
    # span elements: random XOR combinations of training feature rows
    for _ in range(50):
        sel = rng.integers(0, 2, size=len(feats)).astype(bool)
        f = feats[sel].sum(axis=0) % 2
        assert np.array_equal(gf2_apply(M, f), gf2_apply(Wp, f))


def _check_context(wl, fit, c):
    n = int(wl.n_bits[c])
    fw = (n + 64) // 64
    W = fw + 2
    m = int(wl.m_rows[c])
    piv, B, M = fit.context(c)
    r = int(fit.rank[c])
    assert r <= min(m, n + 1)
    # fully reduced: each pivot column is set only in its own row
    for i, p in enumerate(int(v) for v in piv):
        col = [(int(B[k, p // 64]) >> (p % 64)) & 1 for k in range(r)]
        assert col == [int(k == i) for k in range(r)]
    injected = bool(wl.contra[c]) and m >= 2
    assert bool(fit.flags[c] & oracle.CTX_CONTRADICTION) == injected
    if injected:
        assert fit.n_contra[c] == 1 and fit.first_contra[c] == wl.contra_row[c]
    rows = wl.rows[wl.row_off[c]:wl.row_off[c + 1]].reshape(m, W)
    for i in range(m):
        if injected and i == wl.contra_row[c]:
            continue
        ok, acc, res = oracle.reduce_query(piv, B, n, rows[i, :fw])
        assert ok and np.array_equal(acc, rows[i, fw:]), (c, i)


@pytest.mark.parametrize("recipe,num_ctx", [(1, 1), (2, 300), (3, 1500)])
def test_generated_workload_invariants(recipe, num_ctx):
    wl = synth.fit_workload(recipe, num_ctx=num_ctx)
    fit = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    for c in range(wl.num_ctx):
        _check_context(wl, fit, c)
    if recipe in (1, 2):
        # reserved top bit is never observed: rank = active bits + constant
        assert np.all(fit.rank == wl.n_bits)


def test_recipe4_context_full_rank():
    wl = synth.fit_workload(4, num_ctx=1)
    fit = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    assert fit.rank[0] == 4096 and fit.flags[0] == 0


def test_shuffle_invariance_consistent():
    wl = synth.fit_workload(3, num_ctx=200)
    rng = np.random.default_rng(9)
    for c in range(wl.num_ctx):
        if wl.contra[c]:
            continue
        n = int(wl.n_bits[c])
        W = (n + 64) // 64 + 2
        rows = wl.rows[wl.row_off[c]:wl.row_off[c + 1]].reshape(-1, W)
        a = oracle.fit_context(rows, n)
        b = oracle.fit_context(rows[rng.permutation(len(rows))], n)
        assert a[0] == b[0] and np.array_equal(a[1], b[1]) and np.array_equal(a[2], b[2]) and np.array_equal(a[3], b[3])


@pytest.mark.parametrize("recipe", [2, 3])
def test_resume_from_basis(recipe):
    wl = synth.fit_workload(recipe, num_ctx=150)
    rng = np.random.default_rng(recipe)
    for c in range(wl.num_ctx):
        n = int(wl.n_bits[c])
        W = (n + 64) // 64 + 2
        rows = wl.rows[wl.row_off[c]:wl.row_off[c + 1]].reshape(-1, W)
        m = len(rows)
        cut = int(rng.integers(0, m + 1))
        full = oracle.fit_context(rows, n)
        pre = oracle.fit_context(rows[:cut], n)
        resumed = oracle.fit_context(np.concatenate([pre[2], rows[cut:]]), n)
        assert full[0] == resumed[0]
        assert np.array_equal(full[1], resumed[1]) and np.array_equal(full[2], resumed[2])
        assert np.array_equal(full[3], resumed[3])
        assert full[4] == pre[4] + resumed[4]


@pytest.mark.parametrize("recipe,num_ctx,nq,stride,frac,zipf", [(1, 1, 1000, 1, 0.1, 0.0), (2, 200, 20000, 2, 0.02, 0.0),
                                                                  (3, 2000, 20000, 4, 0.01, 1.1)])
def test_generated_queries(recipe, num_ctx, nq, stride, frac, zipf):
    wl = synth.fit_workload(recipe, num_ctx=num_ctx)
    fit = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    ctx, x, planted = synth.queries(wl, nq, stride, frac, zipf)
    words, qf = oracle.encode_batch(fit, ctx, x, stride)
    assert np.array_equal((qf & oracle.Q_OUT_OF_SPAN) != 0, planted != 0)
    assert np.array_equal((qf & oracle.Q_CTX_CONTRADICTORY) != 0, (fit.flags[ctx] & oracle.CTX_CONTRADICTION) != 0)
    assert 0.5 * frac < planted.mean() < 1.5 * frac + 0.01
    # linearity on the span: XOR of three training rows encodes to the XOR of their outputs
    rng = np.random.default_rng(recipe)
    cs, xs, want = [], [], []
    for _ in range(300):
        c = int(rng.integers(0, wl.num_ctx))
        if wl.contra[c] or wl.m_rows[c] == 0:
            continue
        n = int(wl.n_bits[c])
        W = (n + 64) // 64 + 2
        rows = wl.rows[wl.row_off[c]:wl.row_off[c + 1]].reshape(-1, W)
        pick = rows[rng.integers(0, len(rows), size=3)]
        f = pick[0] ^ pick[1] ^ pick[2]
        xv = np.zeros(stride, np.uint64)
        xv[:min(stride, W - 2)] = f[:min(stride, W - 2)]
        if n // 64 < stride:
            xv[n // 64] &= ~(np.uint64(1) << np.uint64(n % 64))
        cs.append(c)
        xs.append(xv)
        want.append(f[W - 2:])
    w2, q2 = oracle.encode_batch(fit, np.array(cs, np.int32), np.concatenate(xs), stride)
    assert np.all(q2 & oracle.Q_OUT_OF_SPAN == 0)
    assert np.array_equal(w2, np.array(want))


def test_generator_prefix_stability():
    a = synth.fit_workload(3, num_ctx=50)
    b = synth.fit_workload(3, num_ctx=120)
    assert np.array_equal(a.n_bits, b.n_bits[:50]) and np.array_equal(a.rows, b.rows[:a.rows.size])
