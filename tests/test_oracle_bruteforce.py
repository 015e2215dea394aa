"""Oracle against brute force and an independent elimination, on tiny systems.

Brute force (pure Python sets over all XOR combinations, Eqs. 6-9):
  * kept rows are the rows outside the span of all earlier rows;
  * T is the unique linear map on that span with T(phi_i) = y_i on kept rows;
  * a contradiction is a non-kept row with y_i != T(phi_i);
  * the reduced basis row of pivot p is the unique span vector whose highest
    priority bit is p and which is zero on every other pivot column;
  * every query q in F2^d: supported iff q in the span, word = T(q).

Independent algorithm: column-scan elimination (numpy boolean matrices) that
picks, for each column in priority order, the earliest remaining row as pivot
and only adds earlier rows into later ones, then back-substitutes.
"""
import numpy as np
import pytest

import oracle


def prio(n):
    """storage bits in descending priority: x_{n-1} .. x_0, then the constant (bit n)"""
    return list(range(n - 1, -1, -1)) + [n]


def top_bit(v, n):
    for s in prio(n):
        if (v >> s) & 1:
            return s
    return -1


def brute(n, feats, ys):
    d = n + 1
    S = {0: 0}   # span element -> T value (built from kept rows only)
    kept, contra = [], []
    for i, (f, y) in enumerate(zip(feats, ys)):
        if f in S:
            if S[f] != y:
                contra.append(i)
        else:
            kept.append(i)
            S.update({s ^ f: t ^ y for s, t in list(S.items())})
    P = sorted({top_bit(v, n) for v in S if v}, key=lambda s: prio(n).index(s))
    pmask = sum(1 << p for p in P)
    basis = []
    for p in P:
        cands = [v for v in S if v and top_bit(v, n) == p and (v & pmask) == (1 << p)]
        assert len(cands) == 1
        basis.append((p, cands[0], S[cands[0]]))
    return kept, contra, S, basis


def randbits(rng, k):
    return int.from_bytes(rng.bytes((k + 7) // 8), "little") & ((1 << k) - 1)


def rand_system(rng, n, m, mode):
    d = n + 1
    Wp = [randbits(rng, 128) for _ in range(d)]
    # feature vectors from a random low-dimensional pool so that dependencies are frequent
    pool = [randbits(rng, d) for _ in range(max(1, int(rng.integers(1, d + 2))))]
    feats, ys = [], []
    for _ in range(m):
        f = 0
        for p in pool:
            if rng.integers(0, 2):
                f ^= p
        if rng.random() < 0.1:
            f = 0
        y = 0
        for j in range(d):
            if (f >> j) & 1:
                y ^= Wp[j]
        if mode == "noisy" and rng.random() < 0.3:
            y ^= 1 << int(rng.integers(0, 128))
        feats.append(f)
        ys.append(y)
    return feats, ys


def pack(n, feats, ys, rng=None):
    fw = (n + 64) // 64
    rows = np.zeros((len(feats), fw + 2), np.uint64)
    for i, (f, y) in enumerate(zip(feats, ys)):
        for w in range(fw):
            rows[i, w] = (f >> (64 * w)) & ((1 << 64) - 1)
        if rng is not None:  # junk in padding bits above the constant must be ignored
            pad = int(rng.integers(0, 1 << 20)) << (n + 1)
            rows[i, fw - 1] |= np.uint64(pad & ((1 << 64) - 1) & ~((1 << (n + 1 - 64 * (fw - 1))) - 1))
        rows[i, fw] = y & ((1 << 64) - 1)
        rows[i, fw + 1] = y >> 64
    return rows


def as_int(words):
    return sum(int(w) << (64 * i) for i, w in enumerate(words))


CASES = [(s, n, m, mode) for s in range(60) for (n, m, mode) in
         [(s % 6, 1 + s % 11, "clean" if s % 3 == 0 else "noisy")]]


@pytest.mark.parametrize("seed,n,m,mode", CASES)
def test_fit_matches_brute_force(seed, n, m, mode):
    rng = np.random.default_rng(1000 + seed)
    feats, ys = rand_system(rng, n, m, mode)
    kept, contra, S, basis = brute(n, feats, ys)
    rows = pack(n, feats, ys, rng)
    r, piv, B, M, nc, fc = oracle.fit_context(rows, n)
    assert r == len(kept) == (len(S).bit_length() - 1)
    assert nc == len(contra)
    assert fc == (contra[0] if contra else -1)
    assert [int(p) for p in piv] == [p for p, _, _ in basis]
    fw = (n + 64) // 64
    for i, (p, v, t) in enumerate(basis):
        assert as_int(B[i, :fw]) == v
        assert as_int(B[i, fw:]) == t
    pset = {p: t for p, _, t in basis}
    for j in range(n + 1):
        assert as_int(M[j]) == pset.get(j, 0)
    # every query of the ambient space (explicit feature vectors, constant bit as given)
    for q in range(1 << (n + 1)):
        qw = np.array([(q >> (64 * w)) & ((1 << 64) - 1) for w in range(fw)], np.uint64)
        ok, acc, res = oracle.reduce_query(piv, B, n, qw)
        assert ok == (q in S)
        if ok:
            assert as_int(acc) == S[q]


def column_scan(n, feats, ys):
    """independent elimination: columns in priority order, earliest remaining row as pivot"""
    m = len(feats)
    cols = prio(n)
    A = np.array([[(f >> s) & 1 for s in cols] for f in feats], dtype=bool).reshape(m, n + 1)
    Y = np.array([[(y >> b) & 1 for b in range(128)] for y in ys], dtype=bool).reshape(m, 128)
    pivoted = np.zeros(m, bool)
    piv_row = {}
    for ci in range(n + 1):
        cand = np.nonzero(A[:, ci] & ~pivoted)[0]
        if len(cand) == 0:
            continue
        i = cand[0]
        pivoted[i] = True
        piv_row[ci] = i
        for j in cand[1:]:
            A[j] ^= A[i]
            Y[j] ^= Y[i]
    kept = sorted(piv_row.values())
    contra = [i for i in range(m) if not pivoted[i] and Y[i].any()]
    # back-substitution, lowest-priority pivot column first
    for ci in sorted(piv_row, reverse=True):
        i = piv_row[ci]
        for cj, j in piv_row.items():
            if j != i and A[j, ci]:
                A[j] ^= A[i]
                Y[j] ^= Y[i]
    basis = []
    for ci in sorted(piv_row):
        i = piv_row[ci]
        v = sum(1 << cols[k] for k in range(n + 1) if A[i, k])
        t = sum(1 << b for b in range(128) if Y[i, b])
        basis.append((cols[ci], v, t))
    return kept, contra, basis


@pytest.mark.parametrize("seed", range(40))
def test_fit_matches_column_scan(seed):
    rng = np.random.default_rng(5000 + seed)
    n = int(rng.integers(0, 70))   # crosses the one-word boundary
    m = int(rng.integers(0, 40))
    feats, ys = rand_system(rng, n, m, "noisy" if seed % 2 else "clean")
    kept, contra, basis = column_scan(n, feats, ys)
    r, piv, B, M, nc, fc = oracle.fit_context(pack(n, feats, ys), n)
    fw = (n + 64) // 64
    assert r == len(kept)
    assert nc == len(contra) and fc == (contra[0] if contra else -1)
    assert [int(p) for p in piv] == [p for p, _, _ in basis]
    for i, (p, v, t) in enumerate(basis):
        assert as_int(B[i, :fw]) == v and as_int(B[i, fw:]) == t


def test_encode_batch_conventions():
    """x bits past the width, the constant of Eq. 1, bad context ids, contradictory contexts, 0-row contexts."""
    rng = np.random.default_rng(3)
    n_bits, rows_list, feats_all = [], [], []
    for c, (n, mode) in enumerate([(5, "clean"), (3, "noisy"), (4, "clean")]):
        m = 0 if c == 2 else 12
        feats, ys = rand_system(rng, n, m, mode)
        feats = [f | (1 << n) for f in feats]  # affine rows: constant feature set
        ys = [y for y in ys]
        n_bits.append(n)
        rows_list.append(pack(n, feats, ys) if m else np.zeros((0, (n + 64) // 64 + 2), np.uint64))
        feats_all.append((feats, ys))
    import synth
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    fit = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    Q = []
    for c in range(3):
        n = n_bits[c]
        for x in range(1 << n):
            Q.append((c, x))
        Q.append((c, 1 << n))        # a bit at the width itself: outside the ambient space
        Q.append((c, 1 << 63))       # far outside
    Q += [(-1, 0), (3, 0), (7, 1)]
    ctx = np.array([c for c, _ in Q], np.int32)
    x = np.array([v for _, v in Q], np.uint64)
    words, qf = oracle.encode_batch(fit, ctx, x, 1)
    for i, (c, xv) in enumerate(Q):
        if c < 0 or c >= 3:
            assert qf[i] == oracle.Q_BAD_CTX and words[i].sum() == 0
            continue
        n = n_bits[c]
        feats, ys = feats_all[c]
        kept, contra, S, _ = brute(n, feats, ys)
        cflag = oracle.Q_CTX_CONTRADICTORY if contra else 0
        q = xv | (1 << n)
        if xv >> n or q not in S:
            assert qf[i] == cflag | oracle.Q_OUT_OF_SPAN and words[i].sum() == 0
        else:
            assert qf[i] == cflag and as_int(words[i]) == S[q]
