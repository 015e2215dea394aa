"""GPU parity of the Eq. 1 row builder and the post-encode word merge against
the oracle (oracle/words.py), bit for bit, through the C ABI; and the chain
values -> rows -> fit -> encode -> merge against the oracle chain."""
import numpy as np
import pytest

import oracle
from oracle import words as W
import parity

pytestmark = pytest.mark.gpu
ALL = 2 ** 64 - 1


@pytest.fixture(scope="module")
def f2(require_gpu):
    from paper_2608_20532_amd import f2gpu
    return f2gpu


def _u64(rng, shape):
    return rng.integers(0, 2 ** 63, size=shape, dtype=np.uint64) * np.uint64(2) + rng.integers(0, 2, size=shape, dtype=np.uint64)


def _vectorize_gpu(f2, vals, y, R, k, keep):
    import torch
    out = torch.full((max(R * (k + 3), 1),), -1, dtype=torch.int64, device="cuda")
    vd = parity.to_dev(vals if vals.size else np.zeros(1, np.uint64))
    yd = parity.to_dev(y) if y is not None else None
    assert f2.f2_vectorize_rows(vd if k else None, yd, R, k, keep, out) == 0
    torch.cuda.synchronize()
    return parity.host(out, np.uint64)[:R * (k + 3)]


@pytest.mark.parametrize("k,R", [(0, 300), (1, 1), (2, 257), (5, 1000), (8, 777), (63, 130)])
def test_vectorize_rows_parity(f2, k, R):
    rng = np.random.default_rng(100 + k)
    vals = _u64(rng, R * k)
    y = _u64(rng, 2 * R)
    for keep, with_y in (((ALL, ALL), True), ((ALL, ALL & ~((1 << 58) | (1 << 60))), True), ((ALL, ALL), False)):
        got = _vectorize_gpu(f2, vals, y if with_y else None, R, k, keep)
        exp = W.vectorize_rows(vals, k, y if with_y else None, keep) if R else np.zeros(0, np.uint64)
        if k == 0 and not with_y:
            exp = np.tile(np.array([1, 0, 0], np.uint64), R)
        assert np.array_equal(got, exp), (k, R, keep, with_y)


def test_vectorize_rows_large_sampled(f2):
    """7.24M rows of k = 4 values; the oracle checks 20,000 sampled rows."""
    rng = np.random.default_rng(7)
    R, k = 7_240_070, 4
    vals = _u64(rng, R * k)
    y = _u64(rng, 2 * R)
    got = _vectorize_gpu(f2, vals, y, R, k, (ALL, ALL)).reshape(R, k + 3)
    sample = rng.choice(R, size=20_000, replace=False)
    for r in sample:
        exp = W.vectorize_row([int(v) for v in vals[r * k:(r + 1) * k]], int(y[2 * r]), int(y[2 * r + 1]), ALL, ALL)
        assert [int(v) for v in got[r]] == exp, r


@pytest.mark.parametrize("shift,width", [(0, 64), (0, 1), (63, 1), (64, 64), (55, 17), (105, 17), (111, 17), (127, 1), (30, 40)])
def test_merge_words_parity(f2, shift, width):
    import torch
    rng = np.random.default_rng(shift * 131 + width)
    Q = 4099
    words = _u64(rng, 2 * Q)
    field = _u64(rng, Q)
    state = _u64(rng, 2 * Q)
    for mask, use_state, use_field in (((0, 0), False, True), ((0, (1 << 58) | (1 << 60)), True, True),
                                       ((0x00ff00ff, ALL), True, False), ((ALL, 0), False, False)):
        out = torch.empty(2 * Q, dtype=torch.int64, device="cuda")
        st = f2.f2_merge_words(parity.to_dev(words), parity.to_dev(field) if use_field else None, shift, width, mask,
                               parity.to_dev(state) if use_state else None, Q, out)
        assert st == 0
        torch.cuda.synchronize()
        exp = W.merge_words(words, field if use_field else None, shift, width, mask, state if use_state else None)
        assert np.array_equal(parity.host(out, np.uint64), exp), (mask, use_state, use_field)


def test_merge_in_place(f2):
    import torch
    rng = np.random.default_rng(9)
    Q = 1000
    words, field = _u64(rng, 2 * Q), _u64(rng, Q)
    d = parity.to_dev(words)
    assert f2.f2_merge_words(d, parity.to_dev(field), 105, 17, (0, 0), None, Q, d) == 0
    torch.cuda.synchronize()
    assert np.array_equal(parity.host(d, np.uint64), W.merge_words(words, field, 105, 17))


def test_values_rows_fit_encode_merge_chain(f2):
    """Parsed values of three contexts (k = 1, 2, 5) -> rows -> fit -> encode -> merge, on the GPU
    and through the oracle, word for word."""
    import torch
    rng = np.random.default_rng(11)
    mask = (0, (1 << 58) | (1 << 60))
    keep = (ALL, ALL & ~mask[1])
    rows_list, n_bits, q_ctx, q_vals = [], [], [], []
    for c, (k, R) in enumerate(((1, 200), (2, 400), (5, 120))):
        vals = _u64(rng, (R, k))
        if k == 5:
            vals[:, 3:] = 0      # a rank-deficient context: two values never vary
        # outputs: a planted affine map of the row's feature bits (each set bit (w, b)
        # contributes a fixed 128-bit vector), restricted to the learned bits
        rows = W.vectorize_rows(vals.reshape(-1), k, None, keep).reshape(R, k + 3)
        A = _u64(rng, (k + 1, 2))
        for r in range(R):
            acc = [0, 0]
            for w in range(k + 1):
                for b in range(64):
                    if (int(rows[r, w]) >> b) & 1:
                        for h in range(2):
                            acc[h] ^= (int(A[w, h]) * (b + 1)) & ALL
            rows[r, k + 1], rows[r, k + 2] = acc[0] & keep[0], acc[1] & keep[1]
        rows_list.append(rows)
        n_bits.append(64 * k)
        sel = rng.integers(0, R, size=300)
        q_ctx.append(np.full(300, c, np.int32))
        qv = np.zeros((300, 5), np.uint64)
        qv[:, :k] = vals[sel]
        qv[::7, :k] ^= _u64(rng, (len(qv[::7]), k)) & np.uint64(0xF0)   # some queries leave the span
        q_vals.append(qv)
    import synth
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    model = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    parity.compare_fit(model, ref)
    ctx = np.concatenate(q_ctx)
    x = np.concatenate(q_vals).reshape(-1)
    words, qf = f2.encode(model, parity.to_dev(ctx), parity.to_dev(x), 5)
    sc = _u64(rng, len(ctx)) & np.uint64((1 << 17) - 1)
    state = _u64(rng, 2 * len(ctx))
    out = torch.empty_like(words).reshape(-1)
    assert f2.f2_merge_words(words.reshape(-1), parity.to_dev(sc), 105, 17, mask, parity.to_dev(state), len(ctx), out) == 0
    torch.cuda.synchronize()
    rw, rq = oracle.encode_batch(ref, ctx, x, 5)
    parity.compare_encode(words, qf, rw, rq)
    exp = W.merge_words(rw.reshape(-1), sc, 105, 17, mask, state)
    assert np.array_equal(parity.host(out, np.uint64), exp)
    assert (rq & oracle.Q_OUT_OF_SPAN).any() and (rq == 0).any()
