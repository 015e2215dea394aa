"""Pins of the feature-vectorizer and word-merge oracle (oracle/words.py).

Every expected value comes from the paper's numbers or from a plain
definition written independently here (shifts of Python integers, per-bit
checks), never from the oracle itself.
"""
import numpy as np

from oracle import words as W

ALL = 2 ** 64 - 1


def test_feature_dimension_eq1():
    # d = 1 + 64k: 321 features for k = 5 (the tensor-core example), 513 for k = 8
    for k, d in ((5, 321), (8, 513), (1, 65), (0, 1)):
        assert len(W.phi_bits([0] * k)) == d
        row = W.vectorize_row([0] * k, 0, 0, ALL, ALL)
        assert len(row) == k + 3                      # ceil(d / 64) feature words + 2 output words
        assert row[k] == 1                            # the constant: storage bit n = 64k


def test_single_bits_land_at_feature_index_minus_one():
    # feature index 1 + 64j + b is bit b of v_j; it is stored at storage bit 64j + b
    rng = np.random.default_rng(0)
    for _ in range(200):
        k = int(rng.integers(1, 9))
        j, b = int(rng.integers(0, k)), int(rng.integers(0, 64))
        vals = [0] * k
        vals[j] = 1 << b
        row = W.vectorize_row(vals, 0, 0, ALL, ALL)
        feat = sum(int(row[w]) << (64 * w) for w in range(k + 1))
        assert feat == (1 << (64 * j + b)) | (1 << (64 * k))


def test_appendix_c_feature_indices():
    # App. C's five-row decomposition has pivots at feature indices 259, 199, 196, 135, 3
    # of a k = 5 vector: v_4 bit 2, v_3 bit 6, v_3 bit 3, v_2 bit 6, v_0 bit 2
    vals = [0] * 5
    for l in (259, 199, 196, 135, 3):
        j, b = divmod(l - 1, 64)
        vals[j] |= 1 << b
    assert vals == [1 << 2, 0, 1 << 6, (1 << 6) | (1 << 3), 1 << 2]
    phi = W.phi_bits(vals)
    assert [l for l, bit in enumerate(phi) if bit] == [0, 3, 135, 196, 199, 259]
    row = W.vectorize_row(vals, 0, 0, ALL, ALL)
    feat = sum(int(row[w]) << (64 * w) for w in range(6))
    assert [i for i in range(6 * 64) if (feat >> i) & 1] == [2, 134, 195, 198, 258, 320]


def test_outputs_restricted_to_learned_bits():
    rng = np.random.default_rng(1)
    for _ in range(100):
        ylo, yhi, klo, khi = (int(v) for v in rng.integers(0, 2 ** 63, size=4))
        row = W.vectorize_row([5, 7], ylo, yhi, klo, khi)
        assert row[3] == ylo & klo and row[4] == yhi & khi


def test_merge_is_xor_of_shifted_field():
    # y_full = y XOR (sc << s) over 128 bits, checked bit by bit
    rng = np.random.default_rng(2)
    for _ in range(300):
        width = int(rng.integers(1, 65))
        shift = int(rng.integers(0, 129 - width))
        sc = int(rng.integers(0, 2 ** 63)) * 2 + int(rng.integers(0, 2))
        ylo, yhi = (int(v) for v in rng.integers(0, 2 ** 63, size=2))
        lo, hi = W.merge_word(ylo, yhi, sc, shift, width, 0, 0, None)
        for bit in range(128):
            src = (ylo >> bit) & 1 if bit < 64 else (yhi >> (bit - 64)) & 1
            fb = bit - shift
            if 0 <= fb < width:
                src ^= (sc >> fb) & 1
            got = (lo >> bit) & 1 if bit < 64 else (hi >> (bit - 64)) & 1
            assert got == src


def test_merge_field_spanning_the_word_boundary():
    # a 17-bit field at position 55 covers bits 55..71: 9 bits in the low word, 8 in the high word
    lo, hi = W.merge_word(0, 0, (1 << 17) - 1, 55, 17, 0, 0, None)
    assert lo == ((1 << 9) - 1) << 55 and hi == (1 << 8) - 1
    # the field is cut to its width: bits above it are ignored
    lo, hi = W.merge_word(0, 0, (1 << 20) - 1, 105, 17, 0, 0, None)
    assert lo == 0 and hi == ((1 << 17) - 1) << 41


def test_opaque_bits_restored_from_state():
    # an opaque mask on bits 122 and 124 (the paper's two ambiguous positions): after the
    # merge those bits come from the recorded state, every other bit from the merged word
    mask_hi = (1 << 58) | (1 << 60)
    for state_hi in (0, ALL, 1 << 58, 1 << 60):
        lo, hi = W.merge_word(0x1234, ALL, None, 0, 0, 0, mask_hi, (0, state_hi))
        assert lo == 0x1234
        assert hi == (ALL & ~mask_hi) | (state_hi & mask_hi)
    # restore without a state clears the masked bits
    assert W.merge_word(ALL, ALL, None, 0, 0, ALL, 0, None) == (0, ALL)


def test_merge_round_trip():
    # XOR-merging the same field twice gives the learned word back; restoring is idempotent
    rng = np.random.default_rng(3)
    for _ in range(100):
        ylo, yhi, sc = (int(v) for v in rng.integers(0, 2 ** 63, size=3))
        a = W.merge_word(ylo, yhi, sc, 105, 17, 0, 0, None)
        assert W.merge_word(a[0], a[1], sc, 105, 17, 0, 0, None) == (ylo, yhi)
        m = (int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2 ** 63)))
        st = (int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2 ** 63)))
        b = W.merge_word(ylo, yhi, None, 0, 0, m[0], m[1], st)
        assert W.merge_word(b[0], b[1], None, 0, 0, m[0], m[1], st) == b


def test_vectorized_rows_fit_and_encode_with_the_core_oracle():
    # rows built by the vectorizer are ordinary fit rows: a planted affine map over the
    # values is recovered by the core oracle, and the values encode as queries with stride k
    import oracle
    rng = np.random.default_rng(4)
    k, R = 2, 300
    vals = rng.integers(0, 2 ** 63, size=(R, k), dtype=np.uint64) * np.uint64(2) + rng.integers(0, 2, size=(R, k), dtype=np.uint64)
    A = [int(v) for v in rng.integers(0, 2 ** 63, size=2 * 128)]  # planted map: row i of W over 128 value bits + bias
    bias = int(rng.integers(0, 2 ** 63))
    y = np.zeros(2 * R, np.uint64)
    for r in range(R):
        xv = int(vals[r, 0]) | (int(vals[r, 1]) << 64)
        out = bias
        for i in range(64):   # output bit i = parity(A_i & x) XOR bias_i, low word only
            out ^= (bin(xv & (A[2 * i] | (A[2 * i + 1] << 64))).count("1") & 1) << i
        y[2 * r] = out
    rows = W.vectorize_rows(vals.reshape(-1), k, y)
    ref = oracle.fit_batch(rows, np.array([0, rows.size], np.int64), np.array([64 * k], np.int32))
    assert ref.rank[0] == 129 and ref.flags[0] == 0
    words, qf = oracle.encode_batch(ref, np.zeros(R, np.int32), vals.reshape(-1), k)
    assert (qf == 0).all() and np.array_equal(words.reshape(-1, 2)[:, 0], y.reshape(-1, 2)[:, 0])
