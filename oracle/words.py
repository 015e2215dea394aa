"""TEST INFRASTRUCTURE -- CPU oracle of the feature vectorizer and the
post-encode word merges.

Plain Python integers, one row or word at a time; only the tests, the smoke
check and the benchmark's CPU-baseline leg use it.

vectorize_rows -- the feature vector of Eq. 1: phi = [1 | bits64(v_0) | ... |
    bits64(v_{k-1})], d = 1 + 64k features.  Feature index l = 0 is the constant
    and index 1 + 64j + b is bit b of value v_j (App. C numbers the features of
    its worked decomposition this way).  A fit row stores feature index l >= 1
    at storage bit l - 1 and the constant at storage bit n = 64k, followed by
    the 128-bit output word; the output is restricted to the learned bits.
merge_words -- the assembly of a final word from the learned word (Sec. 4,
    the worked example that closes the method): a separately supplied field is
    shifted into place and XORed in (y_full = y XOR (sc << s)), then the bits of
    an opaque mask, which are excluded from learning, are restored from the
    recorded state.
"""
from __future__ import annotations

import numpy as np

MASK128 = (1 << 128) - 1


def to_int128(lo: int, hi: int) -> int:
    return (int(lo) & (2 ** 64 - 1)) | ((int(hi) & (2 ** 64 - 1)) << 64)


def from_int128(v: int):
    return v & (2 ** 64 - 1), (v >> 64) & (2 ** 64 - 1)


def phi_bits(values) -> list:
    """Eq. 1 as a list of bits in feature-index order: [1, bits(v_0) (LSB first), ...]."""
    bits = [1]
    for v in values:
        v = int(v)
        bits.extend((v >> b) & 1 for b in range(64))
    return bits


def vectorize_row(values, y_lo: int, y_hi: int, keep_lo: int, keep_hi: int) -> list:
    """One fit row (k + 3 uint64 words) from k parsed 64-bit values and an output word."""
    k = len(values)
    n = 64 * k
    phi = phi_bits(values)
    feat = 0
    for l, bit in enumerate(phi):
        if bit:
            feat |= 1 << (n if l == 0 else l - 1)   # storage bit of feature index l
    words = [(feat >> (64 * w)) & (2 ** 64 - 1) for w in range(k + 1)]
    y = to_int128(y_lo, y_hi) & to_int128(keep_lo, keep_hi)
    return words + list(from_int128(y))


def vectorize_rows(values, k: int, y=None, keep=(2 ** 64 - 1, 2 ** 64 - 1)) -> np.ndarray:
    """values uint64 [R*k], y uint64 [R*2] or None -> rows uint64 [R*(k+3)]."""
    values = np.asarray(values, np.uint64).reshape(-1, k) if k else np.zeros((len(y) // 2 if y is not None else 0, 0), np.uint64)
    R = values.shape[0] if k else (0 if y is None else len(y) // 2)
    out = np.zeros((R, k + 3), np.uint64)
    for r in range(R):
        ylo, yhi = (int(y[2 * r]), int(y[2 * r + 1])) if y is not None else (0, 0)
        out[r] = vectorize_row([int(v) for v in values[r]] if k else [], ylo, yhi, keep[0], keep[1])
    return out.reshape(-1)


def merge_word(y_lo: int, y_hi: int, field, shift: int, width: int, mask_lo: int, mask_hi: int, state) -> tuple:
    """y_full = y XOR (field << shift) over 128 bits, then the masked bits taken from the state."""
    y = to_int128(y_lo, y_hi)
    if field is not None:
        y ^= ((int(field) & ((1 << width) - 1)) << shift) & MASK128
    m = to_int128(mask_lo, mask_hi)
    s = to_int128(*state) if state is not None else 0
    y = (y & ~m & MASK128) | (s & m)
    return from_int128(y)


def merge_words(words, field, shift: int, width: int, mask=(0, 0), state=None) -> np.ndarray:
    """words uint64 [Q*2], field uint64 [Q] or None, state uint64 [Q*2] or None -> uint64 [Q*2]."""
    words = np.asarray(words, np.uint64)
    Q = len(words) // 2
    out = np.zeros(2 * Q, np.uint64)
    for q in range(Q):
        st = (int(state[2 * q]), int(state[2 * q + 1])) if state is not None else None
        f = int(field[q]) if field is not None else None
        out[2 * q], out[2 * q + 1] = merge_word(int(words[2 * q]), int(words[2 * q + 1]), f, shift, width,
                                                mask[0], mask[1], st)
    return out
