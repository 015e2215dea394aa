"""Pins of the interleaved-stream grouping oracle (oracle/group.py): a worked
stream written out by hand, and the invariants that define the grouping (each
context's rows in stream order, every valid row exactly once, invalid rows
dropped)."""
import numpy as np

from oracle import group as G


def test_hand_worked_stream():
    # contexts: 0 (n = 3: 3-word rows), 1 (n = 70: 4-word rows), 2 (n = 5), stride 4 words
    n_bits = [3, 70, 5]
    ids = [1, 0, 2, 0, 7, 1, -1, 0]
    rows = np.zeros((8, 4), np.uint64)
    for r in range(8):
        rows[r] = [10 * r + 1, 10 * r + 2, 10 * r + 3, 10 * r + 4]
    out, off, dropped = G.group_rows(ids, rows, 4, n_bits)
    assert dropped == 2                                   # ids 7 and -1
    assert off.tolist() == [0, 9, 17, 20]                 # 3 rows x 3, 2 rows x 4, 1 row x 3
    assert out[0:9].tolist() == [11, 12, 13, 31, 32, 33, 71, 72, 73]
    assert out[9:17].tolist() == [1, 2, 3, 4, 51, 52, 53, 54]
    assert out[17:20].tolist() == [21, 22, 23]


def test_grouping_invariants_random_stream():
    rng = np.random.default_rng(3)
    C, R, S = 50, 3000, 6
    n_bits = rng.integers(0, 260, size=C)
    n_bits[3] = 5000                                      # outside the supported widths
    ids = rng.integers(-2, C + 2, size=R)
    rows = rng.integers(0, 2 ** 63, size=(R, S), dtype=np.uint64)
    out, off, dropped = G.group_rows(ids, rows, S, n_bits)
    W = [(int(n) + 64) // 64 + 2 for n in n_bits]
    kept = 0
    for c in range(C):
        mine = [r for r in range(R) if ids[r] == c]
        if n_bits[c] > 4095 or W[c] > S:
            assert off[c + 1] == off[c]
            continue
        got = out[off[c]:off[c + 1]].reshape(-1, W[c])
        assert len(got) == len(mine)
        assert np.array_equal(got, rows[mine, :W[c]])     # stream order, trimmed
        kept += len(mine)
    assert kept + dropped == R and off[-1] == len(out)
