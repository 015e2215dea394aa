"""Oracle pinned to the values the paper prints.

* App. B worked example: every basis state, the redundant observation, its
  contradictory variant and both query traces (fixture ``golden/appendix_b.json``).
* App. C structure: feature index 1 + 64 j + b of Eq. 1, the pivot of a row that
  mixes the constant with v0 bits, and a five-row decomposition of phi(v).  The
  output words there are synthetic; the paper's instruction words are not used.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "appendix_b.json")))

# App. B uses 4 feature bits with no constant: x_j = q_j, constant column (storage bit 4) always 0.
N_B = 4


def _row(q, y):
    return [int(q, 2), int(y, 2), 0]


def _basis_dict(piv, B):
    return {int(p): (format(int(B[i, 0]), "04b"), format(int(B[i, 1]), "08b")) for i, p in enumerate(piv)}


def test_appendix_b_states_after_each_observation():
    obs = GOLD["observations"]
    for k in range(1, len(obs) + 1):
        rows = np.array([_row(o["q"], o["y"]) for o in obs[:k]], np.uint64)
        r, piv, B, M, nc, fc = oracle.fit_context(rows, N_B)
        want = {int(p): tuple(v) for p, v in GOLD["basis_after"][k - 1].items()}
        assert _basis_dict(piv, B) == want, f"after observation {k}"
        assert r == len(want)
        assert nc == 0 and fc == -1
        # basis order: descending pivot priority
        assert list(piv) == sorted(want, reverse=True)


def test_appendix_b_contradiction_variant():
    obs = [dict(o) for o in GOLD["observations"]]
    var = GOLD["contradictory_variant"]
    obs[var["replace_observation"] - 1]["y"] = var["y"]
    rows = np.array([_row(o["q"], o["y"]) for o in obs], np.uint64)
    r, piv, B, M, nc, fc = oracle.fit_context(rows, N_B)
    assert r == 3
    assert nc == 1 and fc == 3
    # the contradictory row is discarded: the basis is the rank-3 basis of the first three observations
    want = {int(p): tuple(v) for p, v in GOLD["basis_after"][2].items()}
    assert _basis_dict(piv, B) == want
    # its residual: reduce the row's features and output with the basis
    q = np.array([int(obs[3]["q"], 2)], np.uint64)
    ok, acc, res = oracle.reduce_query(piv, B, N_B, q)
    assert ok and int(res[0]) == int(var["residual"][0], 2)
    assert int(acc[0]) ^ int(var["y"], 2) == int(var["residual"][1], 2)


def test_appendix_b_queries():
    rows = np.array([_row(o["q"], o["y"]) for o in GOLD["observations"]], np.uint64)
    r, piv, B, M, nc, fc = oracle.fit_context(rows, N_B)
    for qd in GOLD["queries"]:
        q = np.array([int(qd["q"], 2)], np.uint64)
        ok, acc, res = oracle.reduce_query(piv, B, N_B, q)
        assert ok == qd["supported"]
        if ok:
            assert format(int(acc[0]), "08b") == qd["word"] and int(acc[1]) == 0
            # replay the printed trace: XOR of the visited basis words in order
            acc_t, cur = 0, int(qd["q"], 2)
            bd = {int(p): (int(B[i, 0]), int(B[i, 1])) for i, p in enumerate(piv)}
            for k, want in zip(qd["pivots_visited"], qd["acc_trace"]):
                assert (cur >> k) & 1
                cur ^= bd[k][0]
                acc_t ^= bd[k][1]
                assert format(acc_t, "08b") == want
            assert cur == 0
        else:
            assert format(int(res[0]), "04b") == qd["residual"]
    # the canonical map: column p = z_p for pivots, zero columns elsewhere; M q = T(q) on the span
    assert [format(int(M[j, 0]), "08b") for j in (3, 2, 1)] == ["10100101", "00111010", "11000011"]
    assert int(M[0, 0]) == 0 and int(M[4, 0]) == 0


def _phi_indices(values):
    """Eq. 1: index 0 is the constant, bit b of value j has index 1 + 64 j + b."""
    idx = {0}
    for j, v in enumerate(values):
        for b in range(64):
            if (v >> b) & 1:
                idx.add(1 + 64 * j + b)
    return idx


def _storage(ell, n):
    """paper feature index -> storage bit (x_i at bit i, constant at bit n)"""
    return n if ell == 0 else ell - 1


def _vec(indices, n):
    fw = (n + 64) // 64
    v = np.zeros(fw, np.uint64)
    for ell in indices:
        s = _storage(ell, n)
        v[s // 64] |= np.uint64(1) << np.uint64(s % 64)
    return v


def test_appendix_c_structure():
    # five parsed values -> d = 1 + 64*5 = 321 features
    values = (7, 4, 68, 72, 4)
    n = 64 * len(values)
    assert n + 1 == 321
    phi = _phi_indices(values)
    assert phi == {0, 1, 2, 3, 67, 131, 135, 196, 199, 259}
    # the five basis rows of the decomposition (feature sets from the paper's table); synthetic outputs
    rows_idx = {259: {67, 131, 259}, 199: {199}, 196: {196}, 135: {135}, 3: {0, 1, 2, 3}}
    rng = np.random.default_rng(7)
    z = {k: rng.integers(0, 2 ** 63, size=2, dtype=np.uint64) for k in rows_idx}
    fw = (n + 64) // 64
    rows = np.zeros((len(rows_idx), fw + 2), np.uint64)
    for i, (k, s) in enumerate(sorted(rows_idx.items())):
        rows[i, :fw] = _vec(s, n)
        rows[i, fw:] = z[k]
    r, piv, B, M, nc, fc = oracle.fit_context(rows, n)
    assert r == 5 and nc == 0
    # pivots are the highest feature index of each row; the constant (index 0) never wins
    assert [int(p) for p in piv] == [_storage(k, n) for k in (259, 199, 196, 135, 3)]
    ok, acc, res = oracle.reduce_query(piv, B, n, _vec(phi, n))
    assert ok
    want = np.zeros(2, np.uint64)
    for k in rows_idx:
        want ^= z[k]
    assert np.array_equal(acc, want)
    # dropping v1[2] (index 67, a non-pivot bit of r_259) leaves residual {67}
    ok2, _, res2 = oracle.reduce_query(piv, B, n, _vec(phi - {67}, n))
    assert not ok2
    assert np.array_equal(res2, _vec({67}, n))


@pytest.mark.parametrize("k,d", [(5, 321), (8, 513)])
def test_feature_dimension(k, d):
    # Eq. 1 and the UTCOMMA example: k parsed values give 1 + 64 k features
    assert 1 + 64 * k == d
