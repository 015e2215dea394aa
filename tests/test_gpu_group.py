"""GPU parity of interleaved-stream ingestion (f2_group_rows) against the grouping
oracle (oracle/group.py), and at the size of the 80,000-context fit workload
against the rows the interleaving was made from."""
import numpy as np
import pytest

import parity
import synth
from oracle import group as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def f2(require_gpu):
    from paper_2608_20532_amd import f2gpu
    return f2gpu


def _run(f2, ids, rows, stride, n_bits):
    import torch
    out, off, dropped = f2.group(parity.to_dev(np.asarray(ids, np.int32)), parity.to_dev(rows.reshape(-1)), stride,
                                 parity.to_dev(np.asarray(n_bits, np.int32)))
    torch.cuda.synchronize()
    off_h = parity.host(off, np.int64)
    return parity.host(out, np.uint64)[:int(off_h[-1])], off_h, int(parity.host(dropped, np.int64)[0])


@pytest.mark.parametrize("C,R,S", [(300, 200_000, 6), (3, 1000, 4), (70_000, 150_000, 7), (300_000, 400_000, 5)])
def test_group_random_stream(f2, C, R, S):
    """Random ids (some out of range), widths up to 300 (some rows wider than the
    stride, one width outside the supported range): rows, offsets and the dropped
    count equal the oracle's; 300 contexts take one radix pass, 70,000 two and
    300,000 three."""
    rng = np.random.default_rng(C)
    n_bits = rng.integers(0, 300, size=C).astype(np.int32)
    n_bits[0] = 4096 if C > 1 else n_bits[0]
    ids = rng.integers(-3, C + 3, size=R)
    rows = rng.integers(0, 2 ** 63, size=(R, S), dtype=np.uint64)
    out, off, dropped = _run(f2, ids, rows, S, n_bits)
    r_out, r_off, r_drop = G.group_rows(ids, rows, S, n_bits)
    assert dropped == r_drop and np.array_equal(off, r_off) and np.array_equal(out, r_out)


def test_group_empty_inputs(f2):
    out, off, dropped = _run(f2, np.zeros(0, np.int32), np.zeros((0, 4), np.uint64), 4, [5, 7])
    assert off.tolist() == [0, 0, 0] and dropped == 0
    out, off, dropped = _run(f2, np.array([0, 0], np.int32), np.ones((2, 4), np.uint64), 4, [])
    assert off.tolist() == [0] and dropped == 2


def test_group_recovers_the_fit_workload_and_fits_it(f2):
    """The rows of the 80,000-context workload interleaved at random with each
    context's order kept: grouping gives back its rows and offsets word for word,
    and the fit of the grouped rows equals the fit of the original."""
    import torch
    wl = synth.fit_workload(3)
    W = (wl.n_bits.astype(np.int64) + 64) // 64 + 2
    S = int(W.max())
    rng = np.random.default_rng(5)
    ids = np.repeat(np.arange(wl.num_ctx, dtype=np.int32), wl.m_rows)
    ids = ids[rng.permutation(len(ids))]               # the k-th occurrence of c is c's k-th row
    start = np.concatenate([[0], np.cumsum(wl.m_rows)[:-1]])
    order = np.argsort(ids, kind="stable")
    rank = np.empty(len(ids), np.int64)
    rank[order] = np.arange(len(ids)) - start[ids[order]]
    rows = np.zeros((len(ids), S), np.uint64)
    src = wl.row_off[ids] + rank * W[ids]
    for w in range(S):
        ok = w < W[ids]
        rows[ok, w] = wl.rows[src[ok] + w]
    out, off, dropped = _run(f2, ids, rows, S, wl.n_bits)
    assert dropped == 0 and np.array_equal(off, wl.row_off) and np.array_equal(out, wl.rows)
    a = parity.gpu_fit(f2, out, off, wl.n_bits)
    b = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    torch.cuda.synchronize()
    ga, gb = parity.model_to_host(a), parity.model_to_host(b)
    for k in ("rank", "flags", "maps", "basis"):
        assert np.array_equal(ga[k], gb[k]), k
