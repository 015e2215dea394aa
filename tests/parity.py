"""Helpers shared by the GPU parity tests: run the HIP library and the CPU
oracle on the same seeded inputs and compare every output element by element
(all outputs are bits or integers, so the bar is bit-exact equality)."""
import numpy as np

import oracle


def to_dev(a, dtype=None):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    t = torch.from_numpy(a)
    return t.to("cuda")


def host(t, np_dtype):
    return t.detach().cpu().numpy().view(np_dtype)


def gpu_fit(f2, rows, row_off, n_bits):
    import torch
    model = f2.fit(to_dev(rows if rows.size else np.zeros(1, np.uint64)), to_dev(row_off), n_bits)
    torch.cuda.synchronize()
    return model


def model_to_host(model):
    return dict(
        basis=host(model.basis, np.uint64), pivots=host(model.pivots, np.int32), maps=host(model.maps, np.uint64),
        tables=host(model.tables, np.uint64),
        rank=host(model.rank, np.int32)[:model.num_ctx], flags=host(model.ctx_flags, np.uint32)[:model.num_ctx],
        n_contra=host(model.n_contra, np.int32)[:model.num_ctx],
        first=host(model.first_contra_row, np.int64)[:model.num_ctx])


def compare_fit(model, ref: "oracle.FitResult", ctx=None):
    """Bit-exact comparison of every defined output; returns the number of contexts checked."""
    g = model_to_host(model)
    C = model.num_ctx
    assert np.array_equal(g["flags"], ref.flags[:C]), "ctx_flags"
    assert np.array_equal(g["rank"], ref.rank[:C]), "rank"
    assert np.array_equal(g["n_contra"], ref.n_contra[:C]), "n_contra"
    assert np.array_equal(g["first"], ref.first_contra[:C]), "first_contra_row"
    # layouts agree (same documented capacities)
    assert np.array_equal(model.basis_off_host, ref.basis_off)
    assert np.array_equal(model.piv_off_host, ref.piv_off)
    assert np.array_equal(model.map_off_host, ref.map_off)
    n = np.clip(ref.n_bits[:C].astype(np.int64), 0, oracle.MAX_N)
    W = (n + 64) // 64 + 2
    ok_ctx = (ref.flags[:C] & (oracle.CTX_BAD_WIDTH | oracle.CTX_BAD_OUTPUT)) == 0
    # pivots [0, rank) and basis rows [0, rank) of every context
    pmask = np.zeros(len(ref.pivots), bool)
    bmask = np.zeros(len(ref.basis), bool)
    mmask = np.zeros(len(ref.maps), bool)
    r = ref.rank[:C].astype(np.int64)
    for arr, off, length in ((pmask, ref.piv_off, r), (bmask, ref.basis_off, r * W), (mmask, ref.map_off, 2 * (n + 1))):
        length = np.where(ok_ctx, length, 0)
        starts = off[:C]
        idx = np.repeat(starts - np.concatenate([[0], np.cumsum(length)[:-1]]), length) + np.arange(length.sum())
        arr[idx] = True
    assert np.array_equal(g["pivots"][:len(pmask)][pmask], ref.pivots[pmask]), "pivots"
    bad = np.nonzero(g["basis"][:len(bmask)][bmask] != ref.basis[bmask])[0]
    assert len(bad) == 0, f"basis mismatch at {len(bad)} words"
    assert np.array_equal(g["maps"][:len(mmask)][mmask], ref.maps[mmask]), "maps"
    check = np.nonzero(ok_ctx & ((ref.flags[:C] & oracle.CTX_BAD_SEGMENT) == 0))[0]
    if ctx is not None:
        check = np.intersect1d(check, np.asarray(ctx))
    for c in check:
        d = int(ref.n_bits[c]) + 1
        if d - int(ref.rank[c]) > int(ref.rank[c]):
            continue  # no parity rows: encoding reduces by the basis
        exp = expected_table(ref, int(c))
        got = g["tables"][ref.basis_off[c]:ref.basis_off[c] + exp.size]
        assert np.array_equal(got, exp), f"parity-check rows of context {c}"
    return C


def expected_table(ref: "oracle.FitResult", c: int) -> np.ndarray:
    """Parity-check rows of context c derived from the oracle's basis: for each free
    (non-pivot) column f in ascending order, fw words holding bit f and the pivot of
    every basis row that has bit f set (the layout documented for f2_model.tables)."""
    piv, B, M = ref.context(c)
    n = int(ref.n_bits[c])
    d = n + 1
    fw = (n + 64) // 64
    is_piv = np.zeros(d, bool)
    is_piv[piv] = True
    free = np.nonzero(~is_piv)[0]
    hb = np.zeros((len(free), 64 * fw), bool)
    hb[np.arange(len(free)), free] = True
    if len(piv) and len(free):
        feat = np.unpackbits(np.ascontiguousarray(B[:, :fw]).view(np.uint8), axis=1, bitorder="little")
        sel = feat[:, free].astype(bool)          # [rank, t]: basis row k holds free column f
        for k, p in enumerate(piv):
            hb[sel[k], p] = True
    return np.packbits(hb, axis=1, bitorder="little").view(np.uint64).ravel()


def compare_encode(words_dev, qf_dev, ref_words, ref_qf, sample=None):
    w = host(words_dev, np.uint64).reshape(-1, 2)
    q = host(qf_dev, np.uint8)
    if sample is not None:
        w, q = w[sample], q[sample]
    assert np.array_equal(q, ref_qf), f"qflags differ at {np.count_nonzero(q != ref_qf)} queries"
    bad = np.nonzero((w != ref_words).any(axis=1))[0]
    assert len(bad) == 0, f"words differ at {len(bad)} queries, first {bad[:5]}"


def _threads():
    import os
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def oracle_fit_threads(rows, row_off, n_bits, threads=None) -> "oracle.FitResult":
    """oracle.fit_batch over context ranges on several host threads (the single-threaded C
    oracle releases the GIL; each range writes its own slice of the shared output arrays at
    the documented offsets), for full-size workloads."""
    import ctypes
    from concurrent.futures import ThreadPoolExecutor
    L = oracle.lib()
    rows = np.ascontiguousarray(rows, np.uint64)
    row_off = np.ascontiguousarray(row_off, np.int64)
    n_bits = np.ascontiguousarray(n_bits, np.int32)
    C = len(n_bits)
    nb = np.clip(n_bits, 0, oracle.MAX_N)
    bo, po, mo = oracle.layout(nb)
    basis = np.zeros(max(int(bo[-1]), 1), np.uint64)
    pivots = np.full(max(int(po[-1]), 1), -1, np.int32)
    maps = np.zeros(max(int(mo[-1]), 1), np.uint64)
    rank = np.zeros(C, np.int32)
    flags = np.zeros(C, np.uint32)
    n_contra = np.zeros(C, np.int32)
    first = np.full(C, -1, np.int64)
    # ranges of about equal row words
    T = threads or _threads()
    cuts = np.searchsorted(row_off, np.linspace(0, row_off[-1], 4 * T + 1)[1:-1]).tolist()
    bounds = sorted(set([0] + [min(max(c, 0), C) for c in cuts] + [C]))

    def addr(a, k):
        return ctypes.c_void_p(a.ctypes.data + k * a.itemsize)

    def run(c0, c1):
        L.oracle_fit_batch(addr(rows, 0), rows.size, addr(row_off, c0), addr(n_bits, c0), c1 - c0,
                           addr(bo, c0), int(bo[-1]), addr(po, c0), int(po[-1]), addr(mo, c0), int(mo[-1]),
                           addr(basis, 0), addr(pivots, 0), addr(maps, 0), addr(rank, c0), addr(flags, c0),
                           addr(n_contra, c0), addr(first, c0))

    with ThreadPoolExecutor(T) as ex:
        list(ex.map(lambda b: run(*b), [(a, b) for a, b in zip(bounds[:-1], bounds[1:]) if b > a]))
    return oracle.FitResult(n_bits, bo, po, mo, basis, pivots, maps, rank, flags, n_contra, first)


def oracle_encode_threads(ref: "oracle.FitResult", ctx_id, x, stride, threads=None):
    """oracle.encode_batch over query ranges on several host threads; same outputs."""
    from concurrent.futures import ThreadPoolExecutor
    ctx_id = np.ascontiguousarray(ctx_id, np.int32)
    x = np.ascontiguousarray(x, np.uint64)
    Q = len(ctx_id)
    T = threads or _threads()
    step = max(1, -(-Q // (4 * T)))
    parts = [(a, min(Q, a + step)) for a in range(0, Q, step)]
    words = np.zeros((Q, 2), np.uint64)
    qf = np.zeros(Q, np.uint8)

    def run(a, b):
        w, q = oracle.encode_batch(ref, ctx_id[a:b], x[a * stride:b * stride], stride)
        words[a:b] = w
        qf[a:b] = q

    with ThreadPoolExecutor(T) as ex:
        list(ex.map(lambda p: run(*p), parts))
    return words, qf
