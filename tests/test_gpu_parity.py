"""GPU parity: the HIP library against the CPU oracle, bit for bit, through the C ABI.

Workloads: the four fit recipes at full size (all 64 contexts of the wide
recipe), random batches covering every feature-word count 1..64 with
rank-deficient and contradictory data, the degenerate contexts the method has,
and the query streams of the encode recipes, the 100M-query streams compared
query by query.  Full-size workloads run the oracle on several host threads
(context or query ranges; the oracle itself is single-threaded).
"""
import numpy as np
import pytest

import oracle
import synth
import parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def f2(require_gpu):
    from paper_2608_20532_amd import f2gpu
    return f2gpu


def _fit_and_compare(f2, wl):
    print(f"fit parity: recipe {wl.recipe}, {wl.num_ctx} contexts, {wl.total_rows} rows", flush=True)
    ref = parity.oracle_fit_threads(wl.rows, wl.row_off, wl.n_bits)
    model = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    parity.compare_fit(model, ref)
    return model, ref


@pytest.mark.parametrize("recipe,num_ctx", [(1, 1), (2, 4096), (3, 80000), (4, 64)])
def test_fit_recipes(f2, recipe, num_ctx):
    wl = synth.fit_workload(recipe, num_ctx=num_ctx)
    model, ref = _fit_and_compare(f2, wl)
    assert np.array_equal((ref.flags & 1) != 0, wl.contra.astype(bool) & (wl.m_rows >= 2))


def _random_batch(seed, widths, max_rows=300):
    rng = np.random.default_rng(seed)
    n_bits, rows_list = [], []
    for n in widths:
        n = int(n)
        fw = (n + 64) // 64
        m = int(rng.choice([0, 1, 2, 63, 64, 65, 127, 129, int(rng.integers(0, max_rows))]))
        kind = rng.integers(0, 4)
        d = n + 1
        # feature vectors from a random pool of k generators (k small -> many dependent rows)
        k = int(rng.integers(1, min(d, 96) + 1)) if kind else d
        pool = rng.integers(0, 2 ** 63, size=(k, fw), dtype=np.uint64) ^ (rng.integers(0, 2, size=(k, fw), dtype=np.uint64) << np.uint64(63))
        Wp = rng.integers(0, 2 ** 63, size=(k, 2), dtype=np.uint64)
        rows = np.zeros((m, fw + 2), np.uint64)
        for i in range(m):
            sel = rng.integers(0, 2, size=k).astype(bool)
            if kind == 3 and rng.random() < 0.2:
                sel[:] = False
            rows[i, :fw] = np.bitwise_xor.reduce(pool[sel], axis=0) if sel.any() else 0
            rows[i, fw:] = np.bitwise_xor.reduce(Wp[sel], axis=0) if sel.any() else 0
            if kind == 2 and rng.random() < 0.1:   # flip an output bit: contradictions
                rows[i, fw + int(rng.integers(0, 2))] ^= np.uint64(1) << np.uint64(int(rng.integers(0, 64)))
        # junk in padding bits above the constant
        vb = d - 64 * (fw - 1)
        if vb < 64 and m:
            rows[:, fw - 1] |= np.uint64(((1 << 64) - 1) ^ ((1 << vb) - 1)) & rng.integers(0, 2 ** 63, size=m, dtype=np.uint64)
        n_bits.append(n)
        rows_list.append(rows)
    return synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)


@pytest.mark.parametrize("seed", range(4))
def test_fit_random_small_widths(f2, seed):
    rng = np.random.default_rng(seed)
    widths = list(rng.integers(0, 512, size=300)) + [0, 1, 62, 63, 64, 65, 127, 128, 255, 256, 511]
    _fit_and_compare(f2, _random_batch(seed, widths))


def test_fit_random_large_widths(f2):
    widths = [512, 575, 576, 1000, 1023, 1024, 2047, 2500, 4094, 4095]
    _fit_and_compare(f2, _random_batch(77, widths, max_rows=200))


def _large_context(rng, n, m, kind):
    """One wide context (n >= 512) of m rows.  kind 'uniform': x uniform, y = W phi (full rank once
    m > n, later rows run the consistency check); 'pool': x from k random generators (rank <= k, many
    dependent rows); 'mixed': a pool prefix then uniform rows.  About 1% of rows get one output bit
    flipped, and some rows are zero or repeat an earlier row."""
    fw = (n + 64) // 64
    d = n + 1
    W = np.empty((d, 2), np.uint64)
    W[:] = rng.integers(0, 2 ** 63, size=(d, 2), dtype=np.uint64) ^ (rng.integers(0, 2, size=(d, 2), dtype=np.uint64) << np.uint64(63))
    rows = np.zeros((m, fw + 2), np.uint64)
    x = rng.integers(0, 2 ** 63, size=(m, fw), dtype=np.uint64) ^ (rng.integers(0, 2, size=(m, fw), dtype=np.uint64) << np.uint64(63))
    if kind != "uniform":
        k = int(rng.integers(20, min(d, 400)))
        pool = rng.integers(0, 2 ** 63, size=(k, fw), dtype=np.uint64) ^ (rng.integers(0, 2, size=(k, fw), dtype=np.uint64) << np.uint64(63))
        cut = m if kind == "pool" else m // 2
        for i in range(cut):
            sel = rng.integers(0, 2, size=k).astype(bool)
            x[i] = np.bitwise_xor.reduce(pool[sel], axis=0) if sel.any() else 0
    vb = d - 64 * (fw - 1)
    x[:, fw - 1] &= np.uint64((1 << vb) - 1) if vb < 64 else np.uint64((1 << 64) - 1)
    # constant bit set on most rows (affine), cleared on a few (linear rows)
    cw, cb = n // 64, n % 64
    const = rng.random(m) < 0.97
    x[const, cw] |= np.uint64(1 << cb)
    x[~const, cw] &= ~np.uint64(1 << cb)
    for i in np.nonzero(rng.random(m) < 0.02)[0]:
        x[i] = 0 if rng.random() < 0.5 else x[int(rng.integers(0, i + 1))]
    bits = np.unpackbits(x.view(np.uint8).reshape(m, fw, 8)[:, :, ::-1], axis=2).reshape(m, fw, 64)[:, :, ::-1].reshape(m, 64 * fw)[:, :d]
    y = np.zeros((m, 2), np.uint64)
    for j0 in range(0, d, 512):
        blk = bits[:, j0:j0 + 512].astype(bool)
        y ^= np.bitwise_xor.reduce(np.where(blk[:, :, None], W[None, j0:j0 + 512, :], np.uint64(0)), axis=1)
    flip = np.nonzero(rng.random(m) < 0.01)[0]
    for i in flip:
        y[i, int(rng.integers(0, 2))] ^= np.uint64(1) << np.uint64(int(rng.integers(0, 64)))
    rows[:, :fw] = x
    rows[:, fw:] = y
    # junk in the padding bits above the constant
    if vb < 64:
        rows[:, fw - 1] |= np.uint64(((1 << 64) - 1) ^ ((1 << vb) - 1)) & rng.integers(0, 2 ** 63, size=m, dtype=np.uint64)
    return rows


def test_fit_large_long_contexts(f2):
    """Wide contexts over many 64-row blocks: full rank reached mid-stream (consistency phase after it),
    rank-deficient streams with many dependent rows, contradictions before and after full rank."""
    rng = np.random.default_rng(4242)
    specs = [(513, 640, "uniform"), (575, 1300, "uniform"), (1000, 1100, "uniform"), (4095, 200, "uniform"),
             (700, 900, "pool"), (2047, 1500, "pool"), (4095, 1000, "pool"), (600, 2000, "mixed"),
             (513, 64, "pool"), (1024, 129, "uniform"), (3000, 3100, "uniform"), (1535, 1700, "mixed")]
    n_bits, rows_list = [], []
    for n, m, kind in specs:
        n_bits.append(n)
        rows_list.append(_large_context(rng, n, m, kind))
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    model, ref = _fit_and_compare(f2, wl)
    full = ref.rank == np.array([n + 1 for n in n_bits])
    assert full.sum() >= 4 and (~full).sum() >= 4        # both regimes exercised
    assert ((ref.flags & 1) != 0).sum() >= 6            # contradictions found


def test_group_barrier_timeout_is_reported(f2, monkeypatch):
    """A few wide contexts, each fitted by a group of workgroups that exchange partial
    sums across a bounded wait.  With the wait bound forced to zero from the host
    (F2GPU_GROUP_SPIN_LIMIT=0: every wait gives up at once) every kernel still
    finishes, every such context comes back flagged F2_CTX_SYNC_TIMEOUT, and its
    queries are reported as bad contexts; with the default bound the same batch
    matches the oracle and carries no such flag."""
    import torch
    rng = np.random.default_rng(91)
    n_bits, rows_list = [], []
    for k in range(8):
        n = int(rng.integers(600, 1200))
        n_bits.append(n)
        rows_list.append(_large_context(rng, n, 300, "uniform" if k % 2 else "pool"))
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    monkeypatch.setenv("F2GPU_GROUP_SPIN_LIMIT", "0")
    model = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    flags = parity.host(model.ctx_flags, np.uint32)[:wl.num_ctx]
    assert ((flags & f2.CTX_SYNC_TIMEOUT) != 0).all(), flags
    ctx = np.repeat(np.arange(wl.num_ctx, dtype=np.int32), 16)
    x = np.zeros(len(ctx) * 16, np.uint64)
    words, qf = f2.encode(model, parity.to_dev(ctx), parity.to_dev(x), 16)
    torch.cuda.synchronize()
    assert (parity.host(qf, np.uint8) == oracle.Q_BAD_CTX).all()
    assert not parity.host(words, np.uint64).any()
    monkeypatch.delenv("F2GPU_GROUP_SPIN_LIMIT")
    model2, ref = _fit_and_compare(f2, wl)
    assert not (parity.host(model2.ctx_flags, np.uint32)[:wl.num_ctx] & f2.CTX_SYNC_TIMEOUT).any()


@pytest.mark.parametrize("num_ctx", [100, 200])
def test_fit_many_wide_contexts(f2, num_ctx):
    """More wide contexts than a quarter (100) or half (200) of the workgroups: each context is then
    fitted by 2 workgroups or by 1, instead of 4."""
    rng = np.random.default_rng(num_ctx)
    n_bits, rows_list = [], []
    for c in range(num_ctx):
        n = int(rng.integers(512, 900))
        m = int(rng.integers(60, 700))
        n_bits.append(n)
        rows_list.append(_large_context(rng, n, m, ["uniform", "pool", "mixed"][c % 3]))
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    _fit_and_compare(f2, wl)


def test_fit_degenerate_contexts(f2):
    """n=0; 0 rows; all-zero rows; zero features with nonzero output; linear (bias 0) rows; duplicates."""
    rows_list, n_bits = [], []
    # n = 0: only the constant column
    n_bits.append(0); rows_list.append(np.array([[1, 5, 0], [1, 5, 0], [1, 6, 0], [0, 0, 0]], np.uint64))
    # 0 rows
    n_bits.append(10); rows_list.append(np.zeros((0, 3), np.uint64))
    # all-zero rows, then zero features with nonzero output
    n_bits.append(20); rows_list.append(np.array([[0, 0, 0], [0, 0, 0], [0, 1, 0], [0, 0, 1 << 63]], np.uint64))
    # linear rows (constant 0) and duplicates (App. B shape)
    n_bits.append(4); rows_list.append(np.array([[12, 159, 0], [8, 165, 0], [10, 102, 0], [6, 249, 0], [6, 248, 0], [12, 159, 0]], np.uint64))
    # 64-bit boundary: n = 63 (constant at bit 63), n = 64 (constant alone in word 1)
    n_bits.append(63); rows_list.append(np.array([[(1 << 63) | 5, 1, 2], [(1 << 63) | 3, 4, 8]], np.uint64))
    n_bits.append(64); rows_list.append(np.array([[5, 1, 1, 2], [3, 1, 4, 8], [0, 1, 7, 7]], np.uint64))
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    _fit_and_compare(f2, wl)


def test_fit_bad_segments_and_widths(f2):
    """Malformed segments, widths and output offsets are flagged per context; others still fit."""
    import torch
    wl = synth.fit_workload(2, num_ctx=8)
    n_bits = wl.n_bits.copy()
    row_off = wl.row_off.copy()
    n_bits[1] = 5000                       # too wide
    n_bits[2] = -3                         # negative width
    row_off[4] += 1                        # segment 3 no longer a multiple of the row size (and 4 shifted)
    layout_n = np.clip(n_bits, 0, oracle.MAX_N)
    ref = oracle.fit_batch(wl.rows, row_off, n_bits)
    from paper_2608_20532_amd import f2gpu
    model = f2gpu.Model(layout_n)
    model.n_bits = parity.to_dev(n_bits)
    model._struct = None
    nb = f2gpu.f2_fit_workspace_bytes(model.num_ctx)
    ws = f2gpu.workspace(nb)
    rows_d, off_d = parity.to_dev(wl.rows), parity.to_dev(row_off)
    assert f2gpu.f2_fit_batch(rows_d, wl.rows.size, off_d, model, ws, nb) == 0
    torch.cuda.synchronize()
    g = parity.model_to_host(model)
    assert g["flags"][1] == oracle.CTX_BAD_WIDTH and g["flags"][2] == oracle.CTX_BAD_WIDTH
    assert g["flags"][3] == oracle.CTX_BAD_SEGMENT
    assert np.array_equal(g["flags"], ref.flags) and np.array_equal(g["rank"], ref.rank)
    # output offsets past the buffers
    model2 = f2gpu.Model(wl.n_bits)
    bo = model2.basis_off_host.copy(); bo[5] = int(bo[-1])
    model2.basis_off = parity.to_dev(bo)
    model2._struct = None
    assert f2gpu.f2_fit_batch(parity.to_dev(wl.rows), wl.rows.size, parity.to_dev(wl.row_off), model2, ws, nb) == 0
    torch.cuda.synchronize()
    assert parity.host(model2.ctx_flags, np.uint32)[5] == oracle.CTX_BAD_OUTPUT


def test_fit_declared_width_bound(f2):
    """max_n_bits is a contract: a context wider than the declared bound is flagged
    F2_CTX_BAD_WIDTH with rank 0 and the others fit as usual, whether the bound lets
    the wide-context kernel launch or not."""
    import torch
    from paper_2608_20532_amd import f2gpu
    widths = [40, 100, 700, 63, 200, 511, 512]
    wl = _random_batch(5, widths)
    ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    rows_d, off_d = parity.to_dev(wl.rows), parity.to_dev(wl.row_off)
    for bound in (99, 511, 700, -1):
        print(f"declared width bound {bound}", flush=True)
        model = f2gpu.Model(wl.n_bits, max_n_bits=bound)
        nb = f2gpu.f2_fit_workspace_bytes(model.num_ctx)
        ws = f2gpu.workspace(nb)
        assert f2gpu.f2_fit_batch(rows_d, wl.rows.size, off_d, model, ws, nb) == 0
        torch.cuda.synchronize()
        g = parity.model_to_host(model)
        over = (wl.n_bits > bound) if bound >= 0 else np.zeros(len(widths), bool)
        assert (g["flags"][over] == oracle.CTX_BAD_WIDTH).all() and not g["rank"][over].any()
        ok = ~over
        for k, r in (("flags", ref.flags), ("rank", ref.rank), ("n_contra", ref.n_contra), ("first", ref.first_contra)):
            assert np.array_equal(g[k][ok], r[ok]), k
        for c in np.nonzero(ok)[0]:
            d, W, r = int(wl.n_bits[c]) + 1, (int(wl.n_bits[c]) + 64) // 64 + 2, int(ref.rank[c])
            mo, bo = int(ref.map_off[c]), int(ref.basis_off[c])
            assert np.array_equal(g["maps"][mo:mo + 2 * d], ref.maps[mo:mo + 2 * d]), f"maps of context {c}"
            assert np.array_equal(g["basis"][bo:bo + r * W], ref.basis[bo:bo + r * W]), f"basis of context {c}"


@pytest.mark.parametrize("num_ctx", [40, 1000, 5000])
def test_fit_invalid_contexts_each_launch_path(f2, num_ctx):
    """Invalid contexts among valid ones under a declared width bound below 512: the
    one-launch path of small batches (40 contexts) and the planned class kernels (1000,
    5000).  A width above the bound, two malformed segments and output offsets past the
    buffers are flagged with rank 0; every other context matches the oracle's fit of
    the unmodified batch."""
    import torch
    from paper_2608_20532_amd import f2gpu
    wl = synth.fit_workload(2, num_ctx=num_ctx)
    ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    n_bits = wl.n_bits.copy()
    row_off = wl.row_off.copy()
    n_bits[1] = 300                 # above the declared bound
    row_off[4] += 1                 # segments 3 and 4 no longer whole rows
    model = f2gpu.Model(n_bits, max_n_bits=127)
    bo = model.basis_off_host.copy()
    bo[6] = int(bo[-1])             # basis past the buffer
    model.basis_off = parity.to_dev(bo)
    model._struct = None
    nb = f2gpu.f2_fit_workspace_bytes(model.num_ctx)
    ws = f2gpu.workspace(nb)
    assert f2gpu.f2_fit_batch(parity.to_dev(wl.rows), wl.rows.size, parity.to_dev(row_off), model, ws, nb) == 0
    torch.cuda.synchronize()
    g = parity.model_to_host(model)
    assert g["flags"][1] == oracle.CTX_BAD_WIDTH
    assert g["flags"][3] == oracle.CTX_BAD_SEGMENT and g["flags"][4] == oracle.CTX_BAD_SEGMENT
    assert g["flags"][6] == oracle.CTX_BAD_OUTPUT
    bad = np.zeros(num_ctx, bool)
    bad[[1, 3, 4, 6]] = True
    assert not g["rank"][bad].any()
    ok = ~bad
    for k, r in (("flags", ref.flags), ("rank", ref.rank), ("n_contra", ref.n_contra), ("first", ref.first_contra)):
        assert np.array_equal(g[k][ok], r[ok]), k
    rb = ref.basis_off
    for c in np.nonzero(ok)[0][:300]:
        d, W, r = int(wl.n_bits[c]) + 1, (int(wl.n_bits[c]) + 64) // 64 + 2, int(ref.rank[c])
        assert np.array_equal(g["basis"][int(bo[c]):int(bo[c]) + r * W], ref.basis[int(rb[c]):int(rb[c]) + r * W]), c
        mo, rmo = int(model.map_off_host[c]), int(ref.map_off[c])
        assert np.array_equal(g["maps"][mo:mo + 2 * d], ref.maps[rmo:rmo + 2 * d]), c


def test_fit_host_errors(f2):
    from paper_2608_20532_amd import f2gpu
    wl = synth.fit_workload(1)
    model = f2gpu.Model(wl.n_bits)
    nb = f2gpu.f2_fit_workspace_bytes(1)
    ws = f2gpu.workspace(nb)
    rows_d, off_d = parity.to_dev(wl.rows), parity.to_dev(wl.row_off)
    assert f2gpu.f2_fit_batch(rows_d, wl.rows.size, off_d, model, ws, nb - 1) == f2gpu.F2_EWORKSPACE
    assert f2gpu.f2_fit_batch(rows_d, -1, off_d, model, ws, nb) == f2gpu.F2_EINVAL
    assert f2gpu.f2_fit_batch(rows_d, wl.rows.size, None, model, ws, nb) == f2gpu.F2_EINVAL


def test_fit_deterministic(f2):
    wl = synth.fit_workload(3, num_ctx=3000)
    a = parity.model_to_host(parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits))
    b = parity.model_to_host(parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits))
    ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    for k in ("rank", "flags", "n_contra", "first"):
        assert np.array_equal(a[k], b[k])
    assert np.array_equal(a["maps"], b["maps"])


def _encode_and_compare(f2, wl, model, ref, nq, stride, frac, zipf, sample=None):
    print(f"encode parity: recipe {wl.recipe}, {nq} queries, stride {stride}", flush=True)
    ctx, x, planted = synth.queries(wl, nq, stride, frac, zipf)
    words, qf = f2.encode(model, parity.to_dev(ctx), parity.to_dev(x), stride)
    import torch
    torch.cuda.synchronize()
    if sample is None:
        rw, rq = oracle.encode_batch(ref, ctx, x, stride)
        parity.compare_encode(words, qf, rw, rq)
    else:
        xs = x.reshape(nq, stride)[sample].reshape(-1)
        rw, rq = oracle.encode_batch(ref, ctx[sample], xs, stride)
        parity.compare_encode(words, qf, rw, rq, sample)
    return planted


@pytest.mark.parametrize("recipe,num_ctx,nq,stride,frac,zipf", [
    (1, 1, 1000, 1, 0.10, 0.0),
    (2, 4096, 1_000_000, 2, 0.02, 0.0),
    (3, 80000, 1_000_000, 4, 0.01, 1.1),
    (3, 6000, 400_000, 4, 0.01, 1.1),   # one context per sort bin: the staged wavefront path, stride 4
    (3, 10000, 400_000, 4, 0.01, 1.1),  # two contexts per bin, 40 queries per context: regrouped chunks
])
def test_encode_recipes(f2, recipe, num_ctx, nq, stride, frac, zipf):
    wl = synth.fit_workload(recipe, num_ctx=num_ctx)
    ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    model = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    _encode_and_compare(f2, wl, model, ref, nq, stride, frac, zipf)


def test_encode_random_widths_and_bad_ids(f2):
    rng = np.random.default_rng(5)
    widths = list(rng.integers(0, 600, size=60)) + [0, 63, 64, 4095]
    wl = _random_batch(11, widths, max_rows=120)
    ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    model = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    stride = 64
    nq = 20000
    ctx = rng.integers(-2, wl.num_ctx + 2, size=nq).astype(np.int32)
    x = np.zeros((nq, stride), np.uint64)
    for i in range(nq):
        c = int(ctx[i])
        if not (0 <= c < wl.num_ctx):
            continue
        n = int(wl.n_bits[c]); fw = (n + 64) // 64; W = fw + 2
        m = int(wl.m_rows[c])
        rows = wl.rows[wl.row_off[c]:wl.row_off[c + 1]].reshape(-1, W)
        mode = rng.integers(0, 4)
        if m and mode < 3:   # combination of training rows (constant bit stripped)
            sel = rows[rng.integers(0, m, size=int(rng.integers(1, 4)))]
            v = np.bitwise_xor.reduce(sel[:, :fw], axis=0)
            x[i, :fw] = v
            x[i, n // 64] &= ~(np.uint64(1) << np.uint64(n % 64))
        if mode == 2:        # one random bit anywhere in the stride (inside or outside the width)
            b = int(rng.integers(0, 64 * stride))
            x[i, b // 64] ^= np.uint64(1) << np.uint64(b % 64)
        if mode == 3:
            x[i] = rng.integers(0, 2 ** 63, size=stride, dtype=np.uint64) if rng.random() < 0.5 else 0
    words, qf = f2.encode(model, parity.to_dev(ctx), parity.to_dev(x.reshape(-1)), stride)
    import torch
    torch.cuda.synchronize()
    rw, rq = oracle.encode_batch(ref, ctx, x.reshape(-1), stride)
    parity.compare_encode(words, qf, rw, rq)
    assert (rq & oracle.Q_OUT_OF_SPAN).any() and (rq == 0).any() and (rq & oracle.Q_BAD_CTX).any()


def _encode_full_size(f2, wl, nq, stride, frac, zipf):
    """Fit a full-size workload on the GPU (checked against the oracle), encode a
    full-size query stream against it and compare every word and flag."""
    import torch
    model, ref = _fit_and_compare(f2, wl)
    ctx, x, planted = synth.queries(wl, nq, stride, frac, zipf)
    print(f"encode parity: {nq} queries, stride {stride}, all compared", flush=True)
    words, qf = f2.encode(model, parity.to_dev(ctx), parity.to_dev(x), stride)
    torch.cuda.synchronize()
    rw, rq = parity.oracle_encode_threads(ref, ctx, x, stride)
    parity.compare_encode(words, qf, rw, rq)
    assert abs(planted.mean() - frac) < 0.2 * frac
    return rq


def test_encode_recipe5_full_size(f2):
    """The 100M-query Zipf stream of the encode recipe at full size, every query compared."""
    wl = synth.fit_workload(5)
    nq, stride, frac, zipf = synth.QUERY_RECIPE[5]
    rq = _encode_full_size(f2, wl, nq, stride, frac, zipf)
    assert 0.008 < ((rq & oracle.Q_OUT_OF_SPAN) != 0).mean() < 0.012


def test_bench_step_full_size(f2):
    """The benchmark's default step exactly: the 80,000-context fit, then 100M Zipf queries
    (stride 4, 1% out of span) against the maps just fitted, every output compared."""
    wl = synth.fit_workload(3)
    _encode_full_size(f2, wl, 100_000_000, 4, 0.01, 1.1)


@pytest.mark.parametrize("stride", [3, 1, 7])
def test_encode_grouped_path_random_widths(f2, stride):
    """A batch large enough for the context-grouped encode, with every context class and
    bad ids mixed in; strides of 1 word (x read a word at a time), 3, and 7 (words past
    the first four checked for bits outside the width)."""
    rng = np.random.default_rng(21)
    widths = list(rng.integers(0, 190, size=300)) + list(rng.integers(190, 600, size=30)) + [0, 63, 64, 4095]
    wl = _random_batch(23, widths, max_rows=100)
    ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    model = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    nq = 200_000   # grouped from 196,608 queries (and 4 per context) on
    ctx = rng.integers(-3, wl.num_ctx + 3, size=nq).astype(np.int32)
    x = np.zeros((nq, stride), np.uint64)
    ok = (ctx >= 0) & (ctx < wl.num_ctx)
    # half the queries: the x of a training row with the constant set (in span when the width fits
    # the stride), half random junk
    for i in np.nonzero(ok)[0][: nq // 2]:
        c = int(ctx[i]); n = int(wl.n_bits[c]); fw = (n + 64) // 64; m = int(wl.m_rows[c])
        if m == 0:
            continue
        rows_c = wl.rows[wl.row_off[c]:wl.row_off[c + 1]].reshape(-1, fw + 2)
        affine = np.nonzero((rows_c[:, n // 64] >> np.uint64(n % 64)) & np.uint64(1))[0]
        if len(affine) == 0:
            continue
        row = rows_c[affine[int(rng.integers(0, len(affine)))]]
        k = min(stride, fw)
        x[i, :k] = row[:k]
        for w in range(k):  # keep only x_0 .. x_{n-1}: drop the constant and the row's padding bits
            lo = 64 * w
            if n - lo < 64:
                x[i, w] &= np.uint64((1 << max(n - lo, 0)) - 1)
    junk = np.nonzero(ok)[0][nq // 2:]
    x[junk] = rng.integers(0, 2 ** 63, size=(len(junk), stride), dtype=np.uint64) & np.uint64(0xFF)
    words, qf = f2.encode(model, parity.to_dev(ctx), parity.to_dev(x.reshape(-1)), stride)
    import torch
    torch.cuda.synchronize()
    rw, rq = oracle.encode_batch(ref, ctx, x.reshape(-1), stride)
    parity.compare_encode(words, qf, rw, rq)
    assert (rq == 0).sum() > 1000 and (rq & oracle.Q_OUT_OF_SPAN).sum() > 1000 and (rq & oracle.Q_BAD_CTX).any()


@pytest.mark.parametrize("stride", [1, 2, 5])
def test_encode_large_batch_random_widths(f2, stride):
    """A batch above 4,194,304 queries (fine sort bins; staged pass for contexts of up to
    2 feature words, second pass for wider ones and for crowded wavefronts) over every
    width class, with in-span queries, single-bit flips inside and outside the width,
    junk words and ids out of range; every query compared."""
    import torch
    rng = np.random.default_rng(100 + stride)
    widths = list(rng.integers(1, 140, size=300)) + [0, 0, 1, 2, 3, 62, 63, 64, 65, 126, 127, 128, 129, 255, 256,
                                                     300, 511, 600, 4095]
    wl = _random_batch(200 + stride, widths, max_rows=160)
    ref = parity.oracle_fit_threads(wl.rows, wl.row_off, wl.n_bits)
    model = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    C = wl.num_ctx
    # a pool of 8 candidate x per context: XOR of 1-3 training rows, the constant and padding dropped
    pool = np.zeros((C, 8, stride), np.uint64)
    for c in range(C):
        n = int(wl.n_bits[c]); fw = (n + 64) // 64; m = int(wl.m_rows[c])
        if m == 0:
            continue
        rows_c = wl.rows[wl.row_off[c]:wl.row_off[c + 1]].reshape(-1, fw + 2)
        for k in range(8):
            sel = rows_c[rng.integers(0, m, size=int(rng.integers(1, 4)))]
            v = np.bitwise_xor.reduce(sel[:, :fw], axis=0)
            for w in range(min(fw, stride)):
                lo = 64 * w
                keep = min(max(n - lo, 0), 64)
                pool[c, k, w] = v[w] & np.uint64((1 << keep) - 1)
    nq = 4_500_000
    ctx = rng.integers(-2, C + 2, size=nq).astype(np.int32)
    ok = (ctx >= 0) & (ctx < C)
    cc = np.where(ok, ctx, 0)
    x = pool[cc, rng.integers(0, 8, size=nq)].copy()
    mode = rng.integers(0, 10, size=nq)
    # mode 0-1: one random bit of the stride flipped (inside or outside the width); 2: junk; else as drawn
    flip = np.nonzero(mode <= 1)[0]
    b = rng.integers(0, 64 * stride, size=len(flip))
    x[flip, b // 64] ^= np.uint64(1) << (b % 64).astype(np.uint64)
    junk = np.nonzero(mode == 2)[0]
    x[junk] = rng.integers(0, 2 ** 63, size=(len(junk), stride), dtype=np.uint64) >> rng.integers(0, 64, size=(len(junk), 1)).astype(np.uint64)
    x = x.reshape(-1)
    print(f"large-batch encode parity: {nq} queries, stride {stride}, {C} contexts", flush=True)
    words, qf = f2.encode(model, parity.to_dev(ctx), parity.to_dev(x), stride)
    torch.cuda.synchronize()
    rw, rq = parity.oracle_encode_threads(ref, ctx, x, stride)
    parity.compare_encode(words, qf, rw, rq)
    assert (rq == 0).sum() > 300_000 and (rq & oracle.Q_OUT_OF_SPAN).sum() > 500_000
    assert (rq & oracle.Q_BAD_CTX).sum() > 10_000 and (rq & oracle.Q_CTX_CONTRADICTORY).any()


@pytest.mark.parametrize("stride", [2, 4])
def test_encode_unaligned_x(f2, stride):
    """x starting 8 bytes past a 16-byte boundary: the grouped passes take their
    word-by-word x loads instead of the 16-byte ones (recipe 2's maps, a grouped batch,
    5% of the queries outside the span); every query compared."""
    import torch
    wl = synth.fit_workload(2)
    ref = parity.oracle_fit_threads(wl.rows, wl.row_off, wl.n_bits)
    model = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    nq = 250_000  # grouped: 196,608 queries or more, four per context
    ctx, x, _ = synth.queries(wl, nq, stride, 0.05, 0.0)
    xd = parity.to_dev(np.concatenate([np.zeros(1, np.uint64), x]))[1:]
    assert xd.data_ptr() % 16 == 8
    print(f"unaligned-x encode parity: {nq} queries, stride {stride}", flush=True)
    words, qf = f2.encode(model, parity.to_dev(ctx), xd, stride)
    torch.cuda.synchronize()
    rw, rq = parity.oracle_encode_threads(ref, ctx, x, stride)
    parity.compare_encode(words, qf, rw, rq)
    assert (rq == 0).sum() > 200_000 and (rq & oracle.Q_OUT_OF_SPAN).sum() > 5_000


def _bad_context_model(f2):
    """40 contexts of recipe 2's shape with two malformed ones (1: too wide; 3: a segment
    that is not a whole number of rows), fitted on the GPU; returns (wl, oracle fit, model)."""
    wl = synth.fit_workload(2, num_ctx=40)
    n_bits = wl.n_bits.copy()
    row_off = wl.row_off.copy()
    n_bits[1] = 5000        # too wide
    row_off[4] += 1         # context 3: segment not a multiple of the row size
    ref = oracle.fit_batch(wl.rows, row_off, n_bits)
    model = f2.Model(np.clip(n_bits, 0, oracle.MAX_N))
    model.n_bits = parity.to_dev(n_bits)
    model._struct = None
    nb = f2.f2_fit_workspace_bytes(model.num_ctx)
    ws = f2.workspace(nb)
    assert f2.f2_fit_batch(parity.to_dev(wl.rows), wl.rows.size, parity.to_dev(row_off), model, ws, nb) == 0
    return wl, ref, model


def _bad_context_queries(wl, nq, stride, seed):
    """Queries of recipe 2's stream with ids out of range and queries of the malformed contexts."""
    ctx, x, _ = synth.queries(wl, nq, stride, 0.05, 0.0)
    rng = np.random.default_rng(seed)
    idx = rng.choice(nq, size=3000, replace=False)
    ctx[idx[:1000]] = rng.choice(np.array([-1, 40, 12345, -7], np.int32), size=1000)
    ctx[idx[1000:2000]] = 1
    ctx[idx[2000:]] = 3
    return ctx, x


def test_encode_sorted_and_gather_paths_agree_with_bad_contexts(f2):
    """One query batch through the context-grouped path (whole batch) and the per-query path
    (slices below its size threshold), against the oracle, with malformed contexts in the
    model and context ids out of range."""
    import torch
    wl, ref, model = _bad_context_model(f2)
    nq, stride = 240_000, 2   # the whole batch is grouped (196,608 queries or more), its halves are not
    ctx, x = _bad_context_queries(wl, nq, stride, 41)
    rw, rq = oracle.encode_batch(ref, ctx, x, stride)
    words, qf = f2.encode(model, parity.to_dev(ctx), parity.to_dev(x), stride)    # grouped path
    torch.cuda.synchronize()
    parity.compare_encode(words, qf, rw, rq)
    half = nq // 2
    for a, b in ((0, half), (half, nq)):                                          # per-query path
        w2, q2 = f2.encode(model, parity.to_dev(ctx[a:b]), parity.to_dev(x[a * stride:b * stride]), stride)
        torch.cuda.synchronize()
        parity.compare_encode(w2, q2, rw[a:b], rq[a:b])
    assert (rq & oracle.Q_BAD_CTX).sum() >= 3000 and (rq & oracle.Q_OUT_OF_SPAN).sum() > 1000
    # x at an 8-byte (not 16-byte) aligned address: the grouped path reads words one at a time
    xd = parity.to_dev(np.concatenate([np.zeros(1, np.uint64), x]))[1:]
    assert xd.data_ptr() % 16 == 8
    w3, q3 = f2.encode(model, parity.to_dev(ctx), xd, stride)
    torch.cuda.synchronize()
    parity.compare_encode(w3, q3, rw, rq)


@pytest.mark.parametrize("window", [None, 1_000_000, 300_007, 65_536])
def test_encode_windowed_sort_with_bad_contexts(f2, monkeypatch, window):
    """A batch above 4,194,304 queries (fine sort bins), sorted as one window or, with the
    window lowered from the host, window by window (5 windows of 1M, 15 of 300,007 rounded
    up to whole regroup chunks, about 60 of 65,536 with three count blocks each; a ragged
    last one); results written straight to their queries and only the nonzero flag bytes
    over the cleared ones.  Every query is checked, bad contexts and ids out of range
    included."""
    import torch
    wl, ref, model = _bad_context_model(f2)
    nq, stride = 4_300_000, 2
    ctx, x = _bad_context_queries(wl, nq, stride, 43)
    rw, rq = oracle.encode_batch(ref, ctx, x, stride)
    if window is not None:
        monkeypatch.setenv("F2GPU_ENCODE_WINDOW", str(window))
    words, qf = f2.encode(model, parity.to_dev(ctx), parity.to_dev(x), stride)
    torch.cuda.synchronize()
    parity.compare_encode(words, qf, rw, rq)
    assert (rq & oracle.Q_BAD_CTX).sum() >= 3000 and (rq & oracle.Q_OUT_OF_SPAN).sum() > 100_000
    assert (rq & oracle.Q_CTX_CONTRADICTORY).any() and (rq == 0).sum() > 1_000_000


def _late_pivot_batch(seed, widths, rows_choices, kmax=40):
    """Long contexts whose rows first span a small subspace and only later reveal new
    pivots (one generator added every few hundred rows), with contradictions late."""
    rng = np.random.default_rng(seed)
    n_bits, rows_list = [], []
    for n in widths:
        n = int(n)
        fw = (n + 64) // 64
        d = n + 1
        m = int(rng.choice(rows_choices))
        k = int(rng.integers(1, min(d, kmax) + 1))
        pool = rng.integers(0, 2 ** 63, size=(k, fw), dtype=np.uint64) ^ (rng.integers(0, 2, size=(k, fw), dtype=np.uint64) << np.uint64(63))
        vb = d - 64 * (fw - 1)
        if vb < 64:
            pool[:, fw - 1] &= np.uint64((1 << vb) - 1)
        Wp = rng.integers(0, 2 ** 63, size=(k, 2), dtype=np.uint64)
        rows = np.zeros((m, fw + 2), np.uint64)
        for i in range(m):
            avail = max(1, min(k, 1 + (i * k) // max(1, m)))   # generators unlocked gradually
            sel = rng.integers(0, 2, size=avail).astype(bool)
            rows[i, :fw] = np.bitwise_xor.reduce(pool[:avail][sel], axis=0) if sel.any() else 0
            rows[i, fw:] = np.bitwise_xor.reduce(Wp[:avail][sel], axis=0) if sel.any() else 0
            if rng.random() < (0.01 if n % 2 else 0.0002):
                rows[i, fw + int(rng.integers(0, 2))] ^= np.uint64(1) << np.uint64(int(rng.integers(0, 64)))
        n_bits.append(n)
        rows_list.append(rows)
    return synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)


def test_fit_long_contexts_late_pivots(f2):
    rng = np.random.default_rng(31)
    widths = [int(w) for w in rng.integers(0, 512, size=40)] + [0, 63, 64, 127, 191, 192, 255, 256, 319, 447, 511]
    _fit_and_compare(f2, _late_pivot_batch(31, widths, [200, 257, 300, 700, 1500, 2600]))


def test_fit_long_high_rank_contexts(f2):
    """Long contexts of 2-4 feature words whose rank grows past 100 over many rounds: the
    LDS basis reduces through Four-Russians tables (rebuilt after each growth), for widths
    whose positions outrun the tables too (d = 256)."""
    widths = [100, 130, 150, 191, 200, 230, 250, 255, 254, 180, 120, 240]
    _fit_and_compare(f2, _late_pivot_batch(57, widths, [1100, 1800, 3000], kmax=256))


def _subspace_rows(rng, n, m, k, contra_rows=(), grow_rows=()):
    """m rows of width n whose features come from a k-dimensional subspace (random
    generators, constant bit included as drawn), outputs linear in the generators;
    the listed rows get a flipped output bit (contradictions) or a fresh random
    feature vector (a new pivot, unless it happens to lie in the span)."""
    fw = (n + 64) // 64
    d = n + 1
    vb = d - 64 * (fw - 1)
    top = np.uint64(((1 << vb) - 1) if vb < 64 else (1 << 64) - 1)
    pool = rng.integers(0, 2 ** 63, size=(k, fw), dtype=np.uint64) ^ (rng.integers(0, 2, size=(k, fw), dtype=np.uint64) << np.uint64(63))
    pool[:, fw - 1] &= top
    Wp = rng.integers(0, 2 ** 63, size=(k, 2), dtype=np.uint64)
    rows = np.zeros((m, fw + 2), np.uint64)
    sel = rng.integers(0, 2, size=(m, k)).astype(bool)
    for i in range(m):
        rows[i, :fw] = np.bitwise_xor.reduce(pool[sel[i]], axis=0) if sel[i].any() else 0
        rows[i, fw:] = np.bitwise_xor.reduce(Wp[sel[i]], axis=0) if sel[i].any() else 0
    for i in contra_rows:
        rows[i, fw] ^= np.uint64(1) << np.uint64(int(rng.integers(0, 64)))
    for i in grow_rows:
        rows[i, :fw] = rng.integers(0, 2 ** 63, size=fw, dtype=np.uint64) ^ (rng.integers(0, 2, size=fw, dtype=np.uint64) << np.uint64(63))
        rows[i, fw - 1] &= top
        rows[i, fw:] = rng.integers(0, 2 ** 63, size=2, dtype=np.uint64)
    return rows


def test_fit_late_rows_after_saturation(f2):
    """Long contexts at every width class (one to eight feature words), of full rank
    and of low rank (rank below d / 2), whose rank saturates early: contradictions
    only long after saturation (counted, first row kept), a new pivot at the very
    last row, one deep inside the stream, one right after the first blocks of 64,
    and a contradiction among the first rows.  More than 64 contexts, so the
    planned path (class lists, LDS-basis and register kernels) runs."""
    rng = np.random.default_rng(2026)
    cases = []
    for n in (20, 40, 63, 100, 150, 191, 200, 255, 300, 447, 511):
        d = n + 1
        for k in (max(1, d // 8), min(d, int(0.7 * d) + 1)):
            cases.append((n, 3 * d + 400, k, (3 * d + 100, 3 * d + 101, 3 * d + 399), ()))   # contradictions late
            cases.append((n, 3 * d + 400, k, (5,), (3 * d + 399,)))                           # new pivot at the end
            cases.append((n, 2 * d + 300, k, (), (2 * d + 150,)))                             # new pivot mid-suffix
        cases.append((n, d + 700, min(d, 30), (d + 650,), (64 * ((d + 95) // 64),)))           # right after the first blocks
    n_bits, rows_list = [], []
    for (n, m, k, contra, grow) in cases:
        n_bits.append(n)
        rows_list.append(_subspace_rows(rng, n, m, k, contra, grow))
    # filler contexts: more than the small-batch bound, so the planned path runs
    for i in range(80):
        n = int(rng.integers(0, 200))
        n_bits.append(n)
        rows_list.append(_subspace_rows(rng, n, int(rng.integers(0, 300)), int(rng.integers(1, n + 2))))
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    model, ref = _fit_and_compare(f2, wl)
    assert (ref.n_contra[:len(cases)] > 0).sum() >= 20


def _ctx_outputs(h, model, i):
    """Every output of context i of a fitted model (host copy h), independent of its position in the batch."""
    r = int(h["rank"][i])
    n = int(h["n_bits"][i])
    fw = (n + 64) // 64
    W = fw + 2
    bo, po, mo = int(model.basis_off_host[i]), int(model.piv_off_host[i]), int(model.map_off_host[i])
    t = (n + 1) - r
    tables = h["tables"][bo:bo + t * fw] if t <= r else np.zeros(0, np.uint64)
    return (r, int(h["flags"][i]), int(h["n_contra"][i]), int(h["first"][i]),
            h["basis"][bo:bo + r * W].tobytes(), h["pivots"][po:po + r].tobytes(),
            h["maps"][mo:mo + 2 * (n + 1)].tobytes(), tables.tobytes())


def _fit_subset(f2, wl, order):
    """Fit the contexts of wl in the given order (a list of context indices) as one batch."""
    rows = [wl.rows[wl.row_off[c]:wl.row_off[c + 1]].reshape(-1, (int(wl.n_bits[c]) + 64) // 64 + 2) for c in order]
    sub = synth.custom_workload(wl.n_bits[order], [len(r) for r in rows], rows)
    model = parity.gpu_fit(f2, sub.rows, sub.row_off, sub.n_bits)
    h = parity.model_to_host(model)
    h["n_bits"] = np.asarray(sub.n_bits)
    return model, h


def test_fit_deterministic_across_launch_geometries(f2):
    """The same contexts fitted under different launch geometries give identical outputs:
    a batch of at most 64 contexts (one workgroup per context, no plan) against the same
    contexts spread through a batch of 3,000 (plan, class kernels, different workgroups
    and list positions); wide contexts fitted by groups of 4, 2 and 1 workgroups (alone,
    among 100 and among 200 other wide contexts)."""
    rng = np.random.default_rng(77)
    widths = [int(w) for w in rng.integers(0, 512, size=36)] + [0, 63, 64, 511]
    small = _random_batch(78, widths, max_rows=600)
    filler = synth.fit_workload(3, num_ctx=3000)
    # one workload holding both: the 40 targets first, then the filler contexts
    rows = [small.rows[small.row_off[c]:small.row_off[c + 1]].reshape(-1, (int(small.n_bits[c]) + 64) // 64 + 2)
            for c in range(small.num_ctx)]
    rows += [filler.rows[filler.row_off[c]:filler.row_off[c + 1]].reshape(-1, (int(filler.n_bits[c]) + 64) // 64 + 2)
             for c in range(filler.num_ctx)]
    both = synth.custom_workload(list(small.n_bits) + list(filler.n_bits), [len(r) for r in rows], rows)
    T = small.num_ctx
    m1, h1 = _fit_subset(f2, both, list(range(T)))                      # small-batch kernel
    pos = rng.permutation(both.num_ctx)                                 # targets at random list positions
    m2, h2 = _fit_subset(f2, both, list(pos))
    inv = np.argsort(pos)
    for i in range(T):
        assert _ctx_outputs(h1, m1, i) == _ctx_outputs(h2, m2, int(inv[i])), f"context {i} (n={widths[i]})"
    ref = oracle.fit_batch(small.rows, small.row_off, small.n_bits)
    parity.compare_fit(m1, ref)

    # wide contexts: groups of 4 (alone), 2 (with 100 others) and 1 (with 200 others)
    wide_rows, wide_n = [], []
    for n, m, kind in ((700, 900, "uniform"), (1500, 400, "pool"), (2100, 2300, "mixed")):
        wide_n.append(n)
        wide_rows.append(_large_context(rng, n, m, kind))
    fill_n = [512 + int(k) for k in rng.integers(0, 200, size=200)]
    fill_rows = [_large_context(rng, n, 40, "pool") for n in fill_n]
    allw = synth.custom_workload(wide_n + fill_n, [len(r) for r in wide_rows + fill_rows], wide_rows + fill_rows)
    outs = []
    for extra in (0, 100, 200):
        mw, hw = _fit_subset(f2, allw, list(range(3 + extra)))
        outs.append([_ctx_outputs(hw, mw, i) for i in range(3)])
    assert outs[0] == outs[1] == outs[2]


@pytest.mark.parametrize("stride,chunk", [(4, 1_000_003), (5, 150_001)])
def test_encode_chunked_batches_match(f2, monkeypatch, stride, chunk):
    """Batches above the chunk size (2^30 queries) are encoded chunk by chunk; with the
    chunk lowered from the host, 3M queries in chunks of about 1M (grouped path, ragged
    tail) and of 150,001 (gather path; with stride 5 the chunks' x start at odd word
    offsets) give the words and flags of the one-call encode, which matches the oracle."""
    import torch
    wl = synth.fit_workload(3)
    model = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
    nq = 3_000_000
    ctx, x, planted = synth.queries(wl, nq, stride, 0.01, 1.1)
    ctx_d, x_d = parity.to_dev(ctx), parity.to_dev(x)
    w0, q0 = f2.encode(model, ctx_d, x_d, stride)
    monkeypatch.setenv("F2GPU_ENCODE_CHUNK", str(chunk))
    w1, q1 = f2.encode(model, ctx_d, x_d, stride)
    monkeypatch.delenv("F2GPU_ENCODE_CHUNK")
    torch.cuda.synchronize()
    assert torch.equal(w0, w1) and torch.equal(q0, q1)
    ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
    sel = np.sort(np.random.default_rng(5).choice(nq, 100_000, replace=False))
    rw, rq = oracle.encode_batch(ref, ctx[sel], x.reshape(nq, stride)[sel].reshape(-1), stride)
    assert np.array_equal(w1.cpu().numpy().view(np.uint64)[sel], rw.reshape(-1, 2))
    assert np.array_equal(q1.cpu().numpy()[sel], rq)
