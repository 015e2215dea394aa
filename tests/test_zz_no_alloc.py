"""The allocation-free fit (f2_fit_batch_noalloc: the plan in the library's fixed
device array, no workspace) against the workspace fit (f2_fit_batch) on the same
inputs, every defined output compared bit for bit, over consecutive calls that
share the array: the 80,000-context workload, then a batch of wide contexts (the
grouped wide-context kernel keeps its barrier counters in the plan), then a smaller
batch of 300 contexts."""
import numpy as np
import pytest

import oracle
import parity
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def f2(require_gpu):
    from paper_2608_20532_amd import f2gpu
    return f2gpu


def _wide_batch(seed, count):
    rng = np.random.default_rng(seed)
    n_bits, rows_list = [], []
    for _ in range(count):
        n = int(rng.integers(512, 1500))
        fw = (n + 64) // 64
        m = int(rng.integers(100, 900))
        x = rng.integers(0, 2 ** 63, size=(m, fw), dtype=np.uint64) << np.uint64(1)
        x ^= rng.integers(0, 2, size=(m, fw), dtype=np.uint64)
        vb = n + 1 - 64 * (fw - 1)
        if vb < 64:
            x[:, fw - 1] &= np.uint64((1 << vb) - 1)
        x[:, n // 64] |= np.uint64(1 << (n % 64))
        y = rng.integers(0, 2 ** 63, size=(m, 2), dtype=np.uint64)
        rows = np.concatenate([x, y], axis=1)
        rows[m // 2:] = rows[rng.integers(0, m // 2, size=m - m // 2)]   # repeated rows (redundant)
        rows[m - 1, fw] ^= np.uint64(1)                                   # and a contradictory one
        n_bits.append(n)
        rows_list.append(rows)
    return synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)


def _compare_models(a, b, n_bits):
    ga, gb = parity.model_to_host(a), parity.model_to_host(b)
    for k in ("rank", "flags", "n_contra", "first"):
        assert np.array_equal(ga[k], gb[k]), k
    n = np.asarray(n_bits, np.int64)
    W = (n + 64) // 64 + 2
    r = ga["rank"].astype(np.int64)
    for c in range(len(n)):
        p0, b0, m0 = int(a.piv_off_host[c]), int(a.basis_off_host[c]), int(a.map_off_host[c])
        assert np.array_equal(ga["pivots"][p0:p0 + r[c]], gb["pivots"][p0:p0 + r[c]]), c
        assert np.array_equal(ga["basis"][b0:b0 + r[c] * W[c]], gb["basis"][b0:b0 + r[c] * W[c]]), c
        assert np.array_equal(ga["maps"][m0:m0 + 2 * (n[c] + 1)], gb["maps"][m0:m0 + 2 * (n[c] + 1)]), c
        d = int(n[c]) + 1
        if d - r[c] <= r[c]:  # parity-check rows present
            t = (d - r[c]) * ((n[c] + 64) // 64)
            assert np.array_equal(ga["tables"][b0:b0 + t], gb["tables"][b0:b0 + t]), c


def test_noalloc_fit_matches_workspace_fit(f2):
    import torch
    batches = [synth.fit_workload(3), _wide_batch(7, 20), synth.fit_workload(2, num_ctx=300)]
    for wl in batches:
        print(f"no-alloc fit: {wl.num_ctx} contexts, {wl.total_rows} rows", flush=True)
        ref = parity.gpu_fit(f2, wl.rows, wl.row_off, wl.n_bits)
        model = f2.Model(wl.n_bits)
        rows_d = parity.to_dev(wl.rows)
        off_d = parity.to_dev(wl.row_off)
        assert f2.f2_fit_batch_noalloc(rows_d, rows_d.numel(), off_d, model) == f2.F2_OK
        torch.cuda.synchronize()
        _compare_models(model, ref, wl.n_bits)
    # and the allocation-free fit of the wide batch agrees with the oracle too
    wl = batches[1]
    model = f2.Model(wl.n_bits)
    rows_d, off_d = parity.to_dev(wl.rows), parity.to_dev(wl.row_off)
    assert f2.f2_fit_batch_noalloc(rows_d, rows_d.numel(), off_d, model) == f2.F2_OK
    torch.cuda.synchronize()
    parity.compare_fit(model, oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits))
