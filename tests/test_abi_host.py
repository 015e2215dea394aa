"""Host-side checks of the C-ABI library (no GPU needed): it loads, exports every
entry point include/f2gpu.h declares, and its host helpers follow the documented
layout and argument rules."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions(header="f2gpu.h", prefix="f2_"):
    src = open(os.path.join(ROOT, "include", header)).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(" + prefix + r"[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    from paper_2608_20532_amd import f2gpu
    names = declared_functions()
    assert len(names) >= 6
    L = ctypes.CDLL(f2gpu.LIB_PATH)
    for name in names:
        assert hasattr(L, name), name
    assert set(f2gpu.EXPORTS) == set(names)


def test_probe_library_exports_every_declared_symbol():
    from paper_2608_20532_amd import f2probe
    names = declared_functions("f2probe.h", "f2probe_")
    assert len(names) == 3
    L = ctypes.CDLL(f2probe.LIB_PATH)
    for name in names:
        assert hasattr(L, name), name
    assert set(f2probe.EXPORTS) == set(names)
    # argument errors return before any device work
    assert L.f2probe_copy(None, None, 4, None) == -1
    assert L.f2probe_copy(None, None, 0, None) == 0
    assert L.f2probe_bitops(None, 1, 1, 0, None) == -1
    L.f2probe_scatter.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_void_p, ctypes.c_void_p]
    assert L.f2probe_scatter(None, 1 << 20, 1, 1, 1, None, None) == -1


def test_layout_matches_documented_capacities():
    from paper_2608_20532_amd import f2gpu
    n = np.array([0, 1, 62, 63, 64, 127, 128, 4095, 33], np.int32)
    got = f2gpu.f2_fit_layout(n)
    want = oracle.layout(n)   # the oracle's own copy of the documented rule
    for g, w in zip(got, want):
        assert np.array_equal(g, w)


def test_layout_errors():
    from paper_2608_20532_amd import f2gpu
    with pytest.raises(RuntimeError, match="F2_MAX_N_BITS|above"):
        f2gpu.f2_fit_layout(np.array([4096], np.int32))
    with pytest.raises(RuntimeError, match="invalid"):
        f2gpu.f2_fit_layout(np.array([-1], np.int32))
    assert f2gpu.f2_fit_layout(np.zeros(0, np.int32))[0].tolist() == [0]


def test_status_strings_and_workspace_sizes():
    from paper_2608_20532_amd import f2gpu
    for st in (0, -1, -2, -3, -4, -5):
        assert f2gpu.f2_status_string(st) != "unknown status"
    assert f2gpu.f2_status_string(7) == "unknown status"
    assert f2gpu.f2_fit_workspace_bytes(-1) == 0
    # the fit plan holds a context list and a sort key per context
    assert f2gpu.f2_fit_workspace_bytes(100_000) >= 8 * 100_000 > f2gpu.f2_fit_workspace_bytes(10) > 0
    assert f2gpu.f2_fit_workspace_bytes(10) % 256 == 0
    m = f2gpu.f2_model()
    m.num_ctx, m.basis_words = 10, 1000
    small = f2gpu.lib.f2_encode_workspace_bytes(ctypes.byref(m), 1000)
    big = f2gpu.lib.f2_encode_workspace_bytes(ctypes.byref(m), 1 << 20)
    assert 0 < small <= big and small % 256 == 0 and big % 256 == 0
    assert f2gpu.lib.f2_encode_workspace_bytes(ctypes.byref(m), -1) == 0


def test_encode_workspace_is_one_chunk(monkeypatch):
    """Batches above the chunk size are encoded chunk by chunk through one chunk-sized
    workspace: 2^30 queries by default, less under F2GPU_ENCODE_CHUNK."""
    from paper_2608_20532_amd import f2gpu
    m = f2gpu.f2_model()
    m.num_ctx, m.basis_words = 80_000, 1000
    ws = lambda q: f2gpu.lib.f2_encode_workspace_bytes(ctypes.byref(m), q)
    assert ws(3 << 30) == ws(1 << 30) > ws((1 << 30) - (1 << 20)) > 0
    monkeypatch.setenv("F2GPU_ENCODE_CHUNK", "1000003")
    assert ws(50_000_000) == ws(1_000_003)
    for bad in ("0", "-5", "x", str((1 << 30) + 1)):   # ignored: the default chunk
        monkeypatch.setenv("F2GPU_ENCODE_CHUNK", bad)
        assert ws(3 << 30) == ws(1 << 30)


def test_calls_with_bad_host_arguments_enqueue_nothing():
    """Argument errors are returned before any device work (so these run without a GPU)."""
    from paper_2608_20532_amd import f2gpu
    L = f2gpu.lib
    assert L.f2_fit_batch(None, 0, None, None, None, 0, None) == f2gpu.F2_EINVAL
    m = f2gpu.f2_model()
    m.num_ctx = -1
    assert L.f2_fit_batch(None, 0, None, ctypes.byref(m), None, 0, None) == f2gpu.F2_EINVAL
    m.num_ctx = 0
    assert L.f2_fit_batch(None, 0, None, ctypes.byref(m), None, 0, None) == f2gpu.F2_OK   # nothing to do
    assert L.f2_encode_batch(ctypes.byref(m), None, None, 0, 5, None, None, None, 0, None) == f2gpu.F2_EINVAL
    assert L.f2_encode_batch(ctypes.byref(m), None, None, 1, 0, None, None, None, 0, None) == f2gpu.F2_OK
    m.num_ctx = 3
    assert L.f2_fit_batch(None, 0, None, ctypes.byref(m), None, 0, None) == f2gpu.F2_EINVAL


def test_vectorize_and_merge_argument_errors():
    """The row builder and the word merge reject bad sizes before any device work."""
    from paper_2608_20532_amd import f2gpu
    keep = (2 ** 64 - 1, 2 ** 64 - 1)
    V = f2gpu.f2_vectorize_rows
    assert V(None, None, 10, 64, keep, None, 0) == f2gpu.F2_EINVAL       # k above 63
    assert V(None, None, 10, -1, keep, None, 0) == f2gpu.F2_EINVAL
    assert V(None, None, -1, 2, keep, None, 0) == f2gpu.F2_EINVAL
    assert V(None, None, 0, 2, keep, None, 0) == f2gpu.F2_OK              # nothing to do
    assert V(None, None, 5, 2, keep, None, 0) == f2gpu.F2_EINVAL          # values and output missing
    assert f2gpu.lib.f2_vectorize_rows(None, None, 5, 0, None, None, None) == f2gpu.F2_EINVAL  # no keep mask
    M = f2gpu.f2_merge_words

    class Fake:  # a non-null device pointer stand-in: the call must fail before using it
        def data_ptr(self):
            return 256
    f = Fake()
    for shift, width in ((0, 0), (0, 65), (-1, 5), (100, 29), (64, 65)):
        assert M(f, f, shift, width, (0, 0), None, 8, f, 0) == f2gpu.F2_EINVAL, (shift, width)
    assert M(None, None, 0, 0, (0, 0), None, 0, None, 0) == f2gpu.F2_OK
    assert M(None, None, 0, 0, (0, 0), None, 3, None, 0) == f2gpu.F2_EINVAL
    assert M(f, None, 0, 0, (0, 0), None, -2, f, 0) == f2gpu.F2_EINVAL
    assert f2gpu.lib.f2_merge_words(None, None, 0, 0, None, None, 0, None, None) == f2gpu.F2_EINVAL


def test_noalloc_fit_rejects_batches_beyond_its_fixed_plan():
    """The allocation-free fit refuses more contexts than its fixed plan holds, and bad
    arguments, before any device work."""
    from paper_2608_20532_amd import f2gpu
    m = f2gpu.f2_model()
    for name in ("n_bits", "basis_off", "piv_off", "map_off", "basis", "pivots", "maps", "tables", "rank",
                 "ctx_flags", "n_contra", "first_contra_row"):
        setattr(m, name, 256)
    m.num_ctx = f2gpu.F2_NOALLOC_MAX_CTX + 1
    L = f2gpu.lib
    assert L.f2_fit_batch_noalloc(256, 0, 256, ctypes.byref(m), None) == f2gpu.F2_ESCRATCH
    assert "allocation-free" in f2gpu.f2_status_string(f2gpu.F2_ESCRATCH)
    m.num_ctx = 0
    assert L.f2_fit_batch_noalloc(None, 0, None, ctypes.byref(m), None) == f2gpu.F2_OK
    m.num_ctx = 5
    assert L.f2_fit_batch_noalloc(None, 0, None, ctypes.byref(m), None) == f2gpu.F2_EINVAL
    assert L.f2_fit_batch_noalloc(None, 0, None, None, None) == f2gpu.F2_EINVAL
