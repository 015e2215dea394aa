"""Thin ctypes binding of ``libf2gpu.so`` (declared in ``include/f2gpu.h``).

Functions carry the C names and only marshal arguments: every step of fit and
encode runs in the HIP kernels of the library.  PyTorch supplies device memory
(``tensor.data_ptr()``) and the stream (``torch.cuda.current_stream()``).
uint64 buffers are held in ``torch.int64`` tensors (bit patterns).

If the library is not built this module raises on import: there is no CPU
fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# F2GPU_LIB may name another build of the same source (the host-sanitizer build of the CPU tests)
LIB_PATH = os.environ.get("F2GPU_LIB") or os.path.join(_HERE, "libf2gpu.so")

F2_OK, F2_EINVAL, F2_EWORKSPACE, F2_EDEVICE, F2_ETOOWIDE, F2_ESCRATCH = 0, -1, -2, -3, -4, -5
F2_NOALLOC_MAX_CTX = 131072
F2_MAX_N_BITS = 4095
CTX_CONTRADICTION, CTX_BAD_SEGMENT, CTX_BAD_WIDTH, CTX_BAD_OUTPUT, CTX_SYNC_TIMEOUT = 1, 2, 4, 8, 16
Q_OUT_OF_SPAN, Q_CTX_CONTRADICTORY, Q_BAD_CTX = 1, 2, 4
POOL_SHARED, POOL_CONTRADICTION, POOL_WIDTH_MISMATCH, POOL_MASK_MISMATCH, POOL_BAD_MEMBER = 1, 2, 4, 8, 16

# every entry point the header declares
EXPORTS = ("f2_fit_layout", "f2_fit_workspace_bytes", "f2_fit_batch", "f2_fit_batch_noalloc", "f2_encode_workspace_bytes",
           "f2_encode_batch", "f2_vectorize_rows", "f2_merge_words", "f2_pool_workspace_bytes", "f2_pool_bases",
           "f2_group_workspace_bytes", "f2_group_rows", "f2_status_string")


class f2_model(ctypes.Structure):
    _fields_ = [
        ("num_ctx", ctypes.c_int32),
        ("n_bits", ctypes.c_void_p),
        ("basis_off", ctypes.c_void_p),
        ("piv_off", ctypes.c_void_p),
        ("map_off", ctypes.c_void_p),
        ("basis_words", ctypes.c_int64),
        ("piv_entries", ctypes.c_int64),
        ("map_words", ctypes.c_int64),
        ("basis", ctypes.c_void_p),
        ("pivots", ctypes.c_void_p),
        ("maps", ctypes.c_void_p),
        ("tables", ctypes.c_void_p),
        ("rank", ctypes.c_void_p),
        ("ctx_flags", ctypes.c_void_p),
        ("n_contra", ctypes.c_void_p),
        ("first_contra_row", ctypes.c_void_p),
        ("max_n_bits", ctypes.c_int32),
    ]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run __graft_entry__.build() (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    MP = ctypes.POINTER(f2_model)
    L.f2_fit_layout.argtypes = [P, i32, P, P, P]
    L.f2_fit_layout.restype = ctypes.c_int
    L.f2_fit_workspace_bytes.argtypes = [i32]
    L.f2_fit_workspace_bytes.restype = sz
    L.f2_fit_batch.argtypes = [P, i64, P, MP, P, sz, P]
    L.f2_fit_batch.restype = ctypes.c_int
    L.f2_fit_batch_noalloc.argtypes = [P, i64, P, MP, P]
    L.f2_fit_batch_noalloc.restype = ctypes.c_int
    L.f2_encode_workspace_bytes.argtypes = [MP, i64]
    L.f2_encode_workspace_bytes.restype = sz
    L.f2_encode_batch.argtypes = [MP, P, P, i32, i64, P, P, P, sz, P]
    L.f2_encode_batch.restype = ctypes.c_int
    L.f2_vectorize_rows.argtypes = [P, P, i64, i32, P, P, P]
    L.f2_vectorize_rows.restype = ctypes.c_int
    L.f2_merge_words.argtypes = [P, P, i32, i32, P, P, i64, P, P]
    L.f2_merge_words.restype = ctypes.c_int
    L.f2_pool_workspace_bytes.argtypes = [MP, i32]
    L.f2_pool_workspace_bytes.restype = sz
    L.f2_pool_bases.argtypes = [MP, P, P, P, i64, MP, P, P, sz, P]
    L.f2_pool_bases.restype = ctypes.c_int
    L.f2_group_workspace_bytes.argtypes = [i32, i64]
    L.f2_group_workspace_bytes.restype = sz
    L.f2_group_rows.argtypes = [P, P, i32, i64, P, i32, P, i64, P, P, P, sz, P]
    L.f2_group_rows.restype = ctypes.c_int
    L.f2_status_string.argtypes = [ctypes.c_int]
    L.f2_status_string.restype = ctypes.c_char_p
    return L


lib = _load()


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream(stream) -> int:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    return int(stream) if isinstance(stream, int) else int(stream.cuda_stream)


def f2_status_string(status: int) -> str:
    return lib.f2_status_string(status).decode()


def _check(status: int, what: str):
    if status != F2_OK:
        raise RuntimeError(f"{what}: {f2_status_string(status)} ({status})")


def f2_fit_layout(n_bits_host):
    """Host helper: (basis_off, piv_off, map_off) int64 numpy arrays of num_ctx+1 entries."""
    n = np.ascontiguousarray(n_bits_host, np.int32)
    C = len(n)
    offs = [np.zeros(C + 1, np.int64) for _ in range(3)]
    st = lib.f2_fit_layout(n.ctypes.data if C else None, C, *(o.ctypes.data for o in offs))
    _check(st, "f2_fit_layout")
    return tuple(offs)


def f2_fit_workspace_bytes(num_ctx: int) -> int:
    return int(lib.f2_fit_workspace_bytes(num_ctx))


def f2_encode_workspace_bytes(model: "Model", num_queries: int) -> int:
    return int(lib.f2_encode_workspace_bytes(ctypes.byref(model.struct()), int(num_queries)))


class Model:
    """Device buffers of a fitted model (the f2_model struct), allocated with torch."""

    def __init__(self, n_bits_host, device="cuda", max_n_bits=None):
        import torch
        n_bits_host = np.ascontiguousarray(n_bits_host, np.int32)
        self.num_ctx = len(n_bits_host)
        self.n_bits_host = n_bits_host
        # declared width bound (f2_model.max_n_bits): the largest width by default
        self.max_n_bits = (int(n_bits_host.max()) if self.num_ctx else 0) if max_n_bits is None else int(max_n_bits)
        bo, po, mo = f2_fit_layout(n_bits_host)
        self.basis_off_host, self.piv_off_host, self.map_off_host = bo, po, mo
        dev = torch.device(device)
        C = max(self.num_ctx, 1)
        self.n_bits = torch.from_numpy(n_bits_host.copy()).to(dev) if self.num_ctx else torch.zeros(1, dtype=torch.int32, device=dev)
        self.basis_off = torch.from_numpy(bo).to(dev)
        self.piv_off = torch.from_numpy(po).to(dev)
        self.map_off = torch.from_numpy(mo).to(dev)
        self.basis = torch.zeros(max(int(bo[-1]), 1), dtype=torch.int64, device=dev)
        self.pivots = torch.zeros(max(int(po[-1]), 1), dtype=torch.int32, device=dev)
        self.maps = torch.zeros(max(int(mo[-1]), 1), dtype=torch.int64, device=dev)
        self.tables = torch.zeros(max(int(bo[-1]), 1), dtype=torch.int64, device=dev)
        self.rank = torch.zeros(C, dtype=torch.int32, device=dev)
        self.ctx_flags = torch.zeros(C, dtype=torch.int32, device=dev)
        self.n_contra = torch.zeros(C, dtype=torch.int32, device=dev)
        self.first_contra_row = torch.zeros(C, dtype=torch.int64, device=dev)
        self._struct = None

    def struct(self) -> f2_model:
        if self._struct is None:
            self._struct = f2_model(
                self.num_ctx, _ptr(self.n_bits), _ptr(self.basis_off), _ptr(self.piv_off), _ptr(self.map_off),
                int(self.basis_off_host[-1]), int(self.piv_off_host[-1]), int(self.map_off_host[-1]),
                _ptr(self.basis), _ptr(self.pivots), _ptr(self.maps), _ptr(self.tables), _ptr(self.rank),
                _ptr(self.ctx_flags),
                _ptr(self.n_contra), _ptr(self.first_contra_row),
                self.max_n_bits)
        return self._struct


def f2_fit_batch(rows, rows_words: int, row_off, model: Model, workspace, workspace_bytes: int, stream=None) -> int:
    """Enqueue the fit of every context; returns the status code."""
    return int(lib.f2_fit_batch(_ptr(rows), int(rows_words), _ptr(row_off), ctypes.byref(model.struct()),
                                _ptr(workspace), int(workspace_bytes), _stream(stream)))


def f2_fit_batch_noalloc(rows, rows_words: int, row_off, model: Model, stream=None) -> int:
    """Enqueue the fit without a workspace (the plan in the library's fixed device array); returns the status."""
    return int(lib.f2_fit_batch_noalloc(_ptr(rows), int(rows_words), _ptr(row_off), ctypes.byref(model.struct()),
                                        _stream(stream)))


def f2_encode_batch(model: Model, ctx_id, x, x_stride_words: int, num_queries: int, words_out, qflags_out,
                    workspace, workspace_bytes: int, stream=None) -> int:
    """Enqueue the encode of a query batch; returns the status code."""
    return int(lib.f2_encode_batch(ctypes.byref(model.struct()), _ptr(ctx_id), _ptr(x), int(x_stride_words),
                                   int(num_queries), _ptr(words_out), _ptr(qflags_out), _ptr(workspace),
                                   int(workspace_bytes), _stream(stream)))


def _host_words2(v) -> ctypes.Array:
    a = (ctypes.c_uint64 * 2)()
    a[0], a[1] = int(v[0]) & (2 ** 64 - 1), int(v[1]) & (2 ** 64 - 1)
    return a


def f2_vectorize_rows(values, y, num_rows: int, k: int, keep, rows_out, stream=None) -> int:
    """Enqueue the Eq. 1 row builder; keep is a pair of host words; returns the status code."""
    return int(lib.f2_vectorize_rows(_ptr(values), _ptr(y), int(num_rows), int(k), _host_words2(keep),
                                     _ptr(rows_out), _stream(stream)))


def f2_merge_words(words, field, shift: int, width: int, mask, state, num_words: int, out, stream=None) -> int:
    """Enqueue the post-encode merge; mask is a pair of host words; returns the status code."""
    return int(lib.f2_merge_words(_ptr(words), _ptr(field), int(shift), int(width), _host_words2(mask),
                                  _ptr(state), int(num_words), _ptr(out), _stream(stream)))


def f2_pool_workspace_bytes(members_model: "Model", num_pools: int) -> int:
    return int(lib.f2_pool_workspace_bytes(ctypes.byref(members_model.struct()), int(num_pools)))


def f2_pool_bases(members_model: "Model", out_mask, pool_off, members, num_members: int, pooled: "Model", pool_flags,
                  workspace, workspace_bytes: int, stream=None) -> int:
    """Enqueue the pooling of member bases into the pooled model; returns the status code."""
    return int(lib.f2_pool_bases(ctypes.byref(members_model.struct()), _ptr(out_mask), _ptr(pool_off), _ptr(members),
                                 int(num_members), ctypes.byref(pooled.struct()), _ptr(pool_flags), _ptr(workspace),
                                 int(workspace_bytes), _stream(stream)))


def f2_group_workspace_bytes(num_ctx: int, num_rows: int) -> int:
    return int(lib.f2_group_workspace_bytes(int(num_ctx), int(num_rows)))


def f2_group_rows(ctx_id, rows, row_stride_words: int, num_rows: int, n_bits, num_ctx: int, rows_out,
                  rows_out_words: int, row_off_out, dropped_out, workspace, workspace_bytes: int, stream=None) -> int:
    """Enqueue the grouping of an interleaved row stream by context; returns the status code."""
    return int(lib.f2_group_rows(_ptr(ctx_id), _ptr(rows), int(row_stride_words), int(num_rows), _ptr(n_bits),
                                 int(num_ctx), _ptr(rows_out), int(rows_out_words), _ptr(row_off_out),
                                 _ptr(dropped_out), _ptr(workspace), int(workspace_bytes), _stream(stream)))


# ---- convenience wrappers used by tests and the benchmark (allocation + one call) ----

def workspace(nbytes: int, device="cuda"):
    import torch
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def fit(rows_dev, row_off_dev, n_bits_host, stream=None):
    """Allocate a Model for n_bits_host and fit it from device rows/row_off; returns the Model."""
    model = Model(n_bits_host, device=rows_dev.device)
    nb = f2_fit_workspace_bytes(model.num_ctx)
    ws = workspace(nb, rows_dev.device)
    _check(f2_fit_batch(rows_dev, rows_dev.numel(), row_off_dev, model, ws, nb, stream), "f2_fit_batch")
    model._fit_ws = ws
    return model


def group(ctx_id_dev, rows_dev, stride: int, n_bits_dev, stream=None):
    """Group an interleaved row stream by context; returns (rows_out, row_off, dropped) device tensors."""
    import torch
    dev = rows_dev.device
    R = int(ctx_id_dev.numel())
    C = int(n_bits_dev.numel())
    rows_out = torch.empty(max(R * stride, 1), dtype=torch.int64, device=dev)
    row_off = torch.empty(C + 1, dtype=torch.int64, device=dev)
    dropped = torch.empty(1, dtype=torch.int64, device=dev)
    nb = f2_group_workspace_bytes(C, R)
    ws = workspace(nb, dev)
    _check(f2_group_rows(ctx_id_dev, rows_dev, stride, R, n_bits_dev, C, rows_out, R * stride, row_off, dropped,
                         ws, nb, stream), "f2_group_rows")
    out_ws = ws  # kept alive with the outputs until the stream has run
    rows_out._group_ws = out_ws
    return rows_out, row_off, dropped


def pool(members_model: Model, pool_off_dev, members_dev, pooled_n_host, out_mask_dev=None, stream=None):
    """Pool member bases; returns (pooled Model, pool_flags uint32-as-int32 device tensor)."""
    import torch
    dev = members_model.basis.device
    pooled = Model(pooled_n_host, device=dev)
    P = pooled.num_ctx
    flags = torch.zeros(max(P, 1), dtype=torch.int32, device=dev)
    nb = f2_pool_workspace_bytes(members_model, P)
    ws = workspace(nb, dev)
    _check(f2_pool_bases(members_model, out_mask_dev, pool_off_dev, members_dev, int(members_dev.numel()), pooled,
                         flags, ws, nb, stream), "f2_pool_bases")
    pooled._pool_ws = ws
    return pooled, flags


def encode(model: Model, ctx_dev, x_dev, stride: int, stream=None):
    """Encode a device query batch; returns (words int64 [Q, 2], qflags uint8 [Q]) device tensors."""
    import torch
    Q = int(ctx_dev.numel())
    words = torch.empty((max(Q, 1), 2), dtype=torch.int64, device=ctx_dev.device)
    qf = torch.empty(max(Q, 1), dtype=torch.uint8, device=ctx_dev.device)
    nb = f2_encode_workspace_bytes(model, Q)
    ws = workspace(nb, ctx_dev.device)
    _check(f2_encode_batch(model, ctx_dev, x_dev, stride, Q, words, qf, ws, nb, stream), "f2_encode_batch")
    return words[:Q], qf[:Q]
