"""Thin ctypes binding of ``libf2probe.so`` (``include/f2probe.h``): the copy,
integer-issue and scattered-access probes whose measured rates are reported beside
the vendor peaks.
Raises on import if the library is not built."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libf2probe.so")
EXPORTS = ("f2probe_copy", "f2probe_bitops", "f2probe_scatter")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run __graft_entry__.build() (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.f2probe_copy.argtypes = [P, P, i64, P]
    L.f2probe_copy.restype = ctypes.c_int
    L.f2probe_bitops.argtypes = [P, i32, i32, i32, P]
    L.f2probe_bitops.restype = ctypes.c_int
    L.f2probe_scatter.argtypes = [P, i64, i32, i32, i32, P, P]
    L.f2probe_scatter.restype = ctypes.c_int
    return L


lib = _load()


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def f2probe_copy(src, dst, words: int, stream) -> int:
    return int(lib.f2probe_copy(_ptr(src), _ptr(dst), int(words), int(stream)))


def f2probe_bitops(out, blocks: int, iters: int, op: int, stream) -> int:
    return int(lib.f2probe_bitops(_ptr(out), int(blocks), int(iters), int(op), int(stream)))


def f2probe_scatter(buf, nbytes: int, blocks: int, per: int, op: int, out, stream) -> int:
    return int(lib.f2probe_scatter(_ptr(buf), int(nbytes), int(blocks), int(per), int(op), _ptr(out), int(stream)))
