"""ctypes front end of the multi-threaded host memory manager (baselines/cpu_manager.c):
completion recycling and page allocation over numpy copies of the cache state, with a
persistent pool of worker threads."""
import ctypes as C
import os

import numpy as np

from . import build as _build

_lib = None


class _State(C.Structure):
    _fields_ = [("table", C.c_void_p), ("pages", C.c_void_p), ("len", C.c_void_p),
                ("ring", C.c_void_p), ("ring_ptr", C.c_void_p), ("status", C.c_void_p),
                ("num_pages", C.c_int64), ("num_tables", C.c_int32), ("p_max", C.c_int32),
                ("tokens_per_page", C.c_int32 * 2)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = C.CDLL(_build.LIB)
        L.cm_pool_create.restype = C.c_void_p
        L.cm_pool_create.argtypes = [C.c_int]
        L.cm_pool_destroy.argtypes = [C.c_void_p]
        L.cm_compact.argtypes = [C.c_void_p, C.POINTER(_State), C.c_void_p]
        L.cm_alloc.argtypes = [C.c_void_p, C.POINTER(_State), C.c_void_p]
        L.cm_alloc.restype = C.c_int
        _lib = L
    return _lib


def _p(a):
    return a.ctypes.data_as(C.c_void_p)


class Manager:
    """Cache state (numpy, owned here) plus a worker pool of `threads` threads."""

    def __init__(self, table, pages, len_, ring, ring_ptr, tokens_per_page, threads):
        self.table = np.ascontiguousarray(table, np.int32).copy()
        self.pages = np.ascontiguousarray(pages, np.int32).copy()
        self.len = np.ascontiguousarray(len_, np.int32).copy()
        self.ring = np.ascontiguousarray(ring, np.int32).copy()
        self.ring_ptr = np.ascontiguousarray(ring_ptr, np.int64).copy()
        self.status = np.zeros(1, np.uint32)
        self.threads = int(threads)
        self._st = _State(_p(self.table), _p(self.pages), _p(self.len), _p(self.ring),
                          _p(self.ring_ptr), _p(self.status), self.ring.size, self.table.shape[0],
                          self.table.shape[1], (C.c_int32 * 2)(*tokens_per_page))
        self._pool = lib().cm_pool_create(self.threads)

    def compact(self, release):
        rel = np.ascontiguousarray(release, np.uint8)
        assert rel.shape == self.table.shape
        lib().cm_compact(self._pool, C.byref(self._st), _p(rel))

    def alloc(self, demand):
        d = np.ascontiguousarray(demand, np.int32)
        assert d.shape == (self.table.shape[0], 2) and (d >= 0).all()
        return lib().cm_alloc(self._pool, C.byref(self._st), _p(d))

    def close(self):
        if self._pool:
            lib().cm_pool_destroy(self._pool)
            self._pool = None

    def __del__(self):
        self.close()
