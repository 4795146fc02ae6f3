"""CPU oracle for the f-gram embedding path (test infrastructure).

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this module; the product path never does.  It wraps
``scone_oracle.cpp`` (plain C++17: a std::unordered_map keyed by the raw bytes
of each f-gram and a memcpy row copy), which shares no code with the GPU
library.  See that file for the passage of the paper each function follows.

Pins (what checks this oracle against something other than itself) live in
``tests/test_oracle_pins.py``: a hand-worked example of Algorithm 1, a
brute-force linear scan over the f-gram list, the match invariants, and the
special cases that reduce to plain indexing.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "scone_oracle.cpp")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None
_lock = threading.Lock()

OR_OK, OR_BAD_ARG, OR_BAD_LENGTH, OR_BAD_ID, OR_DUPLICATE, OR_BAD_ROW = range(6)


class OracleError(RuntimeError):
    def __init__(self, code, what):
        super().__init__(f"oracle {what} failed with code {code}")
        self.code = code


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (it is a checker, built alongside the library)."""
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    subprocess.check_call(["g++", "-std=c++17", "-O2", "-shared", "-fPIC", "-o", tmp, _SRC])
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH):
            build()
        _lib = bind(ctypes.CDLL(_LIB_PATH))
        return _lib


def bind(lib):
    """Declare the C signatures on a loaded oracle library and return it."""
    P = ctypes.c_void_p
    I64, I32 = ctypes.c_int64, ctypes.c_int32
    lib.oracle_build.argtypes = [P, P, P, I64, I32, ctypes.POINTER(P)]
    lib.oracle_build.restype = ctypes.c_int
    lib.oracle_destroy.argtypes = [P]
    lib.oracle_destroy.restype = None
    lib.oracle_size.argtypes = [P]
    lib.oracle_size.restype = I64
    lib.oracle_lookup.argtypes = [P, P, I64, I64, I32, P, P]
    lib.oracle_lookup.restype = I64
    lib.oracle_gather.argtypes = [P, I64, P, I64, I64, P]
    lib.oracle_gather.restype = ctypes.c_int
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None and a.size else None


class OracleTable:
    """The f-gram dictionary of Section 2 (hash dictionary to row indices)."""

    def __init__(self, fgrams, lengths, ids):
        lib = _load()
        fg = np.ascontiguousarray(fgrams, dtype=np.int32)
        if fg.ndim != 2:
            raise ValueError("fgrams must be [n, stride]")
        ln = np.ascontiguousarray(lengths, dtype=np.int32)
        idv = np.ascontiguousarray(ids, dtype=np.int32)
        n = len(ln)
        if fg.shape[0] != n or len(idv) != n:
            raise ValueError("fgrams, lengths and ids disagree on n")
        h = ctypes.c_void_p()
        rc = lib.oracle_build(_ptr(fg), _ptr(ln), _ptr(idv), n, max(fg.shape[1], 1),
                              ctypes.byref(h))
        if rc != OR_OK:
            raise OracleError(rc, "build")
        self._h = h
        self.queries = 0

    def __len__(self):
        return int(_load().oracle_size(self._h))

    def lookup(self, tokens, max_n: int):
        """(ids [B,T] int32, match_len [B,T] int8) by the longest-suffix rule."""
        X = np.ascontiguousarray(tokens, dtype=np.int32)
        if X.ndim == 1:
            X = X.reshape(1, -1)
        B, T = X.shape
        ids = np.empty((B, T), dtype=np.int32)
        ml = np.empty((B, T), dtype=np.int8)
        q = _load().oracle_lookup(self._h, _ptr(X), B, T, max_n, _ptr(ids), _ptr(ml))
        if q < 0:
            raise OracleError(-1, "lookup")
        self.queries = int(q)
        return ids, ml

    def close(self):
        if getattr(self, "_h", None):
            _load().oracle_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def gather(ids, table: np.ndarray) -> np.ndarray:
    """out[k] = table[ids[k]] as raw bytes; table is [n_rows, ...] contiguous."""
    lib = _load()
    tb = np.ascontiguousarray(table)
    idv = np.ascontiguousarray(ids, dtype=np.int32).reshape(-1)
    n_rows = tb.shape[0]
    row_bytes = tb.nbytes // max(n_rows, 1) if n_rows else 1
    out = np.empty((idv.size,) + tb.shape[1:], dtype=tb.dtype)
    rc = lib.oracle_gather(_ptr(idv), idv.size, _ptr(tb), n_rows, row_bytes, _ptr(out))
    if rc != OR_OK:
        raise OracleError(rc, "gather")
    return out.reshape(tuple(np.shape(ids)) + tb.shape[1:])
