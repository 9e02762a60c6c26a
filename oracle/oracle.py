"""ctypes wrapper of the serial C oracle in ``geot_oracle.c`` (test infrastructure only).

Every function takes host numpy arrays and returns host numpy arrays. The C
source states the definition it follows (segment reduction, Section II-B of
the GeoT paper; fused gather-weight form, Sections IV and V-D).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "geot_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
OPS = {"sum": 0, "mean": 1, "max": 2}
_ERRORS = {1: "invalid argument", 2: "index not sorted", 3: "index or column out of range"}


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(_ERRORS.get(code, f"oracle error {code}"))
        self.code = code


MT_SOURCE = os.path.join(_HERE, "geot_oracle_mt.c")
_MT_LIB = os.path.join(_HERE, "liboracle_mt.so")


def lib_path() -> str:
    return _LIB


def host_threads() -> int:
    """Threads for the multi-threaded oracle: OMP_NUM_THREADS when set (the host share the
    machine gives this process), else the CPUs this process may run on."""
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        return min(int(env), 256)
    return max(1, min(len(os.sched_getaffinity(0)), 256))


def build(src: str = SOURCE, out: str = _LIB) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-std=c11", "-shared", "-fPIC",
           "-o", out, src, "-lm"]
    subprocess.run(cmd, check=True)
    return out


def build_mt(src: str = MT_SOURCE, out: str = _MT_LIB) -> str:
    """Compile the multi-threaded oracle (same flags, POSIX threads)."""
    cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-std=c11", "-pthread", "-shared", "-fPIC",
           "-o", out, src, "-lm"]
    subprocess.run(cmd, check=True)
    return out


def build_all() -> None:
    build()
    build_mt()


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _i64(a):
    return np.ascontiguousarray(a, dtype=np.int64)


def _check(rc: int):
    if rc != 0:
        raise OracleError(rc)


class OracleLib:
    """One loaded copy of the oracle shared library."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        lib.oracle_check_index.argtypes = [p, i64, i64]
        lib.oracle_segment_reduce.argtypes = [p, p, i64, i64, i64, ctypes.c_int, p]
        lib.oracle_gather_scatter.argtypes = [p, i64, p, p, p, i64, i64, i64, ctypes.c_int, p]
        lib.oracle_abs_term_sum.argtypes = [p, i64, p, p, p, i64, i64, i64, ctypes.c_int, p]
        lib.oracle_index_stats.argtypes = [p, i64, i64, p, p, p, p, p]
        lib.oracle_segment_reduce_backward.argtypes = [p, p, i64, i64, i64, ctypes.c_int, p, p, p]
        lib.oracle_gather_scatter_backward.argtypes = [p, i64, p, p, p, i64, i64, i64, ctypes.c_int,
                                                       p, p, ctypes.c_int, p, p]
        for name in ("oracle_check_index", "oracle_segment_reduce", "oracle_gather_scatter",
                     "oracle_abs_term_sum", "oracle_index_stats", "oracle_segment_reduce_backward",
                     "oracle_gather_scatter_backward"):
            getattr(lib, name).restype = ctypes.c_int
        self._lib = lib
        self.path = path

    def check_index(self, index, num_segments: int) -> int:
        index = _i64(index)
        return self._lib.oracle_check_index(_ptr(index), index.size, int(num_segments))

    def segment_reduce(self, src, index, num_segments: int, op: str = "sum") -> np.ndarray:
        """out[s] = op over rows i with index[i] == s (fp64 accumulation for sum/mean)."""
        src = _f32(src)
        if src.ndim == 1:
            src = src.reshape(-1, 1)
        index = _i64(index)
        F = src.shape[1]
        nnz = index.size
        if src.shape[0] != nnz:
            raise ValueError("src rows must equal index length")
        out = np.empty((int(num_segments), F), dtype=np.float32)
        _check(self._lib.oracle_segment_reduce(_ptr(src), _ptr(index), nnz, int(num_segments), F,
                                               OPS[op], _ptr(out)))
        return out

    def gather_scatter(self, X, col, weight, row, num_rows: int, op: str = "sum") -> np.ndarray:
        """out[r] = op over edges e with row[e] == r of weight[e] * X[col[e]] (weight None: 1)."""
        X = _f32(X)
        col = _i64(col)
        row = _i64(row)
        w = None if weight is None else _f32(weight)
        F = X.shape[1]
        nnz = row.size
        if col.size != nnz or (w is not None and w.size != nnz):
            raise ValueError("col, weight and row must have one entry per edge")
        out = np.empty((int(num_rows), F), dtype=np.float32)
        _check(self._lib.oracle_gather_scatter(_ptr(X), X.shape[0], _ptr(col), _ptr(w), _ptr(row),
                                               nnz, int(num_rows), F, OPS[op], _ptr(out)))
        return out

    def abs_term_sum(self, rows, index, num_segments: int, op: str = "sum", col=None,
                     weight=None) -> np.ndarray:
        """Per output element, sum of |term| in fp64 (terms divided by the count for mean)."""
        rows = _f32(rows)
        if rows.ndim == 1:
            rows = rows.reshape(-1, 1)
        index = _i64(index)
        c = None if col is None else _i64(col)
        w = None if weight is None else _f32(weight)
        F = rows.shape[1]
        out = np.empty((int(num_segments), F), dtype=np.float64)
        _check(self._lib.oracle_abs_term_sum(_ptr(rows), rows.shape[0], _ptr(c), _ptr(w),
                                             _ptr(index), index.size, int(num_segments), F,
                                             OPS[op], _ptr(out)))
        return out

    def segment_reduce_backward(self, grad_out, index, op: str = "sum", src=None, out=None):
        """grad_src of segment_reduce given grad_out [S x F] (src and out needed for max)."""
        grad_out = _f32(grad_out)
        index = _i64(index)
        S, F = grad_out.shape
        g = np.empty((index.size, F), dtype=np.float32)
        s_ = None if src is None else _f32(src)
        o_ = None if out is None else _f32(out)
        if op == "max" and (s_ is None or o_ is None):
            raise ValueError("max needs src and out")
        _check(self._lib.oracle_segment_reduce_backward(_ptr(grad_out), _ptr(index), index.size, S, F,
                                                        OPS[op], _ptr(s_), _ptr(o_), _ptr(g)))
        return g

    def gather_scatter_backward(self, X, col, weight, row, grad_out, op: str = "sum", out=None,
                                absolute: bool = False):
        """(grad_X [n_x x F] fp64, grad_w [nnz] fp64 or None) of gather_scatter."""
        X = _f32(X)
        col = _i64(col)
        row = _i64(row)
        w = None if weight is None else _f32(weight)
        grad_out = _f32(grad_out)
        o_ = None if out is None else _f32(out)
        if op == "max" and o_ is None:
            raise ValueError("max needs out")
        R, F = grad_out.shape
        gX = np.empty(X.shape, dtype=np.float64)
        gw = np.empty(row.size, dtype=np.float64) if w is not None else None
        _check(self._lib.oracle_gather_scatter_backward(_ptr(X), X.shape[0], _ptr(col), _ptr(w), _ptr(row),
                                                        row.size, R, F, OPS[op], _ptr(grad_out), _ptr(o_),
                                                        int(absolute), _ptr(gX), _ptr(gw)))
        return gX, gw

    def index_stats(self, index, num_segments: int) -> dict:
        """mean, population variance, max length, empty count and sum of squared lengths."""
        index = _i64(index)
        mean, var = ctypes.c_double(), ctypes.c_double()
        mx, ne, sq = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(self._lib.oracle_index_stats(_ptr(index), index.size, int(num_segments),
                                            ctypes.byref(mean), ctypes.byref(var), ctypes.byref(mx),
                                            ctypes.byref(ne), ctypes.byref(sq)))
        return dict(mean_len=mean.value, var_len=var.value, max_len=mx.value,
                    num_empty=ne.value, sum_len_sq=sq.value)


class OracleMT:
    """The multi-threaded oracle (geot_oracle_mt.c): the serial oracle's forward
    definitions with the output segments split across threads; bit-identical results."""

    def __init__(self, path: str, threads: int | None = None):
        lib = ctypes.CDLL(path)
        i64, p, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
        lib.oracle_mt_segment_reduce.argtypes = [p, p, i64, i64, i64, ci, p, ci]
        lib.oracle_mt_gather_scatter.argtypes = [p, i64, p, p, p, i64, i64, i64, ci, p, ci]
        lib.oracle_mt_abs_term_sum.argtypes = [p, i64, p, p, p, i64, i64, i64, ci, p, ci]
        for name in ("oracle_mt_segment_reduce", "oracle_mt_gather_scatter", "oracle_mt_abs_term_sum"):
            getattr(lib, name).restype = ctypes.c_int
        self._lib = lib
        self.path = path
        self.threads = int(threads) if threads else host_threads()

    def segment_reduce(self, src, index, num_segments: int, op: str = "sum") -> np.ndarray:
        src = _f32(src)
        if src.ndim == 1:
            src = src.reshape(-1, 1)
        index = _i64(index)
        if src.shape[0] != index.size:
            raise ValueError("src rows must equal index length")
        out = np.empty((int(num_segments), src.shape[1]), dtype=np.float32)
        _check(self._lib.oracle_mt_segment_reduce(_ptr(src), _ptr(index), index.size, int(num_segments),
                                                  src.shape[1], OPS[op], _ptr(out), self.threads))
        return out

    def gather_scatter(self, X, col, weight, row, num_rows: int, op: str = "sum") -> np.ndarray:
        X, col, row = _f32(X), _i64(col), _i64(row)
        w = None if weight is None else _f32(weight)
        if col.size != row.size or (w is not None and w.size != row.size):
            raise ValueError("col, weight and row must have one entry per edge")
        out = np.empty((int(num_rows), X.shape[1]), dtype=np.float32)
        _check(self._lib.oracle_mt_gather_scatter(_ptr(X), X.shape[0], _ptr(col), _ptr(w), _ptr(row), row.size,
                                                  int(num_rows), X.shape[1], OPS[op], _ptr(out), self.threads))
        return out

    def abs_term_sum(self, rows, index, num_segments: int, op: str = "sum", col=None, weight=None) -> np.ndarray:
        rows = _f32(rows)
        if rows.ndim == 1:
            rows = rows.reshape(-1, 1)
        index = _i64(index)
        c = None if col is None else _i64(col)
        w = None if weight is None else _f32(weight)
        out = np.empty((int(num_segments), rows.shape[1]), dtype=np.float64)
        _check(self._lib.oracle_mt_abs_term_sum(_ptr(rows), rows.shape[0], _ptr(c), _ptr(w), _ptr(index),
                                                index.size, int(num_segments), rows.shape[1], OPS[op], _ptr(out),
                                                self.threads))
        return out


_default = None
_default_mt = None


def mt() -> OracleMT:
    """The multi-threaded oracle built in this directory (built with gcc on first use)."""
    global _default_mt
    if _default_mt is None:
        if not os.path.exists(_MT_LIB):
            build_mt()
        _default_mt = OracleMT(_MT_LIB)
    return _default_mt


def default() -> OracleLib:
    """The oracle built in this directory (built with gcc on first use if missing)."""
    global _default
    if _default is None:
        if not os.path.exists(_LIB):
            build()
        _default = OracleLib(_LIB)
    return _default


def check_index(index, num_segments):
    return default().check_index(index, num_segments)


def segment_reduce(src, index, num_segments, op="sum"):
    return default().segment_reduce(src, index, num_segments, op)


def gather_scatter(X, col, weight, row, num_rows, op="sum"):
    return default().gather_scatter(X, col, weight, row, num_rows, op)


def abs_term_sum(rows, index, num_segments, op="sum", col=None, weight=None):
    return default().abs_term_sum(rows, index, num_segments, op, col, weight)


def index_stats(index, num_segments):
    return default().index_stats(index, num_segments)


def segment_reduce_backward(grad_out, index, op="sum", src=None, out=None):
    return default().segment_reduce_backward(grad_out, index, op, src, out)


def gather_scatter_backward(X, col, weight, row, grad_out, op="sum", out=None, absolute=False):
    return default().gather_scatter_backward(X, col, weight, row, grad_out, op, out, absolute)
