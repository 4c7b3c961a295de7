"""CPU oracle (ctypes wrapper over ``liboracle.so``).

TEST INFRASTRUCTURE ONLY.  The test suite, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg are the only callers.  The product package
never imports this module and shares no code with it.

The C source (``oracle.c``) holds the arithmetic; this module only builds it
with gcc and marshals numpy arrays.  Array conventions: fp32 inputs are
``float32`` arrays, bf16 inputs are ``uint16`` arrays holding the raw bit
patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCES = (os.path.join(_HERE, "oracle.c"), os.path.join(_HERE, "message.c"))
_SO = os.path.join(_HERE, "liboracle.so")

DTYPE_CODE = {"f32": 0, "bf16": 1}


def build(verbose: bool = False, srcs=SOURCES, out: str = _SO) -> str:
    """Compile the oracle with gcc (plain -O2, no fast-math, no OpenMP)."""
    tmp = f"{out}.tmp{os.getpid():x}"   # one per process: builds may run side by side
    cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-Wall", "-I", _HERE, *srcs,
           "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _dtype_of(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return 0
    if a.dtype == np.uint16:
        return 1
    raise TypeError(f"oracle inputs are float32 or uint16 (bf16 bits), got {a.dtype}")


def _check(rc: int, what: str):
    if rc != 0:
        raise RuntimeError(f"{what} failed with status {rc}")


class Oracle:
    """numpy-level wrapper over one build of the oracle library."""

    def __init__(self, so_path: str = _SO):
        if not os.path.exists(so_path):
            build(out=so_path)
        lib = ctypes.CDLL(so_path)
        i64, i32, dbl, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_double, ctypes.c_void_p
        lib.cbo_keep_count.argtypes = [i64, dbl]
        lib.cbo_keep_count.restype = i64
        lib.cbo_score.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, i32, i64, dbl, vp, vp]
        lib.cbo_score.restype = i32
        lib.cbo_select.argtypes = [vp, i64, i64, i64, vp]
        lib.cbo_select.restype = i32
        lib.cbo_select_f32.argtypes = [vp, i64, i64, i64, vp]
        lib.cbo_select_f32.restype = i32
        lib.cbo_compact.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, i64, i64, vp, vp]
        lib.cbo_compact.restype = i32
        lib.cbo_position_score.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, i32, i64, dbl,
                                           i32, dbl, dbl, vp, vp, vp]
        lib.cbo_position_score.restype = i32
        lib.cbo_budget_fanout.argtypes = [i64, i64]
        lib.cbo_budget_fanout.restype = i64
        lib.cbo_budget_chain.argtypes = [i64, i64, i64, i32, i64]
        lib.cbo_budget_chain.restype = i64
        lib.cbo_select_spans.argtypes = [vp, i64, i64, i64, i32, vp]
        lib.cbo_select_spans.restype = i64
        lib.cbo_select_spans_f64.argtypes = [vp, i64, i64, i64, i32, vp]
        lib.cbo_select_spans_f64.restype = i64
        lib.cbo_gather_rows.argtypes = [vp, i32, i64, i64, vp, i64, vp]
        lib.cbo_gather_rows.restype = i32
        self.lib = lib
        self.path = so_path

    def keep_count(self, T: int, keep_ratio: float) -> int:
        return int(self.lib.cbo_keep_count(int(T), float(keep_ratio)))

    def score(self, q: np.ndarray, k: np.ndarray, scale: float = 0.0, with_lse: bool = False):
        """Importance [S][L][Hkv][T] (fp64) for q [L][Hq][m][D] and
        k [S][L][Hkv][T][D].  Returns ``importance`` or ``(importance,
        row_lse)`` with row_lse [S][L][Hq][m] in natural-log units."""
        q = np.ascontiguousarray(q)
        k = np.ascontiguousarray(k)
        dt = _dtype_of(q)
        if _dtype_of(k) != dt:
            raise TypeError("q and k must share a dtype")
        L, Hq, m, D = q.shape
        S, L2, Hkv, T, D2 = k.shape
        if L2 != L or D2 != D:
            raise ValueError("q/k shape mismatch")
        imp = np.empty((S, L, Hkv, T), dtype=np.float64)
        lse = np.empty((S, L, Hq, m), dtype=np.float64) if with_lse else None
        rc = self.lib.cbo_score(_ptr(q), _ptr(k), dt, S, L, Hq, Hkv, D, m, T, float(scale),
                                _ptr(imp), _ptr(lse) if with_lse else None)
        _check(rc, "cbo_score")
        return (imp, lse) if with_lse else imp

    def select(self, importance: np.ndarray, keep: int) -> np.ndarray:
        """Top-``keep`` of each row of ``importance`` [..., T] as ascending
        int32 indices.  fp64 keys use cbo_select, fp32 keys cbo_select_f32."""
        imp = np.ascontiguousarray(importance)
        T = imp.shape[-1]
        units = int(np.prod(imp.shape[:-1])) if imp.ndim > 1 else 1
        out = np.empty(imp.shape[:-1] + (keep,), dtype=np.int32)
        if imp.dtype == np.float64:
            rc = self.lib.cbo_select(_ptr(imp), units, T, keep, _ptr(out))
        elif imp.dtype == np.float32:
            rc = self.lib.cbo_select_f32(_ptr(imp), units, T, keep, _ptr(out))
        else:
            raise TypeError("importance must be float64 or float32")
        _check(rc, "cbo_select")
        return out

    def compact(self, k: np.ndarray, v: np.ndarray, idx: np.ndarray):
        """Row gather: k, v [S][L][Hkv][T][D] and idx [S][L][Hkv][keep] ->
        (k_out, v_out) [L][Hkv][S*keep][D]."""
        k = np.ascontiguousarray(k)
        v = np.ascontiguousarray(v)
        idx = np.ascontiguousarray(idx, dtype=np.int32)
        dt = _dtype_of(k)
        S, L, Hkv, T, D = k.shape
        keep = idx.shape[-1]
        k_out = np.empty((L, Hkv, S * keep, D), dtype=k.dtype)
        v_out = np.empty_like(k_out)
        rc = self.lib.cbo_compact(_ptr(k), _ptr(v), _ptr(idx), dt, S, L, Hkv, D, T, keep,
                                  _ptr(k_out), _ptr(v_out))
        _check(rc, "cbo_compact")
        return k_out, v_out

    def position_score(self, q: np.ndarray, k: np.ndarray, scale: float = 0.0,
                       pool_width: int = 7, p: float = 2.0, alpha: float = 2.0):
        """Position-level scores of every sender (Appendix C.1): returns
        (score, qscore, corr), each [S][T] fp64: S_t = Q_t * C_{p,t}^alpha,
        the mean query attention Q_t and the correction C_{p,t}."""
        q = np.ascontiguousarray(q)
        k = np.ascontiguousarray(k)
        dt = _dtype_of(q)
        if _dtype_of(k) != dt:
            raise TypeError("q and k must share a dtype")
        L, Hq, m, D = q.shape
        S, L2, Hkv, T, D2 = k.shape
        if L2 != L or D2 != D:
            raise ValueError("q/k shape mismatch")
        score = np.empty((S, T))
        qs = np.empty((S, T))
        corr = np.empty((S, T))
        rc = self.lib.cbo_position_score(_ptr(q), _ptr(k), dt, S, L, Hq, Hkv, D, m, T,
                                         float(scale), int(pool_width), float(p), float(alpha),
                                         _ptr(score), _ptr(qs), _ptr(corr))
        _check(rc, "cbo_position_score")
        return score, qs, corr

    def budget_fanout(self, T: int, r: int) -> int:
        return int(self.lib.cbo_budget_fanout(int(T), int(r)))

    def budget_chain(self, T_old: int, T_new: int, r: int, relative: bool, B_max: int = 0) -> int:
        return int(self.lib.cbo_budget_chain(int(T_old), int(T_new), int(r), int(bool(relative)),
                                             int(B_max)))

    def select_spans(self, score: np.ndarray, budget: int, n_latent: int = 40,
                     width: int = 16) -> np.ndarray:
        """Span rule of Appendix C.2 on one sender's scores [T] (fp32 or
        fp64): ascending int32 positions, min(budget, T) of them."""
        sc = np.ascontiguousarray(score)
        T = sc.shape[-1]
        out = np.empty(min(int(budget), T), dtype=np.int32)
        if sc.dtype == np.float32:
            n = self.lib.cbo_select_spans(_ptr(sc), T, int(budget), int(n_latent), int(width),
                                          _ptr(out))
        elif sc.dtype == np.float64:
            n = self.lib.cbo_select_spans_f64(_ptr(sc), T, int(budget), int(n_latent),
                                              int(width), _ptr(out))
        else:
            raise TypeError("scores must be float32 or float64")
        if n < 0:
            raise RuntimeError(f"cbo_select_spans failed with status {n}")
        assert n == len(out)
        return out

    def gather_rows(self, rows: np.ndarray, idx: np.ndarray) -> np.ndarray:
        """rows [S][T][...] (any dtype), idx [S][count] -> [S*count][...]."""
        rows = np.ascontiguousarray(rows)
        idx = np.ascontiguousarray(idx, dtype=np.int32)
        S, T = rows.shape[:2]
        row_bytes = rows[0, 0].nbytes
        count = idx.shape[-1]
        out = np.empty((S * count,) + rows.shape[2:], dtype=rows.dtype)
        rc = self.lib.cbo_gather_rows(_ptr(rows), S, T, row_bytes, _ptr(idx), count, _ptr(out))
        _check(rc, "cbo_gather_rows")
        return out


_default = None


def _get() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default


def keep_count(T, keep_ratio):
    return _get().keep_count(T, keep_ratio)


def score(q, k, scale=0.0, with_lse=False):
    return _get().score(q, k, scale, with_lse)


def select(importance, keep):
    return _get().select(importance, keep)


def compact(k, v, idx):
    return _get().compact(k, v, idx)
