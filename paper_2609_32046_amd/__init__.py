"""MI355X receiver-conditioned KV selection: Python binding of ``libcacheback.so``.

Argument marshalling only.  Every step of the path runs in the HIP kernels
behind the C ABI declared in ``include/cacheback.h``; this module converts
torch tensors (or raw integer device pointers) to pointers, passes the current
HIP stream, and turns status codes into exceptions.  torch is used for device
memory and streams only.

There is no CPU fallback: importing this package raises if the HIP library
has not been built (``python paper_2609_32046_amd/build.py``).
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcacheback.so")

CB_F32, CB_BF16 = 0, 1
STATUS = {0: "CB_OK", -1: "CB_ERR_NULL", -2: "CB_ERR_SHAPE", -3: "CB_ERR_DTYPE",
          -4: "CB_ERR_RATIO", -5: "CB_ERR_WORKSPACE", -6: "CB_ERR_ALIGN", -7: "CB_ERR_HIP",
          -8: "CB_ERR_TIMEOUT"}

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build the HIP library first "
        "(python paper_2609_32046_amd/build.py).  There is no CPU fallback.")

_lib = ctypes.CDLL(LIB_PATH)


class cb_layout(ctypes.Structure):
    _fields_ = [("layers", ctypes.c_int32), ("q_heads", ctypes.c_int32),
                ("kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("q_len", ctypes.c_int32), ("senders", ctypes.c_int32),
                ("seq_len", ctypes.c_int64), ("dtype", ctypes.c_int32),
                ("scale", ctypes.c_float)]


_vp, _i64, _sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
_lib.cb_score_workspace_bytes.argtypes = [ctypes.POINTER(cb_layout)]
_lib.cb_score_workspace_bytes.restype = _sz
_lib.cb_score.argtypes = [_vp, _vp, ctypes.POINTER(cb_layout), _vp, _vp, _vp, _sz, _vp]
_lib.cb_score.restype = ctypes.c_int
_lib.cb_keep_count.argtypes = [_i64, ctypes.c_double]
_lib.cb_keep_count.restype = _i64
_lib.cb_select.argtypes = [_vp, _i64, _i64, ctypes.c_double, _vp, ctypes.POINTER(_i64), _vp]
_lib.cb_select.restype = ctypes.c_int
_lib.cb_select_workspace_bytes.argtypes = [_i64, _i64]
_lib.cb_select_workspace_bytes.restype = _sz
_lib.cb_select_ws.argtypes = [_vp, _i64, _i64, ctypes.c_double, _vp, ctypes.POINTER(_i64), _vp,
                              _sz, _vp]
_lib.cb_select_ws.restype = ctypes.c_int
_lib.cb_select_status.argtypes = [_i64, _i64, _vp, _sz, _vp]
_lib.cb_select_status.restype = ctypes.c_int
_lib.cb_compact.argtypes = [_vp, _vp, _vp, ctypes.POINTER(cb_layout), _i64, _vp, _vp, _vp]
_lib.cb_compact.restype = ctypes.c_int
_lib.cb_pipeline.argtypes = [_vp, _vp, _vp, ctypes.POINTER(cb_layout), ctypes.c_double, _vp, _vp,
                             _vp, _vp, _vp, _vp, _sz, ctypes.POINTER(_i64), _vp]
_lib.cb_pipeline.restype = ctypes.c_int
_lib.cb_pipeline_noalloc.argtypes = [_vp, _vp, _vp, ctypes.POINTER(cb_layout), ctypes.c_double,
                                     _vp, _vp, _vp, _vp, _vp, ctypes.POINTER(_i64), _vp]
_lib.cb_pipeline_noalloc.restype = ctypes.c_int
_lib.cb_score_status.argtypes = [ctypes.POINTER(cb_layout), _vp, _sz, _vp]
_lib.cb_score_status.restype = ctypes.c_int
_lib.cb_set_wait_limit.argtypes = [ctypes.c_uint32]
_lib.cb_set_wait_limit.restype = ctypes.c_uint32
_lib.cb_position_workspace_bytes.argtypes = [ctypes.POINTER(cb_layout)]
_lib.cb_position_workspace_bytes.restype = _sz
_lib.cb_position_score.argtypes = [_vp, _vp, ctypes.POINTER(cb_layout), ctypes.c_double,
                                   ctypes.c_double, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
_lib.cb_position_score.restype = ctypes.c_int
_lib.cb_position_status.argtypes = [ctypes.POINTER(cb_layout), _vp, _sz, _vp]
_lib.cb_position_status.restype = ctypes.c_int
_lib.cb_budget_fanout.argtypes = [_i64, _i64]
_lib.cb_budget_fanout.restype = _i64
_lib.cb_budget_chain.argtypes = [_i64, _i64, _i64, ctypes.c_int, _i64]
_lib.cb_budget_chain.restype = _i64
_lib.cb_spans_workspace_bytes.argtypes = [_i64, _i64, ctypes.c_int32]
_lib.cb_spans_workspace_bytes.restype = _sz
_lib.cb_select_spans.argtypes = [_vp, _i64, _i64, _i64, _i64, ctypes.c_int32, _vp,
                                 ctypes.POINTER(_i64), _vp, _sz, _vp]
_lib.cb_select_spans.restype = ctypes.c_int
_lib.cb_gather_rows.argtypes = [_vp, _i64, _i64, _i64, _vp, _i64, _vp, _vp]
_lib.cb_gather_rows.restype = ctypes.c_int
_lib.cb_status_string.argtypes = [ctypes.c_int]
_lib.cb_status_string.restype = ctypes.c_char_p


class CBError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} "
                         f"({_lib.cb_status_string(status).decode()})")


def _check(status: int, where: str) -> int:
    if status < 0:
        raise CBError(status, where)
    return status


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def layout(layers, q_heads, kv_heads, head_dim, q_len, seq_len, senders=1, dtype=CB_BF16,
           scale=0.0) -> cb_layout:
    if isinstance(dtype, str):
        dtype = {"f32": CB_F32, "bf16": CB_BF16}[dtype]
    return cb_layout(layers, q_heads, kv_heads, head_dim, q_len, senders, seq_len, dtype, scale)


def layout_of(w, scale=0.0) -> cb_layout:
    """cb_layout for a workload description with the usual attribute names."""
    return layout(w.layers, w.q_heads, w.kv_heads, w.head_dim, w.q_len, w.seq_len,
                  w.senders, w.dtype, scale)


def cb_score_workspace_bytes(lay: cb_layout) -> int:
    n = _lib.cb_score_workspace_bytes(ctypes.byref(lay))
    if n == 0:
        raise CBError(-2, "cb_score_workspace_bytes")
    return n


def cb_score(q, k, lay: cb_layout, importance, row_lse=None, ws=None, ws_bytes=None,
             stream=None) -> None:
    if ws_bytes is None:
        ws_bytes = ws.numel() * ws.element_size() if ws is not None and not isinstance(ws, int) else 0
    _check(_lib.cb_score(_ptr(q), _ptr(k), ctypes.byref(lay), _ptr(importance), _ptr(row_lse),
                         _ptr(ws), ws_bytes, _stream(stream)), "cb_score")


def cb_keep_count(T: int, keep_ratio: float) -> int:
    return _check(int(_lib.cb_keep_count(int(T), float(keep_ratio))), "cb_keep_count")


def cb_select(importance, units: int, T: int, keep_ratio: float, idx, stream=None) -> int:
    keep = _i64(0)
    _check(_lib.cb_select(_ptr(importance), int(units), int(T), float(keep_ratio), _ptr(idx),
                          ctypes.byref(keep), _stream(stream)), "cb_select")
    return keep.value


def cb_select_workspace_bytes(units: int, T: int) -> int:
    """Scratch bytes of cb_select_ws for these rows (0: rows are not split)."""
    return _lib.cb_select_workspace_bytes(int(units), int(T))


def cb_select_ws(importance, units: int, T: int, keep_ratio: float, idx, ws, ws_bytes=None,
                 stream=None) -> int:
    keep = _i64(0)
    _check(_lib.cb_select_ws(_ptr(importance), int(units), int(T), float(keep_ratio), _ptr(idx),
                             ctypes.byref(keep), _ptr(ws), _nbytes(ws, ws_bytes),
                             _stream(stream)), "cb_select_ws")
    return keep.value


def cb_select_status(units: int, T: int, ws, ws_bytes=None, stream=None) -> int:
    """Synchronises the stream and returns 0 (CB_OK) or -8 (CB_ERR_TIMEOUT)
    for the last cb_select_ws call on ``ws``; argument errors raise."""
    st = _lib.cb_select_status(int(units), int(T), _ptr(ws), _nbytes(ws, ws_bytes),
                               _stream(stream))
    if st not in (0, -8):
        _check(st, "cb_select_status")
    return st


def cb_compact(k, v, idx, lay: cb_layout, keep: int, k_out, v_out, stream=None) -> None:
    _check(_lib.cb_compact(_ptr(k), _ptr(v), _ptr(idx), ctypes.byref(lay), int(keep),
                           _ptr(k_out), _ptr(v_out), _stream(stream)), "cb_compact")


def cb_pipeline(q, k, v, lay: cb_layout, keep_ratio: float, importance, idx, k_out, v_out,
                ws, row_lse=None, ws_bytes=None, stream=None) -> int:
    if ws_bytes is None:
        ws_bytes = ws.numel() * ws.element_size() if not isinstance(ws, int) else 0
    keep = _i64(0)
    _check(_lib.cb_pipeline(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(lay), float(keep_ratio),
                            _ptr(importance), _ptr(row_lse), _ptr(idx), _ptr(k_out), _ptr(v_out),
                            _ptr(ws), ws_bytes, ctypes.byref(keep), _stream(stream)),
           "cb_pipeline")
    return keep.value


def cb_score_status(lay: cb_layout, ws, ws_bytes=None, stream=None) -> int:
    """Synchronises the stream and returns the status word of the last score
    call on ``ws``: 0 (CB_OK) or -8 (CB_ERR_TIMEOUT); argument errors raise."""
    if ws_bytes is None:
        ws_bytes = ws.numel() * ws.element_size() if not isinstance(ws, int) else 0
    st = _lib.cb_score_status(ctypes.byref(lay), _ptr(ws), ws_bytes, _stream(stream))
    if st not in (0, -8):
        _check(st, "cb_score_status")
    return st


def _nbytes(ws, ws_bytes):
    if ws_bytes is not None:
        return ws_bytes
    return ws.numel() * ws.element_size() if ws is not None and not isinstance(ws, int) else 0


def cb_position_workspace_bytes(lay: cb_layout) -> int:
    n = _lib.cb_position_workspace_bytes(ctypes.byref(lay))
    if n == 0:
        raise CBError(-2, "cb_position_workspace_bytes")
    return n


def cb_position_score(q, k, lay: cb_layout, score, ws, p=2.0, alpha=2.0, qscore=None, corr=None,
                      importance=None, ws_bytes=None, stream=None) -> None:
    _check(_lib.cb_position_score(_ptr(q), _ptr(k), ctypes.byref(lay), float(p), float(alpha),
                                  _ptr(score), _ptr(qscore), _ptr(corr), _ptr(importance),
                                  _ptr(ws), _nbytes(ws, ws_bytes), _stream(stream)),
           "cb_position_score")


def cb_position_status(lay: cb_layout, ws, ws_bytes=None, stream=None) -> int:
    st = _lib.cb_position_status(ctypes.byref(lay), _ptr(ws), _nbytes(ws, ws_bytes),
                                 _stream(stream))
    if st not in (0, -8):
        _check(st, "cb_position_status")
    return st


def cb_budget_fanout(T: int, r: int) -> int:
    return _check(int(_lib.cb_budget_fanout(int(T), int(r))), "cb_budget_fanout")


def cb_budget_chain(T_old: int, T_new: int, r: int, relative: bool, B_max: int = 0) -> int:
    return _check(int(_lib.cb_budget_chain(int(T_old), int(T_new), int(r), int(bool(relative)),
                                           int(B_max))), "cb_budget_chain")


def cb_spans_workspace_bytes(senders: int, T: int, width: int = 16) -> int:
    n = _lib.cb_spans_workspace_bytes(int(senders), int(T), int(width))
    if n == 0:
        raise CBError(-2, "cb_spans_workspace_bytes")
    return n


def cb_select_spans(score, senders: int, T: int, budget: int, idx, ws, n_latent: int = 40,
                    width: int = 16, ws_bytes=None, stream=None) -> int:
    count = _i64(0)
    _check(_lib.cb_select_spans(_ptr(score), int(senders), int(T), int(budget), int(n_latent),
                                int(width), _ptr(idx), ctypes.byref(count), _ptr(ws),
                                _nbytes(ws, ws_bytes), _stream(stream)), "cb_select_spans")
    return count.value


def cb_gather_rows(rows, senders: int, T: int, row_bytes: int, idx, count: int, out,
                   stream=None) -> None:
    _check(_lib.cb_gather_rows(_ptr(rows), int(senders), int(T), int(row_bytes), _ptr(idx),
                               int(count), _ptr(out), _stream(stream)), "cb_gather_rows")


def cb_set_wait_limit(polls: int) -> int:
    return int(_lib.cb_set_wait_limit(int(polls)))


def cb_pipeline_noalloc(q, k, v, lay: cb_layout, keep_ratio: float, importance, idx, k_out, v_out,
                        row_lse=None, stream=None) -> int:
    """cb_pipeline with the library's own per-device workspace (no ws)."""
    keep = _i64(0)
    _check(_lib.cb_pipeline_noalloc(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(lay),
                                    float(keep_ratio), _ptr(importance), _ptr(row_lse), _ptr(idx),
                                    _ptr(k_out), _ptr(v_out), ctypes.byref(keep), _stream(stream)),
           "cb_pipeline_noalloc")
    return keep.value


def cb_status_string(status: int) -> str:
    return _lib.cb_status_string(int(status)).decode()


class Buffers:
    """Device buffers for one layout and keep ratio (torch allocations)."""

    def __init__(self, lay: cb_layout, keep_ratio: float, device="cuda"):
        import torch

        self.lay = lay
        S, L, Hkv, T = lay.senders, lay.layers, lay.kv_heads, lay.seq_len
        self.units = S * L * Hkv
        self.keep = cb_keep_count(T, keep_ratio)
        self.keep_ratio = keep_ratio
        dt = torch.bfloat16 if lay.dtype == CB_BF16 else torch.float32
        self.importance = torch.empty((S, L, Hkv, T), dtype=torch.float32, device=device)
        self.row_lse = torch.empty((S, L, lay.q_heads, lay.q_len), dtype=torch.float32,
                                   device=device)
        self.idx = torch.empty((S, L, Hkv, self.keep), dtype=torch.int32, device=device)
        self.k_out = torch.empty((L, Hkv, S * self.keep, lay.head_dim), dtype=dt, device=device)
        self.v_out = torch.empty_like(self.k_out)
        self.ws = torch.empty(cb_score_workspace_bytes(lay), dtype=torch.uint8, device=device)
        # cb_select_ws scratch for the staged calls (None: rows are not split)
        nsel = cb_select_workspace_bytes(self.units, T)
        self.sel_ws = torch.empty(nsel, dtype=torch.uint8, device=device) if nsel else None


def run_steps(q, k, v, buf: Buffers, want_lse=True, stream=None) -> None:
    """cb_score -> cb_select_ws -> cb_compact on one stream, into ``buf`` (the
    selection splits rows as cb_pipeline does, where it can)."""
    cb_score(q, k, buf.lay, buf.importance, buf.row_lse if want_lse else None, buf.ws,
             stream=stream)
    cb_select_ws(buf.importance, buf.units, buf.lay.seq_len, buf.keep_ratio, buf.idx, buf.sel_ws,
                 stream=stream)
    cb_compact(k, v, buf.idx, buf.lay, buf.keep, buf.k_out, buf.v_out, stream=stream)


def run_pipeline(q, k, v, buf: Buffers, want_lse=True, stream=None) -> None:
    """The fused entry point cb_pipeline, into ``buf``."""
    keep = cb_pipeline(q, k, v, buf.lay, buf.keep_ratio, buf.importance, buf.idx, buf.k_out,
                       buf.v_out, buf.ws, row_lse=buf.row_lse if want_lse else None,
                       stream=stream)
    assert keep == buf.keep


class PositionBuffers:
    """Device buffers of the position-level path for one layout (torch
    allocations): scores, Q, C, importance and the two workspaces."""

    def __init__(self, lay: cb_layout, device="cuda", span_width=16):
        import torch

        S, L, Hkv, T = lay.senders, lay.layers, lay.kv_heads, lay.seq_len
        self.lay = lay
        self.score = torch.empty((S, T), dtype=torch.float32, device=device)
        self.qscore = torch.empty_like(self.score)
        self.corr = torch.empty_like(self.score)
        self.importance = torch.empty((S, L, Hkv, T), dtype=torch.float32, device=device)
        self.ws = torch.empty(cb_position_workspace_bytes(lay), dtype=torch.uint8, device=device)
        self.span_ws = torch.empty(cb_spans_workspace_bytes(S, T, span_width), dtype=torch.uint8,
                                   device=device)


__all__ = ["cb_layout", "layout", "layout_of", "cb_score_workspace_bytes", "cb_score",
           "cb_keep_count", "cb_select", "cb_compact", "cb_status_string", "CBError",
           "cb_pipeline", "cb_score_status", "cb_set_wait_limit", "cb_position_workspace_bytes",
           "cb_position_score", "cb_position_status", "cb_budget_fanout", "cb_budget_chain",
           "cb_spans_workspace_bytes", "cb_select_spans", "cb_gather_rows", "PositionBuffers",
           "cb_pipeline_noalloc", "cb_select_workspace_bytes", "cb_select_ws", "cb_select_status",
           "Buffers", "run_steps", "run_pipeline", "CB_F32", "CB_BF16",
           "LIB_PATH"]
