"""The C-ABI library on a host without a GPU: it loads, exports every symbol
the header declares, and its host-only logic (budget, status strings,
workspace sizing, argument validation that returns before any launch)
behaves as documented."""
import ctypes
import math
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cacheback.h")


@pytest.fixture(scope="module")
def cb():
    import paper_2609_32046_amd as cb

    return cb


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cb_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(
        ["cb_score_workspace_bytes", "cb_score", "cb_keep_count", "cb_select", "cb_compact",
         "cb_pipeline", "cb_score_status", "cb_set_wait_limit", "cb_status_string",
         "cb_position_workspace_bytes", "cb_position_score", "cb_position_status",
         "cb_budget_fanout", "cb_budget_chain", "cb_spans_workspace_bytes", "cb_select_spans",
         "cb_gather_rows", "cb_pipeline_noalloc", "cb_select_workspace_bytes", "cb_select_ws",
         "cb_select_status"])


def test_library_exports_every_declared_symbol(cb):
    out = subprocess.run(["nm", "-D", "--defined-only", cb.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(cb._lib, name)


def test_keep_count_matches_oracle(cb, oracle):
    orc = oracle.Oracle()
    rng = np.random.default_rng(0)
    ratios = [0.07, 0.1, 0.25, 0.5, 0.7, 1.0, 1 / 3, 1 / 16, 1e-9] + rng.random(200).tolist()
    Ts = [1, 2, 3, 10, 100, 512, 1200, 8192, 32768, 65536, 100003, 2**31 - 1]
    for T in Ts:
        for r in ratios:
            if r <= 0:
                continue
            assert cb.cb_keep_count(T, r) == orc.keep_count(T, r), (T, r)
    for bad in (0.0, -1.0, 1.0000001, float("nan")):
        assert cb._lib.cb_keep_count(10, bad) == -4
    assert cb._lib.cb_keep_count(0, 0.5) == -2


def test_status_strings(cb):
    for code in range(-8, 1):
        assert cb.cb_status_string(code) and cb.cb_status_string(code) != "unknown status"
    assert cb.cb_status_string(-99) == "unknown status"


def test_workspace_sizing_and_layout_validation(cb):
    lay = cb.layout(36, 32, 8, 128, 64, 8192)
    n = cb.cb_score_workspace_bytes(lay)
    # at least the per-chunk row statistics (1024-position chunks) for every unit
    assert n >= 288 * 8 * 256 * 8
    for bad in [dict(q_heads=30), dict(head_dim=96), dict(q_len=0), dict(seq_len=2**31),
                dict(seq_len=2**31 - 2**16 + 1),
                dict(q_len=300), dict(dtype=7), dict(scale=-1.0), dict(scale=float("inf"))]:
        kw = dict(layers=36, q_heads=32, kv_heads=8, head_dim=128, q_len=64, seq_len=8192)
        kw.update(bad)
        assert cb._lib.cb_score_workspace_bytes(ctypes.byref(cb.layout(**kw))) == 0, bad


def test_validation_returns_before_any_launch(cb):
    lay = cb.layout(1, 4, 2, 64, 16, 512, dtype="f32")
    ws_n = cb.cb_score_workspace_bytes(lay)
    fake = 1 << 20   # never dereferenced: every call below fails validation first
    L = ctypes.byref
    assert cb._lib.cb_score(None, fake, L(lay), fake, None, fake, ws_n, None) == -1
    assert cb._lib.cb_score(fake, fake, None, fake, None, fake, ws_n, None) == -1
    assert cb._lib.cb_score(fake, fake, L(lay), fake, None, fake, ws_n - 1, None) == -5
    assert cb._lib.cb_score(fake, fake, L(lay), fake, None, None, ws_n, None) == -5
    assert cb._lib.cb_score(fake + 4, fake, L(lay), fake, None, fake, ws_n, None) == -6
    assert cb._lib.cb_score(fake, fake, L(lay), fake, fake + 8, fake, ws_n, None) == -6
    bad = cb.layout(1, 3, 2, 64, 16, 512)
    assert cb._lib.cb_score(fake, fake, L(bad), fake, None, fake, ws_n, None) == -2
    bad = cb.layout(1, 4, 2, 64, 16, 512, dtype=5)
    assert cb._lib.cb_score(fake, fake, L(bad), fake, None, fake, ws_n, None) == -3
    k = ctypes.c_int64(0)
    assert cb._lib.cb_select(None, 2, 512, 0.25, fake, L(k), None) == -1
    assert cb._lib.cb_select(fake, 2, 512, 0.0, fake, L(k), None) == -4
    assert cb._lib.cb_select(fake, 2, 512, float("nan"), fake, L(k), None) == -4
    assert cb._lib.cb_select(fake, 0, 512, 0.25, fake, L(k), None) == -2
    assert cb._lib.cb_select(fake, 2, 2**31, 0.25, fake, L(k), None) == -2
    assert cb._lib.cb_select(fake, 2, 2**31 - 2**16 + 1, 0.25, fake, L(k), None) == -2
    assert cb._lib.cb_select(fake + 4, 2, 512, 0.25, fake, L(k), None) == -6
    assert cb._lib.cb_compact(fake, fake, None, L(lay), 128, fake, fake, None) == -1
    assert cb._lib.cb_compact(fake, fake, fake, L(lay), 0, fake, fake, None) == -2
    assert cb._lib.cb_compact(fake, fake, fake, L(lay), 513, fake, fake, None) == -2
    assert cb._lib.cb_compact(fake, fake, fake, L(lay), 128, fake + 2, fake, None) == -6
    P = cb._lib.cb_pipeline
    assert P(fake, fake, None, L(lay), 0.25, fake, None, fake, fake, fake, fake, ws_n, None, None) == -1
    assert P(fake, fake, fake, L(lay), 0.0, fake, None, fake, fake, fake, fake, ws_n, None, None) == -4
    assert P(fake, fake, fake, L(lay), 0.25, fake, None, fake, fake, fake, fake, 0, None, None) == -5
    assert P(fake, fake, fake, L(lay), 0.25, fake, None, fake + 4, fake, fake, fake, ws_n, None, None) == -6
    assert P(fake, fake, fake, None, 0.25, fake, None, fake, fake, fake, fake, ws_n, None, None) == -1


def test_split_select_sizing_and_validation(cb):
    """cb_select_workspace_bytes is nonzero exactly when rows are split (T >
    16384, at most 256 workgroups in all); cb_select_ws and cb_select_status
    reject bad arguments before any launch or device access."""
    n = cb.cb_select_workspace_bytes
    # 64 rows of 65536: four parts of 16384; a 256-byte-aligned header of
    # 4 + 64*8 words, then per unit the 4 passes x 4 parts x 256 digit counts
    assert n(64, 65536) == 2304 + 64 * (4 * 4 * 256) * 4
    assert n(128, 16385) > 0                  # two parts
    assert n(2, 10**6) > 0                    # 62 parts of 16384
    assert n(64, 16384) == 0                  # short rows: one workgroup per row
    assert n(129, 65536) == 0                 # too many units to split
    assert n(1, 2**31 - 2**16) == 0           # more than 256 parts of 65536
    assert n(0, 65536) == 0 and n(64, 0) == 0 and n(-1, 100) == 0
    fake = 1 << 20
    L = ctypes.byref
    k = ctypes.c_int64(0)
    S = cb._lib.cb_select_ws
    need = n(64, 65536)
    assert S(None, 64, 65536, 0.25, fake, L(k), fake, need, None) == -1
    assert S(fake, 64, 65536, 0.0, fake, L(k), fake, need, None) == -4
    assert S(fake, 0, 65536, 0.25, fake, L(k), fake, need, None) == -2
    assert S(fake + 4, 64, 65536, 0.25, fake, L(k), fake, need, None) == -6
    assert S(fake, 64, 65536, 0.25, fake, L(k), fake, need - 1, None) == -5
    assert S(fake, 64, 65536, 0.25, fake, L(k), fake + 8, need, None) == -6
    st = cb._lib.cb_select_status
    assert st(0, 65536, fake, need, None) == -2
    assert st(64, 16384, None, 0, None) == 0   # rows not split: nothing can time out
    assert st(64, 65536, None, need, None) == -5
    assert st(64, 65536, fake, need - 1, None) == -5


def test_score_status_validates_before_touching_the_device(cb):
    lay = cb.layout(1, 4, 2, 64, 16, 512, dtype="f32")
    ws_n = cb.cb_score_workspace_bytes(lay)
    L = ctypes.byref
    assert cb._lib.cb_score_status(None, 1 << 20, ws_n, None) == -1
    assert cb._lib.cb_score_status(L(lay), None, ws_n, None) == -5
    assert cb._lib.cb_score_status(L(lay), 1 << 20, ws_n - 1, None) == -5
    assert cb._lib.cb_score_status(L(cb.layout(1, 3, 2, 64, 16, 512)), 1 << 20, ws_n, None) == -2


def test_wait_limit_hook_round_trips(cb):
    prev = cb.cb_set_wait_limit(7)
    try:
        assert cb.cb_set_wait_limit(0) == 7
        assert cb.cb_set_wait_limit(prev) == 0
    finally:
        cb.cb_set_wait_limit(prev)
    assert prev == 1 << 21


def test_budgets_match_oracle(cb, oracle):
    orc = oracle.Oracle()
    for T in (1, 2, 41, 100, 8192, 65536, 2**31 - 2**16):
        for r in (1, 2, 4, 8, 16, 32, 64, 128):
            assert cb.cb_budget_fanout(T, r) == orc.budget_fanout(T, r)
    for T_old, T_new, r in [(0, 50, 4), (100, 50, 4), (4096, 16384, 16), (7, 1, 3)]:
        assert cb.cb_budget_chain(T_old, T_new, r, True) == orc.budget_chain(T_old, T_new, r, True)
        for B in (1, 60, 10**6):
            assert cb.cb_budget_chain(T_old, T_new, r, False, B) == \
                orc.budget_chain(T_old, T_new, r, False, B)
    assert cb._lib.cb_budget_fanout(0, 4) == -2 and cb._lib.cb_budget_fanout(5, 0) == -2
    assert cb._lib.cb_budget_chain(-1, 5, 4, 1, 0) == -2
    assert cb._lib.cb_budget_chain(1, 5, 4, 0, 0) == -2


def test_position_path_validation(cb):
    L = ctypes.byref
    lay = cb.layout(36, 32, 8, 128, 64, 8192)
    n = cb.cb_position_workspace_bytes(lay)
    assert n > cb.cb_score_workspace_bytes(lay)
    # G = 16 (more than 8 heads per group) is not taken by the position path
    assert cb._lib.cb_position_workspace_bytes(L(cb.layout(1, 32, 2, 128, 8, 100))) == 0
    fake = 1 << 20
    P = cb._lib.cb_position_score
    assert P(fake, fake, L(lay), 2.0, 2.0, None, None, None, None, fake, n, None) == -1
    assert P(fake, fake, L(lay), 1.0, 2.0, fake, None, None, None, fake, n, None) == -2
    assert P(fake, fake, L(lay), 9.0, 2.0, fake, None, None, None, fake, n, None) == -2
    assert P(fake, fake, L(lay), 2.0, -1.0, fake, None, None, None, fake, n, None) == -2
    assert P(fake, fake, L(lay), 2.0, 2.0, fake, None, None, None, fake, n - 1, None) == -5
    assert P(fake, fake, L(lay), 2.0, 2.0, fake + 4, None, None, None, fake, n, None) == -6
    S = cb._lib.cb_select_spans
    k = ctypes.c_int64(0)
    wsn = cb.cb_spans_workspace_bytes(1, 100, 16)
    assert S(fake, 1, 100, 40, 40, 16, fake, L(k), fake, wsn, None) == -2   # budget < 41 forced
    assert S(fake, 1, 100, 41, 40, 65, fake, L(k), fake, wsn, None) == -2   # width > 64
    assert S(fake, 1, 100, 41, 40, 16, fake, L(k), fake, wsn - 1, None) == -5
    assert S(None, 1, 100, 41, 40, 16, fake, L(k), fake, wsn, None) == -1
    G = cb._lib.cb_gather_rows
    assert G(fake, 1, 100, 6, fake, 5, fake, None) == -2
    assert G(fake + 4, 1, 100, 32, fake, 5, fake, None) == -6
    assert G(fake, 1, 100, 32, fake, 0, fake, None) == -2


def test_noalloc_rejects_before_touching_the_device(cb):
    L = ctypes.byref
    fake = 1 << 20
    N = cb._lib.cb_pipeline_noalloc
    assert N(fake, fake, fake, None, 0.25, fake, None, fake, fake, fake, None, None) == -1
    bad = cb.layout(1, 3, 2, 64, 16, 512)
    assert N(fake, fake, fake, L(bad), 0.25, fake, None, fake, fake, fake, None, None) == -2
    # needs more than the 64 MiB the library holds: rejected, nothing launched
    big = cb.layout(48, 40, 8, 128, 64, 2**20)
    assert cb.cb_score_workspace_bytes(big) > 64 << 20
    assert N(fake, fake, fake, L(big), 0.25, fake, None, fake, fake, fake, None, None) == -5
