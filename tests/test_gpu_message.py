"""The paper's position-level selector and message path on MI355X, through the
C ABI, against the CPU oracle: cb_position_score (Q_t, C_{p,t}, S_t and the
importance it is built from), cb_select_spans (the span rule of Appendix C.2,
bit-exact on the same fp32 scores), cb_gather_rows (continuous rows,
bit-exact), and a four-agent sequential chain with relative and fixed budgets.
"""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest

import cb_workloads as W
from parity import check_importance, rtol_for

pytestmark = pytest.mark.gpu

FLOOR = 2.0 ** -60   # absolute floor for Q and S (see position_tols)


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch():
    import torch as _torch

    assert _torch.cuda.is_available(), "GPU tests need a GPU"
    return _torch


@pytest.fixture(scope="module")
def cb():
    import paper_2609_32046_amd as _cb

    return _cb


@pytest.fixture(scope="module")
def orc(oracle):
    return oracle.Oracle()


def to_dev(torch, a: np.ndarray):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_host(torch, t):
    t = t.cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def position_tols(dtype, p, alpha):
    """Relative tolerances of Q, C and S from the importance tolerance e: Q is
    a sum of weights (e); C^(p-1) is a ratio of two sums of p-th powers of
    weights (2pe), so C errs by 2pe/(p-1) (2e at p = inf, a ratio of two
    maxima); S = Q C^alpha by e + alpha*tol_C.  Positions whose weights all lie
    below 2^-103 lose their correction numerator to fp32 underflow; their S is
    below FLOOR, which is far under any selected score."""
    e = rtol_for(dtype)
    tc = 2 * e if math.isinf(p) else e * 2 * p / (p - 1)
    return e, tc, e + alpha * tc


def run_position(torch, cb, w, q, K, p, alpha):
    lay = cb.layout_of(w)
    buf = cb.PositionBuffers(lay)
    cb.cb_position_score(to_dev(torch, q), to_dev(torch, K), lay, buf.score, buf.ws, p=p,
                         alpha=alpha, qscore=buf.qscore, corr=buf.corr, importance=buf.importance)
    torch.cuda.synchronize()
    assert cb.cb_position_status(lay, buf.ws) == 0
    return dict(score=to_host(torch, buf.score), q=to_host(torch, buf.qscore),
                c=to_host(torch, buf.corr), imp=to_host(torch, buf.importance), buf=buf, lay=lay)


def check_position(orc, w, q, K, out, p, alpha, what, imp_units=None):
    """Q, C and S on every position of every sender; the importance on every
    unit, or on `imp_units` (each computed by the oracle alone)."""
    mG = w.q_len * w.group
    if imp_units is None:
        check_importance(out["imp"], orc.score(q, K), mG, w.dtype, f"{what} importance")
    else:
        for (s, l, g) in imp_units:
            ku = np.ascontiguousarray(K[s, l, g])[None, None, None]
            imp_o = orc.score(W.unit_q(w, q, l, g), ku)[0, 0, 0]
            check_importance(out["imp"][s, l, g], imp_o, mG, w.dtype, f"{what} unit {(s, l, g)}")
    s_o, q_o, c_o = orc.position_score(q, K, p=p, alpha=alpha)
    e, tc, ts = position_tols(w.dtype, p, alpha)
    for name, g, o, tol in (("Q", out["q"], q_o, e), ("S", out["score"], s_o, ts)):
        err = np.abs(g.astype(np.float64) - o)
        bad = err > tol * np.abs(o) + FLOOR
        assert not bad.any(), (f"{what}: {name} off at {bad.sum()} positions; worst "
                               f"{(err / (tol * np.abs(o) + FLOOR)).max():.2f}x tolerance")
    meaningful = s_o > FLOOR * 2.0 ** 20
    err = np.abs(out["c"].astype(np.float64) - c_o)
    bad = (err > tc * c_o) & meaningful
    assert not bad.any(), f"{what}: C off at {bad.sum()} positions (max rel {(err / c_o).max():.2e})"
    rel = (np.abs(out["score"] - s_o) / np.maximum(s_o, FLOOR))[meaningful]
    say(f"  {what}: max rel err S {rel.max():.2e} (tolerance {ts:.1e})")
    return s_o


POS_SWEEP = [
    # (layers, Hq, Hkv, D, m, T, S, dtype, kdist)
    (1, 4, 2, 64, 16, 512, 1, "f32", "normal"),          # the tiny workload's shape, G = 2 -> 4
    (2, 8, 2, 128, 16, 1537, 1, "bf16", "chanscale"),    # G = 4, ragged T
    (1, 32, 8, 128, 64, 3000, 1, "bf16", "chanscale"),   # Qwen3-8B unit shape, several chunks
    (2, 10, 2, 128, 8, 700, 2, "bf16", "peaked"),        # G = 5 -> 8, two senders
    (1, 8, 1, 128, 20, 2100, 1, "bf16", "student_t_outliers"),   # G = 8
    (1, 8, 8, 64, 5, 37, 1, "f32", "normal"),            # G = 1
    (1, 4, 1, 128, 128, 1100, 1, "bf16", "normal"),      # 512 rows
    (1, 8, 1, 64, 80, 300, 1, "f32", "normal"),          # 640 rows: two row groups
    (1, 3, 1, 128, 7, 5, 1, "bf16", "normal"),           # T < 7: windows clipped at both ends
]


@pytest.mark.parametrize("case", POS_SWEEP, ids=[f"L{c[0]}H{c[1]}-{c[2]}D{c[3]}m{c[4]}T{c[5]}S{c[6]}{c[7]}"
                                                 for c in POS_SWEEP])
def test_position_score_sweep(torch, cb, orc, case):
    L, Hq, Hkv, D, m, T, S, dt, kd = case
    w = W.custom(layers=L, q_heads=Hq, kv_heads=Hkv, head_dim=D, q_len=m, seq_len=T, senders=S,
                 dtype=dt, kdist=kd, cfg_id=200 + T)
    say(f"case position {case}")
    q = W.gen_q(w)
    K, _ = W.gen_kv(w, want_v=False)
    for p, alpha in ((2.0, 2.0), (3.0, 1.0), (math.inf, 2.0), (1.5, 0.5), (8.0, 4.0), (2.0, 0.0)):
        out = run_position(torch, cb, w, q, K, p, alpha)
        check_position(orc, w, q, K, out, p, alpha, f"{case} p={p} a={alpha}")
        if (p, alpha) != (2.0, 2.0):
            continue
        # the span rule on the GPU's own scores: bit-exact
        budget = max(orc.budget_fanout(T, 4), min(T, 41))
        check_spans_on(torch, cb, orc, out["score"], budget, 40)


def test_position_score_deterministic(torch, cb, orc):
    w = W.custom(layers=3, q_heads=8, kv_heads=2, head_dim=128, q_len=32, seq_len=5000,
                 kdist="chanscale", cfg_id=299)
    say("case position determinism")
    q = W.gen_q(w)
    K, _ = W.gen_kv(w, want_v=False)
    a = run_position(torch, cb, w, q, K, 2.0, 2.0)
    b = run_position(torch, cb, w, q, K, 2.0, 2.0)
    for key in ("score", "q", "c", "imp"):
        assert a[key].tobytes() == b[key].tobytes(), key


def check_spans_on(torch, cb, orc, scores, budget, n_latent, width=16):
    """cb_select_spans on fp32 scores [S][T] against the oracle's span rule on
    the same scores: identical positions."""
    scores = np.ascontiguousarray(scores, dtype=np.float32)
    S, T = scores.shape
    count = min(budget, T)
    idx = torch.empty((S, count), dtype=torch.int32, device="cuda")
    ws = torch.empty(cb.cb_spans_workspace_bytes(S, T, width), dtype=torch.uint8, device="cuda")
    got_count = cb.cb_select_spans(to_dev(torch, scores), S, T, budget, idx, ws, n_latent=n_latent,
                                   width=width)
    torch.cuda.synchronize()
    assert got_count == count
    got = to_host(torch, idx)
    for s in range(S):
        want = orc.select_spans(scores[s], budget, n_latent, width)
        assert np.array_equal(got[s], want), (T, budget, n_latent, width, s)
    return got


@pytest.mark.parametrize("T", [1, 2, 15, 16, 17, 41, 100, 512, 1537, 8192, 65536, 65537, 100003])
def test_select_spans_cases(torch, cb, orc, T):
    """Hand-made scores (random, constant, heavy ties, increasing) at ragged
    lengths, span widths, latent counts and budgets from the forced count to
    past T; three senders at once."""
    rng = np.random.default_rng(T)
    say(f"case spans T={T}")
    patterns = {
        "random": rng.random((3, T)).astype(np.float32),
        "constant": np.full((3, T), 0.125, np.float32),
        "ties": np.round(rng.random((3, T)) * 3).astype(np.float32) / 4,
        "increasing": np.broadcast_to(np.arange(T, dtype=np.float32), (3, T)).copy(),
    }
    patterns["random"][1, ::5] = np.float32(0.5)
    for name, sc in patterns.items():
        for width in (16, 1, 7, 64):
            for nl in (40, 0, 3):
                nf = min(T, nl + 1)
                for budget in sorted({nf, nf + 1, -(-T // 4), T - 1, T, T + 5}):
                    if budget < nf or budget < 1:
                        continue
                    check_spans_on(torch, cb, orc, sc, budget, nl, width)


@pytest.mark.parametrize("row_bytes", [8192, 4, 8, 20, 16, 256])
def test_gather_rows(torch, cb, orc, row_bytes):
    rng = np.random.default_rng(row_bytes)
    S, T, count = 3, 777, 123
    rows = rng.integers(0, 2**31, size=(S, T, row_bytes // 4), dtype=np.int64).astype(np.int32)
    idx = np.sort(np.stack([rng.choice(T, count, replace=False) for _ in range(S)]), axis=-1)
    idx = idx.astype(np.int32)
    out = torch.empty((S * count, row_bytes // 4), dtype=torch.int32, device="cuda")
    cb.cb_gather_rows(to_dev(torch, rows), S, T, row_bytes, to_dev(torch, idx), count, out)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(torch, out), orc.gather_rows(rows, idx))
    # indices outside [0, T) give zero rows
    bad = idx.copy()
    bad[:, ::10] = -1
    bad[:, 5] = T
    out.fill_(7)
    cb.cb_gather_rows(to_dev(torch, rows), S, T, row_bytes, to_dev(torch, bad), count, out)
    torch.cuda.synchronize()
    want = orc.gather_rows(rows, np.where((bad < 0) | (bad >= T), 0, bad))
    want[((bad < 0) | (bad >= T)).reshape(-1)] = 0
    assert np.array_equal(to_host(torch, out), want)


def test_message_full_size_qwen3_8b(torch, cb, orc):
    """The paper's selector at the Qwen3-8B shape (36 layers, 32/8 heads,
    T = 8192, m = 64, bf16): S_t on every position against the oracle, the
    span rule at 4x (ceil(T/4) positions with the first position and 40
    latents forced) bit-exact, and the 8 KiB continuous rows gathered."""
    w = W.get("qwen3-8b-8k-bf16")
    say("case message qwen3-8b-8k-bf16 (full size)")
    q = W.gen_q(w)
    K, _ = W.gen_kv(w, want_v=False, progress=say)
    out = run_position(torch, cb, w, q, K, 2.0, 2.0)
    say("  oracle position score (all 288 units)")
    check_position(orc, w, q, K, out, 2.0, 2.0, "qwen3-8b", imp_units=W.sample_units(w, 6))
    budget = orc.budget_fanout(w.seq_len, 4)
    idx = check_spans_on(torch, cb, orc, out["score"], budget, 40)
    rows = W.gen_rows(w)
    got = torch.empty((budget, w.d_model), dtype=torch.bfloat16, device="cuda")
    cb.cb_gather_rows(to_dev(torch, rows), 1, w.seq_len, w.d_model * 2, to_dev(torch, idx), budget,
                      got)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(torch, got), orc.gather_rows(rows, idx))


@pytest.mark.parametrize("name", ["fanin-3x16k-bf16", "longctx-32k-bf16", "hybrid-64k-bf16"])
def test_position_score_long_workloads_two_layers(torch, cb, orc, name):
    """Full per-unit shapes of the other workloads (G = 5 for the long-context
    one) on their first two layers."""
    w = W.get(name).with_layers(2)
    say(f"case position {name} first 2 layers")
    q = W.gen_q(w)
    K, _ = W.gen_kv(w, want_v=False)
    out = run_position(torch, cb, w, q, K, 2.0, 2.0)
    check_position(orc, w, q, K, out, 2.0, 2.0, name)
    budget = orc.budget_fanout(w.seq_len, 8)
    check_spans_on(torch, cb, orc, out["score"], budget, 40)


@pytest.mark.parametrize("relative", [True, False])
def test_sequential_chain(torch, cb, orc, relative):
    """Four agents in a chain (LongBench v2 topology): agent i's state is the
    previous message's positions followed by its own new prompt and 40 latent
    positions; all are scored together, the chain budget (relative:
    T_old + ceil(T_new/4); fixed: min(1500, T_old + T_new)) is filled by the
    span rule, and the message carries the selected rows and their source
    ids.  Every step bit-exact against the oracle on the GPU's scores."""
    r, n_latent, B_max = 4, 40, 1500
    base = W.custom(layers=2, q_heads=8, kv_heads=2, head_dim=128, q_len=16, seq_len=1,
                    kdist="chanscale", cfg_id=400 + int(relative))
    rng = np.random.default_rng(41 + int(relative))
    msg_rows = np.zeros((0, base.d_model), np.uint16)
    msg_ids = np.zeros((0,), np.int32)
    say(f"case chain relative={relative}")
    for agent, T_new in enumerate([3000, 2500, 2800, 2600]):
        T_old = len(msg_ids)
        T = T_old + T_new
        w = W.custom(layers=2, q_heads=8, kv_heads=2, head_dim=128, q_len=16, seq_len=T,
                     kdist="chanscale", cfg_id=410 + 2 * agent + int(relative))
        q = W.gen_q(w)
        K, _ = W.gen_kv(w, want_v=False)
        rows = np.concatenate([msg_rows, W.gen_rows(w, T=T_new)[0]])[None]
        ids = np.concatenate([msg_ids, (agent + 1) * 1_000_000 + np.arange(T_new, dtype=np.int32)])
        budget = cb.cb_budget_chain(T_old, T_new, r, relative, B_max)
        assert budget == orc.budget_chain(T_old, T_new, r, relative, B_max)
        out = run_position(torch, cb, w, q, K, 2.0, 2.0)
        idx = check_spans_on(torch, cb, orc, out["score"], budget, n_latent)
        count = idx.shape[1]
        assert count == min(budget, T)
        d_idx = to_dev(torch, idx)
        got_rows = torch.empty((count, w.d_model), dtype=torch.bfloat16, device="cuda")
        got_ids = torch.empty((count,), dtype=torch.int32, device="cuda")
        cb.cb_gather_rows(to_dev(torch, rows), 1, T, w.d_model * 2, d_idx, count, got_rows)
        cb.cb_gather_rows(to_dev(torch, ids[None]), 1, T, 4, d_idx, count, got_ids)
        torch.cuda.synchronize()
        msg_rows = to_host(torch, got_rows)
        msg_ids = to_host(torch, got_ids)
        assert np.array_equal(msg_rows, orc.gather_rows(rows, idx))
        assert np.array_equal(msg_ids, orc.gather_rows(ids[None, :, None], idx)[:, 0])
        # the current latents (last 40 positions) and the first position survive
        assert set(range((agent + 1) * 1_000_000 + T_new - n_latent,
                         (agent + 1) * 1_000_000 + T_new)) <= set(msg_ids.tolist())
        say(f"  agent {agent}: T_old {T_old} + T_new {T_new} -> {count} positions")
    assert len(msg_ids) == len(set(msg_ids.tolist()))


def test_position_wait_timeout_is_reported(torch, cb, orc):
    w = W.custom(layers=2, q_heads=8, kv_heads=2, head_dim=128, q_len=16, seq_len=3000, cfg_id=298)
    say("case position wait timeout")
    q = W.gen_q(w)
    K, _ = W.gen_kv(w, want_v=False)
    lay = cb.layout_of(w)
    buf = cb.PositionBuffers(lay)
    prev = cb.cb_set_wait_limit(0)
    try:
        cb.cb_position_score(to_dev(torch, q), to_dev(torch, K), lay, buf.score, buf.ws)
        assert cb.cb_position_status(lay, buf.ws) == -8
        assert torch.isnan(buf.score).all().item()
    finally:
        cb.cb_set_wait_limit(prev)
    out = run_position(torch, cb, w, q, K, 2.0, 2.0)
    check_position(orc, w, q, K, out, 2.0, 2.0, "after timeout")
