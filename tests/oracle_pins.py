"""Pins for the CPU oracle: facts fixed by the paper or by mathematics.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises AssertionError
when the oracle disagrees with the fact.  None of them retypes the oracle's
formula: they use closed forms, exact special cases, library routines
(numpy matmul, scipy softmax / logsumexp, Python's sort), brute-force
enumeration, invariants, and figures the paper prints (``golden/``).

``test_oracle_pins.py`` runs them against the real oracle and
``test_oracle_mutants.py`` shows that plausible mistakes planted in the
oracle's C source each fail at least one of them.
"""
from __future__ import annotations

import itertools
import math
import os

import numpy as np
from scipy.special import logsumexp, softmax

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rand(rng, shape, dtype="f32", lo=None, hi=None):
    if lo is not None:
        x = rng.integers(lo, hi + 1, size=shape).astype(np.float32)
    else:
        x = rng.standard_normal(shape).astype(np.float32)
    if dtype == "f32":
        return x
    u = x.view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def _as_f64(x):
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def golden(name):
    with open(os.path.join(GOLDEN, "paper_figures.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            key, value, _cite = [p.strip() for p in line.split("|")]
            if key == name:
                return float(value)
    raise KeyError(name)


def library_importance(q, k, scale=None):
    """Importance via numpy matmul + scipy softmax, heads grouped h -> h // G."""
    q64, k64 = _as_f64(q), _as_f64(k)
    L, Hq, m, D = q64.shape
    S, _, Hkv, T, _ = k64.shape
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    out = np.zeros((S, L, Hkv, T))
    for s in range(S):
        for l in range(L):
            for h in range(Hq):
                logits = scale * (q64[l, h] @ k64[s, l, h // G].T)  # [m, T]
                out[s, l, h // G] += softmax(logits, axis=1).sum(axis=0)
    return out


# --- importance -------------------------------------------------------------


def pin_library_softmax(orc):
    """Small random shapes (several GQA groups, ragged T) against numpy+scipy."""
    rng = np.random.default_rng(1)
    for (S, L, Hq, Hkv, D, m, T) in [(1, 1, 4, 2, 8, 3, 13), (2, 2, 6, 2, 4, 2, 7),
                                     (1, 1, 1, 1, 16, 5, 33), (1, 2, 8, 8, 8, 1, 5)]:
        for dtype in ("f32", "bf16"):
            q = _rand(rng, (L, Hq, m, D), dtype)
            k = _rand(rng, (S, L, Hkv, T, D), dtype)
            got = orc.score(q, k)
            want = library_importance(q, k)
            assert np.allclose(got, want, rtol=1e-12, atol=1e-15), (S, L, Hq, Hkv, D, m, T, dtype)


def pin_row_lse(orc):
    rng = np.random.default_rng(2)
    q = _rand(rng, (2, 4, 3, 8))
    k = _rand(rng, (1, 2, 2, 11, 8))
    _, lse = orc.score(q, k, with_lse=True)
    q64, k64 = _as_f64(q), _as_f64(k)
    for l in range(2):
        for h in range(4):
            want = logsumexp(q64[l, h] @ k64[0, l, h // 2].T / math.sqrt(8), axis=1)
            assert np.allclose(lse[0, l, h], want, rtol=1e-13), (l, h)


def pin_zero_query_uniform(orc):
    """q = 0 makes every row uniform: I_t = m*G/T exactly (T a power of two)."""
    rng = np.random.default_rng(3)
    for T in (1, 2, 16, 64):
        q = np.zeros((1, 6, 5, 8), np.float32)
        k = _rand(rng, (1, 1, 2, T, 8))
        imp = orc.score(q, k)
        assert np.all(imp == 5 * 3 / T), T


def pin_identical_rows_uniform(orc):
    rng = np.random.default_rng(4)
    q = _rand(rng, (1, 4, 3, 8))
    row = _rand(rng, (8,))
    k = np.broadcast_to(row, (1, 1, 2, 32, 8)).copy()
    imp = orc.score(q, k)
    assert np.all(imp == 3 * 2 / 32)


def pin_single_position(orc):
    rng = np.random.default_rng(5)
    q = _rand(rng, (2, 8, 7, 16))
    k = _rand(rng, (1, 2, 4, 1, 16))
    assert np.all(orc.score(q, k) == 7 * 2)


def pin_two_token_logistic(orc):
    """Two positions, one query row: the weight on position 0 is the logistic
    function of the scaled logit difference (scale 1/sqrt(D), D = 4 -> 1/2)."""
    q = np.zeros((1, 1, 1, 4), np.float32)
    q[0, 0, 0, 0] = 1.0
    k = np.zeros((1, 1, 1, 2, 4), np.float32)
    for a, b in [(2.0, 0.0), (0.0, 2.0), (5.0, -1.0), (1.5, 1.0)]:
        k[0, 0, 0, 0, 0] = a
        k[0, 0, 0, 1, 0] = b
        imp = orc.score(q, k)[0, 0, 0]
        want0 = 1.0 / (1.0 + math.exp(-(a - b) / 2.0))
        assert abs(imp[0] - want0) < 1e-15 and abs(imp[1] - (1 - want0)) < 1e-15, (a, b)
    # an explicit scale overrides 1/sqrt(D)
    k[0, 0, 0, 0, 0], k[0, 0, 0, 1, 0] = 1.0, 0.0
    imp = orc.score(q, k, scale=3.0)[0, 0, 0]
    assert abs(imp[0] - 1.0 / (1.0 + math.exp(-3.0))) < 1e-15


def pin_gqa_grouping(orc):
    """Query head h reads KV head h // G: with only head 1 of 4 active (G = 2),
    KV head 0 carries head 1's softmax plus head 0's uniform row, and KV head 1
    stays exactly uniform."""
    rng = np.random.default_rng(6)
    T = 16
    q = np.zeros((1, 4, 1, 8), np.float32)
    q[0, 1, 0] = _rand(rng, (8,))
    k = _rand(rng, (1, 1, 2, T, 8))
    imp = orc.score(q, k)[0, 0]
    assert np.all(imp[1] == 2 / T)
    want0 = 1 / T + softmax(_as_f64(q)[0, 1, 0] @ _as_f64(k)[0, 0, 0].T / math.sqrt(8))
    assert np.allclose(imp[0], want0, rtol=1e-13)


def pin_mass_invariant(orc):
    """Each row is a probability distribution: sum_t I = m * G per unit."""
    rng = np.random.default_rng(7)
    q = _rand(rng, (3, 6, 4, 8), "bf16")
    k = _rand(rng, (2, 3, 3, 29, 8), "bf16")
    imp = orc.score(q, k)
    assert np.allclose(imp.sum(axis=-1), 4 * 2, rtol=1e-13)
    assert np.all(imp >= 0)


def pin_shift_invariance(orc):
    """Adding the same vector u to every K row adds a per-row constant to the
    logits, which softmax removes.  Large integer u (logits ~ 1e3..1e4) also
    checks that the oracle survives logits far outside exp's range."""
    rng = np.random.default_rng(8)
    q = _rand(rng, (1, 2, 3, 8), lo=-3, hi=3)
    k = _rand(rng, (1, 1, 1, 20, 8), lo=-3, hi=3)
    base = orc.score(q, k)
    for scale_u in (1, 100, 1000):
        u = _rand(rng, (8,), lo=-scale_u, hi=scale_u)
        shifted = orc.score(q, k + u)
        assert np.all(np.isfinite(shifted))
        assert np.allclose(shifted, base, rtol=1e-9, atol=1e-300), scale_u


def pin_permutation_equivariance(orc):
    rng = np.random.default_rng(9)
    q = _rand(rng, (1, 4, 3, 8))
    k = _rand(rng, (1, 1, 2, 19, 8))
    perm = rng.permutation(19)
    a = orc.score(q, k)
    b = orc.score(q, k[:, :, :, perm])
    assert np.allclose(b, a[..., perm], rtol=1e-13)


def pin_single_row_topk_is_logit_topk(orc):
    """m = G = 1: importance is one softmax row, a monotone map of the logits,
    so the selection equals the top-k of the raw logits."""
    rng = np.random.default_rng(10)
    q = _rand(rng, (1, 1, 1, 16))
    k = _rand(rng, (1, 1, 1, 200, 16))
    imp = orc.score(q, k)
    logits = _as_f64(k)[0, 0, 0] @ _as_f64(q)[0, 0, 0]
    for keep in (1, 7, 50, 199, 200):
        want = np.sort(np.argsort(-logits, kind="stable")[:keep])
        assert np.array_equal(orc.select(imp, keep)[0, 0, 0], want), keep


def pin_bf16_widening(orc):
    """bf16 inputs are read as the exact fp32 values their bits encode."""
    rng = np.random.default_rng(11)
    q = _rand(rng, (1, 2, 2, 8), "bf16")
    k = _rand(rng, (1, 1, 1, 9, 8), "bf16")
    a = orc.score(q, k)
    b = orc.score(_as_f64(q).astype(np.float32), _as_f64(k).astype(np.float32))
    assert np.array_equal(a, b)


# --- selection --------------------------------------------------------------


def _valid_selection(scores, chosen):
    """Every chosen position outranks every other one under (score desc,
    index asc)."""
    others = [t for t in range(len(scores)) if t not in chosen]
    for a in chosen:
        for b in others:
            if not (scores[a] > scores[b] or (scores[a] == scores[b] and a < b)):
                return False
    return True


def pin_select_brute_force(orc):
    """For T <= 8 enumerate all keep-subsets: exactly one satisfies the
    ordering rule, and the oracle returns it in ascending order."""
    rng = np.random.default_rng(12)
    for trial in range(60):
        T = int(rng.integers(1, 9))
        keep = int(rng.integers(1, T + 1))
        scores = rng.integers(0, 4, size=T).astype(np.float64)  # many ties
        got = orc.select(scores[None], keep)[0]
        valid = [set(c) for c in itertools.combinations(range(T), keep)
                 if _valid_selection(scores, set(c))]
        assert len(valid) == 1
        assert set(got.tolist()) == valid[0], (scores, keep, got)
        assert np.all(np.diff(got) > 0)


def pin_select_python_sort(orc):
    rng = np.random.default_rng(13)
    for dtype in (np.float64, np.float32):
        imp = rng.integers(0, 50, size=(3, 300)).astype(dtype) / 7
        for keep in (1, 17, 150, 300):
            got = orc.select(imp, keep)
            for u in range(3):
                want = sorted(sorted(range(300), key=lambda t: (-float(imp[u, t]), t))[:keep])
                assert got[u].tolist() == want, (dtype, keep, u)


def pin_select_ties_and_specials(orc):
    # all equal -> the first keep positions
    assert orc.select(np.full((1, 10), 0.5), 4)[0].tolist() == [0, 1, 2, 3]
    # keep = T -> every position in order
    assert orc.select(np.arange(9.0)[None][:, ::-1].copy(), 9)[0].tolist() == list(range(9))
    # -0 and +0 are equal keys; NaN ranks below everything (fp32 and fp64)
    for dt in (np.float32, np.float64):
        x = np.array([[np.nan, -0.0, 0.0, -1.0, np.nan, 2.0]], dtype=dt)
        assert orc.select(x, 3)[0].tolist() == [1, 2, 5]
        assert orc.select(x, 4)[0].tolist() == [1, 2, 3, 5]
        assert orc.select(x, 5)[0].tolist() == [0, 1, 2, 3, 5]


# --- budget -----------------------------------------------------------------


def pin_keep_count(orc):
    # ceil(T / r) for integer compression ratios r (fan-out budget equation)
    for T in list(range(1, 200)) + [512, 8192, 32768, 65536, 100003, 2**30 + 1, 2**31 - 1]:
        for r in (1, 2, 3, 4, 7, 8, 16, 32, 64, 128):
            assert orc.keep_count(T, 1.0 / r) == -(-T // r), (T, r)
    assert orc.keep_count(10, 0.25) == golden("budget_T10_r4")
    # the paper's removal figures: 75 % at 4x, 94 % (rounded) at 16x
    T = 8192
    assert 1 - orc.keep_count(T, 0.25) / T == golden("removed_fraction_at_4x")
    assert round(100 * (1 - orc.keep_count(T, 1 / 16) / T)) == golden("removed_percent_at_16x_rounded")
    # float noise in ratio*T does not add a position; fractions round up
    assert 0.07 * 100 > 7 and orc.keep_count(100, 0.07) == 7
    assert orc.keep_count(1200, 0.07) == 84
    assert orc.keep_count(32768, 0.10) == 3277
    assert orc.keep_count(5, 1e-9) == 1
    assert orc.keep_count(7, 1.0) == 7
    # a genuine fractional part of 1e-4 at T near 2^31 still rounds up
    # (ratio * T = 2e9 + 1e-4 holds that fraction to within 3e-7)
    T = 2**31 - 1
    r = (2_000_000_000 + 1e-4) / T
    assert abs(r * T - (2_000_000_000 + 1e-4)) < 1e-6
    assert orc.keep_count(T, r) == 2_000_000_001
    for bad in (0.0, -0.5, 1.5, float("nan")):
        assert orc.keep_count(10, bad) < 0


# --- compaction -------------------------------------------------------------


def pin_compact(orc):
    rng = np.random.default_rng(14)
    for dtype in ("f32", "bf16"):
        S, L, Hkv, T, D, keep = 3, 2, 2, 11, 8, 4
        k = _rand(rng, (S, L, Hkv, T, D), dtype)
        v = _rand(rng, (S, L, Hkv, T, D), dtype)
        idx = np.sort(np.stack([rng.choice(T, keep, replace=False)
                                for _ in range(S * L * Hkv)]).reshape(S, L, Hkv, keep), axis=-1)
        ko, vo = orc.compact(k, v, idx)
        for s in range(S):
            for l in range(L):
                for g in range(Hkv):
                    rows = slice(s * keep, (s + 1) * keep)
                    assert np.array_equal(ko[l, g, rows], k[s, l, g][idx[s, l, g]])
                    assert np.array_equal(vo[l, g, rows], v[s, l, g][idx[s, l, g]])
        # keep = T with the identity selection returns the cache unchanged
        k1, v1 = k[:1], v[:1]
        ident = np.broadcast_to(np.arange(T, dtype=np.int32), (1, L, Hkv, T)).copy()
        ko, vo = orc.compact(k1, v1, ident)
        assert ko.tobytes() == k1.tobytes() and vo.tobytes() == v1.tobytes()


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
