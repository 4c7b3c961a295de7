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
from scipy.ndimage import maximum_filter1d
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


# --- position-level score (Appendix C.1) ------------------------------------


def library_attention(q, k, s=0):
    """a[l][h][r][t] of sender s via numpy matmul + scipy softmax."""
    q64, k64 = _as_f64(q), _as_f64(k)
    L, Hq, m, D = q64.shape
    Hkv = k64.shape[2]
    G = Hq // Hkv
    a = np.empty((L, Hq, m, k64.shape[3]))
    for l in range(L):
        for h in range(Hq):
            a[l, h] = softmax(q64[l, h] @ k64[s, l, h // G].T / math.sqrt(D), axis=1)
    return a


def pin_mean_query_attention_against_library(orc):
    """alpha = 0 gives mean query attention: Q_t = Pool_w of the layer sum of
    the mean over query tokens and heads; the pool is scipy's running maximum
    (edge padding leaves a clipped window's maximum unchanged)."""
    rng = np.random.default_rng(21)
    for (L, Hq, Hkv, D, m, T, w) in [(2, 4, 2, 8, 3, 20, 7), (1, 2, 1, 4, 2, 5, 7),
                                     (3, 6, 3, 8, 1, 1, 7), (1, 4, 4, 8, 4, 9, 3),
                                     (2, 2, 2, 4, 5, 13, 1)]:
        q = _rand(rng, (L, Hq, m, D))
        k = _rand(rng, (2, L, Hkv, T, D))
        for s in range(2):
            a = library_attention(q, k, s)
            q_pre = a.mean(axis=(1, 2)).sum(axis=0)
            want = maximum_filter1d(q_pre, size=w, mode="nearest")
            score, qs, _ = orc.position_score(q, k, pool_width=w, alpha=0.0)
            assert np.allclose(qs[s], want, rtol=1e-12, atol=0), (L, Hq, Hkv, T, w)
            assert np.array_equal(score[s], qs[s])


def pin_correction_unpooled_variance_identity(orc):
    """At p = 2 without pooling, C_t = 1 + sum_s Var_r(b) / sum_s (mean_r b)^2
    (population variance over query tokens; b averages the query heads of
    each KV-head group), and S_t = Q_t * C_t^alpha."""
    rng = np.random.default_rng(22)
    for (L, Hq, Hkv, D, m, T) in [(2, 4, 2, 8, 5, 17), (1, 6, 2, 4, 3, 8), (2, 2, 2, 8, 4, 6)]:
        q = _rand(rng, (L, Hq, m, D), "bf16")
        k = _rand(rng, (1, L, Hkv, T, D), "bf16")
        a = library_attention(q, k)
        G = Hq // Hkv
        b = a.reshape(L, Hkv, G, m, T).mean(axis=2)            # [L][Hkv][m][T]
        var = b.var(axis=2).sum(axis=(0, 1))
        mean_sq = (b.mean(axis=2) ** 2).sum(axis=(0, 1))
        for alpha in (2.0, 0.5):
            score, qs, corr = orc.position_score(q, k, pool_width=1, p=2.0, alpha=alpha)
            assert np.allclose(corr[0], 1.0 + var / mean_sq, rtol=1e-12), (L, Hq, Hkv, m, T)
            assert np.allclose(score[0], qs[0] * corr[0] ** alpha, rtol=1e-14)


def _one_hot_query(T=20, p_pos=(10, 12), logit=80.0):
    """m = 2 query tokens, one head (G = 1, D = 4, scale 1/2): token r puts
    essentially all its attention (1 - 1e-33) on position p_pos[r]."""
    q = np.zeros((1, 1, 2, 4), np.float32)
    q[0, 0, 0, 0] = 1.0
    q[0, 0, 1, 1] = 1.0
    k = np.zeros((1, 1, 1, T, 4), np.float32)
    k[0, 0, 0, p_pos[0], 0] = 2.0 * logit
    k[0, 0, 0, p_pos[1], 1] = 2.0 * logit
    return q, k


def pin_correction_closed_forms(orc):
    """Two query tokens peaking at positions 10 and 12.  Unpooled, at a peak
    one token carries all the attention: C_p = ((1/2) / (1/2)^p)^(1/(p-1)) = 2
    for every p.  Pooled over 7 positions, at t = 11 both tokens peak inside
    the window: the numerator pools each token (1 and 1, mean 1), the
    denominator pools the token mean (1/2): C_2 = 1 / (1/2)^2 = 4,
    C_3 = (1 / (1/8))^(1/2) = sqrt(8), C_inf = 1 / (1/2) = 2, and
    Q_11 = 1/2, so S = Q * C^2 = 8 at p = 2.  Far from both peaks the
    attention is uniform (all tokens alike): C = 1."""
    q, k = _one_hot_query()
    for p in (2.0, 3.0, 5.0, math.inf):
        _, _, corr = orc.position_score(q, k, pool_width=1, p=p)
        assert abs(corr[0, 10] - 2.0) < 1e-12 and abs(corr[0, 12] - 2.0) < 1e-12, p
    for p, want in ((2.0, 4.0), (3.0, math.sqrt(8.0)), (math.inf, 2.0)):
        score, qs, corr = orc.position_score(q, k, pool_width=7, p=p, alpha=2.0)
        assert abs(corr[0, 11] - want) < 1e-12, (p, corr[0, 11])
        assert abs(qs[0, 11] - 0.5) < 1e-12
        assert abs(score[0, 11] - 0.5 * want ** 2) < 1e-11
        assert abs(corr[0, 19] - 1.0) < 1e-9 and abs(corr[0, 0] - 1.0) < 1e-9
    # windows are centred: position 15 sees 12 (distance 3), position 16 does not
    _, _, corr = orc.position_score(q, k, pool_width=7, p=2.0)
    assert corr[0, 15] > 1.5 and abs(corr[0, 16] - 1.0) < 1e-9
    assert corr[0, 7] > 1.5 and abs(corr[0, 6] - 1.0) < 1e-9


def pin_correction_is_one_when_both_sums_vanish(orc):
    """A logit 1500 above all others: every other weight underflows to exactly
    0 in fp64, so away from position 0 both sums are 0 and C is set to 1."""
    q = np.zeros((1, 1, 2, 4), np.float32)
    q[0, 0, :, 0] = 1.0
    k = np.zeros((1, 1, 1, 12, 4), np.float32)
    k[0, 0, 0, 0, 0] = 3000.0
    score, qs, corr = orc.position_score(q, k)
    assert np.all(corr[0, 4:] == 1.0) and np.all(score[0, 4:] == 0.0)
    assert np.all(np.isfinite(corr)) and np.all(np.isfinite(score))


def pin_single_query_token_has_no_correction(orc):
    """m = 1: the per-token and the averaged attention coincide, so
    C_{p,t} = 1 exactly (pooled or not, any p) and S = Q."""
    rng = np.random.default_rng(23)
    q = _rand(rng, (2, 4, 1, 8))
    k = _rand(rng, (2, 2, 2, 15, 8))
    for w in (1, 7):
        for p in (2.0, 3.5, math.inf):
            score, qs, corr = orc.position_score(q, k, pool_width=w, p=p)
            assert np.all(corr == 1.0) and np.array_equal(score, qs), (w, p)


def pin_correction_at_least_one(orc):
    """mean_r Pool(b)^p >= (mean_r Pool(b))^p >= Pool(mean_r b)^p (power mean
    and max of means <= mean of maxes), so C_{p,t} >= 1."""
    rng = np.random.default_rng(24)
    q = _rand(rng, (2, 8, 6, 8), "bf16")
    k = _rand(rng, (1, 2, 2, 40, 8), "bf16")
    for p in (2.0, 3.0, math.inf):
        for w in (1, 7):
            _, _, corr = orc.position_score(q, k, pool_width=w, p=p)
            assert corr.min() >= 1.0 - 1e-12, (p, w, corr.min())


def pin_uniform_attention_score(orc):
    """q = 0: every weight is 1/T, so Q_t = L/T, C = 1 and S = L/T."""
    rng = np.random.default_rng(25)
    L, T = 3, 32
    q = np.zeros((L, 4, 2, 8), np.float32)
    k = _rand(rng, (2, L, 2, T, 8))
    score, qs, corr = orc.position_score(q, k)
    assert np.allclose(qs, L / T, rtol=1e-14) and np.allclose(corr, 1.0, rtol=1e-14)
    assert np.allclose(score, L / T, rtol=1e-14)


# --- budgets and span selection (Appendix C.2) -------------------------------


def pin_budgets(orc):
    for T in (1, 2, 41, 100, 8192, 65536, 2**31 - 1):
        for r in (1, 2, 4, 8, 16, 32, 64):
            assert orc.budget_fanout(T, r) == -(-T // r)
    T = 8192
    assert 1 - orc.budget_fanout(T, 4) / T == golden("removed_fraction_at_4x")
    assert round(100 * (1 - orc.budget_fanout(T, 16) / T)) == golden("removed_percent_at_16x_rounded")
    # chain: inherited positions raise the relative budget one for one
    assert orc.budget_chain(100, 50, 4, True) == 100 + 13
    assert orc.budget_chain(0, 50, 4, True) == 13
    assert orc.budget_chain(100, 50, 4, False, 120) == 120
    assert orc.budget_chain(100, 50, 4, False, 1000) == 150
    assert orc.budget_fanout(0, 4) < 0 and orc.budget_chain(1, 0, 4, True) < 0


def pin_spans_keep_all_and_forced_only(orc):
    rng = np.random.default_rng(26)
    nf = int(golden("forced_positions"))
    for T in (41, 100, 1000):
        sc = rng.random(T).astype(np.float32)
        assert np.array_equal(orc.select_spans(sc, T), np.arange(T))
        assert np.array_equal(orc.select_spans(sc, T + 50), np.arange(T))
        forced = np.array(sorted({0} | set(range(T - (nf - 1), T))), dtype=np.int32)
        assert np.array_equal(orc.select_spans(sc, len(forced)), forced), T
    with pytest_raises():
        orc.select_spans(rng.random(100).astype(np.float32), nf - 1)


class pytest_raises:
    def __enter__(self):
        return self

    def __exit__(self, et, ev, tb):
        assert et is RuntimeError, "expected the oracle to reject the call"
        return True


def pin_spans_constant_scores_take_a_prefix(orc):
    """All span means equal: earlier spans win, and inside the partial span
    the top position is its first one, so the selection is the forced set
    plus the first unforced positions."""
    W = int(golden("span_width"))
    for T, B, nl in ((100, 30, 4), (64, 20, 0), (200, 57, 40)):
        sc = np.full(T, 0.25, np.float32)
        forced = {0} | set(range(T - nl, T))
        want = sorted(forced | set([t for t in range(T) if t not in forced][:B - len(forced)]))
        assert orc.select_spans(sc, B, nl, W).tolist() == want, (T, B, nl)


def pin_spans_increasing_scores_take_the_top(orc):
    """s_t = t: spans rank from the last; inside the partial span the top is
    its last position and the interval grows right first, so the result is
    position 0 plus the B-1 highest positions."""
    for T, B, nl in ((100, 30, 4), (97, 41, 40), (300, 77, 0)):
        sc = np.arange(T, dtype=np.float32)
        assert orc.select_spans(sc, B, nl).tolist() == [0] + list(range(T - B + 1, T)), (T, B)


def pin_spans_first_position_gets_the_maximum(orc):
    """Position 0's score is replaced by the maximum before ranking: here it
    lifts the first span from last to second place."""
    sc = np.zeros(48, np.float32)
    sc[1:16] = 0.9
    sc[0] = -100.0
    sc[16:32] = 1.0
    sc[32:48] = 0.5
    assert orc.select_spans(sc, 32, 0).tolist() == list(range(32))


def pin_spans_ties_and_short_last_span(orc):
    """Equal span means favour the earlier span; the last span (8 positions)
    is ranked by its mean, not its sum."""
    sc = np.zeros(40, np.float32)
    sc[16:32] = 0.5
    sc[32:40] = 0.5          # same mean as span 1, a smaller sum
    sc[1:16] = 0.1
    got = orc.select_spans(sc, 1 + 16, 0)
    assert got.tolist() == [0] + list(range(16, 32))
    sc[32:40] = 0.6          # higher mean than span 1, a smaller sum
    got = orc.select_spans(sc, 1 + 8, 0)
    assert got.tolist() == [0] + list(range(32, 40))


def pin_spans_partial_interval_around_the_top(orc):
    """The span that does not fit contributes the unselected positions nearest
    its highest-scoring position, right first on equal distance, clipped to
    the span."""
    sc = np.zeros(64, np.float32)
    sc[1:] = 0.01
    sc[32:48] = 0.5
    sc[40] = 0.9             # span 2's top
    assert orc.select_spans(sc, 1 + 4, 0).tolist() == [0, 39, 40, 41, 42]
    sc[40] = 0.5
    sc[46] = 0.9             # top near the span's end: the interval is clipped
    assert orc.select_spans(sc, 1 + 5, 0).tolist() == [0, 43, 44, 45, 46, 47]


def pin_spans_forced_latents_and_order(orc):
    """Latent positions are kept whatever their scores, count toward the
    budget, and spans holding them add only their other positions."""
    rng = np.random.default_rng(27)
    T, nl = 150, 40
    sc = rng.random(T).astype(np.float32)
    sc[T - nl:] = -1.0
    for B in (41, 42, 60, 149):
        got = orc.select_spans(sc, B, nl)
        assert len(got) == B and np.all(np.diff(got) > 0)
        assert 0 in got and set(range(T - nl, T)) <= set(got.tolist())


def _spans_by_priority_list(sc, B, nl, W):
    """The same rule as one ordering: forced positions, then every span in
    rank order, each span's positions ordered by distance from its top
    (right first); the selection is the first B distinct positions."""
    T = len(sc)
    s = sc.astype(np.float64).copy()
    s[0] = s.max()
    spans = [(-(s[j:j + W].sum() / len(s[j:j + W])), j // W) for j in range(0, T, W)]
    order = [0] + list(range(T - nl, T))
    for _, j in sorted(spans):
        lo, hi = j * W, min(j * W + W, T)
        top = lo + int(np.argmax(s[lo:hi]))
        dist = sorted(range(lo, hi), key=lambda t: (abs(t - top), t < top))
        order += dist
    seen, out = set(), []
    for t in order:
        if t not in seen:
            seen.add(t)
            out.append(t)
    return sorted(out[:B])


def pin_spans_match_the_priority_list_form(orc):
    """Greedy filling equals taking a prefix of one priority order (each span
    either fits whole or is the last one visited)."""
    rng = np.random.default_rng(28)
    for trial in range(60):
        T = int(rng.integers(1, 300))
        nl = int(rng.integers(0, min(T, 45) + 1))
        nf = len({0} | set(range(T - nl, T)))
        B = int(rng.integers(nf, T + 1))
        sc = rng.random(T).astype(np.float32)
        if trial % 3 == 0:
            sc = np.round(sc * 4).astype(np.float32)     # many ties
        assert orc.select_spans(sc, B, nl).tolist() == _spans_by_priority_list(sc, B, nl, 16), \
            (T, B, nl)


def pin_gather_rows(orc):
    rng = np.random.default_rng(29)
    for dt in (np.uint16, np.float32):
        rows = rng.integers(0, 2**15, size=(3, 50, 24)).astype(dt)
        idx = np.sort(np.stack([rng.choice(50, 9, replace=False) for _ in range(3)]), axis=-1)
        out = orc.gather_rows(rows, idx)
        assert np.array_equal(out, np.concatenate([rows[s][idx[s]] for s in range(3)]))


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
