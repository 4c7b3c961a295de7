"""Parity of the HIP path (through the C ABI) with the CPU oracle on MI355X.

Small shapes are compared on every unit.  The full-size workloads run through
the GPU in the launch configuration the benchmark times and are compared on
a seeded sample of units the oracle computes one by one, plus exact checks on
every unit (selection against the oracle's comparison sort on the GPU's own
fp32 scores, bit-exact compaction) and invariants.
"""
from __future__ import annotations

import concurrent.futures
import os
import sys

import numpy as np
import pytest

import cb_workloads as W
from parity import (check_importance, check_invariants, check_lse, check_selection_band,
                    logit_magnitude_rtol)

pytestmark = pytest.mark.gpu


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
    return torch.from_numpy(a).cuda()


def to_host(torch, t):
    t = t.cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def run_gpu(torch, cb, w, q, K, V, keep_ratio, scale=0.0, fused=True):
    """fused: the single cb_pipeline call; otherwise cb_score, cb_select and
    cb_compact one after the other."""
    lay = cb.layout_of(w, scale)
    buf = cb.Buffers(lay, keep_ratio)
    qd, kd, vd = to_dev(torch, q), to_dev(torch, K), to_dev(torch, V)
    (cb.run_pipeline if fused else cb.run_steps)(qd, kd, vd, buf)
    torch.cuda.synchronize()
    out = dict(imp=to_host(torch, buf.importance), lse=to_host(torch, buf.row_lse),
               idx=to_host(torch, buf.idx), k_out=to_host(torch, buf.k_out),
               v_out=to_host(torch, buf.v_out), keep=buf.keep)
    return out


def check_all_units(orc, w, q, K, V, out, scale=0.0, what=""):
    """Oracle on every unit (small shapes)."""
    mG = w.q_len * w.group
    imp_o, lse_o = orc.score(q, K, scale=scale, with_lse=True)
    check_importance(out["imp"], imp_o, mG, w.dtype, what)
    check_lse(out["lse"], lse_o, w.dtype, what)
    keep = out["keep"]
    flat_imp = out["imp"].reshape(-1, w.seq_len)
    flat_idx = out["idx"].reshape(-1, keep)
    # exact: oracle's comparison sort on the GPU's fp32 scores
    assert np.array_equal(orc.select(flat_imp, keep), flat_idx), f"{what}: select not exact"
    orc_idx = orc.select(imp_o.reshape(-1, w.seq_len), keep)
    for uidx in range(flat_idx.shape[0]):
        check_selection_band(flat_idx[uidx], imp_o.reshape(-1, w.seq_len)[uidx], keep, mG,
                             w.dtype, orc_idx[uidx], f"{what} unit {uidx}")
    ko, vo = orc.compact(K, V, out["idx"])
    assert ko.tobytes() == out["k_out"].tobytes() and vo.tobytes() == out["v_out"].tobytes(), \
        f"{what}: compaction not bit-exact"


def oracle_units(orc, w, q, K, units):
    """Oracle importance and row_lse of each listed unit, one unit per call on
    a host thread pool: the oracle is single-threaded and ctypes releases the
    GIL while it runs.  Yields ((s, l, g), importance[T], row_lse[G][m])."""
    def one(u):
        s, l, g = u
        qu = W.unit_q(w, q, l, g)
        ku = np.ascontiguousarray(K[s, l, g])[None, None, None]
        imp, lse = orc.score(qu, ku, with_lse=True)
        return u, imp[0, 0, 0], lse[0, 0]

    threads = min(16, os.cpu_count() or 1)
    with concurrent.futures.ThreadPoolExecutor(threads) as ex:
        for i, res in enumerate(ex.map(one, units)):
            if (i + 1) % max(1, len(units) // 4) == 0:
                say(f"  oracle: {i + 1}/{len(units)} units")
            yield res


def check_units(orc, w, q, K, V, outs, units, what=""):
    """Importance and row_lse against the oracle on the listed units, for
    every output in `outs` (calls on the same inputs, e.g. one per keep
    ratio); selection and compaction exact on every unit of every output."""
    mG = w.q_len * w.group
    T = w.seq_len
    for (s, l, g), imp_o, lse_o in oracle_units(orc, w, q, K, units):
        for out in outs:
            tag = f"{what} keep={out['keep']} unit {(s, l, g)}"
            check_importance(out["imp"][s, l, g], imp_o, mG, w.dtype, tag)
            check_lse(out["lse"][s, l, g * w.group:(g + 1) * w.group], lse_o, w.dtype, tag)
            keep = out["keep"]
            orc_idx = orc.select(imp_o[None], keep)[0]
            check_selection_band(out["idx"][s, l, g], imp_o, keep, mG, w.dtype, orc_idx, tag)
    for out in outs:
        keep = out["keep"]
        flat_imp = out["imp"].reshape(-1, T)
        flat_idx = out["idx"].reshape(-1, keep)
        say(f"  exact select on every unit (keep {keep})")
        assert np.array_equal(orc.select(flat_imp, keep), flat_idx), f"{what}: select not exact"
        check_invariants(flat_imp, flat_idx, keep, mG, w.dtype, what)
        say(f"  bit-exact compaction on every unit (keep {keep})")
        ko, vo = orc.compact(K, V, out["idx"])
        assert np.array_equal(ko, out["k_out"]) and np.array_equal(vo, out["v_out"]), \
            f"{what}: compaction not bit-exact"


def check_sampled(orc, w, q, K, V, out, units, what=""):
    check_units(orc, w, q, K, V, [out], units, what)


def layer_units(w, layers):
    """Every (sender, KV head) of the listed layers."""
    return [(s, l, g) for s in range(w.senders) for l in layers for g in range(w.kv_heads)]


def gen(w):
    q = W.gen_q(w)
    K, V = W.gen_kv(w, progress=say)
    return q, K, V


# --------------------------------------------------------------------------- small


def test_tiny_fp32_all_units(torch, cb, orc):
    w = W.get("tiny-fp32")
    say("case tiny-fp32")
    q, K, V = gen(w)
    out = run_gpu(torch, cb, w, q, K, V, 0.25)
    assert out["keep"] == 128
    check_all_units(orc, w, q, K, V, out, what="tiny-fp32")


SWEEP = [
    # (layers, Hq, Hkv, D, m, T, S, dtype, kdist)
    (1, 1, 1, 64, 1, 1, 1, "f32", "normal"),
    (1, 2, 1, 128, 3, 5, 1, "bf16", "normal"),
    (2, 4, 2, 64, 16, 63, 1, "f32", "normal"),
    (1, 4, 4, 128, 7, 64, 2, "bf16", "chanscale"),
    (1, 8, 2, 128, 5, 65, 1, "bf16", "normal"),
    (2, 10, 2, 128, 13, 511, 1, "bf16", "peaked"),
    (1, 6, 3, 64, 9, 513, 3, "f32", "normal"),
    (1, 16, 2, 128, 70, 700, 1, "bf16", "student_t_outliers"),
    (1, 5, 1, 128, 33, 1000, 1, "bf16", "normal"),
    (1, 32, 8, 128, 64, 1537, 1, "bf16", "chanscale"),
    (1, 8, 1, 128, 80, 300, 1, "bf16", "normal"),        # 640 rows: two row groups
    (1, 8, 1, 64, 128, 257, 1, "f32", "normal"),         # 1024 rows, fp32
    # wave counts that do not divide a K tile's 16-byte chunks evenly
    (1, 3, 1, 128, 32, 777, 1, "bf16", "normal"),        # 96 rows: 3 waves
    (1, 5, 1, 128, 32, 600, 1, "bf16", "student_t_outliers"),  # 160 rows: 5 waves
    (1, 7, 1, 64, 32, 900, 1, "bf16", "chanscale"),      # 224 rows: 7 waves, D = 64
    # 257 to 320 rows: four waves of five 16-row blocks
    (1, 5, 1, 128, 60, 777, 1, "bf16", "normal"),        # 300 rows: last block partly padding
    (2, 10, 2, 64, 64, 1100, 1, "f32", "peaked"),        # 320 rows, fp32, D = 64
    (1, 20, 4, 128, 52, 2049, 2, "bf16", "student_t_outliers"),  # 260 rows, two senders
]


@pytest.mark.parametrize("case", SWEEP, ids=[f"L{c[0]}H{c[1]}-{c[2]}D{c[3]}m{c[4]}T{c[5]}S{c[6]}{c[7]}"
                                             for c in SWEEP])
def test_shape_sweep_all_units(torch, cb, orc, case):
    L, Hq, Hkv, D, m, T, S, dt, kd = case
    w = W.custom(layers=L, q_heads=Hq, kv_heads=Hkv, head_dim=D, q_len=m, seq_len=T, senders=S,
                 dtype=dt, kdist=kd, cfg_id=100 + T)
    say(f"case sweep {case}")
    q, K, V = gen(w)
    for ratio in (0.25, 0.5, 1.0, 1e-6):
        out = run_gpu(torch, cb, w, q, K, V, ratio, fused=ratio != 0.5)
        assert out["keep"] == orc.keep_count(T, ratio)
        if ratio == 0.25:
            check_all_units(orc, w, q, K, V, out, what=f"sweep {case}")
        else:
            flat_imp = out["imp"].reshape(-1, T)
            assert np.array_equal(orc.select(flat_imp, out["keep"]),
                                  out["idx"].reshape(-1, out["keep"])), (case, ratio)
            ko, vo = orc.compact(K, V, out["idx"])
            assert ko.tobytes() == out["k_out"].tobytes() and vo.tobytes() == out["v_out"].tobytes()


def test_keep_all_returns_the_cache_unchanged(torch, cb, orc):
    w = W.custom(layers=2, q_heads=4, kv_heads=2, head_dim=128, q_len=8, seq_len=333)
    say("case keep-all identity")
    q, K, V = gen(w)
    out = run_gpu(torch, cb, w, q, K, V, 1.0)
    assert out["keep"] == 333
    assert np.array_equal(out["idx"], np.broadcast_to(np.arange(333, dtype=np.int32), (1, 2, 2, 333)))
    assert out["k_out"].tobytes() == K[0].tobytes() and out["v_out"].tobytes() == V[0].tobytes()


@pytest.mark.parametrize("dtype,D", [("f32", 64), ("f32", 128), ("bf16", 64), ("bf16", 128)])
def test_compact_out_of_range_indices_give_zero_rows(torch, cb, orc, dtype, D):
    """cb_compact on hand-made indices: entries outside [0, T) give all-zero
    rows, every other row is the oracle's byte copy; two senders, a keep that
    is not a multiple of any row block."""
    w = W.custom(layers=3, q_heads=4, kv_heads=2, head_dim=D, q_len=4, seq_len=300, senders=2,
                 dtype=dtype)
    say(f"case compact out-of-range {dtype} D={D}")
    _, K, V = gen(w)
    keep = 77
    rng = np.random.default_rng(17)
    idx = np.sort(rng.choice(300, size=(2, 3, 2, keep)), axis=-1).astype(np.int32)
    bad = rng.random(idx.shape) < 0.1
    idx[bad] = rng.choice(np.array([-1, -300, 300, 2**31 - 1], dtype=np.int32), size=int(bad.sum()))
    lay = cb.layout_of(w)
    kd, vd, idd = to_dev(torch, K), to_dev(torch, V), to_dev(torch, idx)
    ko = torch.empty((3, 2, 2 * keep, D), dtype=kd.dtype, device=kd.device)
    vo = torch.empty_like(ko)
    ko.fill_(7)
    vo.fill_(7)
    cb.cb_compact(kd, vd, idd, lay, keep, ko, vo)
    torch.cuda.synchronize()
    got_k, got_v = to_host(torch, ko), to_host(torch, vo)
    exp_k, exp_v = orc.compact(K, V, np.where(bad, 0, idx))
    rows_bad = np.zeros((3, 2, 2 * keep), dtype=bool)
    for s in range(2):
        rows_bad[:, :, s * keep:(s + 1) * keep] = bad[s]
    exp_k[rows_bad] = 0
    exp_v[rows_bad] = 0
    assert got_k.tobytes() == exp_k.tobytes()
    assert got_v.tobytes() == exp_v.tobytes()


@pytest.mark.parametrize("T", [1, 511, 2048, 2049, 4097, 8192, 8193, 16384, 16385, 16387, 32768,
                               32769, 40000, 65535, 65536, 65537, 100003])
def test_select_kernel_paths_on_fp32_scores(torch, cb, orc, T):
    """cb_select alone on hand-made fp32 scores, bit-exact against the
    oracle's comparison sort, at the row lengths where the kernel changes
    workgroup size or keys per thread: 4 to 64 keys per thread held in
    registers as 16-byte vectors (T <= 65536; scalar loads when T % 4 != 0),
    or re-read from L2 (longer rows).  Rows mix near-uniform
    values straddling a power of two, exact ties, -0/+0 and NaNs (one row
    with a NaN at every fifth position, so that keeping all positions puts
    the threshold on the NaN key), so that every radix pass and the tie rule
    are exercised; keep runs from 1 to T."""
    rng = np.random.default_rng(T)
    units = 4
    imp = (0.03125 * (1.0 + 0.01 * rng.standard_normal((units, T)))).astype(np.float32)
    imp[1, ::3] = np.float32(0.03125)                   # exact ties at a power of two
    imp[2, : T // 2] = imp[2, T // 2: T // 2 * 2]      # duplicated halves
    imp[3, ::5] = np.float32(np.nan)
    imp[0, 0] = np.float32(-0.0)
    if T > 2:
        imp[0, 1] = np.float32(0.0)
        imp[2, T - 1] = np.float32(np.nan)
    say(f"case select T={T}")
    dimp = to_dev(torch, imp)
    for ratio in (1e-9, 0.1, 0.25, 0.5, 1.0):
        keep = orc.keep_count(T, ratio)
        idx = torch.empty((units, keep), dtype=torch.int32, device="cuda")
        got_keep = cb.cb_select(dimp, units, T, ratio, idx)
        torch.cuda.synchronize()
        assert got_keep == keep
        assert np.array_equal(to_host(torch, idx), orc.select(imp, keep)), (T, ratio)


def test_identical_rows_tie_to_lowest_indices(torch, cb, orc):
    w = W.custom(layers=1, q_heads=4, kv_heads=2, head_dim=128, q_len=16, seq_len=1000)
    say("case identical rows")
    q, K, V = gen(w)
    K[:] = K[:, :, :, :1]   # every position of a unit holds the same key
    out = run_gpu(torch, cb, w, q, K, V, 0.25)
    imp = out["imp"].reshape(-1, 1000)
    assert np.all(imp == imp[:, :1])   # bitwise-equal scores
    assert np.array_equal(out["idx"].reshape(-1, 250), np.broadcast_to(np.arange(250), (2, 250)))
    check_importance(out["imp"], np.full(out["imp"].shape, 16 * 2 / 1000.0), 32, "bf16", "ties")


def test_shift_invariance_with_large_logits(torch, cb, orc):
    """K + u for every position: the logits of each row move by a constant
    (they span about -101 to +72 here); importance must not change beyond
    tolerance and nothing may overflow.  The fp32 tolerance grows with the
    logit magnitude: an absolute logit error d changes a probability by a
    factor exp(d), and the rounding of an fp32 dot product grows with the
    sum of |q_d k_d|.  The test prints the measured error."""
    w = W.custom(layers=1, q_heads=4, kv_heads=1, head_dim=128, q_len=8, seq_len=777, dtype="f32")
    say("case shift invariance")
    q, K, V = gen(w)
    base = run_gpu(torch, cb, w, q, K, V, 0.25)
    rng = np.random.default_rng(3)
    u = (rng.standard_normal(128) * 40).astype(np.float32)
    K2 = (K + u).astype(np.float32)
    out = run_gpu(torch, cb, w, q, K2, V, 0.25)
    assert np.all(np.isfinite(out["imp"]))
    imp_o = orc.score(q, K2)
    logits = (q.reshape(-1, 128).astype(np.float64) @ K2.reshape(-1, 128).astype(np.float64).T
              * 128 ** -0.5)
    rel = np.abs(out["imp"].astype(np.float64) - imp_o) / imp_o
    say(f"  logits {logits.min():.1f} .. {logits.max():.1f}; max rel err {rel.max():.3e}")
    rtol = 1e-5 + logit_magnitude_rtol(q.reshape(-1, 128).astype(np.float64),
                                       K2.reshape(-1, 128).astype(np.float64), 128 ** -0.5)
    check_importance(out["imp"], imp_o, 32, "f32", "shifted", rtol=rtol)
    check_importance(out["imp"], base["imp"].astype(np.float64), 32, "bf16", "shift vs base")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_late_large_logit_takes_the_slow_path(torch, cb, orc, dtype):
    """A position whose logit exceeds the chunk's first positions by far more
    than 100 (log2 units) pushes a row sum past the 2^100 guard, so its tile
    is redone on the online-max path and the row maxima differ between lanes:
    the rescaling merge must then give the same importance as the plain
    definition.  Two such positions, in different chunks; every other
    position keeps weights far below FLT_MIN."""
    w = W.custom(layers=1, q_heads=4, kv_heads=2, head_dim=128, q_len=16, seq_len=3000,
                 dtype=dtype)
    say(f"case late large logit ({dtype})")
    q, K, V = gen(w)
    f32 = (lambda a: W.bf16_bits_to_f32(a)) if dtype == "bf16" else (lambda a: a)
    back = (lambda a: W.round_to_bf16_bits(a)) if dtype == "bf16" else (lambda a: a.astype(np.float32))
    rng = np.random.default_rng(17)
    base = rng.standard_normal(128).astype(np.float32)
    qf = base + 0.3 * rng.standard_normal(f32(q).shape).astype(np.float32)
    Kf = f32(K).copy()
    Kf[..., 700, :] = 8.0 * base      # chunk 0, well past its first 16 positions
    Kf[..., 1500, :] = 7.5 * base     # a later chunk
    q, K = back(qf), back(Kf)
    out = run_gpu(torch, cb, w, q, K, V, 0.25)
    assert np.all(np.isfinite(out["imp"]))
    for row in out["idx"].reshape(-1, out["keep"]):
        assert 700 in row and 1500 in row
    check_all_units(orc, w, q, K, V, out, what=f"late large logit {dtype}")


def test_deterministic_across_runs(torch, cb, orc):
    w = W.custom(layers=3, q_heads=8, kv_heads=2, head_dim=128, q_len=32, seq_len=5000,
                 kdist="chanscale")
    say("case determinism")
    q, K, V = gen(w)
    a = run_gpu(torch, cb, w, q, K, V, 0.25)
    b = run_gpu(torch, cb, w, q, K, V, 0.25)
    c = run_gpu(torch, cb, w, q, K, V, 0.25, fused=False)
    for key in ("imp", "lse", "idx", "k_out", "v_out"):
        assert a[key].tobytes() == b[key].tobytes(), key
        assert a[key].tobytes() == c[key].tobytes(), f"{key}: cb_pipeline vs separate calls"


# --------------------------------------------------------------------------- full size


def test_qwen3_8b_full_size(torch, cb, orc):
    """Qwen3-8B attention shape, T = 8192, m = 64, keep 0.25: the benchmark's
    workload and launch configuration.  Fused and staged calls give bitwise-
    identical outputs; importance and row_lse match the oracle on all 288
    units."""
    w = W.get("qwen3-8b-8k-bf16")
    say("case qwen3-8b-8k-bf16 (full size)")
    q, K, V = gen(w)
    out = run_gpu(torch, cb, w, q, K, V, 0.25)
    staged = run_gpu(torch, cb, w, q, K, V, 0.25, fused=False)
    assert out["keep"] == 2048
    for key in ("imp", "lse", "idx", "k_out", "v_out"):
        assert out[key].tobytes() == staged[key].tobytes(), f"{key}: fused vs staged"
    del staged
    check_units(orc, w, q, K, V, [out], layer_units(w, range(w.layers)), "qwen3-8b")


@pytest.mark.parametrize("name,layers,ratios,nsample", [
    ("fanin-3x16k-bf16", 2, (0.25,), 3),
    ("longctx-32k-bf16", 2, (0.10, 0.25, 0.50), 2),
    ("hybrid-64k-bf16", 2, (0.25,), 2),
])
def test_long_workloads_layer_subset(torch, cb, orc, name, layers, ratios, nsample):
    """Full per-unit shapes (T, heads, m) on the first `layers` layers (a
    smaller launch: other item sizes and work-list lags)."""
    w = W.get(name).with_layers(layers)
    say(f"case {name} first {layers} layers")
    q, K, V = gen(w)
    outs = []
    for ratio in ratios:
        out = run_gpu(torch, cb, w, q, K, V, ratio)
        assert out["keep"] == orc.keep_count(w.seq_len, ratio)
        outs.append(out)
    check_units(orc, w, q, K, V, outs, W.sample_units(w, nsample), name)


@pytest.mark.parametrize("name,ratios", [
    ("fanin-3x16k-bf16", (0.25,)),
    ("longctx-32k-bf16", (0.10, 0.25, 0.50)),
    ("hybrid-64k-bf16", (0.25,)),
])
def test_long_workloads_full_size(torch, cb, orc, name, ratios):
    """Every layer at full size, in the launch configuration the library
    chooses for the whole workload (item size, row groups, resident
    workgroups).  Importance and row_lse against the oracle on every unit of
    the hybrid workload and on every sender and KV head of the first, middle
    and last layer of the others, at every keep ratio; selection and
    compaction exact on all units."""
    w = W.get(name)
    say(f"case {name} full size ({w.units} units)")
    q, K, V = gen(w)
    outs = []
    for ratio in ratios:
        out = run_gpu(torch, cb, w, q, K, V, ratio)
        assert out["keep"] == orc.keep_count(w.seq_len, ratio)
        outs.append(out)
    if w.units <= 64:
        units = layer_units(w, range(w.layers))
    else:
        units = layer_units(w, (0, w.layers // 2, w.layers - 1))
    check_units(orc, w, q, K, V, outs, units, name)


@pytest.mark.parametrize("T", [16387, 16388, 40000, 65536, 65537, 100000])
def test_select_long_rows_with_many_units(torch, cb, orc, T):
    """cb_select with at least as many units as compute units: rows of up to
    65536 scores held in registers (several workgroups per compute unit),
    and longer rows in 512-thread workgroups that re-read the row from L2,
    with scalar loads (T % 4 != 0) and 16-byte loads (T % 4 == 0).
    Bit-exact against the oracle's comparison sort."""
    units = max(300, torch.cuda.get_device_properties(0).multi_processor_count)
    rng = np.random.default_rng(T + 1)
    imp = (0.03125 * (1.0 + 0.01 * rng.standard_normal((units, T)))).astype(np.float32)
    imp[1::3, ::5] = np.float32(0.03125)          # exact ties at a power of two
    imp[2::3, : T // 2] = imp[2::3, T // 2: T // 2 * 2]
    imp[0, 0], imp[0, 1], imp[3, T - 1] = np.float32(-0.0), np.float32(0.0), np.float32(np.nan)
    say(f"case select T={T} units={units}")
    dimp = to_dev(torch, imp)
    for ratio in (0.1, 0.25, 0.5):
        keep = orc.keep_count(T, ratio)
        idx = torch.empty((units, keep), dtype=torch.int32, device="cuda")
        assert cb.cb_select(dimp, units, T, ratio, idx) == keep
        torch.cuda.synchronize()
        assert np.array_equal(to_host(torch, idx), orc.select(imp, keep)), (T, ratio)


def _hand_made_scores(T, units, seed):
    """Near-uniform fp32 scores straddling a power of two, with exact ties,
    duplicated halves, -0/+0, NaNs and a row with a NaN at every fifth
    position."""
    rng = np.random.default_rng(seed)
    imp = (0.03125 * (1.0 + 0.01 * rng.standard_normal((units, T)))).astype(np.float32)
    imp[1 % units, ::3] = np.float32(0.03125)
    imp[2 % units, : T // 2] = imp[2 % units, T // 2: T // 2 * 2]
    imp[3 % units, ::5] = np.float32(np.nan)
    imp[0, 0], imp[0, 1] = np.float32(-0.0), np.float32(0.0)
    imp[units - 1, T - 1] = np.float32(np.nan)
    return imp


@pytest.mark.parametrize("units,T", [(64, 65536), (4, 100003), (100, 40000), (128, 16385),
                                     (2, 65537), (1, 1000003)])
def test_select_split_rows(torch, cb, orc, units, T):
    """cb_select_ws with rows split over several workgroups (16384 to 65536
    positions per part, 2 to 62 parts, read back four parts at a time; the
    last part ragged down to one position, scalar loads when T % 4 != 0):
    bit-exact against the oracle's comparison sort and equal to cb_select,
    keep from 1 to T, status CB_OK."""
    need = cb.cb_select_workspace_bytes(units, T)
    assert need > 0
    imp = _hand_made_scores(T, units, seed=T + units)
    say(f"case split select units={units} T={T}")
    dimp = to_dev(torch, imp)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    for ratio in (1e-9, 0.1, 0.25, 0.5, 1.0):
        keep = orc.keep_count(T, ratio)
        idx = torch.full((units, keep), -7, dtype=torch.int32, device="cuda")
        assert cb.cb_select_ws(dimp, units, T, ratio, idx, ws) == keep
        assert cb.cb_select_status(units, T, ws) == 0
        got = to_host(torch, idx)
        assert np.array_equal(got, orc.select(imp, keep)), (units, T, ratio)
        ref = torch.empty_like(idx)
        cb.cb_select(dimp, units, T, ratio, ref)
        assert torch.equal(idx, ref)


def test_split_select_timeout_is_reported(torch, cb, orc):
    """With the wait limit at 0, the waits between the parts of a split row
    give up: every kernel exits, cb_select_status reports CB_ERR_TIMEOUT and
    every index is -1 or a valid position, including slots that no part's
    ranking reaches once the parts disagree.  Restoring the limit gives an
    exact selection on the same workspace."""
    units, T = 64, 65536
    imp = _hand_made_scores(T, units, seed=5)
    say("case split select timeout")
    dimp = to_dev(torch, imp)
    ws = torch.empty(cb.cb_select_workspace_bytes(units, T), dtype=torch.uint8, device="cuda")
    keep = orc.keep_count(T, 0.25)
    # an out-of-range sentinel in every slot: a slot that no part writes
    # after the waits give up would keep it and fail the range check
    idx = torch.full((units, keep), T + 7, dtype=torch.int32, device="cuda")
    prev = cb.cb_set_wait_limit(0)
    try:
        cb.cb_select_ws(dimp, units, T, 0.25, idx, ws)
        assert cb.cb_select_status(units, T, ws) == -8
        got = to_host(torch, idx)
        assert ((got == -1) | ((got >= 0) & (got < T))).all()
    finally:
        cb.cb_set_wait_limit(prev)
    cb.cb_select_ws(dimp, units, T, 0.25, idx, ws)
    assert cb.cb_select_status(units, T, ws) == 0
    assert np.array_equal(to_host(torch, idx), orc.select(imp, keep))


def test_wait_timeout_is_reported(torch, cb, orc):
    """With the wait limit at 0 from the host, every dependency wait of the
    score kernel gives up at once: every kernel still exits, cb_score_status
    reports CB_ERR_TIMEOUT, importance is NaN, cb_pipeline's selection is -1
    throughout and the compacted rows are zero.  Restoring the limit gives a
    normal run on the same workspace."""
    w = W.custom(layers=2, q_heads=8, kv_heads=2, head_dim=128, q_len=16, seq_len=3000)
    say("case wait timeout")
    q, K, V = gen(w)
    lay = cb.layout_of(w)
    buf = cb.Buffers(lay, 0.25)
    qd, kd, vd = to_dev(torch, q), to_dev(torch, K), to_dev(torch, V)
    prev = cb.cb_set_wait_limit(0)
    try:
        buf.k_out.fill_(1)
        cb.run_pipeline(qd, kd, vd, buf)
        assert cb.cb_score_status(lay, buf.ws) == -8
        assert torch.isnan(buf.importance).all().item()
        assert (buf.idx == -1).all().item()
        assert (buf.k_out.view(torch.int16) == 0).all().item()
        cb.cb_score(qd, kd, lay, buf.importance, buf.row_lse, buf.ws)
        assert cb.cb_score_status(lay, buf.ws) == -8
        assert torch.isnan(buf.row_lse).all().item()
    finally:
        cb.cb_set_wait_limit(prev)
    cb.run_pipeline(qd, kd, vd, buf)
    assert cb.cb_score_status(lay, buf.ws) == 0
    out = dict(imp=to_host(torch, buf.importance), lse=to_host(torch, buf.row_lse),
               idx=to_host(torch, buf.idx), k_out=to_host(torch, buf.k_out),
               v_out=to_host(torch, buf.v_out), keep=buf.keep)
    check_all_units(orc, w, q, K, V, out, what="after timeout")
