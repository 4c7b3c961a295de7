"""The seeded input generators: shapes, determinism, rounding, layout bytes."""
import math

import numpy as np
import pytest

import cb_workloads as W
from oracle_pins import golden


def test_qwen3_8b_layout_matches_paper_bytes_per_position():
    # 144 KiB of bf16 K+V per sender position for Qwen 3 8B.
    w = W.get("qwen3-8b-8k-bf16")
    assert w.kv_bytes_per_position() == golden("kv_bytes_per_position_qwen3_8b_bf16") == 144 * 1024


def test_shapes_of_all_workloads():
    for w in W.WORKLOADS.values():
        assert w.q_heads % w.kv_heads == 0
        assert w.rows == w.group * w.q_len
    assert W.get(2).rows == 256 and W.get(3).rows == 512 and W.get(4).rows == 320
    assert W.get(5).rows == 128 and W.get(1).rows == 32


def test_bf16_rounding_is_nearest_even():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(200000).astype(np.float32)
    # exact halfway cases: low 16 bits = 0x8000, both parities of bit 16
    ties = (np.arange(1000, dtype=np.uint32) << 17 | 0x3F000000 | 0x8000).view(np.float32)
    ties_odd = ((np.arange(1000, dtype=np.uint32) << 17) | 0x3F010000 | 0x8000).view(np.float32)
    x = np.concatenate([x, ties, ties_odd, -ties])
    u = x.view(np.uint32)
    want = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)
    assert np.array_equal(W.round_to_bf16_bits(x), want)


def test_unit_regeneration_is_deterministic_and_independent():
    w = W.custom(layers=2, q_heads=4, kv_heads=2, head_dim=64, seq_len=100, q_len=3,
                 senders=2, kdist="chanscale")
    K, V = W.gen_kv(w, threads=3)
    for s in range(2):
        for l in range(2):
            for g in range(2):
                k, v = W.gen_unit_kv(w, s, l, g)
                assert np.array_equal(K[s, l, g], k) and np.array_equal(V[s, l, g], v)
    assert not np.array_equal(K[0, 0, 0], K[0, 0, 1])
    assert not np.array_equal(K[0, 0, 0], V[0, 0, 0])
    # restricting layers leaves the remaining units bit-identical
    K1, _ = W.gen_kv(w.with_layers(1), threads=2)
    assert np.array_equal(K1[:, 0], K[:, 0])


def test_recipes_have_stated_structure():
    base = dict(layers=1, q_heads=4, kv_heads=1, head_dim=128, seq_len=4000, q_len=2)
    # channel scales in [0.5, 2] / sqrt(D): per-channel std within that band
    k, _ = W.gen_unit_kv(W.custom(kdist="chanscale", **base), 0, 0, 0)
    std = W.bf16_bits_to_f32(k).std(axis=0) * math.sqrt(128)
    assert std.min() > 0.4 and std.max() < 2.2
    # peaked: floor(0.02 T) positions carry a 3*sqrt(D) shift along one direction
    w = W.custom(kdist="peaked", **base)
    k, _ = W.gen_unit_kv(w, 0, 0, 0)
    pos = W.shifted_positions(w, 0)
    assert len(pos) == 80
    kf = W.bf16_bits_to_f32(k)
    mean_shift = kf[pos].mean(axis=0) - kf.mean(axis=0)
    assert abs(np.linalg.norm(mean_shift) - 3 * math.sqrt(128)) < 3.0
    # student-t with 4 outlier channels x20
    k, _ = W.gen_unit_kv(W.custom(kdist="student_t_outliers", **base), 0, 0, 0)
    med = np.median(np.abs(W.bf16_bits_to_f32(k)), axis=0)
    assert (med > 10).sum() == 4


def test_sample_units_includes_ends():
    w = W.get("qwen3-8b-8k-bf16")
    units = W.sample_units(w, 6)
    assert len(units) == 6 and units[0] == (0, 0, 0) and units[-1] == (0, 35, 7)
