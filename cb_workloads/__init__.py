"""Seeded synthetic workloads shaped like the paper's scoring workloads.

This module holds input generation only: shapes, seeds and value
distributions.  It contains none of the method's arithmetic, and it is the
one module that both the oracle-side tests and the GPU path use.

Every array is produced per unit (sender s, layer l, KV head g) from its own
``numpy.random.SeedSequence([ROOT_SEED, cfg_id, s + 1, l, g])``, spawned into
three PCG64 streams (K, V, unit structure), so any single unit can be
regenerated alone.  The receiver query uses ``SeedSequence([ROOT_SEED,
cfg_id, 0])`` and sender-level structure ``SeedSequence([ROOT_SEED, cfg_id,
s + 1])``.  Values are drawn in fp32 and rounded once, to nearest-even, to
the workload dtype; the rounded bytes are the canonical input for every
consumer.  bf16 arrays are returned as ``uint16`` bit patterns.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import math
import os
from typing import Iterable, Optional, Sequence

import numpy as np

ROOT_SEED = 260932046


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    layers: int
    q_heads: int
    kv_heads: int
    head_dim: int
    seq_len: int
    q_len: int
    senders: int
    dtype: str  # "f32" or "bf16"
    keep_ratios: tuple
    kdist: str  # K value recipe, see gen_unit_kv

    @property
    def group(self) -> int:
        return self.q_heads // self.kv_heads

    @property
    def rows(self) -> int:
        return self.group * self.q_len

    @property
    def units(self) -> int:
        return self.senders * self.layers * self.kv_heads

    @property
    def esize(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def d_model(self) -> int:
        """Width of one continuous row (the model's hidden size): q_heads *
        head_dim, 4096 at the Qwen3-8B shape."""
        return self.q_heads * self.head_dim

    def kv_bytes_per_position(self) -> int:
        """K and V bytes one sender position occupies over all layers/heads."""
        return 2 * self.layers * self.kv_heads * self.head_dim * self.esize

    def with_layers(self, layers: int) -> "Workload":
        """Same per-unit shapes and seeds restricted to the first ``layers``
        layers (units of the restricted workload are bit-identical to the
        corresponding units of the full one)."""
        return dataclasses.replace(self, layers=layers)


WORKLOADS = {
    w.name: w
    for w in [
        # 1 layer, 2 KV heads, 4 query heads, D=64, T=512, m=16, fp32, N(0,1).
        Workload("tiny-fp32", 1, 1, 4, 2, 64, 512, 16, 1, "f32", (0.25,), "normal"),
        # Qwen3-8B attention shape: 36 layers, 32/8 heads, D=128, T=8192, m=64.
        Workload("qwen3-8b-8k-bf16", 2, 36, 32, 8, 128, 8192, 64, 1, "bf16", (0.25,),
                 "chanscale"),
        # Fan-in: 3 senders of 16384 positions, one receiver query of 128 tokens.
        Workload("fanin-3x16k-bf16", 3, 36, 32, 8, 128, 16384, 128, 3, "bf16", (0.25,),
                 "chanscale"),
        # Long context: 48 layers, 40/8 heads, T=32768, peaked attention.
        Workload("longctx-32k-bf16", 4, 48, 40, 8, 128, 32768, 64, 1, "bf16",
                 (0.10, 0.25, 0.50), "peaked"),
        # Hybrid: 8 attention layers, T=65536, m=32, heavy-tailed K with outliers.
        Workload("hybrid-64k-bf16", 5, 8, 32, 8, 128, 65536, 32, 1, "bf16", (0.25,),
                 "student_t_outliers"),
    ]
}
BY_ID = {w.cfg_id: w for w in WORKLOADS.values()}


def get(name_or_id) -> Workload:
    if isinstance(name_or_id, int):
        return BY_ID[name_or_id]
    return WORKLOADS[name_or_id]


def custom(name="custom", *, layers, q_heads, kv_heads, head_dim, seq_len, q_len,
           senders=1, dtype="bf16", keep_ratios=(0.25,), kdist="normal", cfg_id=99):
    return Workload(name, cfg_id, layers, q_heads, kv_heads, head_dim, seq_len, q_len,
                    senders, dtype, tuple(keep_ratios), kdist)


# ---------------------------------------------------------------------------
# rounding


def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest, ties to even (finite
    inputs).  Uses torch's CPU conversion, which implements exactly that rule
    and is far faster than a numpy formulation; a test checks the two agree."""
    import torch

    x = np.ascontiguousarray(x, dtype=np.float32)
    t = torch.from_numpy(x).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def _finish(x: np.ndarray, dtype: str) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    return x if dtype == "f32" else round_to_bf16_bits(x)


# ---------------------------------------------------------------------------
# generators


def _streams(w: Workload, s: int, l: int, g: int):
    ss = np.random.SeedSequence([ROOT_SEED, w.cfg_id, s + 1, l, g])
    return [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(3)]


def _sender_stream(w: Workload, s: int):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([ROOT_SEED, w.cfg_id, s + 1])))


def shifted_positions(w: Workload, s: int) -> np.ndarray:
    """Positions of sender s that carry the 'peaked' K shift: floor(0.02 T)
    positions drawn without replacement, shared by all layers and heads."""
    n = int(math.floor(0.02 * w.seq_len))
    rng = _sender_stream(w, s)
    return np.sort(rng.choice(w.seq_len, size=n, replace=False))


def gen_q(w: Workload) -> np.ndarray:
    """Receiver query projections [L][Hq][m][D], N(0,1)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([ROOT_SEED, w.cfg_id, 0])))
    x = rng.standard_normal((w.layers, w.q_heads, w.q_len, w.head_dim), dtype=np.float32)
    return _finish(x, w.dtype)


def gen_unit_kv(w: Workload, s: int, l: int, g: int, want_v: bool = True):
    """K and V slabs [T][D] of one unit.

    Recipes (``kdist``):
      normal            K, V ~ N(0,1)
      chanscale         K = z*c/sqrt(D), z ~ N(0,1), c ~ U(0.5, 2) per channel
                        (one draw of c for K and one for V per unit)
      peaked            K, V ~ N(0,1); the sender's shifted positions get
                        K += 3*sqrt(D)*u with a random unit vector u per unit
      student_t_outliers K ~ Student-t(3) with 4 channels (without
                        replacement, per unit) scaled x20; V ~ N(0,1)
    """
    rk, rv, rs = _streams(w, s, l, g)
    T, D = w.seq_len, w.head_dim
    if w.kdist == "normal":
        k = rk.standard_normal((T, D), dtype=np.float32)
        v = rv.standard_normal((T, D), dtype=np.float32) if want_v else None
    elif w.kdist == "chanscale":
        ck = rs.uniform(0.5, 2.0, size=D).astype(np.float32)
        cv = rs.uniform(0.5, 2.0, size=D).astype(np.float32)
        inv = np.float32(1.0 / math.sqrt(D))
        k = rk.standard_normal((T, D), dtype=np.float32) * (ck * inv)
        v = rv.standard_normal((T, D), dtype=np.float32) * (cv * inv) if want_v else None
    elif w.kdist == "peaked":
        k = rk.standard_normal((T, D), dtype=np.float32)
        u = rs.standard_normal(D)
        u = (u / np.linalg.norm(u) * (3.0 * math.sqrt(D))).astype(np.float32)
        k[shifted_positions(w, s)] += u
        v = rv.standard_normal((T, D), dtype=np.float32) if want_v else None
    elif w.kdist == "student_t_outliers":
        k = rk.standard_t(3, size=(T, D)).astype(np.float32)
        chans = rs.choice(D, size=4, replace=False)
        k[:, chans] *= np.float32(20.0)
        v = rv.standard_normal((T, D), dtype=np.float32) if want_v else None
    else:
        raise ValueError(f"unknown kdist {w.kdist}")
    return _finish(k, w.dtype), (_finish(v, w.dtype) if want_v else None)


def np_dtype(w: Workload):
    return np.float32 if w.dtype == "f32" else np.uint16


def gen_kv(w: Workload, threads: Optional[int] = None, want_v: bool = True,
           progress=None):
    """Full K, V [S][L][Hkv][T][D], generated unit by unit on a thread pool."""
    shape = (w.senders, w.layers, w.kv_heads, w.seq_len, w.head_dim)
    K = np.empty(shape, dtype=np_dtype(w))
    V = np.empty(shape, dtype=np_dtype(w)) if want_v else None
    units = [(s, l, g) for s in range(w.senders) for l in range(w.layers)
             for g in range(w.kv_heads)]

    def job(u):
        s, l, g = u
        k, v = gen_unit_kv(w, s, l, g, want_v)
        K[s, l, g] = k
        if want_v:
            V[s, l, g] = v
        return u

    n = threads or min(16, os.cpu_count() or 1)
    with _cf.ThreadPoolExecutor(n) as ex:
        for i, _ in enumerate(ex.map(job, units)):
            if progress and (i + 1) % max(1, len(units) // 4) == 0:
                progress(f"generated {i + 1}/{len(units)} units of {w.name}")
    return K, V


ROWS_TAG = 1_000_003   # seed-sequence word that separates the row streams


def gen_rows(w: Workload, senders: Optional[Sequence[int]] = None, T: Optional[int] = None):
    """Continuous rows [S][T][d_model], N(0,1), one PCG64 stream per sender
    from SeedSequence([ROOT_SEED, cfg_id, s + 1, ROWS_TAG])."""
    senders = range(w.senders) if senders is None else senders
    T = w.seq_len if T is None else T
    out = []
    for s in senders:
        rng = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence([ROOT_SEED, w.cfg_id, s + 1, ROWS_TAG])))
        out.append(_finish(rng.standard_normal((T, w.d_model), dtype=np.float32), w.dtype))
    return np.stack(out)


def unit_q(w: Workload, q: np.ndarray, l: int, g: int) -> np.ndarray:
    """The G query heads that read KV head g in layer l, as q[1][G][m][D]."""
    G = w.group
    return np.ascontiguousarray(q[l:l + 1, g * G:(g + 1) * G])


def sample_units(w: Workload, count: int, seed: int = 7) -> list:
    """A seeded sample of units (s, l, g) that always includes the first and
    last unit."""
    all_units = [(s, l, g) for s in range(w.senders) for l in range(w.layers)
                 for g in range(w.kv_heads)]
    if count >= len(all_units):
        return all_units
    rng = np.random.default_rng(seed)
    pick = set(rng.choice(len(all_units), size=max(0, count - 2), replace=False).tolist())
    pick |= {0, len(all_units) - 1}
    return [all_units[i] for i in sorted(pick)]
