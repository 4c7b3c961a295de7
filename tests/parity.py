"""Shared parity checks between the HIP path and the CPU oracle.

Tolerances (importance): |gpu - oracle| <= rtol*|oracle| + m*G*2^-126 with
rtol = 1e-5 for fp32 inputs and 2e-3 for bf16 inputs (fp32 accumulation).
The absolute floor is the most probability mass fp32 flush-to-zero can lose
for one position.  Selection: identical to the oracle's exact comparison sort
run on the GPU's own fp32 scores; against the oracle's fp64 scores, identical
outside the band of positions whose oracle score lies within the tolerance
of the keep-th score.  Compaction: bit-exact given the indices.
"""
from __future__ import annotations

import numpy as np

FLT_MIN = 2.0 ** -126


def rtol_for(dtype: str) -> float:
    return 1e-5 if dtype == "f32" else 2e-3


def logit_magnitude_rtol(q64: np.ndarray, k64: np.ndarray, scale: float) -> float:
    """Extra relative importance error fp32 accumulation can cause when
    logits are large: a logit error d moves a probability by a factor
    exp(d), and the rounding of an fp32 dot product grows with the sum of
    |q_d k_d|.  One fp32 rounding unit of the largest such sum (times the
    scale); on the shift-invariance case (logits -101 to +72) this is 2.2e-5
    against a measured maximum error of 1.4e-5 above the plain 1e-5."""
    mag = scale * np.einsum("rd,td->rt", np.abs(q64), np.abs(k64)).max()
    return 2.0 ** -24 * float(mag)


def check_importance(gpu: np.ndarray, orc: np.ndarray, mG: int, dtype: str, what="",
                     rtol=None):
    gpu = gpu.astype(np.float64)
    rtol = rtol_for(dtype) if rtol is None else rtol
    tol = rtol * np.abs(orc) + mG * FLT_MIN
    err = np.abs(gpu - orc)
    bad = err > tol
    if bad.any():
        i = np.unravel_index(np.argmax(err / tol), err.shape)
        raise AssertionError(
            f"{what}: {bad.sum()} of {bad.size} importance values outside tolerance; worst at "
            f"{i}: gpu={gpu[i]!r} oracle={orc[i]!r} err={err[i]:.3e} tol={tol[i]:.3e}")


def check_lse(gpu: np.ndarray, orc: np.ndarray, dtype: str, what=""):
    """Row log-normalisers: within rtol/2 * max(1, |lse|) (an lse error of
    delta moves every probability of the row by a factor exp(delta))."""
    tol = 0.5 * rtol_for(dtype) * np.maximum(1.0, np.abs(orc))
    err = np.abs(gpu.astype(np.float64) - orc)
    assert np.all(err <= tol), f"{what}: row_lse off by up to {err.max():.3e}"


def check_selection_band(gpu_idx: np.ndarray, orc_imp: np.ndarray, keep: int, mG: int,
                         dtype: str, orc_idx: np.ndarray, what=""):
    """gpu_idx/orc_idx: [keep] for one unit; orc_imp: [T] fp64."""
    assert len(gpu_idx) == keep and len(np.unique(gpu_idx)) == keep, what
    assert np.all(np.diff(gpu_idx) > 0), what
    theta = np.sort(orc_imp)[::-1][keep - 1]
    band = np.abs(orc_imp - theta) <= rtol_for(dtype) * abs(theta) + mG * FLT_MIN
    g = set(gpu_idx.tolist()) - set(np.nonzero(band)[0].tolist())
    o = set(orc_idx.tolist()) - set(np.nonzero(band)[0].tolist())
    assert g == o, f"{what}: selections differ outside the threshold band ({len(g ^ o)} positions)"


def check_invariants(imp: np.ndarray, idx: np.ndarray, keep: int, mG: int, dtype: str, what=""):
    """imp [units][T] fp32 from the GPU, idx [units][keep]."""
    sums = imp.astype(np.float64).sum(axis=-1)
    assert np.allclose(sums, mG, rtol=max(1e-4, 10 * rtol_for(dtype))), \
        f"{what}: importance mass {sums.min()}..{sums.max()} != {mG}"
    assert np.all(imp >= 0), what
    assert idx.shape[-1] == keep
    assert np.all(np.diff(idx, axis=-1) > 0), f"{what}: indices not strictly ascending"
    T = imp.shape[-1]
    assert idx.min() >= 0 and idx.max() < T
    # every kept score >= every dropped score, per unit
    for u in range(imp.shape[0]):
        kept = np.zeros(T, bool)
        kept[idx[u]] = True
        if keep < T:
            assert imp[u][kept].min() >= imp[u][~kept].max(), f"{what}: unit {u} ordering"
