"""Plain float64 NumPy oracle for SLiM-Quant, the probabilistic mean-squared-error scale search of
the SLiM chapter (test infrastructure only: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it; the HIP path shares no code with it).

What it computes, and where the thesis defines it
-------------------------------------------------
SLiM-Quant picks one symmetric quantisation parameter alpha for a whole weight matrix by
minimising the expected squared error of quantising a weight drawn from the matrix's magnitude
distribution (SLiM chapter, section "SLiM-Quant quantization method"):

* eq. probabilistic_mse / error_summation: E(alpha) = E_quant(alpha) + E_clip(alpha), where
  E_quant integrates the rounding error over magnitudes below alpha (eq. quantization_error)
  and E_clip the clipping error (alpha - x)^2 above it (eq. clipping_error), both against the
  density f_abs of |w|.
* The density is not a standard one, so the integrals are taken numerically on a histogram of
  |w| (same section, and the SLiM setup for the bin count
  max(512, min(d_in d_out / 1000, 20000))).
* Alg. quantization: a coarse grid of ten candidates over (0, max|w|], then a fine grid of step
  eta_high around the coarse minimum; alpha* is the candidate of least error.

``histogram``, ``estimate_error`` and ``search`` follow those steps; ``pack_alpha`` is the
forward pack (``slim_oracle.pack``'s format) with every group's scale taken from alpha*.

Readings where the thesis is silent or garbled
----------------------------------------------
* Q1  eq. quantization_error prints the reconstruction as alpha round(x / alpha) 2^(1-q), which
      has the garbling of eq. symmetric_quantization. Reading: the quantiser of the path, a
      uniform grid of step delta = alpha / (2^(q-1) - 1) (alpha / 7 at q = 4) with codes in
      [-(2^(q-1) - 1), 2^(q-1) - 1]; a magnitude x <= alpha reconstructs as delta rint(x / delta)
      (ties to even), one above alpha as alpha.
* Q2  Histogram: ``bins`` equal bins over [0, amax], amax = max|w|; |w| falls in bin
      b = floor(|w| bins / amax) computed in float64 (|w| bins is exact there), clamped to
      bins - 1 (the maximum itself). Each bin stands for its count at its centre
      (b + 1/2) amax / bins, i.e. the midpoint rule with f_abs = counts / total.
* Q3  Bin count: max(512, min(floor(N K / 1000), 20000)).
* Q4  Coarse grid: the Alg. writes range(0, M, eta_low), the text ten uniform samples in
      (0, max(W)). alpha = 0 leaves the quantiser undefined, so the ten candidates are
      i eta_low, i = 1 .. 10, eta_low = amax / 10: AbsMax (alpha = amax) is one of them.
* Q5  Fine grid: eta_high = eta_low / 10, candidates (alpha_low - eta_low) + j eta_high for
      j = 0 .. 19 (the Alg.'s range(alpha_low - eta_low, alpha_low + eta_low, eta_high)), the
      positive ones only.
* Q6  alpha* is the argmin over every candidate evaluated, coarse and fine (the Alg. keeps both
      in one dictionary); on equal error the first evaluated wins.
* Q7  All magnitudes zero (amax = 0): alpha* = 0 and no candidate is evaluated.
* Q8  As a pack option, the per-tensor alpha* sets every group's scale to
      s16 = fp16_RNE(fp32(alpha*) / 7.0f), the AbsMax formula with alpha* for the group maximum;
      codes are clamp(rint(w / s16), -7, 7) as in the AbsMax pack, so weights beyond alpha* clip
      to +-7. The mask is unchanged (magnitude top-2 of the fp32 weights).
"""
from __future__ import annotations

import numpy as np

from .slim_oracle import (CODE_OFFSET, GROUP, QMAX, OracleError, _encode, fp16_rne, mask_2of4)

COARSE = 10          # coarse candidates (Alg. quantization, first loop)
FINE = 20            # fine candidates: two coarse steps at a tenth of the step
MAX_CANDIDATES = COARSE + FINE


def bin_count(n: int, k: int) -> int:
    """Histogram size of the SLiM setup: max(512, min(floor(N K / 1000), 20000))."""
    return max(512, min((int(n) * int(k)) // 1000, 20000))


def qmax_of(bits: int) -> int:
    return (1 << (bits - 1)) - 1


def histogram(W, bins: int):
    """Counts of |w| in ``bins`` equal bins over [0, max|w|] (Q2). Returns (counts int64, amax float64)."""
    a = np.abs(np.asarray(W, dtype=np.float32)).astype(np.float64).ravel()
    if not np.all(np.isfinite(a)):
        raise OracleError("non-finite weight")
    if bins < 1:
        raise OracleError("need at least one bin")
    amax = float(a.max()) if a.size else 0.0
    if amax == 0.0:
        counts = np.zeros(bins, dtype=np.int64)
        counts[0] = a.size
        return counts, 0.0
    b = np.floor((a * float(bins)) / amax).astype(np.int64)
    b = np.minimum(b, bins - 1)
    return np.bincount(b, minlength=bins).astype(np.int64), amax


def bin_centres(amax: float, bins: int) -> np.ndarray:
    width = amax / bins
    return (np.arange(bins, dtype=np.float64) + 0.5) * width


def estimate_error(counts, amax: float, alpha: float, bits: int = 4) -> float:
    """EstimateError(alpha) of Alg. quantization: E_quant + E_clip on the histogram (Q1, Q2)."""
    counts = np.asarray(counts, dtype=np.float64)
    bins = counts.size
    c = bin_centres(amax, bins)
    delta = alpha / qmax_of(bits)
    below = c <= alpha
    # eq. quantization_error: rounding to the grid of step delta, magnitudes up to alpha
    e_quant = np.where(below, (delta * np.rint(c / delta) - c) ** 2, 0.0)
    # eq. clipping_error: magnitudes above alpha reconstruct as alpha
    e_clip = np.where(below, 0.0, (alpha - c) ** 2)
    total = counts.sum()
    return float((counts * e_quant).sum() / total + (counts * e_clip).sum() / total)


def candidates_coarse(amax: float) -> list:
    eta_low = amax / COARSE
    return [i * eta_low for i in range(1, COARSE + 1)]


def candidates_fine(amax: float, alpha_low: float) -> list:
    eta_low = amax / COARSE
    eta_high = eta_low / 10
    out = []
    for j in range(FINE):
        a = (alpha_low - eta_low) + j * eta_high
        if a > 0:
            out.append(a)
    return out


def search_hist(counts, amax: float, bits: int = 4) -> dict:
    """Alg. quantization on a histogram: coarse grid, fine grid around its minimum, argmin (Q4-Q7)."""
    if amax == 0.0:
        return {"alpha": 0.0, "error": 0.0, "table": []}
    table = []
    for a in candidates_coarse(amax):
        table.append((a, estimate_error(counts, amax, a, bits)))
    alpha_low = min(table, key=lambda t: t[1])[0]          # first of equal errors wins
    for a in candidates_fine(amax, alpha_low):
        table.append((a, estimate_error(counts, amax, a, bits)))
    best = min(range(len(table)), key=lambda i: (table[i][1], i))
    return {"alpha": table[best][0], "error": table[best][1], "table": table}


def search(W, bits: int = 4, bins: int | None = None) -> dict:
    """SLiM-Quant's alpha* of a weight matrix W [N, K] (or any array), with its histogram."""
    W = np.asarray(W, dtype=np.float32)
    if bins is None:
        n, k = W.shape
        bins = bin_count(n, k)
    counts, amax = histogram(W, bins)
    out = search_hist(counts, amax, bits)
    out.update({"counts": counts, "amax": amax, "bins": bins})
    return out


def pack_alpha(W, alpha: float) -> dict:
    """Forward pack with the per-tensor scale s16 = fp16_RNE(fp32(alpha) / 7) in every group (Q8)."""
    W = np.asarray(W, dtype=np.float32)
    n, k = W.shape
    if k % GROUP or n < 1:
        raise OracleError("need N >= 1 and K a multiple of 128")
    if not np.all(np.isfinite(W)):
        raise OracleError("non-finite weight")
    s = fp16_rne(np.float32(alpha) / np.float32(QMAX))
    if not np.isfinite(s):
        raise OracleError("scale overflows fp16")
    s16 = np.full((n, k // GROUP), s, dtype=np.float16)
    sd = float(s)
    with np.errstate(divide="ignore", invalid="ignore"):
        t = W.astype(np.float64) / sd if sd > 0 else np.zeros(W.shape)
    q = np.clip(np.rint(t), -QMAX, QMAX).astype(np.int8)
    m = mask_2of4(W)
    g = k // 4
    idx = np.sort(np.argsort(-m.reshape(n, g, 4).astype(np.int8), axis=2, kind="stable")[..., :2], axis=2)
    u = np.take_along_axis(q.reshape(n, g, 4), idx, axis=2).astype(np.int16) + CODE_OFFSET
    codes, meta = _encode(u, idx, n, k)
    return {"codes": codes, "meta": meta, "scales": s16.view(np.uint16).copy(), "mask": m}
