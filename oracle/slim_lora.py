"""Plain float64 NumPy oracle for SLiM-LoRA, the saliency-based low-rank adapters of the SLiM chapter
(test infrastructure only: only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` may use it; the HIP path shares no code with it).

What it computes, and where the thesis defines it
-------------------------------------------------
SLiM models quantisation and pruning as additive errors, W^C = W + E_Q + E_S, and fits adapters with
W ~ W^C + L R (section "SLiM-LoRA low-rank adapters"). Weighting the error by a saliency function
F(A) = diag(x) A that is additive and invertible (x: the mean magnitude of each input channel over
a calibration set) turns the fit into a truncated SVD (eq. lora_wanda_objective_function,
eq. lora_svd), as Alg. lora spells out:

    E_C = W^C - W;  x~ = per-channel mean over the calibration samples;  x = x~ + min(|x~|);
    S_C = diag(x) E_C;  L~, R~ = SVD_r(S_C);  L = diag(1/x) L~;  R = R~.

``channel_saliency`` is the calibration statistic, ``saliency_error`` S_C and ``lora`` the
adapters. The SVD itself is NumPy's (LAPACK), a library step.

Readings where the thesis is silent, ambiguous or inconsistent
--------------------------------------------------------------
* L1  Orientation: the thesis writes W as d_in x d_out with L [d_in x r] and R [r x d_out]. Here W is
      [N out x K in] and the layer is Y = X W^T + (X L) R, so the thesis's E_C is (W^C - W)^T [K x N]
      and diag(x) scales its rows, the input channels: S = diag(x) (W^C - W)^T.
* L2  Mean versus mean magnitude: the text defines x as the average absolute value of the inputs;
      the Alg. writes mean(X) and then shifts by min(|x~|). Reading: x~_k = mean_i |X[i, k]|, and
      x = x~ + min_k x~_k (the shift the text describes as adding a small multiple of the identity).
      A channel that is zero in every sample leaves x_k = 0 when it is also the minimum; the
      saliency is then not invertible and the call is rejected.
* L3  Sign: eq. lora_svd carries the minus that Alg. lora drops; with E_C = W^C - W the adapters
      must reproduce W - W^C, so L R = -diag(1/x) S_r, where S_r is the best rank-r approximation.
* L4  Split of the singular values between the factors (unstated): symmetric,
      L~ = U_r Sigma_r^(1/2), R~ = Sigma_r^(1/2) V_r^T, so both factors have the same scale (they are
      stored in fp16 by the layer).
* L5  Sign of each component (the SVD leaves it free): the largest-magnitude entry of each row of R
      is positive (the first such entry on equal magnitudes), and L's column follows.
* L6  Rank: r <= min(N, K); components of zero singular value contribute zero columns and rows.
"""
from __future__ import annotations

import numpy as np

from .slim_oracle import OracleError


def channel_saliency(X) -> np.ndarray:
    """x = x~ + min(x~), x~_k = mean_i |X[i, k]| over the calibration samples (L2). float64 [K]."""
    a = np.abs(np.asarray(X, dtype=np.float64))
    if a.ndim != 2 or a.shape[0] < 1:
        raise OracleError("calibration input must be [samples, K] with at least one sample")
    xt = a.mean(axis=0)
    x = xt + xt.min()
    if np.any(x == 0):
        raise OracleError("an input channel is zero in every calibration sample")
    return x


def saliency_error(W, Wc, x) -> np.ndarray:
    """S = diag(x) (W^C - W)^T, float64 [K, N] (L1)."""
    E = np.asarray(Wc, dtype=np.float64) - np.asarray(W, dtype=np.float32).astype(np.float64)
    return np.asarray(x, dtype=np.float64)[:, None] * E.T


def _fix_signs(L, R):
    for i in range(R.shape[0]):
        j = int(np.argmax(np.abs(R[i])))
        if R[i, j] < 0:
            R[i] *= -1
            L[:, i] *= -1
    return L, R


def lora(W, Wc, X, r: int) -> dict:
    """Alg. lora: L [K, r] and R [r, N] (float64) with W ~ W^C + (L R)^T, and the r singular values."""
    W = np.asarray(W, dtype=np.float32)
    n, k = W.shape
    if not 0 <= r <= min(n, k):
        raise OracleError("rank must lie in [0, min(N, K)]")
    x = channel_saliency(X)
    if x.size != k:
        raise OracleError("calibration input has the wrong width")
    S = saliency_error(W, Wc, x)
    U, s, Vt = np.linalg.svd(S, full_matrices=False)
    sr = s[:r]
    Lt = U[:, :r] * np.sqrt(sr)[None, :]
    Rt = np.sqrt(sr)[:, None] * Vt[:r]
    L = -(Lt / x[:, None])
    R = Rt.copy()
    L, R = _fix_signs(L, R)
    return {"L": L, "R": R, "sigma": sr, "x": x}
