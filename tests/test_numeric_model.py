"""A CPU model of the device's rounding steps, checked against the fp64 oracle (no GPU).

The kernels round operands to fp16 and accumulate in fp32. This file replays those rounding steps
in NumPy (float16 casts for each fp16 rounding, float64 sums standing in for fp32 accumulation,
whose own error is of order 1e-7) and shows two things at gradient-sized inputs:

* folding the backward's scale into dY in fp16 without scaling (one rounding of dY * s16) leaves
  the tolerance gate at |dY| ~ 1e-3 and is far outside it at 1e-5, because the products fall
  into fp16's subnormal range;
* the kernels' per-row power-of-two scaling (largest magnitude brought into [16, 32) before any
  fp16 rounding, undone exactly in fp32) keeps the error at the level of |dY| ~ 1 for every
  magnitude, on both the small-M form (exponents per reduction slice for the sparse product, the
  adapter intermediate accumulated in fp32 and stored in fp16 with its row's exponent) and the
  large-M form (exponents per row throughout).

The model is test infrastructure: it neither calls nor imitates any code of the library, only
the rounding sequence the library's header documents.
"""
import numpy as np
import pytest

from oracle import slim_oracle as O
from paper_2608_24070_amd import synth

GATE = 2e-3
ACT_EXP = 4   # scaled rows have their largest magnitude in [2^4, 2^5)


def f16(x):
    with np.errstate(over="ignore", under="ignore"):
        return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


def bf16(x):
    return synth.bf16_to_f64(synth.bf16_bits(np.asarray(x, dtype=np.float32)))


def row_exp(a, axis=-1):
    """Exponent e per row so that max |a * 2^e| lies in [16, 32) (0 for zero rows)."""
    mx = np.max(np.abs(a), axis=axis, keepdims=True)
    with np.errstate(divide="ignore"):
        e = ACT_EXP - np.floor(np.log2(np.where(mx > 0, mx, 1.0)))
    return np.where(mx > 0, e, 0.0)


def _problem(n, k, r, m, scale, seed):
    W = synth.weights(n, k, seed=seed, name="nm/W")
    _, dY = synth.activations(m, n, seed=seed, name="nm/dY")
    dY = bf16(dY * scale)                       # a bf16 gradient of the given size
    _, _, L, R = synth.adapter(k, n, r, seed=seed, name="nm/")
    pb = O.pack_bwd(O.pack(W), n, k)
    Wrc = O.unpack_bwd(pb["codesT"], pb["metaT"], pb["scalesT"], n, k)       # q * s16, exact
    s = pb["scalesT"].view(np.float16).astype(np.float64)                    # [K/128, N]
    S = np.repeat(s, 128, axis=0).T                                          # s16[n, k / 128], [N, K]
    Q = np.divide(Wrc, S, out=np.zeros_like(Wrc), where=S > 0)              # exact integer codes
    ref = O.bwd_dx(dY, pb, L, R, n, k)
    return dY, Q, s, L, R, ref


def model_bwd_unscaled(dY, Q, s, L, R):
    """The earlier fold: B' = fp16(dY * s16) per (row n, k-group), U = dY R^T rounded to fp16."""
    n, k = Q.shape
    dX = np.zeros((dY.shape[0], k))
    for g in range(k // 128):
        B = f16(f16(dY) * s[g][None, :])                      # fp16 copy of dY, then the fp16 product
        dX[:, 128 * g:128 * g + 128] = B @ Q[:, 128 * g:128 * g + 128]
    U = f16(f16(dY) @ R.T)
    return dX + U @ L.T


def model_bwd_small_m(dY, Q, s, L, R, slice_len=512):
    """M <= 32: exponents per (row, reduction slice) on dY * s16 formed in fp32; U accumulated in
    fp32 and stored in fp16 scaled by the exponent of the row's largest |dY|."""
    n, k = Q.shape
    dX = np.zeros((dY.shape[0], k))
    for g in range(k // 128):
        P = dY * s[g][None, :]                                 # exact in fp32 (8 x 11 bits)
        for a in range(0, n, slice_len):
            Ps = P[:, a:a + slice_len]
            e = row_exp(Ps)
            B = f16(Ps * 2.0 ** e) * 2.0 ** -e
            dX[:, 128 * g:128 * g + 128] += B @ Q[a:a + slice_len, 128 * g:128 * g + 128]
    U = dY @ R.T                                               # fp32 accumulation
    e = row_exp(dY)
    return dX + (f16(U * 2.0 ** e) @ L.T) * 2.0 ** -e


def model_bwd_large_m(dY, Q, s, L, R):
    """M > 32: one exponent per row of dY; B' = fp16(dY' * s16); U' = fp16(dY' R^T); unscaled at the end."""
    n, k = Q.shape
    e = row_exp(dY)
    Ds = f16(dY * 2.0 ** e)
    dX = np.zeros((dY.shape[0], k))
    for g in range(k // 128):
        B = f16(Ds * s[g][None, :])
        dX[:, 128 * g:128 * g + 128] = B @ Q[:, 128 * g:128 * g + 128]
    U = f16(Ds @ R.T)
    return (dX + U @ L.T) * 2.0 ** -e


@pytest.mark.parametrize("scale", [1.0, 1e-3, 1e-5, 1e-7])
def test_backward_models_at_gradient_magnitudes(scale):
    dY, Q, s, L, R, ref = _problem(2048, 256, 32, 8, scale, seed=0)
    for model in (model_bwd_small_m, model_bwd_large_m):
        ok, rf, ma = O.within_tolerance(model(dY, Q, s, L, R), ref)
        assert ok and rf < 5e-4, (model.__name__, scale, rf, ma)
    # the earlier unscaled fold: fine at |dY| ~ 1, out of the gate from 1e-3 on
    ok, rf, _ = O.within_tolerance(model_bwd_unscaled(dY, Q, s, L, R), ref)
    assert ok == (scale == 1.0), (scale, rf)


def model_fwd_large_m(X, p, L, R, n, k):
    """M > 32 forward: X' = fp16(X 2^e) per row, Wc in fp16, T' = fp16(X' L), Y = (X' Wc^T + T' R) 2^-e."""
    Wc = f16(O.unpack(p["codes"], p["meta"], p["scales"], n, k))
    e = row_exp(X)
    Xs = f16(X * 2.0 ** e)
    T = f16(Xs @ L)
    return (Xs @ Wc.T + T @ R) * 2.0 ** -e


def model_fwd_small_m(X, p, L, R, n, k, slice_len=512):
    """M <= 32 forward: exponents per (row, slice) of X; T = X L accumulated in fp32 from rounds of
    128 positions, stored in fp16 scaled by the exponent of the row's largest |X|."""
    Wc = f16(O.unpack(p["codes"], p["meta"], p["scales"], n, k))
    Y = np.zeros((X.shape[0], n))
    for a in range(0, k, slice_len):
        Xa = X[:, a:a + slice_len]
        e = row_exp(Xa)
        Y += (f16(Xa * 2.0 ** e) @ Wc[:, a:a + slice_len].T) * 2.0 ** -e
    T = np.zeros((X.shape[0], L.shape[1]))
    for a in range(0, k, 128):                                 # adapter rounds of 128 positions
        Xa = X[:, a:a + 128]
        e = row_exp(Xa)
        T += (f16(Xa * 2.0 ** e) @ L[a:a + 128]) * 2.0 ** -e
    e = row_exp(X)
    return Y + (f16(T * 2.0 ** e) @ R) * 2.0 ** -e


@pytest.mark.parametrize("scale", [1.0, 1e6, 1e-6])
def test_forward_models_beyond_fp16_range(scale):
    # bf16 activations of 1e6 overflow fp16 (65504) unless scaled; of 1e-6 they are fp16 subnormals
    n, k, r, m = 512, 1024, 32, 8
    W = synth.weights(n, k, seed=1, name="nmf/W")
    _, X = synth.activations(m, k, seed=1, name="nmf/X")
    X = bf16(X * scale)
    _, _, L, R = synth.adapter(k, n, r, seed=1, name="nmf/")
    p = O.pack(W)
    ref = O.linear(X, p, L, R, n, k)
    for model in (model_fwd_small_m, model_fwd_large_m):
        ok, rf, ma = O.within_tolerance(model(X, p, L, R, n, k), ref)
        assert ok and rf < 5e-4, (model.__name__, scale, rf, ma)
    # unscaled: fp16(X) overflows to inf at 1e6
    with np.errstate(over="ignore", invalid="ignore"):
        assert (scale != 1e6) or not np.all(np.isfinite(f16(X)))
