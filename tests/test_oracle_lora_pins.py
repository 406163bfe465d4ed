"""Pins of the SLiM-LoRA oracle (oracle/slim_lora.py) against things other than itself.

* A hand-worked calibration statistic (mean magnitude, then the shift by the smallest channel).
* Planted low rank: when W - W^C has rank <= r the adapters reproduce it exactly.
* Eckart-Young through another routine: the residual of the saliency-weighted fit equals the sum
  of the discarded eigenvalues of S S^T from numpy.linalg.eigvalsh, and the returned singular
  values are the largest ones.
* Constant saliency reduces to plain truncated SVD of W - W^C (computed here from eigh of the
  Gram matrix), which pins the inverse saliency diag(1/x); a dominant input channel gets its error
  fixed first, which pins the side diag(x) acts on.
* The symmetric split of the singular values between the factors, and the sign convention.
No GPU.
"""
import numpy as np
import pytest

from oracle import slim_lora as LR
from oracle import slim_oracle as O
from paper_2608_24070_amd import synth


def _layer(n, k, seed):
    W = synth.weights(n, k, seed=seed, name="lora/W")
    Wc = O.unpack(**{key: v for key, v in O.pack(W).items() if key in ("codes", "meta", "scales")}, n=n, k=k)
    return W, Wc


def _calib(b, k, seed, scale=1.0):
    rng = synth.stream(seed, "lora/X")
    return (rng.standard_normal((b, k)) * scale).astype(np.float32)


def test_channel_saliency_hand_example():
    X = np.array([[1.0, -2.0, 0.5], [3.0, 0.0, -0.5]])
    # mean |X| per channel: 2, 1, 0.5; shifted by the smallest (0.5)
    assert list(LR.channel_saliency(X)) == [2.5, 1.5, 1.0]
    with pytest.raises(O.OracleError):
        LR.channel_saliency(np.array([[1.0, 0.0], [2.0, 0.0]]))


def test_planted_low_rank_error_is_reproduced():
    n, k, r = 48, 64, 5
    rng = synth.stream(1, "lora/planted")
    W = rng.standard_normal((n, k)).astype(np.float32)
    E = rng.standard_normal((n, r)) @ rng.standard_normal((r, k)) * 0.1
    Wc = W.astype(np.float64) + E                       # W^C - W has rank r
    out = LR.lora(W, Wc, _calib(32, k, 1), r)
    assert np.allclose(Wc + (out["L"] @ out["R"]).T, W.astype(np.float64), rtol=0, atol=1e-12)
    assert out["L"].shape == (k, r) and out["R"].shape == (r, n)


@pytest.mark.parametrize("n,k,r", [(96, 128, 8), (64, 256, 16), (128, 128, 1), (256, 128, 20)])
def test_eckart_young_through_eigvalsh(n, k, r):
    W, Wc = _layer(n, k, 2)
    X = _calib(40, k, 2)
    out = LR.lora(W, Wc, X, r)
    x = LR.channel_saliency(X)
    S = x[:, None] * (Wc - W.astype(np.float64)).T
    lam = np.sort(np.linalg.eigvalsh(S @ S.T))[::-1]
    # the residual of the saliency-weighted objective (eq. lora_wanda_objective_function)
    resid = S + x[:, None] * (out["L"] @ out["R"])
    assert np.sum(resid ** 2) == pytest.approx(lam[r:].sum(), rel=1e-9)
    assert np.allclose(out["sigma"] ** 2, lam[:r], rtol=1e-10)
    # and the fit does reduce the weight error it models
    assert np.linalg.norm(W - (Wc + (out["L"] @ out["R"]).T)) < np.linalg.norm(W - Wc)


def test_constant_saliency_is_plain_truncated_svd():
    n, k, r = 80, 128, 6
    W, Wc = _layer(n, k, 3)
    X = np.full((4, k), -1.5)                           # x = 1.5 + 1.5 = 3 for every channel
    out = LR.lora(W, Wc, X, r)
    M = (W.astype(np.float64) - Wc).T                   # [K, N]
    lam, U = np.linalg.eigh(M @ M.T)
    Ur = U[:, np.argsort(lam)[::-1][:r]]
    assert np.allclose(out["L"] @ out["R"], Ur @ Ur.T @ M, rtol=0, atol=1e-12)


def test_dominant_channel_is_fixed_first():
    n, k = 64, 128
    W, Wc = _layer(n, k, 4)
    X = _calib(16, k, 4)
    X[:, 7] *= 1e4                                      # channel 7 far more salient than the rest
    out = LR.lora(W, Wc, X, 1)
    target = (W.astype(np.float64) - Wc)[:, 7]          # the error of input channel 7
    got = (out["L"] @ out["R"])[7]
    assert np.allclose(got, target, rtol=0, atol=1e-6 * np.abs(target).max())


def test_symmetric_split_and_sign_convention():
    n, k, r = 96, 128, 10
    W, Wc = _layer(n, k, 5)
    X = _calib(24, k, 5)
    out = LR.lora(W, Wc, X, r)
    x = out["x"]
    # diag(x) L has column norms sqrt(sigma), and so do the rows of R
    assert np.allclose(np.linalg.norm(x[:, None] * out["L"], axis=0), np.sqrt(out["sigma"]), rtol=1e-10)
    assert np.allclose(np.linalg.norm(out["R"], axis=1), np.sqrt(out["sigma"]), rtol=1e-10)
    # rows of R orthogonal; the largest entry of each row of R is positive
    G = out["R"] @ out["R"].T
    assert np.allclose(G, np.diag(out["sigma"]), rtol=0, atol=1e-12 * out["sigma"][0])
    for i in range(r):
        assert out["R"][i, np.argmax(np.abs(out["R"][i]))] > 0


def test_rank_zero_and_bad_rank():
    W, Wc = _layer(32, 128, 6)
    out = LR.lora(W, Wc, _calib(4, 128, 6), 0)
    assert out["L"].shape == (128, 0) and out["R"].shape == (0, 32)
    with pytest.raises(O.OracleError):
        LR.lora(W, Wc, _calib(4, 128, 6), 33)
