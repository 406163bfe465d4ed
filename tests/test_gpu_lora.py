"""SLiM-LoRA on the GPU (slim_lora) against the oracle in oracle/slim_lora.py.

What is unique is compared directly: the r largest singular values, and the adapter's product
L R = -diag(1/x) P_r S (P_r the projector on the top r singular vectors), which is unique when the
r-th and (r+1)-th singular values differ; individual components are compared up to sign where their
singular value is isolated. The outputs are fp32, so the product carries about 1e-7 of relative
rounding; the bound used is 1e-6 (relative Frobenius) with sampled spectra whose relative gap at r
is far above the float64 eigensolver's error."""
import numpy as np
import pytest
import torch

from oracle import slim_lora as LR
from oracle import slim_oracle as O
from paper_2608_24070_amd import slim, synth
from tests.gpu_common import dev, dev_bits, host

pytestmark = pytest.mark.gpu


def _case(n, k, b, seed, outliers=False, xdtype="bf16"):
    W = synth.weights(n, k, seed=seed, name="lora/W")
    xbits, X = synth.activations(b, k, seed=seed, name="lora/X", dtype=xdtype, outliers=outliers)
    tdt = torch.bfloat16 if xdtype == "bf16" else torch.float16
    return W, xbits, X, tdt


def _run(W, xbits, X, tdt, r):
    n, k = W.shape
    dW = dev(W)
    p = slim.pack(dW)
    got = slim.lora(dW, p, dev_bits(xbits, tdt), r)
    ref_pack = O.pack(W)
    Wc = O.unpack(ref_pack["codes"], ref_pack["meta"], ref_pack["scales"], n, k)
    ref = LR.lora(W, Wc, X, r)
    return got, ref, Wc


def _compare(got, ref, r, tag):
    Lg, Rg = host(got["L"]).astype(np.float64), host(got["R"]).astype(np.float64)
    sg = host(got["sigma"])
    assert np.allclose(sg, ref["sigma"], rtol=1e-10, atol=1e-13 * ref["sigma"][0]), tag
    Pg, Pr = Lg @ Rg, ref["L"] @ ref["R"]
    rel = np.linalg.norm(Pg - Pr) / np.linalg.norm(Pr)
    assert rel <= 1e-6, f"{tag}: product rel {rel:.3g}"
    assert np.abs(Pg - Pr).max() <= 1e-5 * np.abs(Pr).max(), tag
    # isolated components, up to sign
    s = ref["sigma"]
    for c in range(r):
        gap = min(s[c - 1] - s[c] if c > 0 else np.inf, s[c] - s[c + 1] if c + 1 < r else np.inf)
        if gap < 1e-3 * s[0]:
            continue
        sgn = 1.0 if np.dot(Rg[c], ref["R"][c]) >= 0 else -1.0
        assert np.allclose(sgn * Rg[c], ref["R"][c], rtol=0, atol=1e-5 * np.abs(ref["R"][c]).max()), (tag, c)
        assert np.allclose(sgn * Lg[:, c], ref["L"][:, c], rtol=0, atol=1e-5 * np.abs(ref["L"][:, c]).max()), (tag, c)
    return rel


@pytest.mark.parametrize("n,k,r,b,outliers", [
    (256, 128, 16, 64, False),      # K <= N: left Gram (d = 128)
    (128, 256, 16, 64, True),       # N < K: right Gram (d = 128)
    (512, 512, 48, 300, True),
    (400, 1024, 40, 128, False),    # d = 400: padded to 448 for the 32-wide Jacobi blocks
    (1024, 768, 96, 520, True)])
def test_lora_parity(n, k, r, b, outliers):
    print(f"lora n={n} k={k} r={r} b={b} outliers={outliers}", flush=True)
    W, xbits, X, tdt = _case(n, k, b, 1, outliers)
    got, ref, _ = _run(W, xbits, X, tdt, r)
    assert 1 <= got["sweeps"] <= 40
    _compare(got, ref, r, f"n={n} k={k} r={r}")


def test_lora_fp16_calibration_and_full_rank():
    # r = min(N, K): the adapters carry the whole error, W = W^C + (L R)^T up to fp32 rounding
    n, k = 128, 256
    W, xbits, X, tdt = _case(n, k, 48, 2, True, xdtype="fp16")
    got, ref, Wc = _run(W, xbits, X, tdt, n)
    rec = Wc + (host(got["L"]).astype(np.float64) @ host(got["R"]).astype(np.float64)).T
    err = W.astype(np.float64) - Wc
    assert np.linalg.norm(rec - W) <= 1e-6 * np.linalg.norm(err)


def test_lora_rank_zero_and_dead_channel():
    n, k = 64, 128
    W, xbits, X, tdt = _case(n, k, 16, 3)
    dW = dev(W)
    p = slim.pack(dW)
    out = slim.lora(dW, p, dev_bits(xbits, tdt), 0)
    assert out["L"].shape == (k, 0) and out["R"].shape == (0, n)
    # channel 5 zero in every sample, and channel 9 too: the smallest mean is 0, so x_5 = x_9 = 0
    xb = xbits.copy()
    xb[:, [5, 9]] = 0
    with pytest.raises(slim.SlimError) as e:
        slim.lora(dW, p, dev_bits(xb, tdt), 8)
    assert e.value.status == slim.SLIM_ERANGE


def test_lora_decode_layer_full_size():
    # the 4096 x 4096 decode layer at rank 384 with 2048 calibration rows: the singular values against
    # numpy.linalg.eigvalsh of S S^T, the projector property, and the residual identity
    n = k = 4096
    r = 384
    print(f"lora full size n={n} k={k} r={r}", flush=True)
    W, xbits, X, tdt = _case(n, k, 2048, 4, True)
    dW = dev(W)
    p = slim.pack(dW)
    got = slim.lora(dW, p, dev_bits(xbits, tdt), r)
    torch.cuda.synchronize()
    ref_pack = O.pack(W)
    Wc = O.unpack(ref_pack["codes"], ref_pack["meta"], ref_pack["scales"], n, k)
    x = LR.channel_saliency(X)
    S = LR.saliency_error(W, Wc, x)
    lam = np.sort(np.linalg.eigvalsh(S @ S.T))[::-1]
    sg = host(got["sigma"])
    assert np.allclose(sg ** 2, lam[:r], rtol=1e-9, atol=1e-12 * lam[0])
    Lg, Rg = host(got["L"]).astype(np.float64), host(got["R"]).astype(np.float64)
    # rows of R orthogonal with norms sqrt(sigma); diag(x) L columns likewise
    assert np.allclose(Rg @ Rg.T, np.diag(sg), rtol=0, atol=2e-6 * sg[0])
    XL = x[:, None] * Lg
    assert np.allclose(XL.T @ XL, np.diag(sg), rtol=0, atol=2e-6 * sg[0])
    # residual of the saliency-weighted fit = the discarded eigenvalues (Eckart-Young)
    resid = S + x[:, None] * (Lg @ Rg)
    assert np.sum(resid ** 2) == pytest.approx(lam[r:].sum(), rel=1e-5)
