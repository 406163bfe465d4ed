"""SLiM-Quant on the GPU (slim_quant_search, slim_pack_alpha) against the oracle in
oracle/slim_quant.py: bit-exact histograms, the same candidates, errors within float64 summation
order, the same alpha*, bit-exact packs, and the layer on such a pack within the tolerance gate."""
import numpy as np
import pytest
import torch

from oracle import slim_oracle as O
from oracle import slim_quant as Q
from paper_2608_24070_amd import slim, synth
from tests.gpu_common import assert_close, dev, dev_bits, host, host_pack

pytestmark = pytest.mark.gpu


def _weights(n, k, seed, outliers=0):
    W = synth.weights(n, k, seed=seed, name="quant/W")
    if outliers:
        rng = synth.stream(seed, "quant/outliers")
        idx = rng.choice(n * k, size=outliers, replace=False)
        W.reshape(-1)[idx] *= np.float32(12.0)
    return W


def _check_search(W, bits=4, bins=None):
    n, k = W.shape
    got = slim.quant_search(dev(W), bits=bits, bins=bins)
    ref = Q.search(W, bits=bits, bins=bins)
    assert got["bins"] == ref["bins"]
    assert got["amax"] == ref["amax"]
    assert np.array_equal(host(got["hist"]).view(np.uint32).astype(np.int64), ref["counts"])
    # the same candidates in the same order (same float64 operations), errors up to summation order
    ga = [a for a, _ in got["table"]]
    ra = [a for a, _ in ref["table"]]
    assert ga == ra
    ge = np.array([e for _, e in got["table"]])
    re_ = np.array([e for _, e in ref["table"]])
    assert np.allclose(ge, re_, rtol=1e-12, atol=0)
    # alpha*: the oracle's, unless two candidates' errors lie within summation noise of each other
    if got["alpha"] != ref["alpha"]:
        assert got["error"] <= re_.min() * (1 + 1e-12)
        assert abs(re_[ra.index(got["alpha"])] - re_.min()) <= 1e-12 * re_.min()
    assert got["error"] == pytest.approx(ref["error"], rel=1e-12)
    return got, ref


@pytest.mark.parametrize("n,k,bits,bins,outliers", [
    (64, 128, 4, None, 0), (256, 512, 4, 700, 0), (1024, 1024, 4, None, 40), (512, 384, 3, 2048, 5),
    (4096, 4096, 4, None, 0), (160, 256, 2, 20480, 0)])
def test_search_parity(n, k, bits, bins, outliers):
    print(f"quant search n={n} k={k} bits={bits} bins={bins} outliers={outliers}", flush=True)
    _check_search(_weights(n, k, 1, outliers), bits=bits, bins=bins)


def test_search_bins_at_edges():
    # magnitudes on and next to bin edges (including dyadic edges with a non-dyadic bin width)
    vals = [j / 8 for j in range(1, 9)]
    for kq in range(1, 600, 7):
        e = np.float32(kq / 600)
        vals += [np.nextafter(e, np.float32(0)), e, np.nextafter(e, np.float32(2))]
    W = np.zeros((16, 128), dtype=np.float32).reshape(-1)
    W[:len(vals)] = vals
    W[1::2] *= -1
    _check_search(W.reshape(16, 128), bins=600)


def test_search_full_size_70b():
    n, k = 28672, 8192
    print(f"quant search full size n={n} k={k}", flush=True)
    W = _weights(n, k, 2, outliers=1000)
    got, ref = _check_search(W)
    assert ref["bins"] == 20000


def test_search_degenerate_and_errors():
    z = np.zeros((16, 128), dtype=np.float32)
    got = slim.quant_search(dev(z))
    assert got["alpha"] == 0.0 and got["table"] == [] and int(host(got["hist"])[0]) == 16 * 128
    W = _weights(16, 128, 3)
    W[4, 9] = np.inf
    with pytest.raises(slim.SlimError) as e:
        slim.quant_search(dev(W))
    assert e.value.status == slim.SLIM_ENONFINITE
    with pytest.raises(slim.SlimError) as e:
        slim.quant_search(dev(_weights(16, 128, 3)), bins=20481)
    assert e.value.status == slim.SLIM_ESHAPE


@pytest.mark.parametrize("n,k,outliers", [(256, 512, 0), (1024, 1024, 40), (48, 384, 3)])
def test_pack_alpha_bit_exact(n, k, outliers):
    print(f"pack_alpha n={n} k={k} outliers={outliers}", flush=True)
    W = _weights(n, k, 4, outliers)
    dW = dev(W)
    s = slim.quant_search(dW)
    p = host_pack(slim.pack_alpha(dW, s["out"], with_mask=True))
    ref = Q.pack_alpha(W, s["alpha"])
    for key in ("codes", "meta", "scales", "mask"):
        assert np.array_equal(p[key], ref[key]), key


def test_pack_alpha_rejects_bad_alpha():
    W = dev(_weights(16, 128, 5))
    a = torch.tensor([-1.0], dtype=torch.float64, device="cuda")
    with pytest.raises(slim.SlimError) as e:
        slim.pack_alpha(W, a)
    assert e.value.status == slim.SLIM_ERANGE


@pytest.mark.parametrize("m,r", [(16, 64), (300, 64)])
def test_linear_on_slim_quant_pack(m, r):
    # the layer kernels are unchanged; their input is now a pack with one scale for every group
    n, k = 1024, 1024
    print(f"linear on slim-quant pack m={m} r={r}", flush=True)
    W = _weights(n, k, 6, outliers=20)
    xbits, X = synth.activations(m, k, seed=6, name="quant/X", dtype="bf16")
    Lb, Rb, L, R = synth.adapter(k, n, r, seed=6, name="quant/")
    dW = dev(W)
    s = slim.quant_search(dW)
    p = slim.pack_alpha(dW, s["out"])
    ad = slim.pack_adapter(dev_bits(Lb, torch.float16), dev_bits(Rb, torch.float16))
    Y = host(slim.linear(dev_bits(xbits, torch.bfloat16), p, ad))
    ref = O.linear(X, Q.pack_alpha(W, s["alpha"]), L, R, n, k)
    assert_close(Y, ref, f"slim-quant linear m={m}")
