"""PATCH hybrid dense / 2:4 tiles on the GPU (slim_pack_hybrid, slim_linear_hybrid) against the
oracle in oracle/patch_hybrid.py: bit-exact packs; products element by element within the fp32
summation bound. fp16 x fp16 products are exact in fp32, so the only error is the fp32 sum of K
terms: |Y - Y_exact| <= 2 K 2^-24 sum_k |x_k w_k| for any summation order."""
import numpy as np
import pytest
import torch

from oracle import patch_hybrid as P
from paper_2608_24070_amd import slim, synth
from tests.gpu_common import dev, host

pytestmark = pytest.mark.gpu


def _w(n, k, seed, tied=False):
    if tied:
        rng = synth.stream(seed, "ghyb/tied")
        lv = rng.integers(0, 4, size=(n, k)).astype(np.float32) * np.float32(0.5)
        w = lv * np.where(rng.random((n, k)) < 0.5, -1.0, 1.0).astype(np.float32)
        w[rng.random((n, k)) < 0.05] = -0.0
        return w
    return synth.weights(n, k, seed=seed, name="ghyb/W")


def _kinds(n, k, seed, frac):
    return (synth.stream(seed, "ghyb/kinds").random((n // 128, k // 128)) < frac).astype(np.uint8)


def _x(m, k, seed):
    return (synth.stream(seed, "ghyb/X").standard_normal((m, k)) * 1.0).astype(np.float16)


def _check_product(Y, X, Wp, rows=None):
    Xd = X.astype(np.float64)
    ref = Xd @ Wp.T
    bound = 2.0 * X.shape[1] * 2.0 ** -24 * (np.abs(Xd) @ np.abs(Wp).T) + 1e-30
    if rows is not None:
        Y = Y[rows]
    assert Y.shape == ref.shape
    assert np.all(np.abs(Y - ref) <= bound)


@pytest.mark.parametrize("n,k,frac,tied", [(128, 128, 1.0, False), (256, 512, 0.0, False), (384, 640, 0.6, True),
                                           (1024, 768, 0.7, False)])
def test_pack_bit_exact(n, k, frac, tied):
    print(f"hybrid pack n={n} k={k} frac={frac} tied={tied}", flush=True)
    W = _w(n, k, 1, tied)
    kinds = _kinds(n, k, 1, frac)
    p = slim.pack_hybrid(dev(W), kinds)
    ref = P.pack(W, kinds)
    assert np.array_equal(host(p["tile_info"]).view(np.uint64), ref["tile_info"])
    assert np.array_equal(host(p["payload"])[:ref["payload"].size], ref["payload"])


@pytest.mark.parametrize("m", [1, 16, 33, 128, 300])
@pytest.mark.parametrize("frac", [0.0, 0.7, 1.0])
def test_linear_parity(m, frac):
    n, k = 512, 1024
    print(f"hybrid linear m={m} frac={frac}", flush=True)
    W = _w(n, k, 2)
    kinds = _kinds(n, k, 2, frac)
    X = _x(m, k, 2)
    p = slim.pack_hybrid(dev(W), kinds)
    Y = host(slim.linear_hybrid(dev(X), p))
    _check_product(Y, X, P.hybrid_weight(W, kinds))


@pytest.mark.parametrize("n,k,m", [(384, 640, 40), (128, 256, 3), (640, 384, 200)])
def test_linear_odd_tile_rows(n, k, m):
    # N % 256 == 128: the last 256-row block holds one tile row (its second half lies past N)
    print(f"hybrid linear odd tile rows n={n} k={k} m={m}", flush=True)
    W = _w(n, k, 5)
    kinds = _kinds(n, k, 5, 0.5)
    X = _x(m, k, 5)
    p = slim.pack_hybrid(dev(W), kinds)
    Y = host(slim.linear_hybrid(dev(X), p))
    _check_product(Y, X, P.hybrid_weight(W, kinds))


@pytest.mark.parametrize("m", [16, 2048])
def test_llama7b_gate_proj_full_size(m):
    # 11008 x 4096 at 35% sparsity (70% of the tiles 2:4), sampled rows of Y
    n, k = 11008, 4096
    print(f"hybrid full size m={m}", flush=True)
    W = _w(n, k, 3)
    kinds = _kinds(n, k, 3, 0.7)
    X = _x(m, k, 3)
    p = slim.pack_hybrid(dev(W), kinds)
    Y = host(slim.linear_hybrid(dev(X), p))
    rows = np.arange(m) if m <= 16 else np.sort(synth.stream(3, "ghyb/rows").choice(m, size=48, replace=False))
    _check_product(Y, X[rows], P.hybrid_weight(W, kinds), rows=rows)


def test_deterministic_and_errors():
    n, k, m = 256, 2048, 8                                    # small M: split reduction
    W = _w(n, k, 4)
    kinds = _kinds(n, k, 4, 0.5)
    p = slim.pack_hybrid(dev(W), kinds)
    X = dev(_x(m, k, 4))
    a, b = slim.linear_hybrid(X, p), slim.linear_hybrid(X, p)
    assert torch.equal(a, b)
    Wn = W.copy()
    Wn[7, 9] = np.nan
    with pytest.raises(slim.SlimError) as e:
        slim.pack_hybrid(dev(Wn), kinds)
    assert e.value.status == slim.SLIM_ENONFINITE
    with pytest.raises(slim.SlimError) as e:
        slim.slim_linear_hybrid_workspace(4, 256, 200)
    assert e.value.status == slim.SLIM_ESHAPE
