"""Pins of the training-step oracle (oracle/slope_train.py) against things other than itself.

Brute force (pure Python enumeration in oracle/brute.py), closed forms and invariants: a planted
mistake in the oracle (a transposed product, a wrong tie key, a dropped coefficient, values taken
from the wrong positions, a mask ignored) fails at least one of them. No GPU.
"""
import numpy as np
import pytest

from oracle import brute as B
from oracle import slope_train as T
from paper_2608_24070_amd import synth


def _weights(n, k, seed, tied=False):
    rng = synth.stream(seed, "train/W")
    if tied:
        lv = rng.integers(0, 5, size=(n, k)).astype(np.float32) * np.float32(0.25)
        w = lv * np.where(rng.random((n, k)) < 0.5, -1.0, 1.0).astype(np.float32)
        w[rng.random((n, k)) < 0.05] = -0.0
        return w
    return (rng.standard_normal((n, k)) * 0.02).astype(np.float32)


@pytest.mark.parametrize("tied", [False, True])
def test_pack16_matches_brute_force(tied):
    n, k = 8, 32
    W = _weights(n, k, 1, tied)
    p = T.pack16(W)
    vals = p["vals"].view(np.float16).astype(np.float64).reshape(n, k // 2)
    for i in range(n):
        for g in range(k // 4):
            kept = B.top2([float(x) for x in W[i, 4 * g:4 * g + 4]])
            for s, pos in enumerate(sorted(kept)):
                assert vals[i, 2 * g + s] == B.f16_nearest(float(W[i, 4 * g + pos]))
            assert [int(x) for x in p["mask"][i, 4 * g:4 * g + 4]] == [1 if t in kept else 0 for t in range(4)]
    # the dense form is the masked, rounded weight
    dense = T.unpack16(p["vals"], p["meta"], n, k)
    ref = np.where(p["mask"] == 1, W.astype(np.float16).astype(np.float64), 0.0)
    assert np.array_equal(dense, ref)


@pytest.mark.parametrize("tied", [False, True])
def test_pack16_t_matches_brute_column_prune(tied):
    n, k = 16, 16
    W = _weights(n, k, 2, tied)
    p = T.pack16(W)
    Wr = T.unpack16(p["vals"], p["meta"], n, k)
    keep = B.column_prune(Wr.tolist(), p["mask"].tolist())
    pt = T.pack16_t(p["vals"], p["meta"], n, k)
    assert np.array_equal(pt["mask_rc"], np.array(keep, dtype=np.uint8))
    # the transposed pack holds exactly the surviving values
    assert np.array_equal(T.unpack16_t(pt["valsT"], pt["metaT"], n, k), Wr * pt["mask_rc"])
    # and is a 2:4 pack along N for every k
    mt = T.mask_of_meta(pt["metaT"], k, n)
    assert np.all(mt.reshape(k, n // 4, 4).sum(axis=2) == 2)


def test_double_prune_density_matches_lemma():
    # Lemma sparsity_ratio: double pruning a random 2:4 row mask removes 9.375% of the entries
    n, k = 512, 512
    p = T.pack16(_weights(n, k, 3))
    pt = T.pack16_t(p["vals"], p["meta"], n, k)
    drop = p["mask"].mean() - pt["mask_rc"].mean()
    assert abs(drop - 0.09375) < 0.004


def test_grad_w_matches_brute_force():
    m, n, k = 5, 8, 16
    rng = synth.stream(4, "train/g")
    dY = rng.integers(-3, 4, size=(m, n)).astype(np.float64)    # small integers: exact products
    X = rng.integers(-3, 4, size=(m, k)).astype(np.float64)
    p = T.pack16(_weights(n, k, 4))
    g = T.grad_w(dY, X, p["meta"], n, k)
    full = B.matmul(B.transpose(dY.tolist()), X.tolist())          # [n][k]
    for i in range(n):
        kept = [j for j in range(k) if p["mask"][i, j]]
        assert [full[i][j] for j in kept] == list(g[i])


def test_grad_w_is_the_masked_dense_gradient():
    m, n, k = 7, 16, 32
    rng = synth.stream(5, "train/g2")
    dY, X = rng.standard_normal((m, n)), rng.standard_normal((m, k))
    p = T.pack16(_weights(n, k, 5))
    g = T.grad_w(dY, X, p["meta"], n, k)
    # row-major walk of the mask's kept positions gives the compressed order
    ref = (dY.T @ X)[p["mask"] == 1].reshape(n, k // 2)
    assert np.allclose(g, ref, rtol=1e-13, atol=1e-13)
    # a transposed product would not even have this shape
    assert g.shape == (n, k // 2)


def test_sparse_add_closed_forms():
    rng = synth.stream(6, "train/add")
    A = rng.standard_normal(64)
    Bv = rng.standard_normal(64).astype(np.float16)
    assert np.array_equal(T.sparse_add(A, Bv, 1.0, 0.0), A)
    assert np.array_equal(T.sparse_add(A, Bv, 0.0, 1.0), Bv.astype(np.float64))
    assert np.allclose(T.sparse_add(A, Bv, 2.0, -3.0), 2.0 * A - 3.0 * Bv.astype(np.float64))
    # linear in each argument
    assert np.allclose(T.sparse_add(A, Bv, 0.5, 0.25) * 2, T.sparse_add(A, Bv, 1.0, 0.5))


def test_update_pack16_roundtrip_and_rounding():
    p = T.pack16(_weights(8, 32, 7))
    v32 = p["vals"].view(np.float16).astype(np.float32)
    assert np.array_equal(T.update_pack16(v32), p["vals"])
    x = np.array([[1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11]], dtype=np.float32)   # binary16 ties
    got = T.update_pack16(x).view(np.float16).astype(np.float64)[0]
    assert list(got) == [B.f16_nearest(float(v)) for v in x[0]] == [1.0, 1.0 + 2.0 ** -9]


def test_pack16_rejects_non_finite_and_bad_shapes():
    W = _weights(4, 32, 8)
    W[1, 3] = np.inf
    with pytest.raises(T.OracleError):
        T.pack16(W)
    with pytest.raises(T.OracleError):
        T.pack16(_weights(4, 24, 8))


def test_pack16_t_prefers_kept_zeros_over_pruned_slots():
    # column 0 of rows 0..3: row 2 keeps a zero (its group has three zeros), rows 0, 1, 3 drop
    # position 0; the column prune ranks the kept zero before the dropped slots, so it survives
    W = np.zeros((16, 16), dtype=np.float32)
    W[0, :4] = [0.0, 5.0, 5.0, 0.0]
    W[1, :4] = [0.0, 4.0, 3.0, 0.0]
    W[2, :4] = [0.0, 0.0, 0.0, 1.0]
    W[3, :4] = [0.0, 2.0, 0.0, 7.0]
    W[4:, :] = 1.0
    p = T.pack16(W)
    assert list(p["mask"][:4, 0]) == [0, 0, 1, 0]
    pt = T.pack16_t(p["vals"], p["meta"], 16, 16)
    assert list(pt["mask_rc"][:4, 0]) == [0, 0, 1, 0]
    Wr = T.unpack16(p["vals"], p["meta"], 16, 16)
    assert np.array_equal(pt["mask_rc"], np.array(B.column_prune(Wr.tolist(), p["mask"].tolist()), dtype=np.uint8))
