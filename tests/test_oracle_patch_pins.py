"""Pins of the PATCH hybrid-tile oracle (oracle/patch_hybrid.py) against things other than itself.

* Brute force: every group of a sparse tile keeps the pattern pure-Python enumeration picks, with
  the values exhaustive fp16 rounding gives; dense tiles keep every value.
* Special cases: all-dense reduces to the fp16 weight and a plain matmul; one sparse tile changes
  that block only.
* A hand-built tile checks the byte layout (value order, index nibbles, offsets, the sparse bit).
No GPU.
"""
import numpy as np
import pytest

from oracle import brute as B
from oracle import patch_hybrid as P
from oracle import slim_oracle as O
from paper_2608_24070_amd import synth


def _w(n, k, seed, tied=False):
    if tied:
        rng = synth.stream(seed, "patch/tied")
        lv = rng.integers(0, 4, size=(n, k)).astype(np.float32) * np.float32(0.5)
        return lv * np.where(rng.random((n, k)) < 0.5, -1.0, 1.0).astype(np.float32)
    return synth.weights(n, k, seed=seed, name="patch/W")


@pytest.mark.parametrize("tied", [False, True])
def test_sparse_tiles_match_brute_force(tied):
    n, k = 128, 256
    W = _w(n, k, 1, tied)
    kinds = np.array([[1, 0]], dtype=np.uint8)
    Wp = P.hybrid_weight(W, kinds)
    for i in range(0, n, 7):
        for g in range(k // 4):
            ws = [float(x) for x in W[i, 4 * g:4 * g + 4]]
            kept = B.top2(ws) if g < 32 else (0, 1, 2, 3)
            for p in range(4):
                want = B.f16_nearest(ws[p]) if p in kept else 0.0
                assert Wp[i, 4 * g + p] == want, (i, g, p)


def test_all_dense_is_the_fp16_matmul():
    n, k, m = 256, 384, 5
    W = _w(n, k, 2)
    Wp = P.hybrid_weight(W, np.zeros((2, 3), dtype=np.uint8))
    assert np.array_equal(Wp, W.astype(np.float16).astype(np.float64))
    X = synth.stream(2, "patch/X").standard_normal((m, k)).astype(np.float16)
    assert np.allclose(P.linear(X, Wp), X.astype(np.float64) @ W.astype(np.float16).astype(np.float64).T,
                       rtol=1e-12, atol=1e-12)
    assert P.sparsity(np.zeros((2, 3))) == 0.0


def test_one_sparse_tile_changes_only_its_block():
    n, k = 384, 512
    W = _w(n, k, 3)
    kinds = np.zeros((3, 4), dtype=np.uint8)
    kinds[1, 2] = 1
    Wp = P.hybrid_weight(W, kinds)
    dense = W.astype(np.float16).astype(np.float64)
    diff = Wp != dense
    assert not diff[:128].any() and not diff[256:].any()
    assert not diff[128:256, :256].any() and not diff[128:256, 384:].any()
    blk = Wp[128:256, 256:384].reshape(128, 32, 4)
    # the block is 2:4 (exactly two kept of every four; weights here are never exactly zero)
    assert np.all((blk != 0).sum(axis=2) == 2)
    assert P.sparsity(kinds) == pytest.approx(0.5 / 12)


def test_byte_layout_hand_built_tile():
    n, k = 128, 256
    W = np.full((n, k), 0.25, dtype=np.float32)
    W[0, :8] = [4.0, -1.0, 3.0, 0.5, 0.0, -2.0, 2.0, 1.0]
    kinds = np.array([[1, 0]], dtype=np.uint8)
    pk = P.pack(W, kinds)
    info = pk["tile_info"]
    assert int(info[0, 0]) == (1 << 63)                       # sparse, offset 0
    assert int(info[0, 1]) == P.SPARSE_BYTES                  # dense, right after
    pay = pk["payload"]
    assert pay.size == P.SPARSE_BYTES + P.DENSE_BYTES
    vals = pay[:8].view(np.float16)
    # group 0 keeps positions 0, 2 (4, 3); group 1 keeps 5, 6 (-2, 2), lower position first
    assert list(vals) == [4.0, 3.0, -2.0, 2.0]
    # the first half's index words follow its 128 rows x 32 values
    half0 = int(pay[P.TILE * P.TILE // 2:P.TILE * P.TILE // 2 + 2].view("<u2")[0])
    assert half0 & 0xF == (0 | 2 << 2) and (half0 >> 4) & 0xF == (1 | 2 << 2)
    # the dense tile: row 0 of W's columns 128.. as fp16, 256 bytes per row
    d0 = pay[P.SPARSE_BYTES:P.SPARSE_BYTES + 256].view(np.float16)
    assert np.all(d0 == np.float16(0.25))
    assert np.array_equal(P.unpack(info, pay, n, k), P.hybrid_weight(W, kinds))


@pytest.mark.parametrize("seed", [4, 5])
def test_pack_unpack_round_trip(seed):
    n, k = 256, 512
    W = _w(n, k, seed, tied=seed == 5)
    kinds = (synth.stream(seed, "patch/kinds").random((2, 4)) < 0.6).astype(np.uint8)
    pk = P.pack(W, kinds)
    assert pk["payload"].size == P.payload_bytes(kinds)
    assert np.array_equal(P.unpack(pk["tile_info"], pk["payload"], n, k), P.hybrid_weight(W, kinds))
    # the sparse tiles agree with the 2:4 mask the library's pinned pack uses
    m = O.mask_2of4(W)
    tm = P.tile_mask(kinds, n, k)
    assert np.array_equal((P.hybrid_weight(W, kinds) != 0) | (W == 0), np.where(tm == 1, m == 1, True) | (W == 0))


def test_rejects_bad_inputs():
    with pytest.raises(O.OracleError):
        P.hybrid_weight(_w(128, 200, 6), np.zeros((1, 1)))
    W = _w(128, 128, 6)
    W[3, 3] = np.inf
    with pytest.raises(O.OracleError):
        P.pack(W, np.zeros((1, 1)))
