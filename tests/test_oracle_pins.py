"""Pins of the CPU oracle against things other than itself (no GPU needed).

Each test names what fixes the expected value: brute force, a closed form, a value
printed in the thesis, or an invariant of the definition. A planted mistake in the
oracle (a dropped term, a wrong sign or index, a transposed operand, a wrong tie or
rounding rule, a swapped nibble) fails at least one of them.
"""
import math
import os
import struct

import numpy as np
import pytest

from oracle import brute as B
from oracle import slim_oracle as O
from paper_2608_24070_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tied_weights(n, k, seed):
    """Weights with many exact magnitude ties (few levels, random signs) to exercise tie rules."""
    rng = synth.stream(seed, "tied")
    lv = rng.integers(0, 6, size=(n, k)).astype(np.float32) * np.float32(0.013)
    sg = np.where(rng.random((n, k)) < 0.5, -1.0, 1.0).astype(np.float32)
    w = lv * sg
    w[rng.random((n, k)) < 0.05] = -0.0
    return w


# ---------------------------------------------------------------- rounding pins

def test_fp16_rne_matches_exhaustive_search():
    rng = synth.stream(0, "f16pin")
    xs = list(rng.standard_normal(300).astype(np.float32) * np.float32(0.05))
    xs += list((rng.random(100) * 6e-5).astype(np.float32))               # subnormal range
    xs += [np.float32(65504.0), np.float32(65519.0), np.float32(65520.0), np.float32(0.0)]
    # exact midpoints between adjacent binary16 values (ties) in the normal range
    for bits in [0x2C00, 0x2C01, 0x3555, 0x0001, 0x03FF, 0x1234, 0x3BFF]:
        lo = struct.unpack("<e", bits.to_bytes(2, "little"))[0]
        hi = struct.unpack("<e", (bits + 1).to_bytes(2, "little"))[0]
        xs.append(np.float32((lo + hi) / 2))
    xs = np.array(xs, dtype=np.float32)
    got = O.fp16_rne(xs).astype(np.float64)
    want = np.array([B.f16_nearest(float(x)) for x in xs])
    assert np.array_equal(got, want)


def test_scale_uses_fp32_division_then_fp16():
    # a/7 for float32 a, rounded once to fp32 and then to fp16, versus exhaustive search.
    rng = synth.stream(1, "scalepin")
    a = np.abs(rng.standard_normal(200).astype(np.float32)) * np.float32(0.08)
    W = np.zeros((200, 128), dtype=np.float32)
    W[:, 5] = a
    s = O.group_scales(W)[:, 0].astype(np.float64)
    want = [B.f16_nearest(B.to_f32(float(x) / 7.0)) for x in a]
    assert np.array_equal(s, want)


def _exact_rne_f16_of_a_over_7(a):
    """RNE of the exact quotient a/7 to binary16, by exact comparisons against the table of every
    finite binary16 value: 7 t and 2 a are exact in float64 (t has 11 significant bits, a 24),
    and so is 7 (t_lo + t_hi), so no step here rounds."""
    table = B._f16_table()
    a = np.asarray(a, dtype=np.float64)
    lo = np.searchsorted(table, a / 7.0, side="right") - 1
    lo = np.clip(lo, 0, len(table) - 2)
    lo = np.where(7.0 * table[lo] > a, lo - 1, lo)              # t_lo <= a/7 exactly
    lo = np.where(7.0 * table[lo + 1] <= a, lo + 1, lo)         # a/7 < t_hi exactly
    two_a, mid7 = 2.0 * a, 7.0 * (table[lo] + table[lo + 1])
    pick_hi = (two_a > mid7) | ((two_a == mid7) & (lo % 2 == 1))   # ties to the even bit pattern
    return np.where(pick_hi, table[lo + 1], table[lo])


def test_scale_is_exact_rne_of_a_over_7_at_every_fp16_midpoint():
    # Double rounding (a/7 -> fp32 -> fp16) can differ from one rounding of the exact quotient only
    # where the fp32 quotient lands on a binary16 midpoint m. For float32 a that needs
    # |a - 7m| <= 3.5 ulp32(m), while 7m is a float32 whose neighbours are 4 or 8 ulp32(m) away:
    # only a = 7m itself qualifies (an exact tie). This checks every positive midpoint (normal and
    # subnormal binary16) with a = 7m and its two float32 neighbours on each side, against the exact
    # rational rounding. It fails a reciprocal multiply a * fp32(1/7) (17384 of these cases differ)
    # and truncation; computing a/7 in float64 and rounding once to fp16 gives the same scales
    # everywhere, which is why the reading's fp32 division is pinned as exact RNE of a/7.
    table = B._f16_table()
    mids = (table[:-1] + table[1:]) / 2.0
    a0 = (7.0 * mids).astype(np.float32)
    assert np.array_equal(a0.astype(np.float64), 7.0 * mids)
    up1, dn1 = np.nextafter(a0, np.float32(np.inf)), np.nextafter(a0, np.float32(0))
    a = np.concatenate([a0, up1, dn1, np.nextafter(up1, np.float32(np.inf)), np.nextafter(dn1, np.float32(0))])
    a = a[(a > 0) & (a.astype(np.float64) / 7.0 < 65504.0)]
    want = _exact_rne_f16_of_a_over_7(a)
    got = np.empty(len(a))
    for c0 in range(0, len(a), 16384):
        blk = a[c0:c0 + 16384]
        W = np.zeros((len(blk), 128), dtype=np.float32)
        W[:, 77] = blk
        W[:, 3] = -blk * np.float32(0.5)
        got[c0:c0 + len(blk)] = O.group_scales(W)[:, 0].astype(np.float64)
    assert np.array_equal(got, want)
    ties = a0[a0.astype(np.float64) / 7.0 < 65504.0]
    assert len(ties) > 30000                                   # exact ties of both parities are in the set
    spot = synth.stream(2, "spot").choice(len(a), size=64, replace=False)
    assert [B.f16_nearest(B.to_f32(float(a[i]) / 7.0)) for i in spot] == list(want[spot])


# ----------------------------------------------------------- mask (P1, P2, P10)

@pytest.mark.parametrize("seed", [0, 1])
def test_mask_two_of_four_and_bruteforce(seed):
    W = _tied_weights(8, 256, seed)
    m = O.mask_2of4(W)
    assert m.dtype == np.uint8
    assert np.all(m.reshape(8, 64, 4).sum(axis=2) == 2)            # P1: exactly 2 of every 4
    for i in range(8):
        for j in range(64):
            kept = tuple(np.nonzero(m[i, 4 * j:4 * j + 4])[0])
            assert kept == B.top2([float(x) for x in W[i, 4 * j:4 * j + 4]])   # P2


def test_mask_zero_signs_are_ties():
    W = np.zeros((1, 128), dtype=np.float32)
    W[0, 0] = -0.0
    W[0, 1] = 0.0
    W[0, 2] = -0.0
    assert list(O.mask_2of4(W)[0, :4]) == [1, 1, 0, 0]


def test_pack_commutes_with_masking():
    # P10: pack(W) == pack(M (.) W): the group absmax sits in a kept slot (P3),
    # so masking first changes neither the scale nor any kept code.
    W = synth.weights(64, 512, seed=3)
    m = O.mask_2of4(W)
    a, b = O.pack(W), O.pack(W * m)
    for key in ("codes", "meta", "scales", "mask"):
        assert np.array_equal(a[key], b[key]), key


def test_quantize_then_mask_equals_mask_then_quantize():
    W = synth.weights(32, 256, seed=4)
    s = O.group_scales(W)
    q_all = O.quantize(W, s)                           # quantise every weight first
    m = O.mask_2of4(W)                                  # mask from fp32 magnitudes
    Wc_qfirst = m * q_all * np.repeat(s.astype(np.float64), 128, axis=1)
    assert np.array_equal(Wc_qfirst, O.dequant_dense(W))


# ----------------------------------------------------------- scales (P3, P4, P5)

def test_absmax_is_kept():
    W = synth.weights(64, 1024, seed=5)
    m = O.mask_2of4(W)
    a_all = np.abs(W).reshape(64, 8, 128).max(axis=2)
    a_kept = np.abs(W * m).reshape(64, 8, 128).max(axis=2)
    assert np.array_equal(a_all, a_kept)


def test_roundtrip_bound_and_full_scale_code():
    W = synth.weights(64, 1024, seed=6)
    s = O.group_scales(W).astype(np.float64)
    assert np.all(s >= 2.0 ** -14)                      # normal fp16 scales here
    m = O.mask_2of4(W).astype(bool)
    Wc = O.dequant_dense(W)
    S = np.repeat(s, 128, axis=1)
    err = np.abs(W.astype(np.float64) - Wc)
    assert np.all(err[m] <= S[m] / 2)                   # P4: |w - q s| <= s/2
    q = O.quantize(W, O.group_scales(W))
    am = np.abs(W).reshape(64, 8, 128).argmax(axis=2)
    qa = np.take_along_axis(q.reshape(64, 8, 128), am[..., None], axis=2)
    assert np.all(np.abs(qa) == 7)                      # |q| = 7 at the group maximum


def test_rtn_bruteforce_with_exact_ties():
    rng = synth.stream(7, "rtn")
    s16 = np.float16(0.0123)
    s = float(s16)
    ks = rng.integers(-7, 7, size=64)
    ties = ((ks + 0.5) * s).astype(np.float32)          # exact half-way points
    rnd = (rng.standard_normal(192) * 3 * s).astype(np.float32)
    w = np.concatenate([ties, rnd]).astype(np.float32).reshape(2, 128)
    sc = np.full((2, 1), s16, dtype=np.float16)
    q = O.quantize(w, sc)
    for i in range(2):
        for j in range(128):
            assert q[i, j] == B.rtn_code(float(w[i, j]), s), (i, j, w[i, j])


def test_zero_and_tiny_groups():
    W = np.zeros((2, 256), dtype=np.float32)
    W[1, 130] = 1e-8                                     # a/7 underflows fp16 -> s16 = 0
    p = O.pack(W)
    assert np.all(p["scales"] == 0)
    Wc = O.unpack(p["codes"], p["meta"], p["scales"], 2, 256)
    assert np.all(Wc == 0)
    assert np.all(np.ascontiguousarray(p["codes"]).view("<u4") == 0x88888888)


def test_rejects_nonfinite_and_overflow():
    W = np.zeros((1, 128), dtype=np.float32)
    W[0, 3] = np.nan
    with pytest.raises(O.OracleError):
        O.pack(W)
    W[0, 3] = np.inf
    with pytest.raises(O.OracleError):
        O.pack(W)
    W[0, 3] = 7.0 * 65520.0                              # scale rounds to +inf in fp16
    with pytest.raises(O.OracleError):
        O.pack(W)
    with pytest.raises(O.OracleError):
        O.pack(np.zeros((1, 100), dtype=np.float32))


# ------------------------------------------------------------ format (P6, P11)

def _read_fixture(name):
    rows = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            rows[key] = vals
    return rows


def test_worked_example_bytes():
    fx = _read_fixture("pack_worked_example.txt")
    W = np.zeros((1, 128), dtype=np.float32)
    for item in fx["weights"]:
        k, v = item.split(":")
        W[0, int(k)] = np.float32(float(v))
    p = O.pack(W)
    assert p["scales"][0, 0] == int(fx["scale"][0], 16)
    codes = p["codes"][0]
    meta = p["meta"][0]
    assert list(codes[:4]) == [int(b, 16) for b in fx["codes_block0"]]
    assert list(meta[:2]) == [int(b, 16) for b in fx["meta_block0"]]
    other_c = [int(b, 16) for b in fx["codes_other"]]
    other_m = [int(b, 16) for b in fx["meta_other"]]
    for blk in range(1, 8):
        assert list(codes[4 * blk:4 * blk + 4]) == other_c
        assert list(meta[2 * blk:2 * blk + 2]) == other_m


@pytest.mark.parametrize("shape", [(8, 128), (48, 512), (17, 384)])
def test_unpack_of_pack_equals_direct_dequant(shape):
    # P6: decoding the packed bytes gives exactly the weight computed directly from W.
    W = synth.weights(*shape, seed=8)
    p = O.pack(W)
    assert np.array_equal(O.unpack(p["codes"], p["meta"], p["scales"], *shape), O.dequant_dense(W))
    W2 = _tied_weights(*shape, seed=9)
    p2 = O.pack(W2)
    assert np.array_equal(O.unpack(p2["codes"], p2["meta"], p2["scales"], *shape), O.dequant_dense(W2))


def test_dense_weight_matches_bruteforce():
    W = _tied_weights(4, 256, 10) + synth.weights(4, 256, seed=11) * np.float32(0.1)
    W = W.astype(np.float32)
    want = np.array(B.dense_weight([[float(x) for x in row] for row in W]))
    assert np.array_equal(O.dequant_dense(W), want)


def test_pack_sizes_and_index_bits():
    n, k = 96, 1024
    p = O.pack(synth.weights(n, k, seed=12))
    total = p["codes"].nbytes + p["meta"].nbytes + p["scales"].nbytes
    assert total == O.pack_bytes(n, k) == n * k * (1 / 4 + 1 / 8 + 1 / 64)
    assert total * 8 / (n * k) == 3.125                 # bits per dense weight
    for line in open(os.path.join(GOLDEN, "index_bits.txt")):
        if line.strip() and not line.startswith("#"):
            N, M, bits = map(int, line.split())
            assert math.ceil(math.log2(math.comb(M, N))) == bits    # eq. index_bits
    assert 2 * 2 >= 3                                   # 2 bits per kept value >= the 3-bit minimum


def test_pack_is_deterministic():
    W = synth.weights(64, 256, seed=13)
    a, b = O.pack(W), O.pack(W.copy())
    for key in a:
        assert np.array_equal(a[key], b[key])


# ----------------------------------------------------------------- layer (P7, P8)

@pytest.mark.parametrize("m,r", [(1, 0), (2, 1), (3, 2)])
def test_linear_bruteforce_tiny(m, r):
    n, k = 4, 128
    W = synth.weights(n, k, seed=20 + m)
    _, X = synth.activations(m, k, seed=20 + m, dtype="fp16")
    _, _, L, R = synth.adapter(k, n, max(r, 1), seed=20 + m)
    L, R = (L[:, :r], R[:r]) if r else (None, None)
    Y = O.linear(X, O.pack(W), L, R, n, k)
    Yb = np.array(B.linear(X.tolist(), [[float(x) for x in row] for row in W],
                           None if L is None else L.tolist(), None if R is None else R.tolist()))
    assert np.allclose(Y, Yb, rtol=1e-12, atol=1e-14)


def test_linear_reduces_to_plain_matmul_for_exact_weights():
    # W already 2:4 with entries q 2^e and group absmax 7 2^e: quantisation is exact (Wc == W),
    # so with r = 0 the layer is numpy's matmul of X and W^T.
    rng = synth.stream(30, "exact")
    n, k = 32, 256
    W = np.zeros((n, k), dtype=np.float32)
    for i in range(n):
        e = -int(rng.integers(3, 9))
        for j in range(k // 4):
            pos = rng.choice(4, size=2, replace=False)
            q = rng.integers(-7, 8, size=2)
            q[q == 0] = 1
            W[i, 4 * j + pos] = q * 2.0 ** e
        for g in range(k // 128):
            j = 4 * int(rng.integers(0, 32)) + 128 * g
            W[i, j:j + 4] = 0
            W[i, j] = 7 * 2.0 ** e
            W[i, j + 1] = -3 * 2.0 ** e
    assert np.array_equal(O.dequant_dense(W), W.astype(np.float64))
    _, X = synth.activations(5, k, seed=31)
    assert np.allclose(O.linear(X, O.pack(W), None, None, n, k), np.matmul(X, W.astype(np.float64).T),
                       rtol=1e-13, atol=1e-13)


def test_linear_identity_input_exposes_layout():
    n, k, r = 24, 128, 3
    W = synth.weights(n, k, seed=32)
    _, _, L, R = synth.adapter(k, n, r, seed=32)
    Y = O.linear(np.eye(k), O.pack(W), L, R, n, k)
    assert np.allclose(Y, O.dequant_dense(W).T + L @ R, rtol=1e-13, atol=1e-15)


def test_linear_zero_adapter_and_r0_agree():
    n, k, r = 16, 256, 4
    W = synth.weights(n, k, seed=33)
    _, X = synth.activations(3, k, seed=33)
    p = O.pack(W)
    Y0 = O.linear(X, p, None, None, n, k)
    Yz = O.linear(X, p, np.zeros((k, r)), synth.adapter(k, n, r, seed=33)[3], n, k)
    assert np.array_equal(Y0, Yz)
    assert np.allclose(Y0, X @ O.dequant_dense(W).T, rtol=1e-13, atol=1e-15)


# ------------------------------------------------------ double pruning (P9, P7)

def test_lemma_closed_form_matches_printed_values():
    for line in open(os.path.join(GOLDEN, "lemma_sparsity_ratio.txt")):
        if line.strip() and not line.startswith("#"):
            N, M, v = line.split()
            assert abs(O.lemma_extra_sparsity(int(N), int(M)) - float(v)) < 1e-15


def test_double_pruning_extra_sparsity_statistic():
    n, k = 1024, 512
    W = synth.weights(n, k, seed=40)
    p = O.pack(W)
    b = O.pack_bwd(p, n, k)
    mr, mrc = p["mask"].astype(np.int64), b["mask_rc"].astype(np.int64)
    assert np.all(mrc <= mr)                                      # supp(W^{R,C}) within supp(W^R)
    extra = (mr.sum() - mrc.sum()) / mr.size
    assert abs(extra - O.lemma_extra_sparsity(2, 4)) < 2e-3       # Lemma sparsity_ratio, 2:4
    # per column group: exactly max(0, j - 2) forward entries are dropped
    j = mr.T.reshape(k, n // 4, 4).sum(axis=2)
    drop = j - mrc.T.reshape(k, n // 4, 4).sum(axis=2)
    assert np.array_equal(drop, np.maximum(0, j - 2))
    assert np.all(mrc.T.reshape(k, n // 4, 4).sum(axis=2) <= 2)


def test_transposable_mask_loses_nothing():
    pat = np.array([[1, 1, 0, 0], [0, 0, 1, 1], [1, 1, 0, 0], [0, 0, 1, 1]], dtype=np.float32)
    n, k = 32, 256
    P = np.tile(pat, (n // 4, k // 4))
    W = synth.weights(n, k, seed=41)
    W = (np.sign(W) * (0.05 + np.abs(W)) * P + W * np.float32(1e-3) * (1 - P)).astype(np.float32)
    p = O.pack(W)
    assert np.array_equal(p["mask"], P.astype(np.uint8))
    b = O.pack_bwd(p, n, k)
    assert np.array_equal(b["mask_rc"], p["mask"])
    Wc = O.unpack(p["codes"], p["meta"], p["scales"], n, k)
    _, dY = synth.activations(3, n, seed=41)
    assert np.allclose(O.bwd_dx(dY, b, None, None, n, k), dY @ Wc, rtol=1e-13, atol=1e-15)


def test_backward_pack_decodes_to_masked_forward_weight():
    n, k = 64, 384
    W = _tied_weights(n, k, 42)
    p = O.pack(W)
    b = O.pack_bwd(p, n, k)
    Wc = O.unpack(p["codes"], p["meta"], p["scales"], n, k)
    assert np.array_equal(O.unpack_bwd(b["codesT"], b["metaT"], b["scalesT"], n, k), Wc * b["mask_rc"])
    assert np.array_equal(b["scalesT"], p["scales"].T)


@pytest.mark.parametrize("m,r", [(1, 0), (2, 2)])
def test_bwd_bruteforce_tiny(m, r):
    n, k = 16, 128
    W = (_tied_weights(n, k, 50 + m) + synth.weights(n, k, seed=50 + m) * np.float32(0.2)).astype(np.float32)
    _, dY = synth.activations(m, n, seed=50 + m)
    _, _, L, R = synth.adapter(k, n, max(r, 1), seed=50 + m)
    L, R = (L[:, :r], R[:r]) if r else (None, None)
    p = O.pack(W)
    dX = O.bwd_dx(dY, O.pack_bwd(p, n, k), L, R, n, k)
    want = np.array(B.bwd_dx(dY.tolist(), [[float(x) for x in row] for row in W],
                             None if L is None else L.tolist(), None if R is None else R.tolist()))
    assert np.allclose(dX, want, rtol=1e-12, atol=1e-14)


def test_backward_pack_mask_matches_bruteforce():
    n, k = 16, 128
    W = _tied_weights(n, k, 60)
    p = O.pack(W)
    b = O.pack_bwd(p, n, k)
    Wc = O.unpack(p["codes"], p["meta"], p["scales"], n, k)
    want = B.column_prune(Wc.tolist(), p["mask"].tolist())
    assert np.array_equal(b["mask_rc"], np.array(want, dtype=np.uint8))


# ------------------------------------------------------------------ tolerance

def test_tolerance_gate():
    Y = np.ones((4, 4))
    assert O.within_tolerance(Y, Y)[0]
    assert not O.within_tolerance(Y * (1 + 3e-3), Y)[0]
    Z = Y.copy()
    Z[0, 0] += 0.02
    assert not O.within_tolerance(Z, Y)[0]


def test_tolerance_gate_max_abs_leg_alone():
    # One element off by 1.5e-2 of max|Y_ref| in a large array: the relative Frobenius error stays
    # far below 2e-3, so only the max-abs leg (max|Y - Y_ref| <= 1e-2 max|Y_ref|) can reject it.
    Yref = synth.stream(3, "gate").standard_normal((256, 1024))
    inf = np.max(np.abs(Yref))
    Y = Yref.copy()
    Y[17, 333] += 1.5e-2 * inf
    ok, rf, ma = O.within_tolerance(Y, Yref)
    assert rf < 2e-4 and abs(ma - 1.5e-2) < 1e-12
    assert not ok
    # just inside both legs: accepted
    Y[17, 333] = Yref[17, 333] + 0.9e-2 * inf
    assert O.within_tolerance(Y, Yref)[0]
    # and the Frobenius leg alone still rejects a uniform 3e-3 relative error
    assert not O.within_tolerance(Yref * (1 + 3e-3), Yref)[0]


# ------------------------------------------------------ quantized adapters (SLiM-LoRA^Q)

def test_adapter_quant_matches_bruteforce():
    # K = 256 (two groups of L^T rows), r = 48 (one partial group of R^T rows), ties from repeated levels
    K, N, r = 256, 32, 48
    Lb, Rb, L, R = synth.adapter(K, N, r, seed=11, name="aqb/")
    L = L.copy()
    L[5, 3] = L[9, 3] = 0.0                       # zeros and a tie between equal magnitudes
    L[7, 3] = -np.abs(L[:, 3]).max()
    # a group of rank 9 whose maximum is 10 * 2^-24: s16 = fp16(10/7 2^-24) = 2^-24 (subnormal, rounded
    # down), so a / s16 = 10 and the clamp to 7 decides the code
    L[:128, 9] = 0.0
    L[0, 9], L[1, 9] = 10 * 2.0 ** -24, -3 * 2.0 ** -24
    pqt = O.pack_adapter_q(L, R)
    assert pqt["Ls"][9, 0] == 0x0001
    Ld, Rd = O.unpack_adapter_q(pqt, K, N, r)
    assert Ld[0, 9] == 7 * 2.0 ** -24 and Ld[1, 9] == -3 * 2.0 ** -24
    assert np.array_equal(Ld.T, np.array(B.adapter_dequant(L.T.tolist())))
    assert np.array_equal(Rd.T, np.array(B.adapter_dequant(R.T.tolist())))


def test_adapter_quant_roundtrip_bound_and_full_scale_code():
    K, N, r = 512, 256, 80
    _, _, L, R = synth.adapter(K, N, r, seed=12, name="aqr/")
    for A in (L.T, R.T):                          # factors as quantized: rows along the input dimension
        s = O.adapter_group_scales(A).astype(np.float64)
        assert np.all(s >= 2.0 ** -14)
        q = O.adapter_quantize(A, s.astype(np.float16)).astype(np.float64)
        S = np.repeat(s, O.ADAPTER_GROUP, axis=1)[:, :A.shape[1]]
        assert np.all(np.abs(A - q * S) <= S / 2)
        for g in range(s.shape[1]):
            blk = slice(128 * g, 128 * g + 128)
            i = np.argmax(np.abs(A[:, blk]), axis=1)
            assert np.all(np.abs(q[:, blk][np.arange(A.shape[0]), i]) == 7)


def test_adapter_worked_example_bytes():
    # Hand derivation, one row of L^T (rank j = 0, K = 128, r = 8): elements 0..3 are 3.5, -1.0, 0.25,
    # 0.75, the rest 0. Group absmax 3.5: s16 = fp16(fp32(3.5) / 7) = 0.5 (bits 0x3800). Codes
    # q = rint(v / 0.5): 7, -2, rint(0.5) = 0 (tie to even), rint(1.5) = 2 (tie to even); u = q + 8:
    # 15, 6, 8, 10, then 8s. Word 0 holds elements 0..7 with element 2c in nibble c and 2c + 1 in
    # nibble c + 4: nibbles (7..0) = 8 8 A 6 | 8 8 8 F -> 0x88A6888F, bytes 8F 88 A6 88; every other
    # word is 0x88888888.
    L = np.zeros((128, 8))
    L[0, 0], L[1, 0], L[2, 0], L[3, 0] = 3.5, -1.0, 0.25, 0.75
    R = np.zeros((8, 16))
    pq = O.pack_adapter_q(L, R)
    assert list(pq["Lq"][0, :4]) == [0x8F, 0x88, 0xA6, 0x88]
    assert np.all(pq["Lq"][0, 4:] == 0x88) and np.all(pq["Lq"][1:] == 0x88)
    assert pq["Ls"][0, 0] == 0x3800 and np.all(pq["Ls"][1:] == 0)
    assert np.all(pq["Rq"] == 0x88) and np.all(pq["Rs"] == 0)
    Ld, _ = O.unpack_adapter_q(pq, 128, 16, 8)
    assert list(Ld[:4, 0]) == [3.5, -1.0, 0.0, 1.0]


def test_adapter_exact_values_make_linear_qa_equal_linear():
    # factors whose groups hold values q 2^e with a group maximum of 7 2^e dequantize to themselves
    rng = synth.stream(13, "aqx")
    K, N, r, m = 256, 64, 32, 3
    e = rng.integers(-9, -4, size=(r, K // 128))
    Lt = rng.integers(-7, 8, size=(r, K)).astype(np.float64) * np.repeat(2.0 ** e, 128, axis=1)
    Lt[:, ::128] = 7 * 2.0 ** e
    Rt = rng.integers(-7, 8, size=(N, r)).astype(np.float64) * 2.0 ** -6
    Rt[:, 0] = 7 * 2.0 ** -6
    L, R = Lt.T, Rt.T
    pq = O.pack_adapter_q(L, R)
    Ld, Rd = O.unpack_adapter_q(pq, K, N, r)
    assert np.array_equal(Ld, L) and np.array_equal(Rd, R)
    W = synth.weights(N, K, seed=13)
    _, X = synth.activations(m, K, seed=13)
    p = O.pack(W)
    assert np.array_equal(O.linear_qa(X, p, pq, N, K, r), O.linear(X, p, L, R, N, K))


def test_adapter_q_bytes():
    # 4 bits per element plus an fp16 scale per 128: 4.125 bits, 16 / 4.125 = 3.88x fewer bytes than fp16
    K = N = 4096
    r = 384
    assert O.adapter_q_bytes(K, N, r) * 8 == (r * K + N * r) * 4.125
    assert abs(2 * r * (K + N) / O.adapter_q_bytes(K, N, r) - 16 / 4.125) < 1e-12
    pq = O.pack_adapter_q(np.zeros((256, 48)), np.zeros((48, 32)))
    assert sum(v.nbytes for v in pq.values()) == O.adapter_q_bytes(256, 32, 48)
