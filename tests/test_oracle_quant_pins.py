"""Pins of the SLiM-Quant oracle (oracle/slim_quant.py) against things other than itself.

* Brute force on tiny inputs: per-element binning and error sums in plain Python, and the
  candidate search by enumeration.
* Closed forms: for |w| uniform on [0, 1], E(alpha) = alpha delta^2 / 12 + (1 - alpha)^3 / 3 with
  delta = alpha / (2^(q-1) - 1), whose minimiser is 14/15 at q = 4 and 2/3 at q = 2; the grid
  search must land on the grid point of least closed-form error.
* Independent quadrature: the continuous integrals of eq. quantization_error and
  eq. clipping_error against the half-normal density (scipy.integrate.quad over each rounding
  cell) agree with the histogram estimate built from exact bin probabilities.
* Invariants: power-of-two scaling of W scales alpha* exactly; alpha* is never worse than AbsMax.
* The pack option reduces to the pinned AbsMax pack when every group holds the global maximum,
  and clips to the extreme codes beyond alpha (brute-force rounding).
No GPU.
"""
import math

import numpy as np
import pytest
from scipy import integrate, stats

from oracle import brute as B
from oracle import slim_oracle as O
from oracle import slim_quant as Q
from paper_2608_24070_amd import synth


def _weights(n, k, seed, scale=0.02):
    rng = synth.stream(seed, "quant/W")
    return (rng.standard_normal((n, k)) * scale).astype(np.float32)


def _brute_error(ws, bins, amax, alpha, qmax):
    """Mean over the elements of the error at each element's bin centre (pure Python)."""
    delta = alpha / qmax
    tot = 0.0
    for w in ws:
        a = abs(float(w))
        b = min(math.floor((a * bins) / amax), bins - 1)
        c = (b + 0.5) * (amax / bins)
        if c <= alpha:
            q = round(c / delta)                 # Python rounds half to even
            tot += (delta * q - c) ** 2
        else:
            tot += (alpha - c) ** 2
    return tot / len(ws)


@pytest.mark.parametrize("bits", [4, 3])
def test_histogram_error_and_search_match_brute_force(bits):
    W = _weights(6, 40, 1)
    W[0, :3] = [0.0, -0.0, W.max()]               # zeros and a repeated maximum
    ws = [float(x) for x in W.ravel()]
    bins = 16
    amax = max(abs(w) for w in ws)
    counts = [0] * bins
    for w in ws:
        counts[min(math.floor((abs(w) * bins) / amax), bins - 1)] += 1
    r = Q.search(W, bits=bits, bins=bins)
    assert r["amax"] == amax
    assert list(r["counts"]) == counts
    qmax = 2 ** (bits - 1) - 1
    # every tabulated error against the per-element sum
    for a, e in r["table"]:
        assert e == pytest.approx(_brute_error(ws, bins, amax, a, qmax), rel=1e-12, abs=0)
    # the search by enumeration: ten multiples of amax/10, then twenty steps of amax/100
    coarse = [(i * (amax / 10), _brute_error(ws, bins, amax, i * (amax / 10), qmax)) for i in range(1, 11)]
    lo = coarse[min(range(10), key=lambda i: (coarse[i][1], i))][0]
    fine = [(lo - amax / 10) + j * (amax / 10 / 10) for j in range(20)]
    cands = coarse + [(a, _brute_error(ws, bins, amax, a, qmax)) for a in fine if a > 0]
    best = min(range(len(cands)), key=lambda i: (cands[i][1], i))
    assert r["alpha"] == pytest.approx(cands[best][0], rel=1e-15)


@pytest.mark.parametrize("bits,qmax,alpha_star", [(4, 7, 0.93), (2, 1, 0.67)])
def test_uniform_magnitudes_closed_form(bits, qmax, alpha_star):
    bins = 20000
    counts = np.full(bins, 50, dtype=np.int64)     # |w| uniform on [0, 1]

    def closed(a):
        d = a / qmax
        return a * d * d / 12 + (1 - a) ** 3 / 3

    for a in (0.1, 0.37, 0.5, 0.8, 0.93, 1.0):
        assert Q.estimate_error(counts, 1.0, a, bits) == pytest.approx(closed(a), rel=1e-6)
    r = Q.search_hist(counts, 1.0, bits)
    assert r["alpha"] == pytest.approx(alpha_star, abs=1e-12)
    # the analytic minimiser of the closed form lies within one fine step of alpha*
    a_opt = 14 / 15 if bits == 4 else 2 / 3
    assert abs(r["alpha"] - a_opt) < 0.01
    # and alpha* is the grid point of least closed-form error among its fine neighbours
    assert closed(alpha_star) < closed(alpha_star - 0.01) and closed(alpha_star) < closed(alpha_star + 0.01)


def test_half_normal_against_quadrature():
    # exact bin probabilities of |w| for w ~ N(0, 1) truncated at 6 sigma
    amax, bins, bits = 6.0, 20000, 4
    edges = np.linspace(0.0, amax, bins + 1)
    p = 2 * (stats.norm.cdf(edges[1:]) - stats.norm.cdf(edges[:-1]))
    counts = p / p.sum()
    f = lambda x: 2 * stats.norm.pdf(x) / (2 * (stats.norm.cdf(amax) - 0.5))

    def quad_error(alpha):
        d = alpha / 7
        tot = 0.0
        for kq in range(8):          # rounding cells [ (k - 1/2) d, (k + 1/2) d ] clipped to [0, alpha]
            lo, hi = max(0.0, (kq - 0.5) * d), min(alpha, (kq + 0.5) * d)
            if hi > lo:
                tot += integrate.quad(lambda x: f(x) * (kq * d - x) ** 2, lo, hi, epsabs=1e-14)[0]
        tot += integrate.quad(lambda x: f(x) * (alpha - x) ** 2, alpha, amax, epsabs=1e-14)[0]
        return tot

    for a in (1.5, 2.4, 2.6, 3.0, 4.2):
        assert Q.estimate_error(counts, amax, a, bits) == pytest.approx(quad_error(a), rel=2e-4)
    r = Q.search_hist(counts, amax, bits)
    # the fine grid's best point under the quadrature is the oracle's alpha*
    grid = [a for a, _ in r["table"][10:]]
    assert r["alpha"] == pytest.approx(min(grid, key=quad_error), rel=1e-12)


def test_power_of_two_scaling_is_exact():
    W = _weights(64, 256, 3)
    r1 = Q.search(W, bins=700)
    r2 = Q.search(W * np.float32(4.0), bins=700)
    assert np.array_equal(r1["counts"], r2["counts"])
    assert r2["alpha"] == 4.0 * r1["alpha"]
    assert r2["error"] == 16.0 * r1["error"]


def test_alpha_never_worse_than_absmax():
    for seed in range(4):
        W = _weights(128, 256, 10 + seed)
        W[3, 5] = 0.5                                  # an outlier far beyond the bulk
        r = Q.search(W)
        assert r["error"] <= Q.estimate_error(r["counts"], r["amax"], r["amax"], 4)
        assert r["alpha"] < r["amax"]                  # the outlier is clipped


def test_bin_count_formula():
    assert Q.bin_count(512, 512) == 512
    assert Q.bin_count(4096, 4096) == 16777
    assert Q.bin_count(11008, 4096) == 20000
    assert Q.bin_count(28672, 8192) == 20000


def test_pack_alpha_reduces_to_absmax_pack():
    # every 128-group of every row holds +-amax, so each group's AbsMax scale is the global one
    n, k = 16, 512
    W = _weights(n, k, 4)
    amax = np.float32(0.125)
    W = np.clip(W, -0.1, 0.1)
    W[:, ::128] = amax
    W[::2, 64::128] = -amax
    ref = O.pack(W)
    got = Q.pack_alpha(W, float(amax))
    for key in ("codes", "meta", "scales", "mask"):
        assert np.array_equal(got[key], ref[key]), key


def test_pack_alpha_clips_beyond_alpha():
    n, k = 4, 128
    W = _weights(n, k, 5, scale=0.05)
    W[0, :4] = [0.3, -0.29, 0.01, 0.0]               # far beyond alpha: must clip to +-7
    alpha = 0.07
    p = Q.pack_alpha(W, alpha)
    s = float(np.float16(np.float32(alpha) / np.float32(7)))
    dense = O.unpack(p["codes"], p["meta"], p["scales"], n, k)
    m = O.mask_2of4(W)
    for i in range(n):
        for j in range(k):
            want = B.rtn_code(float(W[i, j]), s) * s if m[i, j] else 0.0
            assert dense[i, j] == want
    assert dense[0, 0] == 7 * s and dense[0, 1] == -7 * s


def test_degenerate_inputs():
    z = np.zeros((16, 128), dtype=np.float32)
    r = Q.search(z)
    assert r["alpha"] == 0.0 and r["table"] == []
    p = Q.pack_alpha(z, 0.0)
    assert np.all(p["scales"] == 0)
    W = _weights(16, 128, 6)
    W[2, 3] = np.nan
    with pytest.raises(O.OracleError):
        Q.search(W)


def test_bins_are_exact_rational_floors_at_bin_edges():
    # magnitudes next to every bin edge k amax / B (the float32 neighbours of the exact edge):
    # the bin must be the exact rational floor(|w| B / amax)
    from fractions import Fraction
    bins, amax = 1000, np.float32(3.0)
    vals = []
    for kq in range(1, bins):
        e = np.float32(kq * 3.0 / bins)
        vals += [np.nextafter(e, np.float32(0)), e, np.nextafter(e, np.float32(4))]
    W = np.array(vals + [amax], dtype=np.float32)
    counts, got_amax = Q.histogram(W, bins)
    assert got_amax == 3.0
    ref = [0] * bins
    for w in W:
        ref[min(math.floor(Fraction(float(w)) * bins / Fraction(3.0)), bins - 1)] += 1
    assert list(counts) == ref
    # magnitudes exactly on dyadic edges (j / 8 with amax = 1 and 600 bins: edge 75 j), where a
    # bin width rounded to float64 (1/600 is not dyadic) would put some of them one bin low
    W = np.array([j / 8 for j in range(1, 9)] + [0.0], dtype=np.float32)
    counts, _ = Q.histogram(W, 600)
    assert [int(i) for i in np.nonzero(counts)[0]] == [0] + [75 * j for j in range(1, 8)] + [599]


def test_candidate_grid_and_absmax_optimum():
    # all magnitudes equal: only AbsMax reconstructs them (up to the half bin between the maximum
    # and the centre of its bin); every clipped alpha leaves an error of order (amax - alpha)^2
    W = np.where(_weights(16, 128, 7) < 0, np.float32(-0.25), np.float32(0.25)).astype(np.float32)
    r = Q.search(W, bins=600)
    assert r["alpha"] == 0.25 and r["error"] == pytest.approx((0.25 / 600 / 2) ** 2, rel=1e-9)
    # the coarse candidates are exactly i amax / 10 for i = 1 .. 10, the fine ones step amax / 100
    assert [a for a, _ in r["table"][:10]] == [i * (0.25 / 10) for i in range(1, 11)]
    fine = [a for a, _ in r["table"][10:]]
    assert len(fine) == 20 and fine[0] == 0.25 - 0.025
    assert np.allclose(np.diff(fine), 0.0025, rtol=0, atol=1e-15)
