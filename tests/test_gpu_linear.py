"""slim_linear and slim_linear_bwd_dx against the fp64 oracle, within the tolerance gate
(relative Frobenius error <= 2e-3 and max |error| <= 1e-2 * max |Y_ref|)."""
import numpy as np
import pytest
import torch

from oracle import slim_oracle as O
from paper_2608_24070_amd import slim, synth
from tests.gpu_common import assert_close, dev, dev_bits, host, layer_inputs, oracle_pack_on_device

pytestmark = pytest.mark.gpu


def _fwd_case(n, k, r, m, xdtype="bf16", outliers=False, seed=0, rows=None, ms=None, name="layer",
              use_oracle_pack=False, xscale=1.0):
    print(f"fwd n={n} k={k} r={r} m={m} {xdtype} outliers={outliers} seed={seed} xscale={xscale}", flush=True)
    W, X, L, R, dx, ad = layer_inputs(n, k, r, m, seed=seed, xdtype=xdtype, outliers=outliers, name=name,
                                      xscale=xscale)
    if use_oracle_pack:
        p = oracle_pack_on_device(O.pack(W), n, k)
    else:
        p = slim.pack(dev(W))
    Y = host(slim.linear(dx, p, ad))
    torch.cuda.synchronize()
    rows = np.arange(n) if rows is None else rows
    ms = np.arange(m) if ms is None else ms
    ref = O.linear(X[ms], O.pack(W[rows]), L, None if R is None else R[:, rows], len(rows), k)
    return assert_close(Y[np.ix_(ms, rows)], ref, f"fwd n={n} k={k} r={r} m={m}")


@pytest.mark.parametrize("m,r,xdtype", [(16, 32, "fp16"), (1, 32, "fp16"), (16, 0, "fp16"), (3, 32, "bf16")])
def test_tiny(m, r, xdtype):
    _fwd_case(512, 512, r, m, xdtype=xdtype, name="tiny")


@pytest.mark.parametrize("m", [1, 4, 16])
def test_decode_shape(m):
    _fwd_case(4096, 4096, 384, m, name="decode")


@pytest.mark.parametrize("n,k,m,r", [(16, 128, 1, 0), (16, 128, 5, 16), (80, 384, 32, 16), (80, 384, 7, 0),
                                     (16, 256, 40, 16), (80, 640, 100, 32)])
def test_smallest_shapes(n, k, m, r):
    # one 16-row block, a ragged 64-row tile (80 rows), one to five 128-wide chunks (K = 640 leaves a
    # lane group of the small-M kernel without a chunk), on both paths
    _fwd_case(n, k, r, m, name="edge")


@pytest.mark.parametrize("m", [1, 20])
def test_decode_long_reduction(m):
    # K = 13824: 27 adapter units' worth of 512 positions, so each wave of a unit takes four 128-position
    # slices (7 splits); the last unit's fourth wave lies wholly past K
    _fwd_case(512, 13824, 32, m, name="longk")


@pytest.mark.parametrize("k,r,m", [(4096, 16, 16), (4096, 48, 1), (3200, 80, 16), (1152, 112, 3), (384, 16, 32),
                                   (4096, 272, 20), (2048, 400, 9)])
def test_decode_adapter_ranks(k, r, m):
    # adapter units are 16 ranks wide: one to seven column blocks, one to eight splits, ragged last
    # splits (K = 3200 and 1152 end inside a unit) and a single split (K = 384); ranks 272 and 400
    # give the finish two waves per 16 rows whose rank passes end inside a pass
    _fwd_case(320, k, r, m, name="adranks")


@pytest.mark.parametrize("m", [17, 32, 33, 64])
def test_small_m_multi_fragment(m):
    _fwd_case(1024, 2048, 64, m, name="smallm")


@pytest.mark.parametrize("m,r", [(65, 32), (200, 16), (256, 0), (300, 48), (40, 80)])
def test_tile_kernel_ragged(m, r):
    _fwd_case(768, 1024, r, m, name="ragged")


@pytest.mark.parametrize("k,m", [(128, 100), (256, 97), (384, 130)])
def test_tile_kernel_short_reduction(k, m):
    # one to three 128-wide chunks: the tile kernel's prologue and remainder paths alone
    _fwd_case(528, k, 16, m, name="shortk")


@pytest.mark.parametrize("m", [1, 16, 27])
def test_decode_blocks_run_several_row_tiles(m):
    # 313 row tiles: forward sparse blocks take 3 (m <= 16) or 5 (m > 16) row tiles each, the last
    # block fewer; the sampled rows include the last tiles
    n = 20032
    rows = np.unique(np.concatenate([synth.stream(5, "rows").choice(n, size=384, replace=False),
                                     np.arange(n - 200, n)]))
    _fwd_case(n, 4096, 64, m, rows=rows, name="units")


@pytest.mark.parametrize("m", [1, 16, 27])
def test_decode_long_blocks_repeat(m):
    # K = 8192: 5 (m <= 16) or 8 (m > 16) row tiles per forward sparse block with 8 or 16 splits; a
    # second call on the same workspace gives the same bits and leaves the counters at zero
    n, k = 20032, 8192
    rows = np.unique(np.concatenate([synth.stream(6, "rows").choice(n, size=320, replace=False),
                                     np.arange(n - 160, n)]))
    _fwd_case(n, k, 64, m, rows=rows, name="shared")
    W, X, L, R, dx, ad = layer_inputs(n, k, 64, m, name="shared")
    p = slim.pack(dev(W))
    ws = torch.zeros(slim.slim_linear_workspace(m, n, k, 64), dtype=torch.uint8, device=dx.device)
    y0 = slim.linear(dx, p, ad, ws=ws).clone()
    y1 = slim.linear(dx, p, ad, ws=ws).clone()
    torch.cuda.synchronize()
    assert torch.equal(y0, y1)
    assert int(ws[:COUNTER_BYTES].count_nonzero()) == 0


def test_tile_kernel_wide_tiles_ragged_m():
    # 22 row tiles x 1400 columns: the plan takes 512 x 128 tiles (11 column tiles, the last 120
    # wide); the sampled columns include the last ones
    rows = np.sort(synth.stream(6, "rows").choice(11008, size=256, replace=False))
    ms = np.unique(np.concatenate([synth.stream(6, "ms").choice(1400, size=40, replace=False), np.arange(1380, 1400)]))
    _fwd_case(11008, 2048, 48, 1400, rows=rows, ms=ms, name="wide")


def test_tile_kernel_eight_waves_ragged_rows():
    # the tile kernel runs 8 waves of 64 rows: 2064 rows leave 16 in the last row tile, so one wave
    # there holds 16 rows and seven hold none; 128 column tiles of 128
    rows = np.unique(np.concatenate([synth.stream(7, "rows").choice(2064, size=200, replace=False),
                                     np.arange(2040, 2064)]))
    ms = np.unique(np.concatenate([synth.stream(7, "ms").choice(16384, size=40, replace=False),
                                   np.arange(16380, 16384)]))
    _fwd_case(2064, 5120, 32, 16384, rows=rows, ms=ms, name="w8")


@pytest.mark.parametrize("n,k,r,m", [(4096, 1024, 384, 4096), (4096, 1024, 272, 4096), (768, 1024, 272, 300)])
def test_tile_epilogue_rank_groups(n, k, r, m):
    # the epilogue's adapter product takes tm through LDS in groups of eight 16-rank steps, one
    # activation stage per group: 512 x 128 tiles (two stages) with three groups, the last one whole
    # (r 384) or of one step (r 272), and 512 x 96 tiles (three stages) with r 272
    rows = np.unique(np.concatenate([synth.stream(10, "rows").choice(n, size=min(n, 256), replace=False),
                                     np.arange(n - 16, n)]))
    ms = np.unique(np.concatenate([synth.stream(10, "ms").choice(m, size=40, replace=False), np.arange(m - 8, m)]))
    _fwd_case(n, k, r, m, rows=rows, ms=ms, name="epi")


@pytest.mark.parametrize("n,k,r,m", [(256, 33024, 512, 1900), (128, 16384, 512, 4096), (128, 2048, 512, 32768)])
def test_adapter_gemm_wide_tiles(n, k, r, m):
    # the 256 x 256 adapter GEMM takes shapes whose 256 x 256 tiles times reduction splits of at least
    # 2048 fill 256 blocks: a ragged last m tile (M = 1900, 16 tiles) over 16 splits whose last one is
    # short (reduction 33024 in slices of 2080), 32 tiles over 8 splits of exactly 2048, and 256 tiles
    # with no split (T written in fp16 by the GEMM itself)
    ms = np.unique(np.concatenate([synth.stream(8, "ms").choice(m, size=40, replace=False), np.arange(m - 8, m)]))
    _fwd_case(n, k, r, m, ms=ms, name="adwide")


def test_linear_on_oracle_pack():
    _fwd_case(1024, 1024, 64, 16, use_oracle_pack=True, name="opack")
    _fwd_case(1024, 1024, 64, 256, use_oracle_pack=True, name="opack")


def test_prefill_sampled():
    rows = np.sort(synth.stream(1, "prows").choice(11008, size=1024, replace=False))
    ms = np.sort(synth.stream(1, "pms").choice(2048, size=128, replace=False))
    _fwd_case(11008, 4096, 384, 2048, rows=rows, ms=ms, name="prefill")


def test_prefill_fp16_outliers_sampled():
    rows = np.sort(synth.stream(2, "prows").choice(11008, size=512, replace=False))
    ms = np.sort(synth.stream(2, "pms").choice(2048, size=64, replace=False))
    _fwd_case(11008, 4096, 384, 2048, xdtype="fp16", outliers=True, rows=rows, ms=ms, name="prefill")


def test_block13b_down_proj_sampled():
    rows = np.sort(synth.stream(3, "rows").choice(5120, size=512, replace=False))
    ms = np.sort(synth.stream(3, "ms").choice(4096, size=64, replace=False))
    _fwd_case(5120, 13824, 512, 4096, rows=rows, ms=ms, name="down")


@pytest.mark.parametrize("m", [1, 16, 512, 8192])
def test_mlp70b_fwd_sampled(m):
    rows = np.sort(synth.stream(4, "rows").choice(28672, size=512, replace=False))
    ms = None if m <= 16 else np.sort(synth.stream(4, "ms").choice(m, size=32, replace=False))
    _fwd_case(28672, 8192, 512, m, rows=rows, ms=ms, name="mlp70b")


def test_forward_is_deterministic():
    W, X, L, R, dx, ad = layer_inputs(4096, 4096, 384, 16, name="det")
    p = slim.pack(dev(W))
    a = slim.linear(dx, p, ad).clone()
    b = slim.linear(dx, p, ad).clone()
    assert torch.equal(a, b)
    W, X, L, R, dx, ad = layer_inputs(1024, 1024, 64, 256, name="det2")
    p = slim.pack(dev(W))
    assert torch.equal(slim.linear(dx, p, ad).clone(), slim.linear(dx, p, ad).clone())


@pytest.mark.parametrize("k,n,r", [(512, 512, 32), (4096, 11008, 384), (13824, 5120, 512), (200, 72, 16)])
def test_pack_adapter_is_exact_transpose(k, n, r):
    Lb, Rb, _, _ = synth.adapter(k, n, r, seed=5, name="tp/")
    ad = slim.pack_adapter(dev_bits(Lb, torch.float16), dev_bits(Rb, torch.float16))
    assert np.array_equal(host(ad["Lt"]).view(np.uint16), Lb.T)
    # Rt: R^T in 32 x 16 tiles [ceil(n/32), r/16, 32, 16], rows past n zero
    rt = host(ad["Rt"]).view(np.uint16)
    assert rt.shape == ((n + 31) // 32, r // 16, 32, 16)
    rowmajor = rt.transpose(0, 2, 1, 3).reshape((n + 31) // 32 * 32, r)
    assert np.array_equal(rowmajor[:n], Rb.T)
    assert not rowmajor[n:].any()


# ------------------------------------------------------------------------------ backward

def _bwd_case(n, k, r, m, seed=0, ks=None, ms=None, name="bwd", dydtype="bf16", dyscale=1.0):
    print(f"bwd n={n} k={k} r={r} m={m} seed={seed} {dydtype} dyscale={dyscale}", flush=True)
    W = synth.weights(n, k, seed=seed, name=name + "/W")
    dybits, dY = synth.activations(m, n, seed=seed, name=name + "/dY", dtype=dydtype, scale=dyscale)
    Lb, Rb, L, R = synth.adapter(k, n, max(r, 16), seed=seed, name=name + "/")
    if r == 0:
        L = R = dL = dR = None
    else:
        Lb, Rb, L, R = Lb[:, :r].copy(), Rb[:r].copy(), L[:, :r], R[:r]
        dL, dR = dev_bits(Lb, torch.float16), dev_bits(Rb, torch.float16)
    tdt = torch.bfloat16 if dydtype == "bf16" else torch.float16
    pb = slim.pack_bwd(slim.pack(dev(W)))
    dX = host(slim.bwd_dx(dev_bits(dybits, tdt), pb, dL, dR))
    ms = np.arange(m) if ms is None else ms
    if ks is None:
        ref = O.bwd_dx(dY[ms], O.pack_bwd(O.pack(W), n, k), L, R, n, k)
        return assert_close(dX[ms], ref, f"bwd n={n} k={k} r={r} m={m}")
    for g in ks:   # one 128-column group at a time: the backward pack is separable by K-group
        cols = slice(128 * g, 128 * g + 128)
        ref = O.bwd_dx(dY[ms], O.pack_bwd(O.pack(W[:, cols]), n, 128), None if L is None else L[cols], R, n, 128)
        assert_close(dX[np.ix_(ms, np.arange(128 * g, 128 * g + 128))], ref, f"bwd group {g}")


def test_tile_kernel_exact_tiles():
    # rows and columns that fill whole 512 x 96 tiles: no ragged edge anywhere (two row tiles, four
    # column tiles, a reduction of eight chunks)
    _fwd_case(1024, 1024, 64, 384, name="exact")


@pytest.mark.parametrize("m,r", [(16, 32), (1, 0), (5, 32), (33, 32), (64, 32), (200, 32), (256, 0)])
def test_bwd_small(m, r):
    _bwd_case(512, 512, r, m, name="bwd_small")


@pytest.mark.parametrize("n,k,m,r", [(128, 128, 1, 0), (128, 128, 9, 16), (256, 384, 33, 16), (384, 640, 70, 32)])
def test_bwd_smallest_shapes(n, k, m, r):
    _bwd_case(n, k, r, m, name="bwd_edge")


def test_bwd_decode_shape():
    _bwd_case(4096, 4096, 384, 16, name="bwd_decode")


@pytest.mark.parametrize("n,r,m", [(9216, 48, 16), (3328, 16, 1)])
def test_bwd_decode_adapter_ranks(n, r, m):
    # backward reduction over N: 9216 positions give 18 units' worth of 512, so each wave takes three
    # 128-position slices (6 splits); N = 3328 ends inside the seventh unit
    _bwd_case(n, 256, r, m, name="bwd_adranks")


@pytest.mark.parametrize("m,seed", [(1, 0), (16, 1), (512, 2), (8192, 0)])
def test_bwd_mlp70b_sampled(m, seed):
    ms = None if m <= 16 else np.sort(synth.stream(seed, "bms").choice(m, size=24, replace=False))
    _bwd_case(28672, 8192, 512, m, seed=seed, ks=(0, 31, 63), ms=ms, name="mlp70b")


def test_bwd_wide_tiles_ragged_m():
    # backward rows = K = 11008 (22 row tiles), 1400 columns: 512 x 128 tiles with a ragged last one
    ms = np.unique(np.concatenate([synth.stream(7, "ms").choice(1400, size=24, replace=False), np.arange(1390, 1400)]))
    _bwd_case(2048, 11008, 48, 1400, seed=3, ks=(0, 85), ms=ms, name="bwide")


def test_bwd_adapter_gemm_wide_tiles():
    # U = dY R^T on the 256 x 256 adapter GEMM: r 512, M 1900 (eight m tiles, the last ragged),
    # reduction N = 33024 in 16 splits, the last one short
    ms = np.unique(np.concatenate([synth.stream(9, "ms").choice(1900, size=24, replace=False), np.arange(1892, 1900)]))
    _bwd_case(33024, 256, 512, 1900, seed=4, ks=(0, 1), ms=ms, name="bwd_adwide")


def test_bwd_tile_epilogue_rank_groups():
    # dX = dY W^{R,C} + (dY R^T) L^T at r 272 on 512 x 128 tiles: three groups of rank steps, the
    # last of one step
    ms = np.unique(np.concatenate([synth.stream(11, "ms").choice(4096, size=24, replace=False), np.arange(4088, 4096)]))
    _bwd_case(1024, 4096, 272, 4096, seed=5, ks=(0, 31), ms=ms, name="bwd_epi")


def test_bwd_is_deterministic():
    n, k, m = 4096, 4096, 16
    W = synth.weights(n, k, seed=9)
    dybits, _ = synth.activations(m, n, seed=9)
    Lb, Rb, _, _ = synth.adapter(k, n, 64, seed=9)
    pb = slim.pack_bwd(slim.pack(dev(W)))
    dy = dev_bits(dybits, torch.bfloat16)
    dL, dR = dev_bits(Lb, torch.float16), dev_bits(Rb, torch.float16)
    assert torch.equal(slim.bwd_dx(dy, pb, dL, dR).clone(), slim.bwd_dx(dy, pb, dL, dR).clone())


COUNTER_BYTES = 4096 * 4   # the workspace's leading counter region


def test_decode_counters_return_to_zero():
    # the front of the workspace is a counter region that every call must leave at zero; calls on
    # one workspace give the results of calls on fresh ones
    W, X, L, R, dx, ad = layer_inputs(2048, 1024, 64, 32, name="ctr")
    p = slim.pack(dev(W))
    pb = slim.pack_bwd(p)
    ws = torch.zeros(64 << 20, dtype=torch.uint8, device=dx.device)
    dy = dx.new_empty((16, 2048)).normal_().to(dx.dtype)
    for m in (16, 1, 7, 32, 20):
        Y0 = slim.linear(dx[:m], p, ad).clone()
        Y1 = slim.linear(dx[:m], p, ad, ws=ws)
        Y2 = slim.linear(dx[:m], p, None, ws=ws)
        D0 = slim.bwd_dx(dy[:min(m, 16)], pb, ad["L"], ad["R"]).clone()
        D1 = slim.bwd_dx(dy[:min(m, 16)], pb, ad["L"], ad["R"], ws=ws)
        torch.cuda.synchronize()
        assert torch.equal(Y0, Y1) and torch.equal(D0, D1), m
        assert Y2.shape == (m, 2048) and dx.shape[0] == 32
        assert int(ws[:COUNTER_BYTES].count_nonzero()) == 0, m


# ------------------------------------------------------------ magnitudes outside fp16's range
# The kernels scale each activation row by a power of two before rounding it to fp16, so
# gradient-sized dY (products dY * s16 far below fp16's normal range) and bf16 activations beyond
# fp16's maximum stay within the gate.

@pytest.mark.parametrize("m,dydtype,dyscale", [(16, "bf16", 1e-3), (16, "bf16", 1e-5), (1, "bf16", 1e-7),
                                               (27, "fp16", 1e-4), (200, "bf16", 1e-3), (200, "bf16", 1e-5),
                                               (96, "fp16", 1e-5), (64, "bf16", 1e-7)])
def test_bwd_gradient_magnitudes(m, dydtype, dyscale):
    _bwd_case(1024, 512, 32, m, name="gradmag", dydtype=dydtype, dyscale=dyscale)


@pytest.mark.parametrize("m,r", [(16, 0), (200, 0)])
def test_bwd_gradient_magnitudes_no_adapter(m, r):
    _bwd_case(1024, 512, r, m, name="gradmag0", dyscale=1e-5)


def test_bwd_gradient_magnitudes_mlp70b_sampled():
    # the 70B shape at gradient size on both paths, sampled K groups
    _bwd_case(28672, 8192, 512, 16, seed=1, ks=(0, 40), name="mlp70b", dyscale=1e-5)
    ms = np.sort(synth.stream(1, "gms").choice(512, size=16, replace=False))
    _bwd_case(28672, 8192, 512, 512, seed=1, ks=(7, 63), ms=ms, name="mlp70b", dyscale=1e-5)


@pytest.mark.parametrize("m,r,xscale", [(16, 32, 1e6), (16, 32, 1e-6), (1, 0, 1e6), (20, 48, 3e4),
                                        (200, 32, 1e6), (200, 32, 1e-6), (100, 0, 1e6), (96, 0, 1e-6)])
def test_forward_activations_beyond_fp16_range(m, r, xscale):
    _fwd_case(1024, 2048, r, m, name="xmag", xscale=xscale)


@pytest.mark.parametrize("m", [16, 200])
def test_forward_fp16_small_activations(m):
    # fp16 activations of 1e-5 (near fp16's subnormal range) with an adapter: the adapter's
    # intermediate X L is scaled with the rows
    _fwd_case(1024, 2048, 64, m, xdtype="fp16", name="xmag16", xscale=1e-5)


# ------------------------------------------------------------ every configuration's shapes

@pytest.mark.parametrize("n,k", [(5120, 5120), (13824, 5120)])
def test_block13b_q_and_gate_sampled(n, k):
    rows = np.sort(synth.stream(8, "rows").choice(n, size=512, replace=False))
    ms = np.sort(synth.stream(8, "ms").choice(4096, size=48, replace=False))
    _fwd_case(n, k, 512, 4096, rows=rows, ms=ms, name=f"b13_{n}x{k}")


@pytest.mark.parametrize("m,seed", [(16, 1), (16, 2), (8192, 1), (8192, 2)])
def test_mlp70b_fwd_seeds_sampled(m, seed):
    rows = np.sort(synth.stream(10 + seed, "rows").choice(28672, size=384, replace=False))
    ms = None if m <= 16 else np.sort(synth.stream(10 + seed, "ms").choice(m, size=24, replace=False))
    _fwd_case(28672, 8192, 512, m, seed=seed, rows=rows, ms=ms, name="mlp70b")
