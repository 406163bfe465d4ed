"""4-bit adapters (SLiM-LoRA^Q): slim_pack_adapter_q bit-exact against the oracle, and slim_linear_qa
against the oracle's layer with the dequantized adapters, within the gate."""
import numpy as np
import pytest
import torch

from oracle import slim_oracle as O
from paper_2608_24070_amd import slim, synth
from tests.gpu_common import assert_close, dev, dev_bits, host

pytestmark = pytest.mark.gpu


def _adapter(K, N, r, seed, name):
    Lb, Rb, L, R = synth.adapter(K, N, r, seed=seed, name=name + "/")
    return dev_bits(Lb, torch.float16), dev_bits(Rb, torch.float16), L, R


@pytest.mark.parametrize("K,N,r", [(512, 512, 32), (4096, 4096, 384), (256, 72, 96), (5120, 13824, 512),
                                   (8192, 28672, 512)])
def test_pack_adapter_q_bit_exact(K, N, r):
    print(f"pack_adapter_q K={K} N={N} r={r}", flush=True)
    dL, dR, L, R = _adapter(K, N, r, 1, "qpack")
    q = slim.pack_adapter_q(dL, dR)
    ref = O.pack_adapter_q(L, R)
    for key in ("Lq", "Ls", "Rq", "Rs"):
        got = host(q[key])
        got = got.view(np.uint16) if got.dtype == np.int16 else got
        assert np.array_equal(got, ref[key]), key


def _case(n, k, r, m, xdtype="bf16", rows=None, ms=None, seed=0, name="qa"):
    print(f"linear_qa n={n} k={k} r={r} m={m} {xdtype}", flush=True)
    W = synth.weights(n, k, seed=seed, name=name + "/W")
    xb, X = synth.activations(m, k, seed=seed, name=name + "/X", dtype=xdtype)
    dx = dev_bits(xb, torch.bfloat16 if xdtype == "bf16" else torch.float16)
    dL, dR, L, R = _adapter(k, n, r, seed, name)
    p = slim.pack(dev(W))
    qa = slim.pack_adapter_q(dL, dR)
    Y = slim.linear_qa(dx, p, qa).clone()
    # the same layer through the fp16-adapter path, fed the dequantized factors rounded to fp16 (the
    # values the kernels form in registers): the same kernels and order, so the same bits
    pq = {kk: (host(v).view(np.uint16) if host(v).dtype == np.int16 else host(v)) for kk, v in qa.items()
          if isinstance(v, torch.Tensor)}
    Ld, Rd = O.unpack_adapter_q(pq, k, n, r)
    ad16 = slim.pack_adapter(dev(Ld.astype(np.float16)), dev(Rd.astype(np.float16)))
    Y16 = slim.linear(dx, p, ad16)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y16), "4-bit adapter path differs from the fp16 path on the same values"
    Yh = host(Y)
    rows = np.arange(n) if rows is None else rows
    ms = np.arange(m) if ms is None else ms
    ref = O.linear_qa(X[ms], O.pack(W[rows]), {"Lq": pq["Lq"], "Ls": pq["Ls"], "Rq": pq["Rq"][rows], "Rs": pq["Rs"][rows]},
                      len(rows), k, r)
    assert_close(Yh[np.ix_(ms, rows)], ref, f"linear_qa n={n} k={k} r={r} m={m}")


@pytest.mark.parametrize("m,r,xdtype", [(16, 32, "fp16"), (1, 32, "bf16"), (5, 96, "bf16")])
def test_linear_qa_tiny(m, r, xdtype):
    _case(512, 512, r, m, xdtype=xdtype, name="qtiny")


@pytest.mark.parametrize("m", [1, 4, 16])
def test_linear_qa_decode(m):
    _case(4096, 4096, 384, m, name="qdecode")


@pytest.mark.parametrize("m,r", [(20, 160), (32, 64), (9, 416)])
def test_linear_qa_small_m_ranks(m, r):
    # two 16-row fragments, and ranks whose last group is partial or whose finish passes end inside a pass
    _case(1024, 2048, r, m, name="qsmall")


@pytest.mark.parametrize("m,r", [(200, 64), (33, 96), (300, 32)])
def test_linear_qa_large_m(m, r):
    _case(1024, 1024, r, m, name="qlarge")


def test_linear_qa_prefill_sampled():
    rows = np.sort(synth.stream(21, "rows").choice(11008, size=512, replace=False))
    ms = np.sort(synth.stream(21, "ms").choice(2048, size=48, replace=False))
    _case(11008, 4096, 384, 2048, rows=rows, ms=ms, name="qprefill")


@pytest.mark.parametrize("m", [1, 16])
def test_linear_qa_mlp70b_sampled(m):
    rows = np.sort(synth.stream(22, "rows").choice(28672, size=384, replace=False))
    _case(28672, 8192, 512, m, rows=rows, name="qmlp70b")


def test_pack_adapter_q_rejects_nonfinite():
    dL, dR, _, _ = _adapter(256, 64, 32, 3, "qbad")
    dL[7, 3] = float("inf")
    with pytest.raises(slim.SlimError) as e:
        slim.pack_adapter_q(dL, dR)
    assert e.value.status == slim.SLIM_ENONFINITE
