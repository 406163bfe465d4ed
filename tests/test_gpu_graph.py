"""HIP-graph replays of slim_linear / slim_linear_bwd_dx equal the eager result bit for bit, on every
replay, with unrelated eager work in between (the library records no memsets; its split-K counters
reset themselves)."""
import numpy as np
import pytest
import torch

from paper_2608_24070_amd import slim, synth
from tests.gpu_common import dev, dev_bits, layer_inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n,k,r,m", [(4096, 4096, 384, 16), (1024, 2048, 64, 48), (1024, 1024, 64, 256),
                                     (20032, 8192, 64, 16)])
def test_forward_graph_replays(n, k, r, m):
    print(f"graph fwd n={n} k={k} r={r} m={m}", flush=True)
    W, X, L, R, dx, ad = layer_inputs(n, k, r, m, name="graph")
    p = slim.pack(dev(W))
    ws = torch.zeros(slim.slim_linear_workspace(m, n, k, r), dtype=torch.uint8, device="cuda")
    eager = slim.linear(dx, p, ad, ws=ws).clone()
    out = torch.empty_like(eager)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        slim.linear(dx, p, ad, out=out, ws=ws)
    noise = torch.randn(1 << 20, device="cuda")
    for rep in range(4):
        out.fill_(float("nan"))
        slim.linear(dx, p, ad, ws=ws)         # eager call sharing the workspace in between
        noise.mul_(1.0001).sum()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {rep} differs"


@pytest.mark.parametrize("n,k,r,m", [(4096, 4096, 384, 16), (1024, 1024, 64, 256)])
def test_bwd_graph_replays(n, k, r, m):
    print(f"graph bwd n={n} k={k} r={r} m={m}", flush=True)
    W = synth.weights(n, k, seed=3, name="gbwd/W")
    yb, _ = synth.activations(m, n, seed=3, name="gbwd/dY")
    Lb, Rb, _, _ = synth.adapter(k, n, r, seed=3, name="gbwd/")
    pb = slim.pack_bwd(slim.pack(dev(W)))
    dy, dL, dR = dev_bits(yb, torch.bfloat16), dev_bits(Lb, torch.float16), dev_bits(Rb, torch.float16)
    ws = torch.zeros(slim.slim_bwd_dx_workspace(m, n, k, r), dtype=torch.uint8, device="cuda")
    eager = slim.bwd_dx(dy, pb, dL, dR, ws=ws).clone()
    out = torch.empty_like(eager)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        slim.bwd_dx(dy, pb, dL, dR, out=out, ws=ws)
    for rep in range(3):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {rep} differs"
