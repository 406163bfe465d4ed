"""slim_linear_noalloc (the entry point that allocates nothing; its workspace is the library's own
per-device scratch array) gives bit for bit what slim_linear gives on a caller workspace, on
consecutive calls whose sizes shrink, on both the small-M and the large-M path."""
import numpy as np
import pytest
import torch

from oracle import slim_oracle as O
from paper_2608_24070_amd import slim, synth
from tests.gpu_common import assert_close, dev, host, layer_inputs

pytestmark = pytest.mark.gpu


def _pair(n, k, r, m, xdtype="bf16", name="noalloc", check_oracle=True):
    print(f"noalloc n={n} k={k} r={r} m={m} {xdtype}", flush=True)
    W, X, L, R, dx, ad = layer_inputs(n, k, r, m, xdtype=xdtype, name=name)
    p = slim.pack(dev(W))
    y_ref = slim.linear(dx, p, ad).clone()
    y = slim.linear_noalloc(dx, p, ad)
    torch.cuda.synchronize()
    assert torch.equal(y, y_ref), f"noalloc differs from slim_linear: n={n} k={k} r={r} m={m}"
    if check_oracle:
        rows = np.sort(synth.stream(1, "nar").choice(n, size=min(n, 256), replace=False))
        ms = np.arange(m) if m <= 32 else np.sort(synth.stream(1, "nam").choice(m, size=16, replace=False))
        ref = O.linear(X[ms], O.pack(W[rows]), L, None if R is None else R[:, rows], len(rows), k)
        assert_close(host(y)[np.ix_(ms, rows)], ref, "noalloc vs oracle")


def test_noalloc_small_m_twice_second_smaller():
    _pair(4096, 4096, 384, 16)
    _pair(1024, 2048, 32, 5)


def test_noalloc_large_m_twice_second_smaller():
    _pair(11008, 4096, 384, 2048)
    _pair(1024, 1024, 64, 200, xdtype="fp16")


def test_noalloc_after_other_sizes_and_without_adapter():
    # the shared counters return to zero after every call, so any order of sizes works
    _pair(28672, 8192, 512, 16, check_oracle=False)
    _pair(512, 512, 0, 3)
    _pair(4096, 4096, 384, 1)


def test_noalloc_refuses_oversize_on_device():
    W, X, L, R, dx, ad = layer_inputs(5120, 5120, 512, 8, name="noalloc_big")
    p = slim.pack(dev(W))
    x_big = torch.zeros((4096, 5120), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(slim.SlimError) as e:
        slim.linear_noalloc(x_big, p, ad)
    assert e.value.status == slim.SLIM_EWORKSPACE
