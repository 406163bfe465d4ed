"""Helpers shared by the GPU parity tests (inputs from ``synth``, expected values from ``oracle``)."""
import numpy as np
import torch

from oracle import slim_oracle as O
from paper_2608_24070_amd import slim, synth

TOL_REL_FRO = 2e-3       # relative Frobenius error gate
TOL_MAX_ABS = 1e-2       # max |error| gate, as a fraction of max |Y_ref|


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def dev_bits(bits, dtype):
    """uint16 bit patterns -> a bf16/fp16 device tensor."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(dtype)


def host(t):
    return t.detach().cpu().numpy()


# The device pack keeps rows in blocks of 16 and the reduction in chunks of 128 (codes, meta and
# scales of the forward pack, codesT and metaT of the backward pack): [rows/16, chunks, 16, bytes]
# for 32 code bytes or 16 index bytes per row and chunk, [rows/16, chunks, 16] for the scales.
# The oracle keeps each row whole, [rows, chunks * bytes]. These two permutations convert.
BLOCKED = ("codes", "meta", "scales", "codesT", "metaT")


def unblock(a):
    """Device (blocked) layout -> the oracle's row-major layout."""
    if a.ndim == 4:
        r16, nch, r, b = a.shape
        return np.ascontiguousarray(a.transpose(0, 2, 1, 3)).reshape(r16 * r, nch * b)
    r16, nch, r = a.shape
    return np.ascontiguousarray(a.transpose(0, 2, 1)).reshape(r16 * r, nch)


def block(a, chunk_bytes):
    """The oracle's row-major layout -> device layout; chunk_bytes per row and chunk (32 codes,
    16 index words, 0 for scales, one element per chunk)."""
    rows = a.shape[0]
    if chunk_bytes == 0:
        return np.ascontiguousarray(a.reshape(rows // 16, 16, -1).transpose(0, 2, 1))
    return np.ascontiguousarray(a.reshape(rows // 16, 16, -1, chunk_bytes).transpose(0, 2, 1, 3))


def host_pack(p):
    """Device pack -> numpy arrays in the oracle's dtypes and row-major layout."""
    out = {}
    for k, v in p.items():
        if isinstance(v, torch.Tensor):
            a = host(v)
            a = a.view(np.uint16) if a.dtype == np.int16 else a
            out[k] = unblock(a) if k in BLOCKED else a
        else:
            out[k] = v
    return out


def oracle_pack_on_device(p, n, k):
    """Upload an oracle pack, so the layer kernels can be checked on a pack the GPU did not make."""
    return {"codes": dev(block(p["codes"], 32)), "meta": dev(block(p["meta"], 16)),
            "scales": dev(block(p["scales"], 0).view(np.int16)), "N": n, "K": k}


def layer_inputs(n, k, r, m, seed=0, xdtype="bf16", outliers=False, name="layer", xscale=1.0):
    W = synth.weights(n, k, seed=seed, name=name + "/W")
    xbits, X = synth.activations(m, k, seed=seed, name=name + "/X", dtype=xdtype, outliers=outliers, scale=xscale)
    Lb, Rb, L, R = synth.adapter(k, n, max(r, 16), seed=seed, name=name + "/")
    if r == 0:
        Lb = Rb = L = R = None
    else:
        Lb, Rb, L, R = Lb[:, :r].copy(), Rb[:r].copy(), L[:, :r], R[:r]
    tdt = torch.bfloat16 if xdtype == "bf16" else torch.float16
    dx = dev_bits(xbits, tdt)
    ad = None if Lb is None else slim.pack_adapter(dev_bits(Lb, torch.float16), dev_bits(Rb, torch.float16))
    return W, X, L, R, dx, ad


def assert_close(Y, Yref, what=""):
    ok, rf, ma = O.within_tolerance(Y, Yref, TOL_REL_FRO, TOL_MAX_ABS)
    assert np.all(np.isfinite(Y)), f"{what}: non-finite output"
    assert ok, f"{what}: rel_fro={rf:.3e} (gate {TOL_REL_FRO}), max_abs/inf={ma:.3e} (gate {TOL_MAX_ABS})"
    return rf, ma
