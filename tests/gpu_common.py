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


def host_pack(p):
    """Device pack -> numpy arrays in the oracle's dtypes."""
    out = {}
    for k, v in p.items():
        if isinstance(v, torch.Tensor):
            a = host(v)
            out[k] = a.view(np.uint16) if a.dtype == np.int16 else a
        else:
            out[k] = v
    return out


def oracle_pack_on_device(p, n, k):
    """Upload an oracle pack, so the layer kernels can be checked on a pack the GPU did not make."""
    return {"codes": dev(p["codes"]), "meta": dev(p["meta"]), "scales": dev(p["scales"].view(np.int16)),
            "N": n, "K": k}


def layer_inputs(n, k, r, m, seed=0, xdtype="bf16", outliers=False, name="layer"):
    W = synth.weights(n, k, seed=seed, name=name + "/W")
    xbits, X = synth.activations(m, k, seed=seed, name=name + "/X", dtype=xdtype, outliers=outliers)
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
