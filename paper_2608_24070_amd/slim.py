"""ctypes binding of libslim (``include/slim.h``): argument marshalling only.

Every computation runs in the HIP kernels of ``libslim.so``; this module only turns torch
tensors into device pointers, sizes and the current HIP stream. There is no fallback: if the
library is missing, loading it raises.

Low-level functions carry the C names (``slim_pack``, ``slim_pack_bwd``, ``slim_linear``,
``slim_linear_bwd_dx``, ...) and take raw integers. The tensor-level helpers ``pack``,
``pack_bwd``, ``linear`` and ``bwd_dx`` allocate outputs and a cached workspace with torch.
"""
from __future__ import annotations

import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libslim.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "slim.h")

# slim_status and slim_dtype of include/slim.h (a CPU test checks them against the header)
(SLIM_OK, SLIM_EINVAL, SLIM_ESHAPE, SLIM_EDTYPE, SLIM_EALIGN, SLIM_ENONFINITE, SLIM_EWORKSPACE, SLIM_EDEVICE,
 SLIM_EUNSUPPORTED, SLIM_ERANGE) = range(10)
SLIM_F16, SLIM_BF16, SLIM_F32 = 0, 1, 2

_c_i64 = ctypes.c_int64
_c_p = ctypes.c_void_p
_SIGS = {
    "slim_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "slim_abi_version": (ctypes.c_int, []),
    "slim_pack": (ctypes.c_int, [_c_p, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "slim_pack_bwd": (ctypes.c_int, [_c_p, _c_p, _c_p, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "slim_pack_adapter": (ctypes.c_int, [_c_p, _c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p]),
    "slim_linear_workspace": (ctypes.c_int, [_c_i64, _c_i64, _c_i64, _c_i64, ctypes.POINTER(ctypes.c_size_t)]),
    "slim_bwd_dx_workspace": (ctypes.c_int, [_c_i64, _c_i64, _c_i64, _c_i64, ctypes.POINTER(ctypes.c_size_t)]),
    "slim_workspace_init": (ctypes.c_int, [_c_p, ctypes.c_size_t, _c_p]),
    "slim_linear": (ctypes.c_int, [_c_p, ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i64,
                                   _c_p, _c_p, ctypes.c_size_t, _c_p]),
    "slim_linear_bwd_dx": (ctypes.c_int, [_c_p, ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p, _c_p,
                                          _c_i64, _c_p, _c_p, ctypes.c_size_t, _c_p]),
    "slim_pack_adapter_q": (ctypes.c_int, [_c_p, _c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "slim_linear_qa_workspace": (ctypes.c_int, [_c_i64, _c_i64, _c_i64, _c_i64, ctypes.POINTER(ctypes.c_size_t)]),
    "slim_linear_qa": (ctypes.c_int, [_c_p, ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p,
                                      _c_p, _c_i64, _c_p, _c_p, ctypes.c_size_t, _c_p]),
    "slim_linear_noalloc": (ctypes.c_int, [_c_p, ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p, _c_p,
                                           _c_i64, _c_p, _c_p]),
    "slim_pack16": (ctypes.c_int, [_c_p, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p]),
    "slim_pack16_t": (ctypes.c_int, [_c_p, _c_p, _c_i64, _c_i64, _c_p, _c_p, _c_p]),
    "slim_grad_w": (ctypes.c_int, [_c_p, _c_p, ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p]),
    "slim_sparse_add": (ctypes.c_int, [_c_p, _c_p, ctypes.c_float, ctypes.c_float, _c_p, _c_i64, _c_p]),
    "slim_update_pack16": (ctypes.c_int, [_c_p, _c_i64, _c_p, _c_p]),
    "slim_quant_bins": (ctypes.c_int, [_c_i64, _c_i64]),
    "slim_quant_search": (ctypes.c_int, [_c_p, _c_i64, ctypes.c_int, _c_i64, _c_p, _c_p, _c_p]),
    "slim_pack_alpha": (ctypes.c_int, [_c_p, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "slim_hybrid_layout": (ctypes.c_int, [_c_p, _c_i64, _c_i64, _c_p, ctypes.POINTER(ctypes.c_size_t)]),
    "slim_pack_hybrid": (ctypes.c_int, [_c_p, _c_i64, _c_i64, _c_p, _c_p, _c_p, ctypes.c_size_t, _c_p]),
    "slim_linear_hybrid_workspace": (ctypes.c_int, [_c_i64, _c_i64, _c_i64, ctypes.POINTER(ctypes.c_size_t)]),
    "slim_linear_hybrid": (ctypes.c_int, [_c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_p, ctypes.c_size_t, _c_p, _c_p,
                                          ctypes.c_size_t, _c_p]),
    "slim_lora_workspace": (ctypes.c_int, [_c_i64, _c_i64, _c_i64, _c_i64, ctypes.POINTER(ctypes.c_size_t)]),
    "slim_lora": (ctypes.c_int, [_c_p, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p, ctypes.c_int, _c_i64, _c_i64, _c_p,
                                 _c_p, _c_p, ctypes.POINTER(ctypes.c_int), _c_p, ctypes.c_size_t, _c_p]),
    "slim_timing_enable": (ctypes.c_int, [ctypes.c_int]),
    "slim_timing_reset": (ctypes.c_int, []),
    "slim_timing_read": (ctypes.c_int, [ctypes.c_char_p, ctypes.c_size_t]),
}

_lib = None


class SlimError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)}")


def lib():
    """The loaded libslim.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2608_24070_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def header_symbols() -> list[str]:
    """Entry points declared in include/slim.h."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(slim_\w+)\s*\(", text, flags=re.M)))


def status_string(status: int) -> str:
    return lib().slim_status_string(status).decode()


def _check(status: int, where: str):
    if status != SLIM_OK:
        raise SlimError(status, where)


# ------------------------------------------------------------------ raw C entry points

def slim_abi_version() -> int:
    return lib().slim_abi_version()


def slim_status_string(status: int) -> str:
    return status_string(status)


def slim_pack(W, N, K, codes, meta, scales, mask, stream) -> int:
    return lib().slim_pack(W, N, K, codes, meta, scales, mask, stream)


def slim_quant_bins(N, K) -> int:
    return lib().slim_quant_bins(N, K)


def slim_quant_search(W, count, bits, bins, hist, out, stream) -> int:
    return lib().slim_quant_search(W, count, bits, bins, hist, out, stream)


def slim_pack_alpha(W, N, K, alpha, codes, meta, scales, mask, stream) -> int:
    return lib().slim_pack_alpha(W, N, K, alpha, codes, meta, scales, mask, stream)


def slim_hybrid_layout(kinds, N, K, tile_info, payload_bytes) -> int:
    return lib().slim_hybrid_layout(kinds, N, K, tile_info, payload_bytes)


def slim_pack_hybrid(W, N, K, kinds, tile_info, payload, payload_bytes, stream) -> int:
    return lib().slim_pack_hybrid(W, N, K, kinds, tile_info, payload, payload_bytes, stream)


def slim_linear_hybrid_workspace(M, N, K) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().slim_linear_hybrid_workspace(M, N, K, ctypes.byref(out)), "slim_linear_hybrid_workspace")
    return out.value


def slim_linear_hybrid(X, M, N, K, tile_info, payload, payload_bytes, Y, ws, ws_bytes, stream) -> int:
    return lib().slim_linear_hybrid(X, M, N, K, tile_info, payload, payload_bytes, Y, ws, ws_bytes, stream)


def slim_lora_workspace(N, K, B, r) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().slim_lora_workspace(N, K, B, r, ctypes.byref(out)), "slim_lora_workspace")
    return out.value


def slim_lora(W, N, K, codes, meta, scales, X, xdtype, B, r, L, R, sigma, sweeps, ws, ws_bytes, stream) -> int:
    return lib().slim_lora(W, N, K, codes, meta, scales, X, xdtype, B, r, L, R, sigma, sweeps, ws, ws_bytes, stream)


def slim_pack_bwd(codes, meta, scales, N, K, codesT, metaT, scalesT, mask_rc, stream) -> int:
    return lib().slim_pack_bwd(codes, meta, scales, N, K, codesT, metaT, scalesT, mask_rc, stream)


def slim_pack_adapter(L, R, K, N, r, Lt, Rt, stream) -> int:
    return lib().slim_pack_adapter(L, R, K, N, r, Lt, Rt, stream)


def slim_linear_workspace(M, N, K, r) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().slim_linear_workspace(M, N, K, r, ctypes.byref(out)), "slim_linear_workspace")
    return out.value


def slim_bwd_dx_workspace(M, N, K, r) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().slim_bwd_dx_workspace(M, N, K, r, ctypes.byref(out)), "slim_bwd_dx_workspace")
    return out.value


def slim_workspace_init(ws, nbytes, stream) -> int:
    return lib().slim_workspace_init(ws, nbytes, stream)


def slim_linear(X, xdtype, M, N, K, codes, meta, scales, Lt, Rt, r, Y, ws, ws_bytes, stream) -> int:
    return lib().slim_linear(X, xdtype, M, N, K, codes, meta, scales, Lt, Rt, r, Y, ws, ws_bytes, stream)


def slim_pack_adapter_q(L, R, K, N, r, Lq, Ls, Rq, Rs, stream) -> int:
    return lib().slim_pack_adapter_q(L, R, K, N, r, Lq, Ls, Rq, Rs, stream)


def slim_linear_qa_workspace(M, N, K, r) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().slim_linear_qa_workspace(M, N, K, r, ctypes.byref(out)), "slim_linear_qa_workspace")
    return out.value


def slim_linear_qa(X, xdtype, M, N, K, codes, meta, scales, Lq, Ls, Rq, Rs, r, Y, ws, ws_bytes, stream) -> int:
    return lib().slim_linear_qa(X, xdtype, M, N, K, codes, meta, scales, Lq, Ls, Rq, Rs, r, Y, ws, ws_bytes, stream)


def slim_linear_noalloc(X, xdtype, M, N, K, codes, meta, scales, Lt, Rt, r, Y, stream) -> int:
    return lib().slim_linear_noalloc(X, xdtype, M, N, K, codes, meta, scales, Lt, Rt, r, Y, stream)


SLIM_NOALLOC_SCRATCH_BYTES = 64 << 20


def slim_linear_bwd_dx(dY, dydtype, M, N, K, codesT, metaT, scalesT, L, R, r, dX, ws, ws_bytes, stream) -> int:
    return lib().slim_linear_bwd_dx(dY, dydtype, M, N, K, codesT, metaT, scalesT, L, R, r, dX, ws, ws_bytes, stream)


def slim_pack16(W, N, K, vals, meta, mask, stream) -> int:
    return lib().slim_pack16(W, N, K, vals, meta, mask, stream)


def slim_pack16_t(vals, meta, N, K, valsT, metaT, stream) -> int:
    return lib().slim_pack16_t(vals, meta, N, K, valsT, metaT, stream)


def slim_grad_w(dY, X, dtype, M, N, K, meta, gW, stream) -> int:
    return lib().slim_grad_w(dY, X, dtype, M, N, K, meta, gW, stream)


def slim_sparse_add(A, B, beta, gamma, out, count, stream) -> int:
    return lib().slim_sparse_add(A, B, beta, gamma, out, count, stream)


def slim_update_pack16(Wnew, count, vals, stream) -> int:
    return lib().slim_update_pack16(Wnew, count, vals, stream)


def slim_timing_enable(on: bool) -> int:
    return lib().slim_timing_enable(1 if on else 0)


def slim_timing_reset() -> int:
    return lib().slim_timing_reset()


def slim_timing_read() -> dict:
    """{kernel name: (launches, total_ms, median_ms)} since the last reset (waits for recorded events)."""
    need = lib().slim_timing_read(None, 0)
    buf = ctypes.create_string_buffer(max(need, 1) + 256)
    lib().slim_timing_read(buf, len(buf))
    out = {}
    for line in buf.value.decode().splitlines():
        name, n, ms, med = line.split()
        out[name] = (int(n), float(ms), float(med))
    return out


# ------------------------------------------------------------------ tensor helpers

def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return SLIM_BF16
    if t.dtype == torch.float16:
        return SLIM_F16
    raise TypeError(f"activations must be bf16 or fp16, got {t.dtype}")


def _on_gpu(*ts):
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError("tensors must be contiguous and on the GPU")


_ws_cache: dict = {}


def workspace(nbytes: int, device=None, stream=None):
    """A zero-initialised workspace of at least nbytes, cached per (device, stream)."""
    torch = _torch()
    dev = torch.device(device if device is not None else "cuda")
    key = (dev, _stream(stream))
    ws = _ws_cache.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.zeros(max(nbytes, 1 << 16), dtype=torch.uint8, device=dev)
        _ws_cache[key] = ws
    return ws


def pack(W, with_mask: bool = False, stream=None) -> dict:
    """slim_pack of an fp32 [N, K] weight. Returns codes, meta, scales (and mask)."""
    torch = _torch()
    _on_gpu(W)
    if W.dtype != torch.float32:
        raise TypeError("W must be fp32")
    N, K = W.shape
    dev = W.device
    if N % 16 or K % 128:
        raise ValueError("slim_pack needs N % 16 == 0 and K % 128 == 0")
    # rows in blocks of 16, the reduction in chunks of 128: [N/16, K/128, 16 rows, bytes per row]
    out = {
        "codes": torch.empty((N // 16, K // 128, 16, 32), dtype=torch.uint8, device=dev),
        "meta": torch.empty((N // 16, K // 128, 16, 16), dtype=torch.uint8, device=dev),
        "scales": torch.empty((N // 16, K // 128, 16), dtype=torch.int16, device=dev),
        "N": N, "K": K,
    }
    mask = torch.empty((N, K), dtype=torch.uint8, device=dev) if with_mask else None
    st = slim_pack(_ptr(W), N, K, _ptr(out["codes"]), _ptr(out["meta"]), _ptr(out["scales"]), _ptr(mask),
                   _stream(stream))
    _check(st, "slim_pack")
    if with_mask:
        out["mask"] = mask
    return out


QUANT_OUT_LEN = 4 + 2 * 30     # alpha*, E(alpha*), max|w|, candidate count, then (alpha_i, E_i) pairs


def quant_search(W, bits: int = 4, bins: int | None = None, stream=None) -> dict:
    """slim_quant_search of an fp32 tensor (SLiM-Quant). Returns {"alpha", "error", "amax", "table"
    [(alpha_i, E_i)], "hist" int32 [bins] (uint32 counts), "out" float64 device [64]}; alpha* stays
    on the device in out[0] for slim_pack_alpha."""
    torch = _torch()
    _on_gpu(W)
    if W.dtype != torch.float32 or not W.is_contiguous():
        raise TypeError("W must be a contiguous fp32 tensor")
    if bins is None:
        n, k = W.shape
        bins = slim_quant_bins(n, k)
    hist = torch.empty(bins, dtype=torch.int32, device=W.device)
    out = torch.zeros(QUANT_OUT_LEN, dtype=torch.float64, device=W.device)
    _check(slim_quant_search(_ptr(W), W.numel(), bits, bins, _ptr(hist), _ptr(out), _stream(stream)),
           "slim_quant_search")
    o = out.cpu().tolist()
    c = int(o[3])
    return {"alpha": o[0], "error": o[1], "amax": o[2], "bins": bins, "hist": hist, "out": out,
            "table": [(o[4 + 2 * i], o[5 + 2 * i]) for i in range(c)]}


def pack_alpha(W, alpha, with_mask: bool = False, stream=None) -> dict:
    """slim_pack_alpha: slim_pack with SLiM-Quant's per-tensor alpha (a device float64 tensor whose
    first element is alpha, e.g. quant_search(...)["out"]) in place of each group's absmax."""
    torch = _torch()
    _on_gpu(W)
    if W.dtype != torch.float32:
        raise TypeError("W must be fp32")
    if alpha.dtype != torch.float64 or alpha.device != W.device:
        raise TypeError("alpha must be a float64 tensor on W's device")
    N, K = W.shape
    dev = W.device
    out = {
        "codes": torch.empty((N // 16, K // 128, 16, 32), dtype=torch.uint8, device=dev),
        "meta": torch.empty((N // 16, K // 128, 16, 16), dtype=torch.uint8, device=dev),
        "scales": torch.empty((N // 16, K // 128, 16), dtype=torch.int16, device=dev),
        "N": N, "K": K,
    }
    mask = torch.empty((N, K), dtype=torch.uint8, device=dev) if with_mask else None
    _check(slim_pack_alpha(_ptr(W), N, K, _ptr(alpha), _ptr(out["codes"]), _ptr(out["meta"]), _ptr(out["scales"]),
                           _ptr(mask), _stream(stream)), "slim_pack_alpha")
    if with_mask:
        out["mask"] = mask
    return out


def pack_hybrid(W, kinds, stream=None) -> dict:
    """slim_pack_hybrid: fp32 W [N, K] (device) with a tile map (numpy uint8 [N/128, K/128], 1 = 2:4
    sparse) -> {"tile_info" int64 [N/128, K/128] (uint64 words), "payload" uint8, "N", "K"}."""
    import numpy as np
    torch = _torch()
    _on_gpu(W)
    if W.dtype != torch.float32:
        raise TypeError("W must be fp32")
    N, K = W.shape
    kinds = np.ascontiguousarray(np.asarray(kinds, dtype=np.uint8))
    if kinds.shape != (N // 128, K // 128):
        raise ValueError("the tile map must be [N/128, K/128]")
    nbytes = ctypes.c_size_t(0)
    kp = kinds.ctypes.data_as(ctypes.c_void_p)
    _check(slim_hybrid_layout(kp, N, K, None, ctypes.byref(nbytes)), "slim_hybrid_layout")
    info = torch.empty((N // 128, K // 128), dtype=torch.int64, device=W.device)
    payload = torch.empty(max(nbytes.value, 16), dtype=torch.uint8, device=W.device)
    _check(slim_pack_hybrid(_ptr(W), N, K, kp, _ptr(info), _ptr(payload), nbytes.value, _stream(stream)),
           "slim_pack_hybrid")
    return {"tile_info": info, "payload": payload, "N": N, "K": K}


_hybrid_ws: dict = {}


def linear_hybrid(X, p: dict, out=None, stream=None):
    """slim_linear_hybrid: Y fp32 [M, N] = X Wp^T for fp16 X [M, K] and a hybrid pack."""
    torch = _torch()
    _on_gpu(X)
    if X.dtype != torch.float16:
        raise TypeError("X must be fp16")
    M, K = X.shape
    N = p["N"]
    if K != p["K"]:
        raise ValueError("X width does not match the pack")
    Y = out if out is not None else torch.empty((M, N), dtype=torch.float32, device=X.device)
    nb = slim_linear_hybrid_workspace(M, N, K)
    ws = None
    if nb:
        # its own cache: the split partials must not land in slim_linear's workspace, whose counter
        # region has to stay zero between calls
        key = (X.device, _stream(stream))
        ws = _hybrid_ws.get(key)
        if ws is None or ws.numel() < nb:
            ws = torch.empty(nb, dtype=torch.uint8, device=X.device)
            _hybrid_ws[key] = ws
    _check(slim_linear_hybrid(_ptr(X), M, N, K, _ptr(p["tile_info"]), _ptr(p["payload"]), p["payload"].numel(),
                              _ptr(Y), _ptr(ws), nb, _stream(stream)), "slim_linear_hybrid")
    return Y


def lora(W, packed: dict, X, r: int, stream=None) -> dict:
    """slim_lora (SLiM-LoRA): adapters L fp32 [K, r], R fp32 [r, N] with W ~ W^C + (L R)^T from the
    uncompressed weight W fp32 [N, K], its forward pack and calibration activations X [B, K]
    (bf16/fp16). Returns {"L", "R", "sigma" float64 [r], "sweeps"}."""
    torch = _torch()
    _on_gpu(W)
    _on_gpu(X)
    if W.dtype != torch.float32:
        raise TypeError("W must be fp32")
    N, K = W.shape
    B = X.shape[0]
    if X.shape[1] != K:
        raise ValueError("X must be [B, K]")
    nbytes = slim_lora_workspace(N, K, B, r)
    dev = W.device
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    L = torch.empty((K, r), dtype=torch.float32, device=dev)
    R = torch.empty((r, N), dtype=torch.float32, device=dev)
    sigma = torch.empty(max(r, 1), dtype=torch.float64, device=dev)
    sweeps = ctypes.c_int(0)
    _check(slim_lora(_ptr(W), N, K, _ptr(packed["codes"]), _ptr(packed["meta"]), _ptr(packed["scales"]), _ptr(X),
                     _dtype_code(X), B, r, _ptr(L), _ptr(R), _ptr(sigma), ctypes.byref(sweeps), _ptr(ws), nbytes,
                     _stream(stream)), "slim_lora")
    return {"L": L, "R": R, "sigma": sigma[:r], "sweeps": sweeps.value}


def pack_bwd(packed: dict, with_mask: bool = False, stream=None) -> dict:
    """slim_pack_bwd of a forward pack. Returns codesT, metaT, scalesT (and mask_rc)."""
    torch = _torch()
    N, K = packed["N"], packed["K"]
    dev = packed["codes"].device
    if N % 128:
        raise ValueError("slim_pack_bwd needs N % 128 == 0")
    # rows (k) in blocks of 16, the reduction (n) in chunks of 128; scalesT stays [K/128, N]
    out = {
        "codesT": torch.empty((K // 16, N // 128, 16, 32), dtype=torch.uint8, device=dev),
        "metaT": torch.empty((K // 16, N // 128, 16, 16), dtype=torch.uint8, device=dev),
        "scalesT": torch.empty((K // 128, N), dtype=torch.int16, device=dev),
        "N": N, "K": K,
    }
    mask = torch.empty((N, K), dtype=torch.uint8, device=dev) if with_mask else None
    st = slim_pack_bwd(_ptr(packed["codes"]), _ptr(packed["meta"]), _ptr(packed["scales"]), N, K,
                       _ptr(out["codesT"]), _ptr(out["metaT"]), _ptr(out["scalesT"]), _ptr(mask), _stream(stream))
    _check(st, "slim_pack_bwd")
    if with_mask:
        out["mask_rc"] = mask
    return out


def pack_adapter(L, R, stream=None) -> dict:
    """slim_pack_adapter of fp16 L [K, r] and R [r, N]: returns {"Lt", "Rt", "L", "R"} (the forward
    takes Lt, Rt; the backward takes L, R). Lt is L^T [r, K]; Rt is R^T in 32 x 16 tiles,
    [ceil(N/32), r/16, 32, 16]."""
    torch = _torch()
    _on_gpu(L, R)
    K, r = L.shape
    N = R.shape[1]
    out = {"Lt": torch.empty((r, K), dtype=torch.float16, device=L.device),
           "Rt": torch.empty(((N + 31) // 32, r // 16, 32, 16), dtype=torch.float16, device=L.device),
           "L": L, "R": R}
    _check(slim_pack_adapter(_ptr(L), _ptr(R), K, N, r, _ptr(out["Lt"]), _ptr(out["Rt"]), _stream(stream)),
           "slim_pack_adapter")
    return out


def linear(X, packed: dict, adapter: dict | None = None, out=None, ws=None, stream=None):
    """Y = X Wc^T + (X L) R through slim_linear. X bf16/fp16 [M, K]; adapter from pack_adapter (or None);
    Y fp32 [M, N]."""
    torch = _torch()
    Lt = None if adapter is None else adapter["Lt"]
    Rt = None if adapter is None else adapter["Rt"]
    _on_gpu(X, Lt, Rt, out)
    M, K = X.shape
    N = packed["N"]
    r = 0 if Lt is None else Lt.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=X.device)
    need = slim_linear_workspace(M, N, K, r)
    if ws is None:
        ws = workspace(need, X.device, stream)
    st = slim_linear(_ptr(X), _dtype_code(X), M, N, K, _ptr(packed["codes"]), _ptr(packed["meta"]),
                     _ptr(packed["scales"]), _ptr(Lt), _ptr(Rt), r, _ptr(out), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "slim_linear")
    return out


def bwd_dx(dY, packed_bwd: dict, L=None, R=None, out=None, ws=None, stream=None):
    """dX = dY W^{R,C} + (dY R^T) L^T through slim_linear_bwd_dx. dX fp32 [M, K]."""
    torch = _torch()
    _on_gpu(dY, L, R, out)
    M, N = dY.shape
    K = packed_bwd["K"]
    r = 0 if L is None else L.shape[1]
    if out is None:
        out = torch.empty((M, K), dtype=torch.float32, device=dY.device)
    need = slim_bwd_dx_workspace(M, N, K, r)
    if ws is None:
        ws = workspace(need, dY.device, stream)
    st = slim_linear_bwd_dx(_ptr(dY), _dtype_code(dY), M, N, K, _ptr(packed_bwd["codesT"]),
                            _ptr(packed_bwd["metaT"]), _ptr(packed_bwd["scalesT"]), _ptr(L), _ptr(R), r,
                            _ptr(out), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "slim_linear_bwd_dx")
    return out


def linear_noalloc(X, packed: dict, adapter: dict | None = None, out=None, stream=None):
    """Y = X Wc^T + (X L) R through slim_linear_noalloc (the library's own per-device scratch; no
    workspace). Only `out` is allocated here when not given."""
    torch = _torch()
    Lt = None if adapter is None else adapter["Lt"]
    Rt = None if adapter is None else adapter["Rt"]
    _on_gpu(X, Lt, Rt, out)
    M, K = X.shape
    N = packed["N"]
    r = 0 if Lt is None else Lt.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=X.device)
    st = slim_linear_noalloc(_ptr(X), _dtype_code(X), M, N, K, _ptr(packed["codes"]), _ptr(packed["meta"]),
                             _ptr(packed["scales"]), _ptr(Lt), _ptr(Rt), r, _ptr(out), _stream(stream))
    _check(st, "slim_linear_noalloc")
    return out


def pack_adapter_q(L, R, stream=None) -> dict:
    """slim_pack_adapter_q of fp16 L [K, r] and R [r, N]: {"Lq", "Ls", "Rq", "Rs", "K", "N", "r"}."""
    torch = _torch()
    _on_gpu(L, R)
    K, r = L.shape
    N = R.shape[1]
    dev = L.device
    out = {"Lq": torch.empty((r, K // 2), dtype=torch.uint8, device=dev),
           "Ls": torch.empty((r, (K + 127) // 128), dtype=torch.int16, device=dev),
           "Rq": torch.empty((N, r // 2), dtype=torch.uint8, device=dev),
           "Rs": torch.empty((N, (r + 127) // 128), dtype=torch.int16, device=dev),
           "K": K, "N": N, "r": r}
    _check(slim_pack_adapter_q(_ptr(L), _ptr(R), K, N, r, _ptr(out["Lq"]), _ptr(out["Ls"]), _ptr(out["Rq"]),
                               _ptr(out["Rs"]), _stream(stream)), "slim_pack_adapter_q")
    return out


def linear_qa(X, packed: dict, qadapter: dict, out=None, ws=None, stream=None):
    """Y = X Wc^T + (X L^Q) R^Q through slim_linear_qa (qadapter from pack_adapter_q). Y fp32 [M, N]."""
    torch = _torch()
    _on_gpu(X, out)
    M, K = X.shape
    N, r = packed["N"], qadapter["r"]
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=X.device)
    need = slim_linear_qa_workspace(M, N, K, r)
    if ws is None:
        ws = workspace(need, X.device, stream)
    st = slim_linear_qa(_ptr(X), _dtype_code(X), M, N, K, _ptr(packed["codes"]), _ptr(packed["meta"]),
                        _ptr(packed["scales"]), _ptr(qadapter["Lq"]), _ptr(qadapter["Ls"]), _ptr(qadapter["Rq"]),
                        _ptr(qadapter["Rs"]), r, _ptr(out), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "slim_linear_qa")
    return out


# ------------------------------------------------- training step (value packs, SLoPe)

def pack16(W, with_mask: bool = False, stream=None) -> dict:
    """slim_pack16 of fp32 W [N, K]: {"vals" int16 [N, K/2] (fp16 bits), "meta" uint8 [N, K/8], "N", "K"}
    (+ "mask" uint8 [N, K])."""
    torch = _torch()
    _on_gpu(W)
    N, K = W.shape
    dev = W.device
    out = {"vals": torch.empty((N, K // 2), dtype=torch.int16, device=dev),
           "meta": torch.empty((N, K // 8), dtype=torch.uint8, device=dev), "N": N, "K": K}
    mask = torch.empty((N, K), dtype=torch.uint8, device=dev) if with_mask else None
    _check(slim_pack16(_ptr(W), N, K, _ptr(out["vals"]), _ptr(out["meta"]), _ptr(mask), _stream(stream)),
           "slim_pack16")
    if with_mask:
        out["mask"] = mask
    return out


def pack16_t(p: dict, out: dict | None = None, stream=None) -> dict:
    """slim_pack16_t of a value pack: {"valsT" int16 [K, N/2], "metaT" uint8 [K, N/8]} (into `out` if given)."""
    torch = _torch()
    N, K = p["N"], p["K"]
    dev = p["vals"].device
    if out is None:
        out = {"valsT": torch.empty((K, N // 2), dtype=torch.int16, device=dev),
               "metaT": torch.empty((K, N // 8), dtype=torch.uint8, device=dev)}
    _check(slim_pack16_t(_ptr(p["vals"]), _ptr(p["meta"]), N, K, _ptr(out["valsT"]), _ptr(out["metaT"]),
                         _stream(stream)), "slim_pack16_t")
    return out


def grad_w(dY, X, p: dict, out=None, stream=None):
    """slim_grad_w: fp32 [N, K/2] = (dY^T X) at the kept positions of the value pack `p` (dY [M, N], X [M, K])."""
    torch = _torch()
    _on_gpu(dY, X, out)
    M, N = dY.shape
    K = X.shape[1]
    if dY.dtype != X.dtype:
        raise ValueError("dY and X must have one dtype")
    if out is None:
        out = torch.empty((N, K // 2), dtype=torch.float32, device=dY.device)
    _check(slim_grad_w(_ptr(dY), _ptr(X), _dtype_code(dY), M, N, K, _ptr(p["meta"]), _ptr(out), _stream(stream)),
           "slim_grad_w")
    return out


def sparse_add(A, B, beta: float, gamma: float, out=None, stream=None):
    """slim_sparse_add: beta A + gamma B (A fp32, B fp16 bits as int16 or float16), same shape."""
    torch = _torch()
    _on_gpu(A, B, out)
    if out is None:
        out = torch.empty_like(A)
    _check(slim_sparse_add(_ptr(A), _ptr(B), float(beta), float(gamma), _ptr(out), A.numel(), _stream(stream)),
           "slim_sparse_add")
    return out


def update_pack16(Wnew, p: dict, stream=None) -> dict:
    """slim_update_pack16: new fp32 values [N, K/2] into p["vals"] (in place); returns p."""
    _on_gpu(Wnew)
    _check(slim_update_pack16(_ptr(Wnew), Wnew.numel(), _ptr(p["vals"]), _stream(stream)), "slim_update_pack16")
    return p
