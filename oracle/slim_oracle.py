"""Plain float64 NumPy oracle for the compressed linear layer (test infrastructure only).

What it computes, and where the thesis defines it
-------------------------------------------------
* ``mask_2of4``: keep the two largest-magnitude weights of every aligned group of
  four along the reduction dimension K. N:M sparsity has to lie along the reduction
  dimension to be accelerated (SLoPe, "Double-pruned Backward Pass"; background
  "Sparse Tensor Core Acceleration"); magnitude is the selection criterion of the
  "Magnitude" baselines.
* ``group_scales`` / ``quantize``: symmetric AbsMax quantisation (SLiM preliminaries,
  "Symmetric Quantization"; eq. symmetric_quantization), applied per group of 128
  consecutive weights of a row (group size 128, SLiM setup and "Low-rank adapter
  quantization"), with 4-bit signed codes in [-7, 7].
* ``pack`` / ``unpack``: the packed deployment format (values + 2-bit position
  indices + per-group scales). The thesis only says that 2:4 storage keeps the
  non-zeros contiguously with small index metadata ("Sparse Tensor Core
  Acceleration"; eq. index_bits); the byte layout below is this library's own.
* ``linear``: Y = X Wc^T + (X L) R, the sparse-plus-low-rank layer with the adapter
  as a parallel path (SLoPe eq. sparse_plus_low_rank; SLiM "SLiM-LoRA low-rank
  adapters", W ~ W^C + L R).
* ``pack_bwd`` / ``bwd_dx``: SLoPe's double pruning. The forward weight, already 2:4
  along K (W^R), is pruned 2:4 again along N to give W^{R,C}; the input gradient is
  dX = dY W^{R,C} (eq. sparse_backward_input). The adapter contributes
  (dY R^T) L^T because it is a parallel dense path.
* ``lemma_extra_sparsity``: the closed form of Lemma sparsity_ratio
  (eq. sparsity_ratio).
* ``pack_adapter_q`` / ``linear_qa``: the quantized adapters of SLiM-LoRA^Q (SLiM,
  "Low-rank adapter quantization"): AbsMax 4-bit group quantization with groups of
  128 elements, here along each factor's input dimension (K for L, r for R), with the
  weights' scale and rounding rules; the layer then uses the dequantized factors.

Readings where the thesis is silent, garbled or inconsistent
--------------------------------------------------------------
* Top-2 ties: key (|w| descending, position ascending); -0.0 and +0.0 are equal.
* Quantiser: eq. symmetric_quantization as printed rounds before scaling, so it
  only yields {-1, 0, 1}, and a literal 2^(q-1) = 8 overflows signed int4. The
  reading is round-to-nearest of w/s with s = absmax/7 and codes clamped to
  [-7, 7]. Ties round half to even.
* Scale: s16 = fp16_RNE(fp32(absmax) / 7.0f), using IEEE fp32 division. Codes are
  computed against the stored s16: q = clamp(rint(double(w) / double(s16)), -7, 7),
  and q = 0 when s16 == 0.
* Mask before quantisation: the mask comes from the fp32 magnitudes. The group
  maximum is always kept, so the quantised values equal those of
  quantise-then-prune (pinned in the tests).
* Code encoding: offset binary u = q + 8 (so 1..15; 0 is unused).
* Backward column prune: per column k and aligned group of four rows, keep the
  top two by key (|Wc| descending, forward-mask bit descending, n ascending).
  Entries that are not in the forward mask carry code 8 (value 0).

Packed format
-------------
All multi-byte words are little-endian.

``codes``: uint8 [N, K/4], read as uint32 words [N, K/16]. Word b of row n covers
K positions 16b .. 16b+15, which are four groups of four (c = 0..3). Bits 4c..4c+3
hold u of group c's lower kept position; bits 16+4c..16+4c+3 hold u of its higher
kept position.

``meta``: uint8 [N, K/8], read as uint16 half-words [N, K/16]. Half-word b holds,
for group c of the same 16 positions, i0 in bits 4c..4c+1 and i1 in bits
4c+2..4c+3, where i0 < i1 are the kept offsets inside the group.

``scales``: uint16 [N, K/128], the fp16 bit pattern of s16.

``mask``: uint8 [N, K], 0/1.

The backward pack uses the same code and meta format with the roles of the axes
swapped: ``codesT`` is uint8 [K, N/4] and ``metaT`` is uint8 [K, N/8], both along
n for each k. ``scalesT`` is uint16 [K/128, N], the forward scales transposed.
``mask_rc`` is uint8 [N, K], the support of W^{R,C}.

Parity pins
-----------
Every function here is pinned by a ``-m "not gpu"`` test in
``tests/test_oracle_pins.py`` against something other than itself (brute force,
closed forms, printed values, invariants). The adapter *values* L, R are synthetic
inputs: how SLiM-LoRA computes them is out of scope, so nothing here depends on
them.
"""
from __future__ import annotations

import numpy as np

GROUP = 128          # quantisation group along K
QMAX = 7             # 4-bit symmetric codes in [-7, 7]
CODE_OFFSET = 8      # u = q + 8


class OracleError(ValueError):
    """Input the packed format cannot represent (non-finite weights, scale overflow, bad shape)."""


# ----------------------------------------------------------------------------- mask

def mask_2of4(W: np.ndarray) -> np.ndarray:
    """2:4 magnitude mask along the last axis: keep the two largest |w| of each aligned 4-group.

    Ties are broken by the lower position (stable sort of -|w|). Returns uint8 0/1 of W's shape.
    """
    W = np.asarray(W)
    n, k = W.shape
    if k % 4:
        raise OracleError("reduction length must be a multiple of 4")
    a = np.abs(W.astype(np.float64)).reshape(n, k // 4, 4)
    order = np.argsort(-a, axis=2, kind="stable")
    keep = order[..., :2]
    m = np.zeros((n, k // 4, 4), dtype=np.uint8)
    np.put_along_axis(m, keep, 1, axis=2)
    return m.reshape(n, k)


# ------------------------------------------------------------------------ quantiser

def fp16_rne(x32: np.ndarray) -> np.ndarray:
    """Round float32 values to IEEE binary16, nearest with ties to even (NumPy's half conversion)."""
    with np.errstate(over="ignore"):
        return np.asarray(x32, dtype=np.float32).astype(np.float16)


def group_scales(W: np.ndarray) -> np.ndarray:
    """Per (row, 128-group) AbsMax scale s16 = fp16_RNE(fp32(max|w|) / 7.0f). Returns float16 [N, K/128]."""
    W = np.asarray(W, dtype=np.float32)
    n, k = W.shape
    if k % GROUP:
        raise OracleError("K must be a multiple of 128")
    if not np.all(np.isfinite(W)):
        raise OracleError("non-finite weight")
    a = np.abs(W).reshape(n, k // GROUP, GROUP).max(axis=2)
    s = fp16_rne(a.astype(np.float32) / np.float32(QMAX))
    if not np.all(np.isfinite(s)):
        raise OracleError("group scale overflows fp16")
    return s


def quantize(W: np.ndarray, s16: np.ndarray) -> np.ndarray:
    """Signed codes q = clamp(rint(w / s16), -7, 7) of every weight (0 where s16 == 0). int8 [N, K]."""
    W = np.asarray(W, dtype=np.float32).astype(np.float64)
    n, k = W.shape
    s = np.repeat(s16.astype(np.float64), GROUP, axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.where(s > 0, W / np.where(s > 0, s, 1.0), 0.0)
    q = np.clip(np.rint(t), -QMAX, QMAX)
    return q.astype(np.int8)


def dequant_dense(W: np.ndarray) -> np.ndarray:
    """Wc = M (.) q (.) s16 straight from the weights, as float64 [N, K] (no packing involved)."""
    m = mask_2of4(W)
    s = group_scales(W)
    q = quantize(W, s)
    return m * q.astype(np.float64) * np.repeat(s.astype(np.float64), GROUP, axis=1)


# --------------------------------------------------------------------- pack format

def _encode(u: np.ndarray, idx: np.ndarray, rows: int, length: int):
    """Encode codes u [rows, length/4, 2] and kept offsets idx [rows, length/4, 2] into (codes, meta) bytes."""
    g = length // 4
    u = u.reshape(rows, g // 4, 4, 2).astype(np.uint32)       # [row, block, c, slot]
    idx = idx.reshape(rows, g // 4, 4, 2).astype(np.uint32)
    c = np.arange(4, dtype=np.uint32)
    word = ((u[..., 0] << (4 * c)) | (u[..., 1] << (16 + 4 * c))).sum(axis=2, dtype=np.uint32)
    half = ((idx[..., 0] << (4 * c)) | (idx[..., 1] << (4 * c + 2))).sum(axis=2, dtype=np.uint32)
    codes = word.astype("<u4").view(np.uint8).reshape(rows, length // 4)
    meta = half.astype("<u2").view(np.uint8).reshape(rows, length // 8)
    return np.ascontiguousarray(codes), np.ascontiguousarray(meta)


def _decode(codes: np.ndarray, meta: np.ndarray, rows: int, length: int):
    """Inverse of ``_encode``: returns u [rows, length/4, 2] and idx [rows, length/4, 2]."""
    word = np.ascontiguousarray(codes).view("<u4").reshape(rows, length // 16).astype(np.uint32)
    half = np.ascontiguousarray(meta).view("<u2").reshape(rows, length // 16).astype(np.uint32)
    c = np.arange(4, dtype=np.uint32)
    u0 = (word[..., None] >> (4 * c)) & 0xF
    u1 = (word[..., None] >> (16 + 4 * c)) & 0xF
    i0 = (half[..., None] >> (4 * c)) & 0x3
    i1 = (half[..., None] >> (4 * c + 2)) & 0x3
    u = np.stack([u0, u1], axis=-1).reshape(rows, length // 4, 2)
    idx = np.stack([i0, i1], axis=-1).reshape(rows, length // 4, 2)
    return u, idx


def pack(W: np.ndarray) -> dict:
    """Forward pack of fp32 W [N, K]: mask, scales, int4 codes and 2-bit indices (format in the module docstring)."""
    W = np.asarray(W, dtype=np.float32)
    n, k = W.shape
    if k % GROUP or n < 1:
        raise OracleError("need N >= 1 and K a multiple of 128")
    s16 = group_scales(W)
    m = mask_2of4(W)
    q = quantize(W, s16)
    g = k // 4
    mg = m.reshape(n, g, 4)
    # kept offsets in ascending order: i0 < i1
    idx = np.sort(np.argsort(-mg.astype(np.int8), axis=2, kind="stable")[..., :2], axis=2)
    qk = np.take_along_axis(q.reshape(n, g, 4), idx, axis=2)
    u = qk.astype(np.int16) + CODE_OFFSET
    codes, meta = _encode(u, idx, n, k)
    return {
        "codes": codes,
        "meta": meta,
        "scales": s16.view(np.uint16).copy(),
        "mask": m,
    }


def unpack(codes: np.ndarray, meta: np.ndarray, scales: np.ndarray, n: int, k: int) -> np.ndarray:
    """Materialise the dense dequantised weight Wc [n, k] (float64) from a forward pack."""
    u, idx = _decode(codes, meta, n, k)
    s = np.asarray(scales, dtype=np.uint16).view(np.float16).astype(np.float64).reshape(n, k // GROUP)
    dense = np.zeros((n, k // 4, 4), dtype=np.float64)
    vals = (u.astype(np.float64) - CODE_OFFSET)
    np.put_along_axis(dense, idx.astype(np.int64), vals, axis=2)
    return dense.reshape(n, k) * np.repeat(s, GROUP, axis=1)


def pack_bytes(n: int, k: int) -> int:
    """Bytes of a forward pack: codes K/4 + meta K/8 + scales 2K/128 per row."""
    return n * (k // 4 + k // 8 + 2 * (k // GROUP))


# ------------------------------------------------------------------------- layer

def _f64(a) -> np.ndarray:
    return np.asarray(a).astype(np.float64)


def linear(X, packed: dict, L, R, n: int, k: int) -> np.ndarray:
    """Y = X Wc^T + (X L) R in float64. X [M, K]; L [K, r] and R [r, N], or None for r = 0."""
    Wc = unpack(packed["codes"], packed["meta"], packed["scales"], n, k)
    X = _f64(X)
    Y = X @ Wc.T
    if L is not None and R is not None and np.asarray(L).shape[1] > 0:
        Y = Y + (X @ _f64(L)) @ _f64(R)
    return Y


# ----------------------------------------------------------------- double pruning

def pack_bwd(packed: dict, n: int, k: int) -> dict:
    """Backward pack: prune the forward (already 2:4 along K) weight 2:4 along N as well.

    For each column k and aligned group of four rows, keep the top two by key
    (|Wc| desc, forward-mask bit desc, n asc). The kept slots carry their forward code u
    (8 for a slot the forward mask had dropped). Returns codesT/metaT along N for each k,
    scalesT [K/128, N] and mask_rc [N, K], the support of W^{R,C}.
    """
    if n % 16:
        raise OracleError("backward pack needs N a multiple of 16")
    Wc = unpack(packed["codes"], packed["meta"], packed["scales"], n, k)
    mr = np.asarray(packed["mask"], dtype=np.uint8)
    u_dense = _dense_codes(packed, n, k)                     # [N, K], 8 where not kept
    # work on the transpose: rows k, groups of four along n
    a = np.abs(Wc.T).reshape(k, n // 4, 4)
    f = mr.T.reshape(k, n // 4, 4).astype(np.int64)
    pos = np.broadcast_to(np.arange(4), a.shape)
    order = np.lexsort((pos, -f, -a), axis=-1)
    idx = np.sort(order[..., :2], axis=2)
    uT = np.take_along_axis(u_dense.T.reshape(k, n // 4, 4), idx, axis=2)
    codesT, metaT = _encode(uT, idx, k, n)
    sel = np.zeros((k, n // 4, 4), dtype=np.uint8)
    np.put_along_axis(sel, idx, 1, axis=2)
    mask_rc = (sel.reshape(k, n).T & mr).astype(np.uint8)
    scalesT = np.ascontiguousarray(np.asarray(packed["scales"], dtype=np.uint16).T)
    return {"codesT": codesT, "metaT": metaT, "scalesT": scalesT, "mask_rc": np.ascontiguousarray(mask_rc)}


def _dense_codes(packed: dict, n: int, k: int) -> np.ndarray:
    """Forward codes u placed at their dense positions; 8 (value 0) at pruned positions. uint8 [N, K]."""
    u, idx = _decode(packed["codes"], packed["meta"], n, k)
    dense = np.full((n, k // 4, 4), CODE_OFFSET, dtype=np.uint8)
    np.put_along_axis(dense, idx.astype(np.int64), u.astype(np.uint8), axis=2)
    return dense.reshape(n, k)


def unpack_bwd(codesT, metaT, scalesT, n: int, k: int) -> np.ndarray:
    """Materialise W^{R,C} [n, k] (float64) from a backward pack; the scale of (n, k) is scalesT[k/128, n]."""
    u, idx = _decode(codesT, metaT, k, n)
    dense = np.zeros((k, n // 4, 4), dtype=np.float64)
    np.put_along_axis(dense, idx.astype(np.int64), u.astype(np.float64) - CODE_OFFSET, axis=2)
    s = np.asarray(scalesT, dtype=np.uint16).view(np.float16).astype(np.float64).reshape(k // GROUP, n)
    return dense.reshape(k, n).T * np.repeat(s, GROUP, axis=0).T


def bwd_dx(dY, packed_bwd: dict, L, R, n: int, k: int) -> np.ndarray:
    """dX = dY W^{R,C} + (dY R^T) L^T in float64. dY [M, N]; L [K, r], R [r, N] or None."""
    Wrc = unpack_bwd(packed_bwd["codesT"], packed_bwd["metaT"], packed_bwd["scalesT"], n, k)
    dY = _f64(dY)
    dX = dY @ Wrc
    if L is not None and R is not None and np.asarray(L).shape[1] > 0:
        dX = dX + (dY @ _f64(R).T) @ _f64(L).T
    return dX


def lemma_extra_sparsity(N: int, M: int) -> float:
    """Closed form of Lemma sparsity_ratio: D(A^R) - D(A^{R,C}) for random N:M row masks."""
    from math import comb
    s = N / M
    return sum(comb(M, j) * s ** j * (1 - s) ** (M - j) * (j - N) / M for j in range(N + 1, M + 1))


# ------------------------------------------------- quantized adapters (SLiM-LoRA^Q)

ADAPTER_GROUP = 128   # adapter elements sharing one scale, along each factor's input dimension


def adapter_group_scales(A) -> np.ndarray:
    """AbsMax scales of an adapter factor laid out [rows, length] with groups of 128 consecutive
    elements along `length` (the factor's input dimension; the last group of a row holds
    length % 128 elements when 128 does not divide it): s16 = fp16_RNE(fp32(max|a|) / 7), the
    weights' rule (SLiM "Low-rank adapter quantization": AbsMax group quantization, group 128).
    Returns float16 [rows, ceil(length / 128)]."""
    A = np.asarray(A, dtype=np.float64)
    if not np.all(np.isfinite(A)):
        raise OracleError("non-finite adapter element")
    rows, n = A.shape
    ng = -(-n // ADAPTER_GROUP)
    s = np.zeros((rows, ng), dtype=np.float16)
    for g in range(ng):
        a = np.abs(A[:, ADAPTER_GROUP * g:ADAPTER_GROUP * (g + 1)]).max(axis=1).astype(np.float32)
        s[:, g] = fp16_rne(a / np.float32(QMAX))
    return s


def adapter_quantize(A, s16) -> np.ndarray:
    """Codes q = clamp(rint(a / s16), -7, 7) of every element (0 where s16 == 0); int8 [rows, length]."""
    A = np.asarray(A, dtype=np.float64)
    rows, n = A.shape
    S = np.repeat(s16.astype(np.float64), ADAPTER_GROUP, axis=1)[:, :n]
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.where(S > 0, A / np.where(S > 0, S, 1.0), 0.0)
    return np.clip(np.rint(t), -QMAX, QMAX).astype(np.int8)


def _encode_dense(q: np.ndarray) -> np.ndarray:
    """Dense 4-bit codes u = q + 8 of [rows, length] (length % 8 == 0) as bytes [rows, length / 2]:
    each little-endian 32-bit word holds 8 consecutive elements, element 2c in nibble c and
    element 2c + 1 in nibble c + 4 (c = 0..3)."""
    rows, n = q.shape
    u = (q.astype(np.int16) + CODE_OFFSET).astype(np.uint32).reshape(rows, n // 8, 4, 2)
    c = np.arange(4, dtype=np.uint32)
    word = ((u[..., 0] << (4 * c)) | (u[..., 1] << (4 * c + 16))).sum(axis=2, dtype=np.uint32)
    return np.ascontiguousarray(word.astype("<u4").view(np.uint8).reshape(rows, n // 2))


def _decode_dense(codes: np.ndarray, rows: int, n: int) -> np.ndarray:
    """Inverse of ``_encode_dense``: signed codes int8 [rows, length]."""
    word = np.ascontiguousarray(codes).view("<u4").reshape(rows, n // 8).astype(np.uint32)
    c = np.arange(4, dtype=np.uint32)
    lo = (word[..., None] >> (4 * c)) & 0xF
    hi = (word[..., None] >> (4 * c + 16)) & 0xF
    u = np.stack([lo, hi], axis=-1).reshape(rows, n)
    return (u.astype(np.int16) - CODE_OFFSET).astype(np.int8)


def pack_adapter_q(L, R) -> dict:
    """4-bit AbsMax group-128 pack of the adapter factors for the forward (inference) layer.

    L [K, r] is quantized as L^T [r, K] (groups along K, the input of X L) and R [r, N] as R^T [N, r]
    (groups along r, the input of T R). Returns Lq uint8 [r, K/2], Ls uint16 [r, ceil(K/128)],
    Rq uint8 [N, r/2], Rs uint16 [N, ceil(r/128)] (fp16 bit patterns)."""
    Lt = np.asarray(L, dtype=np.float64).T
    Rt = np.asarray(R, dtype=np.float64).T
    if Lt.shape[0] % 8 or Lt.shape[1] % 8:
        raise OracleError("adapter sizes must be multiples of 8")
    Ls, Rs = adapter_group_scales(Lt), adapter_group_scales(Rt)
    return {"Lq": _encode_dense(adapter_quantize(Lt, Ls)), "Ls": Ls.view(np.uint16).copy(),
            "Rq": _encode_dense(adapter_quantize(Rt, Rs)), "Rs": Rs.view(np.uint16).copy()}


def unpack_adapter_q(pq: dict, K: int, N: int, r: int):
    """Dequantized factors (float64, exact q s16): L [K, r] and R [r, N]."""
    def deq(codes, scales, rows, n):
        q = _decode_dense(codes, rows, n).astype(np.float64)
        S = np.repeat(np.asarray(scales, dtype=np.uint16).view(np.float16).astype(np.float64), ADAPTER_GROUP, axis=1)
        return q * S[:, :n]
    return deq(pq["Lq"], pq["Ls"], r, K).T, deq(pq["Rq"], pq["Rs"], N, r).T


def adapter_q_bytes(K: int, N: int, r: int) -> int:
    """Bytes of a quantized adapter: half a byte per element plus one fp16 scale per group."""
    return r * K // 2 + 2 * r * (-(-K // ADAPTER_GROUP)) + N * r // 2 + 2 * N * (-(-r // ADAPTER_GROUP))


def linear_qa(X, packed: dict, pq: dict, n: int, k: int, r: int) -> np.ndarray:
    """Y = X Wc^T + (X L^Q) R^Q in float64, with the dequantized adapter factors of ``pack_adapter_q``."""
    Lq, Rq = unpack_adapter_q(pq, k, n, r)
    return linear(X, packed, Lq, Rq, n, k)


# ------------------------------------------------------------------ tolerances

def rel_fro(Y, Yref) -> float:
    Y = _f64(Y)
    Yref = _f64(Yref)
    d = np.linalg.norm(Yref)
    return float(np.linalg.norm(Y - Yref) / d) if d > 0 else float(np.linalg.norm(Y))


def within_tolerance(Y, Yref, rel=2e-3, maxabs=1e-2) -> tuple[bool, float, float]:
    """Acceptance test for layer outputs: rel. Frobenius <= rel and max|Y-Yref| <= maxabs * ||Yref||_inf."""
    Y = _f64(Y)
    Yref = _f64(Yref)
    rf = rel_fro(Y, Yref)
    inf = float(np.max(np.abs(Yref))) if Yref.size else 0.0
    ma = float(np.max(np.abs(Y - Yref))) if Y.size else 0.0
    ok = rf <= rel and ma <= maxabs * inf if Yref.size else True
    return ok, rf, (ma / inf if inf > 0 else ma)
