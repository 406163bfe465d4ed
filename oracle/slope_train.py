"""Plain float64 NumPy oracle for the steps of SLoPe's sparse training step that follow the
input gradient (test infrastructure only: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it; the HIP path shares no code with it).

What it computes, and where the thesis defines it
-------------------------------------------------
SLoPe trains a linear layer whose weight keeps the 2:4 row-wise mask M^R fixed from setup
(chapter SLoPe, "Double-pruned Backward Pass"; Alg. "Accelerated Sparse Pretraining Algorithm
for a Linear Layer", the setup steps and the loop body after the input gradient):

* ``pack16`` -- setup of the sparse weight W^R: the 2:4 magnitude mask along K and the kept
  values in half precision (the training backend stores the weight compressed, two values per
  group of four, with index metadata; appendix "Implementation details", "Initialization, sparse
  matrix setup").
* ``pack16_t`` -- the transposed operand of the backward: W^R pruned 2:4 again along N, i.e.
  W^{R,C}, stored compressed along N for each k (eq. sparse_backward_input; the Alg.'s
  transposed setup and its update after every step).
* ``grad_w`` -- BWD-1, grad W = dY^T X (eq. sparse_backward_weight), masked with the same M^R
  and compressed to [N, K/2] ("pruneAndCompress"; appendix "Prune and compress": the gradient
  is pruned with the weight's mask and stored as an N x K/2 matrix).
* ``sparse_add`` -- beta A + gamma B on two compressed matrices with the same pattern
  ("sparseAdd"; appendix "Sparse matrix addition"; in the Alg. with beta = 1/gamma_scale on the
  gradient and the weight decay on the weight).
* ``update_pack16`` -- writing the optimizer's new values into the forward pack
  ("updateSparseMatrix"; appendix "Update Sparse Matrix"); the transposed pack is rebuilt from
  them with ``pack16_t``.

Readings where the thesis is silent
-----------------------------------
* Half precision is IEEE binary16 (the Alg. speaks of a half-precision backward with a gradient
  scaling factor); values are the fp32 weights rounded to nearest, ties to even.
* The 2:4 choice and its ties follow the inference pack (``slim_oracle.mask_2of4``): |w|
  descending, then position ascending.
* The column prune of the transposed pack ranks the stored half-precision values: per column k
  and aligned group of four rows, (|v| descending, forward-mask bit descending, n ascending),
  the same key as the inference pack's double pruning. A kept slot that M^R had dropped holds 0.
* Compressed order: for group g of a row, the value at the lower kept position comes first.
* The gradient is returned in fp32 (accumulated in at least fp32); sparse_add works in fp32 on
  an fp32 A and an fp16 B.

Formats (all row-major, little-endian)
--------------------------------------
``vals``  fp16 bits uint16 [N, K/2]: group g of row n at 2g (lower kept position), 2g + 1.
``meta``  uint8 [N, K/8]: the inference pack's index format (half-word b of a row covers
          positions 16b .. 16b+15; group c of it holds i0 in bits 4c..4c+1, i1 in 4c+2..4c+3).
``valsT`` fp16 bits uint16 [K, N/2] and ``metaT`` uint8 [K, N/8]: the same along n for each k.
``mask``  uint8 [N, K] (M^R) and ``mask_rc`` uint8 [N, K] (support of W^{R,C}).
"""
from __future__ import annotations

import numpy as np

from .slim_oracle import OracleError, _decode, _encode, fp16_rne, mask_2of4


def _kept_idx(mask: np.ndarray) -> np.ndarray:
    """Kept offsets (ascending) of every 4-group of a 0/1 mask [rows, length]: int64 [rows, length/4, 2]."""
    rows, length = mask.shape
    mg = mask.reshape(rows, length // 4, 4)
    if np.any(mg.sum(axis=2) != 2):
        raise OracleError("mask must keep exactly two of every four")
    return np.sort(np.argsort(-mg.astype(np.int8), axis=2, kind="stable")[..., :2], axis=2)


def _meta_of(idx: np.ndarray, rows: int, length: int) -> np.ndarray:
    _, meta = _encode(np.zeros(idx.shape, dtype=np.uint8), idx, rows, length)
    return meta


def idx_of_meta(meta: np.ndarray, rows: int, length: int) -> np.ndarray:
    """Kept offsets [rows, length/4, 2] from index metadata."""
    _, idx = _decode(np.zeros((rows, length // 4), dtype=np.uint8), meta, rows, length)
    return idx.astype(np.int64)


def pack16(W) -> dict:
    """Setup of W^R from fp32 W [N, K]: 2:4 magnitude mask along K, kept values in fp16."""
    W = np.asarray(W, dtype=np.float32)
    n, k = W.shape
    if k % 16:
        raise OracleError("K must be a multiple of 16")
    if not np.all(np.isfinite(W)):
        raise OracleError("non-finite weight")
    m = mask_2of4(W)
    idx = _kept_idx(m)
    v = np.take_along_axis(W.reshape(n, k // 4, 4), idx, axis=2).reshape(n, k // 2)
    return {"vals": fp16_rne(v).view(np.uint16).copy(), "meta": _meta_of(idx, n, k), "mask": m}


def unpack16(vals, meta, n: int, k: int) -> np.ndarray:
    """Dense W^R [n, k] (float64) from a value pack."""
    idx = idx_of_meta(meta, n, k)
    v = np.asarray(vals, dtype=np.uint16).view(np.float16).astype(np.float64).reshape(n, k // 4, 2)
    dense = np.zeros((n, k // 4, 4), dtype=np.float64)
    np.put_along_axis(dense, idx, v, axis=2)
    return dense.reshape(n, k)


def mask_of_meta(meta, n: int, k: int) -> np.ndarray:
    idx = idx_of_meta(meta, n, k)
    m = np.zeros((n, k // 4, 4), dtype=np.uint8)
    np.put_along_axis(m, idx, 1, axis=2)
    return m.reshape(n, k)


def pack16_t(vals, meta, n: int, k: int) -> dict:
    """W^{R,C} along N: per column k and aligned group of four rows keep the top two by
    (|v| desc, M^R bit desc, n asc); returns valsT [K, N/2], metaT [K, N/8], mask_rc [N, K]."""
    if n % 16:
        raise OracleError("N must be a multiple of 16")
    Wr = unpack16(vals, meta, n, k)
    mr = mask_of_meta(meta, n, k)
    a = np.abs(Wr.T).reshape(k, n // 4, 4)
    f = mr.T.reshape(k, n // 4, 4).astype(np.int64)
    pos = np.broadcast_to(np.arange(4), a.shape)
    order = np.lexsort((pos, -f, -a), axis=-1)
    idx = np.sort(order[..., :2], axis=2)
    # values exactly as stored (fp16), 0 for a slot M^R had dropped
    vT = np.take_along_axis(Wr.T.reshape(k, n // 4, 4), idx, axis=2).reshape(k, n // 2)
    sel = np.zeros((k, n // 4, 4), dtype=np.uint8)
    np.put_along_axis(sel, idx, 1, axis=2)
    mask_rc = (sel.reshape(k, n).T & mr).astype(np.uint8)
    return {"valsT": vT.astype(np.float16).view(np.uint16).copy(), "metaT": _meta_of(idx, k, n),
            "mask_rc": np.ascontiguousarray(mask_rc)}


def unpack16_t(valsT, metaT, n: int, k: int) -> np.ndarray:
    """Dense W^{R,C} [n, k] (float64) from a transposed value pack."""
    return unpack16(valsT, metaT, k, n).T


def grad_w(dY, X, meta, n: int, k: int) -> np.ndarray:
    """BWD-1 with the weight's mask: (dY^T X)[n, kept k] in float64, compressed [N, K/2]."""
    dY = np.asarray(dY, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    G = dY.T @ X                                            # [N, K]
    idx = idx_of_meta(meta, n, k)
    return np.take_along_axis(G.reshape(n, k // 4, 4), idx, axis=2).reshape(n, k // 2)


def sparse_add(A, B, beta: float, gamma: float) -> np.ndarray:
    """beta A + gamma B on compressed values with one shared pattern (float64)."""
    return float(beta) * np.asarray(A, dtype=np.float64) + float(gamma) * np.asarray(B, dtype=np.float64)


def update_pack16(Wnew) -> np.ndarray:
    """New compressed fp32 values [N, K/2] -> the forward pack's fp16 values (pattern unchanged)."""
    W = np.asarray(Wnew, dtype=np.float32)
    if not np.all(np.isfinite(W)):
        raise OracleError("non-finite weight")
    return fp16_rne(W).view(np.uint16).copy()
