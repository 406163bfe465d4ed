"""Plain float64 NumPy oracle for PATCH's hybrid dense / 2:4 tile layer (test infrastructure only:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may use
it; the HIP path shares no code with it).

What it computes, and where the thesis defines it
-------------------------------------------------
PATCH decides, per tile of the weight, whether the tile stays dense or is pruned 2:4, which gives
sparsity ratios between 0 and 50% (PATCH chapter; the learned tile-level decisions and the
"PATCH_Tile" variant that learns only those). Deploying it needs a GEMM whose tiles are either
dense or 2:4 sparse in one product ("Efficient deployment of PATCH"; appendix "STOICC
Integration"), with 128 x 128 tiles as the hardware-friendly size the thesis settles on.

* ``hybrid_weight``: the deployed weight: a tile marked sparse keeps the two largest magnitudes of
  each aligned group of four along K (``slim_oracle.mask_2of4``'s rule), a dense tile keeps all;
  kept values in fp16 (round to nearest, ties to even).
* ``linear``: Y = X Wp^T in float64.
* ``pack``: the byte format below, written out from its definition.

Readings
--------
* H1  Tile map: given (PATCH learns it from data; here it is a synthetic input), one byte per
      128 x 128 tile, row-major over (N/128, K/128); 1 = 2:4 sparse, 0 = dense.
* H2  Mask inside a sparse tile: magnitude top-2 of every aligned 4-group along K, ties to the
      lower position (as the 2:4 path of this library); PATCH would learn it.
* H3  Values: fp16 (the deployment keeps the model in half precision; no quantisation).
* H4  Sparsity of a layer = 0.5 x (fraction of sparse tiles).

Format
------
``tile_info`` uint64 [N/128, K/128]: byte offset of the tile's payload (16-byte aligned), with bit
63 set for a sparse tile. Payloads follow each other in row-major tile order.
* dense tile: 128 rows x 128 fp16 (256 bytes per row), 32768 bytes;
* sparse tile: two halves (positions 0..63, then 64..127) of 9216 bytes each: 128 rows x 32 fp16 kept
  values (group g of the half's 16 groups at 2g, 2g+1, the lower kept position first), then 128 rows
  x 4 uint16 index half-words (half-word b covers the half's positions 16b .. 16b+15; group c of it
  holds i0 in bits 4c..4c+1 and i1 in bits 4c+2..4c+3); 18432 bytes.
"""
from __future__ import annotations

import numpy as np

from .slim_oracle import OracleError, fp16_rne, mask_2of4

TILE = 128
DENSE_BYTES = TILE * TILE * 2
SPARSE_HALF = TILE * TILE // 2 + TILE * TILE // 16
SPARSE_BYTES = 2 * SPARSE_HALF
SPARSE_BIT = np.uint64(1) << np.uint64(63)


def _check(W, kinds):
    W = np.asarray(W, dtype=np.float32)
    n, k = W.shape
    if n % TILE or k % TILE:
        raise OracleError("N and K must be multiples of 128")
    kinds = np.asarray(kinds, dtype=np.uint8).reshape(n // TILE, k // TILE)
    if np.any(kinds > 1):
        raise OracleError("tile kinds are 0 (dense) or 1 (2:4 sparse)")
    if not np.all(np.isfinite(W)):
        raise OracleError("non-finite weight")
    return W, kinds, n, k


def tile_mask(kinds, n: int, k: int) -> np.ndarray:
    """0/1 [N, K]: 1 where the position lies in a sparse tile."""
    return np.repeat(np.repeat(np.asarray(kinds, dtype=np.uint8).reshape(n // TILE, k // TILE), TILE, 0), TILE, 1)


def hybrid_weight(W, kinds) -> np.ndarray:
    """The deployed weight Wp [N, K] (float64): 2:4 inside sparse tiles, fp16 values everywhere (H1-H3)."""
    W, kinds, n, k = _check(W, kinds)
    keep = np.where(tile_mask(kinds, n, k) == 1, mask_2of4(W), 1)
    return keep * fp16_rne(W).astype(np.float64)


def sparsity(kinds) -> float:
    return 0.5 * float(np.mean(np.asarray(kinds, dtype=np.float64)))


def linear(X, Wp) -> np.ndarray:
    """Y = X Wp^T in float64."""
    return np.asarray(X, dtype=np.float64) @ np.asarray(Wp, dtype=np.float64).T


def payload_bytes(kinds) -> int:
    kinds = np.asarray(kinds, dtype=np.int64)
    return int(kinds.sum() * SPARSE_BYTES + (kinds.size - kinds.sum()) * DENSE_BYTES)


def pack(W, kinds) -> dict:
    """tile_info uint64 [N/128, K/128] and payload bytes, as the module docstring lays them out."""
    W, kinds, n, k = _check(W, kinds)
    tn, tk = n // TILE, k // TILE
    info = np.zeros((tn, tk), dtype=np.uint64)
    out = np.zeros(payload_bytes(kinds), dtype=np.uint8)
    m = mask_2of4(W)
    h = fp16_rne(W)
    off = 0
    for a in range(tn):
        for b in range(tk):
            rows, cols = slice(a * TILE, (a + 1) * TILE), slice(b * TILE, (b + 1) * TILE)
            if kinds[a, b]:
                info[a, b] = np.uint64(off) | SPARSE_BIT
                mg = m[rows, cols].reshape(TILE, TILE // 4, 4)
                idx = np.sort(np.argsort(-mg.astype(np.int8), axis=2, kind="stable")[..., :2], axis=2)
                vals = np.take_along_axis(h[rows, cols].reshape(TILE, TILE // 4, 4), idx, axis=2)
                c = np.arange(4, dtype=np.uint32)
                ix = idx.reshape(TILE, TILE // 16, 4, 2).astype(np.uint32)
                half = ((ix[..., 0] << (4 * c)) | (ix[..., 1] << (4 * c + 2))).sum(axis=2, dtype=np.uint32)
                for hf in range(2):
                    o = off + hf * SPARSE_HALF
                    v = vals[:, 16 * hf:16 * hf + 16].reshape(TILE, TILE // 4)
                    out[o:o + TILE * TILE // 2] = np.ascontiguousarray(v).view(np.uint8).reshape(-1)
                    hw = np.ascontiguousarray(half[:, 4 * hf:4 * hf + 4]).astype("<u2")
                    out[o + TILE * TILE // 2:o + SPARSE_HALF] = hw.view(np.uint8).reshape(-1)
                off += SPARSE_BYTES
            else:
                info[a, b] = np.uint64(off)
                out[off:off + DENSE_BYTES] = np.ascontiguousarray(h[rows, cols]).view(np.uint8).reshape(-1)
                off += DENSE_BYTES
    return {"tile_info": info, "payload": out}


def unpack(tile_info, payload, n: int, k: int) -> np.ndarray:
    """The dense Wp [n, k] (float64) a hybrid pack holds."""
    tn, tk = n // TILE, k // TILE
    info = np.asarray(tile_info, dtype=np.uint64).reshape(tn, tk)
    Wp = np.zeros((n, k), dtype=np.float64)
    for a in range(tn):
        for b in range(tk):
            off = int(info[a, b] & ~SPARSE_BIT)
            blk = Wp[a * TILE:(a + 1) * TILE, b * TILE:(b + 1) * TILE]
            if int(info[a, b] >> np.uint64(63)):
                vparts, hparts = [], []
                for hf in range(2):
                    o = off + hf * SPARSE_HALF
                    vparts.append(payload[o:o + TILE * TILE // 2].view(np.float16).reshape(TILE, TILE // 4))
                    hparts.append(payload[o + TILE * TILE // 2:o + SPARSE_HALF].view("<u2").reshape(TILE, TILE // 32))
                vals = np.concatenate(vparts, axis=1).reshape(TILE, TILE // 4, 2).astype(np.float64)
                half = np.concatenate(hparts, axis=1)
                c = np.arange(4)
                i0 = (half[..., None].astype(np.int64) >> (4 * c)) & 3
                i1 = (half[..., None].astype(np.int64) >> (4 * c + 2)) & 3
                idx = np.stack([i0, i1], -1).reshape(TILE, TILE // 4, 2)
                d = np.zeros((TILE, TILE // 4, 4))
                np.put_along_axis(d, idx, vals, axis=2)
                blk[:] = d.reshape(TILE, TILE)
            else:
                blk[:] = payload[off:off + DENSE_BYTES].view(np.float16).reshape(TILE, TILE).astype(np.float64)
    return Wp
