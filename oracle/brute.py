"""Pure-Python brute force for tiny shapes (test infrastructure only).

Each step enumerates instead of computing in closed form, so it shares no logic
with ``slim_oracle``:

* the 2:4 choice enumerates the six two-of-four patterns (the candidate set of the
  learnable 2:4 masks in the PATCH chapter) and takes the largest kept magnitude,
  lexicographically first on ties;
* fp16 rounding searches every finite binary16 value;
* the int4 code is the argmin over q in [-7, 7] of |w - q s|, computed in exact
  rational arithmetic, ties to even q;
* the layer products are explicit triple loops.
"""
from __future__ import annotations

import struct
from fractions import Fraction
from itertools import combinations

import numpy as np

PATTERNS = list(combinations(range(4), 2))   # six candidate 2:4 patterns, lexicographic order

_F16_POS = None


def _f16_table():
    """Every finite non-negative binary16 value (as float64, exact) with its bit pattern."""
    global _F16_POS
    if _F16_POS is None:
        vals = [struct.unpack("<e", i.to_bytes(2, "little"))[0] for i in range(0x7C00)]
        _F16_POS = np.array(vals, dtype=np.float64)
    return _F16_POS


def to_f32(x: float) -> float:
    """Round a Python float to the nearest float32 (struct packing rounds to nearest even)."""
    return struct.unpack("<f", struct.pack("<f", x))[0]


def f16_nearest(x: float) -> float:
    """Nearest binary16 value by exhaustive search; ties to the even bit pattern; overflow to inf."""
    if x < 0:
        return -f16_nearest(-x)
    table = _f16_table()
    if x >= 65520.0:
        return float("inf")
    # Distances to all candidates. Both operands are float64 numbers with at most 24
    # significant bits, so the distance to every candidate near x is exact (Sterbenz);
    # far candidates cannot round below the nearest distance.
    d = np.abs(table - x)
    cand = np.nonzero(d == d.min())[0]
    if len(cand) > 1:
        cand = [c for c in cand if c % 2 == 0]
    return float(table[cand[0]])


def top2(ws):
    """Kept positions of one 4-group: the pattern with the largest |w| sum, first in lexicographic order."""
    best, best_sum = None, None
    for p in PATTERNS:
        s = abs(ws[p[0]]) + abs(ws[p[1]])
        if best is None or s > best_sum:
            best, best_sum = p, s
    return best


def rtn_code(w: float, s: float) -> int:
    """argmin over q in [-7, 7] of |w - q s| (exact rationals), ties to even q; 0 when s == 0."""
    if s == 0:
        return 0
    fw, fs = Fraction(w), Fraction(s)
    best, best_d = None, None
    for q in range(-7, 8):
        d = abs(fw - q * fs)
        if best is None or d < best_d or (d == best_d and q % 2 == 0):
            best, best_d = q, d
    return best


def dense_weight(W):
    """Wc as nested lists: mask by ``top2``, scale by exhaustive fp16 search, code by ``rtn_code``."""
    n, k = len(W), len(W[0])
    out = [[0.0] * k for _ in range(n)]
    for i in range(n):
        for g in range(k // 128):
            a = max(abs(W[i][j]) for j in range(128 * g, 128 * g + 128))
            s = f16_nearest(to_f32(to_f32(a) / 7.0))
            for j4 in range(32 * g, 32 * g + 32):
                ws = W[i][4 * j4: 4 * j4 + 4]
                for p in top2(ws):
                    j = 4 * j4 + p
                    out[i][j] = rtn_code(W[i][j], s) * s
    return out


def column_prune(Wc, mask):
    """Support of W^{R,C}: per column and aligned 4-group of rows, the two slots ranked first by
    (|Wc| desc, forward mask desc, row asc), enumerated over the six patterns."""
    n, k = len(Wc), len(Wc[0])
    keep = [[0] * k for _ in range(n)]
    for j in range(k):
        for g in range(n // 4):
            rows = [4 * g + t for t in range(4)]

            def rank_key(p):
                # compare two patterns by the sorted list of member keys (best first)
                keys = sorted(((-abs(Wc[rows[t]][j]), -mask[rows[t]][j], t) for t in p))
                return keys
            best = min(PATTERNS, key=rank_key)
            for t in best:
                if mask[rows[t]][j]:
                    keep[rows[t]][j] = 1
    return keep


def matmul(A, B):
    n, m, k = len(A), len(B[0]), len(B)
    return [[sum(A[i][t] * B[t][j] for t in range(k)) for j in range(m)] for i in range(n)]


def transpose(A):
    return [list(r) for r in zip(*A)]


def linear(X, W, L, R):
    """Y[m][n] = sum_k X[m][k] Wc[n][k] + sum_j (sum_k X[m][k] L[k][j]) R[j][n]."""
    Wc = dense_weight(W)
    M, K, N = len(X), len(X[0]), len(W)
    Y = [[sum(X[m][t] * Wc[n][t] for t in range(K)) for n in range(N)] for m in range(M)]
    if L is not None and len(L[0]) > 0:
        r = len(L[0])
        T = [[sum(X[m][t] * L[t][j] for t in range(K)) for j in range(r)] for m in range(M)]
        for m in range(M):
            for n in range(N):
                Y[m][n] += sum(T[m][j] * R[j][n] for j in range(r))
    return Y


def bwd_dx(dY, W, L, R):
    """dX[m][k] = sum_n dY[m][n] Wrc[n][k] + sum_j (sum_n dY[m][n] R[j][n]) L[k][j]."""
    Wc = dense_weight(W)
    n, k = len(Wc), len(Wc[0])
    # forward mask from the same enumeration
    mask = [[0] * k for _ in range(n)]
    for i in range(n):
        for j4 in range(k // 4):
            for p in top2(W[i][4 * j4: 4 * j4 + 4]):
                mask[i][4 * j4 + p] = 1
    keep = column_prune(Wc, mask)
    M = len(dY)
    dX = [[sum(dY[m][i] * Wc[i][j] * keep[i][j] for i in range(n)) for j in range(k)] for m in range(M)]
    if L is not None and len(L[0]) > 0:
        r = len(L[0])
        U = [[sum(dY[m][i] * R[j][i] for i in range(n)) for j in range(r)] for m in range(M)]
        for m in range(M):
            for j in range(k):
                dX[m][j] += sum(U[m][t] * L[j][t] for t in range(r))
    return dX


def adapter_dequant(A, group=128):
    """Quantize-dequantize of an adapter factor given as rows (lists), groups of `group` consecutive
    elements of a row: scale by exhaustive fp16 search of fp32(max |a|) / 7, codes by ``rtn_code``."""
    out = []
    for row in A:
        q = [0.0] * len(row)
        for g0 in range(0, len(row), group):
            a = max(abs(v) for v in row[g0:g0 + group])
            s = f16_nearest(to_f32(to_f32(a) / 7.0))
            for j in range(g0, min(g0 + group, len(row))):
                q[j] = rtn_code(row[j], s) * s
        out.append(q)
    return out
