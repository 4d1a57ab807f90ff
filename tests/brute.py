"""Brute-force Delta Attention with materialised N x N matrices (tiny N only).

A direct matrix transcription of the method, independent of the oracle's
streaming per-row loops (it shares no code with ``oracle/``):

  X   = Q K^T / sqrt(d)                                   (Sec. 2, Eq. 1)
  A   = softmax over the causal mask M_c (j <= i)
  A*  = softmax over the sparse mask M_s = M_c and (j < s or i - j < w),
        normalised over the kept entries only (Sec. 3)
  Delta = (A V)[delta] - (A* V)[delta], delta = {0, gamma, 2 gamma, ...}  (Alg. 1)
  out[:Lc] = (A* V)[:Lc] + repeat(Delta, gamma)                           (Eq. 6)
  out[Lc:] = (A V)[Lc:]   tail rows computed densely (implementation details)
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even), as uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def masked_softmax(X: np.ndarray, M: np.ndarray) -> np.ndarray:
    Y = np.where(M, X, -np.inf)
    Y = Y - Y.max(axis=1, keepdims=True)
    E = np.where(M, np.exp(Y), 0.0)
    return E / E.sum(axis=1, keepdims=True)


def masks(L: int, window: int, n_sink: int):
    i = np.arange(L)[:, None]
    j = np.arange(L)[None, :]
    Mc = j <= i
    Ms = Mc & ((j < n_sink) | (i - j < window))
    return Mc, Ms


def brute_parts(q, k, v, cu, window, n_sink, gamma):
    """Return (out, dense AV, sparse A*V) as fp64 [T, Hq, d] arrays."""
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    out = np.zeros((T, Hq, d))
    dense = np.zeros((T, Hq, d))
    sparse = np.zeros((T, Hq, d))
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        L = s1 - s0
        if L == 0:
            continue
        Mc, Ms = masks(L, window, n_sink)
        Lc = (L // gamma) * gamma
        anchors = np.arange(0, Lc, gamma)
        for h in range(Hq):
            g = h // G
            Q, K, V = q[s0:s1, h], k[s0:s1, g], v[s0:s1, g]
            X = Q @ K.T / np.sqrt(d)
            AV = masked_softmax(X, Mc) @ V
            AsV = masked_softmax(X, Ms) @ V
            Delta = AV[anchors] - AsV[anchors]
            o = AV.copy()
            o[:Lc] = AsV[:Lc] + np.repeat(Delta, gamma, axis=0)
            out[s0:s1, h] = o
            dense[s0:s1, h] = AV
            sparse[s0:s1, h] = AsV
    return out, dense, sparse


def brute_delta(q, k, v, cu, window, n_sink, gamma):
    return brute_parts(q, k, v, cu, window, n_sink, gamma)[0]
