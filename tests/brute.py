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


# ---- correction variants (Sec. 3 "recompute", interpolation appendix) in matrix form ----

def delta_rows(dense, sparse, L, gamma):
    """Delta_i = dense - sparse at anchors a_i = i*gamma < floor(L/gamma)*gamma: [nA, d]."""
    Lc = (L // gamma) * gamma
    anchors = np.arange(0, Lc, gamma)
    return dense[anchors] - sparse[anchors]


def ema_matrix(n, b):
    """E = W @ D + f * D_0 for E_r = (1-b) E_{r-1} + b D_r, E_{-1} = D_0 (closed form)."""
    r = np.arange(n)[:, None]
    s = np.arange(n)[None, :]
    W = np.where(s <= r, b * (1.0 - b) ** np.clip(r - s, 0, None), 0.0)
    f = (1.0 - b) ** (np.arange(n) + 1.0)
    return W, f


def abg_matrix(n, alpha, beta, gam):
    """o = H @ y for the alpha-beta-gamma filter started at x_0 = (y_0, 0, 0):
    x_i = A x_{i-1} + K y_i with A = (I - K C) F, o_i = C x_i (state-space form)."""
    F = np.array([[1.0, 1.0, 0.5], [0.0, 1.0, 1.0], [0.0, 0.0, 1.0]])
    K = np.array([[alpha], [beta], [gam]])
    C = np.array([[1.0, 0.0, 0.0]])
    A = (np.eye(3) - K @ C) @ F
    H = np.zeros((n, n))
    x0 = np.array([[1.0], [0.0], [0.0]])  # contribution of y_0 through the initial state
    Ap = np.eye(3)
    for i in range(n):
        H[i, 0] = (C @ Ap @ x0)[0, 0]
        Ap = A @ Ap
    for j in range(1, n):
        Ap = np.eye(3)
        for i in range(j, n):
            H[i, j] += (C @ Ap @ K)[0, 0]
            Ap = A @ Ap
    return H


def brute_variant(q, k, v, cu, window, n_sink, gamma, mode, params=(0.0, 0.0, 0.0)):
    """Delta Attention with the correction of step 5 given by mode (0..4), matrix forms."""
    out, dense_all, sparse_all = brute_parts(q, k, v, cu, window, n_sink, gamma)
    if mode == 0:
        return out
    res = dense_all.copy()  # tail rows keep the dense result
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        L = s1 - s0
        Lc = (L // gamma) * gamma
        nA = Lc // gamma
        if nA == 0:
            continue
        for h in range(q.shape[1]):
            sp = sparse_all[s0:s1, h]
            dl = delta_rows(dense_all[s0:s1, h], sp, L, gamma)  # [nA, d]
            if mode == 1:  # recompute: dense rows swapped in at anchors only
                corr = np.zeros((Lc, sp.shape[1]))
                corr[::gamma] = dl
            elif mode == 2:  # linear interpolation towards the next anchor's Delta
                beta = np.linspace(0.0, 1.0, gamma) if gamma > 1 else np.zeros(1)
                nxt = np.vstack([dl[1:], dl[-1:]])
                corr = ((1.0 - beta)[None, :, None] * dl[:, None, :]
                        + beta[None, :, None] * nxt[:, None, :]).reshape(Lc, -1)
            elif mode == 3:  # EMA over repeat(Delta, gamma)
                D = np.repeat(dl, gamma, axis=0)
                W, f = ema_matrix(Lc, params[0])
                corr = W @ D + f[:, None] * D[0][None, :]
            else:  # alpha-beta-gamma filter over Delta_0..Delta_{nA-1}, then repeat
                H = abg_matrix(nA, *params[:3])
                corr = np.repeat(H @ dl, gamma, axis=0)
            res[s0:s0 + Lc, h] = sp[:Lc] + corr
    return res


# ---- f* from key-block lists (other sparse bases) ----

def block_mask(L, ptr_bg, idx, block_q):
    """M[i, j] for one (sequence, kv head): j <= i and tile j//64 is listed for
    query block i//block_q or lies at or after that block's first tile.
    ptr_bg: the [nqb + 1] CSR offsets of this (sequence, kv head)."""
    i = np.arange(L)[:, None]
    j = np.arange(L)[None, :]
    nt = -(-L // 64)
    nq = -(-L // block_q)
    listed = np.zeros((nq, nt), dtype=bool)
    for qb in range(nq):
        diag0 = qb * block_q // 64
        for t in idx[ptr_bg[qb]:ptr_bg[qb + 1]]:
            if 0 <= t < diag0:
                listed[qb, t] = True
    qb_i = i // block_q
    tile_j = j // 64
    return (j <= i) & ((tile_j >= qb_i * block_q // 64) | listed[qb_i, tile_j])


def brute_block_parts(q, k, v, cu, ptr, idx, block_q, gamma):
    """(out, dense AV, sparse A*V) of Algorithm 1 with f* from block lists."""
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
        Mc, _ = masks(L, 1, 0)
        Lc = (L // gamma) * gamma
        anchors = np.arange(0, Lc, gamma)
        for h in range(Hq):
            g = h // G
            Ms = block_mask(L, ptr[b, g], idx, block_q)
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
