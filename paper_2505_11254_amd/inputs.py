"""Seeded synthetic inputs shared by the GPU path's tests/bench and the oracle.

This module draws random numbers and plants structured values; it holds none
of the attention arithmetic.  Both sides receive the very same bf16 tensors:
the oracle reads them back bit for bit, so parity never depends on which
device drew them.
"""
from __future__ import annotations

import torch

from .workloads import Workload

_CHUNK_TOKENS = 1 << 15


def _normal(shape, seed, device, out_dtype, chunk_tokens=_CHUNK_TOKENS, offset=None):
    """N(0,1) values of `shape` = [T, H, d] drawn in token chunks, plus `offset` [H, d]."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    T = shape[0]
    out = torch.empty(shape, dtype=out_dtype, device=device)
    for t0 in range(0, T, chunk_tokens):
        t1 = min(T, t0 + chunk_tokens)
        x = torch.randn((t1 - t0,) + tuple(shape[1:]), generator=g, device=device,
                        dtype=torch.float32)
        if offset is not None:
            x += offset
        out[t0:t1].copy_(x)
    return out


def generate(wl: Workload, device="cpu", dtype=torch.bfloat16):
    """Q [T,Hq,d], K/V [T,Hkv,d] for a workload, plus int32 cu_seqlens on `device`.

    K gets a per-kv-head mean offset with entries N(0, k_offset_std^2) added
    before the cast when the workload asks for it.
    """
    T = wl.total_tokens
    offset = None
    if wl.k_offset_std > 0:
        g = torch.Generator(device=device)
        g.manual_seed(wl.seed_base + 3)
        offset = torch.randn((wl.Hkv, wl.d), generator=g, device=device,
                             dtype=torch.float32) * wl.k_offset_std
    q = _normal((T, wl.Hq, wl.d), wl.seed_base + 0, device, dtype)
    k = _normal((T, wl.Hkv, wl.d), wl.seed_base + 1, device, dtype, offset=offset)
    v = _normal((T, wl.Hkv, wl.d), wl.seed_base + 2, device, dtype)
    cu = torch.tensor(wl.cu_seqlens(), dtype=torch.int32, device=device)
    return q, k, v, cu


def random_qkv(seqlens, Hq, Hkv, d, seed, device="cpu", dtype=torch.bfloat16, std=1.0):
    """I.i.d. N(0, std^2) Q, K, V for an arbitrary (ragged) batch."""
    T = int(sum(seqlens))
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    q = (torch.randn((T, Hq, d), generator=g) * std).to(dtype)
    k = (torch.randn((T, Hkv, d), generator=g) * std).to(dtype)
    v = (torch.randn((T, Hkv, d), generator=g) * std).to(dtype)
    cu = [0]
    for n in seqlens:
        cu.append(cu[-1] + int(n))
    return q.to(device), k.to(device), v.to(device), torch.tensor(cu, dtype=torch.int32,
                                                                  device=device)


def plant_needles(q, k, pairs, heads=None, scale=16.0, seed=0):
    """Make query row i and key row j share one direction for each (i, j) in `pairs`.

    Both rows become scale * u for a random unit vector u (one per pair), so
    the score of (i, j) stands far above the rest and whether key j lies in
    row i's key set decides that row's output.  Rows are global token indices;
    `heads` limits the planting to some query heads (kv heads follow GQA).
    """
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    Hq, d = q.shape[1], q.shape[2]
    Hkv = k.shape[1]
    G = Hq // Hkv
    hs = range(Hq) if heads is None else heads
    for (i, j) in pairs:
        u = torch.randn(d, generator=g)
        u = u / u.norm()
        for h in hs:
            q[i, h] = (scale * u).to(q.dtype)
            k[j, h // G] = (scale * u).to(k.dtype)
    return q, k
