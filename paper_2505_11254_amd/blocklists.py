"""Seeded key-block lists for Delta Attention over other sparse bases.

The method corrects any sparse attention f* (Sec. 3; the paper pairs it with
StreamingLLM, MInference, HiP and Star Attention in Sec. 4).  A block-sparse
f* is described by key-block lists: for sequence b, kv head g and query block
qb (rows qb*block_q .. qb*block_q + block_q - 1 of that sequence), the key
tiles (64 keys each) the block's rows attend to.  The tiles overlapping the
query block itself are always attended (causally) and are not listed.

Layout (the C ABI's and the oracle's): CSR int32 arrays
  ptr [B, Hkv, nqb + 1]  offsets into idx for every (b, g, qb),
  idx [nnz]              ascending unique tile indices < qb * block_q / 64,
with nqb = ceil(max_seqlen / block_q).

This module only draws the lists (no attention arithmetic); the tests, the
benchmark and the oracle take them as inputs.  The layouts stand in for the
selection rules of the sparse methods the paper compares with, not for their
scoring: which tiles are chosen does not change the kernels' cost, only how
many are.
  vertical_slash  a few key columns every query block sees (tile 0 and seeded
                  others) plus a band of recent tiles and diagonals further
                  back (MInference's vertical and slash lines, in tiles);
  block_topk      k seeded tiles per query block, tile 0 always kept (the
                  shape of a per-block top-k selection such as HiP's);
  star            the first `anchor` keys plus the query's own context block
                  of `context` keys (Star Attention's first phase).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

TILE = 64


@dataclass
class BlockLists:
    block_q: int
    ptr: np.ndarray   # int32 [B, Hkv, nqb + 1]
    idx: np.ndarray   # int32 [nnz]

    @property
    def nqb(self) -> int:
        return self.ptr.shape[2] - 1

    def to(self, device):
        """(ptr, idx) as int32 torch tensors on `device` (idx never empty)."""
        import torch
        idx = self.idx if self.idx.size else np.zeros(1, dtype=np.int32)
        return (torch.from_numpy(np.ascontiguousarray(self.ptr)).to(device),
                torch.from_numpy(np.ascontiguousarray(idx)).to(device))

    def tiles(self, b, g, qb) -> np.ndarray:
        return self.idx[self.ptr[b, g, qb]:self.ptr[b, g, qb + 1]]


def _build(seqlens, Hkv, block_q, choose):
    """choose(b, g, qb, diag0) -> iterable of tiles < diag0."""
    assert block_q % TILE == 0 and block_q >= TILE
    nqb = max(1, -(-max(seqlens) // block_q))
    B = len(seqlens)
    ptr = np.zeros((B, Hkv, nqb + 1), dtype=np.int64)
    chunks = []
    n = 0
    for b, L in enumerate(seqlens):
        nq_b = -(-L // block_q)
        for g in range(Hkv):
            for qb in range(nqb):
                ptr[b, g, qb] = n
                if qb < nq_b:
                    diag0 = qb * block_q // TILE
                    t = np.unique(np.asarray(list(choose(b, g, qb, diag0)), dtype=np.int64))
                    t = t[(t >= 0) & (t < diag0)]
                    chunks.append(t)
                    n += len(t)
            ptr[b, g, nqb] = n
    idx = np.concatenate(chunks) if chunks else np.zeros(0, dtype=np.int64)
    assert n < 2 ** 31
    return BlockLists(block_q, ptr.astype(np.int32), idx.astype(np.int32))


def vertical_slash(seqlens, Hkv, block_q=64, n_vertical=8, n_local=8, slash_offsets=(64, 256),
                   seed=0):
    """Vertical columns (tile 0 plus n_vertical - 1 seeded tiles per (b, g)), a
    band of n_local tiles before the query block, and single tiles at the
    given distances (in tiles) before it."""
    rng = np.random.default_rng(seed)
    vert = {}
    for b, L in enumerate(seqlens):
        nt = -(-L // TILE)
        for g in range(Hkv):
            extra = rng.choice(nt, size=min(nt, max(0, n_vertical - 1)), replace=False)
            vert[b, g] = np.concatenate([[0], extra])

    def choose(b, g, qb, diag0):
        band = range(max(0, diag0 - n_local), diag0)
        slash = [diag0 - o for o in slash_offsets]
        return list(vert[b, g]) + list(band) + slash
    return _build(seqlens, Hkv, block_q, choose)


def block_topk(seqlens, Hkv, block_q=64, k=32, seed=0):
    """k seeded tiles per query block (all of them when fewer exist), tile 0 kept."""
    rng = np.random.default_rng(seed)

    def choose(b, g, qb, diag0):
        if diag0 <= k:
            return range(diag0)
        return [0] + list(rng.choice(np.arange(1, diag0), size=k - 1, replace=False))
    return _build(seqlens, Hkv, block_q, choose)


def star(seqlens, Hkv, block_q=64, anchor=2048, context=4096):
    """The first `anchor` keys plus the query's own context block (`context`
    keys, a multiple of block_q) up to the query block."""
    assert anchor % TILE == 0 and context % block_q == 0

    def choose(b, g, qb, diag0):
        c0 = (qb * block_q // context) * context // TILE
        return list(range(anchor // TILE)) + list(range(c0, diag0))
    return _build(seqlens, Hkv, block_q, choose)


def full(seqlens, Hkv, block_q=64):
    """Every tile before the query block: f* becomes dense causal attention."""
    return _build(seqlens, Hkv, block_q, lambda b, g, qb, diag0: range(diag0))


def empty(seqlens, Hkv, block_q=64):
    """No listed tile: each row sees only its own query block's tiles."""
    return _build(seqlens, Hkv, block_q, lambda b, g, qb, diag0: ())


def pair_count(bl: BlockLists, seqlens, Hkv, G):
    """Sum over rows and query heads of |S(i)| (the useful (row, key) pairs)."""
    tot = 0
    for b, L in enumerate(seqlens):
        for g in range(Hkv):
            for qb in range(-(-L // bl.block_q)):
                r0, r1 = qb * bl.block_q, min(L, (qb + 1) * bl.block_q)
                diag0 = r0 // TILE
                listed = len(bl.tiles(b, g, qb)) * TILE
                rows = np.arange(r0, r1, dtype=np.int64)
                tot += int((listed + rows - diag0 * TILE + 1).sum()) * G
    return tot
