"""Row sampling and error metrics for parity checks against the oracle.

A row of Delta Attention depends only on its own key set and on its
anchor's sparse and dense rows, so the oracle can evaluate any subset of
(sequence, head, row) triples exactly; large workloads are checked on such
samples.
"""
from __future__ import annotations

import numpy as np
import torch

# spec tolerances for bf16 I/O with fp32 accumulation
MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def sample_rows(seqlens, Hq, window, n_sink, gamma, n_random=96, seed=0):
    """(b, h, i) triples: every boundary the method has, plus seeded random rows."""
    rng = np.random.default_rng(seed)
    rows = set()
    for b, L in enumerate(seqlens):
        Lc = (L // gamma) * gamma
        first_open = -(-(n_sink + window) // gamma) * gamma  # first anchor with Delta != 0
        special = [0, 1, gamma - 1, gamma, gamma + 1, first_open - gamma, first_open - 1,
                   first_open, first_open + 1, first_open + gamma - 1, window - 1, window,
                   window + 1, n_sink - 1, n_sink, n_sink + window - 1, n_sink + window,
                   Lc - gamma, Lc - gamma + 1, Lc - 1, Lc, L - 2, L - 1]
        for p in special + [int(x) for x in rng.integers(0, L, n_random)]:
            if 0 <= p < L:
                rows.add((b, int(rng.integers(0, Hq)), int(p)))
        p = int(rng.integers(0, L))
        rows |= {(b, h, p) for h in range(Hq)}
    return sorted(rows)


def stratified_rows(seqlens, Hq, window, n_sink, gamma, n_random=64, seed=0):
    """(b, h, i) triples, every query head and every row of whole groups of
    gamma rows, per sequence: the first 4 groups, the groups around the first
    anchor whose Delta is not zero (n_sink + window), the last 4 whole groups,
    n_random seeded groups, and the dense tail rows.  A whole group of all
    heads is a whole workgroup slab of the fused sparse kernel (the
    workloads' slabs hold gamma rows of every head of a GQA group), so every
    XCD's block range is covered.  Sorted by (b, h, i): the oracle evaluates
    each group's anchor rows once."""
    rng = np.random.default_rng(seed)
    rows = []
    for b, L in enumerate(seqlens):
        nA = L // gamma
        groups = set(range(min(4, nA))) | set(range(max(0, nA - 4), nA))
        c = (n_sink + window) // gamma
        groups |= {g for g in (c - 1, c, c + 1) if 0 <= g < nA}
        if nA:
            groups |= {int(g) for g in rng.integers(0, nA, n_random)}
        pos = [g * gamma + j for g in sorted(groups) for j in range(gamma)]
        pos += list(range(nA * gamma, L))
        rows += [(b, h, i) for h in range(Hq) for i in pos]
    return sorted(rows)


def gather_rows(out: torch.Tensor, cu, rows) -> np.ndarray:
    """out[cu[b] + i, h] for every (b, h, i), as fp64 [n, d]."""
    cu = [int(x) for x in cu]
    t = torch.tensor([cu[b] + i for (b, h, i) in rows], dtype=torch.long, device=out.device)
    hh = torch.tensor([h for (b, h, i) in rows], dtype=torch.long, device=out.device)
    return out[t, hh].float().cpu().numpy().astype(np.float64)


def errors(got: np.ndarray, ref: np.ndarray) -> dict:
    e = np.abs(got - ref)
    return {"max_abs": float(e.max()), "mean_abs": float(e.mean()),
            "rel_l2": float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)),
            "nan": int(np.isnan(got).sum())}


def bf16_half_ulp(x: np.ndarray) -> np.ndarray:
    """Half the spacing of bf16 values (8 significant bits) at |x|: the most one
    round-to-nearest to bf16 can move a value of that magnitude."""
    a = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.exp2(e - 8), 0.0)


def assert_parity(got, ref, what="", max_abs=MAX_ABS, mean_abs=MEAN_ABS, slack=None):
    """max-abs and mean-abs against the oracle; `slack` (elementwise, optional) is
    an extra rounding the computation is documented to make, forgiven in the
    max-abs check only."""
    if isinstance(got, torch.Tensor):
        got = got.float().cpu().numpy().astype(np.float64)
    err = errors(got, ref)
    assert err["nan"] == 0, f"{what}: NaN in output {err}"
    worst = err["max_abs"]
    if slack is not None:
        worst = float(np.max(np.maximum(np.abs(got - ref) - slack, 0.0)))
        err["max_abs_beyond_slack"] = worst
    assert worst <= max_abs and err["mean_abs"] <= mean_abs, f"{what}: {err}"
    return err


def to_oracle_bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor (any device) -> uint16 numpy bit patterns the oracle widens exactly."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
