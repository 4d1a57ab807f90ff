"""GPU parity of the fused schedule (dense rows and their merge first, then
the sparse kernel storing bf16(sparse + Delta) itself) against the fp64
oracle and against the unfused schedule, through the C ABI.

Both schedules evaluate Eq. 6; they differ only in rounding: the unfused
one rounds the sparse row to bf16 before adding Delta and rounds again, the
fused one rounds once.  Rows that take no Delta (covered groups), anchor
rows (the dense row) and dense tail rows are bitwise equal under both.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from sampling import assert_parity, to_oracle_bits

pytestmark = pytest.mark.gpu

# (seqlens, Hq, Hkv, d, window, n_sink, gamma): each gamma divides the row
# slab of the fused sparse workgroup for that GQA ratio
CASES = [
    ((777,), 8, 2, 128, 100, 5, 64),              # G 4, 9 dense tail rows
    ((1000, 1, 513, 64), 8, 1, 128, 64, 16, 32),  # varlen, G 8: 32-row slabs, one group each
    ((600,), 4, 4, 64, 40, 2, 8),                 # G 1: 256-row slabs, 32 groups each
    ((300,), 4, 2, 128, 32, 8, 1),                # gamma 1: every row its own anchor
    ((2100,), 4, 1, 128, 128, 4, 128),            # G 4 with gamma 128: two heads per block
    ((3000,), 4, 1, 128, 256, 16, 256),           # gamma 256: one head per block
    ((500,), 2, 1, 64, 16, 2, 2),                 # gamma 2, d 64: the largest LDS exchange
    ((700,), 1, 1, 128, 50, 3, 2),                # gamma 2, d 128: the largest LDS exchange
    ((0, 450, 0, 64), 8, 2, 128, 64, 8, 32),      # empty sequences inside a ragged batch
    # equal lengths through the fixed-length call, several key chunks per dense
    # row: the strided blocks run whole-chunk (row tile, chunk) pairs first
    ((5000, 5000, 5000), 8, 2, 128, 256, 16, 16),  # 3 chunks of 1728 keys, 8 tail rows
    ((4100, 4100), 4, 4, 64, 96, 4, 64),           # G 1, d 64: 3 chunks, 4 tail rows
]


@pytest.fixture(scope="module")
def lib():
    assert torch.cuda.is_available()
    from paper_2505_11254_amd import binding
    binding.load_library()
    return binding


def _run(lib, q, k, v, kw, w, s, gamma, steps):
    from paper_2505_11254_amd import binding
    B_, N = (kw["B"], q.shape[0] // kw["B"]) if "B" in kw else (len(kw["cu_seqlens"]) - 1,
                                                                 kw["max_seqlen"])
    out = torch.full_like(q, float("nan"))
    ws = torch.full((binding.workspace_bytes(B_, N, q.shape[1], k.shape[1], q.shape[2], gamma)
                     // 4,), float("nan"), device=q.device)
    lib.delta_attn_prefill_steps(q, k, v, out, ws, steps, window=w, n_sink=s, gamma=gamma,
                                 B=kw.get("B"), cu_seqlens=kw.get("cu_seqlens"), max_seqlen=N)
    return out


@pytest.mark.parametrize("case", CASES, ids=[f"L{c[0]}-H{c[1]}/{c[2]}-d{c[3]}-g{c[6]}"
                                             for c in CASES])
def test_fused_schedule_matches_oracle_and_unfused(lib, case):
    from paper_2505_11254_amd.inputs import random_qkv
    seqlens, Hq, Hkv, d, w, s, gamma = case
    assert lib.fused_supported(Hq, Hkv, gamma)
    q, k, v, cu = random_qkv(seqlens, Hq, Hkv, d, seed=31 + gamma + len(seqlens))
    qd, kd, vd, cud = (x.cuda() for x in (q, k, v, cu))
    fixed = len(set(seqlens)) == 1
    kw = dict(B=len(seqlens)) if fixed else dict(cu_seqlens=cud, max_seqlen=max(seqlens))
    fused = _run(lib, qd, kd, vd, kw, w, s, gamma, lib.STEP_ALL | lib.STEP_FUSED)
    unfused = _run(lib, qd, kd, vd, kw, w, s, gamma, lib.STEP_ALL)
    default = lib.delta_attn_prefill(qd, kd, vd, window=w, n_sink=s, gamma=gamma, **kw)
    sp = lib.sparse_attn_prefill(qd, kd, vd, window=w, n_sink=s, **kw)
    torch.cuda.synchronize()
    assert torch.equal(default, fused), "the whole-path call takes the fused schedule"

    bits = [to_oracle_bits(x) for x in (q, k, v)]
    cun = cu.numpy().astype(np.int64)
    ref = oracle.delta_attention(*bits, cun, window=w, n_sink=s, gamma=gamma)
    assert_parity(fused, ref, "fused schedule")
    assert_parity(unfused, ref, "unfused schedule")

    # local position and group of every token row
    pos = np.concatenate([np.arange(L) for L in seqlens])
    Ls = np.concatenate([np.full(L, L) for L in seqlens])
    Lc = (Ls // gamma) * gamma
    anc = pos - pos % gamma
    open_group = (pos < Lc) & (anc >= s + w)
    same = torch.from_numpy(~open_group | (pos == anc) | (pos >= Lc))
    assert torch.equal(fused[same.cuda()], unfused[same.cuda()])
    # covered groups keep the sparse rows bit for bit
    cov = torch.from_numpy((pos < Lc) & ~open_group).cuda()
    assert torch.equal(fused[cov], sp[cov])
    # elsewhere the two differ by their roundings only: unfused rounds the
    # sparse row (half an ulp of it) and then the sum, fused rounds the sum
    diff = (fused.float() - unfused.float()).abs()
    bound = sp.float().abs() * 2.0 ** -8 + torch.maximum(fused.float().abs(),
                                                         unfused.float().abs()) * 2.0 ** -7
    # (the factor covers the (1 + 2^-8) terms of the bound's derivation)
    assert bool((diff <= bound * 1.01 + 1e-12).all()), float((diff - bound).max())


def test_recompute_fused_matches_oracle(lib):
    from paper_2505_11254_amd.inputs import random_qkv
    seqlens, Hq, Hkv, d, w, s, gamma = (1500,), 8, 2, 128, 96, 4, 64
    q, k, v, cu = random_qkv(seqlens, Hq, Hkv, d, seed=5)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    got = lib.delta_attn_prefill_correction(qd, kd, vd, window=w, n_sink=s, gamma=gamma,
                                            mode=lib.CORR_RECOMPUTE)
    sp = lib.sparse_attn_prefill(qd, kd, vd, window=w, n_sink=s)
    torch.cuda.synchronize()
    ref = oracle.delta_attention_variant(*(to_oracle_bits(x) for x in (q, k, v)),
                                         cu.numpy().astype(np.int64), window=w, n_sink=s,
                                         gamma=gamma, mode=1, params=(0.0, 0.0, 0.0))
    assert_parity(got, ref, "recompute, fused")
    rows = torch.arange(seqlens[0], device="cuda")
    Lc = (seqlens[0] // gamma) * gamma
    keep = (rows % gamma != 0) & (rows < Lc)
    assert torch.equal(got[keep], sp[keep])


def test_unsupported_gamma_keeps_the_unfused_schedule(lib):
    from paper_2505_11254_amd.inputs import random_qkv
    seqlens, Hq, Hkv, d, w, s, gamma = (900,), 6, 3, 128, 64, 4, 48  # G 2: slabs of 128/256
    assert not lib.fused_supported(Hq, Hkv, gamma)
    q, k, v, cu = random_qkv(seqlens, Hq, Hkv, d, seed=6)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    default = lib.delta_attn_prefill(qd, kd, vd, window=w, n_sink=s, gamma=gamma)
    unfused = _run(lib, qd, kd, vd, dict(B=1), w, s, gamma, lib.STEP_ALL)
    torch.cuda.synchronize()
    assert torch.equal(default, unfused)
