"""GPU parity of the correction variants (recompute, interpolation, EMA,
alpha-beta-gamma filter) against the fp64 oracle, through the C ABI."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from sampling import assert_parity, to_oracle_bits

pytestmark = pytest.mark.gpu

# parameter settings of the paper's interpolation table, plus edge values
MODES = [
    (0, (0.0, 0.0, 0.0)), (1, (0.0, 0.0, 0.0)), (2, (0.0, 0.0, 0.0)),
    (3, (0.5, 0.0, 0.0)), (3, (0.95, 0.0, 0.0)), (3, (1.0, 0.0, 0.0)), (3, (0.0, 0.0, 0.0)),
    (4, (0.05, 1.25e-4, 2.08e-5)), (4, (0.2, 5e-2, 3.5e-3)), (4, (1.0, 0.0, 0.0)),
]
CASES = [
    ((777,), 8, 2, 128, 100, 5, 64),
    ((1000, 1, 513, 64), 8, 1, 128, 64, 16, 32),
    ((600,), 4, 4, 64, 40, 2, 8),
    ((300,), 2, 1, 128, 32, 8, 1),
    ((8192,), 8, 2, 128, 1024, 64, 64),   # 128 anchors through the recurrences
]


@pytest.fixture(scope="module")
def lib():
    assert torch.cuda.is_available()
    from paper_2505_11254_amd import binding
    binding.load_library()
    return binding


@pytest.mark.parametrize("case", CASES, ids=[f"L{c[0]}-g{c[6]}" for c in CASES])
def test_variants_match_oracle(lib, case):
    from paper_2505_11254_amd.inputs import random_qkv
    seqlens, Hq, Hkv, d, w, s, gamma = case
    q, k, v, cu = random_qkv(seqlens, Hq, Hkv, d, seed=len(seqlens) + gamma)
    qd, kd, vd, cud = (x.cuda() for x in (q, k, v, cu))
    kw = (dict(cu_seqlens=cud, max_seqlen=max(seqlens)) if len(seqlens) > 1 else dict(B=1))
    bits = [to_oracle_bits(x) for x in (q, k, v)]
    cun = cu.numpy().astype(np.int64)
    base = lib.delta_attn_prefill(qd, kd, vd, window=w, n_sink=s, gamma=gamma, **kw)
    for mode, params in MODES:
        got = lib.delta_attn_prefill_correction(qd, kd, vd, window=w, n_sink=s, gamma=gamma,
                                                mode=mode, params=params, **kw)
        torch.cuda.synchronize()
        ref = oracle.delta_attention_variant(*bits, cun, window=w, n_sink=s, gamma=gamma,
                                             mode=mode, params=params)
        assert_parity(got, ref, f"mode {mode} {params}")
        if mode == 0:
            assert torch.equal(got, base)


def test_recompute_keeps_sparse_rows_bitwise(lib):
    from paper_2505_11254_amd.inputs import random_qkv
    q, k, v, cu = random_qkv((2048,), 4, 1, 128, seed=9)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    sp = lib.sparse_attn_prefill(qd, kd, vd, window=128, n_sink=4)
    rc = lib.delta_attn_prefill_correction(qd, kd, vd, window=128, n_sink=4, gamma=32, mode=1)
    torch.cuda.synchronize()
    rows = torch.arange(2048, device="cuda")
    assert torch.equal(rc[rows % 32 != 0], sp[rows % 32 != 0])
    assert not torch.equal(rc[rows % 32 == 0], sp[rows % 32 == 0])
