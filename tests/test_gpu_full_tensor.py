"""Whole output tensors of the large workloads against the oracle: every row of
the chosen query heads, in the fused (default) and the unfused schedule.

The oracle evaluates one head per call through its row entry point, which
takes minutes per workload on the host (about 4 s per head at 131K, 13 s for
the ragged batch, 150 s at 1M on 16 threads), so the test runs only when
DA_FULL_TENSOR is set:

    DA_FULL_TENSOR=1 python -m pytest tests/test_gpu_full_tensor.py -m gpu -s

DA_FULL_TENSOR_HEADS (comma-separated) picks the heads; by default every head
at 131K and for the ragged batch, and at 1M one head of each kv head's query
group (heads 0, 4, ..., 28: each kv head's workgroups run on their own XCD).
"""
from __future__ import annotations

import os
import time

import numpy as np
import pytest
import torch

import oracle
from sampling import MAX_ABS, MEAN_ABS, to_oracle_bits

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not os.environ.get("DA_FULL_TENSOR"),
                                 reason="minutes of oracle time per workload: set DA_FULL_TENSOR=1")]


def _heads(wl, default):
    env = os.environ.get("DA_FULL_TENSOR_HEADS")
    return [int(x) for x in env.split(",")] if env else default


@pytest.mark.parametrize("name", ["llama8b_layer_131k", "ragged_b4_gqa8", "llama8b_layer_1m"])
def test_whole_output_matches_oracle(name):
    from paper_2505_11254_amd import WORKLOADS
    from paper_2505_11254_amd import binding as lib
    from paper_2505_11254_amd.inputs import generate
    wl = WORKLOADS[name]
    heads = _heads(wl, list(range(0, wl.Hq, wl.Hq // wl.Hkv)) if name.endswith("_1m")
                   else list(range(wl.Hq)))
    q, k, v, cu = generate(wl, device="cuda")
    kw = dict(B=wl.B) if wl.fixed_length else dict(cu_seqlens=cu, max_seqlen=wl.max_seqlen)
    out = lib.delta_attn_prefill(q, k, v, window=wl.window, n_sink=wl.n_sink, gamma=wl.gamma, **kw)
    ws = torch.empty(lib.workspace_bytes(wl.B, wl.max_seqlen, wl.Hq, wl.Hkv, wl.d, wl.gamma),
                     dtype=torch.uint8, device="cuda")
    out_u = torch.full_like(q, float("nan"))
    lib.delta_attn_prefill_steps(q, k, v, out_u, ws, lib.STEP_ALL, window=wl.window,
                                 n_sink=wl.n_sink, gamma=wl.gamma, B=wl.B,
                                 cu_seqlens=None if wl.fixed_length else cu,
                                 max_seqlen=wl.max_seqlen)
    torch.cuda.synchronize()
    got = {"fused": out.float().cpu().numpy(), "unfused": out_u.float().cpu().numpy()}
    qb, kb, vb = (to_oracle_bits(x) for x in (q, k, v))
    del q, k, v, out, out_u, ws, cu
    torch.cuda.empty_cache()
    cu64 = np.asarray(wl.cu_seqlens(), dtype=np.int64)
    T = int(cu64[-1])
    worst = {s: 0.0 for s in got}
    total = {s: 0.0 for s in got}
    t0 = time.time()
    for h in heads:
        # rows in token order, so that they line up with out[:, h]
        rows = [(b, h, i) for b in range(len(cu64) - 1) for i in range(int(cu64[b + 1] - cu64[b]))]
        ref = oracle.delta_attention_rows(qb, kb, vb, cu64, window=wl.window, n_sink=wl.n_sink,
                                          gamma=wl.gamma, rows=rows)
        for s, g in got.items():
            e = np.abs(g[:, h, :].astype(np.float64) - ref)
            worst[s] = max(worst[s], float(e.max()))
            total[s] += float(e.sum())
        print(f"{name} head {h}: max-abs fused {worst['fused']:.2e} unfused {worst['unfused']:.2e} "
              f"(so far), {time.time() - t0:.0f} s", flush=True)
    n = T * len(heads) * wl.d
    for s in got:
        print(f"{name} {s}: heads {heads}, {T} rows x {wl.d}: max-abs {worst[s]:.3e}, "
              f"mean-abs {total[s] / n:.3e}", flush=True)
        assert worst[s] <= MAX_ABS and total[s] / n <= MEAN_ABS, (s, worst[s], total[s] / n)
