"""The Delta path inside a captured HIP graph.

The path allocates nothing and records no memset (the caller passes the
workspace), so a caller can capture it once and replay it.  Each replay is
checked against the eager call, with eager work and synchronisation between
replays and with the inputs rewritten in place between them.
"""
from __future__ import annotations

import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    assert torch.cuda.is_available()
    from paper_2505_11254_amd import binding
    binding.load_library()
    return binding


# (L, Hq, Hkv, d, window, n_sink, gamma): fused schedule, unfused schedule
CASES = [(4096, 8, 2, 128, 512, 16, 64), (3000, 6, 3, 128, 256, 8, 48)]


@pytest.mark.parametrize("case", CASES, ids=["fused", "unfused"])
def test_delta_path_replays_in_a_graph(lib, case):
    from paper_2505_11254_amd.inputs import random_qkv
    L, Hq, Hkv, d, w, s, gamma = case
    q, k, v, _ = random_qkv((L,), Hq, Hkv, d, seed=21, device="cuda")
    q2, k2, v2, _ = random_qkv((L,), Hq, Hkv, d, seed=22, device="cuda")
    ws = torch.empty(lib.workspace_bytes(1, L, Hq, Hkv, d, gamma), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty_like(q)
    kw = dict(window=w, n_sink=s, gamma=gamma, B=1)
    ref1 = lib.delta_attn_prefill(q, k, v, **kw)
    ref2 = lib.delta_attn_prefill(q2, k2, v2, **kw)
    torch.cuda.synchronize()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm the call on the capturing stream
        lib.delta_attn_prefill(q, k, v, out=out, workspace=ws, **kw)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        lib.delta_attn_prefill(q, k, v, out=out, workspace=ws, **kw)

    qs, ks, vs = q.clone(), k.clone(), v.clone()
    for rep in range(4):
        src = (q2, k2, v2) if rep % 2 else (qs, ks, vs)
        for dst, x in zip((q, k, v), src):
            dst.copy_(x)
        out.fill_(float("nan"))
        ws.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref2 if rep % 2 else ref1), f"replay {rep}"
