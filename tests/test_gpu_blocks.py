"""GPU parity of Delta Attention over key-block-list sparse bases (f* from
per-query-block key tiles) against the fp64 oracle, through the C ABI.

Small cases are compared over whole tensors, for the sparse kernel alone and
for the Delta path in both schedules; a 131K Llama-shaped case with
vertical-slash lists is compared on sampled rows.  Tolerances as for the
sink + window basis: max-abs 2e-2, mean-abs 2e-3.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from sampling import assert_parity, gather_rows, sample_rows, to_oracle_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    assert torch.cuda.is_available()
    from paper_2505_11254_amd import binding
    binding.load_library()
    return binding


def lists(kind, seqlens, Hkv, block_q, seed):
    from paper_2505_11254_amd import blocklists as BL
    if kind == "vertical_slash":
        return BL.vertical_slash(seqlens, Hkv, block_q, n_vertical=4, n_local=3,
                                 slash_offsets=(7, 20), seed=seed)
    if kind == "topk":
        return BL.block_topk(seqlens, Hkv, block_q, k=5, seed=seed)
    if kind == "star":
        return BL.star(seqlens, Hkv, block_q, anchor=256, context=512)
    if kind == "full":
        return BL.full(seqlens, Hkv, block_q)
    if kind == "empty":
        return BL.empty(seqlens, Hkv, block_q)
    if kind == "junk":
        # valid lists plus entries the key set skips: negative, inside and past the
        # query block (the kernel must skip them, not fetch them)
        bl = BL.block_topk(seqlens, Hkv, block_q, k=3, seed=seed)
        rng = np.random.default_rng(seed)
        ptr = np.zeros_like(bl.ptr)
        idx = []
        for b in range(bl.ptr.shape[0]):
            for g in range(Hkv):
                for qb in range(bl.nqb):
                    ptr[b, g, qb] = len(idx)
                    t = [-5] + list(bl.tiles(b, g, qb))
                    t.append(qb * block_q // 64 + int(rng.integers(0, 4)))
                    t.append(1 << 20)
                    idx.extend(t)
                ptr[b, g, bl.nqb] = len(idx)
        return BL.BlockLists(block_q, ptr, np.asarray(idx, dtype=np.int32))
    raise ValueError(kind)


# (seqlens, Hq, Hkv, d, block_q, gamma, list kind)
CASES = [
    ((777,), 8, 2, 128, 64, 64, "vertical_slash"),          # G 4, 9 dense tail rows
    ((1000, 1, 513, 64), 8, 1, 128, 64, 32, "topk"),        # varlen, G 8: 32-row slabs
    ((1500,), 2, 2, 64, 256, 16, "star"),                   # G 1: 256-row slabs
    ((900,), 4, 2, 128, 128, 8, "junk"),                    # G 2, skipped entries
    ((600,), 8, 2, 128, 64, 64, "full"),                    # every tile: dense attention
    ((600,), 8, 2, 64, 64, 16, "empty"),                    # own query block only
    ((1100,), 4, 1, 128, 256, 48, "vertical_slash"),        # gamma fits no slab: unfused
    ((0, 700, 0, 90), 8, 2, 128, 64, 32, "topk"),           # empty sequences in the batch
]


def _run(lib, q, k, v, kw, block_q, ptr, idx, gamma, steps):
    from paper_2505_11254_amd import binding
    B_, N = (kw["B"], q.shape[0] // kw["B"]) if "B" in kw else (len(kw["cu_seqlens"]) - 1,
                                                                 kw["max_seqlen"])
    out = torch.full_like(q, float("nan"))
    ws = torch.full((binding.workspace_bytes(B_, N, q.shape[1], k.shape[1], q.shape[2], gamma)
                     // 4,), float("nan"), device=q.device)
    return lib.delta_attn_prefill_blocksparse(q, k, v, block_q=block_q, block_ptr=ptr,
                                              block_idx=idx, gamma=gamma, out=out, workspace=ws,
                                              steps=steps, **kw)


@pytest.mark.parametrize("case", CASES, ids=[f"L{c[0]}-H{c[1]}/{c[2]}-d{c[3]}-bq{c[4]}-g{c[5]}-"
                                             f"{c[6]}" for c in CASES])
def test_block_lists_match_oracle(lib, case):
    from paper_2505_11254_amd.inputs import random_qkv
    seqlens, Hq, Hkv, d, block_q, gamma, kind = case
    q, k, v, cu = random_qkv(seqlens, Hq, Hkv, d, seed=sum(seqlens) + block_q)
    bl = lists(kind, seqlens, Hkv, block_q, seed=len(seqlens) + gamma)
    qd, kd, vd, cud = (x.cuda() for x in (q, k, v, cu))
    ptr, idx = bl.to("cuda")
    kw = (dict(cu_seqlens=cud, max_seqlen=max(seqlens)) if len(seqlens) > 1 else dict(B=1))
    sp = lib.blocksparse_attn_prefill(qd, kd, vd, block_q=block_q, block_ptr=ptr, block_idx=idx,
                                      **kw)
    default = _run(lib, qd, kd, vd, kw, block_q, ptr, idx, gamma, 0)
    unfused = _run(lib, qd, kd, vd, kw, block_q, ptr, idx, gamma, lib.STEP_ALL)
    fused = None
    if lib.fused_supported_blocksparse(Hq, Hkv, gamma, block_q):
        fused = _run(lib, qd, kd, vd, kw, block_q, ptr, idx, gamma, lib.STEP_ALL | lib.STEP_FUSED)
    torch.cuda.synchronize()
    bits = [to_oracle_bits(x) for x in (q, k, v)]
    cun = cu.numpy().astype(np.int64)
    ref, ref_sp, _ = oracle.block_delta_attention(*bits, cun, blk_ptr=bl.ptr, blk_idx=bl.idx,
                                                  block_q=block_q, gamma=gamma,
                                                  return_parts=True)
    assert_parity(sp, ref_sp, f"{kind} sparse kernel")
    assert_parity(default, ref, f"{kind} delta path")
    assert_parity(unfused, ref, f"{kind} delta path, unfused")
    if fused is not None:
        assert_parity(fused, ref, f"{kind} delta path, fused")
        assert torch.equal(default, fused)
    else:
        assert torch.equal(default, unfused)
    if kind == "full":  # f* is dense attention: the sparse kernel matches the dense one
        de = lib.dense_causal_attn_prefill(qd, kd, vd, **kw)
        torch.cuda.synchronize()
        assert_parity(sp, oracle.attention(*bits, cun, mode=oracle.MODE_DENSE), "full lists")
        assert (sp.float() - de.float()).abs().max().item() <= 2e-2


@pytest.mark.timeout(600)
def test_block_lists_131k_sampled(lib):
    from paper_2505_11254_amd import WORKLOADS
    from paper_2505_11254_amd import blocklists as BL
    from paper_2505_11254_amd.inputs import generate
    wl = WORKLOADS["llama8b_layer_131k"]
    q, k, v, cu = generate(wl, device="cuda")
    bl = BL.vertical_slash(wl.seqlens, wl.Hkv, 64, n_vertical=8, n_local=24,
                           slash_offsets=(64, 256), seed=5)
    ptr, idx = bl.to("cuda")
    out = lib.delta_attn_prefill_blocksparse(q, k, v, block_q=64, block_ptr=ptr, block_idx=idx,
                                             gamma=wl.gamma, B=wl.B)
    torch.cuda.synchronize()
    cun = wl.cu_seqlens()
    rows = sample_rows(wl.seqlens, wl.Hq, 64 * 24, 64, wl.gamma, n_random=64, seed=3)
    got = gather_rows(out, cun, rows)
    del out
    bits = [to_oracle_bits(x) for x in (q, k, v)]
    del q, k, v
    torch.cuda.empty_cache()
    ref = oracle.block_delta_attention_rows(*bits, np.asarray(cun, dtype=np.int64),
                                            blk_ptr=bl.ptr, blk_idx=bl.idx, block_q=64,
                                            gamma=wl.gamma, rows=rows)
    err = assert_parity(got, ref, f"131K vertical-slash lists ({len(rows)} rows)")
    print(f"131K vertical-slash delta path vs oracle on {len(rows)} rows: {err}", flush=True)
