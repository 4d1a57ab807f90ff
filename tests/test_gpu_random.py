"""Seeded random configurations against the fp64 oracle, over whole tensors.

Each case draws a batch and the method's parameters at random: one to three
sequences of 1..2000 tokens (equal lengths through the fixed-length call,
otherwise ragged through cu_seqlens), 1 or 2 kv heads with GQA ratios 1..8,
d = 64 or 128, windows from 1 key to past the longest sequence, 0..300 sinks
and gamma from 1 to past the longest sequence.  The sparse, dense and Delta
calls run through the C ABI, the Delta call in every schedule that applies
(default, unfused, and fused when supported), and every output element is
compared with the oracle.  Tolerances as elsewhere: max-abs 2e-2, mean-abs
2e-3, the max-abs bound taken on top of the output's own bf16 rounding (half a
bf16 ulp of the exact result: with a one-key window outputs reach 8 and more,
where that rounding alone passes 2e-2) and, for the unfused schedule, of its
second rounding (the sparse row is stored in bf16 before Delta is added), up
to half a bf16 ulp of the sparse value.  A second test draws key-block-list
configurations the same way (top-k, vertical-slash and Star layouts), and a
third longer ones, of 2.5K-24K tokens, whose dense rows span several key
chunks, and a fourth edge-shaped ones (empty sequences, GQA ratios 5-7,
sinks and gamma past the sequence).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from sampling import assert_parity, bf16_half_ulp, to_oracle_bits

pytestmark = pytest.mark.gpu


def draw(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 4))
    if rng.random() < 0.3:
        seqlens = (int(rng.integers(1, 1200)),) * B
    else:
        seqlens = tuple(int(x) for x in rng.integers(1, 2000, B))
    Hkv = int(rng.choice([1, 2]))
    G = int(rng.choice([1, 2, 3, 4, 8]))
    d = int(rng.choice([64, 128]))
    Lmax = max(seqlens)
    window = int(rng.choice([1, int(rng.integers(1, 600)), int(rng.integers(1, 600)),
                             Lmax + int(rng.integers(0, 50))]))
    n_sink = int(rng.choice([0, int(rng.integers(0, 8)), int(rng.integers(0, 8)),
                             int(rng.integers(0, 300))]))
    gamma = int(rng.choice([1, 2, int(rng.integers(3, 130)), int(rng.integers(3, 130)), 64,
                            Lmax + 1]))
    return seqlens, Hkv * G, Hkv, d, window, n_sink, gamma


def rounding_slack(ref, ref_sp, unfused):
    """Roundings the Delta outputs are documented to make beyond the computation,
    forgiven in the max-abs check.  Every schedule stores its output in bf16: the
    exact result is not representable, and its nearest bf16 value lies up to half
    a bf16 ulp away (0.031 for outputs in [8, 16), which a one-key window makes
    possible: there the output is v_i + Delta, a sum of unit normals rather than
    an average).  The unfused schedule also stores the sparse row in bf16 before
    adding Delta: a second rounding, up to half a bf16 ulp of the sparse value."""
    slack = bf16_half_ulp(ref)
    return slack + bf16_half_ulp(ref_sp) if unfused else slack


def draw_long(seed):
    """A configuration long enough for several key chunks per dense row (a chunk
    holds at least 2560 keys): 2.5K-24K tokens, GQA 1-4, gamma 8-129."""
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 4))
    if rng.random() < 0.4:
        seqlens = (int(rng.integers(2500, 16000)),) * B
    else:
        seqlens = tuple(int(x) for x in rng.integers(1, 24000, B))
    Hkv = int(rng.choice([1, 2]))
    G = int(rng.choice([1, 2, 4]))
    d = int(rng.choice([64, 64, 128]))
    Lmax = max(seqlens)
    window = int(rng.choice([1, int(rng.integers(1, 1100)), int(rng.integers(1, 1100)),
                             Lmax + int(rng.integers(0, 50))]))
    n_sink = int(rng.choice([0, int(rng.integers(0, 8)), int(rng.integers(0, 300))]))
    gamma = int(rng.choice([8, 16, int(rng.integers(8, 130)), 64]))
    return seqlens, Hkv * G, Hkv, d, window, n_sink, gamma


def draw_edge(seed):
    """An edge-shaped configuration: ragged batches of up to 4 with empty
    sequences, every GQA ratio 1-8 over up to 3 kv heads, sinks up to 2000
    (past the sequence), gamma up to three times the longest sequence."""
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 5))
    seqlens = [int(x) for x in rng.integers(1, 1500, B)]
    for i in range(B):
        if rng.random() < 0.3:
            seqlens[i] = 0
    if max(seqlens) == 0:
        seqlens[int(rng.integers(0, B))] = int(rng.integers(1, 1500))
    seqlens = tuple(seqlens)
    Hkv = int(rng.choice([1, 2, 3]))
    G = int(rng.integers(1, 9))
    d = int(rng.choice([64, 128]))
    Lmax = max(seqlens)
    window = int(rng.choice([1, int(rng.integers(1, 600)), Lmax + int(rng.integers(0, 50))]))
    n_sink = int(rng.choice([0, int(rng.integers(0, 8)), int(rng.integers(0, 2000))]))
    gamma = int(rng.choice([1, 2, int(rng.integers(3, 130)), Lmax + 1, 3 * Lmax + 7]))
    return seqlens, Hkv * G, Hkv, d, window, n_sink, gamma


SEEDS = list(range(100, 132))
LONG_SEEDS = [30000, 30003, 30007, 30008, 30010, 30011, 30012, 30015]
# empty sequences with: sinks and gamma past the sequence; G 5 on 3 kv heads; G 7
# with sinks past it; G 6 on 3 kv heads with gamma 2; G 7, gamma past it; G 5
EDGE_SEEDS = [80004, 80012, 80013, 80028, 80041, 80054]


@pytest.mark.parametrize("seed", SEEDS)
def test_random_configuration_matches_oracle(seed):
    check_configuration(seed, draw(seed))


@pytest.mark.parametrize("seed", LONG_SEEDS)
def test_random_long_configuration_matches_oracle(seed):
    check_configuration(seed, draw_long(seed))


@pytest.mark.parametrize("seed", EDGE_SEEDS)
def test_random_edge_configuration_matches_oracle(seed):
    check_configuration(seed, draw_edge(seed))


def check_configuration(seed, cfg):
    from paper_2505_11254_amd import binding as lib
    from paper_2505_11254_amd.inputs import random_qkv
    seqlens, Hq, Hkv, d, w, s, gamma = cfg
    print(f"seed {seed}: seqlens={seqlens} Hq={Hq} Hkv={Hkv} d={d} window={w} n_sink={s} "
          f"gamma={gamma}", flush=True)
    q, k, v, cu = random_qkv(seqlens, Hq, Hkv, d, seed=seed)
    qd, kd, vd, cud = (x.cuda() for x in (q, k, v, cu))
    fixed = len(set(seqlens)) == 1
    N = max(seqlens)
    kw = dict(B=len(seqlens)) if fixed else dict(cu_seqlens=cud, max_seqlen=N)
    sp = lib.sparse_attn_prefill(qd, kd, vd, window=w, n_sink=s, **kw)
    de = lib.dense_causal_attn_prefill(qd, kd, vd, **kw)
    runs = {"default": lib.delta_attn_prefill(qd, kd, vd, window=w, n_sink=s, gamma=gamma, **kw)}
    schedules = [("unfused", lib.STEP_ALL)]
    if lib.fused_supported(Hq, Hkv, gamma):
        schedules.append(("fused", lib.STEP_ALL | lib.STEP_FUSED))
    for name, steps in schedules:
        out = torch.full_like(qd, float("nan"))
        ws = torch.full((lib.workspace_bytes(len(seqlens), N, Hq, Hkv, d, gamma) // 4,),
                        float("nan"), device=qd.device)
        lib.delta_attn_prefill_steps(qd, kd, vd, out, ws, steps, window=w, n_sink=s, gamma=gamma,
                                     B=len(seqlens), cu_seqlens=None if fixed else cud,
                                     max_seqlen=N)
        runs[name] = out
    torch.cuda.synchronize()
    bits = [to_oracle_bits(x) for x in (q, k, v)]
    cun = cu.numpy().astype(np.int64)
    ref, ref_sp, _ = oracle.delta_attention(*bits, cun, window=w, n_sink=s, gamma=gamma,
                                            return_parts=True)
    assert_parity(sp, ref_sp, f"seed {seed} sparse")
    assert_parity(de, oracle.attention(*bits, cun, mode=oracle.MODE_DENSE), f"seed {seed} dense")
    for name, out in runs.items():
        assert_parity(out, ref, f"seed {seed} delta ({name})",
                      slack=rounding_slack(ref, ref_sp, unfused=name == "unfused" or (
                          name == "default" and not lib.fused_supported(Hq, Hkv, gamma))))


def draw_lists(seed):
    """A random block-list configuration: batch, heads, query block size, gamma and
    a list layout with random parameters."""
    from paper_2505_11254_amd import blocklists as BL
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 4))
    seqlens = tuple(int(x) for x in rng.integers(1, 2000, B))
    Hkv = int(rng.choice([1, 2]))
    G = int(rng.choice([1, 2, 4, 8]))
    d = int(rng.choice([64, 128]))
    # the list mode needs each workgroup's rows of a head (256 / h of them, h the
    # heads of a GQA group sharing a workgroup) inside one query block
    h = 1
    while h * 2 <= 8 and G % (h * 2) == 0:
        h *= 2
    block_q = int(rng.choice([bq for bq in (64, 128, 256) if bq >= 256 // h]))
    gamma = int(rng.choice([1, 2, int(rng.integers(3, 130)), 64, max(seqlens) + 1]))
    kind = int(rng.integers(0, 3))
    if kind == 0:
        bl = BL.block_topk(seqlens, Hkv, block_q, k=int(rng.integers(1, 12)), seed=seed)
    elif kind == 1:
        bl = BL.vertical_slash(seqlens, Hkv, block_q, n_vertical=int(rng.integers(0, 6)),
                               n_local=int(rng.integers(0, 6)),
                               slash_offsets=tuple(int(x) for x in rng.integers(1, 40, 2)),
                               seed=seed)
    else:
        bl = BL.star(seqlens, Hkv, block_q, anchor=64 * int(rng.integers(1, 8)),
                     context=block_q * int(rng.integers(1, 4)))
    return seqlens, Hkv * G, Hkv, d, block_q, gamma, bl


LIST_SEEDS = list(range(200, 216))


@pytest.mark.parametrize("seed", LIST_SEEDS)
def test_random_block_lists_match_oracle(seed):
    from paper_2505_11254_amd import binding as lib
    from paper_2505_11254_amd.inputs import random_qkv
    seqlens, Hq, Hkv, d, block_q, gamma, bl = draw_lists(seed)
    print(f"seed {seed}: seqlens={seqlens} Hq={Hq} Hkv={Hkv} d={d} block_q={block_q} "
          f"gamma={gamma} nnz={bl.idx.size}", flush=True)
    q, k, v, cu = random_qkv(seqlens, Hq, Hkv, d, seed=seed)
    qd, kd, vd, cud = (x.cuda() for x in (q, k, v, cu))
    ptr, idx = bl.to("cuda")
    N = max(seqlens)
    kw = dict(cu_seqlens=cud, max_seqlen=N)
    lkw = dict(block_q=block_q, block_ptr=ptr, block_idx=idx)
    sp = lib.blocksparse_attn_prefill(qd, kd, vd, **lkw, **kw)
    fused_ok = lib.fused_supported_blocksparse(Hq, Hkv, gamma, block_q)
    runs = {}
    for name, steps in [("default", 0), ("unfused", lib.STEP_ALL)] + (
            [("fused", lib.STEP_ALL | lib.STEP_FUSED)] if fused_ok else []):
        out = torch.full_like(qd, float("nan"))
        ws = torch.full((lib.workspace_bytes(len(seqlens), N, Hq, Hkv, d, gamma) // 4,),
                        float("nan"), device=qd.device)
        runs[name] = lib.delta_attn_prefill_blocksparse(qd, kd, vd, gamma=gamma, out=out,
                                                         workspace=ws, steps=steps, **lkw, **kw)
    torch.cuda.synchronize()
    bits = [to_oracle_bits(x) for x in (q, k, v)]
    ref, ref_sp, _ = oracle.block_delta_attention(*bits, cu.numpy().astype(np.int64),
                                                  blk_ptr=bl.ptr, blk_idx=bl.idx,
                                                  block_q=block_q, gamma=gamma, return_parts=True)
    assert_parity(sp, ref_sp, f"seed {seed} sparse (lists)")
    for name, out in runs.items():
        assert_parity(out, ref, f"seed {seed} delta over lists ({name})",
                      slack=rounding_slack(ref, ref_sp, unfused=name == "unfused" or (
                          name == "default" and not fused_ok)))
