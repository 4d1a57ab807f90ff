"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Small cases are compared element by element over whole tensors; the
workload-sized cases on sampled rows the oracle evaluates one by one.
Tolerances: max-abs 2e-2 and mean-abs 2e-3 (bf16 I/O, fp32 accumulation).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from sampling import assert_parity, gather_rows, sample_rows, stratified_rows, to_oracle_bits

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_11254_amd import binding
    binding.load_library()
    props = torch.cuda.get_device_properties(0)
    assert "gfx950" in props.gcnArchName, props.gcnArchName


def B():
    from paper_2505_11254_amd import binding
    return binding


def make(seqlens, Hq, Hkv, d, seed, std=1.0):
    from paper_2505_11254_amd.inputs import random_qkv
    q, k, v, cu = random_qkv(seqlens, Hq, Hkv, d, seed, device="cpu", std=std)
    return q, k, v, cu


def run_all(q, k, v, cu, w, s, gamma):
    """Sparse, dense and Delta outputs of the HIP path (on the GPU)."""
    qd, kd, vd, cud = (x.to(DEV) for x in (q, k, v, cu))
    maxL = int((cu[1:] - cu[:-1]).max())
    kw = dict(cu_seqlens=cud, max_seqlen=maxL) if len(cu) > 2 else dict(B=1)
    sp = B().sparse_attn_prefill(qd, kd, vd, window=w, n_sink=s, **kw)
    de = B().dense_causal_attn_prefill(qd, kd, vd, **kw)
    dl = B().delta_attn_prefill(qd, kd, vd, window=w, n_sink=s, gamma=gamma, **kw)
    torch.cuda.synchronize()
    return sp, de, dl


# (seqlens, Hq, Hkv, d, window, n_sink, gamma)
SMALL = [
    ((1024,), 1, 1, 64, 128, 4, 16),              # the tiny workload shape
    ((777,), 8, 2, 128, 100, 5, 64),              # GQA 4, 777 mod 64 = 9 dense tail rows
    ((1000, 1, 513, 64), 8, 1, 128, 64, 16, 32),  # varlen with a 1-token sequence, GQA 8
    ((600,), 4, 4, 64, 1, 0, 8),                  # window 1, no sinks
    ((400,), 2, 1, 128, 1000, 0, 16),             # window >= N: no correction anywhere
    ((300,), 4, 2, 128, 32, 8, 1),                # gamma 1: every row dense
    ((200,), 2, 2, 64, 16, 4, 512),               # gamma > N: the whole sequence is tail
    ((2500,), 6, 3, 128, 200, 300, 48),           # GQA 2, sinks wider than the window
    ((130, 70), 2, 1, 128, 33, 1, 7),             # odd gamma, short sequences
    ((300,), 4, 1, 128, 2 ** 31 - 1, 0, 16),      # the largest window: sparse = dense
    ((0, 300, 0, 77, 0), 8, 2, 128, 64, 8, 16),   # empty sequences: leading, inner, trailing
    ((0, 0, 129), 4, 4, 64, 32, 4, 64),           # only the last sequence has tokens, d 64
]


@pytest.mark.parametrize("case", SMALL, ids=[f"L{c[0]}-H{c[1]}/{c[2]}-d{c[3]}-w{c[4]}-s{c[5]}-g{c[6]}"
                                             for c in SMALL])
def test_small_cases_match_oracle(case):
    seqlens, Hq, Hkv, d, w, s, gamma = case
    q, k, v, cu = make(seqlens, Hq, Hkv, d, seed=sum(seqlens) + Hq + d)
    sp, de, dl = run_all(q, k, v, cu, w, s, gamma)
    qb, kb, vb = (to_oracle_bits(x) for x in (q, k, v))
    cun = cu.numpy().astype(np.int64)
    ref, ref_sp, _ = oracle.delta_attention(qb, kb, vb, cun, window=w, n_sink=s, gamma=gamma,
                                            return_parts=True)
    ref_de = oracle.attention(qb, kb, vb, cun, mode=oracle.MODE_DENSE)
    assert_parity(sp, ref_sp, "sparse kernel")
    assert_parity(de, ref_de, "dense kernel")
    assert_parity(dl, ref, "delta path")


def test_needles_pin_window_sink_and_anchor_boundaries():
    """Planted query/key pairs make a one-key slip of any boundary an O(1) error."""
    from paper_2505_11254_amd.inputs import plant_needles
    L, Hq, Hkv, d, w, s, gamma = 3000, 4, 1, 128, 256, 16, 64
    q, k, v, cu = make((L,), Hq, Hkv, d, seed=7, std=0.3)
    pairs = [
        (700, 700 - w + 1), (2047, 2047 - w + 1), (2999, 2999 - w + 1),  # oldest key in the window
        (900, 900 - w), (641, 641 - w), (2500, 2500 - w),                # newest key outside it
        (1500, s - 1), (1281, 1),                                        # last sink / a sink
        (1800, s),                                                       # first non-sink key
        (1024, 200), (1023, 300),          # an anchor row and the last row of the group before
        (s + w, 2), (s + w - 1, 3),        # around the first anchor whose Delta is not zero
        (384, 10),
    ]
    uniq = pairs
    q, k = plant_needles(q, k, uniq, seed=3)
    sp, de, dl = run_all(q, k, v, cu, w, s, gamma)
    qb, kb, vb = (to_oracle_bits(x) for x in (q, k, v))
    ref, ref_sp, _ = oracle.delta_attention(qb, kb, vb, None, window=w, n_sink=s, gamma=gamma,
                                            return_parts=True)
    assert_parity(sp, ref_sp, "sparse kernel, needles")
    assert_parity(dl, ref, "delta path, needles")
    assert_parity(de, oracle.attention(qb, kb, vb, None, mode=oracle.MODE_DENSE), "dense, needles")


@pytest.mark.parametrize("n_sink", [4, 0])
def test_logits_rising_along_the_keys_move_the_reference_max(n_sink):
    """Logits that climb by 15-60 log2 units per key tile (up to ~1200 over the sequence): the
    weights would overflow fp32 unless the kernels move their reference max, tile after tile.
    Heads whose logits fall along the keys keep the first reference."""
    L, Hq, Hkv, d, w, gamma = 1200, 4, 1, 128, 700, 16
    q, k, v, cu = make((L,), Hq, Hkv, d, seed=13, std=0.5)
    g = torch.Generator().manual_seed(14)
    u = torch.randn(d, generator=g)
    u /= u.norm()
    ramp = torch.linspace(0.0, 96.0, L)          # key j sits at ramp[j] along u
    k = (0.1 * k.float() + ramp[:, None, None] * u).to(torch.bfloat16)
    gain = torch.tensor([1.0, -1.0, 0.5, 2.0])   # per query head: rising, falling, slower, faster
    q = (0.1 * q.float() + 48.0 * gain[None, :, None] * u).to(torch.bfloat16)
    sp, de, dl = run_all(q, k, v, cu, w, n_sink, gamma)
    for x in (sp, de, dl):
        assert torch.isfinite(x.float()).all()
    qb, kb, vb = (to_oracle_bits(x) for x in (q, k, v))
    ref, ref_sp, _ = oracle.delta_attention(qb, kb, vb, None, window=w, n_sink=n_sink, gamma=gamma,
                                            return_parts=True)
    assert_parity(sp, ref_sp, "sparse kernel, rising logits")
    assert_parity(dl, ref, "delta path, rising logits")
    assert_parity(de, oracle.attention(qb, kb, vb, None, mode=oracle.MODE_DENSE), "dense, rising logits")


def test_covered_groups_equal_sparse_output_bitwise_and_runs_are_deterministic():
    L, Hq, Hkv, d, w, s, gamma = 4096, 8, 2, 128, 512, 64, 64
    q, k, v, cu = make((L,), Hq, Hkv, d, seed=11)
    sp, _, dl = run_all(q, k, v, cu, w, s, gamma)
    covered = ((s + w + gamma - 1) // gamma) * gamma  # rows of groups whose anchor a < s + w
    assert torch.equal(dl[:covered], sp[:covered])
    assert not torch.equal(dl[covered:covered + gamma], sp[covered:covered + gamma])
    _, _, dl2 = run_all(q, k, v, cu, w, s, gamma)
    assert torch.equal(dl, dl2)


def test_every_output_element_is_written():
    L, Hq, Hkv, d, w, s, gamma = 1500, 4, 2, 128, 100, 4, 32
    q, k, v, cu = make((L,), Hq, Hkv, d, seed=12)
    qd, kd, vd = (x.to(DEV) for x in (q, k, v))
    for fn, kw in ((B().sparse_attn_prefill, dict(window=w, n_sink=s)),
                   (B().dense_causal_attn_prefill, {}),
                   (B().delta_attn_prefill, dict(window=w, n_sink=s, gamma=gamma))):
        out = torch.full_like(qd, float("nan"))
        ws = torch.full((B().workspace_bytes(1, L, Hq, Hkv, d, gamma) // 4,), float("nan"),
                        device=DEV)
        if fn is B().delta_attn_prefill:
            fn(qd, kd, vd, out=out, workspace=ws, **kw)
        else:
            fn(qd, kd, vd, out=out, **kw)
        torch.cuda.synchronize()
        assert not torch.isnan(out).any(), fn.__name__


def test_stream_argument_orders_work_on_that_stream():
    L, Hq, Hkv, d, w, s, gamma = 2048, 4, 1, 64, 128, 4, 16
    q, k, v, cu = make((L,), Hq, Hkv, d, seed=13)
    qd, kd, vd = (x.to(DEV) for x in (q, k, v))
    ref = B().delta_attn_prefill(qd, kd, vd, window=w, n_sink=s, gamma=gamma)
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        out = B().delta_attn_prefill(qd, kd, vd, window=w, n_sink=s, gamma=gamma, stream=st)
    st.synchronize()
    torch.cuda.synchronize()
    assert torch.equal(out, ref)


# ---- workload-sized cases: sampled rows ----

def _workload_case(name, check_plain=False, unfused=False):
    """A workload on the stratified rows (every head, whole groups: the first
    and last groups, those around the first corrected anchor, 64 seeded ones,
    tail rows), checked exactly against the oracle's row entry points."""
    from paper_2505_11254_amd import WORKLOADS
    from paper_2505_11254_amd.inputs import generate
    wl = WORKLOADS[name]
    q, k, v, cu = generate(wl, device=DEV)
    kw = (dict(cu_seqlens=cu, max_seqlen=wl.max_seqlen) if not wl.fixed_length
          else dict(B=wl.B))
    out = B().delta_attn_prefill(q, k, v, window=wl.window, n_sink=wl.n_sink, gamma=wl.gamma,
                                 **kw)
    cun = wl.cu_seqlens()
    rows = stratified_rows(wl.seqlens, wl.Hq, wl.window, wl.n_sink, wl.gamma, seed=len(name))
    got = gather_rows(out, cun, rows)
    got_u = got_sp = got_de = None
    if unfused:  # the unfused schedule (sparse, strided rows, in-place epilogue)
        ws = torch.empty(B().workspace_bytes(wl.B, wl.max_seqlen, wl.Hq, wl.Hkv, wl.d, wl.gamma),
                         dtype=torch.uint8, device=DEV)
        B().delta_attn_prefill_steps(q, k, v, out, ws, B().STEP_ALL, window=wl.window,
                                     n_sink=wl.n_sink, gamma=wl.gamma,
                                     cu_seqlens=None if wl.fixed_length else cu,
                                     max_seqlen=wl.max_seqlen, B=wl.B)
        got_u = gather_rows(out, cun, rows)
        del ws
    # the dense kernel on the boundary rows and seeded rows of sample_rows (a
    # dense row costs the oracle up to the whole sequence)
    drows = sample_rows(wl.seqlens, wl.Hq, wl.window, wl.n_sink, wl.gamma, seed=len(name))
    if check_plain:
        sp = B().sparse_attn_prefill(q, k, v, window=wl.window, n_sink=wl.n_sink, **kw)
        got_sp = gather_rows(sp, cun, rows)
        del sp
        de = B().dense_causal_attn_prefill(q, k, v, **kw)
        got_de = gather_rows(de, cun, drows)
        del de
    torch.cuda.synchronize()
    del out
    qb, kb, vb = (to_oracle_bits(x) for x in (q, k, v))
    del q, k, v
    torch.cuda.empty_cache()
    cu64 = np.asarray(cun, dtype=np.int64)
    ref = oracle.delta_attention_rows(qb, kb, vb, cu64, window=wl.window, n_sink=wl.n_sink,
                                      gamma=wl.gamma, rows=rows)
    err = assert_parity(got, ref, f"{name} delta path ({len(rows)} rows)")
    print(f"\n{name}: delta path vs oracle on {len(rows)} (row, head) pairs "
          f"({len(rows) // wl.Hq} rows x {wl.Hq} heads): {err}", flush=True)
    if got_u is not None:
        err = assert_parity(got_u, ref, f"{name} unfused schedule ({len(rows)} rows)")
        print(f"{name}: unfused schedule vs oracle on the same rows: {err}", flush=True)
    if got_sp is not None:
        ref_sp = oracle.attention(qb, kb, vb, cu64, mode=oracle.MODE_SPARSE, window=wl.window,
                                  n_sink=wl.n_sink, rows=rows)
        assert_parity(got_sp, ref_sp, f"{name} sparse kernel ({len(rows)} rows)")
        ref_de = oracle.attention(qb, kb, vb, cu64, mode=oracle.MODE_DENSE, rows=drows)
        assert_parity(got_de, ref_de, f"{name} dense kernel ({len(drows)} rows)")


def test_workload_tiny_full_tensor():
    from paper_2505_11254_amd import WORKLOADS
    from paper_2505_11254_amd.inputs import generate
    wl = WORKLOADS["tiny_n1024_d64"]
    q, k, v, cu = generate(wl, device=DEV)
    out = B().delta_attn_prefill(q, k, v, window=wl.window, n_sink=wl.n_sink, gamma=wl.gamma)
    torch.cuda.synchronize()
    ref = oracle.delta_attention(*(to_oracle_bits(x) for x in (q, k, v)), None,
                                 window=wl.window, n_sink=wl.n_sink, gamma=wl.gamma)
    assert_parity(out.cpu(), ref, "tiny workload")


@pytest.mark.timeout(900)
def test_workload_llama8b_32k_full_tensor():
    """The 32K layer in full: every element of the Delta output and of the
    sparse kernel's output against the oracle (Algorithm 1 over the whole
    sequence), the dense kernel on boundary and seeded rows."""
    from paper_2505_11254_amd import WORKLOADS
    from paper_2505_11254_amd.inputs import generate
    wl = WORKLOADS["llama8b_layer_32k"]
    q, k, v, cu = generate(wl, device=DEV)
    out = B().delta_attn_prefill(q, k, v, window=wl.window, n_sink=wl.n_sink, gamma=wl.gamma)
    sp = B().sparse_attn_prefill(q, k, v, window=wl.window, n_sink=wl.n_sink)
    de = B().dense_causal_attn_prefill(q, k, v)
    torch.cuda.synchronize()
    rows = sample_rows(wl.seqlens, wl.Hq, wl.window, wl.n_sink, wl.gamma, seed=32)
    got_de = gather_rows(de, wl.cu_seqlens(), rows)
    out, sp = out.cpu(), sp.cpu()
    qb, kb, vb = (to_oracle_bits(x) for x in (q, k, v))
    del q, k, v, de
    torch.cuda.empty_cache()
    ref, ref_sp, _ = oracle.delta_attention(qb, kb, vb, None, window=wl.window, n_sink=wl.n_sink,
                                            gamma=wl.gamma, return_parts=True)
    err = assert_parity(out, ref, "32K delta path, whole tensor")
    print(f"\n32K delta path vs oracle, all {ref.size} elements: {err}", flush=True)
    assert_parity(sp, ref_sp, "32K sparse kernel, whole tensor")
    ref_de = oracle.attention(qb, kb, vb, None, mode=oracle.MODE_DENSE, rows=rows)
    assert_parity(got_de, ref_de, f"32K dense kernel ({len(rows)} rows)")


@pytest.mark.timeout(900)
def test_workload_llama8b_131k_stratified():
    _workload_case("llama8b_layer_131k", check_plain=True, unfused=True)


@pytest.mark.timeout(900)
def test_workload_ragged_b4_stratified():
    _workload_case("ragged_b4_gqa8")


@pytest.mark.timeout(900)
def test_workload_llama8b_1m_stratified():
    _workload_case("llama8b_layer_1m")


@pytest.mark.timeout(600)
def test_interleaved_xcd_map_at_scale():
    """Head groups that do not split evenly over the 8 XCDs (here 4 groups of one
    head) take the interleaved-chunk block map, which only engages on grids of
    at least 512 blocks: 64K tokens give 1024 sparse blocks and a strided grid
    of the same order; checked on sampled rows, sparse and Delta outputs."""
    from paper_2505_11254_amd.inputs import random_qkv
    L, Hq, Hkv, d, w, s, gamma = 65536, 4, 4, 64, 512, 16, 32
    q, k, v, cu = random_qkv((L,), Hq, Hkv, d, seed=41, device=DEV)
    out = B().delta_attn_prefill(q, k, v, window=w, n_sink=s, gamma=gamma)
    sp = B().sparse_attn_prefill(q, k, v, window=w, n_sink=s)
    torch.cuda.synchronize()
    rows = sample_rows((L,), Hq, w, s, gamma, n_random=160, seed=5)
    got, got_sp = gather_rows(out, [0, L], rows), gather_rows(sp, [0, L], rows)
    bits = [to_oracle_bits(x) for x in (q, k, v)]
    del q, k, v, out, sp
    cu64 = np.asarray([0, L], dtype=np.int64)
    ref = oracle.delta_attention_rows(*bits, cu64, window=w, n_sink=s, gamma=gamma, rows=rows)
    ref_sp = oracle.attention(*bits, cu64, mode=oracle.MODE_SPARSE, window=w, n_sink=s, rows=rows)
    assert_parity(got, ref, f"interleaved map, delta path ({len(rows)} rows)")
    assert_parity(got_sp, ref_sp, "interleaved map, sparse kernel")

