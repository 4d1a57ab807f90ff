"""Rounding budget of the score scale on peaky logits (GPU).

The kernels multiply each score by c = log2(e)/sqrt(d) in fp32 before the
exponential (Eq. 1's 1/sqrt(d), in base 2).  Folding c into the queries ahead
of the bf16 MFMA instead would round c q to bf16 once more: a relative error
of up to 2^-9 per element, so a logit error proportional to the logit itself.
On unit-normal data that is below the rounding of the bf16 weights P; on
peaky rows (logits near 30 in base 2) it is several times larger.  This test
measures the kernels' error on such rows against the fp64 oracle and against
the error that pre-rounded queries would cause (the oracle evaluated exactly
on those queries, its outputs rounded to bf16 as the kernels store theirs),
and requires the kernels to stay well below it.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
from brute import bf16_bits_to_f64, f32_to_bf16_bits
from sampling import assert_parity, errors, to_oracle_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_11254_amd import binding
    binding.load_library()


@pytest.mark.parametrize("logit_std", [6.0, 8.0])
def test_peaky_logits_keep_the_scale_in_fp32(logit_std):
    from paper_2505_11254_amd import binding
    from paper_2505_11254_amd.inputs import random_qkv
    L, Hq, Hkv, d, w, s, gamma = 1536, 4, 2, 128, 384, 8, 32
    q, k, v, cu = random_qkv((L,), Hq, Hkv, d, seed=31)
    # q.k / sqrt(d) has standard deviation logit_std
    sig = math.sqrt(logit_std)
    q = (q.float() * sig).to(torch.bfloat16)
    k = (k.float() * sig).to(torch.bfloat16)
    qb, kb, vb = (to_oracle_bits(x) for x in (q, k, v))
    qf, kf, vf = (bf16_bits_to_f64(x) for x in (qb, kb, vb))
    c = np.float32(math.log2(math.e) / math.sqrt(d))
    G = Hq // Hkv
    top = max(float((qf[:, h] @ kf[:, h // G].T).max()) / math.sqrt(d) * math.log2(math.e)
              for h in range(Hq))

    qd, kd, vd = (x.cuda() for x in (q, k, v))
    sp = binding.sparse_attn_prefill(qd, kd, vd, window=w, n_sink=s)
    de = binding.dense_causal_attn_prefill(qd, kd, vd)
    dl = binding.delta_attn_prefill(qd, kd, vd, window=w, n_sink=s, gamma=gamma)
    torch.cuda.synchronize()

    ref, ref_sp, _ = oracle.delta_attention(qb, kb, vb, None, window=w, n_sink=s, gamma=gamma,
                                            return_parts=True)
    ref_de = oracle.attention(qb, kb, vb, None, mode=oracle.MODE_DENSE)
    e_sp = assert_parity(sp, ref_sp, "sparse kernel, peaky logits")
    e_de = assert_parity(de, ref_de, "dense kernel, peaky logits")
    e_dl = assert_parity(dl, ref, "delta path, peaky logits")

    # exact attention on the queries bf16(c q) / c, outputs rounded to bf16 as the
    # kernels store them: what pre-scaled bf16 queries would cost
    q_pre = bf16_bits_to_f64(f32_to_bf16_bits(qf.astype(np.float32) * c)) / np.float64(c)
    pre, pre_sp, _ = oracle.delta_attention(q_pre, kf, vf, None, window=w, n_sink=s,
                                            gamma=gamma, return_parts=True)
    pre_de = oracle.attention(q_pre, kf, vf, None, mode=oracle.MODE_DENSE)
    rnd = lambda x: bf16_bits_to_f64(f32_to_bf16_bits(x.astype(np.float32)))
    pre, pre_sp, pre_de = rnd(pre), rnd(pre_sp), rnd(pre_de)
    p_sp, p_de, p_dl = errors(pre_sp, ref_sp), errors(pre_de, ref_de), errors(pre, ref)
    print(f"\nlogit std {logit_std} (largest base-2 logit {top:.1f}): max-abs error")
    for name, e, p in (("sparse", e_sp, p_sp), ("dense", e_de, p_de), ("delta", e_dl, p_dl)):
        print(f"  {name:6s} kernel {e['max_abs']:.2e} (mean {e['mean_abs']:.2e}); "
              f"pre-rounded queries alone {p['max_abs']:.2e} (mean {p['mean_abs']:.2e})")
    assert top > 25.0
    for e, p in ((e_sp, p_sp), (e_de, p_de), (e_dl, p_dl)):
        assert e["max_abs"] < 0.6 * p["max_abs"] and e["mean_abs"] < 0.6 * p["mean_abs"]
