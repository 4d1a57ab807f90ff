"""Synthetic workloads of the Delta Attention prefill path.

Each workload fixes the attention-layer shape (heads, head dim, sequence
lengths) and the sparse pattern (sliding window, sink count, anchor stride
gamma).  Shapes follow the models the paper measures (Llama-3.1-8B attention:
32 query heads, 8 key/value heads, head dim 128; standard gamma = 64 and a
2048-token window, Sec. 4) at the prefill lengths of its latency study
(131K and 1M tokens, Sec. 4.1).  Values are synthetic: i.i.d. normal Q, K, V,
optionally with a per-kv-head mean offset on K.
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class Workload:
    name: str
    seqlens: tuple  # one entry per sequence of the (possibly ragged) batch
    Hq: int
    Hkv: int
    d: int
    window: int
    n_sink: int
    gamma: int
    k_offset_std: float  # std of the per-kv-head mean added to every key (0: none)
    seed_base: int       # Q: base+0, K: base+1, V: base+2, K offset: base+3

    @property
    def B(self) -> int:
        return len(self.seqlens)

    @property
    def total_tokens(self) -> int:
        return int(sum(self.seqlens))

    @property
    def max_seqlen(self) -> int:
        return int(max(self.seqlens))

    @property
    def fixed_length(self) -> bool:
        return len(set(self.seqlens)) == 1

    def cu_seqlens(self) -> list:
        cu = [0]
        for n in self.seqlens:
            cu.append(cu[-1] + int(n))
        return cu

    def describe(self) -> dict:
        return {"workload": self.name, "B": self.B, "seqlens": list(self.seqlens),
                "Hq": self.Hq, "Hkv": self.Hkv, "d": self.d, "window": self.window,
                "n_sink": self.n_sink, "gamma": self.gamma, "dtype_io": "bf16"}


WORKLOADS = {
    # small case the oracle finishes in seconds
    "tiny_n1024_d64": Workload("tiny_n1024_d64", (1024,), 1, 1, 64, 128, 4, 16, 0.0, 1000),
    # Llama-3-8B-shaped attention layer (GQA group 4)
    "llama8b_layer_32k": Workload("llama8b_layer_32k", (32768,), 32, 8, 128, 2048, 64, 64,
                                  0.5, 2000),
    "llama8b_layer_131k": Workload("llama8b_layer_131k", (131072,), 32, 8, 128, 2048, 64, 64,
                                   0.5, 3000),
    "llama8b_layer_1m": Workload("llama8b_layer_1m", (1048576,), 32, 8, 128, 2048, 64, 64,
                                 0.5, 4000),
    # ragged batch packed with cu_seqlens, GQA group 8
    "ragged_b4_gqa8": Workload("ragged_b4_gqa8", (16384, 40000, 65536, 131072), 64, 8, 128,
                               4096, 128, 32, 0.0, 5000),
}

HEADLINE = "llama8b_layer_1m"
