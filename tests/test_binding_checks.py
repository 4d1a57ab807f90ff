"""The Python binding rejects malformed tensors before anything reaches the C
ABI (CPU only: tensors stand in for GPU ones and the library is never called)."""
import os
import sys

import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from paper_2505_11254_amd import binding  # noqa: E402


class Dev:
    """A CPU tensor that reports itself as living on a GPU (only the checks
    look at it; nothing dereferences its pointer)."""

    def __init__(self, t, device="cuda:0", is_cuda=True):
        self.t = t
        self.device = torch.device(device)
        self.is_cuda = is_cuda

    dtype = property(lambda s: s.t.dtype)
    shape = property(lambda s: s.t.shape)

    def dim(self):
        return self.t.dim()

    def is_contiguous(self):
        return self.t.is_contiguous()

    def numel(self):
        return self.t.numel()

    def element_size(self):
        return self.t.element_size()

    def data_ptr(self):
        return self.t.data_ptr()


@pytest.fixture(autouse=True)
def no_library(monkeypatch):
    def refuse(*a, **k):
        raise AssertionError("the C library was reached")
    monkeypatch.setattr(binding, "load_library", refuse)


def good(T=128, Hq=4, Hkv=2, d=64):
    bf = torch.bfloat16
    return dict(q=Dev(torch.zeros(T, Hq, d, dtype=bf)), k=Dev(torch.zeros(T, Hkv, d, dtype=bf)),
                v=Dev(torch.zeros(T, Hkv, d, dtype=bf)), out=Dev(torch.zeros(T, Hq, d, dtype=bf)),
                cu=Dev(torch.tensor([0, 100, 128], dtype=torch.int32)),
                ws=Dev(torch.zeros(1024, dtype=torch.uint8)))


def call_all(t):
    """The checks every entry point runs with these tensors."""
    binding._check(t["q"], t["k"], t["v"], t["out"], t["cu"], t["ws"])


def test_well_formed_tensors_pass():
    call_all(good())


def mutate(name, fn):
    t = good()
    t[name] = fn(t[name])
    return t


BAD = {
    "q on the host": lambda: mutate("q", lambda x: Dev(x.t, "cpu", False)),
    "k on another GPU": lambda: mutate("k", lambda x: Dev(x.t, "cuda:1")),
    "v float32": lambda: mutate("v", lambda x: Dev(x.t.float())),
    "q not contiguous": lambda: mutate("q", lambda x: Dev(x.t.transpose(0, 1))),
    "k shorter than q": lambda: mutate("k", lambda x: Dev(x.t[:100])),
    "v of another shape": lambda: mutate("v", lambda x: Dev(torch.zeros(128, 1, 64, dtype=torch.bfloat16))),
    "k of another head size": lambda: dict(good(), k=Dev(torch.zeros(128, 2, 128, dtype=torch.bfloat16)),
                                           v=Dev(torch.zeros(128, 2, 128, dtype=torch.bfloat16))),
    "q 2-D": lambda: mutate("q", lambda x: Dev(x.t.reshape(128, -1))),
    "out of another shape": lambda: mutate("out", lambda x: Dev(x.t[:64])),
    "out float32": lambda: mutate("out", lambda x: Dev(x.t.float())),
    "out on the host": lambda: mutate("out", lambda x: Dev(x.t, "cpu", False)),
    "cu_seqlens on the host": lambda: mutate("cu", lambda x: Dev(x.t, "cpu", False)),
    "cu_seqlens int64": lambda: mutate("cu", lambda x: Dev(x.t.long())),
    "cu_seqlens with one entry": lambda: mutate("cu", lambda x: Dev(x.t[:1])),
    "workspace on another GPU": lambda: mutate("ws", lambda x: Dev(x.t, "cuda:1")),
}


@pytest.mark.parametrize("case", sorted(BAD))
def test_malformed_tensor_is_rejected(case):
    with pytest.raises(ValueError):
        call_all(BAD[case]())


def test_output_aliasing_an_input_is_rejected():
    t = good()
    with pytest.raises(ValueError):
        binding._check(t["q"], t["k"], t["v"], Dev(t["q"].t))          # out is q
    big = torch.zeros(256, 4, 64, dtype=torch.bfloat16)
    q, out = Dev(big[:128]), Dev(big[64:192])                           # overlapping halves
    with pytest.raises(ValueError):
        binding._check(q, t["k"], t["v"], out)
    binding._check(Dev(big[:128]), t["k"], t["v"], Dev(big[128:]))    # adjacent, disjoint


def test_block_lists_are_checked():
    t = good()
    ptr = Dev(torch.zeros(1 * 2 * 3, dtype=torch.int32))  # B=1, Hkv=2, 128 rows / 64 = 2 blocks
    idx = Dev(torch.zeros(4, dtype=torch.int32))
    binding._check(t["q"], t["k"], t["v"], t["out"], None, t["ws"], ptr, idx)
    binding._blocks(ptr, idx, 1, 2, 128, 64)
    with pytest.raises(ValueError):
        binding._blocks(ptr, idx, 1, 2, 128, 128)  # wrong offset count for these query blocks
    with pytest.raises(ValueError):
        binding._blocks(ptr, idx, 1, 2, 128, 32)   # unsupported query block
    with pytest.raises(ValueError):
        binding._check(t["q"], t["k"], t["v"], t["out"], None, t["ws"],
                       Dev(ptr.t.long()), idx)
    with pytest.raises(ValueError):
        binding._check(t["q"], t["k"], t["v"], t["out"], None, t["ws"], ptr,
                       Dev(idx.t, "cpu", False))


def test_entry_points_check_before_calling():
    """Each public entry point raises ValueError on a host tensor before it
    would load or call the library."""
    t = good()
    q_host = Dev(t["q"].t, "cpu", False)
    calls = [
        lambda: binding.delta_attn_prefill(q_host, t["k"], t["v"], window=8, n_sink=1, gamma=4,
                                           out=t["out"], workspace=t["ws"]),
        lambda: binding.sparse_attn_prefill(t["q"], t["k"], t["v"], window=8, n_sink=1,
                                            out=Dev(t["out"].t.float())),
        lambda: binding.dense_causal_attn_prefill(t["q"], t["k"], Dev(t["v"].t[:7]),
                                                  out=t["out"]),
        lambda: binding.delta_attn_prefill_steps(t["q"], t["k"], t["v"], t["out"],
                                                 Dev(t["ws"].t, "cpu", False), 7, window=8,
                                                 n_sink=1, gamma=4),
    ]
    for c in calls:
        with pytest.raises(ValueError):
            c()
