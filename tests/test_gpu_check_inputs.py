"""da_check_inputs on the GPU: valid cu_seqlens and key-block lists pass, and
each malformed variant is counted (the check kernel reads only within the
arrays' stated sizes, so malformed offsets are never followed)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    assert torch.cuda.is_available()
    from paper_2505_11254_amd import binding
    binding.load_library()
    return binding


def cu_t(x):
    return torch.tensor(x, dtype=torch.int32, device="cuda")


def test_cu_seqlens_rules(lib):
    assert lib.check_inputs(max_seqlen=100, cu_seqlens=cu_t([0, 50, 50, 150])) == 0
    assert lib.check_inputs(max_seqlen=100, cu_seqlens=cu_t([1, 50, 150])) == 1      # not from 0
    assert lib.check_inputs(max_seqlen=100, cu_seqlens=cu_t([0, 60, 50, 90])) == 1   # decreasing
    assert lib.check_inputs(max_seqlen=100, cu_seqlens=cu_t([0, 101, 150])) == 1     # too long
    big = np.arange(0, 5001 * 7, 7, dtype=np.int32)
    assert lib.check_inputs(max_seqlen=7, cu_seqlens=cu_t(big)) == 0                 # 5000 sequences
    big[2500] = big[2499] - 1
    assert lib.check_inputs(max_seqlen=7, cu_seqlens=cu_t(big)) == 2


def test_block_list_rules(lib):
    from paper_2505_11254_amd import blocklists as BL
    seqlens = (3000, 1000)
    bl = BL.vertical_slash(seqlens, 2, 128, n_vertical=4, n_local=3, slash_offsets=(7,), seed=1)
    ptr, idx = bl.to("cuda")
    kw = dict(max_seqlen=max(seqlens), B=2, Hkv=2, block_q=128)
    assert lib.check_inputs(block_ptr=ptr, block_idx=idx, **kw) == 0
    cu = cu_t([0, 3000, 4000])
    assert lib.check_inputs(cu_seqlens=cu, block_ptr=ptr, block_idx=idx, **kw) == 0
    # a repeated entry, then a descending pair, inside one list
    bad = bl.idx.copy()
    b0, b1 = bl.ptr[0, 1, 10], bl.ptr[0, 1, 11]
    assert b1 - b0 >= 3
    bad[b0 + 1] = bad[b0]
    assert lib.check_inputs(block_ptr=ptr, block_idx=torch.from_numpy(bad).cuda(), **kw) == 1
    bad[b0 + 2] = bad[b0] - 1
    assert lib.check_inputs(block_ptr=ptr, block_idx=torch.from_numpy(bad).cuda(), **kw) == 2
    # offsets: decreasing in one (sequence, kv head) row, past nnz in another
    badp = bl.ptr.copy()
    badp[1, 0, 3] = badp[1, 0, 2] - 1
    badp[0, 0, -1] = bl.idx.size + 5
    assert lib.check_inputs(block_ptr=torch.from_numpy(badp).cuda(), block_idx=idx, **kw) == 2
