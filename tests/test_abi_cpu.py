"""Host-side checks of the C ABI: the library loads, exports every declared
symbol, and rejects bad arguments before touching the GPU.

Every call here fails validation, which happens before any HIP call, so the
fake device pointers below are never dereferenced and no kernel is launched.
"""
from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "delta_attn.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2505_11254_amd import binding
    return binding.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^[A-Za-z_][A-Za-z0-9_ \*]*?\b([a-z_][a-z0-9_]*)\s*\(", text, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "defined")))


def test_header_declares_the_expected_entry_points():
    names = declared_functions()
    for n in ("delta_attn_prefill", "delta_attn_prefill_varlen", "sparse_attn_prefill",
              "sparse_attn_prefill_varlen", "dense_causal_attn_prefill",
              "dense_causal_attn_prefill_varlen", "da_workspace_bytes", "da_status_string",
              "da_last_hip_error", "da_abi_version"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for n in declared_functions():
        assert hasattr(lib, n), n


def test_binding_signatures_match_header_arity(lib):
    from paper_2505_11254_amd import binding
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    for name, sig in binding.SIGNATURES.items():
        m = re.search(r"\b" + name + r"\s*\(([^;]*)\);", text, flags=re.S)
        assert m, name
        assert len(m.group(1).split(",")) == len(sig), name


def test_abi_version_and_status_strings(lib):
    assert lib.da_abi_version() == 2
    assert lib.da_status_string(0) == b"DA_OK"
    assert lib.da_status_string(6) == b"DA_ERR_WORKSPACE"
    assert lib.da_last_hip_error() == 0


FAKE = 0x100000  # 16-byte aligned, never dereferenced (validation fails first)


def delta(lib, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, out=FAKE, B=1, Hq=8, Hkv=2, N=1024, d=128, window=64,
             n_sink=4, gamma=16, ws=FAKE, wsz=1 << 40)
    a.update(kw)
    return lib.delta_attn_prefill(a["q"], a["k"], a["v"], a["out"], a["B"], a["Hq"], a["Hkv"],
                                  a["N"], a["d"], a["window"], a["n_sink"], a["gamma"],
                                  a["ws"], a["wsz"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), 1), (dict(out=None), 1), (dict(v=None), 1),
    (dict(B=0), 2), (dict(N=0), 2), (dict(Hq=0), 2), (dict(Hkv=0), 2), (dict(Hq=6, Hkv=4), 2),
    (dict(B=70000, N=70000), 2),
    (dict(window=0), 3), (dict(n_sink=-1), 3), (dict(gamma=0), 3),
    (dict(d=96), 4), (dict(d=256), 4),
    (dict(q=FAKE + 8), 5), (dict(out=FAKE + 2), 5), (dict(k=FAKE + 4), 5),
    (dict(ws=None), 6), (dict(wsz=16), 6), (dict(ws=FAKE + 8), 5),
])
def test_delta_call_rejects_bad_arguments(lib, kw, status):
    assert delta(lib, **kw) == status


def test_varlen_requires_cu_seqlens(lib):
    rc = lib.delta_attn_prefill_varlen(FAKE, FAKE, FAKE, FAKE, None, 2, 128, 8, 2, 128, 16, 2,
                                       4, FAKE, 1 << 40, None)
    assert rc == 1
    assert lib.sparse_attn_prefill_varlen(FAKE, FAKE, FAKE, FAKE, None, 2, 128, 8, 2, 128, 16,
                                          2, None) == 1
    assert lib.dense_causal_attn_prefill_varlen(FAKE, FAKE, FAKE, FAKE, None, 2, 128, 8, 2,
                                                128, None) == 1


def test_plain_calls_reject_bad_arguments(lib):
    assert lib.sparse_attn_prefill(FAKE, FAKE, FAKE, FAKE, 1, 8, 2, 128, 128, 0, 0, None) == 3
    assert lib.sparse_attn_prefill(FAKE, FAKE, FAKE, FAKE, 1, 8, 3, 128, 128, 4, 0, None) == 2
    assert lib.dense_causal_attn_prefill(FAKE, FAKE, FAKE, FAKE, 1, 8, 2, 128, 80, None) == 4
    assert lib.dense_causal_attn_prefill(FAKE + 1, FAKE, FAKE, FAKE, 1, 8, 2, 128, 128,
                                         None) == 5


def test_workspace_size_properties(lib):
    ws = lib.da_workspace_bytes
    assert ws(0, 128, 8, 2, 128, 16) == 0
    assert ws(1, 128, 8, 3, 128, 16) == 0
    assert ws(1, 128, 8, 2, 96, 16) == 0
    # at least the fp32 sparse rows at anchors plus one partial (d + 2 floats) per dense row
    for (B, L, Hq, Hkv, d, g) in [(1, 1024, 1, 1, 64, 16), (1, 32768, 32, 8, 128, 64),
                                   (4, 131072, 64, 8, 128, 32), (1, 1 << 20, 32, 8, 128, 64)]:
        nA = L // g
        assert ws(B, L, Hq, Hkv, d, g) >= B * Hq * (nA * d + (nA + g - 1) * (d + 2)) * 4
        assert ws(B, L, Hq, Hkv, d, g) % 256 == 0
    assert ws(1, 1 << 20, 32, 8, 128, 64) < (5 << 30)
    assert ws(1, 4096, 8, 2, 128, 64) <= ws(1, 8192, 8, 2, 128, 64)


def test_oracle_and_library_share_nothing():
    """The oracle never imports the GPU package, and the GPU sources never name the oracle."""
    osrc = open(os.path.join(ROOT, "oracle", "delta_oracle.c")).read()
    opy = open(os.path.join(ROOT, "oracle", "__init__.py")).read()
    assert "paper_2505_11254_amd" not in osrc + opy and "delta_attn.h" not in osrc
    pkg = os.path.join(ROOT, "paper_2505_11254_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".hpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "delta_oracle" not in text, f


def test_correction_call_rejects_bad_arguments(lib):
    import ctypes as C
    f = lib.delta_attn_prefill_correction

    def call(mode, p0=0.0, p1=0.0, p2=0.0, wsz=1 << 40, gamma=16):
        return f(FAKE, FAKE, FAKE, FAKE, None, 1, 1024, 8, 2, 128, 64, 4, gamma, mode,
                 C.c_float(p0), C.c_float(p1), C.c_float(p2), FAKE, wsz, None)
    assert call(5) == 3 and call(-1) == 3
    assert call(3, p0=1.5) == 3 and call(3, p0=-0.1) == 3
    assert call(4, p1=float("nan")) == 3 and call(4, p2=float("inf")) == 3
    assert call(2, wsz=16) == 6
    assert call(3, gamma=0) == 3
    ws = lib.da_workspace_bytes_correction
    assert ws(1, 1024, 8, 2, 128, 16, 9) == 0
    base = lib.da_workspace_bytes(1, 1024, 8, 2, 128, 16)
    assert ws(1, 1024, 8, 2, 128, 16, 0) == base == ws(1, 1024, 8, 2, 128, 16, 1)
    per = 8 * (1024 // 16) * 128 * 4
    assert ws(1, 1024, 8, 2, 128, 16, 2) == base + per == ws(1, 1024, 8, 2, 128, 16, 4)
    assert ws(1, 1024, 8, 2, 128, 16, 3) == base + 2 * per


def test_fused_schedule_support_and_step_flags(lib):
    sup = lib.da_fused_supported
    assert sup(32, 8, 64) == 1 and sup(64, 8, 32) == 1 and sup(1, 1, 16) == 1
    assert sup(4, 1, 128) == 1 and sup(4, 1, 256) == 1 and sup(300, 300, 1) == 1
    assert sup(4, 1, 512) == 0 and sup(6, 3, 48) == 0 and sup(8, 1, 7) == 0
    assert sup(8, 2, 48) == 0 and sup(4, 1, 3) == 0 and sup(1, 1, 200) == 0
    assert sup(64, 8, 64) == 1  # G 8 takes four heads per block: 64-row slabs
    assert sup(6, 4, 64) == 0 and sup(0, 1, 64) == 0 and sup(8, 2, 0) == 0
    f = lib.delta_attn_prefill_steps

    def call(steps, Hq=8, Hkv=2, gamma=16):
        return f(FAKE, FAKE, FAKE, FAKE, None, 1, 1024, Hq, Hkv, 128, 64, 4, gamma, FAKE, 16,
                 None, steps)
    assert call(8) == 3 and call(16) == 3 and call(0) == 3 and call(7 | 16) == 3
    assert call(7 | 8, Hq=6, Hkv=3, gamma=48) == 4   # fused schedule unavailable: rejected
    assert call(1 | 8) == 6 and call(7) == 6          # valid flags: the tiny workspace fails


def test_blocksparse_calls_validate_before_the_gpu(lib):
    sup = lib.da_fused_supported_blocksparse
    assert sup(32, 8, 64, 64) == 1 and sup(32, 8, 64, 256) == 1
    assert sup(32, 8, 128, 64) == 0            # 64-row slabs cannot hold 128-row groups
    assert sup(8, 8, 16, 256) == 1 and sup(8, 8, 16, 128) == 0 and sup(8, 8, 16, 96) == 0
    f = lib.delta_attn_prefill_blocksparse
    s = lib.blocksparse_attn_prefill

    def delta(Hq=8, Hkv=2, block_q=64, ptr=FAKE, idx=FAKE, wsz=16, steps=0, gamma=16):
        return f(FAKE, FAKE, FAKE, FAKE, None, 1, 1024, Hq, Hkv, 128, block_q, ptr, idx, gamma,
                 FAKE, wsz, None, steps)
    assert delta(ptr=None) == 1 and delta(idx=None) == 1
    assert delta(block_q=96) == 3 and delta(block_q=512) == 3 and delta(block_q=32) == 3
    assert delta(Hq=2, Hkv=2, block_q=64) == 4     # one head per block: 256-row slabs
    assert delta(Hq=2, Hkv=2, block_q=256) == 6    # allowed; the tiny workspace fails
    assert delta(steps=16) == 3
    assert delta(steps=7 | 8, Hq=6, Hkv=3, block_q=256, gamma=48) == 4  # no fused slab fits
    assert delta() == 6
    assert s(FAKE, FAKE, FAKE, FAKE, None, 1, 1024, 8, 2, 128, 64, None, FAKE, None) == 1
    assert s(FAKE, FAKE, FAKE, FAKE, None, 1, 1024, 8, 2, 128, 100, FAKE, FAKE, None) == 3
    assert s(FAKE, FAKE, FAKE, FAKE, None, 1, 1024, 4, 4, 128, 128, FAKE, FAKE, None) == 4


def test_rejected_calls_leave_out_untouched(lib):
    """Validation fails before any access: host buffers standing in for the
    tensors keep their bytes (no HIP call and no write happens)."""
    import numpy as np
    buf = np.full(4096, 0x5A, dtype=np.uint8)
    base = buf.ctypes.data
    p = base + (-base) % 16  # 16-byte aligned inside the buffer
    before = buf.copy()
    # unsupported head size, misaligned k, bad window, too small a workspace
    assert lib.delta_attn_prefill(p, p, p, p, 1, 8, 2, 64, 96, 16, 4, 16, p, 1 << 20, None) == 4
    assert lib.delta_attn_prefill(p, p + 4, p, p, 1, 8, 2, 64, 128, 16, 4, 16, p, 1 << 20,
                                  None) == 5
    assert lib.delta_attn_prefill(p, p, p, p, 1, 8, 2, 64, 128, 0, 4, 16, p, 1 << 20, None) == 3
    assert lib.delta_attn_prefill(p, p, p, p, 1, 8, 2, 64, 128, 16, 4, 16, p, 64, None) == 6
    assert lib.sparse_attn_prefill(p, p, p, p, 1, 8, 3, 64, 128, 16, 4, None) == 2
    assert lib.dense_causal_attn_prefill(p, p, p, p, 0, 8, 2, 64, 128, None) == 2
    assert np.array_equal(buf, before)


def test_check_inputs_validates_its_arguments(lib):
    f = lib.da_check_inputs
    assert f(FAKE, 2, 128, 2, 64, None, None, 0, None, None) == 1         # no result buffer
    assert f(None, 2, 128, 2, 64, None, None, 0, FAKE, None) == 1         # nothing to check
    assert f(FAKE, 0, 128, 2, 64, None, None, 0, FAKE, None) == 2         # B < 1
    assert f(None, 1, 128, 2, 96, FAKE, FAKE, 10, FAKE, None) == 3        # block_q
    assert f(None, 1, 128, 0, 64, FAKE, FAKE, 10, FAKE, None) == 2        # Hkv < 1
    assert f(None, 1, 128, 2, 64, FAKE, None, 10, FAKE, None) == 1        # entries without idx
    assert f(FAKE, 1, 128, 2, 64, None, None, 0, FAKE + 2, None) == 5     # result alignment


def test_launch_plan_validates_and_answers_without_a_gpu(lib):
    from paper_2505_11254_amd import binding
    p = binding.Plan()
    ok = (1, 1 << 20, 32, 8, 128, 64, 0)
    assert lib.da_launch_plan(*ok, ctypes.byref(p)) == 0
    assert (p.fused, p.sparse_heads, p.rows_heads, p.key_chunks, p.chunk_keys) == (1, 4, 4, 16, 65536)
    assert lib.da_launch_plan(*ok, None) == 1                                   # DA_ERR_NULL
    for args, status in [((0, 1024, 4, 2, 64, 8, 0), 2), ((1, 1024, 4, 3, 64, 8, 0), 2),
                         ((1, 1024, 4, 2, 64, 0, 0), 3), ((1, 1024, 4, 2, 64, 8, 32), 3),
                         ((1, 1024, 4, 2, 96, 8, 0), 4),
                         # a 64-row query block cannot hold one head's 128-row slab (G = 2)
                         ((1, 1024, 4, 2, 64, 8, 64), 4)]:
        assert lib.da_launch_plan(*args, ctypes.byref(p)) == status, args


def test_noalloc_call_validates_and_bounds_its_scratch_before_the_gpu(lib):
    """The allocation-free entry point rejects bad arguments like the others,
    and a problem whose workspace cannot fit its static array (even with one
    key chunk) with DA_ERR_WORKSPACE, all before any HIP call."""
    def call(q=FAKE, out=FAKE, cu=None, B=1, N=1024, Hq=8, Hkv=2, d=128, w=64, s=4, g=16):
        return lib.delta_attn_prefill_noalloc(q, FAKE, FAKE, out, cu, B, N, Hq, Hkv, d, w, s, g,
                                              None)
    assert call(q=None) == 1 and call(out=None) == 1
    assert call(B=0) == 2 and call(Hq=6, Hkv=4) == 2
    assert call(w=0) == 3 and call(g=0) == 3
    assert call(d=96) == 4
    assert call(q=FAKE + 8) == 5
    # 1M tokens with 32 query heads: the merged rows alone need 269 MB > 256 MiB
    assert call(N=1 << 20, Hq=32, Hkv=8, w=2048, s=64, g=64) == 6
    # the whole plan of 131072 such tokens (596 MB) does not fit, but fewer key
    # chunks do: that call passes this check (it then needs the GPU)
    from paper_2505_11254_amd import binding
    assert binding.workspace_bytes(1, 1 << 17, 32, 8, 128, 64) > 256 << 20


def test_binding_abi_version_matches_header_and_library(monkeypatch):
    """The binding's structures follow one ABI version: the header's, and the
    built library's; a library of another version is refused at load."""
    from paper_2505_11254_amd import binding
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    header = open(os.path.join(root, "include", "delta_attn.h")).read()
    assert int(re.search(r"#define DA_ABI_VERSION (\d+)", header).group(1)) == binding.ABI_VERSION
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("library not built")
    monkeypatch.setattr(binding, "_lib", None)
    assert binding.load_library().da_abi_version() == binding.ABI_VERSION
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "ABI_VERSION", binding.ABI_VERSION + 1)
    with pytest.raises(RuntimeError, match="ABI version"):
        binding.load_library()
    monkeypatch.setattr(binding, "_lib", None)
