"""Wait states in front of the kernels' LDS DMA, checked in their gfx950
assembly (compiled here from the package's sources; no GPU needed).

The DMA (``buffer_load_dwordx4 ... lds``) is issued from inline asm, where
the compiler inserts no wait states.  Two hazards of the gfx9 family that the
hardware does not interlock apply to it: a VMEM instruction that reads an
SGPR written by a VALU instruction (``v_readfirstlane`` builds the buffer
descriptor) needs 5 wait states after that write, and an LDS DMA needs 1
after M0 is written.  A DMA that reads a stale descriptor word fetches the
wrong bytes (a stale record count: zeros), at random.
"""
from __future__ import annotations

import os
import re
import shutil
import subprocess
import tempfile

import pytest

VMEM_SGPR_WAITS = 5
M0_WAITS = 1

_SREG = re.compile(r"^s(\d+)$")
_SRANGE = re.compile(r"^s\[(\d+):(\d+)\]$")
# VALU instructions that write an SGPR (pair) as their second operand
_SECOND_DST = re.compile(r"^v_(add|sub|subrev|addc|subb|subbrev)_co_|^v_div_scale|^v_mad_[ui]64_[ui]32")


def _sgprs(op: str) -> set:
    op = op.strip()
    if op == "m0":
        return {-1}
    m = _SREG.match(op)
    if m:
        return {int(m.group(1))}
    m = _SRANGE.match(op)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    return set()


def _instructions(lines):
    """(mnemonic, operands) per instruction line; None for a label (block start)."""
    for raw in lines:
        t = raw.split(";", 1)[0].strip()
        if not t:
            continue
        if t.endswith(":"):
            yield None
            continue
        if t.startswith("."):
            continue
        parts = t.split(None, 1)
        ops = [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []
        yield parts[0], ops


def dma_hazards(asm_lines) -> list:
    """Every LDS DMA whose preceding wait states hold a VALU write of an SGPR it
    reads (within 5) or an M0 write (within 1), or that starts a block before
    5 wait states are certain.  Returns (index, reason) pairs."""
    insts = list(_instructions(asm_lines))
    bad = []
    for i, ins in enumerate(insts):
        if ins is None or not (ins[0].startswith("buffer_load") and "lds" in ins[1][-1].split()):
            continue
        ops = ins[1]
        reads = {-1} | _sgprs(ops[1]) | (_sgprs(ops[2].split()[0]) if len(ops) > 2 else set())
        waits, j = 0, i - 1
        while waits < VMEM_SGPR_WAITS:
            if j < 0 or insts[j] is None:
                bad.append((i, "block starts within %d wait states" % VMEM_SGPR_WAITS))
                break
            mn, o = insts[j]
            if mn.startswith("v_"):
                dst = _sgprs(o[0]) if o else set()
                if _SECOND_DST.search(mn) and len(o) > 1:
                    dst |= _sgprs(o[1])
                if dst & reads:
                    names = ["m0" if r < 0 else f"s{r}" for r in sorted(dst & reads)]
                    bad.append((i, f"{mn} writes {','.join(names)} {waits} wait states before"))
                    break
            if waits < M0_WAITS and o and o[0] == "m0":
                bad.append((i, f"{mn} writes m0 right before"))
                break
            m = re.match(r"^s_nop$", mn)
            waits += (int(o[0], 0) + 1) if m and o else 1
            j -= 1
    return bad


def test_checker_flags_the_hazard_and_passes_the_wait():
    stale = """
        v_mul_lo_u32 v36, v36, s69
        s_mov_b32 m0, s67
        v_readfirstlane_b32 s38, v36
        s_nop 0
        buffer_load_dwordx4 v139, s[36:39], 0 offen lds
    """.splitlines()
    assert [r for _, r in dma_hazards(stale)] == ["v_readfirstlane_b32 writes s38 1 wait states before"]
    waited = stale[:4] + ["        s_nop 4"] + stale[5:]
    assert dma_hazards(waited) == []
    m0 = ["v_readfirstlane_b32 s38, v36", "s_nop 4", "s_mov_b32 m0, s67",
          "buffer_load_dwordx4 v1, s[36:39], 0 offen lds"]
    assert [r for _, r in dma_hazards(m0)] == ["s_mov_b32 writes m0 right before"]
    vm0 = ["v_readfirstlane_b32 m0, v3", "s_nop 1", "buffer_load_dwordx4 v1, s[36:39], 0 offen lds"]
    assert [r for _, r in dma_hazards(vm0)] == ["v_readfirstlane_b32 writes m0 2 wait states before"]
    label = ["s_nop 1", ".LBB0_3:", "buffer_load_dwordx4 v1, s[36:39], 0 offen lds"]
    assert len(dma_hazards(label)) == 1
    # a VALU write of an SGPR the load does not read is no hazard
    other = ["v_readfirstlane_b32 s40, v36", "buffer_load_dwordx4 v1, s[36:39], 0 offen lds"]
    assert len(dma_hazards(other)) == 1  # (the block start is still within 5)
    other = ["s_nop 7", "v_readfirstlane_b32 s40, v36",
             "buffer_load_dwordx4 v1, s[36:39], 0 offen lds"]
    assert dma_hazards(other) == []


def test_kernel_dma_has_its_wait_states():
    from paper_2505_11254_amd import build
    cc = build.hipcc()
    if not (os.path.isabs(cc) and os.path.exists(cc)) and shutil.which(cc) is None:
        pytest.skip("hipcc not available")
    flags = [f for f in build.compile_flags() if f not in ("-shared", "-fPIC")]
    with tempfile.TemporaryDirectory() as td:
        out = os.path.join(td, "k.s")
        subprocess.run([cc] + flags + ["--cuda-device-only", "-S", build.SOURCES[0], "-o", out],
                       check=True, capture_output=True)
        text = open(out).read().splitlines()
    n_dma = sum(1 for t in text if "buffer_load_dwordx4" in t and t.rstrip().endswith("lds"))
    assert n_dma > 0
    bad = dma_hazards(text)
    assert bad == [], bad[:5]
