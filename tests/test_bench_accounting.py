"""The flop accounting bench.py reports: executed (row, key) pairs, whole
64-key tiles per 32-row wavefront, computed in closed form with numpy, equal
to a literal walk over the kernels' launch plan and tile classes (every
workgroup, every wavefront, every tile of the workgroup's range, skipped when
no key of the tile is visible to any of the wavefront's rows)."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2505_11254_amd.workloads import WORKLOADS, Workload  # noqa: E402


def walk(wl, kind, hpw, chunk, slab=None):
    ppw = 8 // hpw
    tot = 0
    for L in wl.seqlens:
        nA = L // wl.gamma
        Lc = nA * wl.gamma
        if kind == "dense_rows":
            n_rows = nA + (L - Lc)

            def pos(r):
                return r * wl.gamma if r < nA else Lc + (r - nA)
        else:
            n_rows = L

            def pos(r):
                return r
        rpb = slab if (slab and kind == "sparse") else 32 * ppw
        for R0 in range(0, n_rows, rpb):
            R1 = min(R0 + rpb, n_rows)
            lo, hi = pos(R0), pos(R1 - 1)
            for c in (range(-(-L // chunk)) if kind == "dense_rows" else [None]):
                if kind == "sparse":
                    ta1 = (min(wl.n_sink, hi + 1) + 63) // 64
                    tb0 = max(max(0, lo - wl.window + 1) // 64, ta1)
                    tb1 = max(tb0, hi // 64 + 1)
                    tiles = list(range(ta1)) + list(range(tb0, tb1))
                elif kind == "dense":
                    tiles = list(range(hi // 64 + 1))
                else:
                    kc0 = c * chunk
                    if kc0 > hi:
                        continue
                    kc1 = min(kc0 + chunk, hi + 1)
                    tiles = list(range(kc0 // 64, (kc1 + 63) // 64))
                for sub in range(ppw):
                    wr0 = R0 + 32 * sub
                    if wr0 >= R1:
                        continue
                    wlo, whi = pos(wr0), pos(min(wr0 + 32, R1) - 1)
                    for t in tiles:
                        if 64 * t > whi:
                            continue
                        if (kind == "sparse" and 64 * t >= wl.n_sink
                                and wlo - (64 * t + 63) >= wl.window):
                            continue
                        tot += 64 * 32
    return tot


CASES = [
    Workload("a", (5000,), 8, 2, 128, 300, 10, 16, 0.0, 1),
    Workload("b", (3000, 777, 64), 8, 8, 128, 1000, 0, 7, 0.0, 1),
    Workload("c", (40000,), 32, 8, 128, 2048, 64, 64, 0.0, 1),
    Workload("d", (2049,), 4, 4, 128, 100, 130, 1, 0.0, 1),
    WORKLOADS["tiny_n1024_d64"],
]


@pytest.mark.parametrize("wl", CASES, ids=lambda w: w.name)
@pytest.mark.parametrize("kind", ["sparse", "dense_rows", "dense"])
def test_executed_pairs_match_tile_walk(wl, kind):
    """The closed form equals the walk for every head grouping the kernels
    can take, with the library's own key chunks."""
    plan = bench.launch_plan(wl)
    G = wl.Hq // wl.Hkv
    for hpw in (1, 2, 4, 8):
        if G % hpw == 0:
            p = dict(plan, sparse_heads=hpw, rows_heads=hpw, sparse_slab_rows=256 // hpw)
            assert bench.executed_pairs(wl, kind, p) == walk(wl, kind, hpw, plan["chunk_keys"])
            # a sparse slab of whole groups below the full 256 / hpw rows
            slab = (256 // hpw) // wl.gamma * wl.gamma
            if kind == "sparse" and 0 < slab < 256 // hpw:
                p = dict(p, sparse_slab_rows=slab)
                assert bench.executed_pairs(wl, kind, p) == walk(wl, kind, hpw, plan["chunk_keys"],
                                                                 slab)


def test_library_plan_of_the_workloads():
    """The plan the library reports for the five workloads (da_launch_plan):
    the tiling the kernels run and the counts above depend on."""
    want = {  # fused, sparse heads, strided-row heads, key chunks, keys per chunk
        "tiny_n1024_d64": (1, 1, 1, 1, 1024),
        "llama8b_layer_32k": (1, 4, 4, 13, 2560),
        "llama8b_layer_131k": (1, 4, 4, 16, 8192),
        "llama8b_layer_1m": (1, 4, 4, 16, 65536),
        "ragged_b4_gqa8": (1, 8, 8, 15, 8768),  # 16 chunks would pass the 8 GiB of partials
    }
    for name, w in want.items():
        p = bench.launch_plan(WORKLOADS[name])
        assert (p["fused"], p["sparse_heads"], p["rows_heads"], p["key_chunks"],
                p["chunk_keys"]) == w, name
        assert (p["key_tile"], p["rows_per_wave"], p["waves_per_block"]) == (64, 32, 8)
        assert p["sparse_slab_rows"] == 256 // p["sparse_heads"], name
    # gamma 48 with G = 2: no power-of-two head count makes a slab a multiple of 48
    p = bench.launch_plan(Workload("x", (4096,), 4, 2, 128, 64, 4, 48, 0.0, 1))
    assert p["fused"] == 0 and p["sparse_heads"] == p["rows_heads"] == 2
    assert p["sparse_slab_rows"] == 128


def test_executed_covers_useful():
    # whole tiles hold every useful pair: executed >= useful, and close to it
    # where rows and windows are long against a tile
    for wl in WORKLOADS.values():
        sp, dr, dc = bench.pair_counts(wl.seqlens, wl.window, wl.n_sink, wl.gamma)
        es = bench.executed_pairs(wl, "sparse")
        ed = bench.executed_pairs(wl, "dense_rows")
        ec = bench.executed_pairs(wl, "dense")
        assert es >= sp and ed >= dr and ec >= dc
        if wl.name == "llama8b_layer_1m":
            assert es / sp < 1.04 and ed / dr < 1.003 and ec / dc < 1.0002
