"""Pins of the oracle's block-list sparse basis (Delta Attention over other
sparse attentions f*, given as key-block lists).

The block-list key set is checked against an independent brute-force mask
(tests/brute.py), closed forms with uniform weights, Lemma 1's identity (which
holds for any key set), the dense limit (every tile listed) and planted
mistakes compiled into copies of the oracle.
"""
from __future__ import annotations

import os

import numpy as np
import pytest

import oracle
from brute import bf16_bits_to_f64, brute_block_parts, f32_to_bf16_bits
from paper_2505_11254_amd import blocklists as BL


def rand_problem(seqlens, Hq, Hkv, d, seed, bf16=False):
    rng = np.random.default_rng(seed)
    T = int(sum(seqlens))
    q, k, v = (rng.standard_normal((T, H, d)) for H in (Hq, Hkv, Hkv))
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int64)
    if bf16:
        bits = [f32_to_bf16_bits(x.astype(np.float32)) for x in (q, k, v)]
        return bits, [bf16_bits_to_f64(x) for x in bits], cu
    return (q, k, v), (q, k, v), cu


def random_lists(seqlens, Hkv, block_q, seed, junk=True):
    """Seeded lists with some entries the definition ignores (negative, at or
    past the query block), to pin that they are ignored."""
    rng = np.random.default_rng(seed)
    bl = BL.block_topk(seqlens, Hkv, block_q, k=3, seed=seed)
    if not junk:
        return bl
    idx = []
    ptr = np.zeros_like(bl.ptr)
    for b in range(bl.ptr.shape[0]):
        for g in range(Hkv):
            for qb in range(bl.nqb):
                ptr[b, g, qb] = len(idx)
                t = list(bl.tiles(b, g, qb))
                if rng.random() < 0.3:
                    t.append(qb * block_q // 64 + int(rng.integers(0, 3)))  # inside/after the block
                if rng.random() < 0.2:
                    t.insert(0, -1)
                idx.extend(t)
            ptr[b, g, bl.nqb] = len(idx)
    return BL.BlockLists(block_q, ptr, np.asarray(idx, dtype=np.int32))


# (seqlens, Hq, Hkv, d, block_q, gamma)
GRID = [
    ((1,), 1, 1, 16, 64, 1),
    ((130,), 2, 1, 16, 64, 16),
    ((300,), 4, 2, 16, 128, 8),          # ragged tail: 300 mod 8 = 4
    ((513,), 2, 2, 32, 256, 64),         # 513 mod 64 = 1
    ((200, 1, 70), 4, 2, 16, 64, 7),     # varlen with a length-1 sequence
    ((260,), 8, 1, 16, 64, 300),         # gamma > L: everything is the tail
]


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("case", GRID, ids=[str(c) for c in GRID])
def test_block_oracle_matches_brute_force(case, bf16):
    seqlens, Hq, Hkv, d, block_q, gamma = case
    inp, f64, cu = rand_problem(seqlens, Hq, Hkv, d, seed=sum(seqlens) + d, bf16=bf16)
    bl = random_lists(seqlens, Hkv, block_q, seed=len(seqlens) + block_q)
    out, sp, dl = oracle.block_delta_attention(*inp, cu, blk_ptr=bl.ptr, blk_idx=bl.idx,
                                               block_q=block_q, gamma=gamma, return_parts=True)
    ref, _, ref_sp = brute_block_parts(*f64, cu, bl.ptr, bl.idx, block_q, gamma)
    np.testing.assert_allclose(sp, ref_sp, rtol=0, atol=1e-12)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(oracle.block_attention(*inp, cu, blk_ptr=bl.ptr, blk_idx=bl.idx,
                                                      block_q=block_q), ref_sp, rtol=0, atol=1e-12)


def test_every_tile_listed_is_dense_attention_bitwise():
    seqlens = (333, 64)
    (q, k, v), _, cu = rand_problem(seqlens, 4, 2, 16, seed=2)
    for block_q in (64, 128, 256):
        bl = BL.full(seqlens, 2, block_q)
        out, sp, dl = oracle.block_delta_attention(q, k, v, cu, blk_ptr=bl.ptr, blk_idx=bl.idx,
                                                   block_q=block_q, gamma=16, return_parts=True)
        dense = oracle.attention(q, k, v, cu, mode=oracle.MODE_DENSE)
        assert np.array_equal(sp, dense) and np.array_equal(out, dense)
        assert not dl.any()


def test_uniform_weights_give_means_over_the_selected_tiles():
    """Q = 0 makes every weight equal, so the sparse row is the plain mean of V
    over S(i); with position-coded V the means are exact."""
    L, block_q = 700, 128
    q = np.zeros((L, 2, 16))
    k = np.random.default_rng(3).standard_normal((L, 1, 16))
    v = np.zeros((L, 1, 16))
    v[:, 0, :] = ((np.arange(L) % 11) - 5)[:, None] + np.arange(16)[None, :] * 0.25
    bl = BL.vertical_slash((L,), 1, block_q, n_vertical=3, n_local=2, slash_offsets=(5,), seed=4)
    sp = oracle.block_attention(q, k, v, None, blk_ptr=bl.ptr, blk_idx=bl.idx, block_q=block_q)
    for i in range(L):
        qb = i // block_q
        diag0 = qb * block_q // 64
        keys = [j for t in bl.tiles(0, 0, qb) for j in range(64 * t, 64 * t + 64)]
        keys += list(range(64 * diag0, i + 1))
        np.testing.assert_allclose(sp[i, 0], v[keys, 0].mean(axis=0), rtol=0, atol=1e-12)
        np.testing.assert_allclose(sp[i, 1], sp[i, 0], rtol=0, atol=0)


def test_empty_lists_see_only_the_own_query_block():
    L, block_q = 520, 256
    (q, k, v), _, cu = rand_problem((L,), 1, 1, 16, seed=5)
    bl = BL.empty((L,), 1, block_q)
    for i in (0, 63, 64, 255, 256, 300, 519):
        w, _ = oracle.block_attention_weights(q, k, v, cu, blk_ptr=bl.ptr, blk_idx=bl.idx,
                                              block_q=block_q, i=i)
        lo = (i // block_q) * block_q
        assert np.all(w[:lo] == 0) and np.all(w[lo:] > 0)
        assert abs(w.sum() - 1.0) < 1e-14


def test_lemma1_identity_holds_for_block_lists():
    """Delta_a = sum_{j not in S} a_j v_j - H/(H+T) (A*V)_a for any key set S."""
    L, gamma, block_q = 640, 64, 64
    (q, k, v), _, cu = rand_problem((L,), 1, 1, 32, seed=6)
    bl = BL.block_topk((L,), 1, block_q, k=2, seed=6)
    out, sp, dl = oracle.block_delta_attention(q, k, v, cu, blk_ptr=bl.ptr, blk_idx=bl.idx,
                                               block_q=block_q, gamma=gamma, return_parts=True)
    d = q.shape[2]
    checked = 0
    for a in range(gamma, L, gamma):
        w, _ = oracle.block_attention_weights(q, k, v, cu, blk_ptr=bl.ptr, blk_idx=bl.idx,
                                              block_q=block_q, i=a)
        inS = w > 0
        x = (k[: a + 1, 0] @ q[a, 0]) / np.sqrt(d)
        e = np.exp(x - x.max())
        H, T = e[~inS].sum(), e[inS].sum()
        missing = (e / (H + T))[~inS] @ v[: a + 1, 0][~inS]
        np.testing.assert_allclose(dl[a, 0] - missing, -H / (H + T) * sp[a, 0], rtol=0,
                                   atol=1e-12)
        checked += 1
    assert checked == L // gamma - 1


def test_block_rows_entry_point_equals_full_algorithm():
    seqlens = (300, 129)
    (q, k, v), _, cu = rand_problem(seqlens, 4, 2, 16, seed=7)
    bl = random_lists(seqlens, 2, 64, seed=7)
    full = oracle.block_delta_attention(q, k, v, cu, blk_ptr=bl.ptr, blk_idx=bl.idx, block_q=64,
                                        gamma=32)
    rows = [(b, h, i) for b, L in enumerate(seqlens) for h in range(4) for i in range(0, L, 13)]
    got = oracle.block_delta_attention_rows(q, k, v, cu, blk_ptr=bl.ptr, blk_idx=bl.idx,
                                            block_q=64, gamma=32, rows=rows)
    ref = np.stack([full[cu[b] + i, h] for (b, h, i) in rows])
    assert np.array_equal(got, ref)


def test_generators_follow_their_definitions():
    seqlens = (5000, 700)
    st = BL.star(seqlens, 2, 128, anchor=256, context=1024)
    for b, L in enumerate(seqlens):
        for qb in range(-(-L // 128)):
            diag0 = qb * 2
            c0 = (qb * 128 // 1024) * 1024 // 64
            want = sorted(set(range(4)) | set(range(c0, diag0)))
            assert list(st.tiles(b, 1, qb)) == [t for t in want if t < diag0]
    tk = BL.block_topk(seqlens, 2, 64, k=5, seed=1)
    for qb in range(1, 78):
        t = tk.tiles(0, 0, qb)
        assert len(t) == min(qb, 5) and t[0] == 0 and np.all(np.diff(t) > 0) and t[-1] < qb
    # pair counts of the accounting helper against the oracle's own weights
    L = 300
    (q, k, v), _, cu = rand_problem((L,), 2, 1, 8, seed=9)
    vs = BL.vertical_slash((L,), 1, 64, n_vertical=2, n_local=1, slash_offsets=(3,), seed=2)
    n = 0
    for i in range(L):
        w, _ = oracle.block_attention_weights(q, k, v, cu, blk_ptr=vs.ptr, blk_idx=vs.idx,
                                              block_q=64, i=i)
        n += int((w > 0).sum())
    assert BL.pair_count(vs, (L,), 1, 2) == 2 * n


BLOCK_MUTANTS = {
    "own_block_tiles_dropped": ("sel[t] = (t >= diag0);", "sel[t] = 0;"),
    # (letting listed tiles at or past the query block through changes nothing:
    # those tiles are attended anyway, or masked by causality)
    "listed_tile_zero_dropped": ("if (t >= 0 && t < diag0) sel[t] = 1;",
                                 "if (t > 0 && t < diag0) sel[t] = 1;"),
    "list_by_query_head": ("if (mode == DAO_MODE_BLOCKS) block_row_tiles(P, b, g, i, sel);",
                           "if (mode == DAO_MODE_BLOCKS) block_row_tiles(P, b, h % P->Hkv, i, sel);"),
    # (each mutant must stay in bounds: a slip in the query-block index itself
    # would read past the list offsets)
    "own_block_start_in_query_blocks": ("const int64_t diag0 = qb * P->block_q / DAO_TILE;",
                                        "const int64_t diag0 = qb;"),
}


@pytest.mark.parametrize("name", sorted(BLOCK_MUTANTS))
def test_planted_block_mistake_fails_brute_force(name, tmp_path):
    src = os.path.join(os.path.dirname(oracle.__file__), "delta_oracle.c")
    text = open(src).read()
    old, new = BLOCK_MUTANTS[name]
    assert text.count(old) == 1, name
    mutated = tmp_path / "mutant.c"
    mutated.write_text(text.replace(old, new))
    orc = oracle.Oracle(oracle.build(force=True, src=str(mutated), dst=str(tmp_path / "m.so")))
    failed = False
    for seqlens, block_q in (((300,), 128), ((700,), 64)):
        (q, k, v), _, cu = rand_problem(seqlens, 4, 2, 16, seed=11)
        bl = random_lists(seqlens, 2, block_q, seed=12)
        got = orc.block_delta_attention(q, k, v, cu, blk_ptr=bl.ptr, blk_idx=bl.idx,
                                        block_q=block_q, gamma=16)
        ref = brute_block_parts(q, k, v, cu, bl.ptr, bl.idx, block_q, 16)[0]
        failed |= not np.allclose(got, ref, rtol=0, atol=1e-11)
    assert failed, f"mutant {name} passed"


# ---- the row entry point of sparse attention under block lists ----

BROW_SEQLENS = (300, 0, 129, 1)


def _block_row_pins_pass(orc) -> bool:
    """block_attention(rows=R) equals the whole-tensor call at R bit for bit,
    and the brute-force block-mask softmax, on a ragged GQA batch."""
    (q, k, v), (qf, kf, vf), cu = rand_problem(BROW_SEQLENS, 4, 2, 16, seed=21, bf16=True)
    bl = random_lists(BROW_SEQLENS, 2, 64, seed=22)
    sparse = brute_block_parts(qf, kf, vf, cu, bl.ptr, bl.idx, 64, 1)[2]
    rng = np.random.default_rng(23)
    rows = [(b, h, i) for b, L in enumerate(BROW_SEQLENS) if L for h in range(4)
            for i in {0, L - 1, min(L - 1, 64), min(L - 1, 63)}]
    rows += [(b, int(rng.integers(0, 4)), int(rng.integers(0, L)))
             for b, L in enumerate(BROW_SEQLENS) if L for _ in range(L // 4)]
    rows = [rows[n] for n in rng.permutation(len(rows))]
    try:
        kw = dict(blk_ptr=bl.ptr, blk_idx=bl.idx, block_q=64)
        full = orc.block_attention(q, k, v, cu, **kw)
        got = orc.block_attention(q, k, v, cu, rows=rows, **kw)
    except RuntimeError:
        return False
    for n, (b, h, i) in enumerate(rows):
        t = cu[b] + i
        if not np.array_equal(got[n], full[t, h]):
            return False
        if not np.allclose(got[n], sparse[t, h], rtol=0, atol=1e-12):
            return False
    return True


def test_block_attention_rows_equal_whole_tensor_and_brute_force():
    assert _block_row_pins_pass(oracle.Oracle())


@pytest.mark.parametrize("bad", [(4, 0, 0), (0, 4, 0), (0, 0, 300), (1, 0, 0), (-1, 0, 0)])
def test_block_attention_rows_out_of_range_are_rejected(bad):
    (q, k, v), _, cu = rand_problem(BROW_SEQLENS, 4, 2, 16, seed=24, bf16=True)
    bl = random_lists(BROW_SEQLENS, 2, 64, seed=22)
    with pytest.raises(RuntimeError):
        oracle.block_attention(q, k, v, cu, blk_ptr=bl.ptr, blk_idx=bl.idx, block_q=64,
                               rows=[(0, 0, 0), bad])


BLOCK_ROW_MUTANTS = {
    "block_row_head_and_position_swapped": (
        "        h = (int)rows[3 * it + 1];\n        i = rows[3 * it + 2];\n      } else {",
        "        h = (int)rows[3 * it + 2];\n        i = rows[3 * it + 1];\n      } else {"),
    "block_row_sequence_taken_as_head": (
        "        b = (int)rows[3 * it];\n        h = (int)rows[3 * it + 1];\n        i = rows[3 * it + 2];\n      } else {",
        "        b = (int)rows[3 * it + 1];\n        h = (int)rows[3 * it];\n        i = rows[3 * it + 2];\n      } else {"),
}


@pytest.mark.parametrize("name", sorted(BLOCK_ROW_MUTANTS))
def test_planted_block_row_decode_mistake_fails(name, tmp_path):
    src = os.path.join(os.path.dirname(oracle.__file__), "delta_oracle.c")
    text = open(src).read()
    old, new = BLOCK_ROW_MUTANTS[name]
    assert text.count(old) == 1, name
    mutated = tmp_path / "mutant.c"
    mutated.write_text(text.replace(old, new))
    orc = oracle.Oracle(oracle.build(force=True, src=str(mutated), dst=str(tmp_path / "m.so")))
    assert not _block_row_pins_pass(orc), f"mutant {name} passed"
