"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these checks re-types the oracle's own loops: each compares it with
an independent brute-force matrix form, a closed form, an exact identity
(Lemma 1) or a structural invariant, and the mutation tests at the end show
that plausible slips planted in a copy of the oracle fail at least one pin.
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

import oracle
from brute import bf16_bits_to_f64, brute_parts, f32_to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def rand_problem(seqlens, Hq, Hkv, d, seed, bf16=False, std=1.0):
    rng = np.random.default_rng(seed)
    T = int(sum(seqlens))
    q = rng.standard_normal((T, Hq, d)) * std
    k = rng.standard_normal((T, Hkv, d)) * std
    v = rng.standard_normal((T, Hkv, d))
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int64)
    if bf16:
        qb, kb, vb = (f32_to_bf16_bits(x.astype(np.float32)) for x in (q, k, v))
        return (qb, kb, vb), tuple(bf16_bits_to_f64(x) for x in (qb, kb, vb)), cu
    return (q, k, v), (q, k, v), cu


# (seqlens, Hq, Hkv, d, window, n_sink, gamma)
GRID = [
    ((1,), 1, 1, 16, 1, 0, 1),
    ((2,), 1, 1, 16, 1, 1, 2),
    ((15,), 2, 1, 16, 3, 1, 16),         # gamma = L + 1: all rows are the dense tail
    ((17,), 2, 1, 16, 3, 1, 16),         # gamma +- 1 around L
    ((64,), 4, 2, 16, 8, 2, 4),
    ((257,), 2, 2, 64, 64, 4, 16),       # ragged tail (257 mod 16 = 1)
    ((257,), 4, 1, 16, 3, 0, 3),         # GQA 4, gamma 3, no sinks
    ((130,), 1, 1, 128, 10, 12, 7),      # sinks wider than the window
    ((100,), 2, 1, 16, 200, 0, 8),       # window >= L: no sparsity
    ((40, 1, 77, 16), 4, 2, 16, 5, 2, 8),  # varlen incl. a length-1 sequence
    ((1024,), 1, 1, 64, 128, 4, 16),     # the tiny workload shape
]


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("case", GRID, ids=[f"c{i}" for i in range(len(GRID))])
def test_oracle_matches_brute_force(case, bf16):
    seqlens, Hq, Hkv, d, w, s, gamma = case
    (q, k, v), (qf, kf, vf), cu = rand_problem(seqlens, Hq, Hkv, d, seed=hash(case) % 2**31,
                                               bf16=bf16)
    got, sp, dl = oracle.delta_attention(q, k, v, cu, window=w, n_sink=s, gamma=gamma,
                                         return_parts=True)
    ref, dense, sparse = brute_parts(qf, kf, vf, cu, w, s, gamma)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(sp, sparse, rtol=0, atol=1e-12)
    # plain f and f* from the per-row entry point agree with the matrix forms too
    np.testing.assert_allclose(oracle.attention(q, k, v, cu, mode=oracle.MODE_DENSE), dense,
                               rtol=0, atol=1e-12)
    np.testing.assert_allclose(oracle.attention(q, k, v, cu, mode=oracle.MODE_SPARSE,
                                                window=w, n_sink=s), sparse, rtol=0, atol=1e-12)


def test_gamma_one_is_dense_attention():
    """gamma = 1 makes every row an anchor, so Eq. 6 returns A V exactly."""
    (q, k, v), _, cu = rand_problem((300,), 4, 2, 32, seed=1)
    got = oracle.delta_attention(q, k, v, cu, window=7, n_sink=3, gamma=1)
    dense = oracle.attention(q, k, v, cu, mode=oracle.MODE_DENSE)
    np.testing.assert_allclose(got, dense, rtol=0, atol=1e-12)


@pytest.mark.parametrize("w,s", [(300, 0), (250, 50), (1000, 7)])
def test_full_coverage_gives_zero_delta(w, s):
    """window + sinks >= L: sparse equals dense, Delta is exactly 0, out = A V."""
    (q, k, v), _, cu = rand_problem((300,), 2, 1, 32, seed=2)
    out, sp, dl = oracle.delta_attention(q, k, v, cu, window=w, n_sink=s, gamma=8,
                                         return_parts=True)
    dense = oracle.attention(q, k, v, cu, mode=oracle.MODE_DENSE)
    assert np.all(dl == 0.0)
    assert np.array_equal(sp, dense)
    assert np.array_equal(out, dense)


def test_covered_anchors_have_exactly_zero_delta():
    """Anchors a < s + w see every key j <= a in the sparse set: Delta_a == 0 bitwise."""
    (q, k, v), _, cu = rand_problem((400,), 2, 1, 32, seed=3)
    w, s, gamma = 20, 5, 8
    out, sp, dl = oracle.delta_attention(q, k, v, cu, window=w, n_sink=s, gamma=gamma,
                                         return_parts=True)
    for a in range(0, 400, gamma):
        group = slice(a, a + gamma)
        if a < s + w:
            assert np.all(dl[group] == 0.0), a
            assert np.array_equal(out[group], sp[group])
        else:
            assert np.all(np.abs(dl[a]) > 0), a


@pytest.mark.parametrize("mode", [oracle.MODE_DENSE, oracle.MODE_SPARSE])
def test_softmax_rows_sum_to_one_over_their_key_set(mode):
    (q, k, v), _, cu = rand_problem((200,), 2, 1, 16, seed=4)
    w, s = 9, 3
    for i in (0, 1, 2, 5, 11, 12, 13, 57, 199):
        wts, o = oracle.attention_weights(q, k, v, cu, mode=mode, window=w, n_sink=s, b=0,
                                          h=1, i=i)
        assert abs(wts.sum() - 1.0) < 1e-14
        j = np.arange(i + 1)
        support = np.ones(i + 1, bool) if mode == oracle.MODE_DENSE else (j < s) | (i - j < w)
        assert np.array_equal(wts > 0, support), i
        np.testing.assert_allclose(o, wts @ v[: i + 1, 0], rtol=0, atol=1e-13)


def test_closed_form_window_one_no_sinks():
    """w = 1, s = 0: the sparse row is v_i itself; out_i = v_i + dense_a - v_a."""
    (q, k, v), _, cu = rand_problem((96,), 1, 1, 16, seed=5)
    gamma = 8
    out, sp, dl = oracle.delta_attention(q, k, v, cu, window=1, n_sink=0, gamma=gamma,
                                         return_parts=True)
    assert np.array_equal(sp[:, 0], v[:, 0])
    _, dense, _ = brute_parts(q, k, v, cu, 1, 0, gamma)
    for i in range(96):
        a = (i // gamma) * gamma
        np.testing.assert_allclose(out[i, 0], v[i, 0] + dense[a, 0] - v[a, 0], rtol=0,
                                   atol=1e-12)


@pytest.mark.parametrize("L,w,s,gamma", [(200, 16, 4, 8), (130, 5, 0, 7), (97, 3, 9, 10)])
def test_closed_form_zero_query_is_uniform_mean(L, w, s, gamma):
    """Q = 0 gives uniform weights: every output is a mean of V over an index set.

    V is position-coded with small integers (exact in bf16), so each window,
    sink and anchor boundary shows up in the exact means.
    """
    d = 8
    q = np.zeros((L, 1, d))
    k = np.random.default_rng(6).standard_normal((L, 1, d))
    j = np.arange(L)[:, None]
    c = np.arange(d)[None, :]
    v = (((j * 3 + c * 5) % 7) - 3).astype(np.float64)[:, None, :]
    out = oracle.delta_attention(q, k, v, None, window=w, n_sink=s, gamma=gamma)

    def keyset(i):
        return sorted(set(range(min(s, i + 1))) | set(range(max(0, i - w + 1), i + 1)))

    Lc = (L // gamma) * gamma
    for i in range(L):
        if i >= Lc:
            expect = v[: i + 1, 0].mean(axis=0)
        else:
            a = (i // gamma) * gamma
            expect = (v[keyset(i), 0].mean(axis=0) + v[: a + 1, 0].mean(axis=0)
                      - v[keyset(a), 0].mean(axis=0))
        np.testing.assert_allclose(out[i, 0], expect, rtol=0, atol=1e-12, err_msg=str(i))


def test_lemma1_identity_and_bound():
    """Lemma 1: Delta = sum_{j not in S} a_j v_j + R, R = -H/(H+T) * (A*V)_a exactly,
    with |R| <= H/(H+T) max_{j in S} |v_j| per column (holds for any key set)."""
    (q, k, v), _, cu = rand_problem((512,), 1, 1, 32, seed=7)
    w, s, gamma = 40, 4, 32
    out, sp, dl = oracle.delta_attention(q, k, v, cu, window=w, n_sink=s, gamma=gamma,
                                         return_parts=True)
    d = q.shape[2]
    checked = 0
    for a in range(0, 512, gamma):
        if a < s + w:
            continue
        x = (k[: a + 1, 0] @ q[a, 0]) / np.sqrt(d)
        e = np.exp(x - x.max())
        j = np.arange(a + 1)
        inS = (j < s) | (a - j < w)
        H, T = e[~inS].sum(), e[inS].sum()
        full_w = e / (H + T)
        missing = full_w[~inS] @ v[: a + 1, 0][~inS]
        R = dl[a, 0] - missing
        np.testing.assert_allclose(R, -H / (H + T) * sp[a, 0], rtol=0, atol=1e-12)
        bound = H / (H + T) * np.abs(v[: a + 1, 0][inS]).max(axis=0)
        assert np.all(np.abs(R) <= bound + 1e-15)
        checked += 1
    assert checked > 10


def test_shift_invariance_of_key_offset():
    """Adding one vector mu to every key shifts each score row by a constant: no change."""
    (q, k, v), _, cu = rand_problem((160,), 4, 2, 16, seed=8)
    mu = np.random.default_rng(9).standard_normal((1, 2, 16)) * 0.5
    a = oracle.delta_attention(q, k, v, cu, window=11, n_sink=2, gamma=8)
    b = oracle.delta_attention(q, k + mu, v, cu, window=11, n_sink=2, gamma=8)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_gqa_equals_mha_with_repeated_kv():
    (q, k, v), _, cu = rand_problem((150,), 8, 2, 16, seed=10)
    a = oracle.delta_attention(q, k, v, cu, window=9, n_sink=1, gamma=4)
    k4 = np.repeat(k, 4, axis=1)
    v4 = np.repeat(v, 4, axis=1)
    b = oracle.delta_attention(q, k4, v4, cu, window=9, n_sink=1, gamma=4)
    assert np.array_equal(a, b)


def test_varlen_equals_separate_sequences():
    seqlens = (33, 64, 1, 90)
    (q, k, v), _, cu = rand_problem(seqlens, 4, 2, 16, seed=11)
    packed = oracle.delta_attention(q, k, v, cu, window=6, n_sink=2, gamma=8)
    for b in range(len(seqlens)):
        s0, s1 = cu[b], cu[b + 1]
        alone = oracle.delta_attention(q[s0:s1], k[s0:s1], v[s0:s1], None, window=6,
                                       n_sink=2, gamma=8)
        assert np.array_equal(packed[s0:s1], alone)


def test_empty_sequences_change_nothing():
    """A ragged batch may hold sequences of length zero (repeated offsets): they own no rows
    and leave every other sequence's result as it is without them."""
    seqlens = (0, 70, 0, 33, 0)
    (q, k, v), _, cu = rand_problem(seqlens, 4, 2, 16, seed=13)
    assert list(cu) == [0, 0, 70, 70, 103, 103]
    packed = oracle.delta_attention(q, k, v, cu, window=6, n_sink=2, gamma=8)
    dense = np.array([0, 70, 103])
    assert np.array_equal(packed, oracle.delta_attention(q, k, v, dense, window=6, n_sink=2,
                                                         gamma=8))


def test_row_entry_point_equals_full_algorithm():
    seqlens = (100, 37)
    (q, k, v), _, cu = rand_problem(seqlens, 4, 2, 16, seed=12, bf16=True)
    full, sp, dl = oracle.delta_attention(q, k, v, cu, window=10, n_sink=3, gamma=16,
                                          return_parts=True)
    rng = np.random.default_rng(13)
    rows = [(b, h, i) for b in range(2) for h in range(4) for i in range(seqlens[b])
            if rng.random() < 0.3]
    got, gdl = oracle.delta_attention_rows(q, k, v, cu, window=10, n_sink=3, gamma=16,
                                           rows=rows, return_delta=True)
    for n, (b, h, i) in enumerate(rows):
        assert np.array_equal(got[n], full[cu[b] + i, h])
        assert np.array_equal(gdl[n], dl[cu[b] + i, h])


def key_pair_counts(L, w, s, gamma):
    """(sum_i |S(i)|, sum over anchors of a+1, dense pairs) by direct counting."""
    i = np.arange(L)
    sparse = np.minimum(i + 1, np.minimum(s, i + 1) + np.minimum(w, np.maximum(i + 1 - s, 0)))
    Lc = (L // gamma) * gamma
    anchors = np.arange(0, Lc, gamma)
    tail = np.arange(Lc, L)
    return int(sparse.sum()), int((anchors + 1).sum() + (tail + 1).sum()), L * (L + 1) // 2


def test_key_count_formula_matches_definition():
    """The vectorised |S(i)| used for FLOP accounting equals the set definition."""
    for (L, w, s) in [(300, 20, 5), (50, 100, 3), (64, 1, 0), (99, 7, 30)]:
        direct = sum(len(set(range(min(s, i + 1))) | set(range(max(0, i - w + 1), i + 1)))
                     for i in range(L))
        assert key_pair_counts(L, w, s, 1)[0] == direct


def test_golden_amortised_window_and_overhead():
    """Paper's printed accounting (approx-window appendix; Sec. 4.1 overhead)."""
    with open(os.path.join(GOLDEN, "paper_accounting.json")) as f:
        g = json.load(f)
    aw = g["approx_window"]
    C, w, gamma = aw["context"], aw["window"], aw["gamma"]
    assert w + C // (2 * gamma) == aw["keys_per_row"]
    sp, anc, dense = key_pair_counts(C, w, 0, gamma)
    # exact counts (3055.5 keys/row) sit within 1% of the paper's amortised w + C/(2 gamma);
    # the formula leaves out the w^2/2 start-up triangle of the window
    assert abs((sp + anc) / C - aw["keys_per_row"]) / aw["keys_per_row"] < 1e-2
    ov = g["strided_overhead"]
    frac = anc / dense
    assert abs(frac - ov["fraction_of_full_attention"]) < ov["tolerance"]


# ---- mutation checks: plausible slips planted in a copy of the oracle must fail a pin ----

MUTANTS = {
    "window_edge_inclusive": ("(i - j < window)", "(i - j <= window)"),
    "sink_edge_inclusive": ("(j < n_sink)", "(j <= n_sink)"),
    "diagonal_excluded": ("if (j > i) return 0;", "if (j >= i) return 0;"),
    "delta_sign_flipped": ("dl[c] = dense[c] - spa[c];", "dl[c] = spa[c] - dense[c];"),
    "scale_dropped": ("x[j] = tau * s;", "x[j] = s;"),
    "gqa_interleaved": ("const int g = h / G;", "const int g = h % P->Hkv;"),
    "anchor_of_next_group": ("for (int64_t i = a; i < a + gamma; ++i) {",
                             "for (int64_t i = (a ? a - gamma + 1 : 0); i < a + 1; ++i) {"),
    "tail_not_dense": ("for (int64_t i = Lc; i < L; ++i) {", "for (int64_t i = L; i < L; ++i) {"),
    "sparse_normalised_by_dense": ("if (mode == DAO_MODE_DENSE) return 1;",
                                   "if (mode == DAO_MODE_DENSE || 1) return 1;"),
}


def _pins_pass(orc: oracle.Oracle) -> bool:
    """A compact subset of the pins above, run against one oracle build."""
    cases = [((70,), 4, 2, 16, 6, 3, 8), ((45,), 1, 1, 16, 1, 0, 4)]
    for (seqlens, Hq, Hkv, d, w, s, gamma) in cases:
        (q, k, v), _, cu = rand_problem(seqlens, Hq, Hkv, d, seed=99)
        got = orc.delta_attention(q, k, v, cu, window=w, n_sink=s, gamma=gamma)
        ref, _, _ = brute_parts(q, k, v, cu, w, s, gamma)
        if not np.allclose(got, ref, rtol=0, atol=1e-12):
            return False
    return True


def test_pins_pass_on_the_real_oracle():
    assert _pins_pass(oracle.Oracle())


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_a_pin(name, tmp_path):
    src = os.path.join(os.path.dirname(oracle.__file__), "delta_oracle.c")
    text = open(src).read()
    old, new = MUTANTS[name]
    assert text.count(old) >= 1, f"mutation site for {name} not found"
    mutated = tmp_path / "mutant.c"
    mutated.write_text(text.replace(old, new))
    lib = oracle.build(force=True, src=str(mutated), dst=str(tmp_path / "libmutant.so"))
    assert not _pins_pass(oracle.Oracle(lib)), f"mutant {name} passed the pins"


# ---- correction variants (recompute, interpolation, EMA, alpha-beta-gamma filter) ----

from brute import abg_matrix, brute_variant  # noqa: E402

VARIANT_CASES = [
    ((300,), 2, 1, 16, 20, 3, 16),
    ((257,), 4, 2, 16, 9, 0, 7),           # ragged tail, no sinks
    ((90, 1, 45), 2, 2, 16, 6, 2, 8),      # varlen with a 1-token sequence
    ((64,), 1, 1, 16, 3, 1, 1),            # gamma 1
]
VARIANT_MODES = [(1, (0.0, 0.0, 0.0)), (2, (0.0, 0.0, 0.0)), (3, (0.5, 0.0, 0.0)),
                 (3, (0.95, 0.0, 0.0)), (4, (0.2, 5e-2, 3.5e-3)), (4, (0.05, 1.25e-4, 2.08e-5))]


@pytest.mark.parametrize("case", VARIANT_CASES, ids=[f"v{i}" for i in range(len(VARIANT_CASES))])
@pytest.mark.parametrize("mode,params", VARIANT_MODES, ids=[f"m{m}-{p[0]}" for m, p in VARIANT_MODES])
def test_variant_matches_matrix_form(case, mode, params):
    seqlens, Hq, Hkv, d, w, s, gamma = case
    (q, k, v), _, cu = rand_problem(seqlens, Hq, Hkv, d, seed=sum(seqlens) + mode)
    got = oracle.delta_attention_variant(q, k, v, cu, window=w, n_sink=s, gamma=gamma,
                                         mode=mode, params=params)
    ref = brute_variant(q, k, v, cu, w, s, gamma, mode, params)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-11)


def test_first_anchor_is_always_covered():
    """Anchor 0 sees only key 0 under both f and f*, so Delta_0 is exactly 0."""
    (q, k, v), _, cu = rand_problem((50,), 1, 1, 16, seed=22)
    out, sp, dl = oracle.delta_attention(q, k, v, cu, window=1, n_sink=0, gamma=10,
                                         return_parts=True)
    assert np.all(dl[:10] == 0.0)


def test_variant_special_cases():
    (q, k, v), _, cu = rand_problem((400,), 2, 1, 16, seed=21)
    w, s, g = 30, 2, 16
    base = oracle.delta_attention(q, k, v, cu, window=w, n_sink=s, gamma=g)
    var = lambda m, p=(0.0, 0.0, 0.0): oracle.delta_attention_variant(
        q, k, v, cu, window=w, n_sink=s, gamma=g, mode=m, params=p)
    dense = oracle.attention(q, k, v, cu, mode=oracle.MODE_DENSE)
    sparse = oracle.attention(q, k, v, cu, mode=oracle.MODE_SPARSE, window=w, n_sink=s)
    assert np.array_equal(var(0), base)
    # EMA with weight 1 keeps the newest value: plain Delta
    assert np.array_equal(var(3, (1.0, 0, 0)), base)
    # EMA with weight 0 never moves from D_0 = Delta_0, which is 0 (anchor 0 is covered)
    np.testing.assert_allclose(var(3, (0.0, 0, 0)), sparse, rtol=0, atol=0)
    # filter with alpha=1, beta=gamma=0 follows the measurement: plain Delta
    np.testing.assert_allclose(var(4, (1.0, 0, 0)), base, rtol=0, atol=1e-15)
    # recompute: dense rows at anchors, sparse rows everywhere else
    rec = var(1)
    idx = np.arange(400)
    np.testing.assert_allclose(rec[idx % g == 0], dense[idx % g == 0], rtol=0, atol=1e-12)
    assert np.array_equal(rec[idx % g != 0], sparse[idx % g != 0])
    # interpolation: row a_i carries Delta_i, row a_i + gamma - 1 carries Delta_{i+1}
    itp = var(2)
    delta = base - sparse
    for a in range(0, 400 - 2 * g, g):
        np.testing.assert_allclose(itp[a] - sparse[a], delta[a], rtol=0, atol=1e-12)
        np.testing.assert_allclose(itp[a + g - 1] - sparse[a + g - 1], delta[a + g], rtol=0,
                                   atol=1e-12)


def test_abg_matrix_reproduces_constant_and_ramp_tracking():
    """Independent check of the state-space form: a constant input passes unchanged and
    a critically-tracked ramp converges (the filter is unbiased for polynomial inputs)."""
    H = abg_matrix(400, 0.2, 5e-2, 3.5e-3)
    assert np.allclose(H @ np.ones(400), 1.0, atol=1e-12)
    ramp = np.arange(400.0)
    assert abs((H @ ramp)[-1] - ramp[-1]) < 1e-6


def _closed_loop_radius(a, b, c):
    """Spectral radius of the filter's closed loop (I - g e0^T) F, from its
    eigenvalues (unit step, constant-acceleration transition)."""
    F = np.array([[1.0, 1.0, 0.5], [0.0, 1.0, 1.0], [0.0, 0.0, 1.0]])
    K = np.array([[a], [b], [c]])
    return float(max(abs(np.linalg.eigvals((np.eye(3) - K @ np.array([[1.0, 0.0, 0.0]])) @ F))))


def test_abg_growth_over_many_anchors_matches_the_closed_loop_eigenvalue():
    """The interpolation table's first filter setting is unstable as printed: over
    thousands of anchors the oracle's filtered correction grows by the spectral
    radius of the closed loop per anchor (1.0023), which a factor of 2 or 1/2 on the
    acceleration gain would move to 1.0047 or 1.0007; the table's third setting
    stays bounded.  gamma = 1 makes every row an anchor."""
    (q, k, v), _, cu = rand_problem((3000,), 1, 1, 8, seed=1)
    base = oracle.delta_attention_variant(q, k, v, cu, window=1, n_sink=0, gamma=1, mode=0,
                                          params=(0.0, 0.0, 0.0))

    def envelope(params):
        out = oracle.delta_attention_variant(q, k, v, cu, window=1, n_sink=0, gamma=1, mode=4,
                                             params=params)
        c = np.abs(out - base)[:, 0, :]
        return c[2000:2500].max(), c[2500:3000].max()

    p = (0.05, 1.25e-4, 2.08e-5)
    rho = _closed_loop_radius(*p)
    assert rho > 1.002
    m1, m2 = envelope(p)
    rate = (m2 / m1) ** (1.0 / 500)
    assert abs(rate - rho) < 3e-4, (rate, rho)
    for alt in (2.0, 0.5):
        assert abs(rate - _closed_loop_radius(p[0], p[1], p[2] * alt)) > 1e-3
    p = (0.2, 5e-2, 3.5e-3)
    assert _closed_loop_radius(*p) < 1.0
    m1, m2 = envelope(p)
    assert m2 < 10.0 and m2 < 2 * m1


VARIANT_MUTANTS = {
    "interp_beta_over_gamma": ("(double)kk / (double)(gamma - 1)", "(double)kk / (double)gamma"),
    # (starting the EMA from 0 instead of D_0 is no mistake: anchor 0 only sees key 0,
    # so Delta_0 = D_0 = 0 exactly and both starts agree)
    "ema_weights_swapped": ("ema[c] = (1.0 - p0) * ema[c] + p0 * dl[i * d + c];",
                            "ema[c] = p0 * ema[c] + (1.0 - p0) * dl[i * d + c];"),
    "abg_half_acc_dropped": ("{{1.0, 1.0, 0.5}, {0.0, 1.0, 1.0}, {0.0, 0.0, 1.0}}",
                             "{{1.0, 1.0, 0.0}, {0.0, 1.0, 1.0}, {0.0, 0.0, 1.0}}"),
    "abg_velocity_gain_on_acceleration": ("const double g[3] = {p0, p1, p2};",
                                          "const double g[3] = {p0, p2, p1};"),
    "recompute_applied_everywhere": ("corr = (kk == 0) ? dl[i * d + c] : 0.0;",
                                     "corr = dl[i * d + c];"),
}


@pytest.mark.parametrize("name", sorted(VARIANT_MUTANTS))
def test_planted_variant_mistake_fails_matrix_form(name, tmp_path):
    src = os.path.join(os.path.dirname(oracle.__file__), "delta_oracle.c")
    text = open(src).read()
    old, new = VARIANT_MUTANTS[name]
    assert text.count(old) == 1, name
    mutated = tmp_path / "mutant.c"
    mutated.write_text(text.replace(old, new))
    orc = oracle.Oracle(oracle.build(force=True, src=str(mutated), dst=str(tmp_path / "m.so")))
    (q, k, v), _, cu = rand_problem((200,), 2, 1, 16, seed=5)
    failed = False
    for mode, params in VARIANT_MODES:
        got = orc.delta_attention_variant(q, k, v, cu, window=12, n_sink=2, gamma=8, mode=mode,
                                          params=params)
        ref = brute_variant(q, k, v, cu, 12, 2, 8, mode, params)
        failed |= not np.allclose(got, ref, rtol=0, atol=1e-11)
    assert failed, f"mutant {name} passed"


# ---- the row entry points of plain attention (f and f*), used as checkers at large sizes ----
#
# A row needs only its own key set (Eq. 1; Sec. 3 for f*), so the oracle can be
# evaluated on any list of (sequence, head, row) triples.  These pins hold that
# list form to the whole-tensor form bit for bit, and both to the brute-force
# masked-softmax matrices, on a ragged GQA batch with empty sequences.

ROW_SEQLENS = (57, 0, 90, 1, 33)
ROW_SHAPE = dict(Hq=4, Hkv=2, d=16)
ROW_W, ROW_S = 7, 2


def _row_triples(seqlens, Hq, seed):
    """Every head of the first, last and window-edge rows of each sequence, plus
    random triples, shuffled, with repeats."""
    rng = np.random.default_rng(seed)
    rows = []
    for b, L in enumerate(seqlens):
        for i in {0, L - 1, min(L - 1, ROW_W), min(L - 1, ROW_W + ROW_S)} if L else ():
            rows += [(b, h, i) for h in range(Hq)]
        rows += [(b, int(rng.integers(0, Hq)), int(rng.integers(0, L))) for _ in range(L // 3)] if L else []
    rows += rows[:5]
    order = rng.permutation(len(rows))
    return [rows[n] for n in order]


def _row_pins_pass(orc: oracle.Oracle) -> bool:
    """attention(rows=R) equals the whole-tensor call at R (outputs, score max
    and normaliser) and brute force, for f and f*."""
    (q, k, v), (qf, kf, vf), cu = rand_problem(ROW_SEQLENS, seed=41, bf16=True, **ROW_SHAPE)
    _, dense, sparse = brute_parts(qf, kf, vf, cu, ROW_W, ROW_S, 1)
    rows = _row_triples(ROW_SEQLENS, ROW_SHAPE["Hq"], seed=42)
    try:
        for mode, ref in ((oracle.MODE_DENSE, dense), (oracle.MODE_SPARSE, sparse)):
            full, m, z = orc.attention(q, k, v, cu, mode=mode, window=ROW_W, n_sink=ROW_S,
                                       return_stats=True)
            got, gm, gz = orc.attention(q, k, v, cu, mode=mode, window=ROW_W, n_sink=ROW_S,
                                        rows=rows, return_stats=True)
            for n, (b, h, i) in enumerate(rows):
                t = cu[b] + i
                if not (np.array_equal(got[n], full[t, h]) and gm[n] == m[t, h]
                        and gz[n] == z[t, h]):
                    return False
                if not np.allclose(got[n], ref[t, h], rtol=0, atol=1e-12):
                    return False
    except RuntimeError:
        return False
    return True


def test_attention_rows_equal_whole_tensor_and_brute_force():
    assert _row_pins_pass(oracle.Oracle())


def test_attention_whole_tensor_matches_brute_force():
    (q, k, v), (qf, kf, vf), cu = rand_problem(ROW_SEQLENS, seed=43, bf16=True, **ROW_SHAPE)
    _, dense, sparse = brute_parts(qf, kf, vf, cu, ROW_W, ROW_S, 1)
    for mode, ref in ((oracle.MODE_DENSE, dense), (oracle.MODE_SPARSE, sparse)):
        got = oracle.attention(q, k, v, cu, mode=mode, window=ROW_W, n_sink=ROW_S)
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("bad", [(5, 0, 0), (-1, 0, 0), (0, 4, 0), (0, -1, 0), (0, 0, 57),
                                 (1, 0, 0), (3, 0, 1), (0, 0, -1)])
def test_attention_rows_out_of_range_are_rejected(bad):
    """Triples outside the batch (sequence, head, or row past its sequence,
    including any row of an empty sequence) are an argument error."""
    (q, k, v), _, cu = rand_problem(ROW_SEQLENS, seed=44, bf16=True, **ROW_SHAPE)
    for mode in (oracle.MODE_DENSE, oracle.MODE_SPARSE):
        with pytest.raises(RuntimeError):
            oracle.attention(q, k, v, cu, mode=mode, window=ROW_W, n_sink=ROW_S,
                             rows=[(0, 0, 0), bad])


ROW_MUTANTS = {
    "row_head_and_position_swapped": (
        "        h = (int)rows[3 * it + 1];\n        i = rows[3 * it + 2];\n        o = out + it * d;",
        "        h = (int)rows[3 * it + 2];\n        i = rows[3 * it + 1];\n        o = out + it * d;"),
    "row_sequence_taken_as_head": (
        "        b = (int)rows[3 * it];\n        h = (int)rows[3 * it + 1];\n        i = rows[3 * it + 2];\n        o = out + it * d;",
        "        b = (int)rows[3 * it + 1];\n        h = (int)rows[3 * it];\n        i = rows[3 * it + 2];\n        o = out + it * d;"),
    "row_stats_offset_by_one": (
        "        mo = m_out ? m_out + it : NULL;\n        zo = z_out ? z_out + it : NULL;\n      } else {",
        "        mo = m_out ? m_out + (it + 1) % n_rows : NULL;\n        zo = z_out ? z_out + it : NULL;\n      } else {"),
    "row_position_global_not_local": (
        "        i = rows[3 * it + 2];\n        o = out + it * d;",
        "        i = rows[3 * it + 2] - cu[rows[3 * it]];\n        o = out + it * d;"),
}


@pytest.mark.parametrize("name", sorted(ROW_MUTANTS))
def test_planted_row_decode_mistake_fails_the_row_pins(name, tmp_path):
    src = os.path.join(os.path.dirname(oracle.__file__), "delta_oracle.c")
    text = open(src).read()
    old, new = ROW_MUTANTS[name]
    assert text.count(old) == 1, f"mutation site for {name} not found exactly once"
    mutated = tmp_path / "mutant.c"
    mutated.write_text(text.replace(old, new))
    lib = oracle.build(force=True, src=str(mutated), dst=str(tmp_path / "libmutant.so"))
    assert not _row_pins_pass(oracle.Oracle(lib)), f"mutant {name} passed the row pins"


def test_row_entry_point_is_order_independent():
    """Rows of one group reuse its anchor rows inside the row entry point; the
    result does not depend on how the rows are ordered or interleaved."""
    seqlens = (300, 129)
    (q, k, v), _, cu = rand_problem(seqlens, 4, 2, 16, seed=17, bf16=True)
    full = oracle.delta_attention(q, k, v, cu, window=10, n_sink=3, gamma=16)
    rows = [(b, h, i) for b, L in enumerate(seqlens) for h in range(4) for i in range(L)]
    rng = np.random.default_rng(18)
    for order in (np.arange(len(rows)), rng.permutation(len(rows))):
        rr = [rows[n] for n in order]
        got = oracle.delta_attention_rows(q, k, v, cu, window=10, n_sink=3, gamma=16, rows=rr)
        for n, (b, h, i) in enumerate(rr):
            assert np.array_equal(got[n], full[cu[b] + i, h])
