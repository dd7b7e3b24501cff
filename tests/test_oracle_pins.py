"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-type the oracle's own formulas: each compares it with a
value the paper prints, a closed form the paper prints, an explicit
construction from the basis definitions, a textbook/library routine, an
invariant, or brute force on tiny inputs.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- measurement

def test_flop_table_matches_paper():
    """Appendix C.1 table: the three operation counts the paper prints."""
    with open(os.path.join(GOLDEN, "paper_flop_table.json")) as f:
        g = json.load(f)
    s = g["shape_reading"]
    n = s["N"] // s["block"]
    p = O.num_coeffs(n, s["frames"])
    assert p == 845
    full, conv, solve = O.paper_op_counts(s["N"], s["H"], s["d"], p)
    pr = g["printed_tflops"]
    dec = g["printed_decimals"]
    assert round(full, dec) == pr["full_attention"]
    assert round(conv, dec) == pr["convert_to_sparsity"]
    assert round(solve, dec) == pr["solve_kernel"]


def test_kept_block_flops_full_mask_is_dense_count():
    L, bs, d = 1000, 64, 32          # ragged tail of 40 tokens
    n = O.num_blocks(L, bs)
    full = [[list(range(n)) for _ in range(n)]]
    assert O.kept_block_flops(full, L, bs, d) == 4.0 * d * L * L


# ---------------------------------------------------------------- a1 pooling

def test_pool_bruteforce_ragged():
    rng = np.random.default_rng(0)
    L, d, bs = 150, 5, 64             # blocks of 64, 64, 22
    x = rng.standard_normal((L, d))
    got = O.pool(x, bs)
    assert got.shape == (3, d)
    for j in range(3):
        for c in range(d):
            toks = [x[t, c] for t in range(L) if t // bs == j]
            assert got[j, c] == pytest.approx(sum(toks) / len(toks), rel=1e-14, abs=1e-15)


# ---------------------------------------------------------------- a2 mass

def test_block_mass_aligned_is_softmax_of_block_logits():
    rng = np.random.default_rng(1)
    n, d = 12, 8
    qb, kb = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    G = O.block_mass(qb, kb, np.full(n, 64), 0.3)
    ref = scipy.special.softmax(0.3 * qb @ kb.T, axis=1)
    np.testing.assert_allclose(G, ref, rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(G.sum(axis=1), 1.0, rtol=1e-14)


def test_block_mass_tail_is_mean_field_token_mass():
    """With every key token replaced by its block mean, the mass that a
    query block mean puts on key block j, summed token by token, is G(i, j)."""
    rng = np.random.default_rng(2)
    L, bs, d, s = 200, 64, 6, 0.4     # sizes 64, 64, 64, 8
    q, k = rng.standard_normal((L, d)), rng.standard_normal((L, d))
    qb, kb = O.pool(q, bs), O.pool(k, bs)
    G = O.block_mass(qb, kb, O.block_sizes(L, bs), s)
    n = qb.shape[0]
    for i in range(n):
        logit = [s * float(qb[i] @ kb[t // bs]) for t in range(L)]
        mx = max(logit)
        w = [math.exp(a - mx) for a in logit]
        tot = sum(w)
        for j in range(n):
            mass = sum(w[t] for t in range(L) if t // bs == j) / tot
            assert G[i, j] == pytest.approx(mass, rel=1e-12)


# ---------------------------------------------------------------- geometry

def test_frame_regions_aligned_and_overlapping():
    assert O.frame_regions(1024, 64, 256) == [(0, 3), (4, 7), (8, 11), (12, 15)]
    reg = O.frame_regions(118800, 128, 3600)
    assert len(reg) == 33 and reg[0] == (0, 28) and reg[1] == (28, 56)
    assert reg[-1][1] == O.num_blocks(118800, 128) - 1
    # every 8th frame boundary (8 * 3600 = 225 * 128) is block aligned
    assert reg[7] == (196, 224) and reg[8] == (225, 253)


# ---------------------------------------------------------------- a3 model

CASES = [  # (L, block, frame_tokens)
    (128, 8, 32),       # n 16, 4 aligned frames
    (231, 8, 33),       # n 29 with a 7-token tail, 7 frames straddling blocks
    (240, 10, 48),      # n 24, 5 frames of 4.8 blocks
    (240, 8, 30),       # n 30, 8 frames of 3.75 blocks
    (1024, 64, 256),    # the tiny layer: n 16, 4 frames
    (300, 16, 300),     # a single frame: nullity 2
]


def _case(L, bs, tf):
    n = O.num_blocks(L, bs)
    return n, O.frame_regions(L, bs, tf)


@pytest.mark.parametrize("L,bs,tf", CASES)
def test_normal_matrix_equals_explicit(L, bs, tf):
    n, reg = _case(L, bs, tf)
    M = O.design_matrix(n, reg)
    np.testing.assert_array_equal(O.normal_matrix(n, reg), M.T @ M)


def test_normal_matrix_blocks_printed_in_paper():
    """Appendix B.4: C^T C = diag(n-|delta|), D^T D = nI, C^T D is 0/1 with
    a 1 where the diagonal crosses the column, E^T E = diag(b^2) for frames
    of b blocks."""
    n, b = 16, 4
    reg = O.frame_regions(n * 8, 8, 8 * b)
    N = O.normal_matrix(n, reg)
    deltas = np.arange(-(n - 1), n)
    np.testing.assert_array_equal(np.diag(N)[:2 * n - 1], n - np.abs(deltas))
    CC = N[:2 * n - 1, :2 * n - 1]
    np.testing.assert_array_equal(CC, np.diag(np.diag(CC)))
    np.testing.assert_array_equal(N[2 * n - 1:3 * n - 1, 2 * n - 1:3 * n - 1], n * np.eye(n))
    CD = N[:2 * n - 1, 2 * n - 1:3 * n - 1]
    for a, dl in enumerate(deltas):
        for j in range(n):
            crosses = any(jj - ii == dl for ii in range(n) for jj in [j])
            crosses = crosses and 0 <= j - dl < n
            assert CD[a, j] == (1.0 if crosses else 0.0)
    np.testing.assert_array_equal(N[3 * n - 1:, 3 * n - 1:], b * b * np.eye(n // b))


@pytest.mark.parametrize("L,bs,tf", CASES)
def test_rhs_equals_explicit(L, bs, tf):
    n, reg = _case(L, bs, tf)
    G = np.random.default_rng(3).random((n, n))
    np.testing.assert_allclose(O.rhs(G, reg), O.design_matrix(n, reg).T @ G.ravel(),
                               rtol=1e-13)


@pytest.mark.parametrize("L,bs,tf", CASES)
def test_null_space_is_z(L, bs, tf):
    n, reg = _case(L, bs, tf)
    M = O.design_matrix(n, reg)
    sv = np.linalg.svd(M, compute_uv=False)
    rank = int((sv > sv[0] * 1e-10).sum())
    F = len(reg)
    assert rank == M.shape[1] - 1 if F >= 2 else rank == M.shape[1] - 2
    np.testing.assert_allclose(M @ O.null_vector(n, F), 0.0, atol=1e-12)


@pytest.mark.parametrize("L,bs,tf", CASES)
def test_fit_equals_lstsq_minimum_norm(L, bs, tf):
    n, reg = _case(L, bs, tf)
    if len(reg) < 2:
        pytest.skip("nullity 2")
    G = np.random.default_rng(4).random((n, n))
    X = O.fit(G, reg)
    Xl = O.fit_lstsq(G, reg)
    np.testing.assert_allclose(X, Xl, rtol=0, atol=1e-10 * np.abs(Xl).max())
    assert abs(X @ O.null_vector(n, len(reg))) < 1e-10


@pytest.mark.parametrize("L,bs,tf", CASES)
def test_planted_coefficients_recovered(L, bs, tf):
    n, reg = _case(L, bs, tf)
    F = len(reg)
    if F < 2:
        pytest.skip("nullity 2")
    rng = np.random.default_rng(5)
    z = O.null_vector(n, F)
    Xs = rng.standard_normal(O.num_coeffs(n, F))
    Xs -= (Xs @ z) / (z @ z) * z
    G = (O.design_matrix(n, reg) @ Xs).reshape(n, n)
    np.testing.assert_allclose(O.fit(G, reg), Xs, atol=1e-10)
    np.testing.assert_allclose(O.reconstruct(Xs, n, reg), G, atol=1e-12)


def test_ridge_solution_close_to_minimum_norm():
    """The paper's Tikhonov lambda = 1e-8 (Appendix B.6) lands within
    O(lambda) of the minimum-norm solution used here."""
    n, reg = _case(*CASES[3])
    G = np.random.default_rng(6).random((n, n))
    N = O.normal_matrix(n, reg)
    ridge = np.linalg.solve(N + 1e-8 * np.eye(N.shape[0]), O.rhs(G, reg))
    X = O.fit(G, reg)
    assert np.abs(ridge - X).max() < 1e-6 * max(1.0, np.abs(X).max())


def test_fit_normal_equations_condition_at_workload_shapes():
    """The min-norm system stays well conditioned at the layer shapes used."""
    for L, bs, tf in [(1024, 64, 256), (8192, 128, 1024)]:
        n, reg = _case(L, bs, tf)
        N = O.normal_matrix(n, reg)
        z = O.null_vector(n, len(reg))
        A = N + (n / (z @ z)) * np.outer(z, z)
        assert np.linalg.cond(A) < 1e8


# ---------------------------------------------------------------- a4 prediction

def test_extrapolation_reproduces_linear_sequences():
    rng = np.random.default_rng(7)
    n, F = 6, 2
    a, b = rng.standard_normal(O.num_coeffs(n, F)), rng.standard_normal(O.num_coeffs(n, F))
    X = lambda t: a + b * t  # noqa: E731
    for t1, t2, t in [(4, 5, 9), (5, 15, 22), (10, 20, 20), (3, 7, 5)]:
        c, d = O.extrapolate(X(t1), t1, X(t2), t2, t, n)
        cs, ds, _ = O.split_coeffs(X(t), n)
        np.testing.assert_allclose(c, cs, atol=1e-12)
        np.testing.assert_allclose(d, ds, atol=1e-12)


def test_gauge_invariance_of_scores():
    rng = np.random.default_rng(8)
    n, F = 9, 3
    X = rng.standard_normal(O.num_coeffs(n, F))
    z = O.null_vector(n, F)
    for alpha in (0.3, -2.0):
        c1, d1, _ = O.split_coeffs(X, n)
        c2, d2, _ = O.split_coeffs(X + alpha * z, n)
        np.testing.assert_allclose(O.scores(c1, d1, n), O.scores(c2, d2, n), atol=1e-12)


def test_gate_reading():
    assert O.gate([np.array([0.1, 0.3]), np.array([0.2, 0.05])], 0.0)
    assert not O.gate([np.array([0.1, 0.3]), np.array([-0.2, 0.05])], 0.0)
    assert not O.gate([np.array([0.4])], 0.5)


# ---------------------------------------------------------------- a5 selection

def test_pattern_index_convention_picks_the_planted_diagonal_and_column():
    """Fit a map that is one parallel diagonal (j - i = +3) plus one strong
    column: the top-2 selection of every row must be exactly those."""
    n, bs = 16, 8
    reg = O.frame_regions(n * bs, bs, n * bs // 2)
    G = 0.01 * O.basis_C(n, 3) + 0.05 * O.basis_D(n, 11) + 0.001
    X = O.fit(G, reg)
    c, d, _ = O.split_coeffs(X, n)
    sig = O.scores(c, d, n)
    forced = O.forced_mask(n, reg, False)
    for i, r in enumerate(O.select(sig, forced, "topk", density=2 / n)):
        want = {11} | ({i + 3} if i + 3 < n else set())
        if len(want) == 1:
            assert 11 in set(r.kept.tolist())
        else:
            assert set(r.kept.tolist()) == want


def test_topk_count():
    assert O.topk_count(0.30, 16) == 5
    assert O.topk_count(0.25, 64) == 16
    assert O.topk_count(0.05, 591) == 30
    assert O.topk_count(0.10, 591) == 60
    assert O.topk_count(0.5, 591) == 296
    assert O.topk_count(1.0, 929) == 929
    assert O.topk_count(1e-9, 929) == 1


@pytest.mark.parametrize("seed", range(6))
def test_topk_row_bruteforce(seed):
    rng = np.random.default_rng(100 + seed)
    n = 9
    sig = rng.standard_normal(n)
    forced = rng.random(n) < 0.25
    k = int(rng.integers(1, n + 1))
    got = set(O.select_row_topk(sig, forced, k).kept.tolist())
    free = [j for j in range(n) if not forced[j]]
    kk = min(len(free), max(0, k - int(forced.sum())))
    best = max(itertools.combinations(free, kk), key=lambda s: sum(sig[j] for j in s))
    assert got == set(best) | set(np.flatnonzero(forced).tolist())


@pytest.mark.parametrize("seed", range(6))
def test_mass_row_bruteforce(seed):
    """The kept set is a smallest set (with the forced blocks) whose positive
    mass reaches tau, and among those the heaviest."""
    rng = np.random.default_rng(200 + seed)
    n = 9
    sig = rng.standard_normal(n) + 0.5
    forced = rng.random(n) < 0.2
    tau = float(rng.uniform(0.3, 0.95))
    got = O.select_row_mass(sig, forced, tau)
    pos = np.maximum(sig.astype(np.float32).astype(np.float64), 0)
    target = np.float32(tau) * pos.sum()
    fset = set(np.flatnonzero(forced).tolist())
    free = [j for j in range(n) if not forced[j]]
    fm = sum(pos[j] for j in fset)
    for size in range(0 if fset else 1, len(free) + 1):
        ok = [s for s in itertools.combinations(free, size) if fm + sum(pos[j] for j in s) >= target]
        if ok:
            best = max(ok, key=lambda s: sum(pos[j] for j in s))
            break
    assert set(got.kept.tolist()) == set(best) | fset
    assert sum(pos[j] for j in got.kept) >= target


def test_mass_row_zero_mass_keeps_one_block():
    r = O.select_row_mass(-np.ones(6), np.zeros(6, bool), 0.9)
    assert r.kept.tolist() == [0]


def test_selection_ties_break_by_index():
    r = O.select_row_topk(np.ones(8), np.zeros(8, bool), 3)
    assert r.kept.tolist() == [0, 1, 2] and r.key_gap == 0.0


# ------------------------------------------------------- pattern-level Top-K

def _pattern_mask_bruteforce(c, d, n, K, forced):
    """Kept blocks from explicit pattern sets: choose the K best patterns by
    trying every K-subset of the 3n-1 patterns (values at float32, the
    lexicographically smallest index set among equal sums), then mark the
    blocks each chosen pattern covers from its definition."""
    vals = [float(np.float32(x)) for x in list(c) + list(d)]
    P = len(vals)
    best = max(itertools.combinations(range(P), K),
               key=lambda S: (sum(vals[p] for p in S), [-p for p in S]))
    keep = forced.copy()
    for p in best:
        if p < 2 * n - 1:                      # diagonal delta = p - (n - 1)
            delta = p - (n - 1)
            for i in range(n):
                if 0 <= i + delta < n:
                    keep[i, i + delta] = True
        else:                                  # column j
            keep[:, p - (2 * n - 1)] = True
    return keep


@pytest.mark.parametrize("seed", range(5))
def test_pattern_topk_bruteforce(seed):
    rng = np.random.default_rng(300 + seed)
    n = 4
    c, d = rng.standard_normal(2 * n - 1), rng.standard_normal(n)
    forced = np.zeros((n, n), bool)
    if seed % 2:
        forced[:2, :2] = forced[2:, 2:] = True
    K = int(rng.integers(1, 3 * n))
    got = O.select_patterns(c, d, n, K, forced)
    want = _pattern_mask_bruteforce(c, d, n, K, forced)
    for i in range(n):
        assert got[i].kept.tolist() == np.flatnonzero(want[i]).tolist()


def test_pattern_topk_planted_diagonal_and_column():
    """Fit a map made of one parallel diagonal and one column: the two best
    patterns of the minimum-norm fit are exactly those, and K = 2 keeps the
    union of their blocks."""
    n, bs = 16, 8
    reg = O.frame_regions(n * bs, bs, n * bs // 2)
    G = 0.02 * O.basis_C(n, -2) + 0.05 * O.basis_D(n, 5) + 0.001
    c, d, _ = O.split_coeffs(O.fit(G, reg), n)
    rows = O.select_patterns(c, d, n, 2, np.zeros((n, n), bool))
    for i, r in enumerate(rows):
        want = {5} | ({i - 2} if i >= 2 else set())
        assert set(r.kept.tolist()) == want


def test_pattern_topk_all_patterns_keep_every_block_and_ties():
    n = 6
    rows = O.select_patterns(np.zeros(2 * n - 1), np.zeros(n), n, 3 * n - 1, np.zeros((n, n), bool))
    assert all(r.kept.tolist() == list(range(n)) for r in rows)
    # equal intensities: the lowest pattern indices win (diagonals from the
    # most negative offset, so K = 1 keeps block (n-1, 0) only)
    rows = O.select_patterns(np.zeros(2 * n - 1), np.zeros(n), n, 1, np.zeros((n, n), bool))
    assert [r.kept.tolist() for r in rows] == [[]] * (n - 1) + [[0]]
    assert rows[0].key_gap == 0.0


def test_pattern_topk_invariants():
    rng = np.random.default_rng(7)
    n = 12
    c, d = rng.standard_normal(2 * n - 1), rng.standard_normal(n)
    forced = O.forced_mask(n, [(0, 3), (3, 7), (8, 11)], True)
    K = 9
    rows = O.select_patterns(c, d, n, K, forced)
    vals = np.concatenate([c, d]).astype(np.float32)
    thr = np.sort(vals)[::-1][K - 1]
    for i, r in enumerate(rows):
        for j in range(n):
            covered = vals[j - i + n - 1] >= thr or vals[2 * n - 1 + j] >= thr
            assert (j in r.kept) == (covered or forced[i, j])


# ------------------------------------------------- token-type-aware masking

def _text_case(text_tokens, frames, hh, ww, seed=11):
    rng = np.random.default_rng(seed)
    Lv = frames * hh * ww
    L = Lv + text_tokens
    q, k = rng.standard_normal((1, 2, L, 16)), rng.standard_normal((1, 2, L, 16))
    return Lv, L, q, k


@pytest.mark.parametrize("shape", [(4, 8, 8, 64), (4, 8, 8, 40), (4, 5, 10, 50)])
@pytest.mark.parametrize("mode", ["topk", "mass", "pattern"])
def test_text_rows_and_columns_full_and_video_part(shape, mode):
    """Text blocks' rows keep everything and every row keeps the text blocks.
    Aligned text: the video part of a row is exactly the video-only
    predictor's selection.  Text starting inside a block (shape 3): that
    block is forced into every row, and in TOPK the other video blocks are
    the frame blocks forced by the gate plus the best-scoring others of the
    video-only prediction, the shared block taking one of the k places."""
    frames, hh, ww, text_tokens = shape
    bs = 32
    Lv, L, q, k = _text_case(text_tokens, frames, hh, ww)
    budget = O.Budget(mode, density=0.3, mass=0.6, patterns=9)
    kw = dict(warmup_m=1, delta_t=0)
    P = O.Predictor(1, 2, L, 16, bs, hh * ww, text_tokens=text_tokens, **kw)
    V = O.Predictor(1, 2, Lv, 16, bs, hh * ww, **kw)
    P.collect(q, k, 1)
    V.collect(q[..., :Lv, :], k[..., :Lv, :], 1)
    rows = P.predict(q, k, 2, budget)[0]
    vrows = V.predict(q[..., :Lv, :], k[..., :Lv, :], 2, budget)[0]
    n, nv = O.num_blocks(L, bs), O.num_blocks(Lv, bs)
    tb = list(range(Lv // bs, n))
    mixed = Lv % bs != 0
    kk = O.topk_count(0.3, nv)
    for h in range(2):
        assert len(rows[h]) == n
        ct, dt_ = V.prediction(2)[0][h]
        keys = O.scores(ct, dt_, nv).astype(np.float32)
        for i in range(n):
            kept = rows[h][i].kept.tolist()
            if i in tb:
                assert kept == list(range(n))
                continue
            assert set(tb) <= set(kept)
            video = [j for j in kept if j not in tb]
            if not mixed:
                assert video == vrows[h][i].kept.tolist()
            elif mode == "topk":
                forced = set(np.flatnonzero(O.forced_mask(nv, V.regions, bool(V.gates[0, h]))[i]).tolist())
                forced.add(tb[0])
                cand = [j for j in range(nv) if j not in forced]
                best = sorted(cand, key=lambda j: (-keys[i, j], j))[:max(0, kk - len(forced))]
                assert video == sorted((forced | set(best)) - set(tb))


def test_text_blocks_layout():
    assert list(O.text_blocks(256, 256, 32)) == []
    assert list(O.text_blocks(256, 320, 32)) == [8, 9]          # aligned: text from block 8
    assert list(O.text_blocks(250, 300, 32)) == [7, 8, 9]       # block 7 holds video and text


# ------------------------------------------- Eq. 2 / Eq. 5 attention statistic

@pytest.mark.parametrize("seed", range(3))
def test_attention_statistic_bruteforce(seed):
    """Fractions of softmax probabilities >= eta per kept block, against a
    library softmax over the kept tokens and explicit per-entry counting."""
    rng = np.random.default_rng(400 + seed)
    L, d, bs, scale, eta = 150, 8, 32, 0.4, 3e-3
    q, k = rng.standard_normal((L, d)), rng.standard_normal((L, d))
    n = O.num_blocks(L, bs)
    kept = [sorted(rng.choice(n, size=int(rng.integers(1, n + 1)), replace=False).tolist())
            for _ in range(n)]
    I, _ = O.attention_statistic(q, k, kept, bs, scale, eta)
    for i in range(n):
        rows = range(i * bs, min(L, (i + 1) * bs))
        cols = [c for j in kept[i] for c in range(j * bs, min(L, (j + 1) * bs))]
        for p in rows:
            pr = scipy.special.softmax(scale * np.array([q[p] @ k[c] for c in cols]))
            if p == rows[0]:
                counts = {j: 0 for j in kept[i]}
            for c, v in zip(cols, pr):
                if v >= eta:
                    counts[c // bs] += 1
        for j in range(n):
            if j in kept[i]:
                size = (min(L, (i + 1) * bs) - i * bs) * (min(L, (j + 1) * bs) - j * bs)
                assert I[i, j] == counts[j] / size
            else:
                assert np.isnan(I[i, j])


def test_attention_statistic_uniform_attention_closed_form():
    """q = 0 gives uniform attention 1/m over the m kept tokens of a row:
    eta = 1/m counts every entry, eta slightly above counts none; eta -> 0
    counts all, eta > 1 none."""
    rng = np.random.default_rng(1)
    L, d, bs = 96, 4, 32
    q, k = np.zeros((L, d)), rng.standard_normal((L, d))
    kept = [[0, 2], [1], [0, 1, 2]]
    for i, js in enumerate(kept):
        m = 32 * len(js)
        for eta, want in ((1.0 / m, 1.0), (1.0 / m * (1 + 1e-9), 0.0), (1e-300, 1.0), (1.5, 0.0)):
            I, _ = O.attention_statistic(q, k, kept, bs, 1.0, eta)
            assert all(I[i, j] == want for j in js)


def test_reconstruction_keeps_dropped_blocks():
    rng = np.random.default_rng(2)
    hist = rng.random((5, 5))
    cur = np.full((5, 5), np.nan)
    cur[1, 2], cur[4, 0] = 0.25, 0.75
    out = O.reconstruct_statistic(hist, cur)
    mask = np.zeros((5, 5), bool)
    mask[1, 2] = mask[4, 0] = True
    assert (out[~mask] == hist[~mask]).all() and out[1, 2] == 0.25 and out[4, 0] == 0.75
    with pytest.raises(ValueError):
        O.reconstruct_statistic(None, cur)


def test_attention_predictor_dense_anchor_equals_lstsq_of_dense_map():
    """Two dense warm-up updates: the anchors are the minimum-norm least
    squares fits (library lstsq) of 1 - S of Eq. 2 on the dense maps."""
    rng = np.random.default_rng(3)
    B, H, L, d, bs, tf = 1, 2, 256, 8, 32, 64
    q, k = rng.standard_normal((B, H, L, d)), rng.standard_normal((B, H, L, d))
    P = O.Predictor(B, H, L, d, bs, tf, warmup_m=2, delta_t=0, statistic="attention", eta=2e-3)
    n = P.n
    full = [[[list(range(n))] * n for _ in range(H)] for _ in range(B)]
    P.update(q, k, full, 1)
    P.update(q * 0.9, k, full, 2)
    for h in range(H):
        S = O.sparsity_map(q[0, h] * 0.9, k[0, h], bs, P.scale, 2e-3)
        Msys = O.design_matrix(n, P.regions)
        X, *_ = np.linalg.lstsq(Msys, (1.0 - S).reshape(-1), rcond=None)
        np.testing.assert_allclose(P.anchors[-1][1][0, h], X, atol=1e-10)
    sel = P.predict(None, None, 3, O.Budget("topk", density=0.5))
    assert all(len(r.kept) == O.topk_count(0.5, n) for r in sel[0][0])


# ---------------------------------------------------------------- a6 attention

def test_full_mask_equals_textbook_attention():
    rng = np.random.default_rng(9)
    L, d, bs = 200, 16, 64
    q, k, v = (rng.standard_normal((L, d)) for _ in range(3))
    n = O.num_blocks(L, bs)
    Ob, lse = O.attention(q, k, v, [list(range(n))] * n, bs, 1 / math.sqrt(d))
    A = q @ k.T / math.sqrt(d)
    np.testing.assert_allclose(Ob, scipy.special.softmax(A, axis=1) @ v, atol=1e-12)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(A, axis=1), atol=1e-12)


def test_outputs_are_convex_combinations_of_kept_values():
    """With V = identity the output row is the attention distribution:
    non-negative, summing to one, zero outside the kept blocks."""
    rng = np.random.default_rng(10)
    L, d, bs = 96, 8, 16
    q, k = rng.standard_normal((L, d)), rng.standard_normal((L, d))
    n = O.num_blocks(L, bs)
    lists = [sorted(rng.choice(n, size=int(rng.integers(1, n + 1)), replace=False).tolist())
             for _ in range(n)]
    P, _ = O.attention(q, k, np.eye(L), lists, bs, 0.5)
    assert (P >= 0).all()
    np.testing.assert_allclose(P.sum(axis=1), 1.0, atol=1e-12)
    for i in range(n):
        allowed = np.zeros(L, bool)
        for j in lists[i]:
            allowed[j * bs:(j + 1) * bs] = True
        assert (P[i * bs:(i + 1) * bs][:, ~allowed] == 0).all()


def test_single_block_bruteforce():
    rng = np.random.default_rng(11)
    L, d, bs = 40, 3, 16                 # blocks 16, 16, 8
    q, k, v = (rng.standard_normal((L, d)) for _ in range(3))
    lists = [[2], [0], [1]]
    Ob, lse = O.attention(q, k, v, lists, bs, 0.7)
    for p in range(L):
        j = lists[p // bs][0]
        keys = range(j * bs, min(L, (j + 1) * bs))
        logits = [0.7 * sum(q[p, c] * k[t, c] for c in range(d)) for t in keys]
        mx = max(logits)
        w = [math.exp(a - mx) for a in logits]
        s = sum(w)
        for c in range(d):
            want = sum(wi * v[t, c] for wi, t in zip(w, keys)) / s
            assert Ob[p, c] == pytest.approx(want, abs=1e-12)
        assert lse[p] == pytest.approx(mx + math.log(s), abs=1e-12)


def test_empty_list_gives_zero_output():
    q = np.ones((8, 2))
    Ob, lse = O.attention(q, q, q, [[], [0]], 4, 1.0)
    assert (Ob[:4] == 0).all() and np.isneginf(lse[:4]).all()


# ---------------------------------------------------------------- predictor

def test_predictor_schedule_and_errors():
    rng = np.random.default_rng(12)
    B, H, L, d, bs, tf = 1, 1, 256, 8, 32, 64
    q, k = rng.standard_normal((B, H, L, d)), rng.standard_normal((B, H, L, d))
    P = O.Predictor(B, H, L, d, bs, tf, warmup_m=2, delta_t=3)
    with pytest.raises(ValueError):
        P.predict(q, k, 3, O.Budget("topk", 0.5))
    P.collect(q, k, 1)
    P.collect(q, k, 2)
    with pytest.raises(ValueError):
        P.collect(q, k, 2)
    assert [t for t in range(3, 12) if P.is_anchor_step(t)] == [5, 8, 11]
    P1 = O.Predictor(B, H, L, d, bs, tf, warmup_m=2, delta_t=3, anchor_rule=1)
    assert [t for t in range(3, 12) if P1.is_anchor_step(t)] == [3, 6, 9]
    out = P.predict(q, k, 3, O.Budget("topk", 0.5))
    n = O.num_blocks(L, bs)
    assert all(len(r.kept) >= O.topk_count(0.5, n) for r in out[0][0])


def test_predictor_identical_steps_give_identical_masks():
    """Two identical anchors extrapolate to themselves (zero slope)."""
    rng = np.random.default_rng(13)
    q, k = rng.standard_normal((1, 2, 256, 8)), rng.standard_normal((1, 2, 256, 8))
    P = O.Predictor(1, 2, 256, 8, 32, 64, warmup_m=2, delta_t=0)
    P.collect(q, k, 1)
    P.collect(q, k, 2)
    a = P.predict(q, k, 3, O.Budget("mass", mass=0.8))
    b = P.predict(q, k, 9, O.Budget("mass", mass=0.8))
    for h in range(2):
        for ra, rb in zip(a[0][h], b[0][h]):
            assert ra.kept.tolist() == rb.kept.tolist()


# ---------------------------------------------- one-anchor extrapolation (a4)

def test_extrapolation_one_anchor_is_the_constant_sequence():
    """With one anchor the slope is zero (reading; the paper is silent): the
    prediction is the anchor's c, d at every step, which is what the
    two-anchor formula gives for a constant sequence (two equal anchors)."""
    rng = np.random.default_rng(17)
    n, F = 7, 3
    X2 = rng.standard_normal(O.num_coeffs(n, F))
    c2, d2, _ = O.split_coeffs(X2, n)
    for t2, t in [(1, 2), (5, 6), (5, 50), (3, 3)]:
        c, d = O.extrapolate(None, None, X2, t2, t, n)
        assert np.array_equal(c, c2) and np.array_equal(d, d2)
        cc, dd = O.extrapolate(X2.copy(), t2 - 1, X2, t2, t, n)
        assert np.array_equal(c, cc) and np.array_equal(d, dd)
    # the returned arrays are copies: the anchor is not changed through them
    c, d = O.extrapolate(None, None, X2, 1, 2, n)
    c += 1.0
    assert np.array_equal(O.split_coeffs(X2, n)[0], c2)


# ------------------------------------------------------- diagnostics (O10)

def _ragged_head(seed, L=37, d=4):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((L, d)), rng.standard_normal((L, d))


def test_exact_block_mass_library_softmax_bruteforce():
    """W(i, j) against scipy's softmax of every token row, summed by
    explicit loops over the tokens of each block (ragged: 8, 8, 8, 8, 5)."""
    q, k = _ragged_head(21)
    L, bs, scale = 37, 8, 0.6
    n = O.num_blocks(L, bs)
    W = O.exact_block_mass(q, k, bs, scale)
    for i in range(n):
        toks = [p for p in range(L) if p // bs == i]
        for j in range(n):
            tot = 0.0
            for p in toks:
                pr = scipy.special.softmax(scale * (k @ q[p]))
                tot += sum(pr[c] for c in range(L) if c // bs == j)
            assert W[i, j] == pytest.approx(tot / len(toks), rel=1e-12, abs=1e-15)
    np.testing.assert_allclose(W.sum(axis=1), 1.0, atol=1e-12)
    sub = O.exact_block_mass(q, k, bs, scale, rows=[1, 4])
    np.testing.assert_array_equal(sub[[1, 4]], W[[1, 4]])
    assert np.isnan(sub[[0, 2, 3]]).all()


def test_exact_block_mass_uniform_closed_form():
    """q = 0: uniform attention, W(i, j) = |j| / L (the tail block's share is
    its true size)."""
    _, k = _ragged_head(22)
    L, bs = 37, 8
    W = O.exact_block_mass(np.zeros_like(k), k, bs, 1.0)
    want = O.block_sizes(L, bs) / L
    for i in range(W.shape[0]):
        np.testing.assert_allclose(W[i], want, atol=1e-15)


def test_smfs_token_level_bruteforce():
    """SMFS = ||A . M||_F / ||A||_F with the block lists upsampled to a token
    mask M and A from scipy's softmax, against block_energy + smfs."""
    q, k = _ragged_head(23)
    L, bs, scale = 37, 8, 0.8
    n = O.num_blocks(L, bs)
    rng = np.random.default_rng(24)
    lists = [sorted(rng.choice(n, size=int(rng.integers(1, n + 1)), replace=False).tolist())
             for _ in range(n)]
    A = scipy.special.softmax(scale * (q @ k.T), axis=1)
    Mtok = np.zeros((L, L))
    for p in range(L):
        for c in range(L):
            if (c // bs) in lists[p // bs]:
                Mtok[p, c] = 1.0
    want = math.sqrt(((A * Mtok) ** 2).sum()) / math.sqrt((A ** 2).sum())
    E = O.block_energy(q, k, bs, scale)
    assert O.smfs(E, lists) == pytest.approx(want, rel=1e-12)
    full = [list(range(n))] * n
    assert O.smfs(E, full) == pytest.approx(1.0, rel=1e-14)
    # a subset of query blocks: the same ratio over those token rows
    rows = [0, 3]
    sel = np.array([p // bs in rows for p in range(L)])
    want_r = math.sqrt(((A * Mtok)[sel] ** 2).sum()) / math.sqrt((A[sel] ** 2).sum())
    assert O.smfs(E, lists, rows=rows) == pytest.approx(want_r, rel=1e-12)


def test_smfs_uniform_closed_form():
    """q = 0: every probability of a row is 1/L, so ||A . M||^2 counts the
    kept tokens / L^2 and ||A||^2 = 1: SMFS = sqrt(kept tokens) / L."""
    _, k = _ragged_head(25)
    L, bs = 37, 8
    lists = [[0], [1, 4], [0, 2, 3], [4], [0, 1, 2, 3, 4]]
    sizes = O.block_sizes(L, bs)
    kept_tokens = sum(int(sizes[i]) * int(sizes[lists[i]].sum()) for i in range(5))
    E = O.block_energy(np.zeros_like(k), k, bs, 1.0)
    assert O.smfs(E, lists) == pytest.approx(math.sqrt(kept_tokens) / L, rel=1e-13)


def test_mask_recall_hand_values():
    W = np.array([[0.5, 0.3, 0.2],
                  [0.1, 0.6, 0.3],
                  [0.25, 0.25, 0.5]])
    lists = [[0], [1, 2], [0, 2]]
    # row sums kept: 0.5, 0.9, 0.75 -> mean 0.7166...
    assert O.mask_recall(W, lists) == pytest.approx((0.5 + 0.9 + 0.75) / 3, abs=1e-15)
    assert O.mask_recall(W, lists, rows=[1]) == pytest.approx(0.9, abs=1e-15)
    assert O.mask_recall(W, [[0, 1, 2]] * 3) == pytest.approx(1.0, abs=1e-15)
    assert O.mask_recall(W, [[], [], []]) == 0.0


@pytest.mark.parametrize("L,bs,tf", [(256, 32, 64), (300, 32, 60)])
def test_nae_planted_fit_and_orthogonal_residual(L, bs, tf):
    """NAE(G, X) = ||G - M X|| / ||G||: 0 for a map the model reproduces
    exactly; for a planted map plus a residual orthogonal to the model space
    (projected out with the library least squares on the explicit M) the
    fit recovers the planted part and NAE = ||residual|| / ||G||."""
    n = O.num_blocks(L, bs)
    reg = O.frame_regions(L, bs, tf)
    rng = np.random.default_rng(26)
    Msys = O.design_matrix(n, reg)
    X0 = rng.standard_normal(Msys.shape[1])
    G0 = (Msys @ X0).reshape(n, n)
    assert O.nae(G0, O.fit(G0, reg), reg) < 1e-12
    Rraw = rng.standard_normal(n * n)
    Rperp = Rraw - Msys @ np.linalg.lstsq(Msys, Rraw, rcond=None)[0]
    G = G0 + 0.3 * Rperp.reshape(n, n)
    want = 0.3 * np.linalg.norm(Rperp) / np.linalg.norm(G)
    assert O.nae(G, O.fit(G, reg), reg) == pytest.approx(want, rel=1e-9)
    assert O.nae(G, X0, reg) == pytest.approx(want, rel=1e-9)


def test_sparsity_map_library_softmax_bruteforce():
    """Eq. 2 on the dense map: the fraction of scipy-softmax probabilities
    below eta per block, counted entry by entry (ragged)."""
    q, k = _ragged_head(27)
    L, bs, scale, eta = 37, 8, 0.9, 0.02
    n = O.num_blocks(L, bs)
    S = O.sparsity_map(q, k, bs, scale, eta)
    A = scipy.special.softmax(scale * (q @ k.T), axis=1)
    sizes = O.block_sizes(L, bs)
    for i in range(n):
        for j in range(n):
            below = sum(1 for p in range(L) for c in range(L)
                        if p // bs == i and c // bs == j and A[p, c] < eta)
            assert S[i, j] == below / (sizes[i] * sizes[j])
    # uniform attention (q = 0): 1/L is below eta iff eta > 1/L
    assert (O.sparsity_map(np.zeros_like(q), k, bs, 1.0, 1.0 / L * 1.01) == 1.0).all()
    assert (O.sparsity_map(np.zeros_like(q), k, bs, 1.0, 1.0 / L * 0.99) == 0.0).all()
