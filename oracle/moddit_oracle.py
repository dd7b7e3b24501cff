"""MOD-DiT hot-path oracle: plain, slow, obviously-correct CPU reference in fp64.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check of
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import this
module.  The product path (the HIP library and its Python binding) never
imports it and shares no code, tables or helpers with it.

What is computed (paper: MOD-DiT, arXiv 2601.11641), step by step in the
paper's order and notation, with one deliberate substitution: the block
statistic that the mixture-of-distributions (MOD) model is fitted to is the
*pooled block-mass estimate* G built from block means of Q and K, in place of
the attention sparsity map S of Eq. 2 (which needs the dense N x N attention).

  a1  block pooling            q_bar_i = mean of Q over block i (tail block
                               divided by its true token count)
  a2  block mass estimate      G(i,j) = |j| exp(s q_bar_i . k_bar_j) /
                               sum_j' |j'| exp(s q_bar_i . k_bar_j')
  a3  MOD fit                  Eq. 3/Eq. 4 least squares over the bases
                               C (parallel diagonals), D (verticals),
                               E (frame blocks), Appendix B.3; normal
                               equations M^T M X = M^T vec(G) with M^T M in
                               closed form (Appendix B.4) and the
                               minimum-norm solution (reading of the
                               Tikhonov lambda -> 0 limit, Appendix B.6)
  a4  linear prediction        Section 5.2 extrapolation of c and d from the
                               two latest anchors
  a5  mask                     Section 5.3: ranking of the predicted
                               intensities with the block-diagonal support
                               forced in when min(e) > tau_e
  a6  block-sparse attention   Eq. 1 softmax(A + M) V over the kept blocks

Floating-point convention: everything is fp64, except that the *decision*
of which blocks to keep is taken on float32-rounded scores (the precision of
the kernel's sort keys), with ties broken by ascending block index, and the
cumulative masses of those keys are summed in fp64.

Parity status of each function is stated in its docstring ("pinned by ...").
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

# ----------------------------------------------------------------------------
# geometry: blocks and frame regions
# ----------------------------------------------------------------------------


def num_blocks(L: int, bs: int) -> int:
    """n = ceil(L / B): blocks per dimension (Section 4.1, with a ragged tail).

    Pinned by test_frame_regions_aligned_and_overlapping (the last frame
    region of the 118,800-token layer ends at block n - 1) and
    test_kept_block_flops_full_mask_is_dense_count."""
    return -(-L // bs)


def block_sizes(L: int, bs: int) -> np.ndarray:
    """|j| = number of valid tokens of block j (the last one may be short).

    Pinned by test_block_mass_tail_is_mean_field_token_mass (a short tail
    weighted by its token count) and test_pool_bruteforce_ragged."""
    n = num_blocks(L, bs)
    return np.array([min(bs, L - j * bs) for j in range(n)], dtype=np.int64)


def frame_regions(L: int, bs: int, frame_tokens: int):
    """Block-diagonal regions, one per latent frame (Section 4.2, Appendix B.3).

    Frame f covers tokens [f*T_f, (f+1)*T_f); its region is the inclusive
    block range [floor(f*T_f/B), floor(((f+1)*T_f - 1)/B)].  When frames are
    not multiples of the block size, neighbouring regions share a block.
    Pinned by: explicit construction in the tests (aligned and misaligned).
    """
    if L % frame_tokens:
        raise ValueError("L must be a whole number of frames")
    F = L // frame_tokens
    return [((f * frame_tokens) // bs, ((f + 1) * frame_tokens - 1) // bs) for f in range(F)]


def num_coeffs(n: int, F: int) -> int:
    """|X| = 3n - 1 + |A| (Eq. 4).

    Pinned by test_flop_table_matches_paper (the solve counts of the Appendix
    C table follow from p)."""
    return 3 * n - 1 + F


# ----------------------------------------------------------------------------
# a1: block pooling
# ----------------------------------------------------------------------------


def pool(x: np.ndarray, bs: int) -> np.ndarray:
    """Mean of x over each block of ``bs`` tokens along axis -2.

    x: [..., L, d] (fp64).  Returns [..., n, d].  Pinned by brute force.
    """
    L = x.shape[-2]
    n = num_blocks(L, bs)
    out = np.empty(x.shape[:-2] + (n, x.shape[-1]), dtype=np.float64)
    for j in range(n):
        seg = x[..., j * bs:min(L, (j + 1) * bs), :]
        out[..., j, :] = seg.sum(axis=-2) / seg.shape[-2]
    return out


# ----------------------------------------------------------------------------
# a2: pooled block-mass estimate
# ----------------------------------------------------------------------------


def block_mass(qbar: np.ndarray, kbar: np.ndarray, sizes: np.ndarray, scale: float) -> np.ndarray:
    """G(i, j): attention mass that query block i puts on key block j when
    every token is replaced by its block mean (row-stochastic, n x n).

    qbar, kbar: [..., n, d].  The weight |j| counts the tokens of key block j,
    so a short tail block gets its share of the mass; without a tail this is
    a plain softmax over the block logits.  Pinned by the mean-field token
    brute force and by the plain softmax on aligned shapes.
    """
    logits = scale * np.einsum("...id,...jd->...ij", qbar, kbar)
    logits = logits - logits.max(axis=-1, keepdims=True)
    w = sizes.astype(np.float64) * np.exp(logits)
    return w / w.sum(axis=-1, keepdims=True)


# ----------------------------------------------------------------------------
# a3: the MOD linear model and its least-squares fit
# ----------------------------------------------------------------------------


def basis_C(n: int, delta: int) -> np.ndarray:
    """Parallel-to-main-diagonal basis: 1 where j - i = delta (Appendix B.3).

    Pinned by
    test_pattern_index_convention_picks_the_planted_diagonal_and_column and
    test_null_space_is_z."""
    i, j = np.indices((n, n))
    return (j - i == delta).astype(np.float64)


def basis_D(n: int, col: int) -> np.ndarray:
    """Vertical basis: 1 on column ``col`` (Appendix B.3).

    Pinned by
    test_pattern_index_convention_picks_the_planted_diagonal_and_column and
    test_null_space_is_z."""
    m = np.zeros((n, n))
    m[:, col] = 1.0
    return m


def basis_E(n: int, lo: int, hi: int) -> np.ndarray:
    """Block-diagonal basis: 1 on the square [lo, hi] x [lo, hi] (Appendix B.3).

    Pinned by test_normal_matrix_blocks_printed_in_paper (the closed-form
    blocks of Appendix B.4) and test_null_space_is_z."""
    m = np.zeros((n, n))
    m[lo:hi + 1, lo:hi + 1] = 1.0
    return m


def design_matrix(n: int, regions) -> np.ndarray:
    """M = [vec(C_1..C_{2n-1}), vec(D_1..D_n), vec(E_k)] (Eq. 4, Appendix B.3).

    vec() is row-major.  Column order: diagonal offsets -(n-1)..(n-1),
    then columns 0..n-1, then frame regions.  Only for small n.

    Pinned by test_null_space_is_z (SVD nullity one, spanned by the z of
    Appendix B.5) and test_normal_matrix_blocks_printed_in_paper.
    """
    cols = [basis_C(n, dl).ravel() for dl in range(-(n - 1), n)]
    cols += [basis_D(n, j).ravel() for j in range(n)]
    cols += [basis_E(n, lo, hi).ravel() for lo, hi in regions]
    return np.stack(cols, axis=1)


def normal_matrix(n: int, regions) -> np.ndarray:
    """M^T M in closed form, never building M (Appendix B.4).

    Blocks printed in the paper: C^T C = diag(n - |delta|), D^T D = n I,
    C^T D[delta, j] = 1 iff diagonal delta crosses column j, E^T E = diag(b^2)
    for disjoint frame regions of b blocks.  Blocks the paper leaves out,
    derived from the same basis definitions:
      C^T E[delta, f] = max(0, |R_f| - |delta|)   (cells of the square R_f
                        on diagonal delta)
      D^T E[j, f]     = |R_f| if j in R_f else 0
      E^T E[f, g]     = |R_f intersect R_g|^2     (reduces to b^2 on the
                        diagonal when regions are disjoint)
    Pinned by exact equality with the explicitly built M^T M.
    """
    F = len(regions)
    p = num_coeffs(n, F)
    N = np.zeros((p, p))
    oc, od, oe = 0, 2 * n - 1, 3 * n - 1
    deltas = np.arange(-(n - 1), n)
    for a, dl in enumerate(deltas):
        N[oc + a, oc + a] = n - abs(dl)
        for j in range(n):
            if 0 <= j - dl <= n - 1:
                N[oc + a, od + j] = N[od + j, oc + a] = 1.0
        for f, (lo, hi) in enumerate(regions):
            v = max(0, (hi - lo + 1) - abs(dl))
            N[oc + a, oe + f] = N[oe + f, oc + a] = v
    for j in range(n):
        N[od + j, od + j] = n
        for f, (lo, hi) in enumerate(regions):
            if lo <= j <= hi:
                N[od + j, oe + f] = N[oe + f, od + j] = hi - lo + 1
    for f, (lo, hi) in enumerate(regions):
        for g, (lo2, hi2) in enumerate(regions):
            ov = max(0, min(hi, hi2) - max(lo, lo2) + 1)
            N[oe + f, oe + g] = ov * ov
    return N


def rhs(G: np.ndarray, regions) -> np.ndarray:
    """M^T vec(G) as partitioned sums (Appendix B.4): diagonal sums over
    j - i = delta, column sums, and sums over each frame square.  G: [n, n].
    Pinned by equality with M^T vec(G) from the explicit M.
    """
    n = G.shape[0]
    rc = np.array([np.trace(G, offset=dl) for dl in range(-(n - 1), n)])
    rd = G.sum(axis=0)
    re = np.array([G[lo:hi + 1, lo:hi + 1].sum() for lo, hi in regions])
    return np.concatenate([rc, rd, re])


def null_vector(n: int, F: int) -> np.ndarray:
    """z = [1 (2n-1), -1 (n), 0 (F)]: sum_k C_k = sum_k D_k = all-ones, so
    M z = 0.  For F >= 2 it spans the null space of M (pinned by SVD)."""
    return np.concatenate([np.ones(2 * n - 1), -np.ones(n), np.zeros(F)])


def solve_min_norm(N: np.ndarray, r: np.ndarray, n: int, F: int) -> np.ndarray:
    """Minimum-norm solution of N X = r for N = M^T M with null space span(z).

    Reading of the paper's Tikhonov step (Appendix B.6): its lambda = 1e-8
    picks, up to O(lambda), the minimum-norm least-squares solution, which
    is what is computed here: (N + (n / z.z) z z^T) X = r is nonsingular and,
    because z.r = 0, its solution is orthogonal to z.  Pinned by
    numpy.linalg.lstsq on the explicit M and by planted-coefficient recovery.
    """
    z = null_vector(n, F)
    A = N + (n / z.dot(z)) * np.outer(z, z)
    return np.linalg.solve(A, r)


def fit(G: np.ndarray, regions) -> np.ndarray:
    """X = [c (2n-1), d (n), e (F)] minimising ||vec(G) - M X|| (Eq. 4),
    minimum-norm.  G: [n, n].

    Pinned by test_fit_equals_lstsq_minimum_norm,
    test_planted_coefficients_recovered and
    test_ridge_solution_close_to_minimum_norm."""
    n = G.shape[0]
    return solve_min_norm(normal_matrix(n, regions), rhs(G, regions), n, len(regions))


def fit_lstsq(G: np.ndarray, regions) -> np.ndarray:
    """The same fit through the explicit design matrix and LAPACK's SVD
    least squares (textbook minimum-norm solution).  Small n only.

    Pinned by test_fit_equals_lstsq_minimum_norm (LAPACK minimum-norm least
    squares)."""
    M = design_matrix(G.shape[0], regions)
    return np.linalg.lstsq(M, G.ravel(), rcond=None)[0]


def split_coeffs(X: np.ndarray, n: int):
    """(c, d, e) views of a coefficient vector.

    Pinned by test_extrapolation_reproduces_linear_sequences and
    test_gauge_invariance_of_scores."""
    return X[:2 * n - 1], X[2 * n - 1:3 * n - 1], X[3 * n - 1:]


def reconstruct(X: np.ndarray, n: int, regions) -> np.ndarray:
    """M X as an n x n map: c[j-i] + d[j] + sum of e_f over squares holding (i, j).

    Pinned by test_planted_coefficients_recovered (M X of a planted X)."""
    c, d, e = split_coeffs(X, n)
    i, j = np.indices((n, n))
    out = c[j - i + n - 1] + d[j]
    for f, (lo, hi) in enumerate(regions):
        out[lo:hi + 1, lo:hi + 1] += e[f]
    return out


def nae(G: np.ndarray, X: np.ndarray, regions) -> float:
    """Normalised approximation error ||R|| / ||S|| (Section 4.2) of the fit X
    to the statistic G, R = G - M X.  Reading: the norm is the 2-norm of the
    vectorised map (Eq. 4 fits vec(S)), i.e. the Frobenius norm.  Diagnostic.
    Pinned by a planted fit (NAE 0) and by a planted fit plus a residual
    orthogonal to the model space (NAE = |residual| / |G|)."""
    R = G - reconstruct(X, G.shape[0], regions)
    return float(np.linalg.norm(R) / np.linalg.norm(G))


# ----------------------------------------------------------------------------
# a4: linear prediction, gate
# ----------------------------------------------------------------------------


def extrapolate(X1: np.ndarray | None, t1: int | None, X2: np.ndarray, t2: int, t: int, n: int):
    """Predicted (c~, d~) at step t from anchors (t1, X1), (t2, X2), t1 < t2
    (Section 5.2): x~ = x2 + (x2 - x1) / (t2 - t1) * (t - t2).  With a single
    anchor the slope is taken as zero (the paper is silent; reading).  e is
    not extrapolated (Section 5.3 uses it only through the warm-up gate).
    Pinned by exact reproduction of linear sequences; the one-anchor branch
    by the constant sequence (two equal anchors give the same prediction at
    every step).
    """
    c2, d2, _ = split_coeffs(X2, n)
    if X1 is None:
        return c2.copy(), d2.copy()
    c1, d1, _ = split_coeffs(X1, n)
    w = (t - t2) / (t2 - t1)
    return c2 + (c2 - c1) * w, d2 + (d2 - d1) * w


def gate(e_anchors, tau_e: float) -> bool:
    """Block-diagonal support switch of Section 5.3: kept iff
    min over the warm-up anchors of the frame-averaged e exceeds tau_e.
    (Reading: the paper's e_min aggregates the per-frame e by their mean.)

    Pinned by test_gate_reading."""
    return bool(min(float(np.mean(e)) for e in e_anchors) > tau_e)


# ----------------------------------------------------------------------------
# a5: scores and per-row selection
# ----------------------------------------------------------------------------


def scores(ctil: np.ndarray, dtil: np.ndarray, n: int) -> np.ndarray:
    """sigma(i, j) = n * (c~[j - i] + d~[j]): the predicted diagonal and
    vertical intensities that cover block (i, j) (Section 5.3), scaled by n
    so that a uniform map scores 1.  Invariant under the gauge X -> X + a z.

    Pinned by test_gauge_invariance_of_scores and
    test_pattern_index_convention_picks_the_planted_diagonal_and_column."""
    i, j = np.indices((n, n))
    return n * (ctil[j - i + n - 1] + dtil[j])


def forced_mask(n: int, regions, gate_on: bool) -> np.ndarray:
    """K_E: blocks (i, j) that lie in a frame square R_f x R_f, when the gate
    is on (Section 5.3).  bool [n, n].

    Pinned by test_pattern_topk_invariants and
    test_text_rows_and_columns_full_and_video_part."""
    m = np.zeros((n, n), dtype=bool)
    if gate_on:
        for lo, hi in regions:
            m[lo:hi + 1, lo:hi + 1] = True
    return m


def text_blocks(L_video: int, L: int, bs: int) -> range:
    """Blocks holding at least one text token when a text segment of
    L - L_video tokens follows the video tokens (token-type-aware masking,
    Section 3); empty without text.  A block holding the last video tokens
    and the first text tokens counts as a text block.

    Pinned by test_text_blocks_layout."""
    if L == L_video:
        return range(0)
    return range(L_video // bs, num_blocks(L, bs))


def add_text(rows_video, L_video: int, L: int, bs: int):
    """Token-type-aware masking (Section 3): text tokens attend to and are
    attended by every token.  At block level (reading): the rows of text
    blocks keep every block; every other row keeps its video selection plus
    every text block.  rows_video: RowSelection per video query block (the
    selection over the video blocks, the mixed block already forced).
    Returns one RowSelection per block of the whole sequence.

    Pinned by test_text_rows_and_columns_full_and_video_part."""
    n = num_blocks(L, bs)
    tb = text_blocks(L_video, L, bs)
    if len(tb) == 0:
        return list(rows_video)
    out = []
    for i in range(n):
        if i in tb:
            out.append(RowSelection(np.arange(n), math.inf, math.inf))
        else:
            r = rows_video[i]
            kept = np.union1d(r.kept, np.arange(tb.start, n))
            out.append(RowSelection(kept, r.key_gap, r.mass_margin))
    return out


def topk_count(density: float, n: int) -> int:
    """k = clamp(ceil(rho * n), 1, n), with rho taken at float32 precision
    and a 1e-6 guard so that an integral rho*n is not pushed up by rounding.

    Pinned by test_topk_count."""
    rho = float(np.float32(density))
    return int(min(n, max(1, math.ceil(rho * n - 1e-6))))


@dataclass
class RowSelection:
    kept: np.ndarray          # ascending block indices
    key_gap: float            # boundary gap of the float32 keys (inf if no boundary)
    mass_margin: float        # |cum - tau*P| / P at the boundary (inf for TOPK)


def _order(keys: np.ndarray, cand: np.ndarray) -> np.ndarray:
    """Candidates sorted by (key descending, index ascending).

    Pinned by test_selection_ties_break_by_index and test_topk_row_bruteforce."""
    return cand[np.lexsort((cand, -keys[cand]))]


def select_row_topk(sig_row: np.ndarray, forced_row: np.ndarray, k: int) -> RowSelection:
    """Keep the forced blocks plus the k - |F_i| best-scoring others.

    Pinned by test_topk_row_bruteforce (all subsets of a small row) and
    test_selection_ties_break_by_index."""
    keys = sig_row.astype(np.float32).astype(np.float64)
    forced = np.flatnonzero(forced_row)
    cand = np.flatnonzero(~forced_row)
    order = _order(keys, cand)
    kk = max(0, k - forced.size)
    kk = min(kk, order.size)
    gap = math.inf
    if 0 < kk < order.size:
        gap = keys[order[kk - 1]] - keys[order[kk]]
    kept = np.sort(np.concatenate([forced, order[:kk]]))
    return RowSelection(kept, gap, math.inf)


def select_row_mass(sig_row: np.ndarray, forced_row: np.ndarray, tau: float) -> RowSelection:
    """Keep the forced blocks plus the shortest score-ordered prefix of the
    others whose positive-score mass reaches tau of the row's total
    (at least one block per row).

    Pinned by test_mass_row_bruteforce (shortest prefix by brute force) and
    test_mass_row_zero_mass_keeps_one_block."""
    keys = sig_row.astype(np.float32).astype(np.float64)
    pos = np.maximum(keys, 0.0)
    total = 0.0
    for v in pos:                       # plain sequential fp64 sums
        total += v
    forced = np.flatnonzero(forced_row)
    cand = np.flatnonzero(~forced_row)
    order = _order(keys, cand)
    target = float(np.float32(tau)) * total
    cum = 0.0
    for j in forced:
        cum += pos[j]
    kmin = 0 if forced.size else 1
    cums = [cum]
    for j in order:
        cum += pos[j]
        cums.append(cum)
    kk = order.size
    for t in range(kmin, order.size + 1):
        if cums[t] >= target:
            kk = t
            break
    gap = math.inf
    if 0 < kk < order.size:
        gap = keys[order[kk - 1]] - keys[order[kk]]
    margin = math.inf
    if total > 0:
        margin = (cums[kk] - target) / total
        if kk > kmin:
            margin = min(margin, (target - cums[kk - 1]) / total)
    kept = np.sort(np.concatenate([forced, order[:kk]]))
    return RowSelection(kept, gap, margin)


def pattern_values(ctil: np.ndarray, dtil: np.ndarray) -> np.ndarray:
    """The 3n - 1 predicted pattern intensities in pattern order: diagonals
    delta = -(n-1) .. n-1 (index delta + n - 1), then columns j (index
    2n - 1 + j).

    Pinned by test_pattern_topk_bruteforce and
    test_pattern_topk_planted_diagonal_and_column."""
    return np.concatenate([np.asarray(ctil, dtype=np.float64), np.asarray(dtil, dtype=np.float64)])


def select_patterns(ctil: np.ndarray, dtil: np.ndarray, n: int, K: int, forced: np.ndarray):
    """Section 5.3, pattern form of the mask: rank the predicted intensities
    of the parallel-diagonal and vertical patterns together, keep the K
    largest, and keep block (i, j) iff its diagonal j - i or its column j is
    among them, or it lies in the forced block-diagonal support K_E.  Keys
    are taken at float32 precision, ties by pattern index (reading).  The
    ranking depends on the gauge of (c, d); the minimum-norm solution is
    used.  Rows that no kept pattern reaches keep nothing.  Returns one
    RowSelection per query block; key_gap is the head's boundary gap (the
    K-th minus the (K+1)-th key, inf when K covers every pattern).

    Pinned by test_pattern_topk_bruteforce,
    test_pattern_topk_planted_diagonal_and_column,
    test_pattern_topk_all_patterns_keep_every_block_and_ties and
    test_pattern_topk_invariants."""
    vals = pattern_values(ctil, dtil).astype(np.float32).astype(np.float64)
    P = vals.size
    K = int(min(P, max(1, K)))
    order = np.lexsort((np.arange(P), -vals))
    chosen = np.zeros(P, dtype=bool)
    chosen[order[:K]] = True
    gap = math.inf if K == P else float(vals[order[K - 1]] - vals[order[K]])
    diag, col = chosen[:2 * n - 1], chosen[2 * n - 1:]
    i, j = np.indices((n, n))
    keep = diag[j - i + n - 1] | col[j] | forced
    return [RowSelection(np.flatnonzero(keep[r]), gap, math.inf) for r in range(n)]


def select(sig: np.ndarray, forced: np.ndarray, mode: str, density: float = 1.0,
           mass: float = 1.0):
    """Per-row selection over an n x n score map.  Returns a list of
    RowSelection, one per query block.

    Pinned by
    test_pattern_index_convention_picks_the_planted_diagonal_and_column and
    test_text_rows_and_columns_full_and_video_part."""
    n = sig.shape[0]
    if mode == "topk":
        k = topk_count(density, n)
        return [select_row_topk(sig[i], forced[i], k) for i in range(n)]
    if mode == "mass":
        return [select_row_mass(sig[i], forced[i], mass) for i in range(n)]
    raise ValueError(mode)


# ----------------------------------------------------------------------------
# a6: block-sparse attention
# ----------------------------------------------------------------------------


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, kept_lists, bs: int,
              scale: float, rows=None):
    """Eq. 1 with a block mask: for every query token p of block i,
    O_p = softmax over the tokens of the kept blocks of (scale q_p . k) times V,
    LSE_p = log sum exp(scale q_p . k) (natural log).  One head.

    q, k, v: [L, d] fp64; kept_lists[i]: kept key blocks of query block i.
    ``rows``: optional subset of query blocks (others are left as NaN).
    A query block with no kept block yields O = 0 and LSE = -inf.
    Pinned by dense textbook attention (full mask), convexity and brute force.
    """
    L, d = q.shape
    n = num_blocks(L, bs)
    O = np.full((L, v.shape[1]), np.nan)
    lse = np.full(L, np.nan)
    for i in (range(n) if rows is None else rows):
        qs = slice(i * bs, min(L, (i + 1) * bs))
        blocks = list(kept_lists[i])
        if not blocks:
            O[qs] = 0.0
            lse[qs] = -np.inf
            continue
        idx = np.concatenate([np.arange(j * bs, min(L, (j + 1) * bs)) for j in blocks])
        a = scale * (q[qs] @ k[idx].T)
        m = a.max(axis=1, keepdims=True)
        e = np.exp(a - m)
        s = e.sum(axis=1, keepdims=True)
        O[qs] = (e / s) @ v[idx]
        lse[qs] = (m + np.log(s))[:, 0]
    return O, lse


# ----------------------------------------------------------------------------
# the predictor over denoising steps (Algorithm 1, pooled statistic)
# ----------------------------------------------------------------------------


@dataclass
class Budget:
    mode: str = "topk"        # "topk" | "mass" | "pattern"
    density: float = 1.0      # TOPK: rho
    mass: float = 1.0         # MASS: tau
    patterns: int = 1         # PATTERN: K patterns per head


class Predictor:
    """One layer's mask predictor across denoising steps (Algorithm 1).

    collect(q, k, t)  dense warm-up step t: fit the MOD coefficients on the
                      pooled statistic and record the anchor (t, X).
    predict(q, k, t, budget)
                      sparse step t: on a re-anchor step fit first; then
                      extrapolate from the two latest anchors and select.
    Re-anchor steps: rule 0 uses t = m + i*dt (i >= 1, Section 5 notation);
    rule 1 uses t mod dt == 0 (Algorithm 1).  dt <= 0 never re-anchors.
    The block-diagonal gate is fixed at the first predict from the anchors
    held then (the warm-up anchors m-1, m).
    statistic="attention" fits the Eq. 2 statistic of the attention a step
    computed instead of the pooled block mass: update(q, k, kept, t) after
    the attention of a dense warm-up step or a re-anchor step (Eq. 5 keeps
    the dropped blocks at their history); predict() then never re-anchors
    by itself.
    q, k: fp64 [B, H, L, d].
    """

    def __init__(self, B, H, L, d, bs, frame_tokens, warmup_m, delta_t, tau_e=0.0,
                 anchor_rule=0, scale=None, statistic="pooled", eta=1e-4, text_tokens=0):
        # the MOD machinery runs over the video tokens; a text segment of
        # text_tokens tokens after them only changes the output lists
        self.L_total = L
        self.n_total = num_blocks(L, bs)
        L = L - text_tokens
        self.B, self.H, self.L, self.d, self.bs = B, H, L, d, bs
        self.n = num_blocks(L, bs)
        self.text = text_blocks(L, self.L_total, bs)
        self.regions = frame_regions(L, bs, frame_tokens)
        self.F = len(self.regions)
        self.sizes = block_sizes(L, bs)
        self.m, self.dt, self.tau_e, self.rule = warmup_m, delta_t, tau_e, anchor_rule
        self.scale = 1.0 / math.sqrt(d) if not scale else scale
        self.anchors = []          # list of (t, X [B, H, p])
        self.last_step = None
        self._last_predict = False
        self.gates = None          # bool [B, H]
        self._N = normal_matrix(self.n, self.regions)
        self.statistic, self.eta = statistic, eta
        self.stat = None           # "attention": reconstructed map [B, H, n, n]

    def forced(self, gate_on: bool) -> np.ndarray:
        """Forced video blocks: K_E when the gate is on, plus the block that
        holds the last video tokens and the first text tokens (a text block
        on the key side)."""
        f = forced_mask(self.n, self.regions, gate_on)
        if len(self.text) and self.text.start < self.n:
            f[:, self.text.start] = True
        return f

    def is_anchor_step(self, t: int) -> bool:
        if self.dt <= 0:
            return False
        if self.rule == 0:
            return t > self.m and (t - self.m) % self.dt == 0
        return t % self.dt == 0

    def pooled_mass(self, q, k):
        q, k = q[..., :self.L, :], k[..., :self.L, :]
        qb, kb = pool(q, self.bs), pool(k, self.bs)
        return block_mass(qb, kb, self.sizes, self.scale)

    def fit_all(self, q, k) -> np.ndarray:
        G = self.pooled_mass(q, k)
        X = np.empty((self.B, self.H, num_coeffs(self.n, self.F)))
        for b in range(self.B):
            for h in range(self.H):
                X[b, h] = solve_min_norm(self._N, rhs(G[b, h], self.regions), self.n, self.F)
        return X

    def _advance(self, t, after_predict_ok=False):
        """Steps increase across calls; an update may also follow the
        predict of the same step (it uses that step's attention)."""
        if self.last_step is not None and (t < self.last_step or (
                t == self.last_step and not (after_predict_ok and self._last_predict))):
            raise ValueError("steps must increase")
        self.last_step = t
        self._last_predict = False

    def collect(self, q, k, t):
        if self.statistic != "pooled":
            raise ValueError("collect() is the pooled statistic's entry; use update()")
        self._advance(t)
        self.anchors.append((t, self.fit_all(q, k)))
        self.anchors = self.anchors[-2:]

    def fit_map(self, Smap) -> np.ndarray:
        X = np.empty((self.B, self.H, num_coeffs(self.n, self.F)))
        for b in range(self.B):
            for h in range(self.H):
                X[b, h] = solve_min_norm(self._N, rhs(Smap[b, h], self.regions), self.n, self.F)
        return X

    def update_from_statistic(self, current, t):
        """Anchor at step t from the statistic of the blocks the step kept
        (current [B, H, n, n], NaN where not kept): Eq. 5 reconstruction,
        then the least-squares fit."""
        self._advance(t, after_predict_ok=True)
        self.stat = np.stack([np.stack([reconstruct_statistic(
            None if self.stat is None else self.stat[b, h], current[b, h])
            for h in range(self.H)]) for b in range(self.B)])
        self.anchors.append((t, self.fit_map(self.stat)))
        self.anchors = self.anchors[-2:]

    def update(self, q, k, kept, t, lse=None):
        """Attention statistic (Eq. 2) of step t's attention over the kept
        blocks (kept[b][h][i]: lists; full lists at a dense step), then
        update_from_statistic.  lse: optional [B, H, L] row LSE."""
        if self.statistic != "attention":
            raise ValueError("update() needs statistic='attention'")
        cur = np.empty((self.B, self.H, self.n, self.n))
        for b in range(self.B):
            for h in range(self.H):
                cur[b, h] = attention_statistic(q[b, h], k[b, h], kept[b][h], self.bs, self.scale,
                                                self.eta, None if lse is None else lse[b, h]
                                                )[0][:self.n, :self.n]
        self.update_from_statistic(cur, t)

    def prediction(self, t):
        """(c~, d~) per (b, h) at step t from the anchors held."""
        (t2, X2) = self.anchors[-1]
        (t1, X1) = self.anchors[-2] if len(self.anchors) > 1 else (None, None)
        out = []
        for b in range(self.B):
            row = []
            for h in range(self.H):
                row.append(extrapolate(None if X1 is None else X1[b, h], t1, X2[b, h], t2,
                                       t, self.n))
            out.append(row)
        return out

    def predict(self, q, k, t, budget: Budget):
        if not self.anchors:
            raise ValueError("predict before any collected step")
        self._advance(t)
        self._last_predict = True
        if self.gates is None:
            self.gates = np.array([[gate([split_coeffs(X[b, h], self.n)[2]
                                          for _, X in self.anchors], self.tau_e)
                                    for h in range(self.H)] for b in range(self.B)])
        if self.statistic == "pooled" and self.is_anchor_step(t):
            self.anchors.append((t, self.fit_all(q, k)))
            self.anchors = self.anchors[-2:]
        pred = self.prediction(t)
        result = []
        for b in range(self.B):
            row = []
            for h in range(self.H):
                ct, dt_ = pred[b][h]
                forced = self.forced(bool(self.gates[b, h]))
                if budget.mode == "pattern":
                    sel = select_patterns(ct, dt_, self.n, budget.patterns, forced)
                else:
                    sig = scores(ct, dt_, self.n)
                    sel = select(sig, forced, budget.mode, budget.density, budget.mass)
                row.append(add_text(sel, self.L, self.L_total, self.bs))
            result.append(row)
        return result


# ----------------------------------------------------------------------------
# Eq. 2 / Eq. 5: the attention sparsity statistic of the paper
# ----------------------------------------------------------------------------


def attention_statistic(q: np.ndarray, k: np.ndarray, kept_lists, bs: int, scale: float,
                        eta: float, lse: np.ndarray | None = None, tol: float = 0.0, rows=None,
                        return_lse: bool = False):
    """Eq. 2 on the attention map a step computed: for every kept block
    (i, j), the fraction of its probabilities A(p, q) = exp(scale q_p.k_q -
    LSE_p) that reach eta, where LSE_p normalises over the kept blocks of
    row block i (the masked map of Section 4.1; all blocks at a dense step).
    This is 1 - S(i, j), the informativeness the MOD model is fitted to
    (reading: larger = kept; the fraction is over the block's valid entries,
    so a short tail block is not padded with "sparse" entries).

    q, k: [L, d] fp64 of one head.  lse: optional [L] row LSE to compare
    against (default: the exact masked LSE).  Returns (I, amb): I [n, n]
    with NaN for blocks not kept; amb [n, n] the number of entries whose
    log-probability lies within tol of log(eta) (where two implementations
    may round the decision differently).  rows: optional subset of query
    blocks (the other rows stay NaN / 0).  return_lse: also return the row
    LSE used ([L], NaN outside ``rows``).

    Pinned by test_attention_statistic_bruteforce (entry by entry from the
    dense attention) and
    test_attention_statistic_uniform_attention_closed_form.
    """
    L = q.shape[0]
    n = num_blocks(L, bs)
    I = np.full((n, n), np.nan)
    amb = np.zeros((n, n), dtype=np.int64)
    used = np.full(L, np.nan)
    log_eta = math.log(eta)
    for i in (range(n) if rows is None else rows):
        blocks = list(kept_lists[i])
        if not blocks:
            continue
        qs = slice(i * bs, min(L, (i + 1) * bs))
        idx = np.concatenate([np.arange(j * bs, min(L, (j + 1) * bs)) for j in blocks])
        a = scale * (q[qs] @ k[idx].T)
        if lse is None:
            mx = a.max(axis=1, keepdims=True)
            row_lse = mx + np.log(np.exp(a - mx).sum(axis=1, keepdims=True))
        else:
            row_lse = lse[qs][:, None]
        used[qs] = row_lse[:, 0]
        logp = a - row_lse
        start = 0
        for j in blocks:
            w = min(L, (j + 1) * bs) - j * bs
            blk = logp[:, start:start + w]
            start += w
            I[i, j] = float((blk >= log_eta).sum()) / blk.size
            amb[i, j] = int((np.abs(blk - log_eta) < tol).sum())
    return (I, amb, used) if return_lse else (I, amb)


def reconstruct_statistic(history: np.ndarray | None, current: np.ndarray) -> np.ndarray:
    """Eq. 5 at block level: entries computed at this step (finite in
    ``current``) replace the history; blocks the mask dropped keep their
    historical value.  The first map must be dense (Algorithm 1 starts the
    sequence from the full attention of the warm-up).

    Pinned by test_reconstruction_keeps_dropped_blocks."""
    if history is None:
        if np.isnan(current).any():
            raise ValueError("the first statistic must cover every block (dense step)")
        return current.copy()
    out = history.copy()
    kept = ~np.isnan(current)
    out[kept] = current[kept]
    return out


# ----------------------------------------------------------------------------
# measurement and diagnostics
# ----------------------------------------------------------------------------


def paper_op_counts(N: int, H: int, d: int, p: int):
    """Operation counts in the units of the paper's Appendix C table:
    full attention 2 N^2 d H, conversion to the sparsity map N^2 H (one
    compare per attention entry), dense solve p^3 / 3 (one Cholesky of the
    p x p normal matrix).  Returned in TFLOP.

    Pinned by test_flop_table_matches_paper (the values printed in the
    Appendix C table, tests/golden/paper_flop_table.json)."""
    return 2.0 * N * N * d * H / 1e12, 1.0 * N * N * H / 1e12, p ** 3 / 3.0 / 1e12


def kept_block_flops(kept_lists, L: int, bs: int, d: int) -> float:
    """4 d sum over kept (i, j) of |i| |j|: QK^T and PV multiply-adds counted
    as 2 flops each, valid tokens only.  kept_lists: iterable over heads of
    per-row lists.

    Pinned by test_kept_block_flops_full_mask_is_dense_count (4 d L^2 for a
    full mask)."""
    sizes = block_sizes(L, bs)
    tot = 0
    for rows in kept_lists:
        for i, js in enumerate(rows):
            tot += int(sizes[i]) * int(sizes[np.asarray(js, dtype=np.int64)].sum())
    return 4.0 * d * tot


def exact_block_mass(q: np.ndarray, k: np.ndarray, bs: int, scale: float, rows=None) -> np.ndarray:
    """W(i, j) = (1/|i|) sum_{p in i} sum_{q in j} P(p, q) from the dense
    attention probabilities P of one head (Eq. 1 without a mask): the share
    of query block i's attention that lands in key block j (diagnostic; rows
    sum to 1).  rows: optional subset of query blocks (the others stay NaN).
    Pinned by a library softmax brute force on a ragged shape and by the
    uniform-attention closed form W(i, j) = |j| / L."""
    L = q.shape[0]
    n = num_blocks(L, bs)
    W = np.full((n, n), np.nan)
    for i in (range(n) if rows is None else rows):
        qs = slice(i * bs, min(L, (i + 1) * bs))
        a = scale * (q[qs] @ k.T)
        P = np.exp(a - a.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        for j in range(n):
            W[i, j] = P[:, j * bs:min(L, (j + 1) * bs)].sum() / P.shape[0]
    return W


def block_energy(q: np.ndarray, k: np.ndarray, bs: int, scale: float, rows=None) -> np.ndarray:
    """E(i, j) = sum_{p in i} sum_{q in j} P(p, q)^2 over the dense attention
    probabilities P of one head: the squared Frobenius norm of block (i, j)
    of the attention map, from which the SMFS of a block mask follows
    (diagnostic).  rows: optional subset of query blocks (others NaN).
    Pinned with smfs()."""
    L = q.shape[0]
    n = num_blocks(L, bs)
    E = np.full((n, n), np.nan)
    for i in (range(n) if rows is None else rows):
        qs = slice(i * bs, min(L, (i + 1) * bs))
        a = scale * (q[qs] @ k.T)
        P = np.exp(a - a.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        for j in range(n):
            blk = P[:, j * bs:min(L, (j + 1) * bs)]
            E[i, j] = (blk * blk).sum()
    return E


def smfs(E: np.ndarray, kept_lists, rows=None) -> float:
    """Sparsity Mask Fidelity Score (the paper's SMFS appendix):
    ||A . M||_F / ||A||_F for the dense attention map A and the token mask M
    of the block lists, from the block energies E of block_energy() (over
    the query blocks ``rows``, default all).  The paper calls a lower score
    better although the ratio measures the retained norm; it is reported as
    defined (reading: higher = more of the map retained).  Pinned by a
    token-level brute force with the upsampled mask and by the uniform
    closed form sqrt(kept tokens) / L."""
    rr = range(E.shape[0]) if rows is None else rows
    kept = sum(E[i, np.asarray(kept_lists[i], dtype=np.int64)].sum() for i in rr)
    total = sum(E[i].sum() for i in rr)
    return float(math.sqrt(kept / total))


def sparsity_map(q: np.ndarray, k: np.ndarray, bs: int, scale: float, eta: float) -> np.ndarray:
    """Eq. 2: fraction of attention probabilities below eta in each block
    (probabilities read as the softmax output, as in Algorithm 1).  Diagnostic.
    Pinned by the per-entry library softmax brute force of the statistic
    (its complement on full lists) and the uniform-attention closed form."""
    L = q.shape[0]
    n = num_blocks(L, bs)
    S = np.zeros((n, n))
    for i in range(n):
        qs = slice(i * bs, min(L, (i + 1) * bs))
        a = scale * (q[qs] @ k.T)
        P = np.exp(a - a.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        for j in range(n):
            blk = P[:, j * bs:min(L, (j + 1) * bs)]
            S[i, j] = (blk < eta).mean()
    return S


def mask_recall(W: np.ndarray, kept_lists, rows=None) -> float:
    """Mean over query blocks (``rows``, default all) of the dense attention
    mass the mask keeps: sum over kept j of W(i, j) (diagnostic).  Pinned by
    hand-computed values and the full-mask value 1."""
    rr = range(W.shape[0]) if rows is None else rows
    return float(np.mean([W[i, np.asarray(kept_lists[i], dtype=np.int64)].sum() for i in rr]))
