"""The acceptance rules of the GPU parity tests, exercised on the CPU with
rows the oracle selects and rows planted to be wrong.

A GPU row that differs from the oracle's is excused only when the oracle's
boundary gap is within GAP and the row still satisfies everything a correct
selection satisfies (Section 5.3 with the per-row reading): forced blocks
kept, no dropped block scoring above a kept one, the TOPK count, and for
MASS both reaching the budget and being the shortest such prefix."""
import numpy as np

import oracle as O
from parity import GAP, compare_lists, pattern_head_ok, row_invariants_ok


def _row(n=12, seed=0):
    rng = np.random.default_rng(seed)
    sig = rng.uniform(0.1, 3.0, n)
    forced = np.zeros(n, bool)
    forced[[2, 3]] = True
    return sig, forced


def test_topk_oracle_row_is_valid_and_far_swap_is_not():
    sig, forced = _row()
    n, k = sig.size, 6
    sel = O.select_row_topk(sig, forced, k)
    row = sel.kept.tolist()
    assert row_invariants_ok(row, n, forced, "topk", k, sig, 1.0)
    free_kept = [j for j in row if not forced[j]]
    dropped = [j for j in range(n) if j not in row and not forced[j]]
    best_kept = max(free_kept, key=lambda j: sig[j])
    worst_dropped = min(dropped, key=lambda j: sig[j])
    swapped = sorted(set(row) - {best_kept} | {worst_dropped})
    assert not row_invariants_ok(swapped, n, forced, "topk", k, sig, 1.0)
    # same blocks but a forced one left out, one too many, unsorted, duplicates
    assert not row_invariants_ok([j for j in row if j != 2], n, forced, "topk", k, sig, 1.0)
    assert not row_invariants_ok(sorted(row + [worst_dropped]), n, forced, "topk", k, sig, 1.0)
    assert not row_invariants_ok(row[::-1], n, forced, "topk", k, sig, 1.0)
    assert not row_invariants_ok(row + [row[-1]], n, forced, "topk", k, sig, 1.0)
    assert not row_invariants_ok([], n, forced, "topk", k, sig, 1.0)


def test_topk_tie_at_the_boundary_is_excused():
    sig, forced = _row(seed=1)
    n, k = sig.size, 6
    sel = O.select_row_topk(sig, forced, k)
    row = sel.kept.tolist()
    free_kept = [j for j in row if not forced[j]]
    dropped = [j for j in range(n) if j not in row and not forced[j]]
    last = min(free_kept, key=lambda j: sig[j])
    first_out = max(dropped, key=lambda j: sig[j])
    sig2 = sig.copy()
    sig2[first_out] = sig2[last] - 0.5 * GAP          # a near tie across the boundary
    o = O.select_row_topk(sig2, forced, k)
    assert o.key_gap <= GAP
    swapped = sorted(set(o.kept.tolist()) - {last} | {first_out})
    assert row_invariants_ok(swapped, n, forced, "topk", k, sig2, 1.0)
    sq, fq = np.tile(sig2, (n, 1)), np.tile(forced, (n, 1))    # compare_lists takes n x n maps
    nr, ne, nx, bad = compare_lists([swapped], [o], sq, fq, "topk", k, rows=[0])
    assert (nr, ne, nx, bad) == (1, 0, 1, [])
    # a far swap in a row whose boundary happens to be a near tie is still rejected
    best_kept = max([j for j in o.kept.tolist() if not forced[j]], key=lambda j: sig2[j])
    worst = min([j for j in range(n) if j not in o.kept.tolist() and not forced[j]],
                key=lambda j: sig2[j])
    far = sorted(set(o.kept.tolist()) - {best_kept} | {worst})
    nr, ne, nx, bad = compare_lists([far], [o], sq, fq, "topk", k, rows=[0])
    assert bad == [0]


def test_mass_reach_and_minimality():
    sig, forced = _row(seed=2)
    n, tau = sig.size, 0.6
    o = O.select_row_mass(sig, forced, tau)
    row = o.kept.tolist()
    assert row_invariants_ok(row, n, forced, "mass", 0, sig, tau)
    free_kept = [j for j in row if not forced[j]]
    dropped = [j for j in range(n) if j not in row and not forced[j]]
    # one block more than needed (the best dropped one keeps the ordering): not minimal
    extra = max(dropped, key=lambda j: sig[j])
    assert not row_invariants_ok(sorted(row + [extra]), n, forced, "mass", 0, sig, tau)
    # the last kept block removed: the budget is not reached
    last = min(free_kept, key=lambda j: sig[j])
    assert not row_invariants_ok([j for j in row if j != last], n, forced, "mass", 0, sig, tau)
    # a far swap keeps a count but breaks the ordering
    best = max(free_kept, key=lambda j: sig[j])
    worst = min(dropped, key=lambda j: sig[j])
    assert not row_invariants_ok(sorted(set(row) - {best} | {worst}), n, forced, "mass", 0, sig, tau)


def test_mass_zero_total_keeps_the_minimum():
    n = 6
    sig = -np.ones(n)
    none = np.zeros(n, bool)
    assert row_invariants_ok([0], n, none, "mass", 0, sig, 0.5)
    assert not row_invariants_ok([0, 1], n, none, "mass", 0, sig, 0.5)
    forced = none.copy()
    forced[4] = True
    assert row_invariants_ok([4], n, forced, "mass", 0, sig, 0.5)
    assert not row_invariants_ok([0, 4], n, forced, "mass", 0, sig, 0.5)


def test_pattern_head_validity():
    rng = np.random.default_rng(5)
    n, K = 8, 5
    c, d = rng.uniform(0, 1, 2 * n - 1), rng.uniform(0, 1, n)
    forced = np.zeros((n, n), bool)
    sel = O.select_patterns(c, d, n, K, forced)
    rows = [r.kept.tolist() for r in sel]
    assert pattern_head_ok(rows, c, d, n, K, forced, 1e-7)
    # make the K-th and (K+1)-th patterns tie and choose the other one
    vals = np.concatenate([c, d])
    order = np.lexsort((np.arange(vals.size), -vals))
    a, b = order[K - 1], order[K]
    vals2 = vals.copy()
    vals2[b] = vals2[a]
    c2, d2 = vals2[:2 * n - 1], vals2[2 * n - 1:]
    chosen = np.zeros(vals.size, bool)
    chosen[order[:K]] = True
    chosen[a], chosen[b] = False, True
    i, j = np.indices((n, n))
    keep = chosen[j - i + n - 1] | chosen[2 * n - 1 + j]
    alt = [np.flatnonzero(keep[r]).tolist() for r in range(n)]
    assert pattern_head_ok(alt, c2, d2, n, K, forced, 1e-7)
    # a pattern far below the band chosen instead of the top one: rejected
    bad = chosen.copy()
    bad[order[0]], bad[order[-1]] = False, True
    keep = bad[j - i + n - 1] | bad[2 * n - 1 + j]
    assert not pattern_head_ok([np.flatnonzero(keep[r]).tolist() for r in range(n)], c2, d2, n, K,
                               forced, 1e-7)
    # one block too many
    extra = [list(r) for r in rows]
    missing = [x for x in range(n) if x not in extra[0]]
    extra[0] = sorted(extra[0] + missing[:1])
    assert not pattern_head_ok(extra, c, d, n, K, forced, 1e-7)
