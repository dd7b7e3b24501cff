"""Helpers shared by the GPU parity tests and the smoke check.

They move seeded inputs to the device, drive the library through its C ABI
binding, and compare its outputs with the CPU oracle under the acceptance
rules: index lists bit-exact unless the oracle's boundary gap is at most
GAP (then the GPU row must still satisfy the selection invariants);
attention within MAX_ABS / MEAN_ABS of the fp64 oracle for bf16 inputs.
"""
from __future__ import annotations

import math

import numpy as np

GAP = 1e-5            # float32 score-key gap (and mass margin) below which a row is excused
MAX_ABS = 2e-2        # attention output, max |gpu - oracle|
MEAN_ABS = 2e-3       # attention output, mean |gpu - oracle|
LSE_ABS = 1e-3        # log-sum-exp, max |gpu - oracle|


def bf16_tensor(bits: np.ndarray, device="cuda"):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).to(device)


def bf16_to_f64(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def gpu_lists(kv_idx, kv_cnt) -> list:
    """Per (b, h) list of per-row kept lists from the device outputs."""
    idx = kv_idx.cpu().numpy()
    cnt = kv_cnt.cpu().numpy()
    B, H, n = cnt.shape
    return [[[idx[b, h, i, :cnt[b, h, i]].tolist() for i in range(n)] for h in range(H)]
            for b in range(B)]


def row_invariants_ok(row: list, n: int, forced: np.ndarray, mode: str, k: int,
                      sig_row: np.ndarray, tau: float, tol: float = GAP) -> bool:
    """What any correct selection of the row satisfies, whatever the order of
    keys within ``tol`` of each other (Section 5.3 with the per-row reading):

    * sorted, unique, in [0, n), non-empty, a superset of the forced blocks;
    * ordering: among the non-forced blocks no dropped block's float32 key
      exceeds a kept one's by more than ``tol``;
    * TOPK: exactly max(k, |forced|) blocks (capped at n);
    * MASS: the kept positive key mass reaches tau of the row's total
      (reach), and dropping the lowest-keyed non-forced kept block falls
      below it (minimality), unless that block is the one a row without
      forced blocks must keep.
    """
    if not row or row != sorted(set(row)) or row[0] < 0 or row[-1] >= n:
        return False
    fset = set(np.flatnonzero(forced).tolist())
    rset = set(row)
    if not fset.issubset(rset):
        return False
    keys = sig_row.astype(np.float32).astype(np.float64)
    kept_free = [j for j in row if j not in fset]
    dropped = [j for j in range(n) if j not in rset and j not in fset]
    if kept_free and dropped and keys[kept_free].min() < keys[dropped].max() - tol:
        return False
    if mode == "topk":
        free = n - len(fset)
        return len(row) == len(fset) + min(free, max(0, k - len(fset)))
    pos = np.maximum(keys, 0.0)
    total = math.fsum(pos)
    target = float(np.float32(tau)) * total
    slack = 1e-12 * total               # summation-order rounding of the two sides
    kept_mass = math.fsum(pos[row])
    if kept_mass < target - slack:
        return False
    kmin = 0 if fset else 1
    if len(kept_free) > kmin:
        last = min(kept_free, key=lambda j: (keys[j], -j))   # the last block of the order
        if kept_mass - pos[last] >= target + slack:
            return False
    return True


def pattern_head_ok(gpu_rows: list, ctil: np.ndarray, dtil: np.ndarray, n: int, K: int,
                    forced: np.ndarray, tol: float) -> bool:
    """Validity of a head's pattern-mode mask when keys tie within ``tol``:
    the K chosen patterns must contain every pattern whose float32 key is
    above the band [kth - tol, kth + tol] around the K-th key and none below
    it, so the mask must be (sure patterns) + forced + some band patterns,
    each chosen band pattern fully kept, with room for them in K."""
    vals = np.concatenate([ctil, dtil]).astype(np.float32).astype(np.float64)
    P = vals.size
    order = np.lexsort((np.arange(P), -vals))
    kth = vals[order[min(K, P) - 1]]
    sure = vals > kth + tol
    band = (np.abs(vals - kth) <= tol)
    i, j = np.indices((n, n))
    dg = j - i + n - 1
    col = 2 * n - 1 + j

    def cover(sel):
        return sel[dg] | sel[col]

    mask = np.zeros((n, n), bool)
    for r, js in enumerate(gpu_rows):
        if js != sorted(set(js)) or (js and (js[0] < 0 or js[-1] >= n)):
            return False
        mask[r, js] = True
    base = cover(sure) | forced
    if (base & ~mask).any():
        return False
    # band patterns whose every block is kept are the only ones that can be chosen
    full_band = np.zeros(P, bool)
    for pidx in np.flatnonzero(band):
        cells = (dg == pidx) if pidx < 2 * n - 1 else (col == pidx)
        full_band[pidx] = bool(mask[cells].all())
    explained = base | cover(full_band)
    if (mask & ~explained).any():
        return False
    need = K - int(sure.sum())
    return 0 <= need <= int(full_band.sum())


def compare_lists(gpu_rows: list, oracle_rows: list, sig: np.ndarray, forced: np.ndarray,
                  mode: str, k: int = 0, tau: float = 1.0, rows=None, gap=None):
    """Returns (n_rows, n_exact, n_excused, mismatches) for one head.

    gap: the excuse threshold on the oracle's boundary key gap (and mass
    margin), GAP by default; an array [n] gives one per row (rows whose
    scores carry a known uncertainty).  It is also the ordering tolerance of
    the invariants an excused row must satisfy."""
    n = sig.shape[0]
    exact = excused = 0
    bad = []
    for i in (range(n) if rows is None else rows):
        o = oracle_rows[i]
        g = gpu_rows[i]
        if g == o.kept.tolist():
            exact += 1
            continue
        gi = GAP if gap is None else float(np.broadcast_to(gap, (n,))[i])
        if (o.key_gap <= gi or o.mass_margin <= gi) and \
                row_invariants_ok(g, n, forced[i], mode, k, sig[i], tau, tol=gi):
            excused += 1
            continue
        bad.append(i)
    nrows = n if rows is None else len(rows)
    return nrows, exact, excused, bad


def compare_pattern_head(gpu_rows: list, oracle_rows: list, n: int, ctil=None, dtil=None,
                         K: int = 0, forced=None):
    """Pattern mode decides per head: the GPU lists must equal the oracle's
    unless the head's boundary key gap (scaled by n like the row scores) is
    within GAP, and then the GPU mask must be a valid choice of K patterns
    under ties within GAP / n (pattern_head_ok; checked when the predicted
    ctil, dtil are given).  Returns (n_rows, n_exact, excused_head,
    mismatching rows)."""
    same = [i for i in range(n) if gpu_rows[i] == oracle_rows[i].kept.tolist()]
    if len(same) == n:
        return n, n, False, []
    if n * oracle_rows[0].key_gap <= GAP and (
            ctil is None or pattern_head_ok(gpu_rows, ctil, dtil, n, K, forced, GAP / n)):
        return n, len(same), True, []
    return n, len(same), False, [i for i in range(n) if i not in set(same)]


def attention_errors(o_gpu: np.ndarray, o_ref: np.ndarray):
    diff = np.abs(o_gpu - o_ref)
    return float(diff.max()), float(diff.mean())


def kept_work(lists_bh, L: int, bs: int, d: int) -> float:
    """4 d sum |i||j| over kept pairs of all heads (flop)."""
    sizes = np.array([min(bs, L - j * bs) for j in range(math.ceil(L / bs))], dtype=np.int64)
    tot = 0
    for rows in lists_bh:
        for i, js in enumerate(rows):
            tot += int(sizes[i]) * int(sizes[np.asarray(js, dtype=np.int64)].sum())
    return 4.0 * d * tot
