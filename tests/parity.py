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
                      sig_row: np.ndarray, tau: float) -> bool:
    """What any correct selection of the row satisfies, whatever the tie order."""
    if row != sorted(set(row)) or (row and (row[0] < 0 or row[-1] >= n)) or not row:
        return False
    fset = set(np.flatnonzero(forced).tolist())
    if not fset.issubset(row):
        return False
    free = n - len(fset)
    if mode == "topk":
        return len(row) == len(fset) + min(free, max(0, k - len(fset)))
    keys = np.maximum(sig_row.astype(np.float32).astype(np.float64), 0.0)
    return keys[row].sum() >= np.float32(tau) * keys.sum() - 1e-9 * max(1.0, keys.sum())


def compare_lists(gpu_rows: list, oracle_rows: list, sig: np.ndarray, forced: np.ndarray,
                  mode: str, k: int = 0, tau: float = 1.0, rows=None):
    """Returns (n_rows, n_exact, n_excused, mismatches) for one head."""
    n = sig.shape[0]
    exact = excused = 0
    bad = []
    for i in (range(n) if rows is None else rows):
        o = oracle_rows[i]
        g = gpu_rows[i]
        if g == o.kept.tolist():
            exact += 1
            continue
        if (o.key_gap <= GAP or o.mass_margin <= GAP) and \
                row_invariants_ok(g, n, forced[i], mode, k, sig[i], tau):
            excused += 1
            continue
        bad.append(i)
    nrows = n if rows is None else len(rows)
    return nrows, exact, excused, bad


def compare_pattern_head(gpu_rows: list, oracle_rows: list, n: int):
    """Pattern mode decides per head: the GPU lists must equal the oracle's
    unless the head's boundary key gap (scaled by n like the row scores) is
    within GAP.  Returns (n_rows, n_exact, excused_head, mismatching rows)."""
    same = [i for i in range(n) if gpu_rows[i] == oracle_rows[i].kept.tolist()]
    if len(same) == n:
        return n, n, False, []
    if n * oracle_rows[0].key_gap <= GAP:
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
