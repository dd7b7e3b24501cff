"""Mask quality of the two block statistics at one budget (diagnostic).

TEST INFRASTRUCTURE: runs the CPU oracle only (plain fp64), never the HIP
library.  For a synthetic layer it predicts the masks of the first sparse
step after two warm-up anchors with
  * the pooled block-mass statistic (the hot path's default), and
  * the paper's statistic, I = 1 - S of Eq. 2 on the dense attention map,
at the same cumulative-mass budget, and reports per head
  * the kept density,
  * the mask mass recall: mean over query blocks of the dense attention
    mass the mask keeps,
  * the SMFS of the mask (the paper's SMFS appendix: ||A . M||_F / ||A||_F),
  * the NAE of the MOD fit to the statistic (Section 4.2, ||R|| / ||S||).
Recall and SMFS are taken over all query blocks of the small layer and over
a seeded sample of query blocks (including the last) at 720p.

The warm-up is one dense step (one anchor; the inputs do not drift, so a
second identical anchor would give the same zero-slope prediction).

usage: python oracle/mask_quality.py {small|hunyuan|wan} [rows per head] > out.jsonl
(at 720p, MALLOC_MMAP_MAX_=0 MALLOC_TRIM_THRESHOLD_=100000000000 keep the
large per-block temporaries in the heap instead of mapping them afresh)
"""
from __future__ import annotations

import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle as O  # noqa: E402
import workloads as W  # noqa: E402

WARM = 1
MASS = 0.75


def sampled_heads(cfg):
    """Two heads of each seeded type (the 720p parity tests' heads)."""
    types = W.head_types(cfg)
    heads = []
    for t in (W.HEAD_TEMPORAL, W.HEAD_SPATIAL, W.HEAD_GLOBAL):
        heads += [int(h) for h in np.flatnonzero(types == t)[:2]]
    return sorted(heads)


def head_report(cfg, h, qf, kf, rows):
    scale = 1.0 / math.sqrt(cfg.d)
    n = cfg.n
    budget = O.Budget("mass", mass=MASS)
    full = [list(range(n))] * n
    # pooled statistic
    P0 = O.Predictor(1, 1, cfg.L, cfg.d, cfg.block, cfg.frame_tokens, warmup_m=WARM, delta_t=0)
    P0.collect(qf, kf, WARM)
    sel0 = P0.predict(qf, kf, WARM + 1, budget)[0][0]
    G = P0.pooled_mass(qf, kf)[0, 0]
    nae0 = O.nae(G, P0.anchors[-1][1][0, 0], P0.regions)
    # the paper's statistic (Eq. 2 on the dense map of the warm-up step)
    P1 = O.Predictor(1, 1, cfg.L, cfg.d, cfg.block, cfg.frame_tokens, warmup_m=WARM, delta_t=0,
                     statistic="attention")
    P1.update(qf, kf, [[full]], WARM)
    sel1 = P1.predict(None, None, WARM + 1, budget)[0][0]
    nae1 = O.nae(P1.stat[0, 0], P1.anchors[-1][1][0, 0], P1.regions)
    # dense block mass and energy on the sampled query blocks
    Wm = O.exact_block_mass(qf[0, 0], kf[0, 0], cfg.block, scale, rows=rows)
    E = O.block_energy(qf[0, 0], kf[0, 0], cfg.block, scale, rows=rows)
    out = {"head": h, "type": W.HEAD_TYPE_NAMES[int(W.head_types(cfg)[h])], "rows": len(rows)}
    for name, sel, nae in (("pooled", sel0, nae0), ("paper", sel1, nae1)):
        lists = [r.kept.tolist() for r in sel]
        out[name] = {
            "density": round(sum(len(x) for x in lists) / n ** 2, 4),
            "recall": round(O.mask_recall(Wm, lists, rows=rows), 4),
            "smfs": round(O.smfs(E, lists, rows=rows), 4),
            "nae": round(nae, 4),
        }
    return out


def main():
    name = sys.argv[1] if len(sys.argv) > 1 else "small"
    nrows = int(sys.argv[2]) if len(sys.argv) > 2 else 48
    cfg = W.CONFIGS[name]
    if name == "small":
        heads, rowsel = list(range(cfg.H)), None
    else:
        heads, rowsel = sampled_heads(cfg), nrows
    for h in heads:
        t0 = time.perf_counter()
        q, k, _ = W.generate_heads(cfg, heads=[h])
        qf, kf = W.bf16_bits_to_f64(q), W.bf16_bits_to_f64(k)
        if rowsel is None:
            rows = list(range(cfg.n))
        else:
            rng = np.random.default_rng(1000 + h)
            rows = sorted(set(rng.choice(cfg.n - 1, size=rowsel - 1, replace=False).tolist()) | {cfg.n - 1})
        rep = head_report(cfg, h, qf, kf, rows)
        rep["layer"] = name
        rep["seconds"] = round(time.perf_counter() - t0, 1)
        print(json.dumps(rep), flush=True)


if __name__ == "__main__":
    main()
