#!/usr/bin/env python3
"""Benchmark of the MOD-DiT hot path on one MI355X.

A step is one pass of the whole hot path over one attention layer:
  mod_predict_block_mask at a re-anchor step (block pooling, pooled
  block-mass statistic, MOD fit, extrapolation, per-row selection)
  + mod_block_sparse_attn_fwd over the kept blocks.
Default workload: the HunyuanVideo-shaped 720p layer (B=1, H=24, d=128,
L=118,800 = 33 latent frames x 45x80, block 128) with a cumulative-mass
budget, synthetic seeded inputs already resident in HBM.

Prints one JSON line.  `value` is kept-block TFLOP/s of the whole step
(4*d*sum over kept block pairs of |i||j|, predictor time included);
`roofline` is the attention kernel against the bf16 MFMA peak;
`cpu_baseline` is the fp64 CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
ATTN_SOURCE = os.path.join(ROOT, "paper_2601_11641_amd", "csrc", "attn_fwd.hip")
PRED_SOURCE = os.path.join(ROOT, "paper_2601_11641_amd", "csrc", "predictor.hip")
COUNTER_SUMMARY = os.path.join(ROOT, "profiles", "attn_fwd_hunyuan720p_counters.json")

# rocprofv3 counter passes behind COUNTER_SUMMARY (one run each, see that file)
COUNTER_PASSES = {
    "A": "SQ_INSTS_VALU SQ_INSTS_MFMA SQ_INSTS_LDS SQ_INSTS_SALU SQ_INSTS_VALU_TRANS_F32 "
         "SQ_WAVES SQ_BUSY_CYCLES SQ_WAVE_CYCLES",
    "B": "SQ_VALU_MFMA_BUSY_CYCLES SQ_VALU_MFMA_COEXEC_CYCLES SQ_ACTIVE_INST_VALU "
         "SQ_ACTIVE_INST_LDS SQ_WAIT_INST_LDS SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_WAIT_ANY "
         "GRBM_GUI_ACTIVE",
    "C": "FETCH_SIZE",
    "D": "WRITE_SIZE TCC_HIT_sum TCC_MISS_sum",
    "E": "FETCH_SIZE",      # with --calibrate-copy
    "F": "WRITE_SIZE",      # with --calibrate-copy
}
METRIC = "ms/layer + kept-block TFLOP/s (% bf16 MFMA peak) at 720p video shapes"

WORKLOADS = {
    # name: (layer config, budget mode, budget value)
    "hunyuan-720p": ("hunyuan", "mass", 0.75),
    "wan-720p-d50": ("wan", "topk", 0.50),
    "wan-720p-d25": ("wan", "topk", 0.25),
    "wan-720p-d10": ("wan", "topk", 0.10),
    "wan-720p-d05": ("wan", "topk", 0.05),
    "hunyuan-720p-dense": ("hunyuan", "topk", 1.0),
    "hunyuan-720p-pattern": ("hunyuan", "pattern", 929),   # K = n patterns per head
    # 256 text tokens after the video (token-type-aware masking): 931 blocks
    "hunyuan-720p-text256": ("hunyuan+text256", "mass", 0.75),
    "small": ("small", "topk", 0.25),
    "small-d50": ("small", "topk", 0.50),
    "small-d100": ("small", "topk", 1.0),
    # one GPU's share when a layer is sharded by head over 8 GPUs
    "hunyuan-720p-h3": ("hunyuan@h3", "mass", 0.75),
    "wan-720p-h5": ("wan@h5", "mass", 0.75),
}


def layer_config(W, name):
    """A layer of the workload set; "<layer>+text<T>" appends T text tokens,
    "<layer>@h<H>" keeps its first H heads (one GPU's share of a layer
    sharded by head)."""
    name, _, heads = name.partition("@h")
    base, _, text = name.partition("+text")
    cfg = W.CONFIGS[base]
    if text:
        cfg = W.with_text(cfg, int(text))
    if heads:
        cfg = W.with_heads(cfg, int(heads))
    return cfg
WARMUP_M = 5          # dense warm-up steps before the timed sparse steps


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="hunyuan-720p", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=48,
                    help="query blocks of head 0 in the CPU-baseline attention sample")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run one plain device copy of 1 GiB (reference for the HBM "
                         "byte counters) and exit")
    ap.add_argument("--sweep", action="store_true",
                    help="Wan 720p layer at TOPK densities 0.5/0.25/0.10/0.05: attention time, "
                         "kept work, per-head imbalance and a linear time model; one JSON line "
                         "per density and one for the fit")
    ap.add_argument("--schedule", action="store_true",
                    help="50-step denoising schedule on the Hunyuan 720p shape (5 dense warm-up "
                         "steps, 45 predicted sparse steps) for re-anchor intervals 10 and 1; one "
                         "JSON line per interval")
    ap.add_argument("--share", action="store_true",
                    help="one GPU's share of a layer sharded by head over 8 GPUs (Hunyuan 3 of 24 "
                         "heads, Wan 5 of 40) against the whole layer on the same GPU, mass 0.75: "
                         "attention time, rate, per-head imbalance and the share's time over the "
                         "kept-work-proportional part of the whole layer's time; one JSON line "
                         "per layer")
    ap.add_argument("--count", action="store_true",
                    help="the Eq. 2 count pass of a dense step on the Hunyuan 720p layer alone "
                         "(mod_update_stats over full lists with the dense attention's LSE): "
                         "time per update and the rate on its QK^T flops; one JSON line")
    ap.add_argument("--trace-summary", nargs=2, metavar=("STATS_CSV", "BENCH_LOG"),
                    help="format a rocprofv3 --kernel-trace --stats CSV of a bench run (and the JSON "
                         "line that run printed) into profiles/hunyuan720p_step_kernel_stats.md and exit")
    ap.add_argument("--counter-summary", metavar="PMC_DIR",
                    help="summarise rocprofv3 counter passes A..F found under PMC_DIR/<pass>/ "
                         "into profiles/ and exit")
    return ap.parse_args()


# The attention source also holds the Eq. 2 count kernel after this banner;
# the attention's digest covers the text before it (the helpers, the work
# plan, the merge, the attention kernel and its launch).
ATTN_SECTION_END = "// Eq. 2 statistic of the attention map"


def source_digest(path: str = ATTN_SOURCE, upto: str | None = ATTN_SECTION_END) -> str:
    """Digest of a kernel source's code (the text before ``upto`` when the
    source holds it): comments dropped (string and character literals kept
    as written) and whitespace runs collapsed, so that an edit of the
    comments alone leaves it unchanged."""
    import hashlib
    with open(path, encoding="utf-8") as f:
        text = f.read()
    if upto is not None and upto in text:
        text = text[:text.index(upto)]
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            out.append(" ")
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    code = " ".join("".join(out).split())
    return hashlib.sha256(code.encode("utf-8")).hexdigest()[:16]


TRACE_SUMMARY = os.path.join(ROOT, "profiles", "hunyuan720p_step_kernel_stats.md")
TRACE_COMMAND = ("rocprofv3 --kernel-trace --stats -d gpurun_out/prof -o bench --output-format csv "
                 "-- python3 bench.py --steps 5 --warmup 2 --no-cpu-baseline")


def summarize_trace(stats_csv: str, bench_log: str):
    """Per-kernel time table of one profiled bench run (rocprofv3 kernel
    statistics), with the attention kernel's average checked against the
    event timing that bench.py printed for the same launches."""
    import csv
    import re
    with open(stats_csv) as f:
        rows = list(csv.DictReader(f))
    line = None
    with open(bench_log) as f:
        for t in f:
            if t.startswith("{"):
                line = json.loads(t)
    cfg = line["config"]
    total = sum(float(r["TotalDurationNs"]) for r in rows if "moddit" in r["Name"])
    out = ["# Kernel time summary: hunyuan-720p layer step", "",
           "Command (repo root, MI355X):", "", "    " + TRACE_COMMAND, "",
           f"Workload: {cfg['workload']}, {cfg['budget']} budget, kept density "
           f"{cfg['kept_density']}, kept work {cfg['kept_tflop']} TFLOP per step.",
           f"bench.py under the profiler reported attn_ms {cfg['attn_ms']} (HIP events on the launch "
           f"stream), predict_ms {cfg['predict_ms']}.", "",
           "| kernel | calls | avg us | share |", "|---|---|---|---|"]
    attn_avg = None
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        if "moddit" not in r["Name"]:
            continue
        name = re.sub(r"^void ", "", r["Name"])
        name = re.sub(r"moddit::\(anonymous namespace\)::", "", name)
        name = re.sub(r"\(.*$", "", name)
        avg = float(r["AverageNs"]) / 1e3
        if name.startswith("attn_fwd_kernel"):
            attn_avg = avg
        out.append(f"| {name} | {r['Calls']} | {avg:.1f} | {100 * float(r['TotalDurationNs']) / total:.2f}% |")
    out += ["", "Torch helper kernels of the kept-flop accounting (after the timed region) are omitted.",
            f"attn_fwd_kernel average {attn_avg:.1f} us against bench.py's event timing of the same "
            f"launches ({cfg['attn_ms']} ms)."]
    with open(TRACE_SUMMARY, "w") as f:
        f.write("\n".join(out) + "\n")
    print("\n".join(out))


def summarize_counters(pmc_dir: str):
    """Attention-kernel counters and HBM bytes from the rocprofv3 passes.

    FETCH_SIZE / WRITE_SIZE (KiB per dispatch) are scaled by what the same
    counters read for a plain 1 GiB device copy (bytes moved / bytes read by
    the counter)."""
    import csv
    import glob

    def load(name, match):
        vals = {}
        for f in glob.glob(os.path.join(pmc_dir, name, "**", "*counter_collection.csv"),
                           recursive=True):
            per = {}
            for r in csv.DictReader(open(f)):
                if match(r["Kernel_Name"]):
                    key = int(r["Dispatch_Id"])
                    per.setdefault(key, {}).setdefault(r["Counter_Name"], 0.0)
                    per[key][r["Counter_Name"]] += float(r["Counter_Value"])
                    per[key]["_ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
            if per:
                vals.update(per[max(per)])   # the last dispatch (a timed step)
        return vals
    attn = lambda k: "attn_fwd_kernel" in k   # noqa: E731
    copy = lambda k: "copy" in k.lower() or "elementwise" in k   # noqa: E731
    a = {}
    for p in "ABCD":
        a.update(load(p, attn))
    cf, cw = load("E", copy), load("F", copy)
    gib = float(1 << 30)
    fetch_scale = gib / (cf["FETCH_SIZE"] * 1024.0)
    write_scale = gib / (cw["WRITE_SIZE"] * 1024.0)
    fetch = a["FETCH_SIZE"] * 1024.0 * fetch_scale
    write = a["WRITE_SIZE"] * 1024.0 * write_scale
    xcd_cycles = a["GRBM_GUI_ACTIVE"] / 8.0
    mf = a["SQ_INSTS_MFMA"]
    out = {
        "kernel": "attn_fwd_kernel<128, 128>",
        "workload": "hunyuan-720p layer, mass budget 0.75 (bench.py --steps 1 --warmup 0)",
        "attn_source_sha256_16": source_digest(),
        "predictor_source_sha256_16": source_digest(PRED_SOURCE),
        "commands": [f"rocprofv3 --pmc {COUNTER_PASSES[p]} -d gpurun_out/pmc/{p} -o pmc "
                     f"--output-format csv -- python3 bench.py "
                     + ("--calibrate-copy" if p in "EF" else
                        "--steps 1 --warmup 0 --no-cpu-baseline") for p in "ABCDEF"],
        "copy_calibration": {"fetch_scale": round(fetch_scale, 4),
                             "write_scale": round(write_scale, 4)},
        "hbm_fetch_bytes": round(fetch), "hbm_write_bytes": round(write),
        "traffic_bytes": round(fetch + write),
        "mfma_busy_frac": round(a["SQ_VALU_MFMA_BUSY_CYCLES"] / (xcd_cycles * 1024), 4),
        "mfma_valu_coexec_frac": round(a["SQ_VALU_MFMA_COEXEC_CYCLES"]
                                       / a["SQ_VALU_MFMA_BUSY_CYCLES"], 4),
        "valu_per_mfma": round((a["SQ_INSTS_VALU"] - mf) / mf, 3),
        "lds_per_mfma": round(a["SQ_INSTS_LDS"] / mf, 3),
        "trans_per_mfma": round(a["SQ_INSTS_VALU_TRANS_F32"] / mf, 3),
        "lds_bank_conflict_frac": round(a["SQ_LDS_BANK_CONFLICT"] / a["SQ_LDS_IDX_ACTIVE"], 4),
        "l2_hit_rate": round(a["TCC_HIT_sum"] / (a["TCC_HIT_sum"] + a["TCC_MISS_sum"]), 4),
        "shader_clock_ghz": round(xcd_cycles / (a["_ns"] * 1e-9) / 1e9, 3),
        "duration_ms_under_profiler": round(a["_ns"] * 1e-6, 3),
    }
    # the pooling kernel (a1) of the same step: HBM-bound, Q and K read once
    pool = lambda k: "pool_kernel" in k   # noqa: E731
    pc, pd = load("C", pool), load("D", pool)
    if pc and pd:
        import workloads as W
        cfg = W.CONFIGS["hunyuan"]
        alg = 2.0 * cfg.B * cfg.H * cfg.L * cfg.d * 2 + 2.0 * cfg.B * cfg.H * cfg.n * cfg.d * 8
        pf, pw = pc["FETCH_SIZE"] * 1024.0 * fetch_scale, pd["WRITE_SIZE"] * 1024.0 * write_scale
        ns = 0.5 * (pc["_ns"] + pd["_ns"])
        out["pool_kernel"] = {
            "algorithmic_bytes": round(alg), "hbm_fetch_bytes": round(pf), "hbm_write_bytes": round(pw),
            "duration_us_under_profiler": round(ns * 1e-3, 1),
            "algorithmic_GBps": round(alg / (ns * 1e-9) / 1e9, 1),
            "measured_GBps": round((pf + pw) / (ns * 1e-9) / 1e9, 1),
            "frac_of_8TBps": round(alg / (ns * 1e-9) / 8e12, 4),
        }
    with open(COUNTER_SUMMARY, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out, indent=1))


def measured_traffic():
    """HBM bytes per attention launch from the committed counter summary, or
    None when the kernel source has changed since the counters were taken."""
    try:
        with open(COUNTER_SUMMARY) as f:
            c = json.load(f)
    except (OSError, ValueError):
        return None
    if c.get("attn_source_sha256_16") != source_digest():
        return None
    return c.get("traffic_bytes")


def measured_pool():
    """The pooling kernel's HBM figures from the committed counter summary
    (its duration under the profiler and the algorithmic bytes of the 720p
    Hunyuan layer), or None when the predictor source has changed since."""
    try:
        with open(COUNTER_SUMMARY) as f:
            c = json.load(f)
    except (OSError, ValueError):
        return None
    if c.get("predictor_source_sha256_16") != source_digest(PRED_SOURCE) or "pool_kernel" not in c:
        return None
    return c["pool_kernel"]


def calibrate_copy():
    """One device-to-device copy of exactly 1 GiB through torch's copy kernel;
    its FETCH_SIZE / WRITE_SIZE readings scale the counters of other kernels."""
    import torch
    src = torch.ones(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": 1 << 30}), flush=True)


def kept_flops(kv_idx, kv_cnt, L, bs, d):
    """4 d sum_{rows} |i| sum_{t < cnt} |kv_idx[t]| over every (b, h, i) row."""
    import torch
    n = kv_cnt.shape[-1]
    sizes = torch.tensor([min(bs, L - j * bs) for j in range(n)], dtype=torch.float64,
                         device=kv_idx.device)
    cnt = kv_cnt.reshape(-1, n).to(torch.int64)
    idx = kv_idx.reshape(-1, n, n).to(torch.int64)
    valid = torch.arange(n, device=idx.device)[None, None, :] < cnt[..., None]
    js = torch.where(valid, idx, torch.zeros_like(idx))
    colsum = (sizes[js] * valid).sum(-1)                 # [BH, n]
    return float(4.0 * d * (colsum * sizes[None, :]).sum().item())


def cpu_baseline(cfg, host, rows_h0, mode, val, total_flops, sample_rows):
    """Time the fp64 oracle on head 0: one re-anchor predict step for that
    head and the attention of `sample_rows` query blocks, scaled to the
    layer: T = H * t_predict(head) + t_attn(sample) * total / sample flops."""
    import numpy as np
    import oracle as O
    import workloads as W
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    q = W.bf16_bits_to_f64(host[0][:1, :1])
    k = W.bf16_bits_to_f64(host[1][:1, :1])
    v = W.bf16_bits_to_f64(host[2][0, 0])
    P = O.Predictor(1, 1, cfg.L, cfg.d, cfg.block, cfg.frame_tokens, warmup_m=WARMUP_M,
                    delta_t=1, text_tokens=cfg.text_tokens)
    P.collect(q, k, WARMUP_M - 1)
    P.collect(q, k, WARMUP_M)
    budget = O.Budget(mode, density=val if mode == "topk" else 1.0,
                      mass=val if mode == "mass" else 1.0,
                      patterns=int(val) if mode == "pattern" else 1)
    n = P.n_total
    rows = [int(r) for r in np.linspace(0, n - 1, min(sample_rows, n)).round()]
    sizes = O.block_sizes(cfg.L, cfg.block)
    sflops = 4.0 * cfg.d * sum(int(sizes[i]) * int(sizes[np.asarray(rows_h0[i])].sum())
                               for i in rows)

    def timed(step):
        t0 = time.perf_counter()
        P.predict(q, k, step, budget)
        t_pred = time.perf_counter() - t0
        t0 = time.perf_counter()
        O.attention(q[0, 0], k[0, 0], v, rows_h0, cfg.block, 1.0 / math.sqrt(cfg.d), rows=rows)
        t_attn = time.perf_counter() - t0
        return t_pred, t_attn, cfg.B * cfg.H * t_pred + t_attn * total_flops / sflops

    t_pred, t_attn, t_layer = timed(WARMUP_M + 1)
    one_thread = None
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            one_thread = timed(WARMUP_M + 2)[2]
    except Exception:
        pass
    return {
        "value": total_flops / t_layer / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"fp64 numpy oracle on head 0: one re-anchor predict step "
                   f"({t_pred:.2f} s, scaled x{cfg.B * cfg.H} heads) + attention of {len(rows)} "
                   f"of {n} query blocks ({t_attn:.2f} s, scaled by kept flops); "
                   f"layer estimate {t_layer:.1f} s"
                   + (f"; with 1 BLAS thread {one_thread:.1f} s ({total_flops / one_thread / 1e12:.4f} "
                      f"TFLOP/s)" if one_thread else "")),
    }


def _median_ms(fn, reps, stream):
    import numpy as np
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    for a, b in evs:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return float(np.median([a.elapsed_time(b) for a, b in evs]))


def run_sweep(args):
    """Wan 720p density sweep (TOPK): attention ms and kept work per density,
    per-head kept-work imbalance (max / mean over heads), and the least-squares
    model t_attn = a + b * kept TFLOP across the densities."""
    import numpy as np
    import torch

    import paper_2601_11641_amd as M
    import workloads as W

    cfg = W.CONFIGS["wan"]
    host = W.generate(cfg)
    dev = torch.device("cuda:0")
    qd, kd, vd = (torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev) for x in host)
    shape = M.make_shape(cfg.B, cfg.H, cfg.L, cfg.d, cfg.block, cfg.frame_tokens)
    stream = torch.cuda.current_stream()
    out = torch.empty_like(qd)
    rows = []
    for dens in (0.50, 0.25, 0.10, 0.05):
        st = M.Stats(shape, M.make_params(warmup_m=WARMUP_M, delta_t=1))
        n = st.n
        kv_idx = torch.empty((cfg.B, cfg.H, n, n), dtype=torch.int32, device=dev)
        kv_cnt = torch.empty((cfg.B, cfg.H, n), dtype=torch.int32, device=dev)
        M.mod_collect_stats(st.handle, qd, kd, WARMUP_M - 1)
        M.mod_collect_stats(st.handle, qd, kd, WARMUP_M)
        budget = M.make_budget("topk", density=dens)
        step = [WARMUP_M]

        def predict():
            step[0] += 1               # delta_t = 1: every call re-anchors at a new step
            M.mod_predict_block_mask(st.handle, qd, kd, step[0], budget, kv_idx, kv_cnt, stream)
        pred_ms = _median_ms(predict, 5, stream)
        ws_bytes = M.mod_attn_workspace_bytes(shape)
        ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
        attn = lambda: M.mod_block_sparse_attn_fwd(shape, qd, kd, vd, kv_idx, kv_cnt, 0.0, out,  # noqa: E731
                                                   None, ws, ws_bytes, stream)
        for _ in range(args.warmup):
            attn()
        attn_ms = _median_ms(attn, max(args.steps, 5), stream)
        per_head = np.array([kept_flops(kv_idx[:, h:h + 1], kv_cnt[:, h:h + 1], cfg.L, cfg.block, cfg.d)
                             for h in range(cfg.H)])
        flops = float(per_head.sum())
        rows.append((flops / 1e12, attn_ms))
        line = {"workload": "wan-720p layer: B=1 H=40 L=75600 d=128 block=128", "budget": f"topk {dens}",
                "k_blocks": int(kv_cnt[0, 0, 0].item()), "kept_tflop": round(flops / 1e12, 3),
                "predict_ms": round(pred_ms, 3), "attn_ms": round(attn_ms, 3),
                "attn_tflops": round(flops / (attn_ms * 1e-3) / 1e12, 1),
                "head_imbalance": round(float(per_head.max() / per_head.mean()), 3)}
        print(json.dumps(line), flush=True)
        st.close()
    x = np.array([r[0] for r in rows])
    y = np.array([r[1] for r in rows])
    A = np.stack([np.ones_like(x), x], 1)
    (a, b), *_ = np.linalg.lstsq(A, y, rcond=None)
    pred = a + b * x
    r2 = 1.0 - float(((y - pred) ** 2).sum() / ((y - y.mean()) ** 2).sum())
    print(json.dumps({"fit": "attn_ms = a + b * kept_tflop", "a_ms": round(float(a), 3),
                      "b_ms_per_tflop": round(float(b), 4), "r2": round(r2, 5),
                      "marginal_tflops": round(1e3 / float(b), 1)}), flush=True)


def _layer_attention(M, W, cfg, mode, val, args, dev, plan_only=False):
    """Predicted lists (re-anchor step) and the attention's median time on
    one layer; returns (attn_ms, kept flop per head, attn_ms with a
    plan-only workspace (no split walks) or None)."""
    import numpy as np
    import torch
    host = W.generate(cfg)
    qd, kd, vd = (torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev) for x in host)
    del host
    shape = M.make_shape(cfg.B, cfg.H, cfg.L, cfg.d, cfg.block, cfg.frame_tokens)
    stream = torch.cuda.current_stream()
    st = M.Stats(shape, M.make_params(warmup_m=WARMUP_M, delta_t=1))
    n = st.n
    kv_idx = torch.empty((cfg.B, cfg.H, n, n), dtype=torch.int32, device=dev)
    kv_cnt = torch.empty((cfg.B, cfg.H, n), dtype=torch.int32, device=dev)
    M.mod_collect_stats(st.handle, qd, kd, WARMUP_M - 1)
    M.mod_collect_stats(st.handle, qd, kd, WARMUP_M)
    budget = M.make_budget(mode, density=val) if mode == "topk" else M.make_budget(mode, mass=val)
    M.mod_predict_block_mask(st.handle, qd, kd, WARMUP_M + 1, budget, kv_idx, kv_cnt, stream)
    out = torch.empty_like(qd)
    ws_bytes = M.mod_attn_workspace_bytes(shape)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    attn = lambda: M.mod_block_sparse_attn_fwd(shape, qd, kd, vd, kv_idx, kv_cnt, 0.0, out,  # noqa: E731
                                               None, ws, ws_bytes, stream)
    for _ in range(args.warmup):
        attn()
    attn_ms = _median_ms(attn, max(args.steps, 5), stream)
    unsplit_ms = None
    if plan_only:
        pb = M.mod_attn_plan_bytes(shape)
        attn_u = lambda: M.mod_block_sparse_attn_fwd(shape, qd, kd, vd, kv_idx, kv_cnt, 0.0, out,  # noqa: E731
                                                     None, ws, pb, stream)
        for _ in range(args.warmup):
            attn_u()
        unsplit_ms = _median_ms(attn_u, max(args.steps, 5), stream)
        attn_ms = min(attn_ms, _median_ms(attn, max(args.steps, 5), stream))  # interleaved re-take
    per_head = np.array([kept_flops(kv_idx[:, h:h + 1], kv_cnt[:, h:h + 1], cfg.L, cfg.block, cfg.d)
                         for h in range(cfg.H)])
    st.close()
    return attn_ms, per_head, unsplit_ms


def run_share(args):
    """One GPU's share of a layer sharded by head over 8 GPUs, against the
    whole layer on the same GPU (mass 0.75).  makespan_vs_ideal is the
    share's attention time over the whole layer's time scaled by the
    share's fraction of the kept work: 1.0 means the share runs at the whole
    layer's rate, above 1 means the fewer, unevenly dense heads leave part
    of the chip idle."""
    import numpy as np
    import torch

    import paper_2601_11641_amd as M
    import workloads as W

    dev = torch.device("cuda:0")
    layers = {}
    for base, H in (("hunyuan", 3), ("wan", 5), ("hunyuan", 1)):
        full = W.CONFIGS[base]
        if base not in layers:
            layers[base] = _layer_attention(M, W, full, "mass", 0.75, args, dev)[:2]
        t_full, w_full = layers[base]
        share = W.with_heads(full, H)
        t_share, w_share, t_unsplit = _layer_attention(M, W, share, "mass", 0.75, args, dev, plan_only=True)
        assert np.allclose(w_share, w_full[:H])       # the share's heads are the layer's first H
        ideal = t_full * w_share.sum() / w_full.sum()
        print(json.dumps({
            "workload": f"{base}-720p share: heads 0..{H - 1} of {full.H} (B=1 L={full.L} d={full.d} "
                        f"block={full.block}), mass 0.75",
            "share_attn_ms": round(t_share, 3),
            "share_kept_tflop": round(float(w_share.sum()) / 1e12, 3),
            "share_attn_tflops": round(float(w_share.sum()) / (t_share * 1e-3) / 1e12, 1),
            "share_frac": round(float(w_share.sum()) / (t_share * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "share_head_density": [round(float(x) / (4.0 * full.d * full.L * full.L), 4) for x in w_share],
            "share_head_imbalance": round(float(w_share.max() / w_share.mean()), 3),
            "layer_attn_ms": round(t_full, 3),
            "layer_attn_tflops": round(float(w_full.sum()) / (t_full * 1e-3) / 1e12, 1),
            "makespan_vs_ideal": round(t_share / ideal, 3),
            "share_attn_ms_unsplit": round(t_unsplit, 3),
            "makespan_vs_ideal_unsplit": round(t_unsplit / ideal, 3),
        }), flush=True)


def run_count(args):
    """Eq. 2 statistic of a dense step on the Hunyuan 720p layer: one dense
    attention for the row LSE, then --warmup untimed and --steps timed
    mod_update_stats calls over the full lists (the count pass recomputes
    QK^T for every block, then the fit); HIP events on the launch stream."""
    import numpy as np
    import torch

    import paper_2601_11641_amd as M
    import workloads as W

    cfg = W.CONFIGS["hunyuan"]
    dev = torch.device("cuda:0")
    host = W.generate(cfg)
    q, k, v = (torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev) for x in host)
    del host
    shape = M.make_shape(cfg.B, cfg.H, cfg.L, cfg.d, cfg.block, cfg.frame_tokens)
    stream = torch.cuda.current_stream()
    n = cfg.n
    idx = torch.arange(n, dtype=torch.int32, device=dev).repeat(cfg.B * cfg.H * n).reshape(cfg.B, cfg.H, n, n)
    cnt = torch.full((cfg.B, cfg.H, n), n, dtype=torch.int32, device=dev)
    out = torch.empty_like(q)
    lse = torch.empty((cfg.B, cfg.H, cfg.L), dtype=torch.float32, device=dev)
    M.mod_block_sparse_attn_fwd(shape, q, k, v, idx, cnt, 0.0, out, lse, None, 0, stream)
    st = M.Stats(shape, M.make_params(warmup_m=1, statistic="attention"))
    times = []
    for t in range(1, args.warmup + args.steps + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        M.mod_update_stats(st.handle, q, k, lse, idx, cnt, t, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        if t > args.warmup:
            times.append(e0.elapsed_time(e1))
    st.close()
    ms = float(np.median(times))
    tflop = 2.0 * cfg.d * float(cfg.L) * float(cfg.L) * cfg.B * cfg.H / 1e12
    print(json.dumps({
        "workload": f"hunyuan-720p dense Eq. 2 count pass (B={cfg.B} H={cfg.H} L={cfg.L} d={cfg.d} "
                    f"block={cfg.block}), full lists",
        "steps": args.steps, "warmup": args.warmup,
        "update_ms_median": round(ms, 3), "update_ms_min": round(min(times), 3),
        "qk_tflop": round(tflop, 3), "qk_tflops": round(tflop / (ms / 1e3), 1),
        "frac_of_bf16_peak": round(tflop / (ms / 1e3) / PEAK_BF16_TFLOPS, 4),
    }), flush=True)


def run_schedule(args):
    """50 denoising steps on the Hunyuan 720p shape: steps 1-5 dense (full
    lists) with statistics collected at steps 4 and 5, steps 6-50 predicted
    masks (mass 0.75) + block-sparse attention; inputs drift between two draws
    (seeds 1005, 1006) as Q_t = cos(theta_t) Q0 + sin(theta_t) Q1 (same for K).
    Run with the pooled statistic at re-anchor intervals 10 and 1, and with
    the attention statistic of Eq. 2 / Eq. 5 at interval 10 (its re-anchor
    update runs after the step's attention and is counted as predictor
    time)."""
    import numpy as np
    import torch

    import paper_2601_11641_amd as M
    import workloads as W

    T = 50
    cfg = W.CONFIGS["hunyuan"]
    dev = torch.device("cuda:0")
    to_dev = lambda x: torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev)  # noqa: E731
    d0 = W.generate_heads(cfg, seed=1005)
    d1 = W.generate_heads(cfg, seed=1006)
    q0, k0, v0 = (to_dev(x) for x in d0)
    q1, k1 = to_dev(d1[0]), to_dev(d1[1])
    del d0, d1
    shape = M.make_shape(cfg.B, cfg.H, cfg.L, cfg.d, cfg.block, cfg.frame_tokens)
    stream = torch.cuda.current_stream()
    out = torch.empty_like(q0)
    n = cfg.n
    full_idx = torch.arange(n, dtype=torch.int32, device=dev).repeat(cfg.B * cfg.H * n).reshape(
        cfg.B, cfg.H, n, n)
    full_cnt = torch.full((cfg.B, cfg.H, n), n, dtype=torch.int32, device=dev)
    budget = M.make_budget("mass", mass=0.75)

    def inputs(t):
        th = 0.5 * math.pi * (t - 1) / (T - 1)
        c, s_ = math.cos(th), math.sin(th)
        return ((c * q0.float() + s_ * q1.float()).to(torch.bfloat16),
                (c * k0.float() + s_ * k1.float()).to(torch.bfloat16))

    lse = torch.empty((cfg.B, cfg.H, cfg.L), dtype=torch.float32, device=dev)
    for statistic, dt in (("pooled", 10), ("pooled", 1), ("attention", 10)):
        st = M.Stats(shape, M.make_params(warmup_m=WARMUP_M, delta_t=dt, statistic=statistic))
        attn_stat = statistic == "attention"
        kv_idx = torch.empty((cfg.B, cfg.H, n, n), dtype=torch.int32, device=dev)
        kv_cnt = torch.empty((cfg.B, cfg.H, n), dtype=torch.int32, device=dev)
        dense_ms, sparse_ms, pred_anchor, pred_other, collect_ms, dens = [], [], [], [], [], []
        for t in range(1, T + 1):
            qt, kt = inputs(t)
            torch.cuda.synchronize()
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            if t <= WARMUP_M:
                e[0].record(stream)
                M.mod_block_sparse_attn_fwd(shape, qt, kt, v0, full_idx, full_cnt, 0.0, out,
                                            lse if attn_stat else None, None, 0, stream)
                e[1].record(stream)
                if t >= WARMUP_M - 1:
                    if attn_stat:
                        M.mod_update_stats(st.handle, qt, kt, lse, full_idx, full_cnt, t, stream)
                    else:
                        M.mod_collect_stats(st.handle, qt, kt, t, stream)
                e[2].record(stream)
                torch.cuda.synchronize()
                dense_ms.append(e[0].elapsed_time(e[1]))
                if t >= WARMUP_M - 1:
                    collect_ms.append(e[1].elapsed_time(e[2]))
            else:
                anchor = (t - WARMUP_M) % dt == 0
                e.append(torch.cuda.Event(enable_timing=True))
                e[0].record(stream)
                M.mod_predict_block_mask(st.handle, qt, kt, t, budget, kv_idx, kv_cnt, stream)
                e[1].record(stream)
                M.mod_block_sparse_attn_fwd(shape, qt, kt, v0, kv_idx, kv_cnt, 0.0, out,
                                            lse if (attn_stat and anchor) else None, None, 0, stream)
                e[2].record(stream)
                if attn_stat and anchor:      # re-anchor from this step's attention (Eq. 5)
                    M.mod_update_stats(st.handle, qt, kt, lse, kv_idx, kv_cnt, t, stream)
                e[3].record(stream)
                torch.cuda.synchronize()
                (pred_anchor if anchor else pred_other).append(e[0].elapsed_time(e[1])
                                                              + e[2].elapsed_time(e[3]))
                sparse_ms.append(e[1].elapsed_time(e[2]))
                dens.append(kept_flops(kv_idx, kv_cnt, cfg.L, cfg.block, cfg.d)
                            / (4.0 * cfg.d * cfg.L * cfg.L * cfg.B * cfg.H))
        st.close()
        total_attn = sum(dense_ms) + sum(sparse_ms)
        total_pred = sum(pred_anchor) + sum(pred_other) + sum(collect_ms)
        print(json.dumps({
            "workload": "hunyuan-720p 50-step schedule (B=1 H=24 L=118800 d=128 block=128), mass 0.75",
            "statistic": statistic, "delta_t": dt, "steps": T, "dense_steps": WARMUP_M,
            "dense_attn_ms_avg": round(float(np.mean(dense_ms)), 3),
            "sparse_attn_ms_avg": round(float(np.mean(sparse_ms)), 3),
            "kept_density_avg": round(float(np.mean(dens)), 4),
            "kept_density_range": [round(float(min(dens)), 4), round(float(max(dens)), 4)],
            "collect_ms_avg": round(float(np.mean(collect_ms)), 3),
            "predict_anchor_ms_avg": round(float(np.mean(pred_anchor)), 3) if pred_anchor else None,
            "predict_other_ms_avg": round(float(np.mean(pred_other)), 3) if pred_other else None,
            "anchor_steps": len(pred_anchor),
            "total_attn_ms": round(total_attn, 1), "total_predictor_ms": round(total_pred, 1),
            "predictor_share": round(total_pred / (total_attn + total_pred), 4),
            "all_dense_attn_ms": round(float(np.mean(dense_ms)) * T, 1),
        }), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the hot path is measured at one GPU's share (bench.py --share); a layer shards by head "
              "across GPUs with no exchange between them.",
              file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.trace_summary:
        summarize_trace(*args.trace_summary)
        return
    if args.counter_summary:
        summarize_counters(args.counter_summary)
        return
    if args.sweep:
        run_sweep(args)
        return
    if args.schedule:
        run_schedule(args)
        return
    if args.count:
        run_count(args)
        return
    if args.share:
        run_share(args)
        return

    import numpy as np
    import torch

    import paper_2601_11641_amd as M
    import workloads as W

    cfg_name, mode, val = WORKLOADS[args.workload]
    cfg = layer_config(W, cfg_name)
    t0 = time.perf_counter()
    host = W.generate(cfg)
    t_gen = time.perf_counter() - t0

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def to_dev(bits):
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)

    qd, kd, vd = (to_dev(x) for x in host)
    shape = M.make_shape(cfg.B, cfg.H, cfg.L, cfg.d, cfg.block, cfg.frame_tokens, cfg.text_tokens)
    stats = M.Stats(shape, M.make_params(warmup_m=WARMUP_M, delta_t=1, tau_e=0.0, anchor_rule=0))
    n = stats.n
    budget = (M.make_budget(mode, density=val) if mode == "topk" else
              M.make_budget(mode, mass=val) if mode == "mass" else M.make_budget(mode, patterns=val))
    kv_idx = torch.empty((cfg.B, cfg.H, n, n), dtype=torch.int32, device=dev)
    kv_cnt = torch.empty((cfg.B, cfg.H, n), dtype=torch.int32, device=dev)
    out = torch.empty_like(qd)
    ws_bytes = M.mod_attn_workspace_bytes(shape)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    # dense warm-up anchors (untimed setup of the predictor state)
    M.mod_collect_stats(stats.handle, qd, kd, WARMUP_M - 1)
    M.mod_collect_stats(stats.handle, qd, kd, WARMUP_M)
    step = WARMUP_M

    def one_step(ev=None):
        nonlocal step
        step += 1                      # delta_t = 1: every sparse step re-anchors
        if ev is not None:
            ev[0].record(stream)
        M.mod_predict_block_mask(stats.handle, qd, kd, step, budget, kv_idx, kv_cnt, stream)
        if ev is not None:
            ev[1].record(stream)
        M.mod_block_sparse_attn_fwd(shape, qd, kd, vd, kv_idx, kv_cnt, 0.0, out, None,
                                    ws, ws_bytes, stream)
        if ev is not None:
            ev[2].record(stream)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for s in range(args.steps):
        one_step(evs[s])
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_step = total_ms / args.steps
    pred_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    attn_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))

    flops = kept_flops(kv_idx, kv_cnt, cfg.L, cfg.block, cfg.d)
    dense = 4.0 * cfg.d * cfg.L * cfg.L * cfg.B * cfg.H
    density = flops / dense
    attn_tflops = flops / (attn_ms * 1e-3) / 1e12
    line = {
        "metric": METRIC,
        "value": round(flops / (ms_step * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s (kept blocks, whole step)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload} layer: B={cfg.B} H={cfg.H} L={cfg.L} d={cfg.d} "
                        f"block={cfg.block} ({cfg.frames} frames x {cfg.hs}x{cfg.ws}"
                        + (f" + {cfg.text_tokens} text tokens)" if cfg.text_tokens else ")"),
            "budget": f"{mode} {val}",
            "kept_density": round(density, 4),
            "kept_tflop": round(flops / 1e12, 3),
            "predict_ms": round(pred_ms, 4),
            "attn_ms": round(attn_ms, 4),
            "attn_tflops": round(attn_tflops, 1),
            "input_generation_s": round(t_gen, 1),
        },
        "roofline": {
            "bound": "mfma",
            "achieved": round(attn_tflops, 1),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": measured_traffic() if args.workload == "hunyuan-720p" else None,
        },
    }
    # the predictor's HBM-bound kernel (block pooling: Q and K read once) against
    # the HBM peak, from the committed rocprofv3 counter passes of this layer
    pool = measured_pool() if args.workload == "hunyuan-720p" else None
    line["predictor"] = {
        "kernel": "pool_kernel",
        "bound": "hbm",
        "achieved": pool["algorithmic_GBps"] if pool else None,
        "peak": PEAK_HBM_GBS,
        "unit": "GB/s",
        "frac": pool["frac_of_8TBps"] if pool else None,
        "bytes": pool["algorithmic_bytes"] if pool else None,
        "kernel_us": pool["duration_us_under_profiler"] if pool else None,
        "predict_ms": round(pred_ms, 4),
        "predict_share_of_step": round(pred_ms / ms_step, 4),
    }
    if not args.no_cpu_baseline:
        idx = kv_idx[0, 0].cpu().numpy()
        cnt = kv_cnt[0, 0].cpu().numpy()
        rows_h0 = [idx[i, :cnt[i]].tolist() for i in range(n)]
        line["cpu_baseline"] = cpu_baseline(cfg, host, rows_h0, mode, val, flops, args.cpu_rows)
    stats.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
