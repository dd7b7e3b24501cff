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
    "small": ("small", "topk", 0.25),
}
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
    ap.add_argument("--counter-summary", metavar="PMC_DIR",
                    help="summarise rocprofv3 counter passes A..F found under PMC_DIR/<pass>/ "
                         "into profiles/ and exit")
    return ap.parse_args()


def source_digest() -> str:
    import hashlib
    with open(ATTN_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


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
                    delta_t=1)
    P.collect(q, k, WARMUP_M - 1)
    P.collect(q, k, WARMUP_M)
    budget = O.Budget(mode, density=val if mode == "topk" else 1.0,
                      mass=val if mode == "mass" else 1.0)
    t0 = time.perf_counter()
    P.predict(q, k, WARMUP_M + 1, budget)
    t_pred = time.perf_counter() - t0
    n = P.n
    rows = [int(r) for r in np.linspace(0, n - 1, min(sample_rows, n)).round()]
    t0 = time.perf_counter()
    O.attention(q[0, 0], k[0, 0], v, rows_h0, cfg.block, 1.0 / math.sqrt(cfg.d), rows=rows)
    t_attn = time.perf_counter() - t0
    sizes = O.block_sizes(cfg.L, cfg.block)
    sflops = 4.0 * cfg.d * sum(int(sizes[i]) * int(sizes[np.asarray(rows_h0[i])].sum())
                               for i in rows)
    t_layer = cfg.B * cfg.H * t_pred + t_attn * total_flops / sflops
    return {
        "value": total_flops / t_layer / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"fp64 numpy oracle on head 0: one re-anchor predict step "
                   f"({t_pred:.2f} s, scaled x{cfg.B * cfg.H} heads) + attention of {len(rows)} "
                   f"of {n} query blocks ({t_attn:.2f} s, scaled by kept flops); "
                   f"layer estimate {t_layer:.1f} s"),
    }


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the hot path is measured at one GPU's share, see DESIGN.md for sharding.",
              file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.counter_summary:
        summarize_counters(args.counter_summary)
        return

    import numpy as np
    import torch

    import paper_2601_11641_amd as M
    import workloads as W

    cfg_name, mode, val = WORKLOADS[args.workload]
    cfg = W.CONFIGS[cfg_name]
    t0 = time.perf_counter()
    host = W.generate(cfg)
    t_gen = time.perf_counter() - t0

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def to_dev(bits):
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)

    qd, kd, vd = (to_dev(x) for x in host)
    shape = M.make_shape(cfg.B, cfg.H, cfg.L, cfg.d, cfg.block, cfg.frame_tokens)
    stats = M.Stats(shape, M.make_params(warmup_m=WARMUP_M, delta_t=1, tau_e=0.0, anchor_rule=0))
    n = stats.n
    budget = M.make_budget(mode, density=val) if mode == "topk" else M.make_budget(mode, mass=val)
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
                        f"block={cfg.block} ({cfg.frames} frames x {cfg.hs}x{cfg.ws})",
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
            "traffic": measured_traffic(),
        },
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
