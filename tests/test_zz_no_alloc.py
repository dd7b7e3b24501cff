"""The no-allocation attention entry point against the one with a caller
workspace, through the C ABI: identical outputs on two calls in a row (the
second on a smaller layer, so the library's array holds the first call's
plan when the second starts), both within the oracle's tolerance on
sampled query blocks, and shapes whose plan would not fit rejected on the
host before anything is enqueued."""
import math

import numpy as np
import pytest

import oracle as O
import workloads as W
from parity import LSE_ABS, MAX_ABS, MEAN_ABS, attention_errors, bf16_tensor, bf16_to_f64

import paper_2601_11641_amd as M

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _random_lists(cfg, seed, density):
    """Seeded ascending lists of about density * n blocks per row (at least one)."""
    n = cfg.n
    rng = np.random.default_rng(seed)
    idx = np.zeros((cfg.B, cfg.H, n, n), np.int32)
    cnt = np.zeros((cfg.B, cfg.H, n), np.int32)
    rows = [[[None] * n for _ in range(cfg.H)] for _ in range(cfg.B)]
    for b in range(cfg.B):
        for h in range(cfg.H):
            for i in range(n):
                m = int(rng.integers(1, max(2, int(density * n) + 1)))
                js = np.sort(rng.choice(n, size=m, replace=False)).astype(np.int32)
                idx[b, h, i, :m] = js
                cnt[b, h, i] = m
                rows[b][h][i] = js.tolist()
    return torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda(), rows


def _both(cfg, host, dev, seed, density):
    qd, kd, vd = dev
    shape = M.make_shape(cfg.B, cfg.H, cfg.L, cfg.d, cfg.block, cfg.frame_tokens)
    assert M.mod_attn_workspace_bytes(shape) <= M.MOD_ATTN_NOALLOC_MAX_BYTES
    idx, cnt, rows = _random_lists(cfg, seed, density)
    o_ws = torch.zeros_like(qd)
    l_ws = torch.zeros((cfg.B, cfg.H, cfg.L), dtype=torch.float32, device="cuda")
    M.mod_block_sparse_attn_fwd(shape, qd, kd, vd, idx, cnt, 0.0, o_ws, l_ws)
    o_na = torch.full_like(qd, float("nan"))
    l_na = torch.full((cfg.B, cfg.H, cfg.L), float("nan"), dtype=torch.float32, device="cuda")
    M.mod_block_sparse_attn_fwd_noalloc(shape, qd, kd, vd, idx, cnt, 0.0, o_na, l_na)
    torch.cuda.synchronize()
    # the same kernels over the same lists: bit-identical outputs
    assert torch.equal(o_na.view(torch.int16), o_ws.view(torch.int16))
    assert torch.equal(l_na, l_ws)
    og, lg = bf16_to_f64(o_na), l_na.cpu().numpy().astype(np.float64)
    rng = np.random.default_rng(seed + 1)
    for b, h in {(0, 0), (cfg.B - 1, cfg.H - 1)}:
        sample = sorted(set(rng.choice(cfg.n, size=min(4, cfg.n), replace=False).tolist())
                        | {cfg.n - 1})
        qf, kf, vf = (W.bf16_bits_to_f64(x[b, h]) for x in host)
        Oo, Lo = O.attention(qf, kf, vf, rows[b][h], cfg.block, 1.0 / math.sqrt(cfg.d), rows=sample)
        for i in sample:
            sl = slice(i * cfg.block, min(cfg.L, (i + 1) * cfg.block))
            mx, mean = attention_errors(og[b, h, sl], Oo[sl])
            assert mx <= MAX_ABS and mean <= MEAN_ABS, (b, h, i, mx, mean)
            assert np.abs(lg[b, h, sl] - Lo[sl]).max() <= LSE_ABS


def test_noalloc_matches_workspace_entry_on_two_calls():
    big = W.CONFIGS["small"]                     # H=8, L=8192, d=128, block 128
    print(f"no-alloc call 1: {big.name} B={big.B} H={big.H} L={big.L} d={big.d}", flush=True)
    host = W.generate(big)
    _both(big, host, tuple(bf16_tensor(x) for x in host), seed=71, density=0.4)
    small = W.CONFIGS["tiny"]                    # H=2, L=1024, d=64, block 64: fewer items
    print(f"no-alloc call 2: {small.name} B={small.B} H={small.H} L={small.L} d={small.d}", flush=True)
    host = W.generate(small)
    _both(small, host, tuple(bf16_tensor(x) for x in host), seed=72, density=0.3)


def test_noalloc_rejects_plans_beyond_the_array():
    cfg = W.CONFIGS["tiny"]
    host = W.generate(cfg)
    qd, kd, vd = (bf16_tensor(x) for x in host)
    n = cfg.n
    idx = torch.zeros((cfg.B, cfg.H, n, n), dtype=torch.int32, device="cuda")
    cnt = torch.ones((cfg.B, cfg.H, n), dtype=torch.int32, device="cuda")
    o = torch.empty_like(qd)
    # 300 heads of 4096 blocks: a plan of 4 * (288 + 300 * 2059) bytes > 2 MiB
    big = M.make_shape(1, 300, 4096 * 128, 128, 128)
    assert M.mod_attn_workspace_bytes(big) > M.MOD_ATTN_NOALLOC_MAX_BYTES
    with pytest.raises(M.ModError) as e:
        M.mod_block_sparse_attn_fwd_noalloc(big, qd, kd, vd, idx, cnt, 0.0, o)
    assert e.value.status == M.MOD_ERR_UNSUPPORTED
    with pytest.raises(M.ModError) as e:
        M.mod_block_sparse_attn_fwd_noalloc(M.make_shape(cfg.B, cfg.H, cfg.L, cfg.d, cfg.block),
                                            qd, kd, vd, idx, cnt, 0.0, None)
    assert e.value.status == M.MOD_ERR_INVALID_ARG
