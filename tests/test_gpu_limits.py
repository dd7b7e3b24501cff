"""GPU parity at the size limits of the kernels, through the C ABI.

* The selection keeps a row's npad = 256 * E keys in registers (E keys per
  thread, E = 1, 2, 4, 8, 16 by n); the other parity tests reach E = 1
  (n <= 256) and E = 4 (the 720p layers).  Rows of n = 300, 1172 and 2063
  blocks (E = 2, 8, 16, each with a short tail block) are checked here
  against the oracle's predictor, whole layer, both budget modes.
* The attention handles n up to the ABI limit of 4096 blocks (the union
  list of two rows is held in LDS).  A layer of exactly 4096 blocks (short
  tail block) with rows that keep every block, long random lists, and short
  lists is checked on sampled query blocks: every full row, the first and
  the tail block, and a few others.
* The work plan keeps the counts of up to 16384 pairs in LDS; a layer of
  40 heads x 1024 blocks (20480 pairs) takes its path that reads them from
  memory.
"""
import math

import numpy as np
import pytest

import oracle as O
import workloads as W
from parity import LSE_ABS, MAX_ABS, MEAN_ABS, attention_errors, bf16_tensor, bf16_to_f64, gpu_lists

import paper_2601_11641_amd as M
from test_gpu_parity import _check_predictor, _run_predictor

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

MAX_BLOCKS = 4096   # largest n the ABI accepts


def _layer(name, H, frames, hs, ws, seed):
    return W.LayerConfig(name=name, B=1, H=H, d=64, frames=frames, hs=hs, ws=ws, block=64, seed=seed)


SELECT = {
    # 3 frames of 80x80: L = 19200, n = 300 (E = 2), no tail
    "n300": _layer("n300", 2, 3, 80, 80, 21),
    # 3 frames of 125x200: L = 75000, n = 1172 (E = 8), tail 56
    "n1172": _layer("n1172", 1, 3, 125, 200, 22),
    # 3 frames of 200x220: L = 132000, n = 2063 (E = 16), tail 32
    "n2063": _layer("n2063", 1, 3, 200, 220, 23),
}


@pytest.mark.parametrize("name", sorted(SELECT))
@pytest.mark.parametrize("budget", [("topk", 0.2), ("mass", 0.7)])
def test_select_register_widths(name, budget):
    cfg = SELECT[name]
    host = W.generate(cfg)
    dev = tuple(bf16_tensor(x) for x in host)
    params = dict(warmup_m=1, delta_t=0)
    st, kv_idx, kv_cnt, P, sel, qf, kf = _run_predictor(cfg, dev, host, [1], 2, budget, params)
    _check_predictor(cfg, st, kv_idx, kv_cnt, P, sel, qf, kf, budget, 2)
    st.close()


@pytest.mark.parametrize("budget", [("topk", 0.2), ("mass", 0.7)])
@pytest.mark.parametrize("tau_e", [-1.0, 1.0])
def test_select_tied_scores_work_group(budget, tau_e):
    """The one-work-group-per-row selection (n > 1024) on tied scores: every Q
    token and every K token the same vector, so a row's scores take one or
    two float32 values and the lists rest on the tie rule (ascending j), the
    frame blocks forced (tau_e below the zero frame energy) or not."""
    cfg = SELECT["n1172"]
    q, k, v = W.generate(cfg)
    q = np.ascontiguousarray(np.broadcast_to(q[:, :, :1, :], q.shape))
    k = np.ascontiguousarray(np.broadcast_to(k[:, :, :1, :], k.shape))
    host = (q, k, v)
    dev = tuple(bf16_tensor(x) for x in host)
    params = dict(warmup_m=1, delta_t=0, tau_e=tau_e)
    st, kv_idx, kv_cnt, P, sel, qf, kf = _run_predictor(cfg, dev, host, [1], 2, budget, params)
    assert P.gates.all() == (tau_e < 0) and P.gates.any() == (tau_e < 0)
    ct, dt_ = P.prediction(2)[0][0]
    keys = O.scores(ct, dt_, st.n).astype(np.float32)
    assert max(len(set(r.tolist())) for r in keys) <= 2      # the ties are there
    rows = gpu_lists(kv_idx, kv_cnt)
    for i in range(st.n):
        assert rows[0][0][i] == sel[0][0][i].kept.tolist(), i
    _check_predictor(cfg, st, kv_idx, kv_cnt, P, sel, qf, kf, budget, 2)
    st.close()


def _max_block_rows(n: int, H: int):
    """Per head: full rows every 97 blocks, 700-block random lists every 13,
    otherwise {i, its pair partner, 0, n-1, a head-dependent block}."""
    rows = []
    for h in range(H):
        rng = np.random.default_rng(500 + h)
        r = []
        for i in range(n):
            if i % 97 == 5:
                r.append(list(range(n)))
            elif i % 13 == 0:
                r.append(sorted(rng.choice(n, size=700, replace=False).tolist()))
            else:
                r.append(sorted({i, i ^ 1 if (i ^ 1) < n else i, 0, n - 1, (i * 37 + 11 * h) % n}))
        rows.append(r)
    return rows


def test_attention_at_max_blocks():
    # 2 frames of 50x2621: L = 262100, block 64: n = 4096, tail 20
    cfg = _layer("maxblocks", 2, 2, 50, 2621, 24)
    n = math.ceil(cfg.L / cfg.block)
    assert n == MAX_BLOCKS
    host = W.generate(cfg)
    qd, kd, vd = (bf16_tensor(x) for x in host)
    shape = M.make_shape(cfg.B, cfg.H, cfg.L, cfg.d, cfg.block, cfg.frame_tokens)
    assert M.mod_num_blocks(shape) == n
    rows = _max_block_rows(n, cfg.H)
    idx = torch.zeros((cfg.B, cfg.H, n, n), dtype=torch.int32)
    cnt = torch.zeros((cfg.B, cfg.H, n), dtype=torch.int32)
    for h in range(cfg.H):
        for i, js in enumerate(rows[h]):
            cnt[0, h, i] = len(js)
            idx[0, h, i, :len(js)] = torch.tensor(js, dtype=torch.int32)
    o = torch.empty_like(qd)
    lse = torch.empty((cfg.B, cfg.H, cfg.L), dtype=torch.float32, device="cuda")
    M.mod_block_sparse_attn_fwd(shape, qd, kd, vd, idx.cuda(), cnt.cuda(), 0.0, o, lse)
    torch.cuda.synchronize()
    og = bf16_to_f64(o)
    lg = lse.cpu().numpy().astype(np.float64)
    scale = 1.0 / math.sqrt(cfg.d)
    for h in range(cfg.H):
        full = [i for i in range(n) if i % 97 == 5]
        sample = sorted(set(full[::8]) | {0, 1, 13, 26, 2048, 2049, n - 2, n - 1})
        qf, kf, vf = (W.bf16_bits_to_f64(x[0, h]) for x in host)
        Oo, Lo = O.attention(qf, kf, vf, rows[h], cfg.block, scale, rows=sample)
        for i in sample:
            sl = slice(i * cfg.block, min(cfg.L, (i + 1) * cfg.block))
            mx, mean = attention_errors(og[0, h, sl], Oo[sl])
            assert mx <= MAX_ABS and mean <= MEAN_ABS, (h, i, mx, mean)
            assert np.abs(lg[0, h, sl] - Lo[sl]).max() <= LSE_ABS, (h, i)


def test_attention_plan_beyond_count_cache():
    """The work plan keeps both counts of up to 16384 pairs in LDS and reads
    them from memory beyond that; every other test stays below.  40 heads of
    1024 blocks (20480 pairs), each row a band of five blocks around the
    diagonal plus 0–40 seeded random blocks, heads of uneven cost (the
    random part grows with the head index), sampled query blocks of three
    heads against the oracle."""
    H, L, d, bs = 40, 65536, 64, 64
    n = L // bs
    assert H * ((n + 1) // 2) > 16384
    rng = np.random.default_rng(31)
    host = tuple(W.to_bf16_bits(rng.standard_normal((1, H, L, d)).astype(np.float32)) for _ in range(3))
    qd, kd, vd = (bf16_tensor(x) for x in host)
    shape = M.make_shape(1, H, L, d, bs, L)
    assert M.mod_num_blocks(shape) == n
    rows = []
    for h in range(H):
        rh = []
        for i in range(n):
            band = set(range(max(0, i - 2), min(n, i + 3)))
            extra = rng.integers(0, n, size=int(rng.integers(0, 1 + h)))
            rh.append(sorted(band | set(extra.tolist())))
        rows.append(rh)
    idx = np.zeros((1, H, n, n), np.int32)
    cnt = np.zeros((1, H, n), np.int32)
    for h in range(H):
        for i, js in enumerate(rows[h]):
            cnt[0, h, i] = len(js)
            idx[0, h, i, :len(js)] = js
    o = torch.empty_like(qd)
    lse = torch.empty((1, H, L), dtype=torch.float32, device="cuda")
    M.mod_block_sparse_attn_fwd(shape, qd, kd, vd, torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda(),
                                0.0, o, lse)
    torch.cuda.synchronize()
    og = bf16_to_f64(o)
    lg = lse.cpu().numpy().astype(np.float64)
    scale = 1.0 / math.sqrt(d)
    sample = [0, 1, 2, 255, 511, 512, 777, n - 2, n - 1]
    for h in (0, 17, H - 1):
        qf, kf, vf = (W.bf16_bits_to_f64(x[0, h]) for x in host)
        Oo, Lo = O.attention(qf, kf, vf, rows[h], bs, scale, rows=sample)
        for i in sample:
            sl = slice(i * bs, (i + 1) * bs)
            mx, mean = attention_errors(og[0, h, sl], Oo[sl])
            assert mx <= MAX_ABS and mean <= MEAN_ABS, (h, i, mx, mean)
            assert np.abs(lg[0, h, sl] - Lo[sl]).max() <= LSE_ABS, (h, i)
