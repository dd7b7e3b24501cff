"""Seeded synthetic attention-layer inputs for the MOD-DiT hot path.

This module is shared by the oracle-side tests, the GPU parity tests and the
benchmark, and it holds none of the method's arithmetic.  It only draws
Q, K, V tensors with the shapes, value distributions and spatiotemporal
structure of video-DiT attention layers and rounds them to bfloat16:

* tokens are laid out frame-first: token (f, y, x) sits at index
  f*Hs*Ws + y*Ws + x (the layout the paper assumes in Section 4.4);
* every token carries sinusoidal 3-D positional features: d/4 dimensions
  for the frame axis, 3d/8 for each spatial axis, as sin/cos pairs at
  geometric frequencies omega_{a,r} = omega_{a,0} * 0.7**r, scaled so the
  feature vector of every token has RMS ``kappa`` over its d entries;
* each head rotates the features by its own random orthogonal matrix
  R_h (QR of a Gaussian matrix) and mixes in Gaussian noise:
  Q = 0.7*phi*R_h + 0.3*N(0,1), K likewise with independent noise,
  V ~ N(0,1);
* heads come in three seeded types: temporal-local (fast frame-axis
  frequencies), spatial-local (fast spatial frequencies) and global
  (slow frequencies plus attention sinks: half the tokens of ~2% of the
  key blocks are pushed along a shared unit direction g that every query
  also leans towards, which produces vertical stripes).

Every random draw is made with numpy's PCG64 from a seed sequence keyed by
(seed, batch, head), so any single head can be regenerated on its own.
"""
from __future__ import annotations

import concurrent.futures
import math
import os
from dataclasses import dataclass, field

import numpy as np

HEAD_TEMPORAL = 0
HEAD_SPATIAL = 1
HEAD_GLOBAL = 2
HEAD_TYPE_NAMES = {HEAD_TEMPORAL: "temporal-local", HEAD_SPATIAL: "spatial-local",
                   HEAD_GLOBAL: "global"}

# Frequencies (radians per latent-grid step) of the first sin/cos pair per axis.
_OMEGA = {
    HEAD_TEMPORAL: (1.0, 0.05),
    HEAD_SPATIAL: (0.05, 1.0),
    HEAD_GLOBAL: (0.05, 0.05),
}
_DECAY = 0.7
_FEATURE_WEIGHT = 0.7
_NOISE_WEIGHT = 0.3
_SINK_BLOCK_FRACTION = 0.02
# Logit boost (in units of the softmax argument, i.e. after the 1/sqrt(d)
# scale) that an anchor key receives from every query.
_ANCHOR_LOGIT = 4.0

# Feature RMS.  Chosen once on the 8-frame 32x32 small layer so that, under
# dense attention, the top 25% of KV blocks of a query block hold at least
# 80% of its attention mass on average.
KAPPA = 3.0


@dataclass(frozen=True)
class LayerConfig:
    """Shape of one synthetic attention layer (one DiT attention call)."""
    name: str
    B: int
    H: int
    d: int
    frames: int
    hs: int
    ws: int
    block: int
    seed: int
    head_types: tuple = field(default=())   # empty: seeded 1/3 each
    text_tokens: int = 0                    # text segment appended after the video

    @property
    def frame_tokens(self) -> int:
        return self.hs * self.ws

    @property
    def L_video(self) -> int:
        return self.frames * self.frame_tokens

    @property
    def L(self) -> int:
        return self.L_video + self.text_tokens

    @property
    def n_video(self) -> int:
        return -(-self.L_video // self.block)

    @property
    def n(self) -> int:
        return -(-self.L // self.block)


CONFIGS = {
    # 4 frames x 16x16 latent grid, block 64: 16x16 block grid.
    "tiny": LayerConfig("tiny", B=1, H=2, d=64, frames=4, hs=16, ws=16, block=64, seed=1001),
    # 8 frames x 32x32, block 128: 64x64 block grid.
    "small": LayerConfig("small", B=1, H=8, d=128, frames=8, hs=32, ws=32, block=128,
                         seed=1002),
    # HunyuanVideo-shaped 720p layer: 33 latent frames x 45x80, L = 118,800.
    "hunyuan": LayerConfig("hunyuan", B=1, H=24, d=128, frames=33, hs=45, ws=80, block=128,
                           seed=1003),
    # Wan-style 720p layer: 21 latent frames x 45x80, L = 75,600.
    "wan": LayerConfig("wan", B=1, H=40, d=128, frames=21, hs=45, ws=80, block=128,
                       seed=1004),
}


def with_heads(cfg: LayerConfig, H: int, name: str | None = None) -> LayerConfig:
    """The layer's first H heads (each keeps its seed and type: the types of
    the whole layer are fixed explicitly, since the seeded draw depends on
    the head count)."""
    if not 1 <= H <= cfg.H:
        raise ValueError(f"with_heads keeps 1..{cfg.H} heads, got {H}")
    types = tuple(int(t) for t in head_types(cfg))
    return LayerConfig(name or cfg.name, cfg.B, H, cfg.d, cfg.frames, cfg.hs, cfg.ws,
                       cfg.block, cfg.seed, types, cfg.text_tokens)


def with_text(cfg: LayerConfig, text_tokens: int, name: str | None = None) -> LayerConfig:
    """The same layer with a text segment of `text_tokens` tokens appended
    after the video tokens (the video part is drawn identically)."""
    return LayerConfig(name or f"{cfg.name}+text{text_tokens}", cfg.B, cfg.H, cfg.d, cfg.frames,
                       cfg.hs, cfg.ws, cfg.block, cfg.seed, cfg.head_types, text_tokens)


# ----------------------------------------------------------------------------
# bfloat16 plumbing (round-to-nearest-even on the float32 bit pattern)
# ----------------------------------------------------------------------------

def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 array -> uint16 array of bfloat16 bit patterns (RNE)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(b).astype(np.float64)


# ----------------------------------------------------------------------------
# structure
# ----------------------------------------------------------------------------

def head_types(cfg: LayerConfig) -> np.ndarray:
    """Seeded head type per head: temporal / spatial / global, 1/3 each."""
    if cfg.head_types:
        return np.asarray(cfg.head_types[:cfg.H], dtype=np.int64)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, 7777])))
    base = np.arange(3 * (-(-cfg.H // 3))) % 3
    return rng.permutation(base)[:cfg.H].astype(np.int64)


def _axis_features(coord: np.ndarray, n_dims: int, omega0: float) -> np.ndarray:
    r = np.arange(n_dims // 2, dtype=np.float64)
    w = omega0 * _DECAY ** r
    ang = coord[:, None].astype(np.float64) * w[None, :]
    return np.concatenate([np.sin(ang), np.cos(ang)], axis=1)


def head_bandwidths(cfg: LayerConfig, b: int, h: int, htype: int):
    """(omega_t0, omega_s0) of one head: its type's base frequencies times a
    seeded per-head factor in [e^-0.5, e^0.5] (random locality bandwidth)."""
    rng = _head_rng(cfg.seed, b, h, tag=1)
    ft, fs = np.exp(rng.uniform(-0.5, 0.5, size=2))
    wt, wsp = _OMEGA[htype]
    return wt * ft, wsp * fs


def axis_features(cfg: LayerConfig, omega_t: float, omega_s: float, kappa: float = KAPPA):
    """Per-axis positional features (frame [F, d/4], row [Hs, 3d/8], column
    [Ws, 3d/8]) for the given base frequencies; the feature of token (f, y, x)
    is their concatenation, which has RMS ``kappa`` over its d entries."""
    d = cfg.d
    dt = d // 4
    ds = (d - dt) // 2
    # every sin/cos pair has squared norm 1, so sqrt(2)*kappa gives RMS kappa
    a = math.sqrt(2.0) * kappa
    return (a * _axis_features(np.arange(cfg.frames), dt, omega_t),
            a * _axis_features(np.arange(cfg.hs), ds, omega_s),
            a * _axis_features(np.arange(cfg.ws), ds, omega_s))


def positional_features(cfg: LayerConfig, omega_t: float, omega_s: float,
                        kappa: float = KAPPA) -> np.ndarray:
    """phi [L, d] float32 in frame-first token order."""
    ft, fy, fx = axis_features(cfg, omega_t, omega_s, kappa)
    dt, ds = ft.shape[1], fy.shape[1]
    phi = np.empty((cfg.frames, cfg.hs, cfg.ws, cfg.d), dtype=np.float64)
    phi[..., :dt] = ft[:, None, None, :]
    phi[..., dt:dt + ds] = fy[None, :, None, :]
    phi[..., dt + ds:] = fx[None, None, :, :]
    return phi.reshape(cfg.L, cfg.d).astype(np.float32)


def _head_rng(seed: int, b: int, h: int, tag: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, b, h, tag])))


def _draw_head(cfg: LayerConfig, b: int, h: int, htype: int, axes, seed: int | None = None):
    """float32 Q, K, V [L, d] of one head before bf16 rounding.  ``axes``:
    the per-axis features; phi R is formed as the sum of the three axis
    blocks times the matching rows of R (same product, fewer flops)."""
    rng = _head_rng(cfg.seed if seed is None else seed, b, h)
    d, L = cfg.d, cfg.L_video
    R, _ = np.linalg.qr(rng.standard_normal((d, d)))
    ft, fy, fx = axes
    dt, ds = ft.shape[1], fy.shape[1]
    w = _FEATURE_WEIGHT
    at = (w * ft @ R[:dt]).astype(np.float32)
    ay = (w * fy @ R[dt:dt + ds]).astype(np.float32)
    ax = (w * fx @ R[dt + ds:]).astype(np.float32)
    base = np.empty((cfg.frames, cfg.hs, cfg.ws, d), dtype=np.float32)
    np.add(at[:, None, None, :], ay[None, :, None, :], out=base)
    base += ax[None, None, :, :]
    base = base.reshape(L, d)
    q = base + np.float32(_NOISE_WEIGHT) * rng.standard_normal((L, d), dtype=np.float32)
    k = base + np.float32(_NOISE_WEIGHT) * rng.standard_normal((L, d), dtype=np.float32)
    v = rng.standard_normal((L, d), dtype=np.float32)
    if htype == HEAD_GLOBAL:
        # attention sinks: half the tokens of ~2% of the key blocks
        g = rng.standard_normal(d)
        g = (g / np.linalg.norm(g)).astype(np.float32)
        bs, n = cfg.block, cfg.n_video
        sinks = np.sort(rng.choice(n, size=max(1, int(round(_SINK_BLOCK_FRACTION * n))),
                                   replace=False))
        idx = []
        for j in sinks:
            lo, hi = j * bs, min(L, (j + 1) * bs)
            idx.append(lo + rng.choice(hi - lo, size=max(1, (hi - lo) // 2), replace=False))
        idx = np.sort(np.concatenate(idx))
        amp = math.sqrt(_ANCHOR_LOGIT * math.sqrt(d))   # alpha = beta, alpha*beta/sqrt(d) = boost
        q += np.float32(amp) * g[None, :]
        k[idx] += np.float32(amp) * g[None, :]
    if cfg.text_tokens:
        # text tokens: unstructured features at the video tokens' RMS, from a
        # stream of their own (the video part does not depend on them)
        trng = _head_rng(cfg.seed if seed is None else seed, b, h, tag=2)
        T = cfg.text_tokens
        rms = float(np.sqrt(np.mean(base * base) + _NOISE_WEIGHT ** 2))
        tq = rms * trng.standard_normal((T, d), dtype=np.float32)
        tk = rms * trng.standard_normal((T, d), dtype=np.float32)
        tv = trng.standard_normal((T, d), dtype=np.float32)
        q, k, v = (np.concatenate([a, t]) for a, t in ((q, tq), (k, tk), (v, tv)))
    return q, k, v


def generate_heads(cfg: LayerConfig, heads=None, batches=None, seed: int | None = None,
                   kappa: float = KAPPA):
    """bf16 bit patterns of Q, K, V for the selected (batch, head) pairs.

    Returns three uint16 arrays of shape [len(batches), len(heads), L, d].
    ``seed`` overrides the config seed (used for the second draw of the
    denoising-schedule drift).
    """
    heads = list(range(cfg.H)) if heads is None else list(heads)
    batches = list(range(cfg.B)) if batches is None else list(batches)
    types = head_types(cfg)
    shape = (len(batches), len(heads), cfg.L, cfg.d)
    out = [np.empty(shape, dtype=np.uint16) for _ in range(3)]

    def one(bi, b, hi, h):
        t = int(types[h])
        axes = axis_features(cfg, *head_bandwidths(cfg, b, h, t), kappa=kappa)
        q, k, v = _draw_head(cfg, b, h, t, axes, seed)
        out[0][bi, hi] = to_bf16_bits(q)
        out[1][bi, hi] = to_bf16_bits(k)
        out[2][bi, hi] = to_bf16_bits(v)

    jobs = [(bi, b, hi, h) for bi, b in enumerate(batches) for hi, h in enumerate(heads)]
    # heads draw from their own generators, so the result does not depend on
    # the number of worker threads
    workers = max(1, min(len(jobs), os.cpu_count() or 1, 16))
    if workers == 1:
        for j in jobs:
            one(*j)
    else:
        with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(lambda j: one(*j), jobs))
    return out[0], out[1], out[2]


def generate(cfg: LayerConfig, kappa: float = KAPPA):
    """bf16 bit patterns of the whole layer: Q, K, V uint16 [B, H, L, d]."""
    return generate_heads(cfg, kappa=kappa)


def drift_mix(bits0: np.ndarray, bits1: np.ndarray, step: int, total_steps: int) -> np.ndarray:
    """Smooth per-step drift between two draws of the same layer.

    X_t = cos(theta_t) X0 + sin(theta_t) X1, theta_t = (pi/2)(t-1)/(T-1),
    rounded back to bf16.
    """
    theta = 0.5 * math.pi * (step - 1) / max(1, total_steps - 1)
    x = math.cos(theta) * bf16_bits_to_f32(bits0) + math.sin(theta) * bf16_bits_to_f32(bits1)
    return to_bf16_bits(x.astype(np.float32))
