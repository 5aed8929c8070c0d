"""Seeded synthetic workloads for the action-guided sparse denoising step.

This module only draws inputs: model weights, per-step token activations with
planted, drifting action-relevant blobs, and the timestep embedding. It holds
none of the method's arithmetic (no scoring, selection, packing or block
computation), so the CPU oracle and the HIP path consume identical arrays
without sharing any code of the method.

Token layout of one sequence (the paper leaves the order open; this is the
reading adopted here): ``[context | future frames, frame-major, row-major inside
a frame | action tokens]``.  Sequences of a batch are concatenated row-wise.
A multi-view frame (several cameras of unequal resolution) is the views'
row-major token grids concatenated, so a frame has N_s = sum_v h_v w_v tokens
and is described to the step as one frame of 1 x N_s.

Every array is float32.  For bf16 configurations every value is already on the
bf16 grid (round-to-nearest-even), so converting to ``torch.bfloat16`` is exact.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "SwamConfig", "preset", "PRESETS", "budgets", "rng_for", "block_weights",
    "timestep_embedding", "StepInputs", "make_inputs", "blob_direction",
    "time_embedding", "latent_io_weights", "SamplerInputs", "make_sampler_inputs", "view_grids",
]


# ---------------------------------------------------------------------------
# configuration
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class SwamConfig:
    """Shape and policy of one workload.

    ``k_core``/``k_anchor`` are the per-frame budgets K_c / K_s of the paper's
    selection rule (Sec. 4.1); ``mass_threshold`` > 0 replaces the fixed K_c by
    a per-frame count from a score-mass threshold (an extension used by the
    ragged batched workload).
    """
    name: str
    batch: int
    d_model: int
    n_heads: int
    n_blocks: int
    n_ctx: int
    n_frames: int
    frame_h: int
    frame_w: int
    n_act: int
    k_core: int
    k_anchor: int
    reuse_R: int
    n_steps: int
    dtype: str                  # "f32" or "bf16"
    seed: int
    blob_sigma: float = 3.0     # fixed blob width (tokens) for single-blob workloads
    blob_count: tuple = (1, 1)  # inclusive range of blobs per sequence
    blob_sigma_range: tuple | None = None  # (lo, hi): sigma ~ U[lo, hi] per blob
    action_dof: int = 0         # > 0: actions are DoF vectors embedded to d
    head_dim: int = 64
    mlp_ratio: int = 4
    d_temb: int = 128
    k_layer: int = 6
    cv_penalty: float = 1.0
    mass_threshold: float = 0.0
    retain_percent: int = 0     # informational: per-frame core percent
    rope: int = 0               # backbone variant: rotary embedding at original positions
    qk_norm: int = 0            # backbone variant: RMS-normalised q and k per head
    cfg_pairs: int = 0          # guidance: sequences [P, 2P) are the unconditional partners of [0, P)
    guidance: float = 1.0       # guidance scale g of the sampler (with cfg_pairs)
    views: tuple = ()           # multi-view frames: ((h, w), ...) per camera; frame is 1 x sum(h w)

    # derived sizes ----------------------------------------------------------
    @property
    def n_s(self) -> int:
        return self.frame_h * self.frame_w

    @property
    def n_fut(self) -> int:
        return self.n_frames * self.n_s

    @property
    def l_full(self) -> int:
        return self.n_ctx + self.n_fut + self.n_act

    @property
    def g(self) -> int:
        return self.n_act // self.n_frames

    @property
    def k_ret(self) -> int:
        return self.k_core + self.k_anchor

    @property
    def n_scored(self) -> int:
        """Sequences that are scored and selected: the conditional half with
        guidance pairs, else every sequence."""
        return self.batch // 2 if self.cfg_pairs else self.batch

    @property
    def t_pack_fixed(self) -> int:
        """Packed length of one sequence in fixed-budget mode."""
        return self.n_ctx + self.n_frames * self.k_ret + self.n_act

    def replace(self, **kw) -> "SwamConfig":
        return dataclasses.replace(self, **kw)


def budgets(n_s: int, percent: int, n_anchor: int) -> tuple[int, int]:
    """Per-frame budgets from "retain p% per frame plus top-N positions".

    K_c = round-half-up(p * N_s / 100); K_s = N clamped to N_s - K_c, so that a
    100% retention keeps every position as a core token and no anchors.
    """
    k_c = (percent * n_s + 50) // 100
    k_s = min(n_anchor, n_s - k_c)
    return k_c, k_s


def _cfg1() -> SwamConfig:
    k_c, k_s = budgets(64, 25, 4)
    return SwamConfig(name="tiny-fp32-1blk-d128", batch=1, d_model=128, n_heads=2,
                      n_blocks=1, n_ctx=16, n_frames=2, frame_h=8, frame_w=8, n_act=8,
                      k_core=k_c, k_anchor=k_s, reuse_R=2, n_steps=4, dtype="f32",
                      seed=0, blob_sigma=1.5, retain_percent=25)


def _cfg2() -> SwamConfig:
    k_c, k_s = budgets(256, 30, 16)
    return SwamConfig(name="bf16-8blk-d1024", batch=1, d_model=1024, n_heads=16,
                      n_blocks=8, n_ctx=256, n_frames=4, frame_h=16, frame_w=16, n_act=32,
                      k_core=k_c, k_anchor=k_s, reuse_R=2, n_steps=10, dtype="bf16",
                      seed=1, blob_sigma=3.0, retain_percent=30)


def _cfg3() -> SwamConfig:
    k_c, k_s = budgets(1200, 25, 64)
    return SwamConfig(name="bf16-28blk-d1536-wam", batch=1, d_model=1536, n_heads=24,
                      n_blocks=28, n_ctx=512, n_frames=8, frame_h=30, frame_w=40, n_act=48,
                      k_core=k_c, k_anchor=k_s, reuse_R=2, n_steps=10, dtype="bf16",
                      seed=2, blob_sigma=3.0, action_dof=7, retain_percent=25)


def _cfg4(percent: int = 25, reuse_R: int = 2) -> SwamConfig:
    k_c, k_s = budgets(1024, percent, 64)
    return SwamConfig(name=f"bf16-28blk-d2048-r{percent}-R{reuse_R}", batch=1,
                      d_model=2048, n_heads=32, n_blocks=28, n_ctx=1024, n_frames=16,
                      frame_h=32, frame_w=32, n_act=64, k_core=k_c, k_anchor=k_s,
                      reuse_R=reuse_R, n_steps=16, dtype="bf16", seed=3, blob_sigma=3.0,
                      retain_percent=percent)


def _cfg5() -> SwamConfig:
    n_s = 24 * 32
    return SwamConfig(name="bf16-ragged-b8-12blk-d1536", batch=8, d_model=1536,
                      n_heads=24, n_blocks=12, n_ctx=256, n_frames=4, frame_h=24,
                      frame_w=32, n_act=32, k_core=n_s, k_anchor=0, reuse_R=2,
                      n_steps=10, dtype="bf16", seed=4, blob_count=(1, 4),
                      blob_sigma_range=(2.0, 6.0), mass_threshold=0.8)


def _cfg6() -> SwamConfig:
    # three cameras (one wrist view and two smaller third-person views) of
    # 340 tokens per future frame, 8 future frames, 4 denoising steps with one
    # full step per chunk, K_c + K_s = 80 + 104, guidance pairs at scale 3.0,
    # 28 blocks (the shape of the paper's 28-layer backbone, App. B.2 table)
    views = ((14, 14), (8, 9), (8, 9))
    n_s = sum(h * w for h, w in views)
    return SwamConfig(name="bf16-28blk-d1536-3view-340tok-cfg3", batch=2, d_model=1536,
                      n_heads=24, n_blocks=28, n_ctx=n_s, n_frames=8, frame_h=1, frame_w=n_s,
                      n_act=32, k_core=80, k_anchor=104, reuse_R=4, n_steps=4, dtype="bf16",
                      seed=6, blob_count=(1, 3), blob_sigma_range=(1.5, 3.0), views=views,
                      cfg_pairs=1, guidance=3.0)


def _cfg7() -> SwamConfig:
    # two cameras of 98 tokens per future frame in total, 2 future frames,
    # 16 aligned action queries per frame, 10 steps with one full step,
    # K_c + K_s = 19 + 12, no guidance, 30 blocks (App. B.2 table)
    views = ((7, 7), (7, 7))
    n_s = sum(h * w for h, w in views)
    return SwamConfig(name="bf16-30blk-d1536-2view-98tok", batch=1, d_model=1536,
                      n_heads=24, n_blocks=30, n_ctx=n_s, n_frames=2, frame_h=1, frame_w=n_s,
                      n_act=32, k_core=19, k_anchor=12, reuse_R=10, n_steps=10, dtype="bf16",
                      seed=7, blob_count=(1, 2), blob_sigma_range=(1.0, 2.0), views=views)


PRESETS = {1: _cfg1, 2: _cfg2, 3: _cfg3, 4: _cfg4, 5: _cfg5, 6: _cfg6, 7: _cfg7}


def preset(n: int, **kw) -> SwamConfig:
    """Named workload ``n`` (1..7); config 4 takes ``percent`` and ``reuse_R``.
    6 and 7 are multi-view workloads at the shapes of the paper's backbone
    table (App. B.2)."""
    if n == 4:
        return _cfg4(**kw)
    cfg = PRESETS[n]()
    return cfg.replace(**kw) if kw else cfg


# ---------------------------------------------------------------------------
# random streams
# ---------------------------------------------------------------------------
_STREAM_WEIGHTS = 1
_STREAM_BASE = 2
_STREAM_ACTION = 3
_STREAM_BLOB = 4


def rng_for(cfg: SwamConfig, *stream: int) -> np.random.Generator:
    """Independent PCG64 stream keyed by (seed, stream ids...)."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, *stream])))


def _to_bf16_grid(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 value (ties to even), on a copy.

    In uint32 arithmetic: for every finite float32 the bit pattern plus
    0x7FFF + 1 stays below 2^32, so nothing wraps."""
    x = np.array(x, dtype=np.float32, order="C")
    u = x.view(np.uint32)
    lsb = (u >> 16) & np.uint32(1)
    u += np.uint32(0x7FFF)
    u += lsb
    u &= np.uint32(0xFFFF0000)
    return x


def _storage(cfg: SwamConfig, x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float32)
    return _to_bf16_grid(x) if cfg.dtype == "bf16" else np.ascontiguousarray(x)


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(std)


def block_weights(cfg: SwamConfig, layer: int) -> dict:
    """Weights of block ``layer``; each matrix is [out_features][in_features].

    Entries are N(0, 1/fan_in) (fan_in = d for d-input layers, 4d for the MLP
    down projection, d_temb for the adaLN projection); biases use the same
    standard deviation as their matrix.
    """
    d, dt, hidden = cfg.d_model, cfg.d_temb, cfg.mlp_ratio * cfg.d_model
    rng = rng_for(cfg, _STREAM_WEIGHTS, layer)
    sd, sdt, sdh = 1.0 / math.sqrt(d), 1.0 / math.sqrt(dt), 1.0 / math.sqrt(hidden)
    w = {}
    w["w_ada"] = _normal(rng, (6 * d, dt), sdt)
    w["b_ada"] = _normal(rng, (6 * d,), sdt)
    w["w_qkv"] = _normal(rng, (3 * d, d), sd)
    w["b_qkv"] = _normal(rng, (3 * d,), sd)
    w["w_o"] = _normal(rng, (d, d), sd)
    w["b_o"] = _normal(rng, (d,), sd)
    w["w_1"] = _normal(rng, (hidden, d), sd)
    w["b_1"] = _normal(rng, (hidden,), sd)
    w["w_2"] = _normal(rng, (d, hidden), sdh)
    w["b_2"] = _normal(rng, (d,), sdh)
    return {k: _storage(cfg, v) for k, v in w.items()}


def time_embedding(cfg: SwamConfig, t: float) -> np.ndarray:
    """Sinusoidal embedding of a model time t, layout [cos | sin]."""
    half = cfg.d_temb // 2
    freqs = np.exp(-math.log(10000.0) * np.arange(half, dtype=np.float64) / half)
    arg = float(t) * freqs
    return np.concatenate([np.cos(arg), np.sin(arg)]).astype(np.float32)


def timestep_embedding(cfg: SwamConfig, tau: int) -> np.ndarray:
    """Sinusoidal embedding of t = 1000 (N - tau) / N, layout [cos | sin]."""
    t = 1000.0 * (cfg.n_steps - tau) / cfg.n_steps
    half = cfg.d_temb // 2
    freqs = np.exp(-math.log(10000.0) * np.arange(half, dtype=np.float64) / half)
    arg = t * freqs
    return np.concatenate([np.cos(arg), np.sin(arg)]).astype(np.float32)


# ---------------------------------------------------------------------------
# activations with planted drifting blobs
# ---------------------------------------------------------------------------
@dataclass
class _Blob:
    sigma: float
    centers: np.ndarray   # [F][2] (row, col) at tau = 0
    dirs: np.ndarray      # [F][2] unit grid step per denoising step
    view: int = -1        # multi-view frames: the camera the blob lives in


@dataclass
class StepInputs:
    """Per-sequence base tokens and blob parameters; ``x(tau)`` draws nothing."""
    cfg: SwamConfig
    base: list = field(default_factory=list)      # per sequence: [L_full][d] float32
    blobs: list = field(default_factory=list)     # per sequence: list[_Blob]
    direction: list = field(default_factory=list)  # per sequence: [F][d] float32 (rows of norm sqrt(d))

    def x(self, tau: int) -> np.ndarray:
        """x_full at step tau, [B * L_full][d] float32 on the storage grid."""
        cfg = self.cfg
        out = []
        for b in range(cfg.batch):
            xb = self.base[b].copy()
            w = _blob_weights(cfg, self.blobs[b], tau)           # [F][N_s]
            fut = xb[cfg.n_ctx:cfg.n_ctx + cfg.n_fut].reshape(cfg.n_frames, cfg.n_s, cfg.d_model)
            fut += 0.5 * w[:, :, None].astype(np.float32) * self.direction[b][:, None, :]
            out.append(xb)
        return _storage(cfg, np.concatenate(out, axis=0))

    def temb(self, tau: int) -> np.ndarray:
        return timestep_embedding(self.cfg, tau)


def view_grids(cfg: SwamConfig):
    """(offset in the frame, h, w) of every camera view; one view of
    frame_h x frame_w for single-view workloads."""
    if not cfg.views:
        return [(0, cfg.frame_h, cfg.frame_w)]
    out, off = [], 0
    for h, w in cfg.views:
        out.append((off, h, w))
        off += h * w
    return out


def _blob_weights(cfg: SwamConfig, blobs, tau: int) -> np.ndarray:
    """Sum over blobs of exp(-dist^2 / (2 sigma^2)) on the torus of the blob's
    view, [F][N_s]."""
    if cfg.views:
        acc = np.zeros((cfg.n_frames, cfg.n_s))
        grids = view_grids(cfg)
        for bl in blobs:
            off, hh, ww = grids[bl.view]
            sub = cfg.replace(frame_h=hh, frame_w=ww, views=())
            acc[:, off:off + hh * ww] += _blob_weights(sub, [dataclasses.replace(bl, view=-1)], tau)
        return acc
    hh, ww = cfg.frame_h, cfg.frame_w
    rows = np.arange(hh)[:, None].astype(np.float64)
    cols = np.arange(ww)[None, :].astype(np.float64)
    acc = np.zeros((cfg.n_frames, hh, ww))
    for bl in blobs:
        for f in range(cfg.n_frames):
            cr = (bl.centers[f, 0] + tau * bl.dirs[f, 0]) % hh
            cc = (bl.centers[f, 1] + tau * bl.dirs[f, 1]) % ww
            dr = np.abs(rows - cr)
            dr = np.minimum(dr, hh - dr)
            dc = np.abs(cols - cc)
            dc = np.minimum(dc, ww - dc)
            acc[f] += np.exp(-(dr ** 2 + dc ** 2) / (2.0 * bl.sigma ** 2))
    return acc.reshape(cfg.n_frames, cfg.n_s)


def blob_direction(cfg: SwamConfig, w_qkv0: np.ndarray, act_tokens: np.ndarray) -> np.ndarray:
    """Token-space direction, per future frame, that raises the logits of the
    frame's own action queries, [F][d].

    Frame f is scored by its group of g = H / F action queries (rows
    f*g .. f*g + g - 1 of the action block).  The mean action token of that
    group is mapped to query space by block 0's query projection and back to
    token space by the transpose of its key projection, then scaled to the
    typical token norm sqrt(d).
    """
    d = cfg.d_model
    g = cfg.n_act // cfg.n_frames
    w_q = w_qkv0[0:d].astype(np.float64)
    w_k = w_qkv0[d:2 * d].astype(np.float64)
    out = np.empty((cfg.n_frames, d), np.float32)
    for f in range(cfg.n_frames):
        a_mean = act_tokens[f * g:(f + 1) * g].astype(np.float64).mean(axis=0)
        u = w_k.T @ (w_q @ a_mean)
        out[f] = u * (math.sqrt(d) / np.linalg.norm(u))
    return out


def make_inputs(cfg: SwamConfig, w_qkv0: np.ndarray | None = None) -> StepInputs:
    """Draw base tokens and blobs for every sequence of the batch.

    ``w_qkv0`` is block 0's QKV matrix (drawn if not given).
    """
    if w_qkv0 is None:
        w_qkv0 = block_weights(cfg, 0)["w_qkv"]
    d = cfg.d_model
    inp = StepInputs(cfg=cfg)
    for b in range(cfg.batch):
        rng = rng_for(cfg, _STREAM_BASE, b)
        ctx = rng.standard_normal((cfg.n_ctx, d), dtype=np.float32)
        fut = rng.standard_normal((cfg.n_fut, d), dtype=np.float32)
        if cfg.action_dof > 0:
            ra = rng_for(cfg, _STREAM_ACTION, b)
            w_emb = _normal(ra, (d, cfg.action_dof), 1.0 / math.sqrt(cfg.action_dof))
            dof = ra.standard_normal((cfg.n_act, cfg.action_dof), dtype=np.float32)
            act = dof @ w_emb.T
        else:
            act = rng.standard_normal((cfg.n_act, d), dtype=np.float32)
        inp.base.append(np.concatenate([ctx, fut, act], axis=0).astype(np.float32))
        rb = rng_for(cfg, _STREAM_BLOB, b)
        lo, hi = cfg.blob_count
        nb = int(rb.integers(lo, hi + 1))
        blobs = []
        steps = np.array([[1, 0], [-1, 0], [0, 1], [0, -1]], dtype=np.float64)
        for _ in range(nb):
            if cfg.blob_sigma_range is not None:
                sigma = float(rb.uniform(*cfg.blob_sigma_range))
            else:
                sigma = float(cfg.blob_sigma)
            view, hh, ww = -1, cfg.frame_h, cfg.frame_w
            if cfg.views:
                view = int(rb.integers(0, len(cfg.views)))
                hh, ww = cfg.views[view]
            centers = np.stack([rb.integers(0, hh, cfg.n_frames),
                                rb.integers(0, ww, cfg.n_frames)], axis=1).astype(np.float64)
            dirs = steps[rb.integers(0, 4, cfg.n_frames)]
            blobs.append(_Blob(sigma=sigma, centers=centers, dirs=dirs, view=view))
        inp.blobs.append(blobs)
        inp.direction.append(blob_direction(cfg, w_qkv0, act))
    return inp


# ---------------------------------------------------------------------------
# closed-loop sampling: latent embedding / velocity read-out and initial noise
# ---------------------------------------------------------------------------
_STREAM_LATENT_W = 5
_STREAM_LATENT_Z = 6


def latent_io_weights(cfg: SwamConfig, d_latent: int = 16) -> dict:
    """Latent embedding w_in [d][c], b_in [d] (std 1/sqrt(c), so unit-variance
    latents give unit-variance tokens) and velocity head w_v [c][d], b_v [c]
    (std 1/sqrt(d)), on the storage grid of the configuration."""
    d, c = cfg.d_model, d_latent
    rng = rng_for(cfg, _STREAM_LATENT_W)
    w = {"w_in": _normal(rng, (d, c), 1.0 / math.sqrt(c)),
         "b_in": _normal(rng, (d,), 1.0 / math.sqrt(c)),
         "w_v": _normal(rng, (c, d), 1.0 / math.sqrt(d)),
         "b_v": _normal(rng, (c,), 1.0 / math.sqrt(d))}
    return {k: _storage(cfg, v) for k, v in w.items()}


@dataclass
class SamplerInputs:
    """Context tokens per sequence ([B][n_ctx][d], storage grid) and the
    initial latent noise z0 ([B * (F*N_s + H)][c] float32, future then action
    tokens of each sequence)."""
    ctx: np.ndarray
    z0: np.ndarray


def make_sampler_inputs(cfg: SwamConfig, d_latent: int = 16) -> SamplerInputs:
    base = make_inputs(cfg)
    ctx = np.stack([b[:cfg.n_ctx] for b in base.base]).astype(np.float32)
    rng = rng_for(cfg, _STREAM_LATENT_Z)
    # one latent state per pair with guidance (both branches denoise the same z)
    z0 = rng.standard_normal((cfg.n_scored * (cfg.l_full - cfg.n_ctx), d_latent), dtype=np.float32)
    return SamplerInputs(ctx=_storage(cfg, ctx), z0=z0)
