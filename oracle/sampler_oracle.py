"""Plain CPU oracle of the sampling update around the sparse step.

TEST INFRASTRUCTURE ONLY: imported by the test suite and the benchmark's
CPU-baseline leg, never by the product path; shares no code with the HIP path.

What it computes (Sparse-WAM, Sec. 4.2 "sampling updates for omitted
regions", and App. B.2 for the schedule shift), in float64 with the same
storage points as the GPU path:

* the latent tokens (future frames, then actions) enter the network through a
  linear embedding, x = z W_in^T + b_in (the context tokens are conditioning
  and stay as given);
* the network output of a latent token is read out by a velocity head,
  v = LN(y) W_v^T + b_v (LayerNorm without affine, eps 1e-6);
* a full step caches the visual (future-token) velocity; a sparse step uses
  the current velocity at retained future positions and the cached one
  elsewhere, M * v(tau) + (1 - M) * v(tau_d) (the paper's merge equation);
  action velocities are always the current ones;
* the sampler is the flow-matching Euler step z <- z + (sigma_next - sigma) v
  over a shifted schedule sigma(s) = shift s / (1 + (shift - 1) s), s = 1 - i/N,
  shift 5.0 (App. B.2), with the model time t = 1000 sigma;
* with classifier-free guidance (scale g, App. B.2) the batch holds P
  conditional sequences and their P unconditional partners, both branches
  denoise one latent state per pair, the guided velocity is
  v = v_u + g (v_c - v_u), and that guided velocity is what a full step
  caches and a sparse step merges; the selection comes from the conditional
  branch and the partner reuses it.

The linear embedding / head, the LayerNorm in the head and the Euler
integrator are readings (the paper names the merge, the shift and that the
original sampler updates every latent); they are listed in the design notes.
Pins: tests/test_oracle_sampler.py.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .swam_oracle import (round_f32, storage_round, layer_norm, is_refresh, refresh_step,
                          sparse_step, dense_step, n_scored)

SCHEDULE_SHIFT = 5.0     # App. B.2: noise schedule shift of every backbone


def sigmas(n_steps: int, shift: float = SCHEDULE_SHIFT) -> np.ndarray:
    """sigma_i for i = 0..N: the shifted flow schedule, from 1 (noise) to 0."""
    s = 1.0 - np.arange(n_steps + 1, dtype=np.float64) / n_steps
    return shift * s / (1.0 + (shift - 1.0) * s)


def latent_rows(cfg) -> np.ndarray:
    """Full-layout rows of the latent tokens (future frames, then actions) of
    every sequence, in latent order [B][F*N_s + H]."""
    per = np.arange(cfg.n_ctx, cfg.l_full)
    return (np.arange(cfg.batch)[:, None] * cfg.l_full + per[None, :]).reshape(-1)


def embed(z, w_in, b_in, dtype):
    """Tokens of latent rows: z [n][c] -> x [n][d], stored in the config dtype."""
    z = np.asarray(z, np.float64)
    return storage_round(dtype)(z @ np.asarray(w_in, np.float64).T + np.asarray(b_in, np.float64))


def velocity(y, w_v, b_v):
    """Velocity read-out of output tokens y [n][d] -> v [n][c] (float32 values)."""
    h = layer_norm(np.asarray(y, np.float64))
    return round_f32(h @ np.asarray(w_v, np.float64).T + np.asarray(b_v, np.float64))


def merge_velocity(v_cur, v_cached, keep):
    """The paper's merge: current prediction where the position was retained,
    the cached full-step prediction elsewhere (keep: bool per row)."""
    keep = np.asarray(keep, bool)
    return np.where(keep[:, None], np.asarray(v_cur, np.float64), np.asarray(v_cached, np.float64))


def guided_velocity(v_cond, v_uncond, g):
    """Classifier-free guidance of two branch velocities: v_u + g (v_c - v_u)."""
    vc = np.asarray(v_cond, np.float64)
    vu = np.asarray(v_uncond, np.float64)
    return vu + float(g) * (vc - vu)


def euler_update(z, v, dsigma):
    """One flow-matching Euler step of the float32 latent state."""
    return round_f32(np.asarray(z, np.float64) + float(dsigma) * np.asarray(v, np.float64))


@dataclass
class SamplerTrace:
    z: list          # latent state after each step, [B*L_lat][c]
    kinds: list      # 1 = refresh (full step), 2 = sparse
    v_tilde: list    # merged velocity used at each step
    x: list          # network input of each step (full layout)


def run_sampler(cfg, model, io, ctx_tokens, z0, temb_of_t, n_steps=None,
                shift=SCHEDULE_SHIFT, dense=False):
    """Closed-loop sampling: at every step the latent rows of the network input
    are re-embedded from z; refresh steps (tau mod R == 0) run the dense step
    with scoring and selection and cache the visual velocity, sparse steps run
    the packed blocks and merge.  ``dense=True`` runs every step dense (the
    reference the sparse sampler approximates).

    io: dict w_in [d][c], b_in [d], w_v [c][d], b_v [c];
    ctx_tokens: [B][n_ctx][d]; z0: [P*L_lat][c] (P = B, or B/2 with guidance
    pairs); temb_of_t(t) -> [d_temb]."""
    n = cfg.n_steps if n_steps is None else n_steps
    sig = sigmas(n, shift)
    rows = latent_rows(cfg)
    L_lat = cfg.l_full - cfg.n_ctx
    P = n_scored(cfg)
    pairs = P != cfg.batch
    g = float(getattr(cfg, "guidance", 1.0))
    fut = np.tile(np.arange(L_lat) < cfg.n_fut, P)
    cond_rows = rows[:P * L_lat]

    def branch_velocity(v_all):
        # per-sequence read-outs [B*L_lat][c] -> the velocity of each latent state
        if not pairs:
            return v_all
        return guided_velocity(v_all[:P * L_lat], v_all[P * L_lat:], g)

    x = np.zeros((cfg.batch * cfg.l_full, cfg.d_model))
    for b in range(cfg.batch):
        x[b * cfg.l_full:b * cfg.l_full + cfg.n_ctx] = ctx_tokens[b]
    z = np.asarray(z0, np.float64)
    v_cache = np.zeros_like(z)
    pm = None
    tr = SamplerTrace(z=[], kinds=[], v_tilde=[], x=[])
    for tau in range(n):
        x = x.copy()
        z_rows = np.concatenate([z, z]) if pairs else z
        x[rows] = embed(z_rows, io["w_in"], io["b_in"], cfg.dtype)
        temb = temb_of_t(1000.0 * sig[tau])
        if dense:
            y = dense_step(x, model, temb, cfg)
            v_t = branch_velocity(velocity(y[rows], io["w_v"], io["b_v"]))
            kind = 0
        elif is_refresh(tau, cfg.reuse_R):
            r = refresh_step(x, model, temb, cfg)
            pm = r.packmap
            v_t = branch_velocity(velocity(r.y[rows], io["w_v"], io["b_v"]))
            v_cache = np.where(fut[:, None], v_t, v_cache)
            kind = 1
        else:
            y = sparse_step(x, model, temb, cfg, pm)
            v_cur = branch_velocity(velocity(y[rows], io["w_v"], io["b_v"]))
            keep = (pm.pack_pos[cond_rows] >= 0) | ~fut
            v_t = merge_velocity(v_cur, v_cache, keep)
            kind = 2
        z = euler_update(z, v_t, sig[tau + 1] - sig[tau])
        tr.z.append(z)
        tr.kinds.append(kind)
        tr.v_tilde.append(v_t)
        tr.x.append(x)
    return tr
