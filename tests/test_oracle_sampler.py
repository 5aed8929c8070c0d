"""Pins of the sampling-update oracle (Sec. 4.2 merge; App. B.2 shift) against
closed forms, textbook routines and invariants -- CPU only."""
import dataclasses

import numpy as np
import pytest
import torch

import workload as W
from oracle import sampler_oracle as SO
from oracle import swam_oracle as O


def test_sigmas_closed_form_n4():
    # s = 1, 3/4, 1/2, 1/4, 0 and sigma = 5s / (1 + 4s)
    want = [1.0, 3.75 / 4.0, 5.0 / 6.0, 1.25 / 2.0, 0.0]
    np.testing.assert_allclose(SO.sigmas(4), want, rtol=0, atol=1e-15)


def test_sigmas_shift_one_is_linear_and_odds_scale_with_shift():
    np.testing.assert_allclose(SO.sigmas(10, shift=1.0), 1.0 - np.arange(11) / 10.0, atol=1e-15)
    s = 1.0 - np.arange(1, 10) / 10.0
    sig = SO.sigmas(10, shift=5.0)[1:10]
    # the shift multiplies the noise-to-signal odds: sigma / (1 - sigma) = 5 s / (1 - s)
    np.testing.assert_allclose(sig / (1 - sig), 5.0 * s / (1 - s), rtol=1e-12)
    assert np.all(np.diff(SO.sigmas(10)) < 0)


def test_euler_integrates_the_straight_flow_exactly():
    # z(sigma) = x0 + sigma (eps - x0) has the constant velocity eps - x0; the
    # Euler steps over any schedule from sigma 1 to 0 land on x0
    rng = np.random.default_rng(0)
    x0 = rng.standard_normal((50, 16)).astype(np.float32)
    eps = rng.standard_normal((50, 16)).astype(np.float32)
    v = eps.astype(np.float64) - x0
    z = eps.astype(np.float64)
    sig = SO.sigmas(7)
    for i in range(7):
        z = SO.euler_update(z, v, sig[i + 1] - sig[i])
    np.testing.assert_allclose(z, x0, atol=2e-6)


def test_merge_selects_current_or_cached_rowwise():
    rng = np.random.default_rng(1)
    cur, cache = rng.standard_normal((9, 4)), rng.standard_normal((9, 4))
    np.testing.assert_array_equal(SO.merge_velocity(cur, cache, np.ones(9, bool)), cur)
    np.testing.assert_array_equal(SO.merge_velocity(cur, cache, np.zeros(9, bool)), cache)
    keep = rng.random(9) < 0.5
    out = SO.merge_velocity(cur, cache, keep)
    for r in range(9):
        np.testing.assert_array_equal(out[r], cur[r] if keep[r] else cache[r])


def test_velocity_head_matches_torch_layernorm_linear():
    rng = np.random.default_rng(2)
    y = rng.standard_normal((13, 96))
    w = rng.standard_normal((8, 96)) / 10
    b = rng.standard_normal(8)
    t = torch.nn.functional.linear(
        torch.nn.functional.layer_norm(torch.from_numpy(y), (96,), eps=1e-6),
        torch.from_numpy(w), torch.from_numpy(b)).numpy()
    np.testing.assert_allclose(SO.velocity(y, w, b), O.round_f32(t), rtol=0, atol=1e-6)


def test_embedding_matches_torch_linear_on_the_storage_grid():
    rng = np.random.default_rng(3)
    z = rng.standard_normal((11, 16)).astype(np.float32)
    w = rng.standard_normal((64, 16)).astype(np.float32) / 4
    b = rng.standard_normal(64).astype(np.float32)
    t = torch.nn.functional.linear(torch.from_numpy(z).double(), torch.from_numpy(w).double(),
                                   torch.from_numpy(b).double()).numpy()
    np.testing.assert_array_equal(SO.embed(z, w, b, "bf16"), O.round_bf16(t))
    np.testing.assert_array_equal(SO.embed(z, w, b, "f32"), O.round_f32(t))


def test_latent_rows_are_future_then_action_rows():
    cfg = W.preset(5)
    rows = SO.latent_rows(cfg).reshape(cfg.batch, -1)
    for b in range(cfg.batch):
        np.testing.assert_array_equal(rows[b], np.arange(b * cfg.l_full + cfg.n_ctx, (b + 1) * cfg.l_full))


def _sampler_case(cfg, n_steps=4):
    model = [W.block_weights(cfg, l) for l in range(cfg.n_blocks)]
    io = W.latent_io_weights(cfg)
    si = W.make_sampler_inputs(cfg)
    temb = lambda t: W.time_embedding(cfg, t)  # noqa: E731
    return model, io, si, temb, n_steps


def test_full_retention_sampler_equals_dense_sampler():
    cfg = dataclasses.replace(W.preset(1), k_core=64, k_anchor=0)
    model, io, si, temb, n = _sampler_case(cfg)
    sp = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, n)
    de = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, n, dense=True)
    assert sp.kinds == [1, 2, 1, 2]
    for a, b in zip(sp.z, de.z):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_refresh_every_step_equals_dense_sampler():
    cfg = dataclasses.replace(W.preset(1), reuse_R=1)
    model, io, si, temb, n = _sampler_case(cfg)
    sp = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, n)
    de = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, n, dense=True)
    assert sp.kinds == [1, 1, 1, 1]
    for a, b in zip(sp.z, de.z):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_sparse_step_uses_cache_at_pruned_and_current_elsewhere():
    cfg = W.preset(1)
    model, io, si, temb, n = _sampler_case(cfg)
    tr = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, n)
    assert tr.kinds == [1, 2, 1, 2]
    rows = SO.latent_rows(cfg)
    fut = np.arange(cfg.l_full - cfg.n_ctx) < cfg.n_fut
    # recompute the pieces of step 1 (sparse, selection of step 0)
    sig = SO.sigmas(n)
    r0 = O.refresh_step(tr.x[0], model, temb(1000 * sig[0]), cfg)
    v0 = SO.velocity(r0.y[rows], io["w_v"], io["b_v"])
    y1 = O.sparse_step(tr.x[1], model, temb(1000 * sig[1]), cfg, r0.packmap)
    v1 = SO.velocity(y1[rows], io["w_v"], io["b_v"])
    kept = r0.packmap.pack_pos[rows] >= 0
    pruned_fut = fut & ~kept
    assert pruned_fut.any() and (fut & kept).any()
    np.testing.assert_array_equal(tr.v_tilde[1][pruned_fut], v0[pruned_fut])
    np.testing.assert_array_equal(tr.v_tilde[1][fut & kept], v1[fut & kept])
    np.testing.assert_array_equal(tr.v_tilde[1][~fut], v1[~fut])     # actions always current
    # and the state moved by exactly that merged velocity
    np.testing.assert_array_equal(tr.z[1], SO.euler_update(tr.z[0], tr.v_tilde[1], sig[2] - sig[1]))


def test_latent_inputs_reach_the_network_every_step():
    cfg = W.preset(1)
    model, io, si, temb, n = _sampler_case(cfg)
    tr = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, n)
    rows = SO.latent_rows(cfg)
    np.testing.assert_array_equal(tr.x[0][rows], SO.embed(si.z0, io["w_in"], io["b_in"], cfg.dtype))
    np.testing.assert_array_equal(tr.x[2][rows], SO.embed(tr.z[1], io["w_in"], io["b_in"], cfg.dtype))
    np.testing.assert_array_equal(tr.x[3][:cfg.n_ctx], si.ctx[0])
