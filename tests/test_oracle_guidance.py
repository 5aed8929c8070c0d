"""Pins of classifier-free guidance in the oracle (App. B.2 guidance scale;
Sec. 4.2 selection from the dense conditional forward) -- CPU only.

A batch of 2P sequences holds P conditional sequences and, at [P, 2P), their
unconditional partners.  The pins reduce guidance to runs without it: at
g = 1 the guided sampler is the plain sampler on the conditional half; at
g = 0 and without pruning it is the plain sampler on the unconditional half;
full retention makes the guided sparse sampler equal the guided dense one.
"""
import dataclasses

import numpy as np

import workload as W
from oracle import sampler_oracle as SO
from oracle import swam_oracle as O


def _pair_case(g, **kw):
    """A guided config (B = 2) and its two halves as plain B = 1 runs."""
    base = dataclasses.replace(W.preset(1), **kw)
    cfg = base.replace(batch=2, cfg_pairs=1, guidance=g)
    model = [W.block_weights(base, l) for l in range(base.n_blocks)]
    io = W.latent_io_weights(base)
    si = W.make_sampler_inputs(cfg)
    temb = lambda t: W.time_embedding(base, t)  # noqa: E731
    return base, cfg, model, io, si, temb


def test_guidance_pairs_score_the_conditional_half_and_share_its_selection():
    base, cfg, model, io, si, temb = _pair_case(3.0)
    inp = W.make_inputs(cfg, model[0]["w_qkv"])
    x = inp.x(0)
    r = O.refresh_step(x, model, inp.temb(0), cfg)
    assert r.S_all.shape[0] == 1 and len(r.selection) == 1
    # the conditional half alone, as a plain batch of one, gives the same scores and selection
    r1 = O.refresh_step(x[:cfg.l_full], model, inp.temb(0), base)
    np.testing.assert_array_equal(r.S_all[0], r1.S_all[0])
    keep = r.packmap.pack_pos.reshape(2, cfg.l_full) >= 0
    np.testing.assert_array_equal(keep[0], keep[1])
    np.testing.assert_array_equal(keep[0], r1.packmap.pack_pos >= 0)
    # both halves ran dense: the partner's output is its own plain dense block stack
    y_u = O.dense_step(x[cfg.l_full:], model, inp.temb(0), base)
    np.testing.assert_array_equal(r.y[cfg.l_full:], y_u)


def test_guidance_one_is_the_conditional_sampler():
    base, cfg, model, io, si, temb = _pair_case(1.0)
    tr = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, 4)
    plain = SO.run_sampler(base, model, io, si.ctx[:1], si.z0, temb, 4)
    assert tr.kinds == plain.kinds == [1, 2, 1, 2]
    for a, b in zip(tr.z, plain.z):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_guidance_zero_dense_is_the_unconditional_sampler():
    base, cfg, model, io, si, temb = _pair_case(0.0)
    tr = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, 3, dense=True)
    plain = SO.run_sampler(base, model, io, si.ctx[1:], si.z0, temb, 3, dense=True)
    for a, b in zip(tr.z, plain.z):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_guided_full_retention_equals_guided_dense():
    base, cfg, model, io, si, temb = _pair_case(3.0, k_core=64, k_anchor=0)
    sp = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, 4)
    de = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, 4, dense=True)
    for a, b in zip(sp.z, de.z):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_guided_velocity_is_affine_in_the_scale_and_extrapolates_away_from_uncond():
    rng = np.random.default_rng(4)
    vc, vu = rng.standard_normal((6, 3)), rng.standard_normal((6, 3))
    v1, v3 = SO.guided_velocity(vc, vu, 1.0), SO.guided_velocity(vc, vu, 3.0)
    np.testing.assert_allclose(v1, vc, atol=1e-15)
    np.testing.assert_allclose(SO.guided_velocity(vc, vu, 0.0), vu, atol=1e-15)
    # g = 3 lies on the line through v_u and v_c, three times as far from v_u as v_c
    np.testing.assert_allclose(v3 - vu, 3.0 * (vc - vu), atol=1e-12)


def test_guided_sparse_step_caches_the_guided_velocity():
    base, cfg, model, io, si, temb = _pair_case(3.0)
    tr = SO.run_sampler(cfg, model, io, si.ctx, si.z0, temb, 2)
    rows = SO.latent_rows(cfg)
    L_lat = cfg.l_full - cfg.n_ctx
    sig = SO.sigmas(2)
    r0 = O.refresh_step(tr.x[0], model, temb(1000 * sig[0]), cfg)
    v_all = SO.velocity(r0.y[rows], io["w_v"], io["b_v"])
    v0 = v_all[L_lat:] + 3.0 * (v_all[:L_lat] - v_all[L_lat:])
    # step 1 is sparse: pruned future rows take step 0's guided velocity
    pruned = (r0.packmap.pack_pos[rows[:L_lat]] < 0)
    assert pruned.any()
    np.testing.assert_array_equal(tr.v_tilde[1][pruned], v0[pruned])
    np.testing.assert_array_equal(tr.v_tilde[0], v0)
