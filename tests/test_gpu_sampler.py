"""GPU parity of the sampling-update calls (swam_embed, swam_velocity,
swam_sample_update, swam_sample_step) against the sampler oracle.

Tolerances: embedded tokens within one unit in the last place of their
storage type plus the fp32 error bound of the c-term accumulation (which
dominates where the sum cancels); velocities 1e-4 max-relative (fp32
LayerNorm and dot products against float64); the Euler update within one
fp32 ulp (one FMA against a float64 value rounded once); the closed fp32
sampler 1e-4 max-relative per step; rows that a call must not touch are
bit-identical.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle as O
import workload as W
from helpers import act_dtype, dev, host, maxrel, model_for
from oracle import sampler_oracle as SO

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _small_bf16(**kw):
    base = dict(name="bf16-small", batch=2, d_model=256, n_heads=4, n_blocks=2, n_ctx=20,
                n_frames=2, frame_h=8, frame_w=9, n_act=8, k_core=18, k_anchor=6, reuse_R=2,
                n_steps=4, dtype="bf16", seed=7, blob_sigma=1.5)
    base.update(kw)
    return W.SwamConfig(**base)


def _io(cfg, c=16):
    from paper_2609_38984_amd import swam
    w = W.latent_io_weights(cfg, c)
    return w, swam.LatentIO({k: dev(v, act_dtype(cfg)) for k, v in w.items()}, act_dtype(cfg))


def _embed_bound(z, w_in, b_in, want, ulp_rel):
    """Per element: one storage ulp of the result plus the fp32 error bound of
    a c-term accumulation, 2^-24 * c * sum_k |z_k w_k| (+ |b|), which dominates
    where the sum cancels."""
    mag = np.abs(z).astype(np.float64) @ np.abs(w_in).astype(np.float64).T + np.abs(b_in)
    return ulp_rel * np.abs(want) + 2.0 ** -24 * (z.shape[1] + 1) * mag


@pytest.mark.parametrize("cfg_fn", [lambda: W.preset(1), lambda: _small_bf16()], ids=["f32", "bf16"])
def test_embed_writes_latent_rows_only(cfg_fn):
    from paper_2609_38984_amd import swam
    cfg = cfg_fn()
    print(f"embed {cfg.name}", flush=True)
    w, io = _io(cfg)
    rng = np.random.default_rng(11)
    n_lat = cfg.batch * (cfg.l_full - cfg.n_ctx)
    z = rng.standard_normal((n_lat, 16)).astype(np.float32)
    x0 = W.make_inputs(cfg).x(0)
    ctx = swam.Context(cfg)
    xd = dev(x0, act_dtype(cfg))
    ctx.embed(io, dev(z), xd)
    torch.cuda.synchronize()
    got = host(xd)
    rows = SO.latent_rows(cfg)
    want = SO.embed(z, w["w_in"], w["b_in"], cfg.dtype)
    other = np.setdiff1d(np.arange(cfg.batch * cfg.l_full), rows)
    np.testing.assert_array_equal(got[other], x0[other])
    # one ulp is at most 2^-7 (bf16) / 2^-23 (fp32) of the value
    bound = _embed_bound(z, w["w_in"], w["b_in"], want, 2.0 ** -7 if cfg.dtype == "bf16" else 2.0 ** -23)
    err = np.abs(got[rows] - want)
    worst = np.unravel_index(np.argmax(err - bound), err.shape)
    assert np.all(err <= bound), (worst, got[rows][worst], want[worst], bound[worst])


@pytest.mark.parametrize("cfg_fn", [lambda: W.preset(1), lambda: _small_bf16(),
                                    lambda: dataclasses.replace(_small_bf16(), name="bf16-c40")],
                         ids=["f32", "bf16", "bf16-c40"])
def test_velocity_all_rows_and_retained_rows(cfg_fn):
    from paper_2609_38984_amd import swam
    cfg = cfg_fn()
    c = 40 if cfg.name == "bf16-c40" else 16
    print(f"velocity {cfg.name} c={c}", flush=True)
    w, io = _io(cfg, c)
    blocks, dblocks, model = model_for(cfg)
    x = W.make_inputs(cfg, blocks[0]["w_qkv"]).x(0)
    ctx = swam.Context(cfg)
    xd = dev(x, act_dtype(cfg))
    yd = torch.empty_like(xd)
    ctx.step(model, xd, dev(W.timestep_embedding(cfg, 0)), 0, yd)      # refresh: selection cached
    n_lat = cfg.batch * (cfg.l_full - cfg.n_ctx)
    v_all = torch.full((n_lat, c), 12345.0, dtype=torch.float32, device="cuda:0")
    v_ret = torch.full((n_lat, c), 12345.0, dtype=torch.float32, device="cuda:0")
    ctx.velocity(io, yd, v_all)
    ctx.velocity(io, yd, v_ret, retained_only=True)
    pack_pos = torch.empty(cfg.batch * cfg.l_full, dtype=torch.int32, device="cuda:0")
    ctx.export(pack_pos=pack_pos)
    torch.cuda.synchronize()
    rows = SO.latent_rows(cfg)
    want = SO.velocity(host(yd)[rows], w["w_v"], w["b_v"])
    assert maxrel(host(v_all), want) < 1e-4
    kept = host(pack_pos)[rows] >= 0
    assert kept.any() and (~kept).any()
    vr = host(v_ret)
    assert maxrel(vr[kept], want[kept]) < 1e-4
    assert np.all(vr[~kept] == 12345.0)


@pytest.mark.parametrize("kind", [0, 1, 2])
def test_sample_update_kinds(kind):
    from paper_2609_38984_amd import swam
    cfg = _small_bf16()
    print(f"sample update kind={kind}", flush=True)
    blocks, dblocks, model = model_for(cfg)
    ctx = swam.Context(cfg)
    x = W.make_inputs(cfg, blocks[0]["w_qkv"]).x(0)
    xd = dev(x, act_dtype(cfg))
    ctx.step(model, xd, dev(W.timestep_embedding(cfg, 0)), 0, torch.empty_like(xd))
    n_lat = cfg.batch * (cfg.l_full - cfg.n_ctx)
    rng = np.random.default_rng(kind)
    z, v, vc = (rng.standard_normal((n_lat, 16)).astype(np.float32) for _ in range(3))
    zd, vd, vcd = dev(z), dev(v), dev(vc)
    dsig = float(np.float32(-0.0625))
    ctx.sample_update(16, vd, vcd, zd, dsig, kind)
    pack_pos = torch.empty(cfg.batch * cfg.l_full, dtype=torch.int32, device="cuda:0")
    ctx.export(pack_pos=pack_pos)
    torch.cuda.synchronize()
    fut = np.tile(np.arange(cfg.l_full - cfg.n_ctx) < cfg.n_fut, cfg.batch)
    if kind == 2:
        keep = (host(pack_pos)[SO.latent_rows(cfg)] >= 0) | ~fut
        vt = SO.merge_velocity(v, vc, keep)
    else:
        vt = v
    want = SO.euler_update(z, vt, dsig)
    np.testing.assert_allclose(host(zd), want, rtol=1.2e-7, atol=1e-30)
    want_cache = np.where(fut[:, None], v, vc) if kind == 1 else vc
    np.testing.assert_array_equal(host(vcd), want_cache)


def test_sparse_update_without_selection_is_a_state_error():
    from paper_2609_38984_amd import swam
    cfg = _small_bf16()
    ctx = swam.Context(cfg)
    n = cfg.batch * (cfg.l_full - cfg.n_ctx) * 16
    t = torch.zeros(n, dtype=torch.float32, device="cuda:0")
    with pytest.raises(swam.SwamError) as e:
        ctx.sample_update(16, t, t.clone(), t.clone(), -0.1, swam.KIND_SPARSE)
    assert e.value.code == -4


def test_closed_loop_sampler_fp32_matches_oracle():
    from paper_2609_38984_amd import swam
    cfg = W.preset(1)
    print("closed loop fp32 config 1", flush=True)
    blocks, dblocks, model = model_for(cfg)
    w, io = _io(cfg)
    si = W.make_sampler_inputs(cfg)
    temb_of_t = lambda t: W.time_embedding(cfg, t)  # noqa: E731
    tr = SO.run_sampler(cfg, blocks, w, si.ctx, si.z0, temb_of_t)
    ctx = swam.Context(cfg)
    n_lat = cfg.batch * (cfg.l_full - cfg.n_ctx)
    zd = dev(si.z0)
    vd = torch.zeros(n_lat, 16, dtype=torch.float32, device="cuda:0")
    vcd = torch.zeros_like(vd)
    x = np.zeros((cfg.batch * cfg.l_full, cfg.d_model), np.float32)
    for b in range(cfg.batch):
        x[b * cfg.l_full:b * cfg.l_full + cfg.n_ctx] = si.ctx[b]
    xd = dev(x)
    yd = torch.empty_like(xd)
    sig = swam.flow_sigmas(cfg.n_steps)
    kinds = []
    for tau in range(cfg.n_steps):
        temb = dev(temb_of_t(1000.0 * sig[tau]))
        kinds.append(ctx.sample_step(model, io, zd, vd, vcd, xd, yd, temb, tau,
                                     sig[tau + 1] - sig[tau]))
        torch.cuda.synchronize()
        e = maxrel(host(zd), tr.z[tau])
        print(f"  step {tau} kind {kinds[-1]} z max-rel {e:.2e}", flush=True)
        assert e < 1e-4
    assert kinds == tr.kinds == [1, 2, 1, 2]


def test_sample_step_rejects_aliased_buffers():
    from paper_2609_38984_amd import swam
    cfg = _small_bf16()
    _, _, model = model_for(cfg)
    _, io = _io(cfg)
    ctx = swam.Context(cfg)
    n_lat = cfg.batch * (cfg.l_full - cfg.n_ctx)
    z = torch.zeros(n_lat, 16, dtype=torch.float32, device="cuda:0")
    x = torch.zeros(cfg.batch * cfg.l_full, cfg.d_model, dtype=torch.bfloat16, device="cuda:0")
    with pytest.raises(swam.SwamError) as e:
        ctx.sample_step(model, io, z, z.clone(), z.clone(), x, x,
                        dev(W.time_embedding(cfg, 1000.0)), 0, -0.1)
    assert e.value.code == -1


def test_closed_loop_sampler_bf16_step_properties():
    """bf16 closed loop over the schedule: the sparse steps move pruned future
    latents by exactly dsigma times the cached velocity, retained ones by the
    velocity of the current output, and the selection stays fixed between
    refreshes."""
    from paper_2609_38984_amd import swam
    cfg = _small_bf16()
    print("closed loop bf16 properties", flush=True)
    blocks, dblocks, model = model_for(cfg)
    w, io = _io(cfg)
    si = W.make_sampler_inputs(cfg)
    ctx = swam.Context(cfg)
    n_lat = cfg.batch * (cfg.l_full - cfg.n_ctx)
    zd = dev(si.z0)
    vd = torch.zeros(n_lat, 16, dtype=torch.float32, device="cuda:0")
    vcd = torch.zeros_like(vd)
    x = np.zeros((cfg.batch * cfg.l_full, cfg.d_model), np.float32)
    for b in range(cfg.batch):
        x[b * cfg.l_full:b * cfg.l_full + cfg.n_ctx] = si.ctx[b]
    xd = dev(x, torch.bfloat16)
    yd = torch.empty_like(xd)
    sig = swam.flow_sigmas(cfg.n_steps)
    rows = SO.latent_rows(cfg)
    fut = np.tile(np.arange(cfg.l_full - cfg.n_ctx) < cfg.n_fut, cfg.batch)
    pack_pos = torch.empty(cfg.batch * cfg.l_full, dtype=torch.int32, device="cuda:0")
    for tau in range(cfg.n_steps):
        z_before = host(zd)
        cache_before = host(vcd)
        kind = ctx.sample_step(model, io, zd, vd, vcd, xd, yd,
                               dev(W.time_embedding(cfg, 1000.0 * sig[tau])), tau,
                               sig[tau + 1] - sig[tau])
        ctx.export(pack_pos=pack_pos)
        torch.cuda.synchronize()
        z_after, v_now, y = host(zd), host(vd), host(yd)
        dsig = float(np.float32(sig[tau + 1] - sig[tau]))     # the call takes dsigma as fp32
        keep = (host(pack_pos)[rows] >= 0) | ~fut
        if kind == swam.KIND_SPARSE:
            pruned = fut & ~keep
            assert pruned.any()
            np.testing.assert_allclose(z_after[pruned],
                                       SO.euler_update(z_before[pruned], cache_before[pruned], dsig),
                                       rtol=1.2e-7, atol=1e-30)
        # retained (or all, after a full step) rows move by the head of the current output
        sel = keep if kind == swam.KIND_SPARSE else np.ones_like(keep)
        v_ref = SO.velocity(y[rows][sel], w["w_v"], w["b_v"])
        assert maxrel(v_now[sel], v_ref) < 1e-4
        np.testing.assert_allclose(z_after[sel], SO.euler_update(z_before[sel], v_now[sel], dsig),
                                   rtol=1.2e-7, atol=1e-30)
    # the network input of the last step embedded the latents of the step before
    assert np.isfinite(host(zd)).all()
