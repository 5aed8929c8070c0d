"""Parity at the full workload sizes, in the launch configuration bench.py times.

Blocks are checked on sampled rows that the oracle computes one by one (keys
and values over the whole sequence, queries and the rest only for the sample);
whole steps are checked through properties that hold at any size: attention
normalisers, score mass bounds, selection structure, pruned rows byte-identical,
full retention equal to the dense step, reuse equal to re-selection, determinism.
"""
import numpy as np
import pytest
import torch

import oracle as O
import workload as W
from helpers import act_dtype, dev, host, lse_from_qkv, maxrel, model_for
from test_oracle_blob import blob_centres

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _ctx(cfg):
    from paper_2609_38984_amd import swam
    return swam.Context(cfg)


def _sample_rows(cu, per_seq, rng):
    rows = []
    for a, b in zip(cu[:-1], cu[1:]):
        if b > a:
            rows += [a, b - 1]
            rows += list(rng.integers(a, b, per_seq))
    return np.unique(np.asarray(rows, np.int64))


def _sampled_block(cfg, cu, x, per_seq=24):
    print(f"full-size block {cfg.name} rows={int(cu[-1])} seqs={len(cu) - 1}", flush=True)
    blocks, dblocks, _ = model_for(cfg, 1)
    temb = W.timestep_embedding(cfg, 0)
    n_rows = int(cu[-1])
    ctx = _ctx(cfg)
    xd = dev(x[:n_rows], act_dtype(cfg))
    lse = torch.empty(n_rows, cfg.n_heads, dtype=torch.float32, device="cuda:0")
    qkv = torch.empty(n_rows, 3 * cfg.d_model, dtype=act_dtype(cfg), device="cuda:0")
    ctx.block(dblocks[0], dev(temb), xd, n_rows, dev(np.asarray(cu, np.int32)), len(cu) - 1, lse,
              qkv)
    torch.cuda.synchronize()
    rows = _sample_rows(cu, per_seq, np.random.default_rng(5))
    y_ref, l_ref = O.block_rows(x[:n_rows], blocks[0], temb, cu, rows, cfg.n_heads, cfg.dtype)
    e_y = maxrel(host(xd)[rows], y_ref)
    e_l = float(np.abs(host(lse)[rows] - l_ref).max())
    # the kernel's normaliser against the log-sum-exp of its own q and k (every head)
    e_own = float(np.abs(host(lse)[rows] - lse_from_qkv(host(qkv), cu, rows, cfg.n_heads)).max())
    print(f"  sampled {len(rows)} rows: y max-rel {e_y:.2e}, lambda abs {e_l:.2e}, "
          f"lambda abs on own qkv {e_own:.2e}", flush=True)
    assert e_y < 2e-2 and e_l < 1e-2 and e_own < 1e-5


def test_block_wam_dense_10160_sampled():
    cfg = W.preset(3)
    x = W.make_inputs(cfg, W.block_weights(cfg, 0)["w_qkv"]).x(0)
    _sampled_block(cfg, O.dense_cu(cfg), x)


def test_block_wam_packed_3472_sampled():
    """The packed sequence of the WAM workload as the bench times it: the
    4-wave attention, the 192x128 out projection, the 192x256 MLP up tile
    and the down projection split along K in three."""
    cfg = W.preset(3)
    x = W.make_inputs(cfg, W.block_weights(cfg, 0)["w_qkv"]).x(0)
    _sampled_block(cfg, np.array([0, cfg.t_pack_fixed]), x)


def test_block_ragged_batch_sampled():
    cfg = W.preset(5)
    rng = np.random.default_rng(9)
    lens = rng.integers(600, cfg.l_full + 1, cfg.batch)
    cu = np.concatenate([[0], np.cumsum(lens)])
    x = W.make_inputs(cfg, W.block_weights(cfg, 0)["w_qkv"]).x(0)
    _sampled_block(cfg, cu, x, per_seq=6)


def test_block_2048_packed_3744_sampled():
    """The packed sequence of the d = 2048 workload at 10% + 64 retention
    (3,744 rows, 32 heads): 480 attention workgroups of 8 waves, the 192x256
    QKV tile and the down projection split along K in two."""
    cfg = W.preset(4, percent=10).replace(n_blocks=1)
    assert cfg.t_pack_fixed == 3744
    x = W.make_inputs(cfg, W.block_weights(cfg, 0)["w_qkv"]).x(0)
    _sampled_block(cfg, np.array([0, cfg.t_pack_fixed]), x, per_seq=24)


def test_block_wam_packed_4200_sampled():
    """4,200 packed rows of the WAM width (24 heads): the 4-wave attention
    kernel with its four-waves-per-SIMD register cap (33 query tiles per head,
    too few for the 8-wave kernel), the 128x128 QKV tile and the down
    projection split along K in two."""
    cfg = W.preset(3)
    x = W.make_inputs(cfg, W.block_weights(cfg, 0)["w_qkv"]).x(0)
    _sampled_block(cfg, np.array([0, 4200]), x)


@pytest.mark.parametrize("pct,rows", [(25, 6208), (50, 10304)])
def test_block_2048_packed_sampled(pct, rows):
    """The packed sequences of the d = 2048 workload at 25% + 64 (the bench's
    second point: 800 workgroups of the 8-wave attention, 256x256 projections)
    and 50% + 64 retention (the out projection on the 192x256 tile, the down
    projection split along K in three)."""
    cfg = W.preset(4, percent=pct).replace(n_blocks=1)
    assert cfg.t_pack_fixed == rows
    x = W.make_inputs(cfg, W.block_weights(cfg, 0)["w_qkv"]).x(0)
    _sampled_block(cfg, np.array([0, rows]), x, per_seq=16)


def test_block_2048_dense_sampled():
    cfg = W.preset(4, percent=25).replace(n_blocks=1)
    x = W.make_inputs(cfg, W.block_weights(cfg, 0)["w_qkv"]).x(0)
    _sampled_block(cfg, O.dense_cu(cfg), x, per_seq=16)


def _check_selection(cfg, ki, kc, pp, ga, cu):
    ki = ki.reshape(cfg.batch, cfg.n_frames, -1)
    kc = kc.reshape(cfg.batch, cfg.n_frames)
    for b in range(cfg.batch):
        keep_full = np.zeros(cfg.l_full, bool)
        keep_full[:cfg.n_ctx] = True
        keep_full[cfg.n_ctx + cfg.n_fut:] = True
        for f in range(cfg.n_frames):
            r = ki[b, f, :kc[b, f]]
            assert (np.diff(r) > 0).all() and r.min() >= 0 and r.max() < cfg.n_s
            assert (ki[b, f, kc[b, f]:] == -1).all()
            if cfg.mass_threshold == 0:
                assert kc[b, f] == cfg.k_core + cfg.k_anchor
            keep_full[cfg.n_ctx + f * cfg.n_s + r] = True
        seg = pp[b * cfg.l_full:(b + 1) * cfg.l_full]
        assert ((seg >= 0) == keep_full).all()
        kept = seg[seg >= 0]
        assert (np.diff(kept) == 1).all() and kept[0] == cu[b] and kept[-1] == cu[b + 1] - 1
        np.testing.assert_array_equal(ga[cu[b]:cu[b + 1]], b * cfg.l_full + np.nonzero(keep_full)[0])
    # anchors are shared: every frame of a sequence contains the same K_s positions outside its core


def test_step_wam_fullsize_properties():
    from paper_2609_38984_amd import swam
    cfg = W.preset(3)
    print(f"full-size step {cfg.name}", flush=True)
    blocks, dblocks, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ctx = _ctx(cfg)
    x0, x1 = dev(inp.x(0), torch.bfloat16), dev(inp.x(1), torch.bfloat16)
    t0, t1 = dev(inp.temb(0)), dev(inp.temb(1))
    y0 = torch.empty_like(x0)
    assert ctx.step(model, x0, t0, 0, y0) == swam.KIND_REFRESH
    n_s, F, L = cfg.n_s, cfg.n_frames, cfg.n_blocks
    S = torch.empty(L * F * n_s, dtype=torch.float32, device="cuda:0")
    ki = torch.empty(F * ctx.k_max, dtype=torch.int32, device="cuda:0")
    kc = torch.empty(F, dtype=torch.int32, device="cuda:0")
    pp = torch.empty(cfg.l_full, dtype=torch.int32, device="cuda:0")
    ga = torch.empty(cfg.l_full, dtype=torch.int32, device="cuda:0")
    cu = torch.empty(2, dtype=torch.int32, device="cuda:0")
    ctx.export(s_all=S, keep_idx=ki, keep_cnt=kc, pack_pos=pp, gather=ga, cu_seqlens=cu)
    torch.cuda.synchronize()
    Sh = host(S).reshape(L, F, n_s)
    assert (Sh >= 0).all() and (Sh.sum(axis=2) <= 1 + 1e-5).all()
    assert np.isfinite(host(y0)).all()
    cuh = cu.cpu().numpy()
    assert cuh[-1] == cfg.t_pack_fixed == ctx.packed_rows()
    _check_selection(cfg, ki.cpu().numpy(), kc.cpu().numpy(), pp.cpu().numpy(), ga.cpu().numpy(), cuh)
    # the planted action-relevant blob: its centre is a core token of every
    # frame (the oracle's select on the kernel's V and A reproduces the
    # kernel's selection bit for bit, so its core sets are the kernel's)
    Vd = torch.empty(F * n_s, dtype=torch.float32, device="cuda:0")
    Ad = torch.empty(n_s, dtype=torch.float32, device="cuda:0")
    ctx.export(v=Vd, a=Ad)
    torch.cuda.synchronize()
    Vh = Vd.cpu().numpy().reshape(F, n_s)
    sel = O.select(Vh, Ad.cpu().numpy(), cfg.k_core, cfg.k_anchor)
    kih = ki.cpu().numpy().reshape(F, -1)
    for f, centres in enumerate(blob_centres(inp, cfg, 0, 0)):
        for j in centres:
            rank = int((Vh[f] > Vh[f, j]).sum())
            print(f"  frame {f}: blob centre {j} ranks {rank} of {n_s}", flush=True)
            assert j in set(int(i) for i in sel.core[f]) and j in set(int(i) for i in kih[f])
    # reuse: re-selecting on the exported scores in a fresh context gives the cached selection
    ctx2 = _ctx(cfg)
    V = torch.empty(F * n_s, dtype=torch.float32, device="cuda:0")
    A = torch.empty(n_s, dtype=torch.float32, device="cuda:0")
    ctx2.score_reduce(S, V, A)
    ki2 = torch.empty_like(ki)
    ctx2.select(None, None, ki2)
    torch.cuda.synchronize()
    assert torch.equal(ki2, ki)
    # sparse step: pruned rows keep x(1) byte for byte
    y1 = torch.empty_like(x1)
    assert ctx.step(model, x1, t1, 1, y1) == swam.KIND_SPARSE
    torch.cuda.synchronize()
    pruned = torch.from_numpy(pp.cpu().numpy() < 0)
    assert torch.equal(y1.cpu()[pruned].view(torch.int16), x1.cpu()[pruned].view(torch.int16))
    assert np.isfinite(host(y1)).all()
    # determinism: a second refresh gives identical bytes
    y0b = torch.empty_like(x0)
    ctx.step(model, x0, t0, 0, y0b)
    S2 = torch.empty_like(S)
    ctx.export(s_all=S2)
    torch.cuda.synchronize()
    assert torch.equal(y0b.view(torch.int16), y0.view(torch.int16)) and torch.equal(S2, S)


def test_refresh_scores_equal_layerwise_scoring_fullsize():
    """At the WAM shape a bf16 refresh scores every layer but the last inside
    its MLP up projection launch and the last one with the scoring kernel on
    the side stream.  Chaining the blocks one call at a time and scoring each
    layer's own q, k and lambda with the standalone kernel must give the same
    S bit for bit (the same scoring arithmetic in a fixed order), and the same
    step output."""
    from paper_2609_38984_amd import swam
    cfg = W.preset(3).replace(n_blocks=4)
    print(f"refresh scores vs layerwise scoring {cfg.name} L={cfg.n_blocks}", flush=True)
    blocks, dblocks, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ctx = _ctx(cfg)
    assert cfg.batch == 1 and ctx.n_scored == 1
    x0, t0 = dev(inp.x(0), torch.bfloat16), dev(inp.temb(0))
    y0 = torch.empty_like(x0)
    assert ctx.step(model, x0, t0, 0, y0) == swam.KIND_REFRESH
    n_s, F, L, d = cfg.n_s, cfg.n_frames, cfg.n_blocks, cfg.d_model
    S = torch.empty(L * F * n_s, dtype=torch.float32, device="cuda:0")
    ctx.export(s_all=S)
    act0 = cfg.n_ctx + cfg.n_fut
    ld = 3 * d
    x = x0.clone()
    lse = torch.empty(cfg.l_full, cfg.n_heads, dtype=torch.float32, device="cuda:0")
    qkv = torch.empty(cfg.l_full, ld, dtype=torch.bfloat16, device="cuda:0")
    S_lay = torch.empty(L, F * n_s, dtype=torch.float32, device="cuda:0")
    ctx2 = _ctx(cfg)
    for l in range(L):
        ctx2.block(dblocks[l], t0, x, None, None, 0, lse, qkv)
        flat = qkv.view(-1)
        ctx2.score(flat[act0 * ld:], cfg.l_full * ld, ld, flat[cfg.n_ctx * ld + d:],
                   cfg.l_full * ld, ld, S_lay[l], lse_act=lse[act0:].contiguous())
    torch.cuda.synchronize()
    Sh, Lh = host(S).reshape(L, F, n_s), host(S_lay).reshape(L, F, n_s)
    for l in range(L):
        diff = float(np.abs(Sh[l] - Lh[l]).max())
        print(f"  layer {l}: max |S_step - S_layer| {diff:.3e}", flush=True)
    assert torch.equal(S.view(L, -1), S_lay)
    assert torch.equal(y0.view(torch.int16), x.view(torch.int16))


def test_attention_normalisers_sum_to_one_fullsize():
    """sum over all keys of exp(q.k/8 - lambda) = 1 for the action rows, with the
    kernel's own q, k and lambda (a property at any size)."""
    cfg = W.preset(3)
    blocks, dblocks, _ = model_for(cfg, 1)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ctx = _ctx(cfg)
    x = dev(inp.x(0), torch.bfloat16)
    qkv = torch.empty(cfg.l_full, 3 * cfg.d_model, dtype=torch.bfloat16, device="cuda:0")
    lse = torch.empty(cfg.l_full, cfg.n_heads, dtype=torch.float32, device="cuda:0")
    ctx.block(dblocks[0], dev(inp.temb(0)), x, None, None, 0, lse, qkv)
    torch.cuda.synchronize()
    q = host(qkv)
    lam = host(lse)
    d = cfg.d_model
    act = np.arange(cfg.n_ctx + cfg.n_fut, cfg.l_full)
    for h in range(0, cfg.n_heads, 5):
        c = slice(h * 64, (h + 1) * 64)
        logits = q[act][:, c] @ q[:, d:2 * d][:, c].T / 8.0
        tot = np.exp(logits - lam[act, h][:, None]).sum(axis=1)
        np.testing.assert_allclose(tot, 1.0, atol=2e-5)


def test_full_retention_sparse_equals_dense_fullsize():
    """rho = 100%: the packed sequence is the full sequence in the same order, so
    the sparse step reproduces the dense step byte for byte (2048-wide blocks)."""
    from paper_2609_38984_amd import swam
    cfg = W.preset(4, percent=100).replace(n_blocks=2)
    print(f"full retention {cfg.name}", flush=True)
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ctx = _ctx(cfg)
    x0, x1 = dev(inp.x(0), torch.bfloat16), dev(inp.x(1), torch.bfloat16)
    y = torch.empty_like(x0)
    ctx.step(model, x0, dev(inp.temb(0)), 0, y)
    assert ctx.packed_rows() == cfg.l_full
    ys = torch.empty_like(x1)
    yd = torch.empty_like(x1)
    assert ctx.step(model, x1, dev(inp.temb(1)), 1, ys) == swam.KIND_SPARSE
    assert ctx.step(model, x1, dev(inp.temb(1)), 1, yd, swam.FORCE_DENSE) == swam.KIND_DENSE
    torch.cuda.synchronize()
    assert torch.equal(ys.view(torch.int16), yd.view(torch.int16))


def test_ragged_mass_threshold_step_fullsize():
    """Batched ragged workload: mass-threshold selection gives per-frame counts,
    packed lengths are ragged, pruned rows stay byte-identical."""
    from paper_2609_38984_amd import swam
    cfg = W.preset(5).replace(n_blocks=2)
    print(f"ragged step {cfg.name}", flush=True)
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ctx = _ctx(cfg)
    x0, x1 = dev(inp.x(0), torch.bfloat16), dev(inp.x(1), torch.bfloat16)
    y = torch.empty_like(x0)
    ctx.step(model, x0, dev(inp.temb(0)), 0, y)
    ki = torch.empty(cfg.batch * cfg.n_frames * ctx.k_max, dtype=torch.int32, device="cuda:0")
    kc = torch.empty(cfg.batch * cfg.n_frames, dtype=torch.int32, device="cuda:0")
    pp = torch.empty(cfg.batch * cfg.l_full, dtype=torch.int32, device="cuda:0")
    ga = torch.empty(cfg.batch * cfg.l_full, dtype=torch.int32, device="cuda:0")
    cu = torch.empty(cfg.batch + 1, dtype=torch.int32, device="cuda:0")
    ctx.export(keep_idx=ki, keep_cnt=kc, pack_pos=pp, gather=ga, cu_seqlens=cu)
    torch.cuda.synchronize()
    cuh = cu.cpu().numpy()
    _check_selection(cfg, ki.cpu().numpy(), kc.cpu().numpy(), pp.cpu().numpy(), ga.cpu().numpy(), cuh)
    lens = np.diff(cuh)
    print(f"  packed lengths {lens.tolist()}", flush=True)
    assert cuh[-1] == ctx.packed_rows()
    y1 = torch.empty_like(x1)
    assert ctx.step(model, x1, dev(inp.temb(1)), 1, y1) == swam.KIND_SPARSE
    torch.cuda.synchronize()
    pruned = torch.from_numpy(pp.cpu().numpy() < 0)
    assert torch.equal(y1.cpu()[pruned].view(torch.int16), x1.cpu()[pruned].view(torch.int16))
    assert np.isfinite(host(y1)).all()


def test_closed_loop_sampler_wam_fullsize_properties():
    """Closed-loop sampling at the 10,160-token d=1536 shape for one refresh
    and one sparse step: pruned future latents move by exactly dsigma times
    the cached velocity, retained and action latents by the read-out of the
    current output (checked against the oracle read-out on sampled rows)."""
    from oracle import sampler_oracle as SO
    from paper_2609_38984_amd import swam
    cfg = W.preset(3)
    print("sampler fullsize", flush=True)
    blocks, dblocks, model = model_for(cfg)
    wio = W.latent_io_weights(cfg)
    io = swam.LatentIO({k: dev(v, torch.bfloat16) for k, v in wio.items()}, torch.bfloat16)
    si = W.make_sampler_inputs(cfg)
    ctx = swam.Context(cfg)
    n_lat = cfg.batch * (cfg.l_full - cfg.n_ctx)
    z = dev(si.z0)
    v, vc = torch.zeros_like(z), torch.zeros_like(z)
    x = torch.zeros(cfg.batch * cfg.l_full, cfg.d_model, dtype=torch.bfloat16, device="cuda:0")
    x[:cfg.n_ctx] = dev(si.ctx[0], torch.bfloat16)
    y = torch.empty_like(x)
    sig = swam.flow_sigmas(cfg.n_steps)
    rows = SO.latent_rows(cfg)
    fut = np.arange(cfg.l_full - cfg.n_ctx) < cfg.n_fut
    rng = np.random.default_rng(0)
    pack_pos = torch.empty(cfg.l_full, dtype=torch.int32, device="cuda:0")
    for tau in range(2):
        z0, c0 = host(z), host(vc)
        kind = ctx.sample_step(model, io, z, v, vc, x, y,
                               dev(W.time_embedding(cfg, 1000.0 * sig[tau])), tau,
                               sig[tau + 1] - sig[tau])
        ctx.export(pack_pos=pack_pos)
        torch.cuda.synchronize()
        dsig = float(np.float32(sig[tau + 1] - sig[tau]))
        z1, vn = host(z), host(v)
        keep = (host(pack_pos)[rows] >= 0) | ~fut
        assert kind == (swam.KIND_REFRESH if tau == 0 else swam.KIND_SPARSE)
        if kind == swam.KIND_SPARSE:
            pruned = ~keep
            np.testing.assert_allclose(z1[pruned], SO.euler_update(z0[pruned], c0[pruned], dsig),
                                       rtol=1.2e-7, atol=1e-30)
            live = np.nonzero(keep)[0]
        else:
            live = np.arange(n_lat)
        pick = rng.choice(live, 64, replace=False)
        ref = SO.velocity(host(y)[rows[pick]], wio["w_v"], wio["b_v"])
        assert maxrel(vn[pick], ref) < 1e-4
        np.testing.assert_allclose(z1[pick], SO.euler_update(z0[pick], vn[pick], dsig),
                                   rtol=1.2e-7, atol=1e-30)
