"""GPU parity on multi-view frames: cameras of unequal resolution concatenated
inside each frame (N_s = sum of the views' token counts, not a rectangle),
at a small fp32 size against the oracle and at the shapes of the paper's
backbone table (App. B.2: three views of 340 tokens per frame with guidance
pairs, two views of 98 tokens with 16 aligned queries per frame).

Tolerances: fp32 outputs 1e-4 max-relative and the selection bit-exact;
bf16 outputs 2e-2 max-relative on retained rows and the selection bit-exact
when the oracle selects on the GPU's own scores; pruned rows byte-identical.
"""
import numpy as np
import pytest
import torch

import oracle as O
import workload as W
from helpers import act_dtype, dev, host, maxrel, model_for
from test_gpu_fullsize import _check_selection

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _ctx(cfg):
    from paper_2609_38984_amd import swam
    return swam.Context(cfg)


def _small_multiview(**kw):
    views = ((5, 7), (3, 4), (3, 4))                       # 35 + 12 + 12 = 59 tokens per frame
    n_s = sum(h * w for h, w in views)
    base = dict(name="f32-3view-59tok", batch=2, d_model=128, n_heads=2, n_blocks=2, n_ctx=20,
                n_frames=2, frame_h=1, frame_w=n_s, n_act=8, k_core=12, k_anchor=5, reuse_R=2,
                n_steps=4, dtype="f32", seed=11, blob_count=(1, 2), blob_sigma_range=(1.0, 2.0),
                views=views, cfg_pairs=1, guidance=3.0, rope=1, qk_norm=1)
    base.update(kw)
    return W.SwamConfig(**base)


def test_multiview_guided_rope_schedule_fp32_matches_oracle():
    from paper_2609_38984_amd import swam
    cfg = _small_multiview()
    print(f"multi-view schedule {cfg.name} N_s={cfg.n_s}", flush=True)
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ys, refr = O.run_schedule(cfg, blocks, inp.x, inp.temb)
    ctx = _ctx(cfg)
    kinds = []
    for tau in range(cfg.n_steps):
        x = dev(inp.x(tau))
        y = torch.empty_like(x)
        kinds.append(ctx.step(model, x, dev(inp.temb(tau)), tau, y))
        torch.cuda.synchronize()
        err = maxrel(host(y), ys[tau])
        print(f"  tau {tau} kind {kinds[-1]} max-rel {err:.2e}", flush=True)
        assert err < 1e-4
        if tau in refr:
            ki = torch.empty(cfg.batch * cfg.n_frames * ctx.k_max, dtype=torch.int32,
                             device="cuda:0")
            ctx.export(keep_idx=ki)
            torch.cuda.synchronize()
            want = np.concatenate([np.asarray(r) for r in refr[tau].selection[0].retained])
            got = ki.cpu().numpy().reshape(cfg.batch, -1)
            np.testing.assert_array_equal(got[0], want)
            np.testing.assert_array_equal(got[1], want)
    assert kinds == [swam.KIND_REFRESH, swam.KIND_SPARSE] * 2


def _gpu_selection(ctx, cfg):
    ki = torch.empty(cfg.batch * cfg.n_frames * ctx.k_max, dtype=torch.int32, device="cuda:0")
    kc = torch.empty(cfg.batch * cfg.n_frames, dtype=torch.int32, device="cuda:0")
    pp = torch.empty(cfg.batch * cfg.l_full, dtype=torch.int32, device="cuda:0")
    ga = torch.empty(cfg.batch * cfg.l_full, dtype=torch.int32, device="cuda:0")
    cu = torch.empty(cfg.batch + 1, dtype=torch.int32, device="cuda:0")
    S = torch.empty(cfg.n_scored * cfg.n_blocks * cfg.n_frames * cfg.n_s, dtype=torch.float32,
                    device="cuda:0")
    ctx.export(s_all=S, keep_idx=ki, keep_cnt=kc, pack_pos=pp, gather=ga, cu_seqlens=cu)
    torch.cuda.synchronize()
    return (host(S).reshape(cfg.n_scored, cfg.n_blocks, cfg.n_frames, cfg.n_s),
            ki.cpu().numpy(), kc.cpu().numpy(), pp.cpu().numpy(), ga.cpu().numpy(),
            cu.cpu().numpy())


@pytest.mark.parametrize("n", [6, 7])
def test_multiview_table_shapes_two_blocks_match_oracle(n):
    """Both table shapes with two blocks: refresh, then a sparse step, against
    the oracle on the GPU's selection."""
    from paper_2609_38984_amd import swam
    cfg = W.preset(n).replace(n_blocks=2)
    print(f"multi-view {cfg.name} (2 blocks) B={cfg.batch} N_s={cfg.n_s} g={cfg.g}", flush=True)
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ctx = _ctx(cfg)
    x0 = dev(inp.x(0), act_dtype(cfg))
    y0 = torch.empty_like(x0)
    assert ctx.step(model, x0, dev(inp.temb(0)), 0, y0) == swam.KIND_REFRESH
    S, ki, kc, pp, ga, cu = _gpu_selection(ctx, cfg)
    _check_selection(cfg, ki, kc, pp, ga, cu)
    _, sel, pm = O.selection_from_scores(cfg, S)
    for b in range(cfg.batch):
        want = np.concatenate([np.asarray(r) for r in sel[b % cfg.n_scored].retained])
        np.testing.assert_array_equal(ki.reshape(cfg.batch, -1)[b], want)
    np.testing.assert_array_equal(pp, pm.pack_pos)
    # the refresh output is the dense blocks' output
    y_ref = O.dense_step(inp.x(0), blocks, inp.temb(0), cfg)
    e0 = maxrel(host(y0), y_ref)
    # a sparse step on that selection
    x1 = dev(inp.x(1), act_dtype(cfg))
    y1 = torch.empty_like(x1)
    assert ctx.step(model, x1, dev(inp.temb(1)), 1, y1) == swam.KIND_SPARSE
    torch.cuda.synchronize()
    y1_ref = O.sparse_step(inp.x(1), blocks, inp.temb(1), cfg, pm)
    kept = pm.pack_pos >= 0
    e1 = maxrel(host(y1)[kept], y1_ref[kept])
    print(f"  refresh max-rel {e0:.2e}, sparse kept rows max-rel {e1:.2e}", flush=True)
    assert e0 < 2e-2 and e1 < 2e-2
    assert host(y1)[~kept].tobytes() == host(x1)[~kept].tobytes()


def test_multiview_guided_fullsize_step_properties():
    """All 28 blocks of the three-view guided shape: selection structure,
    partners sharing it, score mass bounds, pruned rows byte-identical."""
    from paper_2609_38984_amd import swam
    cfg = W.preset(6)
    print(f"multi-view full size {cfg.name}", flush=True)
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ctx = _ctx(cfg)
    x0 = dev(inp.x(0), act_dtype(cfg))
    y0 = torch.empty_like(x0)
    assert ctx.step(model, x0, dev(inp.temb(0)), 0, y0) == swam.KIND_REFRESH
    S, ki, kc, pp, ga, cu = _gpu_selection(ctx, cfg)
    assert (S >= 0).all() and (S.sum(axis=3) <= 1 + 1e-5).all()
    _check_selection(cfg, ki, kc, pp, ga, cu)
    kk = ki.reshape(cfg.batch, -1)
    np.testing.assert_array_equal(kk[0], kk[1])
    assert cu[-1] == cfg.batch * cfg.t_pack_fixed == ctx.packed_rows()
    for tau in (1, 2, 3):
        x = dev(inp.x(tau), act_dtype(cfg))
        y = torch.empty_like(x)
        assert ctx.step(model, x, dev(inp.temb(tau)), tau, y) == swam.KIND_SPARSE
        torch.cuda.synchronize()
        pruned = torch.from_numpy(pp < 0)
        assert torch.equal(y.cpu()[pruned].view(torch.int16), x.cpu()[pruned].view(torch.int16))
        assert np.isfinite(host(y)).all()
