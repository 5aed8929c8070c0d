"""Whole bf16 schedules against the oracle, step by step.

The 8-block d = 1024 workload (1,312 tokens, 4 frames of 16 x 16, 77 + 16
retained per frame, 10 steps, reuse R = 2) runs through swam_step.  At every
refresh the oracle reduces and selects on the kernel's own fp32 scores S_all
(Sec. 4.1, App. A.1): indices, counts, pack map, gather list and cu_seqlens
must match bit for bit.  Each sparse step is compared with the oracle's sparse
step on that packing (Sec. 4.2 compact execution) within 2e-2 max-relative,
with pruned rows byte-identical to the input; the first refresh's dense output
is compared with the oracle's dense step the same way.  The same schedule
replayed from captured HIP graphs (swam_step_graph) is checked against the
oracle in the same way.  One-block schedules (the block that packs is the one
that scatters back), in place and out of place, one and two sequences.
"""
import numpy as np
import pytest
import torch

import oracle as O
import workload as W
from helpers import dev, host, maxrel, model_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _exported_selection(ctx, cfg):
    F, n_s = cfg.n_frames, cfg.n_s
    out = dict(s_all=torch.empty(cfg.n_scored * cfg.n_blocks * F * n_s, dtype=torch.float32, device="cuda:0"),
               keep_idx=torch.empty(cfg.batch * F * ctx.k_max, dtype=torch.int32, device="cuda:0"),
               keep_cnt=torch.empty(cfg.batch * F, dtype=torch.int32, device="cuda:0"),
               pack_pos=torch.empty(cfg.batch * cfg.l_full, dtype=torch.int32, device="cuda:0"),
               gather=torch.empty(cfg.batch * cfg.l_full, dtype=torch.int32, device="cuda:0"),
               cu_seqlens=torch.empty(cfg.batch + 1, dtype=torch.int32, device="cuda:0"))
    ctx.export(**out)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def _check_selection_on_own_scores(cfg, got, kmax):
    S = got["s_all"].reshape(cfg.n_scored, cfg.n_blocks, cfg.n_frames, cfg.n_s)
    assert (S >= 0).all() and (S.sum(axis=3) <= 1 + 1e-5).all()
    _, sel, pm = O.selection_from_scores(cfg, S)
    want_idx = np.full((cfg.batch, cfg.n_frames, kmax), -1, np.int64)
    for b in range(cfg.batch):
        for f, r in enumerate(sel[b % cfg.n_scored].retained):
            want_idx[b, f, :len(r)] = r
    np.testing.assert_array_equal(got["keep_idx"].reshape(want_idx.shape), want_idx)
    np.testing.assert_array_equal(got["keep_cnt"].reshape(cfg.batch, cfg.n_frames),
                                  (want_idx >= 0).sum(axis=2))
    np.testing.assert_array_equal(got["pack_pos"], pm.pack_pos)
    np.testing.assert_array_equal(got["cu_seqlens"], pm.cu_seqlens)
    np.testing.assert_array_equal(got["gather"][:pm.cu_seqlens[-1]], pm.gather)
    return pm


def _run_schedule_against_oracle(cfg, use_graph, dense_check_at=(0,), in_place=False):
    from paper_2609_38984_amd import swam
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    stream = torch.cuda.Stream() if use_graph else None
    with torch.cuda.stream(stream) if use_graph else torch.cuda.device(0):
        ctx = swam.Context(cfg, stream=stream) if use_graph else swam.Context(cfg)
        pm = None
        for tau in range(cfg.n_steps):
            x = dev(inp.x(tau), torch.bfloat16)
            x_in = x.clone()
            y = x if in_place else torch.empty_like(x)
            t = dev(inp.temb(tau))
            if use_graph:
                kind = ctx.step_graph(model, x, t, tau, y)
                ctx.step_graph(model, x, t, tau, y)          # a second replay of the same graph
            else:
                kind = ctx.step(model, x, t, tau, y)
            torch.cuda.synchronize()
            xh = inp.x(tau)
            if kind == swam.KIND_REFRESH:
                pm = _check_selection_on_own_scores(cfg, _exported_selection(ctx, cfg), ctx.k_max)
                if tau in dense_check_at:
                    err = maxrel(host(y), O.dense_step(xh, blocks, inp.temb(tau), cfg))
                    print(f"  tau {tau} refresh: selection bit-exact, dense max-rel {err:.2e}", flush=True)
                    assert err < 2e-2
                else:
                    print(f"  tau {tau} refresh: selection bit-exact", flush=True)
            else:
                assert kind == swam.KIND_SPARSE and pm is not None
                ref = O.sparse_step(xh, blocks, inp.temb(tau), cfg, pm)
                err = maxrel(host(y), ref)
                pruned = pm.pack_pos < 0
                yb = y.view(torch.int16).cpu().numpy()
                xb = x_in.view(torch.int16).cpu().numpy()
                print(f"  tau {tau} sparse ({int(pm.cu_seqlens[-1])} rows): max-rel {err:.2e}", flush=True)
                assert err < 2e-2
                assert np.array_equal(yb[pruned], xb[pruned])


def test_bf16_8block_schedule_matches_oracle():
    cfg = W.preset(2)
    print(f"schedule {cfg.name}: {cfg.n_steps} steps, R = {cfg.reuse_R}", flush=True)
    _run_schedule_against_oracle(cfg, use_graph=False)


@pytest.mark.parametrize("in_place", [False, True])
@pytest.mark.parametrize("batch", [1, 2])
def test_bf16_one_block_schedule_matches_oracle(batch, in_place):
    # one block: the sparse step's gather-pack (first LayerNorm) and its
    # scatter back (the MLP down projection's store) are in the same block;
    # in place the scatter writes into the latent the pack read from, and with
    # two sequences the scattered rows cross a sequence boundary
    cfg = W.preset(2).replace(n_blocks=1, batch=batch, n_steps=4)
    print(f"one-block schedule {cfg.name}: batch {batch}, in place {in_place}", flush=True)
    _run_schedule_against_oracle(cfg, use_graph=False, in_place=in_place)


def test_bf16_graph_schedule_matches_oracle():
    cfg = W.preset(2).replace(n_steps=4)
    print(f"graph schedule {cfg.name}: {cfg.n_steps} steps", flush=True)
    _run_schedule_against_oracle(cfg, use_graph=True, dense_check_at=())


def test_fp32_graph_schedule_matches_oracle():
    from paper_2609_38984_amd import swam
    cfg = W.preset(1).replace(n_steps=6)
    print(f"graph schedule {cfg.name}", flush=True)
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ys, _ = O.run_schedule(cfg, blocks, inp.x, inp.temb)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        ctx = swam.Context(cfg, stream=stream)
        xs = [dev(inp.x(t)) for t in range(cfg.n_steps)]
        tb = [dev(inp.temb(t)) for t in range(cfg.n_steps)]
        y = torch.empty_like(xs[0])
        for rep in range(2):
            for tau in range(cfg.n_steps):
                ctx.step_graph(model, xs[tau], tb[tau], tau, y)
                stream.synchronize()
                err = maxrel(host(y), ys[tau])
                assert err < 1e-4, (rep, tau, err)
