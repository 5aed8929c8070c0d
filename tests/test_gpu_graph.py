"""Graph-captured steps replay exactly what the eager steps compute.

Each schedule is run eagerly in one context and through swam_step_graph in
another (on a non-default stream); every replay -- with eager work and
synchronisations in between -- must match the eager output byte for byte.
A context moved between two streams step by step (swam_set_stream, no host
synchronisation) must match a one-stream run the same way.
"""
import numpy as np
import pytest
import torch

import workload as W
from helpers import act_dtype, dev, model_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _small(**kw):
    base = dict(name="bf16-graph", batch=2, d_model=256, n_heads=4, n_blocks=3, n_ctx=20,
                n_frames=2, frame_h=8, frame_w=9, n_act=8, k_core=18, k_anchor=6, reuse_R=2,
                n_steps=6, dtype="bf16", seed=11, blob_sigma=1.5)
    base.update(kw)
    return W.SwamConfig(**base)


# "guided" records the partner copies of the selection (device-to-device copy
# nodes); "rope_qknorm" the QKV projection with its fused rotary / norm store
@pytest.mark.parametrize("cfg", [_small(), _small(mass_threshold=0.8, k_core=72, k_anchor=0),
                                 W.preset(1).replace(n_steps=6),
                                 _small(cfg_pairs=1, guidance=3.0),
                                 _small(rope=1, qk_norm=1)],
                         ids=["fixed", "mass", "fp32", "guided", "rope_qknorm"])
def test_graph_replays_match_eager(cfg):
    from paper_2609_38984_amd import swam
    print(f"graph case {cfg.name} mass={cfg.mass_threshold}", flush=True)
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    dt = act_dtype(cfg)
    xs = [dev(inp.x(t), dt) for t in range(cfg.n_steps)]
    tb = [dev(inp.temb(t)) for t in range(cfg.n_steps)]
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        eager = swam.Context(cfg, stream=stream)
        graph = swam.Context(cfg, stream=stream)
        ye = torch.empty_like(xs[0])
        yg = torch.empty_like(xs[0])
        for rep in range(3):                       # the same graphs replay on every pass
            for tau in range(cfg.n_steps):
                ke = eager.step(model, xs[tau], tb[tau], tau, ye)
                kg = graph.step_graph(model, xs[tau], tb[tau], tau, yg)
                stream.synchronize()
                assert ke == kg
                assert torch.equal(yg.view(torch.int16 if dt == torch.bfloat16 else torch.int32),
                                   ye.view(torch.int16 if dt == torch.bfloat16 else torch.int32)), \
                    (rep, tau)
                scratch = torch.randn(1 << 16, device="cuda:0") * 2.0   # eager work in between
                del scratch
        graph.graph_clear()
        kg = graph.step_graph(model, xs[1], tb[1], 1, yg)
        eager.step(model, xs[1], tb[1], 1, ye)
        stream.synchronize()
        assert torch.equal(yg, ye)


def test_graph_needs_non_default_stream():
    from paper_2609_38984_amd import swam
    cfg = W.preset(1)
    _, _, model = model_for(cfg)
    ctx = swam.Context(cfg, stream=torch.cuda.default_stream())
    x = torch.zeros(cfg.l_full, cfg.d_model, device="cuda:0")
    with pytest.raises(swam.SwamError) as e:
        ctx.step_graph(model, x, torch.zeros(cfg.d_temb, device="cuda:0"), 0, torch.empty_like(x))
    assert e.value.code == -4


def test_stream_switch_orders_after_queued_work():
    """swam_set_stream between the steps of a schedule, with no host
    synchronisation: every sparse step on the second stream reads the
    selection the refresh on the first stream wrote, and the outputs equal a
    one-stream run byte for byte."""
    from paper_2609_38984_amd import swam
    cfg = _small()
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    dt = act_dtype(cfg)
    xs = [dev(inp.x(t), dt) for t in range(cfg.n_steps)]
    ts = [dev(inp.temb(t)) for t in range(cfg.n_steps)]
    ref = [torch.empty_like(x) for x in xs]
    got = [torch.empty_like(x) for x in xs]
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    one = swam.Context(cfg, stream=s1)
    for t in range(cfg.n_steps):
        one.step(model, xs[t], ts[t], t, ref[t])
    two = swam.Context(cfg, stream=s1)
    kinds = []
    for t in range(cfg.n_steps):
        two.set_stream(s1 if t % 2 == 0 else s2)
        kinds.append(two.step(model, xs[t], ts[t], t, got[t]))
    torch.cuda.synchronize()
    print(f"step kinds {kinds}", flush=True)
    assert swam.KIND_SPARSE in kinds
    for t in range(cfg.n_steps):
        assert torch.equal(got[t].view(torch.int16), ref[t].view(torch.int16)), t
