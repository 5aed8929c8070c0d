"""On-stream launch timers: every launch of an enabled class bracketed once and
tagged with the kind of the step that enqueued it; a stride brackets every
stride-th launch of a class (ordinals counted from the last enable / reset),
so a timed loop pays for fewer event pairs.  Counts are exact; durations are
checked only for being positive and for the per-kind sums adding up."""
import pytest
import torch

import workload as W
from helpers import dev, model_for

pytestmark = pytest.mark.gpu

# 4 blocks, R = 2: steps 0, 2, 4 refresh, 1, 3, 5 sparse
CFG = W.preset(1).replace(n_blocks=4, n_steps=6)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _run(ctx, model, inp, steps, flags=0):
    kinds = []
    for tau in range(steps):
        x = dev(inp.x(tau))
        y = torch.empty_like(x)
        kinds.append(ctx.step(model, x, dev(inp.temb(tau)), tau, y, flags))
    torch.cuda.synchronize()
    return kinds


def test_timer_counts_by_kind_and_stride():
    from paper_2609_38984_amd import swam
    cfg = CFG
    blocks, dblocks, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ctx = swam.Context(cfg)
    L = cfg.n_blocks
    ctx.timer_enable(["ATTN", "PACK", "SCORE"], capacity=256)
    kinds = _run(ctx, model, inp, cfg.n_steps)
    n_ref, n_sp = kinds.count(swam.KIND_REFRESH), kinds.count(swam.KIND_SPARSE)
    print(f"kinds {kinds}", flush=True)
    assert (n_ref, n_sp) == (3, 3)
    want = {swam.KIND_REFRESH: L * n_ref, swam.KIND_SPARSE: L * n_sp, swam.KIND_DENSE: 0,
            swam.KIND_NONE: 0}
    tot_ms = 0.0
    for kind, n in want.items():
        got, ms = ctx.timer_read("ATTN", kind)
        assert got == n, (kind, got, n)
        assert (ms > 0) == (n > 0)
        tot_ms += ms
    n_any, ms_any = ctx.timer_read("ATTN")
    assert n_any == L * cfg.n_steps
    assert abs(ms_any - tot_ms) <= 1e-9 * max(ms_any, 1.0)
    # the pack runs once per sparse step, the scoring once per layer of a refresh
    assert ctx.timer_read("PACK", swam.KIND_SPARSE)[0] == n_sp
    assert ctx.timer_read("PACK", swam.KIND_REFRESH)[0] == 0
    assert ctx.timer_read("SCORE", swam.KIND_REFRESH)[0] == L * n_ref
    assert ctx.timer_read("SCORE", swam.KIND_SPARSE)[0] == 0

    # stride 2 over 4 launches per step: launches 0 and 2 of every step
    ctx.timer_stride(2)
    assert ctx.timer_read("ATTN")[0] == 0                    # the stride drops old brackets
    _run(ctx, model, inp, cfg.n_steps)
    assert ctx.timer_read("ATTN", swam.KIND_REFRESH)[0] == 2 * n_ref
    assert ctx.timer_read("ATTN", swam.KIND_SPARSE)[0] == 2 * n_sp
    assert ctx.timer_read("PACK", swam.KIND_SPARSE)[0] == 2   # ordinals 0 and 2 of 3
    # stride 3 over 4 per step: ordinals 0, 3, ..., 21 of 24 launches
    ctx.timer_stride(3)
    _run(ctx, model, inp, cfg.n_steps)
    assert ctx.timer_read("ATTN")[0] == 8
    # launches outside a step are tagged as such
    ctx.timer_stride(1)
    x = dev(inp.x(0))
    cu = torch.tensor([0, cfg.l_full], dtype=torch.int32, device="cuda:0")
    ctx.block(dblocks[0], dev(inp.temb(0)), x, cfg.l_full, cu, 1)
    assert ctx.timer_read("ATTN", swam.KIND_NONE)[0] == 1
    assert ctx.timer_read("ATTN")[0] == 1
    # a forced dense step
    ctx.timer_reset()
    _run(ctx, model, inp, 1, swam.FORCE_DENSE)
    assert ctx.timer_read("ATTN", swam.KIND_DENSE)[0] == L
    with pytest.raises(swam.SwamError):
        ctx.timer_stride(0)
    with pytest.raises(swam.SwamError):
        ctx.timer_read("ATTN", 7)


def test_captured_steps_are_not_bracketed():
    """Launches recorded into a HIP graph (and its replays) take no event
    brackets; an eager step on the same context still does."""
    from paper_2609_38984_amd import swam
    cfg = CFG
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        ctx = swam.Context(cfg, stream=stream)
        ctx.timer_enable(["ATTN"], capacity=64)
        x = dev(inp.x(0))
        y = torch.empty_like(x)
        temb = dev(inp.temb(0))
        for tau in range(4):                 # refresh and sparse captured, then replayed
            ctx.step_graph(model, x, temb, tau, y)
        stream.synchronize()
        assert ctx.timer_read("ATTN")[0] == 0
        ctx.step(model, x, temb, 0, y)
        stream.synchronize()
        assert ctx.timer_read("ATTN", swam.KIND_REFRESH)[0] == cfg.n_blocks
