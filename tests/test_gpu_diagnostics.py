"""GPU parity of the diagnostics and selection/schedule variants against the
oracle: the overlap measure (App. C), anchor-only and core-only selections
(bit-exact on the oracle's fp32 V and A), and refresh schedules other than
a fixed interval (the paper's default of a single full step per chunk, and
an explicit step set through SWAM_STEP_FORCE_REFRESH).

Tolerances: overlap 1e-6 relative (float64 sums on both sides, fp32 result);
selections bit-exact; fp32 step outputs 1e-4 max-relative.
"""
import numpy as np
import pytest
import torch

import oracle as O
import workload as W
from helpers import dev, host, maxrel, model_for
from test_gpu_parity import _select_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def test_overlap_matches_oracle():
    from paper_2609_38984_amd import swam
    print("overlap", flush=True)
    cfg = W.preset(3)
    ctx = swam.Context(cfg)
    rng = np.random.default_rng(5)
    n_maps, n = 19, 1200
    p = rng.random((n_maps, n)).astype(np.float32) ** 4
    q = rng.random((n_maps, n)).astype(np.float32) ** 4
    p[3] = 0.0                                   # a map of zero mass
    q[7] = p[7]                                  # identical maps
    q[8, :600], p[8, 600:] = 0.0, 0.0            # disjoint supports
    out = torch.empty(n_maps, dtype=torch.float32, device="cuda:0")
    ctx.overlap(dev(p), dev(q), out)
    got = host(out)
    want = np.array([O.overlap(p[m], q[m]) for m in range(n_maps)])
    np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-7)
    assert got[3] == 0.0 and got[8] == 0.0 and abs(got[7] - 1.0) < 1e-6


def test_select_anchor_only_bitexact():
    print("select anchor only", flush=True)
    _select_case(W.preset(2).replace(n_blocks=2, k_core=0, k_anchor=40), 91)


def test_select_core_only_bitexact():
    print("select core only", flush=True)
    _select_case(W.preset(2).replace(n_blocks=2, k_anchor=0), 92)


@pytest.mark.parametrize("refresh_at", [(0,), (0, 3)], ids=["initial-only", "steps-0-3"])
def test_schedule_as_step_set_matches_oracle(refresh_at):
    from paper_2609_38984_amd import swam
    print(f"schedule refresh_at={refresh_at}", flush=True)
    cfg = W.preset(1).replace(reuse_R=100)        # no automatic refresh after tau = 0
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    n = 5
    ys, refr = O.run_schedule(cfg, blocks, inp.x, inp.temb, n_steps=n, refresh_at=set(refresh_at))
    ctx = swam.Context(cfg)
    for tau in range(n):
        x = dev(inp.x(tau))
        y = torch.empty_like(x)
        flags = swam.FORCE_REFRESH if tau in refresh_at else 0
        kind = ctx.step(model, x, dev(inp.temb(tau)), tau, y, flags)
        torch.cuda.synchronize()
        assert kind == (swam.KIND_REFRESH if tau in refresh_at else swam.KIND_SPARSE)
        assert maxrel(host(y), ys[tau]) < 1e-4
