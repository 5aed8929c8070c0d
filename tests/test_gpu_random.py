"""GPU parity of the random-selection baseline (the component ablation's
random tokens at the same per-frame budget) against the oracle: the
Philox4x64-10 keys bit-exact, the selection and packing metadata bit-exact,
a sparse step on the random selection 1e-4 max-relative (fp32) with pruned
rows byte-identical."""
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


def _ctx(cfg):
    from paper_2609_38984_amd import swam
    return swam.Context(cfg)


@pytest.mark.parametrize("n,seed", [(1, 0), (3, 12345), (5, 2 ** 64 - 3)])
def test_random_keys_and_selection_bitexact(n, seed):
    cfg = W.preset(n)
    if cfg.mass_threshold > 0:
        cfg = cfg.replace(mass_threshold=0.0, k_core=100, k_anchor=20)
    print(f"random selection {cfg.name} seed {seed}", flush=True)
    ctx = _ctx(cfg)
    B, F, n_s = cfg.batch, cfg.n_frames, cfg.n_s
    ki = torch.empty(B * F * ctx.k_max, dtype=torch.int32, device="cuda:0")
    pp = torch.empty(B * cfg.l_full, dtype=torch.int32, device="cuda:0")
    ctx.select_random(seed, keep_idx=ki, pack_pos=pp)
    v = torch.empty(B * F * n_s, dtype=torch.float32, device="cuda:0")
    ctx.export(v=v)
    torch.cuda.synchronize()
    keys = O.random_keys(seed, B, F, n_s)
    np.testing.assert_array_equal(host(v).reshape(B, F, n_s), keys)
    got = ki.cpu().numpy().reshape(B, F, -1)
    retained = []
    for b in range(B):
        sel = O.random_selection(keys[b], cfg.k_ret)
        retained.append(sel.retained)
        for f in range(F):
            np.testing.assert_array_equal(got[b, f], sel.retained[f])
    pm = O.pack_map(O.keep_mask(cfg, retained), B)
    np.testing.assert_array_equal(pp.cpu().numpy(), pm.pack_pos)


def test_sparse_step_on_random_selection_matches_oracle():
    from paper_2609_38984_amd import swam
    cfg = W.preset(1)
    blocks, _, model = model_for(cfg)
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ctx = _ctx(cfg)
    x0 = dev(inp.x(0))
    y0 = torch.empty_like(x0)
    ctx.step(model, x0, dev(inp.temb(0)), 0, y0, swam.FORCE_DENSE)
    ctx.select_random(7)
    keys = O.random_keys(7, 1, cfg.n_frames, cfg.n_s)
    pm = O.pack_map(O.keep_mask(cfg, [O.random_selection(keys[0], cfg.k_ret).retained]), 1)
    x1 = dev(inp.x(1))
    y1 = torch.empty_like(x1)
    assert ctx.step(model, x1, dev(inp.temb(1)), 1, y1) == swam.KIND_SPARSE
    torch.cuda.synchronize()
    want = O.sparse_step(inp.x(1), blocks, inp.temb(1), cfg, pm)
    err = maxrel(host(y1), want)
    print(f"  sparse step on the random selection: max-rel {err:.2e}", flush=True)
    assert err < 1e-4
    pruned = pm.pack_pos < 0
    assert y1.cpu().numpy()[pruned].tobytes() == x1.cpu().numpy()[pruned].tobytes()


def test_random_selection_with_guidance_pairs_is_shared_and_seeded():
    cfg = W.preset(1).replace(batch=4, cfg_pairs=1, guidance=3.0)
    ctx = _ctx(cfg)
    ki = torch.empty(cfg.batch * cfg.n_frames * ctx.k_max, dtype=torch.int32, device="cuda:0")
    ctx.select_random(99, keep_idx=ki)
    a = ki.cpu().numpy().reshape(cfg.batch, -1)
    np.testing.assert_array_equal(a[:2], a[2:])
    assert not np.array_equal(a[0], a[1])          # the two conditional sequences differ
    ctx.select_random(99, keep_idx=ki)
    np.testing.assert_array_equal(ki.cpu().numpy().reshape(cfg.batch, -1), a)
    ctx.select_random(100, keep_idx=ki)
    assert not np.array_equal(ki.cpu().numpy().reshape(cfg.batch, -1), a)


def test_random_selection_rejects_mass_threshold_mode():
    from paper_2609_38984_amd import swam
    ctx = _ctx(W.preset(5))
    with pytest.raises(swam.SwamError) as e:
        ctx.select_random(1)
    assert e.value.code == -7
