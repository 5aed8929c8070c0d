"""The seeded input generator: determinism, storage grid, shapes and budgets."""
import numpy as np
import torch

import workload as W


def test_budgets_of_the_workloads():
    assert (W.preset(1).k_core, W.preset(1).k_anchor) == (16, 4)
    assert (W.preset(2).k_core, W.preset(2).k_anchor) == (77, 16)
    assert (W.preset(3).k_core, W.preset(3).k_anchor) == (300, 64)
    for pct, want in ((10, (102, 64)), (25, (256, 64)), (50, (512, 64)), (100, (1024, 0))):
        c = W.preset(4, percent=pct)
        assert (c.k_core, c.k_anchor) == want
    assert W.preset(3).l_full == 10160 and W.preset(3).t_pack_fixed == 3472
    assert W.preset(4, percent=25).t_pack_fixed == 6208
    assert W.preset(5).mass_threshold == 0.8 and W.preset(5).k_anchor == 0


def test_inputs_deterministic_and_on_storage_grid():
    cfg = W.preset(2).replace(n_blocks=1)
    a = W.make_inputs(cfg)
    b = W.make_inputs(cfg)
    x0, x0b = a.x(0), b.x(0)
    assert x0.shape == (cfg.l_full, cfg.d_model) and x0.dtype == np.float32
    assert x0.tobytes() == x0b.tobytes()
    t = torch.from_numpy(x0)
    assert torch.equal(t.to(torch.bfloat16).float(), t)
    w = W.block_weights(cfg, 0)
    assert w["w_qkv"].shape == (3 * cfg.d_model, cfg.d_model)
    assert torch.equal(torch.from_numpy(w["w_2"]).to(torch.bfloat16).float(), torch.from_numpy(w["w_2"]))
    # the blob drifts: future rows change between steps, context and action rows do not
    x1 = a.x(1)
    fut = slice(cfg.n_ctx, cfg.n_ctx + cfg.n_fut)
    assert not np.array_equal(x0[fut], x1[fut])
    np.testing.assert_array_equal(x0[:cfg.n_ctx], x1[:cfg.n_ctx])
    np.testing.assert_array_equal(x0[cfg.n_ctx + cfg.n_fut:], x1[cfg.n_ctx + cfg.n_fut:])


def test_ragged_workload_draws_blob_counts_and_widths():
    cfg = W.preset(5).replace(d_model=64, n_heads=1)
    inp = W.make_inputs(cfg)
    counts = [len(bl) for bl in inp.blobs]
    assert len(counts) == 8 and min(counts) >= 1 and max(counts) <= 4
    sig = [b.sigma for bl in inp.blobs for b in bl]
    assert all(2.0 <= s <= 6.0 for s in sig)
    assert inp.x(0).shape == (8 * cfg.l_full, 64)


def test_timestep_embedding():
    cfg = W.preset(1)
    e = W.timestep_embedding(cfg, 0)
    assert e.shape == (128,)
    assert e[0] == np.float32(np.cos(1000.0)) and e[64] == np.float32(np.sin(1000.0))


def test_multi_view_frames_concatenate_unequal_views():
    for n, views, n_s in ((6, ((14, 14), (8, 9), (8, 9)), 340), (7, ((7, 7), (7, 7)), 98)):
        cfg = W.preset(n)
        assert cfg.views == views and cfg.n_s == n_s and (cfg.frame_h, cfg.frame_w) == (1, n_s)
        grids = W.view_grids(cfg)
        assert [g[0] for g in grids] == list(np.cumsum([0] + [h * w for h, w in views])[:-1])


def test_multi_view_blobs_stay_inside_their_view():
    cfg = W.preset(6).replace(n_blocks=1, d_model=128, n_heads=2)
    inp = W.make_inputs(cfg)
    grids = W.view_grids(cfg)
    for b in range(cfg.batch):
        base = inp.base[b][cfg.n_ctx:cfg.n_ctx + cfg.n_fut].reshape(cfg.n_frames, cfg.n_s, -1)
        got = inp.x(0)[b * cfg.l_full + cfg.n_ctx:b * cfg.l_full + cfg.n_ctx + cfg.n_fut]
        moved = np.abs(got.reshape(cfg.n_frames, cfg.n_s, -1) - W._storage(cfg, base)).max(axis=2) > 0
        views = {bl.view for bl in inp.blobs[b]}
        for v, (off, h, w) in enumerate(grids):
            if v not in views:
                assert not moved[:, off:off + h * w].any()
        assert moved.any()
