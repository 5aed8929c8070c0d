"""Pins of the backbone variants (rotary embedding at original positions,
QK-norm) in the oracle -- CPU only."""
import numpy as np

import oracle as O
import workload as W


def test_rope_closed_form_single_pair_and_identity_at_zero():
    x = np.array([[1.0, 0.0], [0.0, 1.0], [2.0, 3.0]])
    pos = np.array([0.0, 0.7, 2.5])
    y = O.apply_rope(x, pos, 1)          # head dim 2: one pair, angle = pos
    np.testing.assert_allclose(y[0], [1.0, 0.0], atol=1e-15)
    np.testing.assert_allclose(y[1], [-np.sin(0.7), np.cos(0.7)], atol=1e-15)
    c, s = np.cos(2.5), np.sin(2.5)
    np.testing.assert_allclose(y[2], [2 * c - 3 * s, 2 * s + 3 * c], atol=1e-14)


def test_rope_is_a_rotation_with_relative_position_logits():
    rng = np.random.default_rng(0)
    a, b = rng.standard_normal((1, 128)), rng.standard_normal((1, 128))
    ra = O.apply_rope(a, [37], 2)
    np.testing.assert_allclose(np.linalg.norm(ra[0, :64]), np.linalg.norm(a[0, :64]), rtol=1e-13)
    for m, n, sft in ((5, 9, 100), (300, 2, 1234), (0, 0, 17)):
        d0 = (O.apply_rope(a, [m], 2) * O.apply_rope(b, [n], 2))[0, :64].sum()
        d1 = (O.apply_rope(a, [m + sft], 2) * O.apply_rope(b, [n + sft], 2))[0, :64].sum()
        assert abs(d0 - d1) < 1e-10


def test_qk_norm_gives_unit_rms_heads():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 192)) * 3
    y = O.qk_rms_norm(x, 3).reshape(5, 3, 64)
    np.testing.assert_allclose((y * y).mean(axis=2), 1.0, rtol=1e-5)


def _variant_cfg(**kw):
    return W.preset(1).replace(rope=1, qk_norm=1, **kw)


def test_packed_rows_keep_their_original_positions():
    # the retained rows' q and k in the packed run equal those of the dense run
    cfg = _variant_cfg()
    blocks = [W.block_weights(cfg, l) for l in range(cfg.n_blocks)]
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    x = inp.x(0)
    r = O.refresh_step(x, blocks, inp.temb(0), cfg)
    pm = r.packmap
    _, tr_dense = O.block(x, blocks[0], inp.temb(1), O.dense_cu(cfg), cfg.n_heads, cfg.dtype,
                          O.dense_positions(cfg), True, True)
    xp = O.pack(x, pm)
    _, tr_pack = O.block(xp, blocks[0], inp.temb(1), pm.cu_seqlens, cfg.n_heads, cfg.dtype,
                         pm.gather % cfg.l_full, True, True)
    d = cfg.d_model
    np.testing.assert_array_equal(tr_pack.qkv[:, :2 * d], tr_dense.qkv[pm.gather, :2 * d])
    # numbering the packed rows 0..T-1 instead would rotate them differently
    _, tr_wrong = O.block(xp, blocks[0], inp.temb(1), pm.cu_seqlens, cfg.n_heads, cfg.dtype,
                          np.arange(len(pm.gather)), True, True)
    assert not np.array_equal(tr_wrong.qkv[:, :2 * d], tr_dense.qkv[pm.gather, :2 * d])


def test_full_retention_with_variants_equals_dense_step():
    cfg = _variant_cfg(k_core=64, k_anchor=0)
    blocks = [W.block_weights(cfg, l) for l in range(cfg.n_blocks)]
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    r = O.refresh_step(inp.x(0), blocks, inp.temb(0), cfg)
    y_sparse = O.sparse_step(inp.x(1), blocks, inp.temb(1), cfg, r.packmap)
    y_dense = O.dense_step(inp.x(1), blocks, inp.temb(1), cfg)
    np.testing.assert_array_equal(y_sparse, y_dense)


def test_block_rows_matches_block_with_variants():
    cfg = W.preset(2).replace(rope=1, qk_norm=1, n_blocks=1)
    w = W.block_weights(cfg, 0)
    inp = W.make_inputs(cfg, w["w_qkv"])
    x = inp.x(0)
    pos = O.dense_positions(cfg)
    y, tr = O.block(x, w, inp.temb(0), O.dense_cu(cfg), cfg.n_heads, cfg.dtype, pos, True, True)
    rows = np.array([0, 5, 300, 1311])
    yr, lr = O.block_rows(x, w, inp.temb(0), O.dense_cu(cfg), rows, cfg.n_heads, cfg.dtype, pos,
                          True, True)
    np.testing.assert_array_equal(yr, y[rows])
    np.testing.assert_array_equal(lr, tr.lse[rows])
