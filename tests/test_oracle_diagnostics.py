"""Pins of the overlap diagnostic (App. C attention-overlap eq.), the
selection variants (core-only, anchor-only) and refresh schedules beyond a
fixed interval (App. C.2) -- CPU only."""
import dataclasses

import numpy as np
import pytest

import oracle as O
import workload as W


def test_overlap_closed_forms():
    rng = np.random.default_rng(0)
    P = rng.random(50)
    assert O.overlap(P, P) == pytest.approx(1.0, abs=1e-15)
    assert O.overlap(P, 3.5 * P) == pytest.approx(1.0, abs=1e-15)       # scale invariant
    Q = rng.random(50)
    assert O.overlap(P, Q) == pytest.approx(O.overlap(Q, P), abs=1e-15)  # symmetric
    a, b = np.zeros(50), np.zeros(50)
    a[:20], b[30:] = 1.0, 1.0
    assert O.overlap(a, b) == 0.0                                          # disjoint supports
    # uniform on A vs uniform on B: |A and B| * min(1/|A|, 1/|B|)
    a[:] = 0
    b[:] = 0
    a[0:20] = 1.0
    b[10:40] = 1.0
    assert O.overlap(a, b) == pytest.approx(10 / 30, abs=1e-15)
    assert O.overlap(np.zeros(5), np.ones(5)) == 0.0


def test_overlap_brute_force_formula():
    rng = np.random.default_rng(1)
    P, Q = rng.random(17), rng.random(17)
    want = sum(min(p / P.sum(), q / Q.sum()) for p, q in zip(P, Q))
    assert O.overlap(P, Q) == pytest.approx(want, abs=1e-14)


def test_anchor_only_selection_is_topk_of_anchor_key():
    # K_c = 0: no cores, E is every position, each frame keeps the same top-K_s of A
    rng = np.random.default_rng(2)
    V = rng.random((3, 40)).astype(np.float32)
    A = rng.random(40).astype(np.float32)
    sel = O.select(V, A, k_core=0, k_anchor=7)
    want = np.sort(np.argsort(-A.astype(np.float64), kind="stable")[:7])
    for f in range(3):
        np.testing.assert_array_equal(sel.retained[f], want)


def test_core_only_selection_is_per_frame_topk():
    # K_s = 0: the pool is every position and each frame keeps its own top-K_c of V
    rng = np.random.default_rng(3)
    V = rng.random((3, 40)).astype(np.float32)
    A = rng.random(40).astype(np.float32)
    sel = O.select(V, A, k_core=9, k_anchor=0)
    for f in range(3):
        want = np.sort(np.argsort(-V[f].astype(np.float64), kind="stable")[:9])
        np.testing.assert_array_equal(sel.retained[f], want)


def test_initial_only_schedule_reuses_the_first_selection():
    cfg = W.preset(1)
    blocks = [W.block_weights(cfg, l) for l in range(cfg.n_blocks)]
    inp = W.make_inputs(cfg, blocks[0]["w_qkv"])
    ys, refr = O.run_schedule(cfg, blocks, inp.x, inp.temb, n_steps=4, refresh_at={0})
    assert list(refr) == [0]
    pm = refr[0].packmap
    for tau in (1, 2, 3):
        want = O.sparse_step(inp.x(tau), blocks, inp.temb(tau), cfg, pm)
        np.testing.assert_array_equal(ys[tau], want)
    # the default interval schedule is the refresh_at set {tau : tau mod R == 0}
    ys2, refr2 = O.run_schedule(cfg, blocks, inp.x, inp.temb, n_steps=4, refresh_at={0, 2})
    ys3, refr3 = O.run_schedule(cfg, blocks, inp.x, inp.temb, n_steps=4)
    assert list(refr2) == list(refr3) == [0, 2]
    for a, b in zip(ys2, ys3):
        np.testing.assert_array_equal(a, b)
