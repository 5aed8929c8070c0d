"""Pins of the CPU oracle: paper-printed constants, closed forms, invariants the
paper states, library routines and brute force on tiny inputs.

Each test names the pin it provides; a plausible mistake in the oracle (a
dropped term, a wrong sign or index, a transposed operand, a wrong normaliser)
fails at least one of them.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import torch

import oracle as O
import workload as W


# ---------------------------------------------------------------------------
# paper-printed constants
# ---------------------------------------------------------------------------
def test_alpha_printed_values(golden):
    a4 = golden["alpha_g4"]
    want = np.array(a4["numerators"], float) / a4["denominator"]
    np.testing.assert_allclose(O.alpha_weights(4), want, rtol=0, atol=1e-15)
    a16 = golden["alpha_g16"]
    w = O.alpha_weights(16)
    central = Fraction(*a16["central"])
    outer = Fraction(*a16["outer"])
    vals = sorted(Fraction(x).limit_denominator(1000) for x in w)
    assert vals.count(central) == a16["n_central"]
    assert vals.count(outer) == a16["n_outer"]


@pytest.mark.parametrize("g", list(range(1, 65)))
def test_alpha_nonnegative_sums_to_one_centre_double(g):
    w = O.alpha_weights(g)
    assert (w > 0).all()
    assert abs(w.sum() - 1.0) < 1e-14
    assert np.allclose(w, w[::-1])                       # symmetric about the centre
    assert w.max() / w.min() in (1.0, 2.0)
    if g >= 4:
        assert w[g // 2] == pytest.approx(2 * w[0])      # centre twice the outer quarter


def test_groups_printed(golden):
    for case in golden["groups"]["cases"]:
        groups = O.frame_groups(case["H"], case["F"])
        assert len(groups) == case["F"]
        assert all(len(I) == case["group_size"] for I in groups)
        flat = [i for I in groups for i in I]
        assert flat == list(range(case["H"]))           # consecutive, disjoint, covering
    with pytest.raises(ValueError):
        O.frame_groups(30, 8)


def test_printed_budgets_give_fixed_length(golden):
    """K_c + K_s tokens per frame at the printed budgets, every frame."""
    rng = np.random.default_rng(5)
    for case in golden["budgets"]["cases"]:
        assert case["K_c"] + case["K_s"] == case["retained"]
        V = rng.random((4, case["N_s"])).astype(np.float32)
        A = rng.random(case["N_s"]).astype(np.float32)
        sel = O.select(V, A, case["K_c"], case["K_s"])
        assert all(len(r) == case["retained"] for r in sel.retained)


def test_pruning_ratio_printed(golden):
    """r = 1 - K_ret/N_s: exactly one integer budget reproduces each printed ratio."""
    pr = golden["pruning_ratio"]
    n_s = pr["N_s"]
    for pct in pr["printed_percent"]:
        hits = [k for k in range(n_s + 1) if round(100 * (1 - k / n_s), 2) == pct]
        assert len(hits) == 1
    assert {256, 112} == {k for k in range(n_s + 1)
                          if round(100 * (1 - k / n_s), 2) in pr["printed_percent"]}


# ---------------------------------------------------------------------------
# attention normaliser and scores
# ---------------------------------------------------------------------------
def _rand_qkv(rng, T, n_heads, hd=64, scale=1.0):
    return [rng.standard_normal((T, n_heads * hd)) * scale for _ in range(3)]


def test_attention_rows_sum_to_one_and_match_library():
    """Sum over all visible keys of exp(x - lambda) is 1 (P-1); output and lambda
    equal torch softmax attention and scipy logsumexp."""
    rng = np.random.default_rng(0)
    T, nh, hd = 37, 3, 64
    q, k, v = _rand_qkv(rng, T, nh, hd, 1.5)
    cu = np.array([0, 20, 37])
    o, lse = O.attention(q, k, v, cu, nh)
    for b in range(2):
        s0, s1 = cu[b], cu[b + 1]
        for h in range(nh):
            c = slice(h * hd, (h + 1) * hd)
            x = q[s0:s1, c] @ k[s0:s1, c].T / 8.0
            np.testing.assert_allclose(np.exp(x - lse[s0:s1, h][:, None]).sum(1), 1.0, atol=1e-12)
            np.testing.assert_allclose(lse[s0:s1, h], scipy.special.logsumexp(x, axis=1), rtol=1e-13)
            tq = torch.tensor(q[s0:s1, c]).view(1, 1, s1 - s0, hd)
            tk = torch.tensor(k[s0:s1, c]).view(1, 1, s1 - s0, hd)
            tv = torch.tensor(v[s0:s1, c]).view(1, 1, s1 - s0, hd)
            ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)
            np.testing.assert_allclose(o[s0:s1, c], ref[0, 0].numpy(), rtol=1e-11, atol=1e-12)


def _score_via_full_attention(q_act, k_all, n_ctx, F, n_s, nh, alpha):
    """E1 then E2: head-mean of the full attention matrix, weighted per group."""
    H = q_act.shape[0]
    hd = q_act.shape[1] // nh
    g = H // F
    U = np.zeros((H, k_all.shape[0]))
    for h in range(nh):
        c = slice(h * hd, (h + 1) * hd)
        logits = torch.tensor(q_act[:, c] @ k_all[:, c].T / math.sqrt(hd))
        U += torch.softmax(logits, dim=1).numpy()
    U /= nh
    S = np.zeros((F, n_s))
    for f in range(F):
        for a in range(g):
            i = f * g + a
            S[f] += alpha[a] * U[i, n_ctx + f * n_s: n_ctx + (f + 1) * n_s]
    return S


@pytest.mark.parametrize("F,g,nh", [(2, 4, 2), (3, 6, 1), (4, 8, 3)])
def test_score_equals_head_mean_attention(F, g, nh):
    """The reused-normaliser scorer equals E2 applied to E1 built from the full
    softmax matrix (normalised over all visible keys)."""
    rng = np.random.default_rng(F * 100 + g)
    n_ctx, n_s, H, hd = 5, 12, F * g, 64
    L = n_ctx + F * n_s + H
    k_all = rng.standard_normal((L, nh * hd)) * 1.3
    q_act = rng.standard_normal((H, nh * hd)) * 1.3
    lam = np.stack([scipy.special.logsumexp(
        q_act[:, h * hd:(h + 1) * hd] @ k_all[:, h * hd:(h + 1) * hd].T / 8.0, axis=1)
        for h in range(nh)], axis=1)
    S = O.score(q_act, k_all[n_ctx:n_ctx + F * n_s], lam, F, n_s, nh)
    ref = _score_via_full_attention(q_act, k_all, n_ctx, F, n_s, nh, O.alpha_weights(g))
    np.testing.assert_allclose(S, ref, rtol=2e-7, atol=1e-12)
    # attention mass on a frame never exceeds one (P-2)
    assert (S >= 0).all() and (S.sum(axis=1) <= 1 + 1e-6).all()
    # mode B: lambda over all keys equals the library logsumexp
    np.testing.assert_allclose(O.lse_all_keys(q_act, k_all, nh), lam, rtol=1e-7)


def test_score_hand_example():
    """One head, two queries, logits chosen by hand: S = sum_i alpha_i e^{x - lambda_i}."""
    hd = 64
    q = np.zeros((2, hd)); q[0, 0] = 8.0; q[1, 0] = 16.0      # logits x = c_j and 2 c_j
    k = np.zeros((3, hd)); k[:, 0] = [0.0, 1.0, -1.0]
    lam = np.array([[0.5], [1.5]])
    S = O.score(q, k, lam, 1, 3, 1)
    c = np.array([0.0, 1.0, -1.0])
    want = 0.5 * np.exp(c - 0.5) + 0.5 * np.exp(2 * c - 1.5)  # g = 2: both outer, 1/2 each
    np.testing.assert_allclose(S[0], want, rtol=1e-7)


def test_uniform_attention_closed_form():
    """Zero queries: every logit is 0, so S = 1/L_full, R = N_s/L_full, E = 1,
    Q = 0 and the zero-weight fallback gives V = A = 1/L_full (P-3)."""
    rng = np.random.default_rng(1)
    n_ctx, F, n_s, H, nh = 6, 2, 16, 8, 2
    L = n_ctx + F * n_s + H
    k_all = rng.standard_normal((L, nh * 64))
    q_act = np.zeros((H, nh * 64))
    lam = O.lse_all_keys(q_act, k_all, nh)
    np.testing.assert_allclose(lam, math.log(L), rtol=1e-7)
    S = O.score(q_act, k_all[n_ctx:n_ctx + F * n_s], lam, F, n_s, nh)
    np.testing.assert_allclose(S, 1.0 / L, rtol=1e-6)
    S_all = np.stack([S, S, S])
    R, E, Q = O.layer_quality(S_all)
    np.testing.assert_allclose(R, n_s / L, rtol=1e-6)
    np.testing.assert_allclose(E, 1.0, atol=1e-12)
    np.testing.assert_allclose(Q, 0.0, atol=1e-12)
    red = O.score_reduce(S_all, k_layer=2)
    np.testing.assert_allclose(red.V, 1.0 / L, rtol=1e-6)
    np.testing.assert_allclose(red.A, 1.0 / L, rtol=1e-6)


def test_block_zero_query_weights_give_log_L_normaliser():
    cfg = W.preset(1)
    w = W.block_weights(cfg, 0)
    d = cfg.d_model
    w["w_qkv"] = w["w_qkv"].copy(); w["b_qkv"] = w["b_qkv"].copy()
    w["w_qkv"][:d] = 0.0
    w["b_qkv"][:d] = 0.0
    x = W.make_inputs(cfg).x(0)
    _, tr = O.block(x, w, W.timestep_embedding(cfg, 0), O.dense_cu(cfg), cfg.n_heads, "f64")
    np.testing.assert_allclose(tr.lse, math.log(cfg.l_full), rtol=1e-7)


# ---------------------------------------------------------------------------
# layer quality, core score, anchors
# ---------------------------------------------------------------------------
def test_entropy_closed_forms():
    """One-hot frames: E = 0 and Q = R (P-4); two equal spots out of four: E = 1/2."""
    F, n_s = 3, 4
    S1 = np.zeros((1, F, n_s))
    S1[0, 0, 1] = 0.3; S1[0, 1, 3] = 0.6; S1[0, 2, 0] = 0.9
    R, E, Q = O.layer_quality(S1)
    assert R[0] == pytest.approx(1.8 / 3)
    assert E[0] == 0.0 and Q[0] == pytest.approx(R[0])
    S2 = np.zeros((1, 1, 4)); S2[0, 0, :2] = 0.25
    R, E, Q = O.layer_quality(S2)
    assert E[0] == pytest.approx(0.5, abs=1e-15)
    assert Q[0] == pytest.approx(0.5 * 0.5)
    # an all-zero frame contributes nothing (0 log 0 = 0, Sbar = 0)
    S3 = np.zeros((1, 2, 4)); S3[0, 0, 2] = 1.0
    R, E, Q = O.layer_quality(S3)
    assert E[0] == 0.0 and R[0] == 0.5


def test_core_layers_topk_and_ties():
    Q = np.array([0.1, 0.5, 0.5, 0.2, 0.9, 0.0, 0.5])
    assert list(O.core_layers(Q, 3)) == [1, 2, 4]          # ties to the lowest index
    assert list(O.core_layers(Q[:2], 6)) == [0, 1]          # min(K_layer, L)


def test_weighted_mean_closed_forms():
    rng = np.random.default_rng(3)
    S_all = rng.random((4, 2, 5))
    np.testing.assert_allclose(O.weighted_mean(S_all, np.ones(4), range(4)), S_all.mean(0))
    np.testing.assert_allclose(O.weighted_mean(S_all, np.array([0, 0, 3.0, 0]), [2]), S_all[2])
    Q = np.array([1.0, 3.0, 0.0, 0.0])
    np.testing.assert_allclose(O.weighted_mean(S_all, Q, [0, 1]), (S_all[0] + 3 * S_all[1]) / 4)
    np.testing.assert_allclose(O.weighted_mean(S_all, np.zeros(4), [1, 3]), (S_all[1] + S_all[3]) / 2)


def test_anchor_key_closed_forms():
    mu = 0.25
    const = np.full((4, 3), mu)
    np.testing.assert_allclose(O.anchor_key(const), mu)                  # CV = 0
    two = np.array([[0.0, 0.0, 1.0], [2 * mu, 0.0, 1.0]])
    A = O.anchor_key(two)
    assert A[0] == pytest.approx(mu / 2)                                  # CV = 1
    assert A[1] == 0.0                                                    # mu = 0
    assert A[2] == pytest.approx(1.0)
    np.testing.assert_allclose(O.anchor_key(two, cv_penalty=0.0), [mu, 0.0, 1.0])
    three = np.array([[1.0], [2.0], [3.0]])                              # population std
    assert O.anchor_key(three)[0] == pytest.approx(2.0 / (1 + math.sqrt(2 / 3) / 2))


# ---------------------------------------------------------------------------
# top-k and the selection sets (brute force)
# ---------------------------------------------------------------------------
def _topk_bruteforce(scores, cand, k):
    """The unique k-subset whose every member beats every non-member under
    (score descending, index ascending)."""
    def beats(a, b):
        return scores[a] > scores[b] or (scores[a] == scores[b] and a < b)
    hits = [set(T) for T in itertools.combinations(cand, k)
            if all(beats(a, b) for a in T for b in set(cand) - set(T))]
    assert len(hits) == 1
    return sorted(hits[0])


def test_topk_exhaustive_with_ties():
    for n in range(1, 6):
        for vals in itertools.product([0.0, 1.0, 2.0], repeat=n):
            s = np.array(vals, np.float32)
            for k in range(n + 1):
                assert list(O.topk(s, range(n), k)) == _topk_bruteforce(s, list(range(n)), k)


def test_topk_random_candidates_and_signed_zero():
    rng = np.random.default_rng(9)
    for _ in range(200):
        n = int(rng.integers(2, 9))
        s = rng.integers(-2, 3, n).astype(np.float32)
        cand = sorted(rng.choice(n, int(rng.integers(1, n + 1)), replace=False).tolist())
        k = int(rng.integers(0, len(cand) + 1))
        assert list(O.topk(s, cand, k)) == _topk_bruteforce(s, cand, k)
    s = np.array([0.0, -0.0, 0.0], np.float32)
    s[1] = -0.0
    assert list(O.topk(s, range(3), 2)) == [0, 1]            # -0 ties +0


def _select_bruteforce(V, A, kc, ks):
    F, n_s = V.shape
    J = list(range(n_s))
    m = V.max(axis=0)
    P = _topk_bruteforce(m, J, n_s - ks)
    C = [_topk_bruteforce(V[f], P, kc) for f in range(F)]
    E = [j for j in J if all(j not in c for c in C)]
    S = _topk_bruteforce(A, E, ks)
    return P, C, E, S


def test_select_matches_literal_definition_and_invariants():
    rng = np.random.default_rng(11)
    for _ in range(300):
        n_s = int(rng.integers(2, 9))
        F = int(rng.integers(1, 4))
        ks = int(rng.integers(0, n_s))
        kc = int(rng.integers(0, n_s - ks + 1))
        V = rng.integers(0, 4, (F, n_s)).astype(np.float32)
        A = rng.integers(0, 3, n_s).astype(np.float32)
        sel = O.select(V, A, kc, ks)
        P, C, E, S = _select_bruteforce(V, A, kc, ks)
        assert list(sel.pool) == P and list(sel.anchors) == S and list(sel.unused) == E
        assert [list(c) for c in sel.core] == C
        assert len(P) == n_s - ks and len(E) >= ks                       # availability
        for f in range(F):
            assert set(C[f]) <= set(P) and len(C[f]) == kc
            assert not set(C[f]) & set(S)                                  # disjoint
            R = list(sel.retained[f])
            assert R == sorted(R) and len(R) == kc + ks
            assert set(R) == set(C[f]) | set(S)


def test_mass_threshold_bruteforce_and_monotone():
    rng = np.random.default_rng(12)
    for _ in range(200):
        n_s = int(rng.integers(2, 12))
        ks = int(rng.integers(0, n_s))
        # values on a 2^-20 grid so the 2^-40 code is exact
        v = (rng.integers(0, 1 << 12, n_s) / float(1 << 20)).astype(np.float32)
        V = v[None, :]
        P = O.select(V, np.zeros(n_s, np.float32), 0, ks).pool
        for theta in (0.05, 0.5, 0.8, 0.999, 1.0):
            ranked = sorted(P, key=lambda j: (-float(v[j]), j))
            T = sum(Fraction(float(x)) for x in v)
            want = len(ranked)
            run = Fraction(0)
            for k, j in enumerate(ranked, start=1):
                run += Fraction(float(v[j]))
                if run >= Fraction(theta).limit_denominator(1000) * T:
                    want = k
                    break
            assert O.mass_count(v, P, theta) == want
        ks_ = [O.mass_count(v, P, t) for t in (0.1, 0.3, 0.5, 0.7, 0.9, 1.0)]
        assert ks_ == sorted(ks_)
    v = np.linspace(0.1, 0.2, 10).astype(np.float32)
    assert O.mass_count(v, np.arange(10), 1.0) == 10                      # all q_j > 0
    z = np.zeros(6, np.float32)
    assert O.mass_count(z, np.arange(6), 0.8) == 1                        # smallest k >= 1


def _mass_bruteforce(v, pool, frac, rounding):
    """The mass rule literally: codes rounding(V 2^40) of the exact fp32 values
    (clamped to [0, 2^40]), the pool walked in (score desc, index asc) order,
    the smallest k >= 1 whose prefix reaches frac * T."""
    def q(x):
        x = Fraction(float(x))
        return 0 if x <= 0 else (1 << 40) if x >= 1 else rounding(x * (1 << 40))
    codes = [q(x) for x in v]
    T = sum(codes)
    ranked = sorted((int(j) for j in pool), key=lambda j: (-float(v[j]), j))
    run = 0
    for k, j in enumerate(ranked, start=1):
        run += codes[j]
        if run >= frac * T:
            return k
    return len(ranked)


def test_mass_code_floors_values_off_the_grid():
    """Scores of a few 2^-40 units with fractional parts: the count must follow
    floor(V 2^40), and the cases are chosen so that rounding to nearest or up
    would change it somewhere."""
    rng = np.random.default_rng(13)
    differ_round = differ_ceil = 0
    for _ in range(300):
        n_s = int(rng.integers(3, 10))
        v = (rng.uniform(0.05, 6.0, n_s) * 2.0 ** -40).astype(np.float32)
        pool = np.arange(n_s)
        for theta in (0.2, 0.5, 0.8, 0.95):
            frac = O.threshold_fraction(theta)
            want = _mass_bruteforce(v, pool, frac, math.floor)
            assert O.mass_count(v, pool, theta) == want
            differ_round += want != _mass_bruteforce(v, pool, frac, lambda x: math.floor(x + Fraction(1, 2)))
            differ_ceil += want != _mass_bruteforce(v, pool, frac, math.ceil)
        # single codes straight from the definition
        for x in v:
            assert O.mass_code(x) == math.floor(Fraction(float(x)) * (1 << 40))
    assert differ_round > 0 and differ_ceil > 0
    # codes saturate at 1 and vanish at or below 0
    assert O.mass_code(np.float32(1.0)) == O.mass_code(np.float32(3.0)) == 1 << 40
    assert O.mass_code(np.float32(0.0)) == O.mass_code(np.float32(-1.0)) == 0
    assert O.mass_code(np.float32(2.0 ** -41)) == 0 and O.mass_code(np.float32(2.0 ** -40)) == 1


def test_threshold_fraction_rounds_the_float32_value():
    """theta = num / 1000 with num the integer nearest to 1000 times the float32
    threshold (the value the configuration carries)."""
    assert O.threshold_fraction(0.0125) == Fraction(13, 1000)   # float32(0.0125) > 1/80
    assert O.threshold_fraction(0.0004) == 0                     # below 1/2000: zero
    assert O.threshold_fraction(0.0005) == Fraction(1, 1000)     # float32(0.0005) > 1/2000
    assert O.threshold_fraction(0.8) == Fraction(4, 5)
    assert O.threshold_fraction(1.0) == 1
    rng = np.random.default_rng(14)
    for t in rng.uniform(0.0, 1.0, 2000).astype(np.float32):
        exact = Fraction(float(t)) * 1000
        num = O.threshold_fraction(float(t)) * 1000
        assert num.denominator == 1 and abs(exact - num) < Fraction(1, 2)
    # a zero numerator keeps one core token per frame
    v = np.array([0.1, 0.5, 0.2, 0.2], np.float32)
    assert O.mass_count(v, np.arange(4), 0.0004) == 1


# ---------------------------------------------------------------------------
# packing, steps, reuse
# ---------------------------------------------------------------------------
def test_pack_unpack_invariants():
    cfg = W.preset(1).replace(batch=3)
    rng = np.random.default_rng(4)
    retained = [[np.sort(rng.choice(cfg.n_s, int(rng.integers(1, cfg.n_s)), replace=False))
                 for _ in range(cfg.n_frames)] for _ in range(cfg.batch)]
    mask = O.keep_mask(cfg, retained)
    pm = O.pack_map(mask, cfg.batch)
    kept = pm.pack_pos[pm.pack_pos >= 0]
    assert (np.diff(kept) == 1).all() and kept[0] == 0                     # strictly increasing
    for b in range(cfg.batch):
        n = cfg.n_ctx + cfg.n_act + sum(len(r) for r in retained[b])
        assert pm.cu_seqlens[b + 1] - pm.cu_seqlens[b] == n
    x = rng.standard_normal((cfg.batch * cfg.l_full, 8)).astype(np.float32)
    xp = O.pack(x, pm)
    y = O.unpack(xp * 3.0, x, pm)
    pruned = pm.pack_pos < 0
    assert y[pruned].astype(np.float32).tobytes() == x[pruned].tobytes()   # bit-identical (P-12)
    np.testing.assert_array_equal(y[~pruned], 3.0 * x[~pruned].astype(np.float64))
    np.testing.assert_array_equal(O.unpack(O.pack(x, pm), x, pm), x)


def test_varlen_attention_isolates_sequences():
    rng = np.random.default_rng(6)
    nh = 2
    cu = np.array([0, 9, 9, 30, 41])                                        # includes an empty one
    q, k, v = _rand_qkv(rng, 41, nh)
    o, lse = O.attention(q, k, v, cu, nh)
    for b in range(4):
        s0, s1 = cu[b], cu[b + 1]
        if s1 > s0:
            ob, lb = O.attention(q[s0:s1], k[s0:s1], v[s0:s1], [0, s1 - s0], nh)
            np.testing.assert_array_equal(o[s0:s1], ob)
            np.testing.assert_array_equal(lse[s0:s1], lb)
    k2 = k.copy(); k2[10:30] += 1.0
    o2, _ = O.attention(q, k2, v, cu, nh)
    np.testing.assert_array_equal(o2[:9], o[:9])
    np.testing.assert_array_equal(o2[30:], o[30:])


def test_block_matches_torch_composition():
    """The block equals layer_norm / linear / SDPA / gelu(tanh) from torch in fp64 (P-10)."""
    cfg = W.preset(1)
    w = W.block_weights(cfg, 0)
    x = W.make_inputs(cfg).x(1)
    temb = W.timestep_embedding(cfg, 1)
    cu = np.array([0, 70, cfg.l_full])
    y, tr = O.block(x, w, temb, cu, cfg.n_heads, "f64")
    F = torch.nn.functional
    T = {k: torch.tensor(v, dtype=torch.float64) for k, v in w.items()}
    tx = torch.tensor(x, dtype=torch.float64)
    m = F.linear(F.silu(torch.tensor(temb, dtype=torch.float64)), T["w_ada"], T["b_ada"])
    m = m.float().double()
    sh1, sc1, g1, sh2, sc2, g2 = m.chunk(6)
    d = cfg.d_model
    ys = []
    for s0, s1 in zip(cu[:-1], cu[1:]):
        xs = tx[s0:s1]
        h = F.layer_norm(xs, (d,), eps=1e-6) * (1 + sc1) + sh1
        qkv = F.linear(h, T["w_qkv"], T["b_qkv"])
        q, k, v = qkv.split(d, dim=1)
        sh = lambda t: t.view(s1 - s0, cfg.n_heads, 64).transpose(0, 1)
        o = F.scaled_dot_product_attention(sh(q), sh(k), sh(v)).transpose(0, 1).reshape(s1 - s0, d)
        x1 = xs + g1 * F.linear(o, T["w_o"], T["b_o"])
        h2 = F.layer_norm(x1, (d,), eps=1e-6) * (1 + sc2) + sh2
        ys.append(x1 + g2 * F.linear(F.gelu(F.linear(h2, T["w_1"], T["b_1"]), approximate="tanh"),
                                     T["w_2"], T["b_2"]))
    np.testing.assert_allclose(y, torch.cat(ys).numpy(), rtol=1e-11, atol=1e-11)


def test_storage_rounding_bf16_ties_to_even():
    vals = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 1.0 + 2 ** -8 + 2 ** -20])
    np.testing.assert_array_equal(O.round_bf16(vals),
                                  [1.0, 1.0 + 4 * 2 ** -8, -1.0, 1.0 + 2 * 2 ** -8])
    assert torch.tensor(vals, dtype=torch.float32).to(torch.bfloat16).double().numpy().tolist() \
        == O.round_bf16(vals).tolist()


def _tiny_model(cfg):
    return [W.block_weights(cfg, l) for l in range(cfg.n_blocks)]


def test_full_retention_equals_dense():
    """rho = 100% (K_c = N_s, K_s = 0): identity pack map and the sparse step is
    the dense step exactly (P-11)."""
    cfg = W.preset(1).replace(k_core=64, k_anchor=0)
    model = _tiny_model(cfg)
    inp = W.make_inputs(cfg, model[0]["w_qkv"])
    r = O.refresh_step(inp.x(0), model, inp.temb(0), cfg)
    np.testing.assert_array_equal(r.packmap.gather, np.arange(cfg.l_full))
    x1, t1 = inp.x(1), inp.temb(1)
    ys = O.sparse_step(x1, model, t1, cfg, r.packmap)
    yd = O.dense_step(x1, model, t1, cfg)
    assert ys.tobytes() == yd.tobytes()


def test_refresh_is_dense_and_reuse_equals_reselection():
    """The refresh step returns the dense output; with interval R every step uses
    select(cached scores from step R floor(tau/R)) (P-13)."""
    cfg = W.preset(1).replace(n_steps=6, reuse_R=3)
    model = _tiny_model(cfg)
    inp = W.make_inputs(cfg, model[0]["w_qkv"])
    ys, refr = O.run_schedule(cfg, model, inp.x, inp.temb)
    assert sorted(refr) == [0, 3]
    for tau in range(cfg.n_steps):
        x, t = inp.x(tau), inp.temb(tau)
        base = cfg.reuse_R * (tau // cfg.reuse_R)
        if tau == base:
            np.testing.assert_array_equal(ys[tau], O.dense_step(x, model, t, cfg))
        else:
            _, _, pm = O.selection_from_scores(cfg, refr[base].S_all)
            np.testing.assert_array_equal(ys[tau], O.sparse_step(x, model, t, cfg, pm))
            pruned = pm.pack_pos < 0
            assert ys[tau][pruned].tobytes() == np.asarray(x, np.float64)[pruned].tobytes()
    # R = 1 refreshes every step
    _, refr1 = O.run_schedule(cfg.replace(reuse_R=1), model, inp.x, inp.temb, n_steps=3)
    assert sorted(refr1) == [0, 1, 2]


def test_refresh_scores_use_block_normalisers():
    """Scores in the step use the block's own q, k and lambda; recomputing lambda
    over all keys (mode B) gives the same S."""
    cfg = W.preset(1)
    model = _tiny_model(cfg)
    inp = W.make_inputs(cfg, model[0]["w_qkv"])
    x = inp.x(0)
    _, tr = O.block(x, model[0], inp.temb(0), O.dense_cu(cfg), cfg.n_heads, cfg.dtype)
    d = cfg.d_model
    act = slice(cfg.n_ctx + cfg.n_fut, cfg.l_full)
    lam_b = O.lse_all_keys(tr.qkv[act, :d], tr.qkv[:, d:2 * d], cfg.n_heads)
    np.testing.assert_allclose(lam_b, tr.lse[act], rtol=1e-6)
    S_a = O.layer_scores(cfg, tr)[0]
    S_b = O.score(tr.qkv[act, :d], tr.qkv[cfg.n_ctx:cfg.n_ctx + cfg.n_fut, d:2 * d], lam_b,
                  cfg.n_frames, cfg.n_s, cfg.n_heads)
    np.testing.assert_allclose(S_a, S_b, rtol=1e-5)


def test_anchor_statistics_use_all_layers():
    """Core score uses L_core only; the anchor key aggregates every layer
    (App. A.1).  Two one-hot layers, K_layer = 1: Q = (0.5, 0.2), so
    V = S_0 while V_all = (0.5 S_0 + 0.2 S_1) / 0.7 (constant across frames,
    CV = 0, A = mu)."""
    F, n_s = 3, 4
    S_all = np.zeros((2, F, n_s))
    S_all[0, :, 0] = 0.5
    S_all[1, :, 1] = 0.2
    red = O.score_reduce(S_all, k_layer=1)
    assert list(red.L_core) == [0]
    np.testing.assert_allclose(red.Q, [0.5, 0.2], rtol=1e-7)
    np.testing.assert_allclose(red.V, S_all[0], rtol=1e-7)
    np.testing.assert_allclose(red.A, [0.25 / 0.7, 0.04 / 0.7, 0.0, 0.0], rtol=1e-6)


@pytest.mark.parametrize("dtype", ["f64", "bf16"])
def test_block_rows_equals_full_block(dtype):
    """The row-sampled block gives exactly the rows of the full block."""
    cfg = W.preset(1).replace(batch=2)
    w = W.block_weights(cfg, 0)
    x = W.make_inputs(cfg).x(2)
    temb = W.timestep_embedding(cfg, 2)
    cu = np.array([0, 100, cfg.batch * cfg.l_full])
    y, tr = O.block(x, w, temb, cu, cfg.n_heads, dtype)
    rows = np.array([0, 5, 99, 100, 101, 250, 303])
    yr, lr = O.block_rows(x, w, temb, cu, rows, cfg.n_heads, dtype)
    np.testing.assert_allclose(yr, y[rows], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lr, tr.lse[rows], rtol=1e-6)
