"""The oracle's pins catch plausible mistakes: each case plants one (a dropped
term, a wrong sign, index or order, a transposed operand, a wrong normaliser)
into the oracle on the CPU and checks that the pin named beside it fails.

Mistakes are planted by swapping one oracle function for a wrong variant
(monkeypatch, in the package namespace and in the module the other oracle
functions look it up in); nothing is changed on disk.
"""
import math

import numpy as np
import pytest

import oracle as O
import oracle.sampler_oracle as SA
import oracle.swam_oracle as SO
import test_oracle_pins as P
import test_oracle_sampler as PS
import test_oracle_variants as PV


def _plant(monkeypatch, name, fn):
    if hasattr(SA, name) and not hasattr(SO, name):
        monkeypatch.setattr(SA, name, fn)          # sampler oracle
        return
    monkeypatch.setattr(SO, name, fn)
    monkeypatch.setattr(O, name, fn)


def _ln_uncentred(x):
    x = np.asarray(x, np.float64)
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + SO.LN_EPS)


def _gelu_no_cubic(u):
    u = np.asarray(u, np.float64)
    return 0.5 * u * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * u))


def _round_bf16_truncate(x):
    x32 = np.ascontiguousarray(np.asarray(x, np.float64).astype(np.float32))
    bits = x32.view(np.uint32) & np.uint32(0xFFFF0000)
    return bits.view(np.float32).astype(np.float64)


def _topk_high_index_ties(scores, candidates, k):
    cand = np.asarray(sorted(int(c) for c in candidates), dtype=np.int64)
    s = np.asarray(scores)[cand]
    order = np.lexsort((-cand, -s.astype(np.float64)))
    return np.sort(cand[order[:k]])


def mass_code_nearest(val):
    val = float(np.float32(val))
    if not val > 0.0:
        return 0
    if val >= 1.0:
        return 1 << SO.MASS_SCALE_BITS
    return round(val * (1 << SO.MASS_SCALE_BITS))


def threshold_float64(theta):
    from fractions import Fraction
    return Fraction(max(1, int(round(theta * 1000))), 1000)


def _mutants():
    ln, mod, score, att = SO.layer_norm, SO.modulation, SO.score, SO.attention
    lq, wm, ak, pm, mc = SO.layer_quality, SO.weighted_mean, SO.anchor_key, SO.pack_map, SO.mass_count

    def mod_swapped(w, b, t):
        s = mod(w, b, t)
        return [s[1], s[0], s[2], s[4], s[3], s[5]]          # shift and scale exchanged

    def score_lambda_off(q, k, lse, F, n_s, nh, alpha=None):
        return score(q, k, np.asarray(lse) + 1.0, F, n_s, nh, alpha)

    def attention_one_sequence(q, k, v, cu, nh):
        return att(q, k, v, np.array([0, int(np.asarray(cu)[-1])]), nh)

    def attention_scale_hd(q, k, v, cu, nh):
        return att(np.asarray(q, np.float64) / 8.0, k, v, cu, nh)  # 1/hd instead of 1/sqrt(hd)

    def quality_sign(S):
        R, E, _ = lq(S)
        return R, E, R * (1.0 + E)

    def mean_unweighted(S, Q, layers):
        return wm(S, np.ones(len(np.asarray(Q))), layers)

    def anchor_no_penalty(V, c=1.0):
        return ak(V, 0.0)

    def pack_inclusive(mask, batch):
        r = pm(mask, batch)
        r.pack_pos[r.pack_pos >= 0] += 1
        return r

    def mass_plus_one(v, pool, theta):
        return min(mc(v, pool, theta) + 1, len(list(pool)))

    sig, eul, mrg = SA.sigmas, SA.euler_update, SA.merge_velocity
    rope, qkn = SO.apply_rope, SO.qk_rms_norm

    def sigmas_unshifted(n, shift=SA.SCHEDULE_SHIFT):
        return sig(n, 1.0)

    def euler_wrong_sign(z, v, dsigma):
        return eul(z, v, -dsigma)

    def merge_swapped(v_cur, v_cached, keep):
        return mrg(v_cur, v_cached, ~np.asarray(keep, bool))

    def rope_reversed(x, positions, nh):
        return rope(x, -np.asarray(positions), nh)

    def qk_norm_sum(x, nh, eps=SO.LN_EPS):
        return qkn(x, nh, eps) / 8.0                 # root of the sum, not the mean, of squares

    return {
        "layer norm without centring": ("layer_norm", _ln_uncentred,
                                        [P.test_block_matches_torch_composition]),
        "shift and scale exchanged": ("modulation", mod_swapped,
                                      [P.test_block_matches_torch_composition]),
        "GELU without its cubic term": ("gelu_tanh", _gelu_no_cubic,
                                        [P.test_block_matches_torch_composition]),
        "attention scaled by 1/hd": ("attention", attention_scale_hd,
                                     [P.test_attention_rows_sum_to_one_and_match_library]),
        "attention across sequences": ("attention", attention_one_sequence,
                                       [P.test_varlen_attention_isolates_sequences]),
        "score normaliser off by one": ("score", score_lambda_off,
                                        [lambda: P.test_score_equals_head_mean_attention(2, 4, 2),
                                         P.test_score_hand_example]),
        "uniform query weights": ("alpha_weights", lambda g: np.full(g, 1.0 / g),
                                  [lambda: P.test_alpha_printed_values(_golden())]),
        "quality with the entropy's sign flipped": ("layer_quality", quality_sign,
                                                    [P.test_entropy_closed_forms]),
        "unweighted core-layer mean": ("weighted_mean", mean_unweighted,
                                       [P.test_weighted_mean_closed_forms]),
        "anchor key without the CV penalty": ("anchor_key", anchor_no_penalty,
                                              [P.test_anchor_key_closed_forms]),
        "top-k ties to the highest index": ("topk", _topk_high_index_ties,
                                            [P.test_topk_exhaustive_with_ties]),
        "mass count one too many": ("mass_count", mass_plus_one,
                                    [P.test_mass_threshold_bruteforce_and_monotone]),
        "mass code rounded to nearest": ("mass_code", mass_code_nearest,
                                         [P.test_mass_code_floors_values_off_the_grid]),
        "threshold numerator from the float64 value, at least 1": (
            "threshold_fraction", threshold_float64,
            [P.test_threshold_fraction_rounds_the_float32_value]),
        "inclusive prefix sum in the pack map": ("pack_map", pack_inclusive,
                                                 [P.test_pack_unpack_invariants]),
        "bf16 storage by truncation": ("round_bf16", _round_bf16_truncate,
                                       [P.test_storage_rounding_bf16_ties_to_even]),
        "refresh on the last step of each interval": (
            "is_refresh", lambda tau, R: tau % R == R - 1,
            [P.test_refresh_is_dense_and_reuse_equals_reselection]),
        "flow schedule without its shift": ("sigmas", sigmas_unshifted,
                                            [PS.test_sigmas_closed_form_n4]),
        "Euler step with the wrong sign": ("euler_update", euler_wrong_sign,
                                           [PS.test_euler_integrates_the_straight_flow_exactly]),
        "merge takes the cache at retained rows": (
            "merge_velocity", merge_swapped,
            [PS.test_merge_selects_current_or_cached_rowwise]),
        "rotary angles reversed": ("apply_rope", rope_reversed,
                                   [PV.test_rope_closed_form_single_pair_and_identity_at_zero]),
        "QK-norm by the root sum of squares": ("qk_rms_norm", qk_norm_sum,
                                               [PV.test_qk_norm_gives_unit_rms_heads]),
    }


def _golden():
    import json
    import os
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    with open(os.path.join(root, "tests", "golden", "paper_constants.json")) as fh:
        return json.load(fh)


MUTANTS = _mutants()


@pytest.mark.parametrize("name", list(MUTANTS))
def test_pins_catch_planted_mistake(name, monkeypatch):
    target, fn, pins = MUTANTS[name]
    for pin in pins:
        pin()                                   # passes on the unchanged oracle
    _plant(monkeypatch, target, fn)
    caught = 0
    for pin in pins:
        try:
            pin()
        except Exception:                      # a failed check, or the pin cannot run
            caught += 1
    assert caught > 0, f"no pin caught: {name}"
