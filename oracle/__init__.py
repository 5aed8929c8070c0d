"""CPU oracle of the action-guided sparse denoising step.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the package smoke check
and the benchmark's CPU-baseline leg, never by the product path.
"""
from .swam_oracle import *  # noqa: F401,F403
from .swam_oracle import (  # noqa: F401
    round_f32, round_bf16, storage_round, silu, gelu_tanh, layer_norm, modulation,
    attention, block, block_rows, BlockTrace, frame_groups, alpha_weights, score, lse_all_keys,
    layer_quality, topk, core_layers, weighted_mean, anchor_key, score_reduce, Reduced,
    threshold_fraction, mass_count, MASS_SCALE_BITS, select, Selection, keep_mask,
    pack_map, PackMap, pack, unpack, dense_cu, run_blocks, dense_step, layer_scores,
    selection_from_scores, refresh_step, sparse_step, is_refresh, run_schedule,
    RefreshResult, overlap, rope_angles, apply_rope, qk_rms_norm, qk_post, dense_positions,
    n_scored, philox4x64_10, random_keys, random_selection,
)
