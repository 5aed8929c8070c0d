"""swam_select_noalloc (the selection for callers that cannot allocate) gives
exactly what swam_select gives, through the C ABI, on consecutive calls that
share the library's static scratch array: a ragged mass-threshold batch, then
a smaller fixed-budget one, then the first again; oversize calls are refused
on the host."""
import numpy as np
import pytest
import torch

import workload as W
from helpers import dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _scores(cfg, seed):
    rng = np.random.default_rng(seed)
    V = rng.gamma(0.3, 1.0, (cfg.batch, cfg.n_frames, cfg.n_s))
    V /= V.sum(axis=2, keepdims=True)
    A = rng.gamma(0.3, 1.0, (cfg.batch, cfg.n_s)) / cfg.n_s
    return dev(V.astype(np.float32)), dev(A.astype(np.float32))


def _outputs(cfg, k_max):
    i32 = dict(dtype=torch.int32, device="cuda:0")
    return (torch.full((cfg.batch * cfg.n_frames * k_max,), 7, **i32),
            torch.full((cfg.batch * cfg.n_frames,), 7, **i32),
            torch.full((cfg.batch * cfg.l_full,), 7, **i32),
            torch.full((cfg.batch * cfg.l_full,), 7, **i32),
            torch.full((cfg.batch + 1,), 7, **i32))


def _case(cfg, seed):
    from paper_2609_38984_amd import swam
    print(f"no-alloc selection {cfg.name} B={cfg.batch} N_s={cfg.n_s} mass={cfg.mass_threshold}",
          flush=True)
    V, A = _scores(cfg, seed)
    ctx = swam.Context(cfg)
    want = _outputs(cfg, ctx.k_max)
    ctx.select(V, A, *want)
    got = _outputs(cfg, ctx.k_max)
    swam.select_noalloc(cfg.batch, cfg.n_frames, cfg.n_s, cfg.n_ctx, cfg.n_act, cfg.k_core,
                        cfg.k_anchor, cfg.mass_threshold, V, A, *got)
    torch.cuda.synchronize()
    t_pack = int(want[4][-1].item())
    names = ["keep_idx", "keep_cnt", "pack_pos", "gather", "cu_seqlens"]
    for n, w, g in zip(names, want, got):
        if n == "gather":
            w, g = w[:t_pack], g[:t_pack]
        assert torch.equal(w, g), n
    return t_pack


def test_select_noalloc_matches_select_on_consecutive_calls():
    big = W.preset(5).replace(n_blocks=2, d_model=64, n_heads=1)          # 8 ragged sequences
    small = W.preset(2).replace(n_blocks=2, d_model=64, n_heads=1)        # one fixed-budget one
    assert _case(big, 91) > 0
    assert _case(small, 92) == small.t_pack_fixed
    _case(big, 93)


def test_select_noalloc_rejects_oversize_and_bad_arguments():
    from paper_2609_38984_amd import swam
    cfg = W.preset(4, percent=25).replace(batch=16, n_blocks=1, d_model=64, n_heads=1)
    V, A = _scores(cfg.replace(batch=1), 94)
    V, A = V.reshape(-1).repeat(16), A.reshape(-1).repeat(16)
    outs = _outputs(cfg, cfg.k_core + cfg.k_anchor)
    with pytest.raises(swam.SwamError) as e:     # 16 x 17,472 keep flags alone are 1.1 MB
        swam.select_noalloc(cfg.batch, cfg.n_frames, cfg.n_s, cfg.n_ctx, cfg.n_act, cfg.k_core,
                            cfg.k_anchor, 0.0, V, A, *outs)
    assert e.value.code == -2 and "SWAM_NOALLOC_SCRATCH_BYTES" in str(e.value)
    lib = swam.load_library()
    assert lib.swam_select_noalloc(1, 2, 8, 0, 2, 2, 0, 0.0, None, None, None, None, None, None,
                                   None, None) == -1
