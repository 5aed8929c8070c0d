"""Host-side checks of the C ABI (no GPU): exports, plan sizes, validation."""
import ctypes as C
import os
import re

import pytest

import workload as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    from paper_2609_38984_amd import swam
    if not os.path.exists(swam.LIB_PATH):
        from paper_2609_38984_amd.build import build
        build()
    return swam.load_library()


def _declared():
    text = open(os.path.join(ROOT, "include", "swam.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(swam_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    from paper_2609_38984_amd import swam
    names = _declared()
    assert len(names) == 31
    assert sorted(swam.EXPORTS) == names
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for code, name in {0: "SWAM_OK", -1: "SWAM_E_INVALID", -4: "SWAM_E_STATE", -5: "SWAM_E_HIP"}.items():
        assert lib.swam_status_str(code).decode() == name


@pytest.mark.parametrize("n,want", [(1, (152, 64, 20)), (2, (1312, 660, 93)), (3, (10160, 3472, 364)),
                                    (5, (3360, -1, 768)), (6, (3092, 1844, 184)),
                                    (7, (326, 192, 31))])
def test_plan_sizes(lib, n, want):
    from paper_2609_38984_amd import swam
    cfg = W.preset(n)
    p = swam.plan(cfg)
    assert (p.l_full, p.t_pack_fixed, p.k_max) == want
    assert p.rows_full == cfg.batch * cfg.l_full
    assert p.group_size == cfg.g and p.n_s == cfg.n_s
    assert p.k_layer_eff == min(6, cfg.n_blocks)
    assert p.workspace_bytes > 0


@pytest.mark.parametrize("bad,code", [
    (dict(n_act=31), -1),              # H not divisible by F
    (dict(k_core=60, k_anchor=8), -1),  # K_c + K_s > N_s
    (dict(k_anchor=64), -1),           # K_s >= N_s
    (dict(head_dim=32), -2),
    (dict(d_model=100), -1),
    (dict(n_blocks=0), -2),
    (dict(reuse_R=0), -1),
    (dict(frame_h=1, frame_w=1), -2),
    (dict(mass_threshold=1.5), -1),
    (dict(n_act=2 * 17, n_frames=2), -2),  # more than 16 queries per group
    (dict(rope=2), -1),
    (dict(qk_norm=-1), -1),
    (dict(cfg_pairs=1, batch=3), -2),  # guidance pairs need an even batch
    (dict(cfg_pairs=1, batch=2, guidance=float("nan")), -1),
    # bf16 QKV buffer beyond 2^31 elements: 64 x 4112 rows x 3 x 4096
    (dict(dtype=1, batch=64, n_heads=64, d_model=4096, n_frames=1, frame_h=64, frame_w=64,
          n_act=16, n_ctx=0, k_core=100, k_anchor=10), -2),
])
def test_plan_rejects_bad_configs(lib, bad, code):
    from paper_2609_38984_amd import swam
    base = W.preset(1)
    cfg = swam.Config.from_obj(base)
    for k, v in bad.items():
        setattr(cfg, k, v)
    info = swam.PlanInfo()
    rc = lib.swam_plan(C.byref(cfg), C.byref(info))
    assert rc == code
    assert lib.swam_last_error(None).decode() != ""
    out = C.c_void_p(123)
    assert lib.swam_create(C.byref(cfg), None, C.byref(out)) == code   # rejected before any HIP call
    assert out.value is None


def test_null_context_is_rejected(lib):
    assert lib.swam_pack(None, None, None) == -1
    assert lib.swam_step(None, None, None, None, 0, None, 0, None) == -1
    assert lib.swam_set_stream(None, None) == -1
    assert lib.swam_packed_rows(None, None) == -1
    assert lib.swam_graph_clear(None) == -1
    assert lib.swam_timer_stride(None, 1) == -1
    n, ms = C.c_int64(), C.c_double()
    assert lib.swam_timer_read_kind(None, 0, -2, C.byref(n), C.byref(ms)) == -1
    assert lib.swam_destroy(None) == 0


def test_sampler_entry_points_reject_bad_arguments_without_a_gpu(lib):
    # NULL context and a latent io outside the supported channel range are
    # rejected on the host before any HIP call
    from paper_2609_38984_amd import swam
    io = swam.LatentIOStruct(0, None, None, None, None)
    assert lib.swam_embed(None, C.byref(io), None, None) == -1
    assert lib.swam_velocity(None, C.byref(io), None, 0, None) == -1
    assert lib.swam_sample_update(None, 16, None, None, None, 0.1, 1) == -1
    assert lib.swam_sample_step(None, None, C.byref(io), None, None, None, None, None, None, 0,
                                0.1, 0, None) == -1


def test_flow_sigmas_host_call(lib):
    from paper_2609_38984_amd import swam
    s = swam.flow_sigmas(4)
    assert s[0] == 1.0 and s[-1] == 0.0
    assert abs(s[2] - 5.0 / 6.0) < 1e-15 and all(a > b for a, b in zip(s, s[1:]))
    assert swam.flow_sigmas(3, 1.0) == [1.0 - i / 3.0 for i in range(4)]   # shift 1: linear
    out = (C.c_double * 5)()
    assert lib.swam_flow_sigmas(0, 5.0, out) == -1
    assert lib.swam_flow_sigmas(4, 0.0, out) == -1
    assert lib.swam_flow_sigmas(4, float("inf"), out) == -1
    assert lib.swam_flow_sigmas(4, 5.0, None) == -1


def test_workspace_does_not_grow_with_block_depth(lib):
    """A refresh scores each layer right after its attention, so one QKV and one
    normaliser slot serve every block: the workspace grows with the block count
    only by the per-block modulation (6 d floats), the per-layer scores
    (F N_s floats per scored sequence) and two per-layer statistics."""
    from paper_2609_38984_amd import swam
    cfg = W.preset(3)
    w28 = swam.plan(cfg).workspace_bytes
    w1 = swam.plan(cfg.replace(n_blocks=1)).workspace_bytes
    per_block = 6 * cfg.d_model * 4 + cfg.n_scored * (cfg.n_frames * cfg.n_s * 4 + 4 + 8 + 2 * 8 * cfg.n_frames)
    assert w28 - w1 <= 27 * per_block + 16 * 256
    # one QKV slot of the 10,160-token, d = 1536 workload is 93.6 MB; 28 of them were 2.6 GB
    assert w28 < 512 << 20


def test_select_noalloc_validates_on_the_host(lib):
    """The allocation-free selection refuses NULL tensors and sizes beyond its
    static scratch before any HIP call (so this runs without a GPU)."""
    assert lib.swam_select_noalloc(1, 2, 8, 0, 2, 2, 0, 0.0, None, None, None, None, None, None,
                                   None, None) == -1
    fake = [C.c_void_p(256)] * 7             # never dereferenced: the size check comes first
    # 16 sequences of 17,472 tokens: 1.1 MB of keep flags alone
    assert lib.swam_select_noalloc(16, 16, 1024, 1024, 64, 256, 64, 0.0, *fake, None) == -2
    assert b"SWAM_NOALLOC_SCRATCH_BYTES" in lib.swam_last_error(None)
    assert lib.swam_select_noalloc(1, 2, 8, 0, 2, 7, 2, 0.0, *fake, None) == -1   # K_c + K_s > N_s
