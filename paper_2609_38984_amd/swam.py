"""Thin ctypes binding of libswam (include/swam.h).

Argument marshalling only: tensors are checked for device, dtype, size and
contiguity, then their device pointers are passed to the C ABI.  Every step of
the path runs in the HIP kernels of libswam.so; if the library is missing the
binding raises instead of computing anything itself.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libswam.so")

SWAM_F32, SWAM_BF16 = 0, 1
STATUS = {0: "SWAM_OK", -1: "SWAM_E_INVALID", -2: "SWAM_E_SHAPE", -3: "SWAM_E_DTYPE",
          -4: "SWAM_E_STATE", -5: "SWAM_E_HIP", -6: "SWAM_E_NOMEM", -7: "SWAM_E_UNSUPPORTED"}
FORCE_DENSE, FORCE_REFRESH = 1, 2
KIND_DENSE, KIND_REFRESH, KIND_SPARSE = 0, 1, 2
KIND_NONE, KIND_ANY = -1, -2   # timer slots outside any step / every slot
TIMERS = ["ADALN", "LNMOD", "GEMM_QKV", "ATTN", "GEMM_OUT", "GEMM_UP", "GEMM_DOWN", "SCORE",
          "REDUCE", "SELECT", "PACK", "UNPACK", "COPY", "SAMPLE", "QK_POST"]
T = {name: i for i, name in enumerate(TIMERS)}

EXPORTS = ["swam_create", "swam_destroy", "swam_set_stream", "swam_plan", "swam_status_str",
           "swam_last_error", "swam_score", "swam_score_reduce", "swam_select",
           "swam_set_selection", "swam_packed_rows", "swam_export", "swam_pack", "swam_unpack",
           "swam_block", "swam_step", "swam_step_graph", "swam_graph_clear", "swam_timer_enable",
           "swam_timer_reset", "swam_timer_read", "swam_timer_stride",
           "swam_timer_read_kind", "swam_embed", "swam_velocity",
           "swam_sample_update", "swam_sample_step", "swam_overlap", "swam_select_random",
           "swam_flow_sigmas", "swam_select_noalloc"]

# the flow-schedule shift of the paper's backbones (App. B.2)
SCHEDULE_SHIFT = 5.0


def flow_sigmas(n_steps: int, shift: float = SCHEDULE_SHIFT) -> list[float]:
    """The n_steps + 1 noise levels of the shifted flow schedule, computed by
    swam_flow_sigmas in the library (a host call, no GPU needed)."""
    lib = load_library()
    out = (C.c_double * (n_steps + 1))()
    _check(lib, None, lib.swam_flow_sigmas(int(n_steps), float(shift), out))
    return list(out)


class SwamError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


class Config(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "batch", "d_model", "n_heads", "head_dim", "mlp_ratio", "n_blocks", "d_temb", "n_ctx",
        "n_frames", "frame_h", "frame_w", "n_act", "k_core", "k_anchor", "k_layer")] + [
        ("cv_penalty", C.c_float), ("mass_threshold", C.c_float), ("reuse_R", C.c_int32),
        ("dtype", C.c_int32), ("rope", C.c_int32), ("qk_norm", C.c_int32),
        ("cfg_pairs", C.c_int32), ("guidance", C.c_float)]

    @classmethod
    def from_obj(cls, o) -> "Config":
        """Build from any object with the workload attributes (dtype 'f32'/'bf16')."""
        c = cls()
        for n, _ in cls._fields_:
            if n == "dtype":
                c.dtype = SWAM_BF16 if o.dtype == "bf16" else SWAM_F32
            elif n in ("rope", "qk_norm", "cfg_pairs"):
                setattr(c, n, int(getattr(o, n, 0)))
            elif n == "guidance":
                c.guidance = float(getattr(o, n, 1.0))
            else:
                setattr(c, n, getattr(o, n))
        return c


class PlanInfo(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("n_s", "group_size", "l_full", "rows_full", "k_max",
                                         "t_pack_fixed", "k_layer_eff", "workspace_bytes")]


WEIGHT_NAMES = ["w_ada", "b_ada", "w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2"]


class BlockWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in WEIGHT_NAMES]


class ModelStruct(C.Structure):
    _fields_ = [("n_blocks", C.c_int32), ("blocks", C.POINTER(BlockWeights))]


LATENT_NAMES = ["w_in", "b_in", "w_v", "b_v"]


class LatentIOStruct(C.Structure):
    _fields_ = [("d_latent", C.c_int32)] + [(n, C.c_void_p) for n in LATENT_NAMES]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libswam.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(the HIP library is required; there is no fallback)")
    lib = C.CDLL(path)
    P, I32, I64, F = C.c_void_p, C.c_int32, C.c_int64, C.c_float
    sig = {
        "swam_create": [C.POINTER(Config), P, C.POINTER(P)],
        "swam_destroy": [P], "swam_set_stream": [P, P],
        "swam_plan": [C.POINTER(Config), C.POINTER(PlanInfo)],
        "swam_score": [P, P, I64, I64, P, I64, I64, P, P, I64, P],
        "swam_score_reduce": [P, P, P, P, P, P],
        "swam_select": [P, P, P, P, P, P, P, P],
        "swam_select_random": [P, C.c_uint64, P, P, P, P, P],
        "swam_set_selection": [P, P, P],
        "swam_packed_rows": [P, C.POINTER(I64)],
        "swam_export": [P, P, P, P, P, P, P, P, P, P],
        "swam_pack": [P, P, P], "swam_unpack": [P, P, P, P],
        "swam_block": [P, C.POINTER(BlockWeights), P, P, I64, P, I32, P, P],
        "swam_step": [P, C.POINTER(ModelStruct), P, P, I32, P, I32, C.POINTER(I32)],
        "swam_step_graph": [P, C.POINTER(ModelStruct), P, P, I32, P, I32, C.POINTER(I32)],
        "swam_graph_clear": [P],
        "swam_timer_enable": [P, C.c_uint32, I32], "swam_timer_reset": [P],
        "swam_timer_read": [P, I32, C.POINTER(I64), C.POINTER(C.c_double)],
        "swam_timer_stride": [P, I32],
        "swam_timer_read_kind": [P, I32, I32, C.POINTER(I64), C.POINTER(C.c_double)],
        "swam_overlap": [P, P, P, I64, I64, P],
        "swam_flow_sigmas": [I32, C.c_double, C.POINTER(C.c_double)],
        "swam_select_noalloc": [I32, I32, I32, I32, I32, I32, I32, F, P, P, P, P, P, P, P, P],
        "swam_embed": [P, C.POINTER(LatentIOStruct), P, P],
        "swam_velocity": [P, C.POINTER(LatentIOStruct), P, I32, P],
        "swam_sample_update": [P, I32, P, P, P, F, I32],
        "swam_sample_step": [P, C.POINTER(ModelStruct), C.POINTER(LatentIOStruct), P, P, P, P, P,
                             P, I32, F, I32, C.POINTER(I32)],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = C.c_int
    lib.swam_status_str.argtypes = [C.c_int]
    lib.swam_status_str.restype = C.c_char_p
    lib.swam_last_error.argtypes = [P]
    lib.swam_last_error.restype = C.c_char_p
    _lib = lib
    return lib


def _check(lib, ctx, rc):
    if rc != 0:
        raise SwamError(rc, lib.swam_last_error(ctx).decode())


def plan(cfg) -> PlanInfo:
    lib = load_library()
    c = cfg if isinstance(cfg, Config) else Config.from_obj(cfg)
    info = PlanInfo()
    _check(lib, None, lib.swam_plan(C.byref(c), C.byref(info)))
    return info


def _ptr(t, dtype=None, numel=None, name="tensor"):
    """Device pointer of a contiguous CUDA tensor (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs {numel}")
    return t.data_ptr()


class Model:
    """Device weights of every block, kept alive with their C descriptors."""

    def __init__(self, blocks: list[dict], act_dtype: torch.dtype):
        self.blocks = blocks
        self._arr = (BlockWeights * len(blocks))()
        for i, w in enumerate(blocks):
            for n in WEIGHT_NAMES:
                setattr(self._arr[i], n, _ptr(w[n], act_dtype, name=n))
        self.struct = ModelStruct(len(blocks), self._arr)


class LatentIO:
    """Device latent embedding / velocity head weights with their C descriptor."""

    def __init__(self, weights: dict, act_dtype: torch.dtype):
        self.weights = weights
        self.d_latent = int(weights["w_in"].shape[1])
        self.struct = LatentIOStruct(self.d_latent, *[_ptr(weights[n], act_dtype, name=n)
                                                      for n in LATENT_NAMES])


NOALLOC_SCRATCH_BYTES = 1 << 20   # SWAM_NOALLOC_SCRATCH_BYTES


def select_noalloc(batch, n_frames, n_s, n_ctx, n_act, k_core, k_anchor, mass_threshold,
                   v, a, keep_idx, keep_cnt, pack_pos, gather, cu_seqlens,
                   stream: torch.cuda.Stream | None = None):
    """swam_select_noalloc: the selection and pack map for explicit sizes,
    without a context and without any allocation (scratch in the library's
    static device array), on `stream` (default: torch's current stream)."""
    lib = load_library()
    l_full = n_ctx + n_frames * n_s + n_act
    k_max = n_s if mass_threshold > 0 else max(1, k_core + k_anchor)
    i32 = torch.int32
    args = [_ptr(v, torch.float32, batch * n_frames * n_s, "v"),
            _ptr(a, torch.float32, batch * n_s, "a"),
            _ptr(keep_idx, i32, batch * n_frames * k_max, "keep_idx"),
            _ptr(keep_cnt, i32, batch * n_frames, "keep_cnt"),
            _ptr(pack_pos, i32, batch * l_full, "pack_pos"),
            _ptr(gather, i32, batch * l_full, "gather"),
            _ptr(cu_seqlens, i32, batch + 1, "cu_seqlens")]
    st = (stream or torch.cuda.current_stream()).cuda_stream
    _check(lib, None, lib.swam_select_noalloc(int(batch), int(n_frames), int(n_s), int(n_ctx),
                                              int(n_act), int(k_core), int(k_anchor),
                                              float(mass_threshold), *args, C.c_void_p(st)))


class Context:
    """One libswam context bound to a stream (default: torch's current stream)."""

    def __init__(self, cfg, stream: torch.cuda.Stream | None = None):
        self.lib = load_library()
        self.cfg = cfg
        self.c_cfg = cfg if isinstance(cfg, Config) else Config.from_obj(cfg)
        self.plan = plan(self.c_cfg)
        self.act_dtype = torch.bfloat16 if self.c_cfg.dtype == SWAM_BF16 else torch.float32
        self.stream = stream or torch.cuda.current_stream()
        h = C.c_void_p()
        _check(self.lib, None, self.lib.swam_create(C.byref(self.c_cfg),
                                                    C.c_void_p(self.stream.cuda_stream),
                                                    C.byref(h)))
        self.h = h

    def close(self):
        if getattr(self, "h", None):
            self.lib.swam_destroy(self.h)
            self.h = None

    def __del__(self):
        self.close()

    def _ok(self, rc):
        _check(self.lib, self.h, rc)

    def set_stream(self, stream: torch.cuda.Stream):
        """swam_set_stream: later calls run on `stream`, after the work already
        queued on the previous one."""
        self._ok(self.lib.swam_set_stream(self.h, C.c_void_p(stream.cuda_stream)))
        self.stream = stream

    # -- sizes -----------------------------------------------------------------
    @property
    def n_s(self):
        return self.plan.n_s

    @property
    def rows_full(self):
        return self.plan.rows_full

    @property
    def k_max(self):
        return self.plan.k_max

    @property
    def n_scored(self):
        """Sequences that are scored and selected (the conditional half with
        guidance pairs)."""
        c = self.c_cfg
        return c.batch // 2 if c.cfg_pairs else c.batch

    # -- (1) scoring -----------------------------------------------------------
    def score(self, q_act, q_seq, q_row, k_fut, k_seq, k_row, s_out, lse_act=None, k_all=None,
              kall_seq=0):
        c = self.c_cfg
        n_s = self.n_s
        _ptr(s_out, torch.float32, self.n_scored * c.n_frames * n_s, "s_out")
        self._ok(self.lib.swam_score(
            self.h, _ptr(q_act, self.act_dtype, name="q_act"), q_seq, q_row,
            _ptr(k_fut, self.act_dtype, name="k_fut"), k_seq, k_row,
            _ptr(lse_act, torch.float32, self.n_scored * c.n_act * c.n_heads, "lse_act"),
            _ptr(k_all, self.act_dtype, name="k_all"), kall_seq, s_out.data_ptr()))

    def score_reduce(self, s_all, v_out, a_out, q_out=None, core_out=None):
        c = self.c_cfg
        self._ok(self.lib.swam_score_reduce(
            self.h, _ptr(s_all, torch.float32, self.n_scored * c.n_blocks * c.n_frames * self.n_s, "s_all"),
            _ptr(q_out, torch.float32, self.n_scored * c.n_blocks, "q_out"),
            _ptr(v_out, torch.float32, self.n_scored * c.n_frames * self.n_s, "v_out"),
            _ptr(a_out, torch.float32, self.n_scored * self.n_s, "a_out"),
            _ptr(core_out, torch.int32, self.n_scored * self.plan.k_layer_eff, "core_out")))

    # -- (2) selection ---------------------------------------------------------
    def select(self, v=None, a=None, keep_idx=None, keep_cnt=None, pack_pos=None, gather=None,
               cu_seqlens=None):
        c = self.c_cfg
        self._ok(self.lib.swam_select(
            self.h, _ptr(v, torch.float32, self.n_scored * c.n_frames * self.n_s, "v"),
            _ptr(a, torch.float32, self.n_scored * self.n_s, "a"),
            _ptr(keep_idx, torch.int32, c.batch * c.n_frames * self.k_max, "keep_idx"),
            _ptr(keep_cnt, torch.int32, c.batch * c.n_frames, "keep_cnt"),
            _ptr(pack_pos, torch.int32, self.rows_full, "pack_pos"),
            _ptr(gather, torch.int32, self.rows_full, "gather"),
            _ptr(cu_seqlens, torch.int32, c.batch + 1, "cu_seqlens")))

    def select_random(self, seed: int, keep_idx=None, keep_cnt=None, pack_pos=None, gather=None,
                      cu_seqlens=None):
        """Random-selection baseline at the configured budget K_c + K_s."""
        c = self.c_cfg
        self._ok(self.lib.swam_select_random(
            self.h, int(seed) & ((1 << 64) - 1),
            _ptr(keep_idx, torch.int32, c.batch * c.n_frames * self.k_max, "keep_idx"),
            _ptr(keep_cnt, torch.int32, c.batch * c.n_frames, "keep_cnt"),
            _ptr(pack_pos, torch.int32, self.rows_full, "pack_pos"),
            _ptr(gather, torch.int32, self.rows_full, "gather"),
            _ptr(cu_seqlens, torch.int32, c.batch + 1, "cu_seqlens")))

    def set_selection(self, keep_idx, keep_cnt=None):
        c = self.c_cfg
        self._ok(self.lib.swam_set_selection(
            self.h, _ptr(keep_idx, torch.int32, c.batch * c.n_frames * self.k_max, "keep_idx"),
            _ptr(keep_cnt, torch.int32, c.batch * c.n_frames, "keep_cnt")))

    def packed_rows(self) -> int:
        r = C.c_int64()
        self._ok(self.lib.swam_packed_rows(self.h, C.byref(r)))
        return r.value

    def export(self, s_all=None, q=None, v=None, a=None, keep_idx=None, keep_cnt=None,
               pack_pos=None, gather=None, cu_seqlens=None):
        c = self.c_cfg
        n_s = self.n_s
        self._ok(self.lib.swam_export(
            self.h, _ptr(s_all, torch.float32, self.n_scored * c.n_blocks * c.n_frames * n_s, "s_all"),
            _ptr(q, torch.float32, self.n_scored * c.n_blocks, "q"),
            _ptr(v, torch.float32, self.n_scored * c.n_frames * n_s, "v"),
            _ptr(a, torch.float32, self.n_scored * n_s, "a"),
            _ptr(keep_idx, torch.int32, c.batch * c.n_frames * self.k_max, "keep_idx"),
            _ptr(keep_cnt, torch.int32, c.batch * c.n_frames, "keep_cnt"),
            _ptr(pack_pos, torch.int32, self.rows_full, "pack_pos"),
            _ptr(gather, torch.int32, self.rows_full, "gather"),
            _ptr(cu_seqlens, torch.int32, c.batch + 1, "cu_seqlens")))

    # -- (3) pack / (5) unpack ---------------------------------------------------
    def pack(self, x_full, x_packed):
        d = self.c_cfg.d_model
        self._ok(self.lib.swam_pack(self.h, _ptr(x_full, self.act_dtype, self.rows_full * d, "x_full"),
                                    _ptr(x_packed, self.act_dtype, self.packed_rows() * d, "x_packed")))

    def unpack(self, y_packed, x_full, y_full):
        d = self.c_cfg.d_model
        self._ok(self.lib.swam_unpack(
            self.h, _ptr(y_packed, self.act_dtype, self.packed_rows() * d, "y_packed"),
            _ptr(x_full, self.act_dtype, self.rows_full * d, "x_full"),
            _ptr(y_full, self.act_dtype, self.rows_full * d, "y_full")))

    # -- (4) block ---------------------------------------------------------------
    def block(self, weights: dict, temb, x, n_rows=None, cu_seqlens=None, n_seqs=0, lse_out=None,
              qkv_out=None):
        c = self.c_cfg
        d = c.d_model
        n_rows = self.rows_full if n_rows is None else int(n_rows)
        bw = BlockWeights()
        for n in WEIGHT_NAMES:
            setattr(bw, n, _ptr(weights[n], self.act_dtype, name=n))
        self._ok(self.lib.swam_block(
            self.h, C.byref(bw), _ptr(temb, torch.float32, c.d_temb, "temb"),
            _ptr(x, self.act_dtype, n_rows * d, "x"), n_rows,
            _ptr(cu_seqlens, torch.int32, None, "cu_seqlens"), n_seqs,
            _ptr(lse_out, torch.float32, n_rows * c.n_heads, "lse_out"),
            _ptr(qkv_out, self.act_dtype, n_rows * 3 * d, "qkv_out")))

    # -- step --------------------------------------------------------------------
    def step(self, model: Model, x_full, temb, tau: int, y_full, flags: int = 0) -> int:
        c = self.c_cfg
        n = self.rows_full * c.d_model
        kind = C.c_int32(-1)
        self._ok(self.lib.swam_step(
            self.h, C.byref(model.struct), _ptr(x_full, self.act_dtype, n, "x_full"),
            _ptr(temb, torch.float32, c.d_temb, "temb"), int(tau),
            _ptr(y_full, self.act_dtype, n, "y_full"), int(flags), C.byref(kind)))
        return kind.value

    def step_graph(self, model: Model, x_full, temb, tau: int, y_full, flags: int = 0) -> int:
        """swam_step through cached HIP graphs (needs a non-default stream)."""
        c = self.c_cfg
        n = self.rows_full * c.d_model
        kind = C.c_int32(-1)
        self._ok(self.lib.swam_step_graph(
            self.h, C.byref(model.struct), _ptr(x_full, self.act_dtype, n, "x_full"),
            _ptr(temb, torch.float32, c.d_temb, "temb"), int(tau),
            _ptr(y_full, self.act_dtype, n, "y_full"), int(flags), C.byref(kind)))
        return kind.value

    def graph_clear(self):
        self._ok(self.lib.swam_graph_clear(self.h))

    # -- diagnostics ---------------------------------------------------------------
    def overlap(self, p, q, out):
        """out[m] = Overlap(p[m], q[m]) of normalised maps (rows of p and q)."""
        n_maps, n = int(p.shape[0]), int(p[0].numel())
        self._ok(self.lib.swam_overlap(self.h, _ptr(p, torch.float32, n_maps * n, "p"),
                                       _ptr(q, torch.float32, n_maps * n, "q"), n_maps, n,
                                       _ptr(out, torch.float32, n_maps, "out")))

    # -- sampling update -----------------------------------------------------------
    def _n_lat(self):
        """Latent rows of every sequence (the rows of v)."""
        c = self.c_cfg
        return c.batch * (self.plan.l_full - c.n_ctx)

    def _n_state(self):
        """Latent rows of the state z and the velocity cache (one per pair
        with guidance)."""
        return self.n_scored * (self.plan.l_full - self.c_cfg.n_ctx)

    def embed(self, io: LatentIO, z, x_full):
        n = self._n_state() * io.d_latent
        self._ok(self.lib.swam_embed(self.h, C.byref(io.struct), _ptr(z, torch.float32, n, "z"),
                                     _ptr(x_full, self.act_dtype, self.rows_full * self.c_cfg.d_model,
                                          "x_full")))

    def velocity(self, io: LatentIO, y_full, v, retained_only: bool = False):
        self._ok(self.lib.swam_velocity(
            self.h, C.byref(io.struct),
            _ptr(y_full, self.act_dtype, self.rows_full * self.c_cfg.d_model, "y_full"),
            int(bool(retained_only)), _ptr(v, torch.float32, self._n_lat() * io.d_latent, "v")))

    def sample_update(self, d_latent: int, v, v_cache, z, dsigma: float, kind: int):
        n = self._n_state() * d_latent
        self._ok(self.lib.swam_sample_update(
            self.h, int(d_latent), _ptr(v, torch.float32, self._n_lat() * d_latent, "v"),
            _ptr(v_cache, torch.float32, n, "v_cache"), _ptr(z, torch.float32, n, "z"),
            float(dsigma), int(kind)))

    def sample_step(self, model: Model, io: LatentIO, z, v, v_cache, x_full, y_full, temb,
                    tau: int, dsigma: float, flags: int = 0) -> int:
        c = self.c_cfg
        n = self._n_state() * io.d_latent
        nt = self.rows_full * c.d_model
        kind = C.c_int32(-1)
        self._ok(self.lib.swam_sample_step(
            self.h, C.byref(model.struct), C.byref(io.struct), _ptr(z, torch.float32, n, "z"),
            _ptr(v, torch.float32, self._n_lat() * io.d_latent, "v"),
            _ptr(v_cache, torch.float32, n, "v_cache"),
            _ptr(x_full, self.act_dtype, nt, "x_full"), _ptr(y_full, self.act_dtype, nt, "y_full"),
            _ptr(temb, torch.float32, c.d_temb, "temb"), int(tau), float(dsigma), int(flags),
            C.byref(kind)))
        return kind.value

    # -- timers ------------------------------------------------------------------
    def timer_enable(self, classes, capacity=8192):
        mask = 0
        for cls in classes:
            mask |= 1 << (T[cls] if isinstance(cls, str) else int(cls))
        self._ok(self.lib.swam_timer_enable(self.h, mask, capacity))

    def timer_reset(self):
        self._ok(self.lib.swam_timer_reset(self.h))

    def timer_stride(self, stride: int):
        self._ok(self.lib.swam_timer_stride(self.h, int(stride)))

    def timer_read(self, cls, kind: int = KIND_ANY) -> tuple[int, float]:
        n, ms = C.c_int64(), C.c_double()
        self._ok(self.lib.swam_timer_read_kind(self.h, T[cls] if isinstance(cls, str) else int(cls),
                                               int(kind), C.byref(n), C.byref(ms)))
        return n.value, ms.value
