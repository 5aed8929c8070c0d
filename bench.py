"""Benchmark of the action-guided sparse denoising step on one MI355X.

A bench "step" is one denoising step of the schedule: a refresh step (dense
forward with per-layer scoring, score reduction, selection and pack map) when
tau mod R == 0, otherwise a sparse step (pack, blocks on the packed sequence,
unpack).  K timed steps therefore cover every part of the hot path.

value = K * batch * l_full / (timed seconds): full-latent tokens advanced per
second over the schedule, inputs already resident in HBM.  Alongside: the
dense, refresh and sparse step rates, the sparse/dense speedup, the score+pack
overhead as a percentage of the dense step, per-phase times, the roofline of
the dominant kernel (HIP events on the library's stream during the timed
steps) and the CPU oracle timed on a bounded sample of the same workload.

Default workload: the 28-block d=1536 WAM-scale DiT (8 frames x 30x40 future
tokens, 512 context, 48 action tokens, 25% + 64 retention, R = 2).
"""
from __future__ import annotations

import argparse
import json
import os
import re
import statistics
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "sparse denoise-step tokens/sec vs dense at 1 MI355X; score+pack overhead %"
PEAK_BF16_TFLOPS = 2500.0
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def workload_from_args(args):
    import workload as W
    if args.config == 4:
        cfg = W.preset(4, percent=args.percent, reuse_R=args.reuse or 2)
    else:
        cfg = W.preset(args.config)
    if args.reuse:
        cfg = cfg.replace(reuse_R=args.reuse)
    if args.rope or args.qk_norm:
        tag = "+rope" * args.rope + "+qknorm" * args.qk_norm
        cfg = cfg.replace(rope=int(args.rope), qk_norm=int(args.qk_norm), name=cfg.name + tag)
    if args.guidance is not None:
        # every sequence gets an unconditional partner: the batch doubles
        cfg = cfg.replace(batch=2 * cfg.batch, cfg_pairs=1, guidance=args.guidance,
                          name=f"{cfg.name}+cfg{args.guidance:g}")
    return cfg


def kernel_work(cfg, cls, rows_per_seq):
    """Algorithmic flops (GEMMs, attention) or bytes (memory-bound phases) of one
    launch of class `cls` on sequences of the given lengths."""
    d = cfg.d_model
    hid = cfg.mlp_ratio * d
    m = sum(rows_per_seq)
    esz = 2 if cfg.dtype == "bf16" else 4
    if cls == "GEMM_QKV":
        return 2.0 * m * 3 * d * d
    if cls == "GEMM_OUT":
        return 2.0 * m * d * d
    if cls == "GEMM_UP":
        return 2.0 * m * hid * d
    if cls == "GEMM_DOWN":
        return 2.0 * m * d * hid
    if cls == "ATTN":
        return float(sum(4.0 * r * r * d for r in rows_per_seq))
    if cls == "SCORE":
        # one read of the future keys, the action queries and normalisers; S written
        return float(cfg.batch * (cfg.n_fut * d * esz + cfg.n_act * d * esz
                                  + cfg.n_act * cfg.n_heads * 4 + cfg.n_fut * 4))
    if cls == "PACK":
        # the gather-pack fused into block 0's first LayerNorm: the retained
        # rows read once, written once packed and once modulated
        return 3.0 * m * d * esz
    if cls == "UNPACK":
        # the packed (retained) rows read once and scattered once; the pruned
        # rows are copied on the side stream while the blocks run
        return 2.0 * m * d * esz
    if cls == "QK_POST":
        # q and k of every row read and written once (the rotation table is L2-resident)
        return 4.0 * m * d * esz
    raise KeyError(cls)


BOUND = {"GEMM_QKV": "mfma", "GEMM_OUT": "mfma", "GEMM_UP": "mfma", "GEMM_DOWN": "mfma",
         "ATTN": "mfma", "SCORE": "hbm", "PACK": "hbm", "UNPACK": "hbm", "QK_POST": "hbm"}


def step_flops(cfg, rows):
    """Flop model of one block on a sequence of `rows` tokens: 24 d^2 T + 4 d T^2."""
    d = cfg.d_model
    return 24.0 * d * d * rows + 4.0 * d * rows * rows


def host_description():
    """CPU model of the host and the BLAS numpy links (threadpoolctl)."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas = []
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            blas.append(f"{i.get('internal_api')} {i.get('version')} "
                        f"({i.get('threading_layer', '?')}, {i.get('num_threads')} threads)")
    except Exception:
        pass
    return model, blas


def cpu_baseline(cfg, kinds, blocks_np, inp):
    """The oracle (plain float64 numpy, never tuned) timed on this host:

    * the 1-block fp32 workload's whole schedule, with every BLAS thread and
      with one;
    * the 8-block d = 1024 workload: one refresh step and one sparse step
      measured whole, its 10-step schedule composed from them;
    * the benched workload on a bounded sample: one packed block, one layer's
      scoring, one reduce + select and (on a fast host) one dense block, scaled
      to the timed schedule (a whole step is hours of numpy).
    `value` is the benched workload's rate; the others are context."""
    import oracle as O
    import workload as W
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threadpool_limits = None
        cores = len(os.sched_getaffinity(0))
    cpu_model, blas = host_description()

    # workload 1 in full
    c1 = W.preset(1)
    b1 = [W.block_weights(c1, l) for l in range(c1.n_blocks)]
    i1 = W.make_inputs(c1, b1[0]["w_qkv"])
    t0 = time.perf_counter()
    O.run_schedule(c1, b1, i1.x, i1.temb)
    t1_n = time.perf_counter() - t0
    t1_1 = None
    if threadpool_limits is not None:
        with threadpool_limits(1):
            t0 = time.perf_counter()
            O.run_schedule(c1, b1, i1.x, i1.temb)
            t1_1 = time.perf_counter() - t0
    # workload 2: one refresh and one sparse step, whole
    c2 = W.preset(2)
    b2 = [W.block_weights(c2, l) for l in range(c2.n_blocks)]
    i2 = W.make_inputs(c2, b2[0]["w_qkv"])
    t0 = time.perf_counter()
    r2 = O.refresh_step(i2.x(0), b2, i2.temb(0), c2)
    t2_f = time.perf_counter() - t0
    t0 = time.perf_counter()
    O.sparse_step(i2.x(1), b2, i2.temb(1), c2, r2.packmap)
    t2_s = time.perf_counter() - t0
    n2_f = sum(1 for t in range(c2.n_steps) if t % c2.reuse_R == 0)
    t2 = n2_f * t2_f + (c2.n_steps - n2_f) * t2_s

    # the benched workload, sampled
    x = inp.x(0)
    temb = inp.temb(0)
    w = blocks_np[0]
    rng = np.random.default_rng(0)
    d = cfg.d_model
    t0 = time.perf_counter()
    for b in range(cfg.batch):
        q = rng.standard_normal((cfg.n_act, d))
        k = rng.standard_normal((cfg.n_fut, d))
        O.score(q, k, np.full((cfg.n_act, cfg.n_heads), 10.0), cfg.n_frames, cfg.n_s, cfg.n_heads)
    t_score = time.perf_counter() - t0
    S_all = rng.random((cfg.batch, cfg.n_blocks, cfg.n_frames, cfg.n_s)) / cfg.n_s
    t0 = time.perf_counter()
    _, _, pm = O.selection_from_scores(cfg, S_all)
    t_select = time.perf_counter() - t0
    t0 = time.perf_counter()
    O.block(O.pack(x, pm), w, temb, pm.cu_seqlens, cfg.n_heads, cfg.dtype)
    t_sparse_block = time.perf_counter() - t0
    packed = [int(pm.cu_seqlens[b + 1] - pm.cu_seqlens[b]) for b in range(cfg.batch)]
    ratio = (sum(step_flops(cfg, cfg.l_full) for _ in range(cfg.batch))
             / sum(step_flops(cfg, r) for r in packed))
    t_dense_block = t_sparse_block * ratio
    how = f"dense block extrapolated by the flop model (x{ratio:.2f})"
    if t_dense_block < 25.0:   # fast host: measure the dense block as well
        t0 = time.perf_counter()
        O.block(x, w, temb, O.dense_cu(cfg), cfg.n_heads, cfg.dtype)
        t_dense_block = time.perf_counter() - t0
        how = f"one dense block ({cfg.batch * cfg.l_full} tokens) {t_dense_block:.1f}s"
    n_ref = sum(1 for k in kinds if k == 1)
    n_sp = len(kinds) - n_ref
    total = (cfg.n_blocks * (n_ref * (t_dense_block + t_score) + n_sp * t_sparse_block)
             + n_ref * t_select)
    tokens = len(kinds) * cfg.batch * cfg.l_full
    return {"value": round(tokens / total, 2), "unit": "tokens/s", "cores": int(cores),
            "kind": "oracle",
            "sample": (f"measured: one packed block ({sum(packed)} tokens) {t_sparse_block:.1f}s, "
                       f"one layer of scoring {t_score:.2f}s, one reduce+select {t_select:.2f}s, "
                       f"{how}; scaled to {cfg.n_blocks} blocks x {len(kinds)} steps "
                       f"({n_ref} refresh, {n_sp} sparse)"),
            "sample_seconds": round(t_sparse_block + t_score + t_select
                                    + (t_dense_block if how.startswith("one") else 0.0), 2),
            "cpu_model": cpu_model, "blas": blas,
            "workload1_full_schedule": {
                "workload": c1.name, "steps": c1.n_steps, "seconds": round(t1_n, 4),
                "tokens_per_s": round(c1.n_steps * c1.l_full / t1_n, 1),
                "seconds_single_thread": round(t1_1, 4) if t1_1 is not None else None,
                "tokens_per_s_single_thread": (round(c1.n_steps * c1.l_full / t1_1, 1)
                                               if t1_1 else None)},
            "workload2_schedule": {
                "workload": c2.name, "steps": c2.n_steps, "refresh_step_s": round(t2_f, 3),
                "sparse_step_s": round(t2_s, 3), "schedule_s": round(t2, 2),
                "tokens_per_s": round(c2.n_steps * c2.l_full / t2, 1),
                "how": f"{n2_f} refresh + {c2.n_steps - n2_f} sparse steps, each kind measured whole once"}}


GEMM_CLASSES = ("GEMM_QKV", "GEMM_OUT", "GEMM_UP", "GEMM_DOWN")   # index = the ROLE template argument
MFMA_CLASSES = ("ATTN",) + GEMM_CLASSES


def kernel_class(name):
    """Timer class of a kernel from its name in a trace: the bf16 GEMM and
    split-K epilogue instantiations carry their projection as the first
    template argument."""
    m = re.search(r"(?:gemm_bf16_nt|splitk_epilogue)<(\d+)", name)
    if m:
        return GEMM_CLASSES[int(m.group(1))]
    if re.search(r"ln_mod_bf16<\d+, true>", name) or "pack_rows" in name:
        return "PACK"
    for sub, cls in (("attn_fwd", "ATTN"), ("score_bf16", "SCORE"), ("score_f32", "SCORE"),
                     ("unpack_", "UNPACK")):
        if sub in name:
            return cls
    return None


def class_units(rows, cls):
    """Launch units of one class in stream order from (id, name, duration) rows:
    [duration, [ids]], a split-K partial launch and its epilogue being one unit
    (one projection)."""
    units = []
    for rid, name, dur in rows:
        if kernel_class(name) != cls:
            continue
        if "splitk_epilogue" in name and units:
            units[-1][0] += dur
            units[-1][1].append(rid)
        else:
            units.append([dur, [rid]])
    return units


def warmup_kinds(res):
    """Step kinds of the untimed warm-up steps (tau = 0 .. warmup - 1)."""
    R = res["config"]["reuse_R"]
    return [1 if t % R == 0 else 2 for t in range(res["warmup"])]


def timed_window(res, cls, units):
    """The units of `cls` issued by exactly the K timed steps, with the step
    kind of each: ATTN and GEMM classes run once per block of every step,
    SCORE once per block of a refresh, PACK / UNPACK once per sparse step."""
    nb = res["config"]["n_blocks"]

    def per_step(kind):
        if cls == "SCORE":
            return nb if kind == 1 else 0
        if cls in ("PACK", "UNPACK"):
            return 1 if kind == 2 else 0
        return nb

    skip = sum(per_step(k) for k in warmup_kinds(res))
    out, i = [], skip
    for k in res["config"]["schedule_kinds"]:
        for _ in range(per_step(k)):
            if i < len(units):
                out.append((k, units[i]))
            i += 1
    return out


def kernel_table(db_path):
    """Launch rows (dispatch id, name, start, end) of a rocprofv3 kernel trace
    and the per-kernel table (calls, average and total duration)."""
    import sqlite3
    con = sqlite3.connect(db_path)
    rows = con.execute("select dispatch_id, name, start, end from kernels order by start").fetchall()
    agg = {}
    for _, name, a, b in rows:
        short = name.split("(")[0].replace("void ", "")
        n, t = agg.get(short, (0, 0))
        agg[short] = (n + 1, t + (b - a))
    lines = [f"{'calls':>7} {'avg_us':>10} {'total_ms':>10}  kernel"]
    for k, (n, t) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        lines.append(f"{n:7d} {t / n / 1e3:10.2f} {t / 1e6:10.2f}  {k}")
    return rows, lines


def summarize_rocprof(db_path, bench_json):
    """Per-kernel table of a rocprofv3 kernel trace of this benchmark, the
    per-class rooflines over exactly the timed steps (dense-layout launches
    of refresh steps and packed launches of sparse steps apart), and the
    dominant class's average against the bench's live HIP-event average."""
    res = json.load(open(bench_json))
    cfg = workload_from_json(res["config"])
    rows, lines = kernel_table(db_path)
    trows = [(rid, name, b - a) for rid, name, a, b in rows]
    full = [cfg.l_full] * cfg.batch
    packed = res["config"]["packed_per_seq"]
    lines += ["", "timed steps, per class and step kind (algorithmic work per launch unit / "
              "average unit duration; a split-K projection is its partial GEMM + epilogue):",
              f"{'class':10s} {'kind':8s} {'units':>6s} {'avg_us':>9s} {'achieved':>10s} {'unit':8s} {'%_of_peak':>9s}"]
    avgs = {}
    for cls in MFMA_CLASSES + ("SCORE", "PACK", "UNPACK"):
        win = timed_window(res, cls, class_units(trows, cls))
        for kind, name in ((1, "refresh"), (2, "sparse")):
            sel = [u for k, u in win if k == kind]
            if not sel:
                continue
            us = sum(u[0] for u in sel) / len(sel) / 1e3
            work = kernel_work(cfg, cls, full if kind == 1 else packed)
            if BOUND[cls] == "mfma":
                ach, unit, peak = work / (us * 1e-6) / 1e12, "TFLOP/s", PEAK_BF16_TFLOPS
            else:
                ach, unit, peak = work / (us * 1e-6) / 1e9, "GB/s", PEAK_HBM_GBS
            lines.append(f"{cls:10s} {name:8s} {len(sel):6d} {us:9.2f} {ach:10.1f} {unit:8s} "
                         f"{100.0 * ach / peak:9.1f}")
        if win:
            avgs[cls] = sum(u[0] for _, u in win) / len(win) / 1e3
    rf = res["roofline"]
    cls = rf["kernel"]
    lines.append("")
    lines.append(f"timed window: {cls} {len(timed_window(res, cls, class_units(trows, cls)))} launch units, "
                 f"avg {avgs.get(cls, float('nan')):.2f} us (bench live HIP-event average "
                 f"{rf['avg_launch_us']:.2f} us over {rf['launches']} launches, every "
                 f"{rf.get('bracketed_every', 1)}th of the class)")
    return "\n".join(lines)


def load_model(cfg, dev, adt):
    """Seeded block weights (every block has its own random stream, so drawing
    them on a thread pool gives the same arrays), copied to the device."""
    import torch
    import workload as W
    from paper_2609_38984_amd import swam
    blocks_np, dblocks = [], []
    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    with ThreadPoolExecutor(workers) as ex:
        for l, b in enumerate(ex.map(lambda i: W.block_weights(cfg, i), range(cfg.n_blocks))):
            if l == 0:
                blocks_np.append(b)
            dblocks.append({k: torch.from_numpy(v).to(dev, adt) for k, v in b.items()})
    return blocks_np, swam.Model(dblocks, adt)


def measure(cfg, model, xs, tembs, steps, warmup, reps):
    """Warm-up, K timed schedule steps, per-kind medians and phase times."""
    import torch
    from paper_2609_38984_amd import swam
    dev = xs[0].device
    n_sched = len(xs)
    y = torch.empty_like(xs[0])
    ctx = swam.Context(cfg)
    ctx.timer_enable(swam.TIMERS, capacity=1 << 15)

    def run(tau, flags=0):
        return ctx.step(model, xs[tau % n_sched], tembs[tau % n_sched], tau, y, flags)

    n_warm = max(warmup, 2)
    warm_kinds = [run(t) for t in range(n_warm)]
    torch.cuda.synchronize()
    phase = {cls: ctx.timer_read(cls) for cls in swam.TIMERS}
    dominant = max(BOUND, key=lambda c: phase[c][1])
    # Each event bracket costs the stream a few microseconds (about 0.2 ms per
    # step with all 28 attention launches bracketed), so the timed region
    # brackets every `stride`-th launch of the dominant class: the largest
    # stride <= 8 dividing its launches per step of every kind, so each step
    # contributes the same launch positions.
    per_step = set()
    for kind in set(warm_kinds):
        n_kind = ctx.timer_read(dominant, kind)[0]
        if n_kind:
            per_step.add(n_kind // warm_kinds.count(kind))
    stride = max(s for s in range(1, 9) if all(n % s == 0 for n in per_step))

    # timed region: exactly K steps, sampled launches of the dominant class bracketed
    ctx.timer_enable([dominant], capacity=max(64, steps * cfg.n_blocks * 2))
    ctx.timer_stride(stride)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    kinds = [run(t) for t in range(steps)]
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start

    full_rows = [cfg.l_full] * cfg.batch
    cu = torch.empty(cfg.batch + 1, dtype=torch.int32, device=dev)
    ctx.export(cu_seqlens=cu)
    cuh = cu.cpu().numpy()
    packed_rows = [int(cuh[b + 1] - cuh[b]) for b in range(cfg.batch)]
    rows_of = {swam.KIND_REFRESH: full_rows, swam.KIND_DENSE: full_rows, swam.KIND_SPARSE: packed_rows}
    # algorithmic work of exactly the bracketed launches, by the kind of their step
    work, n_dom, ms_dom = 0.0, 0, 0.0
    for kind in set(kinds):
        n_kind, ms_kind = ctx.timer_read(dominant, kind)
        work += n_kind * kernel_work(cfg, dominant, rows_of[kind])
        n_dom += n_kind
        ms_dom += ms_kind
    ctx.timer_stride(1)
    bound = BOUND[dominant]
    if bound == "mfma":
        achieved = work / (ms_dom * 1e-3) / 1e12
        peak = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_FP32_TFLOPS
        unit = "TFLOP/s"
    else:
        achieved = work / (ms_dom * 1e-3) / 1e9
        peak = PEAK_HBM_GBS
        unit = "GB/s"
    roofline = {"kernel": dominant, "bound": bound, "achieved": round(achieved, 2), "peak": peak,
                "unit": unit, "frac": round(achieved / peak, 4),
                "traffic": read_traffic(dominant, cfg.name),
                "launches": n_dom, "bracketed_every": stride,
                "avg_launch_us": round(ms_dom * 1e3 / max(n_dom, 1), 2)}

    def median_ms(flags, tau):
        # the paper's protocol: 5 untimed runs, then `reps` timed ones, median
        for _ in range(5):
            run(tau, flags)
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            run(tau, flags)
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return statistics.median(ts)

    ctx.timer_enable([], 1)
    t_dense = median_ms(swam.FORCE_DENSE, 0)
    t_refresh = median_ms(swam.FORCE_REFRESH, 0)
    run(0)                                       # a fresh selection for the sparse medians
    t_sparse = median_ms(0, 1) if cfg.reuse_R > 1 else float("nan")

    def class_times(flags, tau, n=3):
        """(launches, ms) per class and step, every class bracketed by events."""
        ctx.timer_enable(swam.TIMERS, capacity=1 << 14)
        for _ in range(n):
            run(tau, flags)
        got = {c: ctx.timer_read(c) for c in swam.TIMERS}
        ctx.timer_enable([], 1)
        return {c: (k / n, ms / n) for c, (k, ms) in got.items() if k}

    per_kind = {"dense": class_times(swam.FORCE_DENSE, 0), "refresh": class_times(swam.FORCE_REFRESH, 0)}
    if cfg.reuse_R > 1:
        run(0)
        per_kind["sparse"] = class_times(0, 1)
    by_class = class_rooflines(cfg, per_kind, full_rows, packed_rows)
    by_class["hbm"]["SCORE_isolated"] = score_isolated(cfg, ctx)
    in_up = score_in_up(cfg, per_kind)
    if in_up is not None:
        by_class["hbm"]["SCORE_in_up_marginal"] = in_up
    ctx.timer_enable(swam.TIMERS, capacity=1 << 15)
    for t in range(n_sched):
        run(t)
    torch.cuda.synchronize()
    phase_ms = {cls: round(ctx.timer_read(cls)[1] / n_sched, 4) for cls in swam.TIMERS}
    qk_post = None
    if cfg.rope or cfg.qk_norm:
        n_qk, ms_qk = ctx.timer_read("QK_POST")
        if n_qk == 0:
            # applied inside the QKV projection's store (no pass of its own)
            qk_post = {"rope": cfg.rope, "qk_norm": cfg.qk_norm, "launches": 0,
                       "fused_into": "GEMM_QKV"}
        else:
            rows = [full_rows if t % cfg.reuse_R == 0 else packed_rows for t in range(n_sched)]
            work = sum(kernel_work(cfg, "QK_POST", r) * cfg.n_blocks for r in rows)
            gbs = work / (ms_qk * 1e-3) / 1e9
            qk_post = {"rope": cfg.rope, "qk_norm": cfg.qk_norm, "launches": n_qk,
                       "ms_per_step": round(ms_qk / n_sched, 4), "achieved": round(gbs, 1),
                       "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)}
    ctx.timer_enable([], 1)
    over = sum(phase_ms[c] for c in ("SCORE", "REDUCE", "SELECT", "PACK", "UNPACK"))
    # what the overhead costs the schedule: a refresh step's excess over the
    # dense step (scoring overlaps the blocks on a side stream) plus pack and
    # unpack of the sparse steps, per schedule step
    n_ref = sum(1 for t in range(n_sched) if t % cfg.reuse_R == 0)
    exposed = (max(0.0, t_refresh - t_dense) * n_ref / n_sched + phase_ms["PACK"] + phase_ms["UNPACK"])
    tok = cfg.batch * cfg.l_full
    sched_ms = elapsed * 1e3 / steps
    return {
        "elapsed_s": elapsed, "kinds": kinds, "warmup_steps": max(warmup, 2),
        "packed_rows": sum(packed_rows), "packed_per_seq": packed_rows,
        "dense_step_ms": round(t_dense, 4), "refresh_step_ms": round(t_refresh, 4),
        "sparse_step_ms": round(t_sparse, 4), "schedule_step_ms": round(sched_ms, 4),
        "dense_tokens_per_s": round(tok / t_dense * 1e3, 1),
        "sparse_tokens_per_s": round(tok / t_sparse * 1e3, 1) if t_sparse == t_sparse else None,
        "refresh_tokens_per_s": round(tok / t_refresh * 1e3, 1),
        "speedup_sparse_vs_dense": round(t_dense / t_sparse, 3) if t_sparse == t_sparse else None,
        "speedup_schedule_vs_dense": round(t_dense / sched_ms, 3),
        "overhead_pct_of_dense": round(100.0 * over / t_dense, 3),
        "overhead_exposed_pct_of_dense": round(100.0 * exposed / t_dense, 3),
        "overhead_pct_of_schedule_step": round(100.0 * over / sched_ms, 3),
        "phase_ms_per_step": phase_ms, "roofline": roofline, "qk_post": qk_post,
        "roofline_by_class": by_class,
    }


def score_isolated(cfg, ctx, n=None):
    """One layer's scoring per launch, alone on the context stream (swam_score,
    mode A) over a QKV buffer and normalisers of the workload's shape: the
    scorer's own launch time and HBM fraction (in a refresh step the same
    launches overlap the projections on the side stream, which stretches
    them).  Values are random (the work does not depend on them)."""
    import torch
    from paper_2609_38984_amd import swam
    n = n or cfg.n_blocks
    dev = torch.device("cuda:0")
    adt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    d, L = cfg.d_model, cfg.l_full
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    qkv = torch.randn(cfg.batch * L, 3 * d, device=dev, generator=g).to(adt)
    lse = torch.full((cfg.n_scored, cfg.n_act, cfg.n_heads), 8.0, device=dev)
    s = torch.empty(cfg.n_scored * cfg.n_frames * cfg.n_s, device=dev)
    ld = 3 * d
    flat = qkv.view(-1)
    q_act = flat[(cfg.n_ctx + cfg.n_fut) * ld:]
    k_fut = flat[cfg.n_ctx * ld + d:]
    for _ in range(3):
        ctx.score(q_act, L * ld, ld, k_fut, L * ld, ld, s, lse_act=lse)
    # the n launches back to back between one pair of events on the context
    # stream (an event pair around every launch would add its own cost to a
    # launch of about ten microseconds)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(n):
        ctx.score(q_act, L * ld, ld, k_fut, L * ld, ld, s, lse_act=lse)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / n
    gbs = kernel_work(cfg, "SCORE", [cfg.l_full] * cfg.batch) / (us * 1e-6) / 1e9
    return {"us": round(us, 2), "launches": n, "GB/s": round(gbs, 1),
            "frac": round(gbs / PEAK_HBM_GBS, 4)}


def score_in_up(cfg, per_kind):
    """What the scoring of the layers that score in the tail of their MLP up
    projection grid costs the step: the up projection's time in a refresh step
    minus its time in a dense step (the same launches without the scoring
    units), per scored layer, and the scoring's algorithmic bytes over that
    marginal time."""
    up_r = per_kind.get("refresh", {}).get("GEMM_UP")
    up_d = per_kind.get("dense", {}).get("GEMM_UP")
    if not up_r or not up_d:
        return None
    n_side = per_kind["refresh"].get("SCORE", (0, 0.0))[0]   # layers scored on the side stream
    n_in = cfg.n_blocks - int(round(n_side))
    if n_in <= 0:
        return None
    marg_us = (up_r[1] - up_d[1]) * 1e3 / n_in
    out = {"layers_per_refresh": n_in, "marginal_us_per_layer": round(marg_us, 2)}
    if marg_us > 0:
        gbs = kernel_work(cfg, "SCORE", [cfg.l_full] * cfg.batch) / (marg_us * 1e-6) / 1e9
        out["effective_GB/s"] = round(gbs, 1)
    return out


def class_rooflines(cfg, per_kind, full_rows, packed_rows):
    """Per kernel class: average launch time from on-stream HIP events and the
    fraction of its roofline.  MFMA classes (attention and the four
    projections; a split-K projection counts its partial GEMM and epilogue)
    against the bf16 peak, separately for the dense layout (refresh / dense
    steps) and the packed one (sparse steps); scoring, pack and unpack against
    8 TB/s of HBM; reduce and select (latency-bound, at most 2 MB) in us."""
    peak_mfma = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_FP32_TFLOPS
    out = {}
    for kind, rows in (("dense", full_rows), ("sparse", packed_rows)):
        if kind not in per_kind:
            continue
        d = {}
        for cls in MFMA_CLASSES:
            n, ms = per_kind[kind].get(cls, (0, 0.0))
            if not n:
                continue
            us = ms * 1e3 / n
            tf = kernel_work(cfg, cls, rows) / (us * 1e-6) / 1e12
            d[cls] = {"us": round(us, 2), "TFLOP/s": round(tf, 1), "frac": round(tf / peak_mfma, 4)}
        out[kind + "_mfma"] = d
    mem = {}
    for kind, cls, rows in (("refresh", "SCORE", full_rows), ("sparse", "PACK", packed_rows),
                            ("sparse", "UNPACK", packed_rows)):
        n, ms = per_kind.get(kind, {}).get(cls, (0, 0.0))
        if not n:
            if cls == "UNPACK" and cfg.dtype == "bf16" and "sparse" in per_kind:
                # the scatter rides in the last block's MLP down projection store
                mem[cls] = {"launches_per_step": 0, "fused_into": "GEMM_DOWN"}
            continue
        us = ms * 1e3 / n
        gbs = kernel_work(cfg, cls, rows) / (us * 1e-6) / 1e9
        mem[cls] = {"us": round(us, 2), "launches_per_step": round(n, 2), "GB/s": round(gbs, 1),
                    "frac": round(gbs / PEAK_HBM_GBS, 4)}
    out["hbm"] = mem
    out["latency_us_per_refresh"] = {c: round(per_kind["refresh"].get(c, (0, 0.0))[1] * 1e3, 1)
                                     for c in ("REDUCE", "SELECT")}
    return out


def measure_graph(cfg, model, xs, tembs, steps, reps):
    """Schedule and per-kind step times through swam_step_graph (captured once,
    replayed), on a dedicated stream."""
    import torch
    from paper_2609_38984_amd import swam
    n_sched = len(xs)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        y = torch.empty_like(xs[0])
        ctx = swam.Context(cfg, stream=stream)

        def run(tau, flags=0):
            return ctx.step_graph(model, xs[tau % n_sched], tembs[tau % n_sched], tau, y, flags)

        for t in range(max(n_sched, steps)):        # capture every (kind, input) pair once
            run(t)
        stream.synchronize()
        t0 = time.perf_counter()
        for t in range(steps):
            run(t)
        stream.synchronize()
        elapsed = time.perf_counter() - t0

        def median_ms(flags, tau):
            for _ in range(5):
                run(tau, flags)
            ts = []
            for _ in range(reps):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                run(tau, flags)
                e1.record(stream)
                stream.synchronize()
                ts.append(e0.elapsed_time(e1))
            return statistics.median(ts)

        t_dense = median_ms(swam.FORCE_DENSE, 0)
        run(0)
        t_sparse = median_ms(0, 1) if cfg.reuse_R > 1 else float("nan")
    return {"schedule_step_ms": elapsed * 1e3 / steps, "dense_step_ms": t_dense,
            "sparse_step_ms": t_sparse}


def inputs_for(cfg, blocks_np, dev, adt):
    import torch
    import workload as W
    inp = W.make_inputs(cfg, blocks_np[0]["w_qkv"])
    xs = [torch.from_numpy(inp.x(t)).to(dev, adt) for t in range(cfg.n_steps)]
    tembs = [torch.from_numpy(inp.temb(t)).to(dev) for t in range(cfg.n_steps)]
    return inp, xs, tembs


def sweep(args):
    """Retention x reuse sweep of the 2048-wide workload plus the other workloads:
    one markdown row per point (not the driver's JSON line)."""
    import torch
    import workload as W
    dev = torch.device("cuda:0")
    rows = []
    head = ("| workload | retention | R | packed rows | dense ms | refresh ms | sparse ms | "
            "schedule ms/step | sparse/dense | schedule/dense | score+pack % of dense | "
            "exposed % of dense | dominant kernel | MFMA frac | graph dense ms | graph sparse ms | "
            "graph schedule ms/step |")
    print(head)
    print("|" + "---|" * 17)

    def emit(cfg, ret, m, model, xs, tembs):
        g = measure_graph(cfg, model, xs, tembs, cfg.n_steps, args.sweep_reps)
        rf = m["roofline"]
        line = (f"| {cfg.name} | {ret} | {cfg.reuse_R} | {m['packed_rows']} | {m['dense_step_ms']:.2f} | "
                f"{m['refresh_step_ms']:.2f} | {m['sparse_step_ms']:.2f} | {m['schedule_step_ms']:.2f} | "
                f"{m['speedup_sparse_vs_dense']} | {m['speedup_schedule_vs_dense']} | "
                f"{m['overhead_pct_of_dense']:.3f} | {m['overhead_exposed_pct_of_dense']:.3f} | "
                f"{rf['kernel']} | {rf['frac']:.3f} | "
                f"{g['dense_step_ms']:.3f} | {g['sparse_step_ms']:.3f} | {g['schedule_step_ms']:.3f} |")
        print(line, flush=True)

    for n in (1, 2, 3):
        cfg = W.preset(n)
        adt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        blocks_np, model = load_model(cfg, dev, adt)
        _, xs, tembs = inputs_for(cfg, blocks_np, dev, adt)
        emit(cfg, f"{cfg.k_core}+{cfg.k_anchor} of {cfg.n_s}",
             measure(cfg, model, xs, tembs, cfg.n_steps, 2, args.sweep_reps), model, xs, tembs)
        del model, xs
        torch.cuda.empty_cache()
    base = W.preset(4, percent=25)
    blocks_np, model = load_model(base, dev, torch.bfloat16)
    _, xs, tembs = inputs_for(base, blocks_np, dev, torch.bfloat16)
    for pct in (10, 25, 50, 100):
        for R in (1, 2, 4):
            cfg = W.preset(4, percent=pct, reuse_R=R)
            emit(cfg, f"{pct}% ({cfg.k_core}+{cfg.k_anchor})",
                 measure(cfg, model, xs, tembs, cfg.n_steps, 2, args.sweep_reps), model, xs, tembs)
    del model, xs
    torch.cuda.empty_cache()
    cfg = W.preset(5)
    blocks_np, model = load_model(cfg, dev, torch.bfloat16)
    _, xs, tembs = inputs_for(cfg, blocks_np, dev, torch.bfloat16)
    emit(cfg, "mass 0.8", measure(cfg, model, xs, tembs, cfg.n_steps, 2, args.sweep_reps), model, xs,
         tembs)


def second_point(dev, reps):
    """The 2048-wide workload (17,472 tokens, 28 blocks, 32 heads) at 25% + 64
    retention with reuse R = 2: dense / refresh / sparse medians, score+pack
    overhead and per-class rooflines, from the same measurement as the main
    line (two schedule steps of inputs, tau = 0 and 1)."""
    import torch
    import workload as W
    cfg = W.preset(4, percent=25, reuse_R=2)
    log(f"[bench] second point {cfg.name}: L_full={cfg.l_full} d={cfg.d_model}")
    t0 = time.perf_counter()
    blocks_np, model = load_model(cfg, dev, torch.bfloat16)
    inp = W.make_inputs(cfg, blocks_np[0]["w_qkv"])
    xs = [torch.from_numpy(inp.x(t)).to(dev, torch.bfloat16) for t in range(2)]
    tembs = [torch.from_numpy(inp.temb(t)).to(dev) for t in range(2)]
    log(f"[bench] second point resident ({time.perf_counter() - t0:.1f}s)")
    m = measure(cfg, model, xs, tembs, 4, 2, reps)
    n_f = sum(1 for t in range(cfg.n_steps) if t % cfg.reuse_R == 0)
    sched = (n_f * m["refresh_step_ms"] + (cfg.n_steps - n_f) * m["sparse_step_ms"]) / cfg.n_steps
    out = {"workload": cfg.name, "l_full": cfg.l_full, "packed_rows": m["packed_rows"],
           "k_core": cfg.k_core, "k_anchor": cfg.k_anchor, "reuse_R": cfg.reuse_R,
           "schedule_steps": cfg.n_steps,
           "schedule_step_ms_from_medians": round(sched, 4),
           "schedule_tokens_per_s_from_medians": round(cfg.l_full / sched * 1e3, 1)}
    for k in ("dense_step_ms", "refresh_step_ms", "sparse_step_ms", "dense_tokens_per_s",
              "sparse_tokens_per_s", "speedup_sparse_vs_dense", "overhead_pct_of_dense",
              "overhead_exposed_pct_of_dense", "roofline", "roofline_by_class"):
        out[k] = m[k]
    del model, xs
    torch.cuda.empty_cache()
    return out


def overlap_diagnostic(cfg, model, xs, tembs):
    """Mean Overlap (App. C) of the frame score maps V between the first two
    refreshes (cross-step) and between neighbouring frames of the first
    refresh (cross-frame); untimed."""
    import torch
    from paper_2609_38984_amd import swam
    if cfg.reuse_R >= cfg.n_steps:
        return None
    ctx = swam.Context(cfg)
    dev = xs[0].device
    y = torch.empty_like(xs[0])
    F, n_s = cfg.n_frames, cfg.n_s
    vs = []
    for tau in range(cfg.reuse_R + 1):
        ctx.step(model, xs[tau], tembs[tau], tau, y)
        if tau % cfg.reuse_R == 0:
            v = torch.empty(cfg.n_scored * F, n_s, dtype=torch.float32, device=dev)
            ctx.export(v=v)
            vs.append(v)
    out = torch.empty(cfg.n_scored * F, dtype=torch.float32, device=dev)
    ctx.overlap(vs[0], vs[1], out)
    step = float(out.mean().item())
    if F < 2:
        return {"overlap_cross_step": round(step, 4)}
    v0 = vs[0].view(cfg.n_scored, F, n_s)
    p = v0[:, :-1].reshape(-1, n_s).contiguous()
    q = v0[:, 1:].reshape(-1, n_s).contiguous()
    out2 = torch.empty(p.shape[0], dtype=torch.float32, device=dev)
    ctx.overlap(p, q, out2)
    return {"overlap_cross_step": round(step, 4), "overlap_cross_frame": round(float(out2.mean().item()), 4)}


def sampler_bench(args):
    """Closed-loop sampling (embed -> step -> velocity -> cached-velocity merge
    and Euler update) over the workload's schedule: time per sampling step,
    the share of the sampler kernels, and the same with the plain step.
    One JSON line (not the default line)."""
    import torch
    import workload as W
    from paper_2609_38984_amd import swam
    cfg = workload_from_args(args)
    dev = torch.device("cuda:0")
    adt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    c = args.d_latent
    blocks_np, model = load_model(cfg, dev, adt)
    wio = W.latent_io_weights(cfg, c)
    io = swam.LatentIO({k: torch.from_numpy(v).to(dev, adt) for k, v in wio.items()}, adt)
    si = W.make_sampler_inputs(cfg, c)
    n_lat = cfg.batch * (cfg.l_full - cfg.n_ctx)          # rows of v (both branches with pairs)
    n_state = cfg.n_scored * (cfg.l_full - cfg.n_ctx)     # rows of z and the cache
    x = torch.zeros(cfg.batch * cfg.l_full, cfg.d_model, dtype=adt, device=dev)
    for b in range(cfg.batch):
        x[b * cfg.l_full:b * cfg.l_full + cfg.n_ctx] = torch.from_numpy(si.ctx[b]).to(dev, adt)
    y = torch.empty_like(x)
    z0 = torch.from_numpy(si.z0).to(dev)
    z, v, vc = z0.clone(), torch.zeros(n_lat, c, device=dev), torch.zeros(n_state, c, device=dev)
    sig = swam.flow_sigmas(cfg.n_steps)
    tembs = [torch.from_numpy(W.time_embedding(cfg, 1000.0 * sig[t])).to(dev) for t in range(cfg.n_steps)]
    ctx = swam.Context(cfg)

    def run_all():
        z.copy_(z0)
        kinds = []
        for t in range(cfg.n_steps):
            kinds.append(ctx.sample_step(model, io, z, v, vc, x, y, tembs[t], t, sig[t + 1] - sig[t]))
        return kinds

    run_all()
    torch.cuda.synchronize()
    ctx.timer_enable(["SAMPLE"], capacity=1 << 12)
    reps = max(1, args.steps // cfg.n_steps)
    t0 = time.perf_counter()
    for _ in range(reps):
        kinds = run_all()
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    n_sample, ms_sample = ctx.timer_read("SAMPLE")
    ctx.timer_enable([], 1)
    steps = reps * cfg.n_steps
    out = {"mode": "closed-loop sampler", "workload": cfg.name, "d_latent": c,
           "steps": steps, "ms_per_step": round(el * 1e3 / steps, 4),
           "tokens_per_s": round(steps * cfg.batch * cfg.l_full / el, 1),
           "sample_tokens_per_s": round(steps * cfg.n_scored * cfg.l_full / el, 1),
           "cfg_pairs": cfg.cfg_pairs, "guidance": cfg.guidance if cfg.cfg_pairs else None,
           "kinds": kinds,
           "sampler_kernels_ms_per_step": round(ms_sample / steps, 4),
           "sampler_kernels_pct_of_step": round(100.0 * ms_sample / (el * 1e3), 3),
           "latent_tokens": n_lat, "final_z_finite": bool(torch.isfinite(z).all().item())}
    print(json.dumps(out), flush=True)


# sources that define each kernel class (the attention kernel sees only the
# device helpers of common.h; the others also include the launcher header)
KERNEL_SOURCES = {"ATTN": ["k_attn.hip"],
                  "GEMM_QKV": ["k_gemm.hip", "launchers.h"], "GEMM_OUT": ["k_gemm.hip", "launchers.h"],
                  "GEMM_UP": ["k_gemm.hip", "launchers.h"], "GEMM_DOWN": ["k_gemm.hip", "launchers.h"],
                  "SCORE": ["k_score.hip", "launchers.h"], "PACK": ["k_select.hip", "launchers.h"],
                  "UNPACK": ["k_select.hip", "launchers.h"]}


def kernel_source_hash(cls):
    """sha256 over the sources that define a kernel class (and the device-helper header)."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[cls] + ["common.h"]:
        with open(os.path.join(ROOT, "paper_2609_38984_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_file(cls, workload):
    return os.path.join(ROOT, "profiles", f"traffic_{cls.lower()}__{workload}.md")


def summarize_traffic(fetch_db, write_db, bench_json):
    """HBM bytes per launch unit from FETCH_SIZE / WRITE_SIZE counter runs, each
    scaled by its reading for the library's plain copy kernel (copy_chunks:
    rows_full * d * elem bytes read and written per launch), over exactly the
    timed steps, per class and step kind; the dominant class's average over
    all its timed units is what the bench line reports as traffic."""
    import sqlite3
    res = json.load(open(bench_json))
    cfgj = res["config"]
    cfg = workload_from_json(cfgj)
    esz = 2 if res["dtype"] == "bf16" else 4
    copy_bytes = cfgj["batch"] * cfgj["l_full"] * cfgj["d_model"] * esz

    def per_dispatch(db, counter):
        con = sqlite3.connect(db)
        return con.execute("select dispatch_id, name, sum(counter_value) from pmc_events "
                           "where counter_name = ? group by dispatch_id order by dispatch_id",
                           (counter,)).fetchall()

    fetch = per_dispatch(fetch_db, "FETCH_SIZE")
    write = per_dispatch(write_db, "WRITE_SIZE")
    cal_f = [v for _, n, v in fetch if "copy_chunks" in n]
    cal_w = [v for _, n, v in write if "copy_chunks" in n]
    f_fac = copy_bytes / (1024.0 * sum(cal_f) / len(cal_f))
    w_fac = copy_bytes / (1024.0 * sum(cal_w) / len(cal_w))
    full = [cfg.l_full] * cfg.batch
    packed = cfgj["packed_per_seq"]
    lines = [f"calibration: copy_chunks moves {copy_bytes} bytes each way per launch; "
             f"FETCH_SIZE reads {sum(cal_f) / len(cal_f):.1f} KiB (factor {f_fac:.4f}), "
             f"WRITE_SIZE reads {sum(cal_w) / len(cal_w):.1f} KiB (factor {w_fac:.4f})",
             "",
             "timed steps, HBM bytes per launch unit (FETCH + WRITE, calibrated) against the "
             "algorithmic bytes (MFMA classes: operands read once, outputs written once):",
             f"{'class':10s} {'kind':8s} {'units':>6s} {'MB':>9s} {'alg_MB':>9s} {'ratio':>6s}"]
    dom = res["roofline"]["kernel"]
    dom_avg = None
    for cls in MFMA_CLASSES + ("SCORE", "PACK", "UNPACK"):
        wf = timed_window(res, cls, class_units(fetch, cls))
        ww = timed_window(res, cls, class_units(write, cls))
        n = min(len(wf), len(ww))
        if not n:
            continue
        tot = [wf[i][1][0] * 1024.0 * f_fac + ww[i][1][0] * 1024.0 * w_fac for i in range(n)]
        for kind, name in ((1, "refresh"), (2, "sparse")):
            sel = [t for i, t in enumerate(tot) if wf[i][0] == kind]
            if not sel:
                continue
            rows = full if kind == 1 else packed
            alg = algorithmic_bytes(cfg, cls, rows)
            mb = sum(sel) / len(sel) / 1e6
            lines.append(f"{cls:10s} {name:8s} {len(sel):6d} {mb:9.2f} {alg / 1e6:9.2f} {mb * 1e6 / alg:6.2f}")
        if cls == dom:
            dom_avg = sum(tot) / n
    lines += ["",
              f"traffic_per_launch_bytes: {int(dom_avg) if dom_avg else 0}",
              f"kernel_class: {dom}",
              f"workload: {cfgj['workload']}",
              f"source_sha256_16: {kernel_source_hash(dom)}"]
    return "\n".join(lines)


def algorithmic_bytes(cfg, cls, rows_per_seq):
    """Bytes a launch must move at least: memory-bound classes their
    kernel_work; MFMA classes their operands read once and result written once
    (attention: q, k, v and o of every row, lambda; projections: A, B, bias, C,
    and the residual for the gated ones)."""
    if BOUND[cls] == "hbm":
        return kernel_work(cfg, cls, rows_per_seq)
    d, hid, m = cfg.d_model, cfg.mlp_ratio * cfg.d_model, sum(rows_per_seq)
    esz = 2 if cfg.dtype == "bf16" else 4
    if cls == "ATTN":
        return m * 4 * d * esz + m * cfg.n_heads * 4
    n_k = {"GEMM_QKV": (3 * d, d), "GEMM_OUT": (d, d), "GEMM_UP": (hid, d), "GEMM_DOWN": (d, hid)}[cls]
    n, k = n_k
    resid = 2 if cls in ("GEMM_OUT", "GEMM_DOWN") else 1
    return (m * k + n * k + n + resid * m * n) * esz


def read_traffic(cls, workload):
    """Counter-derived bytes per launch if they were taken on the current kernel source."""
    path = traffic_file(cls, workload)
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line:
            k, v = line.split(":", 1)
            vals[k.strip().lstrip("- ")] = v.strip()
    if vals.get("source_sha256_16") != kernel_source_hash(cls):
        return None
    try:
        return int(vals["traffic_per_launch_bytes"])
    except (KeyError, ValueError):
        return None


def summarize_mfma(db_path, bench_json):
    """MFMA-busy share per MFMA kernel class and step kind over the timed
    steps, from one `rocprofv3 --kernel-trace --pmc SQ_VALU_MFMA_BUSY_CYCLES
    SQ_BUSY_CYCLES GRBM_GUI_ACTIVE SQ_INSTS_VALU_MFMA_MOPS_BF16` run of this
    benchmark.  SQ_VALU_MFMA_BUSY_CYCLES counts SIMD-cycles with the matrix
    core busy; it is divided by the launch time x 2.4 GHz x 1024 SIMDs (the
    clock of the 2.5 PFLOP/s peak).  SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 is the
    flops the matrix cores executed (padding of ragged tiles included).
    GRBM_GUI_ACTIVE / 8 XCDs / launch time is the clock the GPU ran at
    (approximate for short launches).  A split-K projection counts its
    partial GEMM and its epilogue."""
    import sqlite3
    res = json.load(open(bench_json))
    cfgj = res["config"]
    cfg = workload_from_json(cfgj)
    con = sqlite3.connect(db_path)
    cnt, names = {}, {}
    for did, name, c, v in con.execute("select dispatch_id, name, counter_name, sum(counter_value) "
                                       "from pmc_events group by dispatch_id, counter_name"):
        cnt.setdefault(did, {})[c] = v
        names[did] = name
    dur = {did: b - a for did, a, b in con.execute("select dispatch_id, start, end from kernels")}
    trows = [(did, names[did], dur.get(did, 0)) for did in sorted(cnt)]
    full = [cfg.l_full] * cfg.batch
    packed = cfgj["packed_per_seq"]
    lines = [f"{'class':10s} {'kind':8s} {'units':>6s} {'avg_us':>8s} {'MFMA_busy_%':>11s} "
             f"{'alg_TFLOP/s':>11s} {'%_of_2.5PF':>10s} {'exec/alg_flops':>14s} {'GRBM_clock_GHz':>14s}"]
    for cls in MFMA_CLASSES:
        win = timed_window(res, cls, class_units(trows, cls))
        for kind, kname in ((1, "refresh"), (2, "sparse")):
            sel = [u for k, u in win if k == kind]
            if not sel:
                continue
            ids = [i for u in sel for i in u[1]]
            t = sum(u[0] for u in sel) * 1e-9
            alg = kernel_work(cfg, cls, full if kind == 1 else packed) * len(sel)
            gui = sum(cnt[i].get("GRBM_GUI_ACTIVE", 0) for i in ids) / 8.0
            busy = sum(cnt[i].get("SQ_VALU_MFMA_BUSY_CYCLES", 0) for i in ids)
            mops = sum(cnt[i].get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0) for i in ids)
            lines.append(f"{cls:10s} {kname:8s} {len(sel):6d} {t / len(sel) * 1e6:8.1f} "
                         f"{100.0 * busy / (t * 2.4e9 * 1024):11.1f} {alg / t / 1e12:11.1f} "
                         f"{100.0 * alg / t / 1e12 / PEAK_BF16_TFLOPS:10.1f} {mops * 512 / alg:14.3f} "
                         f"{gui / t / 1e9:14.2f}")
    return "\n".join(lines)


def library_comparison(args):
    """Same-process comparison with the libraries torch ships, at the workload's
    dense and packed row counts: our attention and projections (per-class HIP
    events around the launches of swam_block, one block, 30 calls) against
    torch's flash and memory-efficient SDPA (same heads, head dim 64, one
    sequence, no normaliser output) and F.linear (hipBLASLt; bias only, where
    ours also fuses GELU or gate + residual).  Two interleaved passes; ours are
    averages over the bracketed launches, the libraries' over 30 back-to-back
    calls.  Only the comparison calls the libraries; the step never does."""
    import torch
    import workload as W
    from paper_2609_38984_amd import swam
    from torch.nn.attention import SDPBackend, sdpa_kernel
    cfg = workload_from_args(args).replace(n_blocks=1)
    if cfg.dtype != "bf16" or cfg.batch != 1 or cfg.t_pack_fixed is None:
        sys.exit("--libcmp: bf16 workloads of one sequence with a fixed token budget only")
    dev = torch.device("cuda:0")
    d, hid, nh = cfg.d_model, cfg.mlp_ratio * cfg.d_model, cfg.n_heads
    blocks_np, model = load_model(cfg, dev, torch.bfloat16)
    wts = model.blocks[0]
    temb = torch.from_numpy(W.timestep_embedding(cfg, 0)).to(dev)
    classes = ["ATTN", "GEMM_QKV", "GEMM_OUT", "GEMM_UP", "GEMM_DOWN"]
    reps = 30
    gen = torch.Generator(device=dev).manual_seed(cfg.seed)

    def ours(rows):
        ctx = swam.Context(cfg)
        x = torch.randn(rows, d, device=dev, generator=gen).to(torch.bfloat16)
        cu = torch.tensor([0, rows], dtype=torch.int32, device=dev)
        lse = torch.empty(rows, nh, dtype=torch.float32, device=dev)
        qkv = torch.empty(rows, 3 * d, dtype=torch.bfloat16, device=dev)
        for i in range(3 + reps):
            if i == 3:
                torch.cuda.synchronize()
                ctx.timer_enable(classes, capacity=8 * reps)
            ctx.block(wts, temb, x.clone(), rows, cu, 1, lse, qkv)
        torch.cuda.synchronize()
        res = {}
        for c in classes:
            n, ms = ctx.timer_read(c)
            res[c] = 1000.0 * ms / n
        return res

    def timed(fn):
        # back-to-back calls between one pair of events: the host's launch
        # latency stays hidden behind the queue, which favours the library
        # (ours carry an event pair around every launch)
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1000.0 / reps

    def libs(rows):
        res = {}
        q, k, v = (torch.randn(1, nh, rows, 64, device=dev, generator=gen).to(torch.bfloat16)
                   for _ in range(3))
        for name, be in (("ATTN_flash", SDPBackend.FLASH_ATTENTION),
                         ("ATTN_efficient", SDPBackend.EFFICIENT_ATTENTION)):
            try:
                with sdpa_kernel([be]):
                    res[name] = timed(lambda: torch.nn.functional.scaled_dot_product_attention(q, k, v))
            except RuntimeError as ex:
                res[name] = f"unavailable: {str(ex)[:60]}"
        lin = torch.nn.functional.linear
        for c, (kk, nn) in (("GEMM_QKV", (d, 3 * d)), ("GEMM_OUT", (d, d)), ("GEMM_UP", (d, hid)),
                            ("GEMM_DOWN", (hid, d))):
            a = torch.randn(rows, kk, device=dev, generator=gen).to(torch.bfloat16)
            w = (torch.randn(nn, kk, device=dev, generator=gen) * kk ** -0.5).to(torch.bfloat16)
            b = torch.zeros(nn, device=dev, dtype=torch.bfloat16)
            res[c + "_hipblaslt"] = timed(lambda: lin(a, w, b))
        return res

    out = {"mode": "library comparison", "workload": cfg.name, "reps": reps, "passes": []}
    for p in range(2):
        row = {}
        for kind, rows in (("dense", cfg.l_full), ("packed", cfg.t_pack_fixed)):
            o, l_ = ours(rows), libs(rows)
            row[kind] = {"rows": rows, "ours_us": {c: round(v, 2) for c, v in o.items()},
                         "library_us": {c: (round(v, 2) if isinstance(v, float) else v)
                                        for c, v in l_.items()}}
            for c in classes:
                work = kernel_work(cfg, c, [rows])
                lib = [v for n, v in l_.items() if n.startswith(c + "_") and isinstance(v, float)]
                best = min(lib) if lib else float("nan")
                log(f"[libcmp] pass {p} {kind:6s} {c:9s} ours {o[c]:8.1f} us "
                    f"({work / o[c] / 1e6:6.1f} TFLOP/s)  library {best:8.1f} us "
                    f"({work / best / 1e6:6.1f} TFLOP/s)  ours/library {o[c] / best:5.2f}")
        out["passes"].append(row)
    print(json.dumps(out))


def workload_from_json(cj):
    import workload as W
    for n in (1, 2, 3, 5):
        c = W.preset(n)
        if c.name == cj["workload"]:
            return c
    for pct in (10, 25, 50, 100):
        for R in (1, 2, 4):
            c = W.preset(4, percent=pct, reuse_R=R)
            if c.name == cj["workload"]:
                return c
    raise KeyError(cj["workload"])


def main():
    if len(sys.argv) > 1 and sys.argv[1] == "--mfma":
        print(summarize_mfma(sys.argv[2], sys.argv[3]))
        return
    if len(sys.argv) > 1 and sys.argv[1] == "--kernels":
        print("\n".join(kernel_table(sys.argv[2])[1]))
        return
    if len(sys.argv) > 1 and sys.argv[1] == "--summarize":
        print(summarize_rocprof(sys.argv[2], sys.argv[3]))
        return
    if len(sys.argv) > 1 and sys.argv[1] == "--traffic":
        print(summarize_traffic(sys.argv[2], sys.argv[3], sys.argv[4]))
        return
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--percent", type=int, default=25, help="retention for workload 4")
    ap.add_argument("--reuse", type=int, default=0, help="override the reuse interval R")
    ap.add_argument("--reps", type=int, default=30,
                    help="timed repetitions per step kind for the medians (after 5 untimed)")
    ap.add_argument("--sweep-reps", type=int, default=5, help="the same, per sweep workload")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-second-point", action="store_true",
                    help="skip the 2048-wide 25%% / R = 2 point of the default line")
    ap.add_argument("--sweep", action="store_true", help="markdown table over all workloads")
    ap.add_argument("--sampler", action="store_true",
                    help="closed-loop sampling with the cached-velocity merge (own JSON line)")
    ap.add_argument("--d-latent", type=int, default=16, help="latent channels for --sampler")
    ap.add_argument("--libcmp", action="store_true",
                    help="our attention and projections against torch's SDPA and F.linear, "
                         "same process (own JSON line)")
    ap.add_argument("--rope", action="store_true",
                    help="backbone variant: rotary embedding at the original positions")
    ap.add_argument("--qk-norm", action="store_true", help="backbone variant: per-head QK-norm")
    ap.add_argument("--guidance", type=float, default=None,
                    help="classifier-free guidance pairs with this scale (the batch doubles)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "one GPU only: the step is single-GPU "
                          "data parallel work with no collectives; run with --gpus 1"}))
        sys.exit(2)

    import torch
    torch.cuda.set_device(0)
    if args.sweep:
        sweep(args)
        return
    if args.sampler:
        sampler_bench(args)
        return
    if args.libcmp:
        library_comparison(args)
        return
    cfg = workload_from_args(args)
    dev = torch.device("cuda:0")
    adt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    log(f"[bench] workload {cfg.name}: B={cfg.batch} L_full={cfg.l_full} d={cfg.d_model} "
        f"blocks={cfg.n_blocks} K_c+K_s={cfg.k_core}+{cfg.k_anchor} R={cfg.reuse_R}")
    t0 = time.perf_counter()
    blocks_np, model = load_model(cfg, dev, adt)
    inp, xs, tembs = inputs_for(cfg, blocks_np, dev, adt)
    log(f"[bench] inputs resident in HBM ({time.perf_counter() - t0:.1f}s)")
    m = measure(cfg, model, xs, tembs, args.steps, args.warmup, args.reps)
    log(f"[bench] timed {args.steps} steps in {m['elapsed_s'] * 1e3:.2f} ms; kinds {m['kinds']}; "
        f"dominant {m['roofline']['kernel']}")
    tok = cfg.batch * cfg.l_full
    out = {
        "metric": METRIC, "value": round(args.steps * tok / m["elapsed_s"], 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": m["warmup_steps"],
        "ms_per_step": round(m["elapsed_s"] * 1e3 / args.steps, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": cfg.name, "batch": cfg.batch, "l_full": cfg.l_full,
                   "d_model": cfg.d_model, "n_blocks": cfg.n_blocks,
                   "frames": f"{cfg.n_frames}x{cfg.frame_h}x{cfg.frame_w}",
                   "n_ctx": cfg.n_ctx, "n_act": cfg.n_act,
                   "k_core": cfg.k_core, "k_anchor": cfg.k_anchor,
                   "mass_threshold": cfg.mass_threshold, "reuse_R": cfg.reuse_R,
                   "rope": cfg.rope, "qk_norm": cfg.qk_norm, "cfg_pairs": cfg.cfg_pairs,
                   "guidance": cfg.guidance if cfg.cfg_pairs else None,
                   "packed_rows": m["packed_rows"], "packed_per_seq": m["packed_per_seq"],
                   "schedule_kinds": m["kinds"]},
    }
    for k in ("dense_step_ms", "refresh_step_ms", "sparse_step_ms", "dense_tokens_per_s",
              "sparse_tokens_per_s", "refresh_tokens_per_s", "speedup_sparse_vs_dense",
              "speedup_schedule_vs_dense", "overhead_pct_of_dense", "overhead_exposed_pct_of_dense",
              "overhead_pct_of_schedule_step", "phase_ms_per_step", "roofline", "roofline_by_class"):
        out[k] = m[k]
    if m["qk_post"] is not None:
        out["qk_post"] = m["qk_post"]
    out["selection_overlap"] = overlap_diagnostic(cfg, model, xs, tembs)
    if args.config == 3 and not args.no_second_point and not (args.rope or args.qk_norm
                                                              or args.guidance is not None):
        del model, xs
        torch.cuda.empty_cache()
        out["point_d2048_r25_R2"] = second_point(dev, args.reps)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(cfg, m["kinds"], blocks_np, inp)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
