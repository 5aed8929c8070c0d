// C ABI of libswam: validation, workspace, the five parts of the sparse
// denoising step and the step orchestrator.  Every device pointer argument
// is owned by the caller; the context owns one workspace arena allocated at
// creation.  All work is enqueued on the context's stream.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <numeric>
#include <new>
#include <string>
#include <vector>

#include "../../include/swam.h"
#include "launchers.h"

#include <cmath>

using namespace swam;

namespace {

thread_local std::string g_err;

struct Derived {
  int64_t n_s, g, l_full, rows_full, k_max, k_eff, d, hidden, esz, t_pack_fixed;
  int64_t n_scored;   // sequences that are scored and selected (the conditional half with pairs)
  int64_t splitk_floats;  // fp32 workspace of the split-K GEMM path (bf16 only)
  int mass_num, mass_den;
};

// workspace layout (offsets into one arena)
struct Layout {
  size_t qkv, h, o, u, xp, lse, mod, alpha, rope, splitk, lse_act, lse_part, s_all, q, qd, core, v, a, vall,
      fsum, fent, pool, corefl, keep_idx, keep_cnt, keep, pack_pos, gather, cu_packed, cu_dense, total;
};

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

int fail(std::string* err, int code, const std::string& msg) {
  if (err) *err = msg;
  return code;
}

// theta = num / den reduced from num / 1000, num the integer nearest to
// 1000 theta: the product of the float32 threshold and 1000 is exact in
// double and never halfway between integers; num = 0 (theta < 0.0005) keeps
// one core token per frame (gcd(0, 1000) = 1000 gives 0 / 1, den > 0 still
// marks mass-threshold mode)
void mass_fraction(float theta, int* num, int* den) {
  const int n = (int)llround((double)theta * 1000.0);
  const int gg = std::gcd(n, 1000);
  *num = n / gg;
  *den = 1000 / gg;
}

int derive(const swam_config* c, Derived* dv, std::string* err) {
  if (!c) return fail(err, SWAM_E_INVALID, "config is NULL");
  if (c->dtype != SWAM_F32 && c->dtype != SWAM_BF16)
    return fail(err, SWAM_E_DTYPE, "dtype must be SWAM_F32 or SWAM_BF16");
  if (c->batch < 1 || c->batch > SWAM_MAX_BATCH)
    return fail(err, SWAM_E_SHAPE, "batch must be in [1, 64]");
  if (c->head_dim != 64) return fail(err, SWAM_E_SHAPE, "head_dim must be 64");
  if (c->n_heads < 1 || c->d_model != c->n_heads * 64)
    return fail(err, SWAM_E_INVALID, "d_model must equal n_heads * 64");
  if (c->mlp_ratio < 1 || c->mlp_ratio > 16) return fail(err, SWAM_E_SHAPE, "mlp_ratio in [1, 16]");
  if (c->n_blocks < 1 || c->n_blocks > SWAM_MAX_BLOCKS)
    return fail(err, SWAM_E_SHAPE, "n_blocks must be in [1, 64]");
  if (c->d_temb < 1 || c->d_temb > 1024) return fail(err, SWAM_E_SHAPE, "d_temb in [1, 1024]");
  if (c->n_ctx < 0) return fail(err, SWAM_E_INVALID, "n_ctx < 0");
  if (c->n_frames < 1 || c->n_frames > SWAM_MAX_FRAMES)
    return fail(err, SWAM_E_SHAPE, "n_frames must be in [1, 64]");
  if (c->frame_h < 1 || c->frame_w < 1) return fail(err, SWAM_E_INVALID, "frame size < 1");
  const int64_t n_s = (int64_t)c->frame_h * c->frame_w;
  if (n_s < 2 || n_s > SWAM_MAX_NS)
    return fail(err, SWAM_E_SHAPE, "tokens per frame must be in [2, 4096]");
  if (c->n_act < 1 || c->n_act % c->n_frames)
    return fail(err, SWAM_E_INVALID, "n_act must be a positive multiple of n_frames");
  const int64_t g = c->n_act / c->n_frames;
  if (g > 16) return fail(err, SWAM_E_SHAPE, "at most 16 action queries per frame group");
  if (!(c->mass_threshold >= 0.0f && c->mass_threshold <= 1.0f))
    return fail(err, SWAM_E_INVALID, "mass_threshold must be in [0, 1]");
  if (c->k_anchor < 0 || c->k_anchor >= n_s)
    return fail(err, SWAM_E_INVALID, "k_anchor must be in [0, N_s)");
  if (c->mass_threshold == 0.0f && (c->k_core < 0 || c->k_core + c->k_anchor > n_s))
    return fail(err, SWAM_E_INVALID, "k_core + k_anchor must be in [0, N_s]");
  if (c->k_layer < 1) return fail(err, SWAM_E_INVALID, "k_layer must be >= 1");
  if (!(c->cv_penalty >= 0.0f) || !isfinite(c->cv_penalty))
    return fail(err, SWAM_E_INVALID, "cv_penalty must be finite and >= 0");
  if (c->reuse_R < 1) return fail(err, SWAM_E_INVALID, "reuse_R must be >= 1");
  if (c->rope != 0 && c->rope != 1) return fail(err, SWAM_E_INVALID, "rope must be 0 or 1");
  if (c->qk_norm != 0 && c->qk_norm != 1) return fail(err, SWAM_E_INVALID, "qk_norm must be 0 or 1");
  if (c->cfg_pairs != 0 && c->cfg_pairs != 1)
    return fail(err, SWAM_E_INVALID, "cfg_pairs must be 0 or 1");
  if (c->cfg_pairs && c->batch % 2)
    return fail(err, SWAM_E_SHAPE, "guidance pairs need an even batch");
  if (!std::isfinite(c->guidance)) return fail(err, SWAM_E_INVALID, "guidance must be finite");
  const int64_t d = c->d_model;
  if (c->dtype == SWAM_BF16 && d > 4096) return fail(err, SWAM_E_SHAPE, "bf16 d_model <= 4096");
  const int64_t l_full = c->n_ctx + (int64_t)c->n_frames * n_s + c->n_act;
  const int64_t rows = (int64_t)c->batch * l_full;
  if (rows >= (1ll << 30)) return fail(err, SWAM_E_SHAPE, "batch * tokens exceeds 2^30");
  // the bf16 attention addresses the QKV buffer with 32-bit element offsets
  if (c->dtype == SWAM_BF16 && rows * 3 * d >= (1ll << 31))
    return fail(err, SWAM_E_SHAPE, "batch * tokens * 3 * d_model must stay below 2^31");
  dv->n_s = n_s;
  dv->n_scored = c->cfg_pairs ? c->batch / 2 : c->batch;
  // split-K partial sums: up to 8 slices of the widest projection, at most 128 MB
  dv->splitk_floats = c->dtype == SWAM_BF16
      ? std::min<int64_t>(8 * rows * std::max<int64_t>(3 * d, (int64_t)c->mlp_ratio * d), 32ll << 20)
      : 0;
  dv->g = g;
  dv->l_full = l_full;
  dv->rows_full = rows;
  dv->d = d;
  dv->hidden = (int64_t)c->mlp_ratio * d;
  dv->esz = c->dtype == SWAM_BF16 ? 2 : 4;
  dv->k_eff = std::min(c->k_layer, c->n_blocks);
  if (c->mass_threshold > 0.0f) {
    mass_fraction(c->mass_threshold, &dv->mass_num, &dv->mass_den);
    dv->k_max = n_s;
    dv->t_pack_fixed = -1;
  } else {
    dv->mass_num = 0;
    dv->mass_den = 0;
    dv->k_max = std::max<int64_t>(1, c->k_core + c->k_anchor);
    dv->t_pack_fixed = c->n_ctx + (int64_t)c->n_frames * (c->k_core + c->k_anchor) + c->n_act;
  }
  return SWAM_OK;
}

Layout layout_for(const swam_config* c, const Derived& dv) {
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return o;
  };
  const int64_t R = dv.rows_full, B = c->batch, F = c->n_frames, Lb = c->n_blocks;
  const int64_t chunks = (dv.l_full + 255) / 256;
  // one QKV / lambda slot: a refresh scores each layer right after its
  // attention, before the next block overwrites the slot
  L.qkv = take(R * 3 * dv.d * dv.esz);
  L.h = take(R * dv.d * dv.esz);
  L.o = take(R * dv.d * dv.esz);
  L.u = take(R * dv.hidden * dv.esz);
  L.xp = take(R * dv.d * dv.esz);
  L.lse = take(R * c->n_heads * 4);
  L.mod = take(Lb * 6 * dv.d * 4);
  L.alpha = take(16 * 4);
  // positions up to batch * l_full - 1: a cu_seqlens sequence of swam_block may
  // span every row of the workspace
  L.rope = take(c->rope ? dv.rows_full * 32 * 8 : 0);
  L.splitk = take(dv.splitk_floats * 4);
  L.lse_act = take(B * c->n_act * c->n_heads * 4);
  L.lse_part = take(B * chunks * c->n_act * c->n_heads * 2 * 4);
  L.s_all = take(B * Lb * F * dv.n_s * 4);
  L.q = take(B * Lb * 4);
  L.qd = take(B * Lb * 8);
  L.core = take(B * dv.k_eff * 4);
  L.v = take(B * F * dv.n_s * 4);
  L.a = take(B * dv.n_s * 4);
  L.vall = take(B * F * dv.n_s * 8);
  L.fsum = take((B * Lb * F + 2 * B) * 8);
  L.fent = take(B * Lb * F * 8);
  L.pool = take(B * dv.n_s);
  L.corefl = take(B * F * dv.n_s);
  L.keep_idx = take(B * F * dv.k_max * 4);
  L.keep_cnt = take(B * F * 4);
  L.keep = take(R * 4);
  L.pack_pos = take(R * 4);
  L.gather = take(R * 4);
  L.cu_packed = take((B + 1) * 4);
  L.cu_dense = take((B + 1) * 4);
  L.total = off;
  return L;
}

}  // namespace

struct swam_ctx {
  swam_config cfg;
  Derived dv;
  Layout lay;
  hipStream_t st = nullptr;
  int device = 0;
  char* arena = nullptr;
  int32_t* host_cu = nullptr;   // pinned
  hipEvent_t order_ev = nullptr; // orders a newly bound stream after the previous one
  // a refresh scores layer l on `side` while the context stream runs the rest
  // of block l; the next block's QKV projection waits for it (ev_score).  An
  // out-of-place sparse step copies the pruned rows on `side` during the
  // blocks and joins it (ev_score) before the scatter of the packed rows.
  hipStream_t side = nullptr;
  hipEvent_t ev_attn = nullptr, ev_score = nullptr;
  bool score_pending = false;
  bool sel_valid = false, scores_valid = false;
  int64_t packed_rows = 0;
  std::string err;
  // timers
  uint32_t tmask = 0;
  int tcap = 0, tused = 0;
  int tstride = 1;                    // bracket every tstride-th launch of a class
  int64_t tcount[SWAM_T_COUNT] = {};  // launches per class since enable / reset
  int step_kind = SWAM_KIND_NONE;     // kind of the step being enqueued
  std::vector<hipEvent_t> ev;   // 2 per slot
  std::vector<int> ev_cls;
  std::vector<int> ev_kind;     // step kind per slot
  // captured steps (swam_step_graph)
  struct GraphEntry {
    int kind;
    const void* x;
    const void* y;
    const float* temb;
    uint64_t wsig;
    int64_t packed;
    hipGraphExec_t exec;
  };
  std::vector<GraphEntry> graphs;
  bool capturing = false;

  template <typename T> T* ptr(size_t off) { return (T*)(arena + off); }
};

namespace {

int set_err(swam_ctx* c, int code, const std::string& msg) {
  if (c) c->err = msg; else g_err = msg;
  return code;
}

int hip_check(swam_ctx* c, hipError_t e, const char* what) {
  if (e == hipSuccess) return SWAM_OK;
  return set_err(c, SWAM_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define SWAM_HIP(ctx, expr, what)                        \
  do {                                                   \
    const int rc_ = hip_check((ctx), (expr), (what));    \
    if (rc_ != SWAM_OK) return rc_;                      \
  } while (0)

// brackets one launch (or phase) of a timed class with events on a stream
// (the context stream unless given)
struct Timed {
  swam_ctx* c;
  hipStream_t s;
  int slot = -1;
  Timed(swam_ctx* ctx, int cls) : Timed(ctx, cls, ctx->st) {}
  Timed(swam_ctx* ctx, int cls, hipStream_t on) : c(ctx), s(on) {
    if (c->capturing || !((c->tmask >> cls) & 1u)) return;
    if (c->tcount[cls]++ % c->tstride != 0 || c->tused >= c->tcap) return;
    slot = c->tused++;
    c->ev_cls[slot] = cls;
    c->ev_kind[slot] = c->step_kind;
    (void)hipEventRecord(c->ev[2 * slot], s);
  }
  ~Timed() {
    if (slot >= 0) (void)hipEventRecord(c->ev[2 * slot + 1], s);
  }
};

// the context stream waits for the scoring launched on the side stream
int join_score(swam_ctx* c) {
  if (!c->score_pending) return SWAM_OK;
  c->score_pending = false;
  SWAM_HIP(c, hipStreamWaitEvent(c->st, c->ev_score, 0), "join scoring");
  return SWAM_OK;
}

// out-of-place sparse step: the pruned rows of y_full are x_full's whatever
// the blocks compute, so they are copied on the side stream while the blocks
// run; the scatter of the packed rows waits for it (ev_score)
int fork_pruned_copy(swam_ctx* c, const void* x_full, void* y_full) {
  SWAM_HIP(c, hipEventRecord(c->ev_attn, c->st), "fork pruned-row copy");
  SWAM_HIP(c, hipStreamWaitEvent(c->side, c->ev_attn, 0), "fork pruned-row copy");
  {
    Timed t(c, SWAM_T_COPY, c->side);
    SWAM_HIP(c, launch_copy_pruned(x_full, y_full, c->ptr<int32_t>(c->lay.pack_pos),
                                   c->dv.rows_full, c->dv.d * c->dv.esz, c->side), "pruned-row copy");
  }
  SWAM_HIP(c, hipEventRecord(c->ev_score, c->side), "pruned-row copy done");
  return SWAM_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// NULL or not 16-byte aligned (the kernels read weights in 16-byte vectors)
bool bad_block(const swam_block_weights* w) {
  if (!w) return true;
  const void* p[10] = {w->w_ada, w->b_ada, w->w_qkv, w->b_qkv, w->w_o,
                       w->b_o,   w->w_1,   w->b_1,   w->w_2,   w->b_2};
  for (const void* q : p)
    if (!q || !aligned16(q)) return true;
  return false;
}

// one block in place on x [n_rows][d]; mod = this block's [6][d] modulation
// pos_mode (rope only): 0 = dense layout, 1 = packed rows of the cached
// selection (original positions), 2 = index inside the cu_seqlens sequence.
// score (refresh only): this layer's action-to-future scores, launched right
// after the attention while the layer's q, k and lambda are fresh in cache
// pack_src (first block of a sparse step): x is filled from the gather-pack of
// pack_src (the full latent) by the block's first LayerNorm kernel itself;
// pruned_dst (with pack_src, out of place): the pruned rows of pack_src are
// copied into it on the side stream, forked after that LayerNorm so the copy
// overlaps the QKV projection rather than the pack
// score_in_up (with score): the scoring runs in the tail of the MLP up
// projection's grid instead of on the side stream (no fork or join)
// scatter_to (bf16, last block of a sparse step): the MLP down projection
// stores row r of its result into scatter_to at the cached gather position of
// r (the scatter back into the full latent) instead of into x
int run_block(swam_ctx* c, const swam_block_weights* w, const float* mod, void* x,
              int64_t n_rows, const int32_t* cu, int n_seqs, float* lse_out, void* qkv,
              int pos_mode, const ScoreArgs* score = nullptr, const void* pack_src = nullptr,
              void* pruned_dst = nullptr, bool score_in_up = false, void* scatter_to = nullptr) {
  const int dt = c->cfg.dtype;
  const int64_t d = c->dv.d, hid = c->dv.hidden;
  void* h = c->ptr<char>(c->lay.h);
  void* o = c->ptr<char>(c->lay.o);
  void* u = c->ptr<char>(c->lay.u);
  hipStream_t st = c->st;
  float* sk = c->ptr<float>(c->lay.splitk);
  const int64_t sk_n = c->dv.splitk_floats;
  const float *sh1 = mod, *sc1 = mod + d, *g1 = mod + 2 * d;
  const float *sh2 = mod + 3 * d, *sc2 = mod + 4 * d, *g2 = mod + 5 * d;
  if (n_rows <= 0) return SWAM_OK;
  if (pack_src) {
    {
      Timed t(c, SWAM_T_PACK);
      SWAM_HIP(c, launch_ln_mod_gather(dt, pack_src, c->ptr<int32_t>(c->lay.gather), x, h, sh1,
                                       sc1, n_rows, (int)d, st), "pack + ln_mod");
    }
    if (pruned_dst)
      if (int rc = fork_pruned_copy(c, pack_src, pruned_dst)) return rc;
  } else {
    Timed t(c, SWAM_T_LNMOD);
    SWAM_HIP(c, launch_ln_mod(dt, x, h, sh1, sc1, n_rows, (int)d, st), "ln_mod");
  }
  // the previous layer's scoring (side stream) still reads the QKV slot and
  // the normalisers: this block's projection and attention overwrite them
  if (int rc = join_score(c)) return rc;
  if (c->cfg.rope || c->cfg.qk_norm) {
    // QKV projection with the QK-norm / rotary embedding of q and k (fused
    // into the projection's store where the shape allows)
    QkPost qp;
    qp.d = (int)d;
    qp.pos_mode = pos_mode;
    qp.gather = c->ptr<int32_t>(c->lay.gather);
    qp.cu = cu;
    qp.n_seqs = n_seqs;
    qp.l_full = (int)c->dv.l_full;
    qp.tab = c->cfg.rope ? c->ptr<float2>(c->lay.rope) : nullptr;
    qp.n_pos = (int)c->dv.rows_full;
    qp.qk_norm = c->cfg.qk_norm;
    Timed t(c, SWAM_T_GEMM_QKV);
    SWAM_HIP(c, launch_gemm_qkv(dt, h, d, w->w_qkv, d, w->b_qkv, qkv, 3 * d, n_rows, 3 * d, d, qp,
                                st, sk, sk_n), "gemm qkv + qk post");
  } else {
    Timed t(c, SWAM_T_GEMM_QKV);
    SWAM_HIP(c, launch_gemm(dt, ROLE_QKV, h, d, w->w_qkv, d, w->b_qkv, nullptr, qkv, 3 * d,
                            n_rows, 3 * d, d, st, sk, sk_n), "gemm qkv");
  }
  {
    Timed t(c, SWAM_T_ATTN);
    SWAM_HIP(c, launch_attention(dt, qkv, o, lse_out, cu, n_seqs, n_rows, c->cfg.n_heads, st),
             "attention");
  }
  if (score && !score_in_up) {
    // fork: the scores of this layer run on the side stream, concurrently
    // with the rest of the block (memory-bound next to MFMA-bound GEMMs)
    SWAM_HIP(c, hipEventRecord(c->ev_attn, st), "fork scoring");
    SWAM_HIP(c, hipStreamWaitEvent(c->side, c->ev_attn, 0), "fork scoring");
    {
      Timed t(c, SWAM_T_SCORE, c->side);
      SWAM_HIP(c, launch_score(dt, *score, c->side), "score");
    }
    SWAM_HIP(c, hipEventRecord(c->ev_score, c->side), "scoring done");
    c->score_pending = true;
  }
  {
    Timed t(c, SWAM_T_GEMM_OUT);
    SWAM_HIP(c, launch_gemm(dt, ROLE_OUT, o, d, w->w_o, d, w->b_o, g1, x, d,
                            n_rows, d, d, st, sk, sk_n), "gemm out");
  }
  {
    Timed t(c, SWAM_T_LNMOD);
    SWAM_HIP(c, launch_ln_mod(dt, x, h, sh2, sc2, n_rows, (int)d, st), "ln_mod 2");
  }
  if (score && score_in_up) {
    // this layer's q, k and lambda stay in place until the next block's QKV
    // projection, which the stream orders after this launch
    Timed t(c, SWAM_T_GEMM_UP);
    SWAM_HIP(c, launch_gemm_up_scored(h, d, w->w_1, d, w->b_1, u, hid, n_rows, hid, d, *score,
                                      st, sk ? sk_n : 0), "gemm up + scoring");
  } else {
    Timed t(c, SWAM_T_GEMM_UP);
    SWAM_HIP(c, launch_gemm(dt, ROLE_UP, h, d, w->w_1, d, w->b_1, nullptr, u, hid, n_rows,
                            hid, d, st, sk, sk_n), "gemm up");
  }
  {
    Timed t(c, SWAM_T_GEMM_DOWN);
    SWAM_HIP(c, launch_gemm(dt, ROLE_DOWN, u, hid, w->w_2, hid, w->b_2, g2, x, d,
                            n_rows, d, hid, st, sk, sk_n, scatter_to,
                            scatter_to ? c->ptr<int32_t>(c->lay.gather) : nullptr),
             scatter_to ? "gemm down + unpack" : "gemm down");
  }
  return SWAM_OK;
}

int run_adaln(swam_ctx* c, const swam_block_weights* blocks, int n_blk, const float* temb) {
  AdalnArgs a{};
  for (int i = 0; i < n_blk; ++i) {
    a.w[i] = blocks[i].w_ada;
    a.b[i] = blocks[i].b_ada;
  }
  Timed t(c, SWAM_T_ADALN);
  SWAM_HIP(c, launch_adaln(c->cfg.dtype, a, n_blk, temb, c->cfg.d_temb, (int)(6 * c->dv.d),
                           c->ptr<float>(c->lay.mod), c->st), "adaln");
  return SWAM_OK;
}

// on: the stream to enqueue on (the context stream when NULL)
int run_reduce(swam_ctx* c, const float* s_all, hipStream_t on = nullptr) {
  const swam_config& cf = c->cfg;
  const hipStream_t st = on ? on : c->st;
  ReduceArgs r{};
  r.s_all = s_all;
  r.frame_sum = c->ptr<double>(c->lay.fsum);
  r.frame_ent = c->ptr<double>(c->lay.fent);
  r.q = c->ptr<float>(c->lay.q);
  r.core = c->ptr<int32_t>(c->lay.core);
  r.qd = c->ptr<double>(c->lay.qd);
  r.v = c->ptr<float>(c->lay.v);
  r.a = c->ptr<float>(c->lay.a);
  r.vall = c->ptr<double>(c->lay.vall);
  r.B = (int)c->dv.n_scored;
  r.L = cf.n_blocks;
  r.F = cf.n_frames;
  r.n_s = (int)c->dv.n_s;
  r.k_layer = cf.k_layer;
  r.cv_penalty = cf.cv_penalty;
  Timed t(c, SWAM_T_REDUCE, st);
  SWAM_HIP(c, launch_score_reduce(r, st), "score_reduce");
  return SWAM_OK;
}

// read the packed sequence offsets back to the host (one synchronisation)
int read_packed_rows(swam_ctx* c, hipStream_t st) {
  const int B = c->cfg.batch;
  SWAM_HIP(c, hipMemcpyAsync(c->host_cu, c->ptr<int32_t>(c->lay.cu_packed), (B + 1) * 4,
                             hipMemcpyDeviceToHost, st), "read cu_seqlens");
  SWAM_HIP(c, hipStreamSynchronize(st), "synchronise");
  c->packed_rows = c->host_cu[B];
  return SWAM_OK;
}

// k_core / k_anchor < 0: the configured budgets; on: the stream to enqueue on
// (the context stream when NULL)
int run_select(swam_ctx* c, const float* v, const float* a, int k_core = -1, int k_anchor = -1,
               hipStream_t on = nullptr) {
  const swam_config& cf = c->cfg;
  const hipStream_t st = on ? on : c->st;
  SelectArgs s{};
  s.v = v;
  s.a = a;
  s.pool = c->ptr<uint8_t>(c->lay.pool);
  s.core = c->ptr<uint8_t>(c->lay.corefl);
  s.keep_idx = c->ptr<int32_t>(c->lay.keep_idx);
  s.keep_cnt = c->ptr<int32_t>(c->lay.keep_cnt);
  s.keep = c->ptr<int32_t>(c->lay.keep);
  s.B = (int)c->dv.n_scored;
  s.F = cf.n_frames;
  s.n_s = (int)c->dv.n_s;
  s.k_core = k_core >= 0 ? k_core : cf.k_core;
  s.k_anchor = k_anchor >= 0 ? k_anchor : cf.k_anchor;
  s.k_max = (int)c->dv.k_max;
  s.mass_num = c->dv.mass_num;
  s.mass_den = c->dv.mass_den;
  s.n_ctx = cf.n_ctx;
  s.n_act = cf.n_act;
  {
    Timed t(c, SWAM_T_SELECT, st);
    SWAM_HIP(c, launch_select(s, st), "select");
    if (cf.cfg_pairs) {
      // the unconditional partner b + B/2 keeps the positions selected for b
      const int64_t P = c->dv.n_scored;
      const size_t kb = (size_t)(P * c->dv.l_full) * 4, ib = (size_t)(P * cf.n_frames * c->dv.k_max) * 4,
                   cb = (size_t)(P * cf.n_frames) * 4;
      SWAM_HIP(c, hipMemcpyAsync((char*)s.keep + kb, s.keep, kb, hipMemcpyDeviceToDevice, st),
               "share keep");
      SWAM_HIP(c, hipMemcpyAsync((char*)s.keep_idx + ib, s.keep_idx, ib, hipMemcpyDeviceToDevice,
                                 st), "share keep_idx");
      SWAM_HIP(c, hipMemcpyAsync((char*)s.keep_cnt + cb, s.keep_cnt, cb, hipMemcpyDeviceToDevice,
                                 st), "share keep_cnt");
    }
    SWAM_HIP(c, launch_packmap(s.keep, c->ptr<int32_t>(c->lay.pack_pos),
                               c->ptr<int32_t>(c->lay.gather), c->ptr<int32_t>(c->lay.cu_packed),
                               cf.batch, c->dv.l_full, st), "packmap");
  }
  if (c->dv.mass_den > 0) {
    const int rc = read_packed_rows(c, st);
    if (rc != SWAM_OK) return rc;
  } else {
    c->packed_rows = (int64_t)cf.batch * c->dv.t_pack_fixed;
  }
  c->sel_valid = true;
  return SWAM_OK;
}

int copy_out(swam_ctx* c, void* dst, size_t src_off, size_t bytes, const char* what) {
  if (!dst) return SWAM_OK;
  SWAM_HIP(c, hipMemcpyAsync(dst, c->arena + src_off, bytes, hipMemcpyDeviceToDevice, c->st),
           what);
  return SWAM_OK;
}

void fill_alpha(int g, float* out) {
  // central half (|i - (g-1)/2| < g/4) weighs twice the outer quarters
  double w[16], s = 0.0;
  for (int i = 0; i < g; ++i) {
    w[i] = fabs(i - (g - 1) / 2.0) < g / 4.0 ? 2.0 : 1.0;
    s += w[i];
  }
  for (int i = 0; i < 16; ++i) out[i] = i < g ? (float)(w[i] / s) : 0.0f;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* swam_status_str(int status) {
  switch (status) {
    case SWAM_OK: return "SWAM_OK";
    case SWAM_E_INVALID: return "SWAM_E_INVALID";
    case SWAM_E_SHAPE: return "SWAM_E_SHAPE";
    case SWAM_E_DTYPE: return "SWAM_E_DTYPE";
    case SWAM_E_STATE: return "SWAM_E_STATE";
    case SWAM_E_HIP: return "SWAM_E_HIP";
    case SWAM_E_NOMEM: return "SWAM_E_NOMEM";
    case SWAM_E_UNSUPPORTED: return "SWAM_E_UNSUPPORTED";
    default: return "SWAM_E_UNKNOWN";
  }
}

const char* swam_last_error(const swam_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_err.c_str();
}

int swam_plan(const swam_config* cfg, swam_plan_info* out) {
  if (!out) return set_err(nullptr, SWAM_E_INVALID, "out is NULL");
  Derived dv{};
  const int rc = derive(cfg, &dv, &g_err);
  if (rc != SWAM_OK) return rc;
  const Layout L = layout_for(cfg, dv);
  out->n_s = dv.n_s;
  out->group_size = dv.g;
  out->l_full = dv.l_full;
  out->rows_full = dv.rows_full;
  out->k_max = dv.k_max;
  out->t_pack_fixed = dv.t_pack_fixed;
  out->k_layer_eff = dv.k_eff;
  out->workspace_bytes = (int64_t)L.total;
  return SWAM_OK;
}

int swam_create(const swam_config* cfg, void* stream, swam_ctx** out) {
  if (!out) return set_err(nullptr, SWAM_E_INVALID, "out is NULL");
  *out = nullptr;
  Derived dv{};
  int rc = derive(cfg, &dv, &g_err);
  if (rc != SWAM_OK) return rc;
  swam_ctx* c = new (std::nothrow) swam_ctx();
  if (!c) return set_err(nullptr, SWAM_E_NOMEM, "context allocation");
  c->cfg = *cfg;
  c->dv = dv;
  c->lay = layout_for(cfg, dv);
  c->st = (hipStream_t)stream;
  hipError_t e = hipGetDevice(&c->device);
  if (e == hipSuccess) e = hipMalloc((void**)&c->arena, c->lay.total);
  if (e != hipSuccess) {
    g_err = std::string("workspace allocation: ") + hipGetErrorString(e);
    delete c;
    return e == hipErrorOutOfMemory ? SWAM_E_NOMEM : SWAM_E_HIP;
  }
  e = hipHostMalloc((void**)&c->host_cu, (cfg->batch + 1) * sizeof(int32_t), 0);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->order_ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_attn, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_score, hipEventDisableTiming);
  // default priority (no priority argument): the side stream of the scoring
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking);
  if (e == hipSuccess) {
    float alpha[16];
    fill_alpha((int)dv.g, alpha);
    e = hipMemcpy(c->ptr<float>(c->lay.alpha), alpha, sizeof(alpha), hipMemcpyHostToDevice);
  }
  if (e == hipSuccess) {
    std::vector<int32_t> cu(cfg->batch + 1);
    for (int b = 0; b <= cfg->batch; ++b) cu[b] = (int32_t)(b * dv.l_full);
    e = hipMemcpy(c->ptr<int32_t>(c->lay.cu_dense), cu.data(), cu.size() * 4,
                  hipMemcpyHostToDevice);
  }
  if (e == hipSuccess && cfg->rope) {
    e = launch_rope_table(c->ptr<float2>(c->lay.rope), (int)dv.rows_full, c->st);
    if (e == hipSuccess) e = hipStreamSynchronize(c->st);
  }
  if (e != hipSuccess) {
    g_err = std::string("context setup: ") + hipGetErrorString(e);
    swam_destroy(c);
    return SWAM_E_HIP;
  }
  *out = c;
  return SWAM_OK;
}

int swam_destroy(swam_ctx* c) {
  if (!c) return SWAM_OK;
  if (c->st || c->arena) (void)hipStreamSynchronize(c->st);
  if (c->side) (void)hipStreamSynchronize(c->side);
  for (auto& g : c->graphs) (void)hipGraphExecDestroy(g.exec);
  for (hipEvent_t ev : c->ev) (void)hipEventDestroy(ev);
  if (c->arena) (void)hipFree(c->arena);
  if (c->host_cu) (void)hipHostFree(c->host_cu);
  if (c->order_ev) (void)hipEventDestroy(c->order_ev);
  if (c->ev_attn) (void)hipEventDestroy(c->ev_attn);
  if (c->ev_score) (void)hipEventDestroy(c->ev_score);
  if (c->side) (void)hipStreamDestroy(c->side);
  delete c;
  return SWAM_OK;
}

int swam_set_stream(swam_ctx* c, void* stream) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (c->capturing) return set_err(c, SWAM_E_STATE, "stream switch during graph capture");
  const hipStream_t next = (hipStream_t)stream;
  if (next != c->st) {
    // work queued on the previous stream uses the same workspace: the new
    // stream waits for it (no host synchronisation)
    SWAM_HIP(c, hipEventRecord(c->order_ev, c->st), "order event record");
    SWAM_HIP(c, hipStreamWaitEvent(next, c->order_ev, 0), "order event wait");
    c->st = next;
  }
  return SWAM_OK;
}

int swam_score(swam_ctx* c, const void* q_act, int64_t q_seq_stride, int64_t q_row_stride,
               const void* k_fut, int64_t k_seq_stride, int64_t k_row_stride,
               const float* lse_act, const void* k_all, int64_t kall_seq_stride, float* s_out) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (!q_act || !k_fut || !s_out) return set_err(c, SWAM_E_INVALID, "q_act, k_fut, s_out required");
  if (!lse_act && !k_all) return set_err(c, SWAM_E_INVALID, "need lse_act (mode A) or k_all (mode B)");
  const int64_t d = c->dv.d;
  if (q_row_stride < d || k_row_stride < d || q_seq_stride < 0 || k_seq_stride < 0 ||
      (!lse_act && kall_seq_stride < 0))
    return set_err(c, SWAM_E_INVALID, "row strides must be >= d_model and seq strides >= 0");
  const swam_config& cf = c->cfg;
  const float* lse = lse_act;
  int64_t lse_seq = (int64_t)cf.n_act * cf.n_heads;
  if (!lse_act) {
    Timed t(c, SWAM_T_SCORE);
    float* ws = c->ptr<float>(c->lay.lse_act);
    SWAM_HIP(c, launch_lse_all(cf.dtype, q_act, q_seq_stride, q_row_stride, k_all,
                               kall_seq_stride, k_row_stride, c->dv.l_full, (int)c->dv.n_scored, cf.n_act,
                               cf.n_heads, ws, c->ptr<float>(c->lay.lse_part), c->st),
             "lse (mode B)");
    lse = ws;
  }
  ScoreArgs a{};
  a.q = q_act; a.q_seq = q_seq_stride; a.q_row = q_row_stride;
  a.k = k_fut; a.k_seq = k_seq_stride; a.k_row = k_row_stride;
  a.lse = lse; a.lse_seq = lse_seq;
  a.s_out = s_out; a.s_seq = (int64_t)cf.n_frames * c->dv.n_s;
  a.alpha = c->ptr<float>(c->lay.alpha);
  a.B = (int)c->dv.n_scored; a.F = cf.n_frames; a.n_s = (int)c->dv.n_s; a.H = cf.n_act;
  a.n_heads = cf.n_heads;
  a.n_layers = 1;
  Timed t(c, SWAM_T_SCORE);
  SWAM_HIP(c, launch_score(cf.dtype, a, c->st), "score");
  return SWAM_OK;
}

int swam_score_reduce(swam_ctx* c, const float* s_all, float* q_out, float* v_out, float* a_out,
                      int32_t* core_out) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (!s_all || !v_out || !a_out) return set_err(c, SWAM_E_INVALID, "s_all, v_out, a_out required");
  int rc = run_reduce(c, s_all);
  if (rc != SWAM_OK) return rc;
  const swam_config& cf = c->cfg;
  const int64_t B = c->dv.n_scored;
  if ((rc = copy_out(c, q_out, c->lay.q, B * cf.n_blocks * 4, "copy Q"))) return rc;
  if ((rc = copy_out(c, v_out, c->lay.v, B * cf.n_frames * c->dv.n_s * 4, "copy V"))) return rc;
  if ((rc = copy_out(c, a_out, c->lay.a, B * c->dv.n_s * 4, "copy A"))) return rc;
  if ((rc = copy_out(c, core_out, c->lay.core, B * c->dv.k_eff * 4, "copy core"))) return rc;
  return SWAM_OK;
}

int swam_select(swam_ctx* c, const float* v, const float* a, int32_t* keep_idx,
                int32_t* keep_cnt, int32_t* pack_pos, int32_t* gather, int32_t* cu_seqlens) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if ((v == nullptr) != (a == nullptr))
    return set_err(c, SWAM_E_INVALID, "v and a must both be given or both NULL");
  if (!v) {
    v = c->ptr<float>(c->lay.v);
    a = c->ptr<float>(c->lay.a);
  }
  int rc = run_select(c, v, a);
  if (rc != SWAM_OK) return rc;
  return swam_export(c, nullptr, nullptr, nullptr, nullptr, keep_idx, keep_cnt, pack_pos, gather,
                     cu_seqlens);
}

int swam_select_random(swam_ctx* c, uint64_t seed, int32_t* keep_idx, int32_t* keep_cnt,
                       int32_t* pack_pos, int32_t* gather, int32_t* cu_seqlens) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (c->dv.mass_den > 0)
    return set_err(c, SWAM_E_UNSUPPORTED, "random selection needs fixed budgets (mass_threshold 0)");
  const swam_config& cf = c->cfg;
  const int64_t n = c->dv.n_scored * cf.n_frames * c->dv.n_s;
  {
    Timed t(c, SWAM_T_SELECT);
    SWAM_HIP(c, launch_random_keys(c->ptr<float>(c->lay.v), n, c->ptr<float>(c->lay.a),
                                   c->dv.n_scored * c->dv.n_s, seed, c->st),
             "random keys");
  }
  int rc = run_select(c, c->ptr<float>(c->lay.v), c->ptr<float>(c->lay.a),
                      cf.k_core + cf.k_anchor, 0);
  if (rc != SWAM_OK) return rc;
  return swam_export(c, nullptr, nullptr, nullptr, nullptr, keep_idx, keep_cnt, pack_pos, gather,
                     cu_seqlens);
}

}  // extern "C"

// ------------------------------------------- selection without allocation
// Scratch of swam_select_noalloc.  In host code `scratch` names a host-side
// stand-in, not device memory: its device address is resolved once per
// device with hipGetSymbolAddress and only that address is used.
static __device__ __align__(256) uint8_t scratch[SWAM_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch[kScratchDevices] = {};

// device address of `scratch` on the current device (resolved on first use)
int scratch_of_current_device(uint8_t** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_err(nullptr, SWAM_E_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kScratchDevices)
    return set_err(nullptr, SWAM_E_UNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_err(nullptr, SWAM_E_HIP, std::string("hipGetSymbolAddress(scratch): ") +
                                          hipGetErrorString(e));
    g_scratch[dev] = (uint8_t*)p;
  }
  *out = g_scratch[dev];
  return SWAM_OK;
}

}  // namespace

extern "C" {

int swam_select_noalloc(int32_t batch, int32_t n_frames, int32_t n_s, int32_t n_ctx,
                        int32_t n_act, int32_t k_core, int32_t k_anchor, float mass_threshold,
                        const float* v, const float* a, int32_t* keep_idx, int32_t* keep_cnt,
                        int32_t* pack_pos, int32_t* gather, int32_t* cu_seqlens, void* stream) {
  if (!v || !a || !keep_idx || !keep_cnt || !pack_pos || !gather || !cu_seqlens)
    return set_err(nullptr, SWAM_E_INVALID, "every tensor argument is required");
  if (batch < 1 || batch > SWAM_MAX_BATCH) return set_err(nullptr, SWAM_E_SHAPE, "batch must be in [1, 64]");
  if (n_frames < 1 || n_frames > SWAM_MAX_FRAMES)
    return set_err(nullptr, SWAM_E_SHAPE, "n_frames must be in [1, 64]");
  if (n_s < 2 || n_s > SWAM_MAX_NS) return set_err(nullptr, SWAM_E_SHAPE, "n_s must be in [2, 4096]");
  if (n_ctx < 0 || n_act < 0) return set_err(nullptr, SWAM_E_INVALID, "n_ctx and n_act must be >= 0");
  if (!(mass_threshold >= 0.0f && mass_threshold <= 1.0f))
    return set_err(nullptr, SWAM_E_INVALID, "mass_threshold must be in [0, 1]");
  if (k_anchor < 0 || k_anchor >= n_s) return set_err(nullptr, SWAM_E_INVALID, "k_anchor must be in [0, n_s)");
  if (mass_threshold == 0.0f && (k_core < 0 || (int64_t)k_core + k_anchor > n_s))
    return set_err(nullptr, SWAM_E_INVALID, "k_core + k_anchor must be in [0, n_s]");
  const int64_t l_full = (int64_t)n_ctx + (int64_t)n_frames * n_s + n_act;
  const size_t pool_b = align_up((size_t)batch * n_s);
  const size_t core_b = align_up((size_t)batch * n_frames * n_s);
  const size_t keep_b = (size_t)batch * l_full * 4;
  if (pool_b + core_b + keep_b > (size_t)SWAM_NOALLOC_SCRATCH_BYTES)
    return set_err(nullptr, SWAM_E_SHAPE,
                   "scratch need " + std::to_string(pool_b + core_b + keep_b) +
                       " bytes exceeds SWAM_NOALLOC_SCRATCH_BYTES (" +
                       std::to_string(SWAM_NOALLOC_SCRATCH_BYTES) + ")");
  uint8_t* base = nullptr;
  int rc = scratch_of_current_device(&base);
  if (rc != SWAM_OK) return rc;
  SelectArgs s{};
  s.v = v;
  s.a = a;
  s.pool = base;
  s.core = base + pool_b;
  s.keep = (int32_t*)(base + pool_b + core_b);
  s.keep_idx = keep_idx;
  s.keep_cnt = keep_cnt;
  s.B = batch;
  s.F = n_frames;
  s.n_s = n_s;
  s.k_core = k_core;
  s.k_anchor = k_anchor;
  s.n_ctx = n_ctx;
  s.n_act = n_act;
  if (mass_threshold > 0.0f) {
    mass_fraction(mass_threshold, &s.mass_num, &s.mass_den);
    s.k_max = n_s;
  } else {
    s.mass_num = 0;
    s.mass_den = 0;
    s.k_max = std::max(1, k_core + k_anchor);
  }
  // every flag the kernels read is written by them first in the same call,
  // so the array's contents from an earlier call never matter
  const hipStream_t st = (hipStream_t)stream;
  hipError_t e = launch_select(s, st);
  if (e == hipSuccess) e = launch_packmap(s.keep, pack_pos, gather, cu_seqlens, batch, l_full, st);
  if (e != hipSuccess) return set_err(nullptr, SWAM_E_HIP, std::string("select: ") + hipGetErrorString(e));
  return SWAM_OK;
}

int swam_set_selection(swam_ctx* c, const int32_t* keep_idx, const int32_t* keep_cnt) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (!keep_idx) return set_err(c, SWAM_E_INVALID, "keep_idx is NULL");
  (void)keep_cnt;  // counts are recomputed from the indices
  const swam_config& cf = c->cfg;
  int32_t* own = c->ptr<int32_t>(c->lay.keep_idx);
  if (keep_idx == own) return set_err(c, SWAM_E_INVALID, "keep_idx aliases the context cache");
  {
    Timed t(c, SWAM_T_SELECT);
    SWAM_HIP(c, launch_keep_from_idx(keep_idx, own, c->ptr<int32_t>(c->lay.keep_cnt),
                                     c->ptr<int32_t>(c->lay.keep), cf.batch, cf.n_frames,
                                     (int)c->dv.n_s, (int)c->dv.k_max, cf.n_ctx, cf.n_act, c->st),
             "import selection");
    SWAM_HIP(c, launch_packmap(c->ptr<int32_t>(c->lay.keep), c->ptr<int32_t>(c->lay.pack_pos),
                               c->ptr<int32_t>(c->lay.gather), c->ptr<int32_t>(c->lay.cu_packed),
                               cf.batch, c->dv.l_full, c->st), "packmap");
  }
  const int rc = read_packed_rows(c, c->st);
  if (rc != SWAM_OK) return rc;
  c->sel_valid = true;
  return SWAM_OK;
}

int swam_packed_rows(swam_ctx* c, int64_t* rows) {
  if (!c || !rows) return set_err(c, SWAM_E_INVALID, "NULL argument");
  if (!c->sel_valid) return set_err(c, SWAM_E_STATE, "no selection cached");
  *rows = c->packed_rows;
  return SWAM_OK;
}

int swam_export(swam_ctx* c, float* s_all, float* q, float* v, float* a, int32_t* keep_idx,
                int32_t* keep_cnt, int32_t* pack_pos, int32_t* gather, int32_t* cu_seqlens) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  const swam_config& cf = c->cfg;
  const int64_t B = cf.batch, F = cf.n_frames, n_s = c->dv.n_s;
  if ((keep_idx || keep_cnt || pack_pos || gather || cu_seqlens) && !c->sel_valid)
    return set_err(c, SWAM_E_STATE, "no selection cached");
  int rc;
  const int64_t Bs = c->dv.n_scored;
  if ((rc = copy_out(c, s_all, c->lay.s_all, Bs * cf.n_blocks * F * n_s * 4, "copy S"))) return rc;
  if ((rc = copy_out(c, q, c->lay.q, Bs * cf.n_blocks * 4, "copy Q"))) return rc;
  if ((rc = copy_out(c, v, c->lay.v, Bs * F * n_s * 4, "copy V"))) return rc;
  if ((rc = copy_out(c, a, c->lay.a, Bs * n_s * 4, "copy A"))) return rc;
  if ((rc = copy_out(c, keep_idx, c->lay.keep_idx, B * F * c->dv.k_max * 4, "copy keep_idx"))) return rc;
  if ((rc = copy_out(c, keep_cnt, c->lay.keep_cnt, B * F * 4, "copy keep_cnt"))) return rc;
  if ((rc = copy_out(c, pack_pos, c->lay.pack_pos, c->dv.rows_full * 4, "copy pack_pos"))) return rc;
  if ((rc = copy_out(c, gather, c->lay.gather, c->dv.rows_full * 4, "copy gather"))) return rc;
  if ((rc = copy_out(c, cu_seqlens, c->lay.cu_packed, (B + 1) * 4, "copy cu"))) return rc;
  return SWAM_OK;
}

int swam_pack(swam_ctx* c, const void* x_full, void* x_packed) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (!x_full || !x_packed) return set_err(c, SWAM_E_INVALID, "NULL tensor");
  if (!aligned16(x_full) || !aligned16(x_packed))
    return set_err(c, SWAM_E_INVALID, "tensors must be 16-byte aligned");
  if (!c->sel_valid) return set_err(c, SWAM_E_STATE, "no selection cached");
  Timed t(c, SWAM_T_PACK);
  SWAM_HIP(c, launch_pack(x_full, x_packed, c->ptr<int32_t>(c->lay.gather), c->packed_rows,
                          c->dv.d * c->dv.esz, c->st), "pack");
  return SWAM_OK;
}

int swam_unpack(swam_ctx* c, const void* y_packed, const void* x_full, void* y_full) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (!y_packed || !x_full || !y_full) return set_err(c, SWAM_E_INVALID, "NULL tensor");
  if (!aligned16(y_packed) || !aligned16(x_full) || !aligned16(y_full))
    return set_err(c, SWAM_E_INVALID, "tensors must be 16-byte aligned");
  if (!c->sel_valid) return set_err(c, SWAM_E_STATE, "no selection cached");
  Timed t(c, SWAM_T_UNPACK);
  const int64_t rb = c->dv.d * c->dv.esz;
  if (y_full == x_full)
    SWAM_HIP(c, launch_unpack_scatter(y_packed, y_full, c->ptr<int32_t>(c->lay.gather),
                                      c->packed_rows, rb, c->st), "unpack");
  else
    SWAM_HIP(c, launch_unpack_merge(y_packed, x_full, y_full, c->ptr<int32_t>(c->lay.pack_pos),
                                    c->dv.rows_full, rb, c->st), "unpack");
  return SWAM_OK;
}

int swam_block(swam_ctx* c, const swam_block_weights* w, const float* temb, void* x,
               int64_t n_rows, const int32_t* cu_seqlens, int32_t n_seqs, float* lse_out,
               void* qkv_out) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (bad_block(w) || !temb || !x) return set_err(c, SWAM_E_INVALID, "NULL or unaligned weight, or NULL tensor");
  if (!aligned16(x) || (qkv_out && !aligned16(qkv_out)))
    return set_err(c, SWAM_E_INVALID, "x and qkv_out must be 16-byte aligned");
  if (n_rows < 0 || n_rows > c->dv.rows_full)
    return set_err(c, SWAM_E_SHAPE, "n_rows must be in [0, batch * l_full]");
  const int32_t* cu = cu_seqlens;
  if (!cu) {
    if (n_rows != c->dv.rows_full)
      return set_err(c, SWAM_E_SHAPE, "dense layout needs n_rows == batch * l_full");
    cu = c->ptr<int32_t>(c->lay.cu_dense);
    n_seqs = c->cfg.batch;
  } else if (n_seqs < 1 || n_seqs > SWAM_MAX_BATCH) {
    return set_err(c, SWAM_E_SHAPE, "n_seqs must be in [1, 64]");
  }
  int rc = run_adaln(c, w, 1, temb);
  if (rc != SWAM_OK) return rc;
  void* qkv = qkv_out ? qkv_out : c->ptr<char>(c->lay.qkv);
  return run_block(c, w, c->ptr<float>(c->lay.mod), x, n_rows, cu, n_seqs, lse_out, qkv,
                   cu_seqlens ? 2 : 0);
}

}  // extern "C"

namespace {

int check_step(swam_ctx* c, const swam_model* model, const void* x_full, const float* temb,
               int32_t tau, void* y_full, int32_t flags, int* kind) {
  const swam_config& cf = c->cfg;
  if (!model || !model->blocks || model->n_blocks != cf.n_blocks)
    return set_err(c, SWAM_E_INVALID, "model must have config.n_blocks blocks");
  for (int l = 0; l < cf.n_blocks; ++l)
    if (bad_block(&model->blocks[l]))
      return set_err(c, SWAM_E_INVALID, "NULL or not 16-byte aligned block weight");
  if (!x_full || !y_full || !temb) return set_err(c, SWAM_E_INVALID, "NULL tensor");
  if (!aligned16(x_full) || !aligned16(y_full))
    return set_err(c, SWAM_E_INVALID, "x_full and y_full must be 16-byte aligned");
  {
    // y_full is x_full itself or a disjoint buffer: the pruned rows are copied
    // and the retained ones scattered assuming one of the two
    const uintptr_t xa = (uintptr_t)x_full, ya = (uintptr_t)y_full;
    const uintptr_t nb = (uintptr_t)(c->dv.rows_full * c->dv.d * c->dv.esz);
    if (xa != ya && xa < ya + nb && ya < xa + nb)
      return set_err(c, SWAM_E_INVALID, "y_full must be x_full itself or not overlap it");
  }
  if (tau < 0) return set_err(c, SWAM_E_INVALID, "tau < 0");
  if (flags & SWAM_STEP_FORCE_DENSE) *kind = SWAM_KIND_DENSE;
  else if ((flags & SWAM_STEP_FORCE_REFRESH) || tau % cf.reuse_R == 0) *kind = SWAM_KIND_REFRESH;
  else *kind = SWAM_KIND_SPARSE;
  if (*kind == SWAM_KIND_SPARSE && !c->sel_valid)
    return set_err(c, SWAM_E_STATE, "sparse step before any selection (run a refresh first)");
  return SWAM_OK;
}

// every launch of one step, in order, on the context stream
// tags the timer slots of the launches enqueued in its scope with a step kind
struct StepKindScope {
  swam_ctx* c;
  int prev;
  StepKindScope(swam_ctx* ctx, int kind) : c(ctx), prev(ctx->step_kind) { c->step_kind = kind; }
  ~StepKindScope() { c->step_kind = prev; }
};

int enqueue_step_launches(swam_ctx* c, const swam_model* model, const void* x_full,
                          const float* temb, int kind, void* y_full);

int enqueue_step(swam_ctx* c, const swam_model* model, const void* x_full, const float* temb,
                 int kind, void* y_full) {
  StepKindScope scope(c, kind);
  return enqueue_step_launches(c, model, x_full, temb, kind, y_full);
}

int enqueue_step_launches(swam_ctx* c, const swam_model* model, const void* x_full,
                          const float* temb, int kind, void* y_full) {
  const swam_config& cf = c->cfg;
  int rc = run_adaln(c, model->blocks, cf.n_blocks, temb);
  if (rc != SWAM_OK) return rc;
  const int64_t d = c->dv.d;
  const float* mod = c->ptr<float>(c->lay.mod);
  void* qkv = c->ptr<char>(c->lay.qkv);
  if (kind != SWAM_KIND_SPARSE) {
    {
      Timed t(c, SWAM_T_COPY);
      SWAM_HIP(c, launch_copy(x_full, y_full, c->dv.rows_full * d * c->dv.esz, c->st), "copy");
    }
    const bool score = kind == SWAM_KIND_REFRESH;
    // scores of layer l from its q, k (in the QKV slot) and lambda, written
    // into S_all[b][l]; the slot is reused by the next block
    ScoreArgs a{};
    if (score) {
      const int64_t ld = 3 * d, es = c->dv.esz;
      const int64_t act0 = cf.n_ctx + (int64_t)cf.n_frames * c->dv.n_s;
      a.q = (const char*)qkv + act0 * ld * es;
      a.q_seq = c->dv.l_full * ld;
      a.q_row = ld;
      a.k = (const char*)qkv + (cf.n_ctx * ld + d) * es;
      a.k_seq = c->dv.l_full * ld;
      a.k_row = ld;
      a.lse = c->ptr<float>(c->lay.lse) + act0 * cf.n_heads;
      a.lse_seq = c->dv.l_full * cf.n_heads;
      a.s_seq = (int64_t)cf.n_blocks * cf.n_frames * c->dv.n_s;
      a.alpha = c->ptr<float>(c->lay.alpha);
      a.B = (int)c->dv.n_scored;
      a.F = cf.n_frames;
      a.n_s = (int)c->dv.n_s;
      a.H = cf.n_act;
      a.n_heads = cf.n_heads;
      a.n_layers = 1;
    }
    // bf16: every layer but the last scores in the tail of its MLP up
    // projection where that grid leaves CUs idle; the last layer scores on the
    // side stream, so that the reduction and selection can follow it there
    const bool in_up = score && cf.dtype == SWAM_BF16 &&
                       gemm_up_scored_slots(c->dv.rows_full, c->dv.hidden, d,
                                            c->dv.splitk_floats) > 0;
    for (int l = 0; l < cf.n_blocks; ++l) {
      a.s_out = c->ptr<float>(c->lay.s_all) + (int64_t)l * cf.n_frames * c->dv.n_s;
      rc = run_block(c, &model->blocks[l], mod + (int64_t)l * 6 * d, y_full, c->dv.rows_full,
                     c->ptr<int32_t>(c->lay.cu_dense), cf.batch,
                     score ? c->ptr<float>(c->lay.lse) : nullptr, qkv, 0,
                     score ? &a : nullptr, nullptr, nullptr, in_up && l + 1 < cf.n_blocks);
      if (rc != SWAM_OK) return rc;
    }
    if (score) {
      // the reduce, the selection and the pack map follow the last layer's
      // scoring on the side stream, overlapping the last block's projections
      // (they read only the scores and write only selection state); the
      // context stream waits for them before the step ends
      c->scores_valid = true;
      if ((rc = run_reduce(c, c->ptr<float>(c->lay.s_all), c->side)) != SWAM_OK) return rc;
      if ((rc = run_select(c, c->ptr<float>(c->lay.v), c->ptr<float>(c->lay.a), -1, -1,
                           c->side)) != SWAM_OK)
        return rc;
      SWAM_HIP(c, hipEventRecord(c->ev_score, c->side), "selection done");
      c->score_pending = true;
    }
    if ((rc = join_score(c)) != SWAM_OK) return rc;
  } else {
    // out of place, the pruned rows are copied on the side stream (forked
    // inside block 0 after the pack, or here when no row is retained)
    const int64_t rb = d * c->dv.esz;
    const bool fork = y_full != x_full;
    if (fork && c->packed_rows <= 0)
      if ((rc = fork_pruned_copy(c, x_full, y_full)) != SWAM_OK) return rc;
    // the gather-pack of x_full runs inside block 0's first LayerNorm kernel;
    // bf16: the scatter of the retained rows into y_full inside the last
    // block's MLP down projection store (the pruned rows of y_full are the
    // copy's, disjoint from these); fp32: a separate scatter pass
    void* xp = c->ptr<char>(c->lay.xp);
    const bool fold_unpack = cf.dtype == SWAM_BF16;
    for (int l = 0; l < cf.n_blocks; ++l) {
      const bool last = l + 1 == cf.n_blocks;
      rc = run_block(c, &model->blocks[l], mod + (int64_t)l * 6 * d, xp, c->packed_rows,
                     c->ptr<int32_t>(c->lay.cu_packed), cf.batch, nullptr, qkv, 1, nullptr,
                     l == 0 ? x_full : nullptr, l == 0 && fork ? y_full : nullptr, false,
                     fold_unpack && last ? y_full : nullptr);
      if (rc != SWAM_OK) return rc;
    }
    if (fork) SWAM_HIP(c, hipStreamWaitEvent(c->st, c->ev_score, 0), "join pruned-row copy");
    if (!fold_unpack) {
      // scatter of the packed rows (the retained ones) into y_full
      Timed t(c, SWAM_T_UNPACK);
      SWAM_HIP(c, launch_unpack_scatter(xp, y_full, c->ptr<int32_t>(c->lay.gather),
                                        c->packed_rows, rb, c->st), "unpack");
    }
  }
  return SWAM_OK;
}

uint64_t weight_signature(const swam_model* m) {
  uint64_t h = 1469598103934665603ull;   // FNV-1a over every weight pointer
  for (int l = 0; l < m->n_blocks; ++l) {
    const void* const* p = (const void* const*)&m->blocks[l];
    for (size_t i = 0; i < sizeof(swam_block_weights) / sizeof(void*); ++i) {
      uint64_t v = (uint64_t)(uintptr_t)p[i];
      for (int k = 0; k < 8; ++k) {
        h ^= (v >> (8 * k)) & 0xFF;
        h *= 1099511628211ull;
      }
    }
  }
  return h;
}

constexpr size_t MAX_GRAPHS = 64;

}  // namespace

extern "C" {

int swam_step(swam_ctx* c, const swam_model* model, const void* x_full, const float* temb,
              int32_t tau, void* y_full, int32_t flags, int32_t* kind_out) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  int kind;
  int rc = check_step(c, model, x_full, temb, tau, y_full, flags, &kind);
  if (rc != SWAM_OK) return rc;
  if ((rc = enqueue_step(c, model, x_full, temb, kind, y_full)) != SWAM_OK) return rc;
  if (kind_out) *kind_out = kind;
  return SWAM_OK;
}

// ---------------------------------------------------------- diagnostics

int swam_overlap(swam_ctx* c, const float* p, const float* q, int64_t n_maps, int64_t n,
                 float* out) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (!p || !q || !out) return set_err(c, SWAM_E_INVALID, "NULL tensor");
  if (n_maps < 0 || n < 1 || n_maps > (1ll << 31) - 1) return set_err(c, SWAM_E_SHAPE, "bad map count or size");
  SWAM_HIP(c, launch_overlap(p, q, n_maps, n, out, c->st), "overlap");
  return SWAM_OK;
}

// ------------------------------------------------------------- sampler


static int check_io(swam_ctx* c, const swam_latent_io* io) {
  if (!io) return set_err(c, SWAM_E_INVALID, "latent io is NULL");
  if (io->d_latent < 1 || io->d_latent > 64)
    return set_err(c, SWAM_E_SHAPE, "d_latent must be in [1, 64]");
  if (!io->w_in || !io->b_in || !io->w_v || !io->b_v)
    return set_err(c, SWAM_E_INVALID, "NULL latent io weight");
  if (!aligned16(io->w_in) || !aligned16(io->b_in) || !aligned16(io->w_v) || !aligned16(io->b_v))
    return set_err(c, SWAM_E_INVALID, "latent io weights must be 16-byte aligned");
  // the velocity head is staged in LDS: 64 KB at most
  if ((int64_t)io->d_latent * c->dv.d * c->dv.esz > 65536)
    return set_err(c, SWAM_E_SHAPE, "d_latent * d_model * element size must be <= 64 KB");
  return SWAM_OK;
}

int swam_embed(swam_ctx* c, const swam_latent_io* io, const float* z, void* x_full) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  int rc = check_io(c, io);
  if (rc != SWAM_OK) return rc;
  if (!z || !x_full) return set_err(c, SWAM_E_INVALID, "NULL tensor");
  if (!aligned16(z) || !aligned16(x_full)) return set_err(c, SWAM_E_INVALID, "tensors must be 16-byte aligned");
  const swam_config& cf = c->cfg;
  const int l_lat = (int)(c->dv.l_full - cf.n_ctx);
  Timed t(c, SWAM_T_SAMPLE);
  SWAM_HIP(c, launch_embed(cf.dtype, z, io->w_in, io->b_in, x_full, (int64_t)cf.batch * l_lat,
                           c->dv.n_scored * l_lat, l_lat, (int)c->dv.l_full, cf.n_ctx,
                           io->d_latent, (int)c->dv.d, c->st),
           "embed");
  return SWAM_OK;
}

int swam_velocity(swam_ctx* c, const swam_latent_io* io, const void* y_full, int32_t retained_only,
                  float* v) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  int rc = check_io(c, io);
  if (rc != SWAM_OK) return rc;
  if (!y_full || !v) return set_err(c, SWAM_E_INVALID, "NULL tensor");
  if (!aligned16(y_full)) return set_err(c, SWAM_E_INVALID, "tensors must be 16-byte aligned");
  if (retained_only && !c->sel_valid) return set_err(c, SWAM_E_STATE, "no selection cached");
  const swam_config& cf = c->cfg;
  const int l_lat = (int)(c->dv.l_full - cf.n_ctx);
  const int32_t* gather = retained_only ? c->ptr<int32_t>(c->lay.gather) : nullptr;
  const int64_t items = retained_only ? c->packed_rows : (int64_t)cf.batch * l_lat;
  Timed t(c, SWAM_T_SAMPLE);
  SWAM_HIP(c, launch_velocity(cf.dtype, y_full, gather, items, io->w_v, io->b_v, v, l_lat,
                              (int)c->dv.l_full, cf.n_ctx, io->d_latent, (int)c->dv.d, c->st),
           "velocity");
  return SWAM_OK;
}

static int sample_update(swam_ctx* c, int c_lat, const float* v, float* v_cache, float* z,
                         float dsigma, int32_t kind) {
  if (!v || !z) return set_err(c, SWAM_E_INVALID, "NULL tensor");
  if (kind != SWAM_KIND_DENSE && kind != SWAM_KIND_REFRESH && kind != SWAM_KIND_SPARSE)
    return set_err(c, SWAM_E_INVALID, "bad step kind");
  if (kind != SWAM_KIND_DENSE && !v_cache) return set_err(c, SWAM_E_INVALID, "NULL velocity cache");
  if (kind == SWAM_KIND_SPARSE && !c->sel_valid) return set_err(c, SWAM_E_STATE, "no selection cached");
  if (!std::isfinite(dsigma)) return set_err(c, SWAM_E_INVALID, "dsigma is not finite");
  const swam_config& cf = c->cfg;
  const int l_lat = (int)(c->dv.l_full - cf.n_ctx);
  Timed t(c, SWAM_T_SAMPLE);
  SWAM_HIP(c, launch_sample_update(v, v_cache, z, c->ptr<int32_t>(c->lay.pack_pos), dsigma, kind,
                                   c->dv.n_scored * l_lat, l_lat, (int)c->dv.l_full, cf.n_ctx,
                                   (int)(cf.n_frames * c->dv.n_s), c_lat, cf.cfg_pairs,
                                   cf.guidance, c->st),
           "sample update");
  return SWAM_OK;
}

int swam_sample_update(swam_ctx* c, int32_t d_latent, const float* v, float* v_cache, float* z,
                       float dsigma, int32_t kind) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (d_latent < 1 || d_latent > 64) return set_err(c, SWAM_E_SHAPE, "d_latent must be in [1, 64]");
  return sample_update(c, d_latent, v, v_cache, z, dsigma, kind);
}

int swam_flow_sigmas(int32_t n_steps, double shift, double* sigmas) {
  if (n_steps < 1 || !sigmas || !std::isfinite(shift) || !(shift > 0.0))
    return set_err(nullptr, SWAM_E_INVALID, "need n_steps >= 1, a finite shift > 0 and sigmas");
  for (int32_t i = 0; i <= n_steps; ++i) {
    const double s = 1.0 - (double)i / n_steps;
    sigmas[i] = shift * s / (1.0 + (shift - 1.0) * s);
  }
  return SWAM_OK;
}

int swam_sample_step(swam_ctx* c, const swam_model* model, const swam_latent_io* io, float* z,
                     float* v, float* v_cache, void* x_full, void* y_full, const float* temb,
                     int32_t tau, float dsigma, int32_t flags, int32_t* kind_out) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  int rc = check_io(c, io);
  if (rc != SWAM_OK) return rc;
  if (!z || !v || !v_cache || !x_full || !y_full) return set_err(c, SWAM_E_INVALID, "NULL tensor");
  if (x_full == y_full)
    return set_err(c, SWAM_E_INVALID, "x_full must not alias y_full (its context rows are reused)");
  int kind;
  if ((rc = check_step(c, model, x_full, temb, tau, y_full, flags, &kind)) != SWAM_OK) return rc;
  StepKindScope scope(c, kind);
  if ((rc = swam_embed(c, io, z, x_full)) != SWAM_OK) return rc;
  if ((rc = enqueue_step(c, model, x_full, temb, kind, y_full)) != SWAM_OK) return rc;
  if ((rc = swam_velocity(c, io, y_full, kind == SWAM_KIND_SPARSE, v)) != SWAM_OK) return rc;
  if ((rc = sample_update(c, io->d_latent, v, v_cache, z, dsigma, kind)) != SWAM_OK) return rc;
  if (kind_out) *kind_out = kind;
  return SWAM_OK;
}

int swam_step_graph(swam_ctx* c, const swam_model* model, const void* x_full,
                    const float* temb, int32_t tau, void* y_full, int32_t flags,
                    int32_t* kind_out) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  int kind;
  int rc = check_step(c, model, x_full, temb, tau, y_full, flags, &kind);
  if (rc != SWAM_OK) return rc;
  if (kind == SWAM_KIND_REFRESH && c->dv.mass_den > 0) {
    // the ragged refresh reads its packed lengths back to the host: run it eagerly
    if ((rc = enqueue_step(c, model, x_full, temb, kind, y_full)) != SWAM_OK) return rc;
    if (kind_out) *kind_out = kind;
    return SWAM_OK;
  }
  if (c->st == nullptr)
    return set_err(c, SWAM_E_STATE, "graph capture needs a non-default stream");
  const uint64_t wsig = weight_signature(model);
  const int64_t packed = kind == SWAM_KIND_SPARSE ? c->packed_rows : -1;
  hipGraphExec_t exec = nullptr;
  for (auto& g : c->graphs)
    if (g.kind == kind && g.x == x_full && g.y == y_full && g.temb == temb && g.wsig == wsig &&
        g.packed == packed) {
      exec = g.exec;
      break;
    }
  if (!exec) {
    c->capturing = true;
    hipError_t e = hipStreamBeginCapture(c->st, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) {
      c->capturing = false;
      return hip_check(c, e, "begin capture");
    }
    rc = enqueue_step(c, model, x_full, temb, kind, y_full);
    hipGraph_t graph = nullptr;
    e = hipStreamEndCapture(c->st, &graph);
    c->capturing = false;
    if (rc != SWAM_OK) {
      if (graph) (void)hipGraphDestroy(graph);
      return rc;
    }
    if (e != hipSuccess) return hip_check(c, e, "end capture");
    e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (e != hipSuccess) return hip_check(c, e, "graph instantiate");
    if (c->graphs.size() >= MAX_GRAPHS) {
      (void)hipGraphExecDestroy(c->graphs.front().exec);
      c->graphs.erase(c->graphs.begin());
    }
    c->graphs.push_back({kind, x_full, y_full, temb, wsig, packed, exec});
  }
  SWAM_HIP(c, hipGraphLaunch(exec, c->st), "graph launch");
  if (kind == SWAM_KIND_REFRESH) {   // host-side effects of a replayed refresh
    c->scores_valid = true;
    c->sel_valid = true;
    c->packed_rows = (int64_t)c->cfg.batch * c->dv.t_pack_fixed;
  }
  if (kind_out) *kind_out = kind;
  return SWAM_OK;
}

int swam_graph_clear(swam_ctx* c) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  SWAM_HIP(c, hipStreamSynchronize(c->st), "synchronise");
  for (auto& g : c->graphs) (void)hipGraphExecDestroy(g.exec);
  c->graphs.clear();
  return SWAM_OK;
}

int swam_timer_enable(swam_ctx* c, uint32_t mask, int32_t capacity) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (mask && capacity < 1) return set_err(c, SWAM_E_INVALID, "capacity must be >= 1");
  SWAM_HIP(c, hipStreamSynchronize(c->st), "synchronise");
  for (hipEvent_t ev : c->ev) (void)hipEventDestroy(ev);
  c->ev.clear();
  c->ev_cls.clear();
  c->ev_kind.clear();
  c->tmask = mask;
  c->tcap = 0;
  c->tused = 0;
  for (int64_t& n : c->tcount) n = 0;
  if (!mask) return SWAM_OK;
  c->ev.resize(2 * (size_t)capacity);
  c->ev_cls.assign(capacity, -1);
  c->ev_kind.assign(capacity, SWAM_KIND_NONE);
  for (auto& ev : c->ev) SWAM_HIP(c, hipEventCreate(&ev), "event create");
  c->tcap = capacity;
  return SWAM_OK;
}

int swam_timer_reset(swam_ctx* c) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  SWAM_HIP(c, hipStreamSynchronize(c->st), "synchronise");
  c->tused = 0;
  for (int64_t& n : c->tcount) n = 0;
  return SWAM_OK;
}

int swam_timer_stride(swam_ctx* c, int32_t stride) {
  if (!c) return set_err(nullptr, SWAM_E_INVALID, "ctx is NULL");
  if (stride < 1) return set_err(c, SWAM_E_INVALID, "stride must be >= 1");
  SWAM_HIP(c, hipStreamSynchronize(c->st), "synchronise");
  c->tstride = stride;
  c->tused = 0;
  for (int64_t& n : c->tcount) n = 0;
  return SWAM_OK;
}

int swam_timer_read_kind(swam_ctx* c, int32_t cls, int32_t kind, int64_t* launches,
                         double* total_ms) {
  if (!c || !launches || !total_ms) return set_err(c, SWAM_E_INVALID, "NULL argument");
  if (cls < 0 || cls >= SWAM_T_COUNT) return set_err(c, SWAM_E_INVALID, "bad timer class");
  if (kind != SWAM_KIND_ANY && kind != SWAM_KIND_NONE && kind != SWAM_KIND_DENSE &&
      kind != SWAM_KIND_REFRESH && kind != SWAM_KIND_SPARSE)
    return set_err(c, SWAM_E_INVALID, "bad step kind");
  SWAM_HIP(c, hipStreamSynchronize(c->st), "synchronise");
  int64_t n = 0;
  double ms = 0.0;
  for (int i = 0; i < c->tused; ++i) {
    if (c->ev_cls[i] != cls || (kind != SWAM_KIND_ANY && c->ev_kind[i] != kind)) continue;
    float e = 0.0f;
    SWAM_HIP(c, hipEventElapsedTime(&e, c->ev[2 * i], c->ev[2 * i + 1]), "elapsed");
    ms += e;
    ++n;
  }
  *launches = n;
  *total_ms = ms;
  return SWAM_OK;
}

int swam_timer_read(swam_ctx* c, int32_t cls, int64_t* launches, double* total_ms) {
  return swam_timer_read_kind(c, cls, SWAM_KIND_ANY, launches, total_ms);
}

}  // extern "C"
