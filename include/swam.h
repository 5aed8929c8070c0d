/*
 * swam.h -- C ABI of the action-guided sparse denoising step (Sparse-WAM,
 * arXiv 2609.38984) on AMD Instinct MI355X (gfx950).
 *
 * One step of a world-action-model diffusion transformer is split into the
 * paper's five parts, each an entry point below:
 *   (1) swam_score / swam_score_reduce : action-to-future attention scoring
 *       with reused log-sum-exp normalisers (Sec. 4.2 "low-overhead attention
 *       profiling"; App. A.2, score-extraction equation), layer quality and
 *       core/anchor scores (Sec. 4.1; App. A.1 layer-quality and
 *       anchor-statistics equations);
 *   (2) swam_select : candidate pool, per-frame core tokens and shared anchors
 *       (Sec. 4.1 pool, core-selection and stable-selection equations), with
 *       the packing metadata of the retained tokens (Sec. 4.2 compact
 *       execution), cached for reuse across denoising steps;
 *   (3) swam_pack : gather of context, retained future and action tokens into
 *       the compact sequence;
 *   (4) swam_block : one adaLN DiT block on a (packed or dense) token set;
 *   (5) swam_unpack : scatter back into the full latent; pruned tokens keep
 *       their input residual stream unchanged.
 * swam_step runs a whole denoising step: a refresh (dense forward + scoring +
 * selection) when tau mod R == 0, otherwise a sparse step on the cached
 * selection (Sec. 4.2 cross-step reuse).
 *
 * Conventions shared by every call
 * --------------------------------
 * Ownership: every tensor argument is a DEVICE pointer owned by the caller.
 *   The context owns only its workspace (allocated once by swam_create) and
 *   the cached scores/selection.  No call other than swam_create /
 *   swam_timer_enable allocates.
 * Streams: every call is asynchronous on the stream given to swam_create
 *   (or swam_set_stream).  Inside a step the context also uses a second
 *   stream of its own (default priority): a refresh scores each layer there
 *   while the block continues, and an out-of-place sparse step copies the
 *   pruned rows there while the blocks run; both are forked from and joined
 *   back into the context stream with events (also under graph capture), so
 *   a step's work is complete when the context stream's is.  Nothing
 *   synchronises except where stated:
 *   swam_select / swam_step in mass-threshold mode and swam_set_selection read
 *   the packed lengths back to the host once; swam_timer_read synchronises.
 * Token layout: row-major [T][d].  One sequence is
 *   [context (n_ctx) | future frames (n_frames * frame_h * frame_w),
 *    frame-major, row-major inside a frame | action tokens (n_act)];
 *   sequences of a batch are concatenated.  Packed sequences keep the original
 *   order of their retained rows and are described by cu_seqlens [B+1]
 *   (int32 row offsets).
 * Element type: activations and weights are float32 (SWAM_F32) or bf16
 *   (SWAM_BF16, raw 16-bit storage) as fixed by swam_config.dtype; scores,
 *   normalisers, timestep embeddings and all statistics are float32.
 * Alignment: block weights (swam_block_weights), activation rows (x, x_full,
 *   y_full, x_packed, y_packed, qkv_out) and the latent-io tensors are read
 *   and written in 16-byte vectors and must be 16-byte aligned; the entry
 *   points that take them return SWAM_E_INVALID otherwise.
 * Errors: every int-returning call returns SWAM_OK (0) or a negative
 *   swam_status.  Arguments are validated on the host before any launch; on
 *   error nothing is launched and swam_last_error() describes the problem.
 *   A context is not thread-safe; use one context per stream.
 */
#ifndef SWAM_H
#define SWAM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SWAM_MAX_BLOCKS 64   /* blocks per model */
#define SWAM_MAX_FRAMES 64   /* future frames per sequence */
#define SWAM_MAX_NS 4096     /* spatial tokens per frame */
#define SWAM_MAX_BATCH 64    /* sequences per call */
/* Also: batch * L_full < 2^30 rows, and in bf16 batch * L_full * 3 * d_model
 * < 2^31 elements (32-bit offsets into the QKV buffer); swam_create rejects
 * larger configurations with SWAM_E_SHAPE. */

typedef enum { SWAM_F32 = 0, SWAM_BF16 = 1 } swam_dtype;

typedef enum {
  SWAM_OK = 0,
  SWAM_E_INVALID = -1,      /* null pointer, bad enum, inconsistent config */
  SWAM_E_SHAPE = -2,        /* a size outside what the kernels support */
  SWAM_E_DTYPE = -3,        /* dtype not supported by this call */
  SWAM_E_STATE = -4,        /* e.g. sparse step before any selection */
  SWAM_E_HIP = -5,          /* HIP runtime or launch error */
  SWAM_E_NOMEM = -6,        /* workspace allocation failed */
  SWAM_E_UNSUPPORTED = -7
} swam_status;

/* Step / selection configuration.  N_s = frame_h * frame_w, H = n_act,
 * g = H / n_frames (H must be divisible by n_frames: App. A.1). */
typedef struct {
  int32_t batch;          /* sequences per call, 1..SWAM_MAX_BATCH */
  int32_t d_model;        /* d = n_heads * head_dim */
  int32_t n_heads;
  int32_t head_dim;       /* must be 64 */
  int32_t mlp_ratio;      /* MLP hidden = mlp_ratio * d */
  int32_t n_blocks;       /* 1..SWAM_MAX_BLOCKS */
  int32_t d_temb;         /* timestep-embedding width, 1..1024 */
  int32_t n_ctx;          /* context (observation) tokens, always kept */
  int32_t n_frames;       /* F, 1..SWAM_MAX_FRAMES */
  int32_t frame_h, frame_w;
  int32_t n_act;          /* H action tokens, always kept */
  int32_t k_core;         /* K_c (ignored when mass_threshold > 0) */
  int32_t k_anchor;       /* K_s; K_c + K_s <= N_s */
  int32_t k_layer;        /* K_layer (paper default 6); min(K_layer, n_blocks) used */
  float cv_penalty;       /* c in mu / (1 + c CV); paper default 1.0 */
  float mass_threshold;   /* 0: fixed K_c.  In (0,1]: per-frame core count is
                             the smallest k >= 1 whose top-k score mass reaches
                             the threshold (an extension giving ragged lengths) */
  int32_t reuse_R;        /* refresh when tau mod R == 0; >= 1 */
  int32_t dtype;          /* swam_dtype */
  /* Backbone variants (0 = off): rope = rotary embedding of q and k at each
   * token's original position in its full sequence (pairs (2i, 2i+1) of a
   * head rotated by pos * 10000^(-2i/64); packed rows of a sparse step keep
   * their original positions, Sec. 4.2); qk_norm = unit-gain RMS
   * normalisation of every q and k head vector (eps 1e-6), applied before
   * the rotation. */
  int32_t rope;
  int32_t qk_norm;
  /* Classifier-free guidance (App. B.2 lists guidance scale 3.0 for two of
   * the backbones).  cfg_pairs = 1: the batch (even) holds P = batch/2
   * conditional sequences followed by their P unconditional partners
   * (sequence P + b pairs with b).  Scoring, score reduction and selection
   * run on the conditional half only (the statistics come from the dense
   * conditional forward, Sec. 4.2); the partner of b keeps b's retained
   * positions.  The sampler entry points keep one latent state per pair and
   * use the guided velocity v_u + guidance * (v_c - v_u).  guidance is read
   * only with cfg_pairs = 1 (must be finite). */
  int32_t cfg_pairs;
  float guidance;
} swam_config;

/* Sizes derived from a configuration (host-only, no GPU needed). */
typedef struct {
  int64_t n_s;            /* tokens per frame */
  int64_t group_size;     /* g = H / F */
  int64_t l_full;         /* tokens per full sequence */
  int64_t rows_full;      /* batch * l_full */
  int64_t k_max;          /* max retained per frame (K_c+K_s, or N_s in mass mode) */
  int64_t t_pack_fixed;   /* packed rows per sequence in fixed mode, else -1 */
  int64_t k_layer_eff;    /* min(k_layer, n_blocks) */
  int64_t workspace_bytes;/* device bytes swam_create allocates */
} swam_plan_info;

/* Weights of one block; each matrix is [out_features][in_features] row-major,
 * element type = config dtype.  Modulation order of w_ada's 6d outputs:
 * shift1, scale1, gate1, shift2, scale2, gate2. */
typedef struct {
  const void* w_ada;  const void* b_ada;   /* [6d][d_temb], [6d] */
  const void* w_qkv;  const void* b_qkv;   /* [3d][d], [3d]; output [q|k|v], heads of 64 */
  const void* w_o;    const void* b_o;     /* [d][d], [d] */
  const void* w_1;    const void* b_1;     /* [hidden][d], [hidden] */
  const void* w_2;    const void* b_2;     /* [d][hidden], [d] */
} swam_block_weights;

typedef struct {
  int32_t n_blocks;                    /* must equal config.n_blocks */
  const swam_block_weights* blocks;    /* HOST array of n_blocks entries */
} swam_model;

typedef struct swam_ctx swam_ctx;

/* ---------------------------------------------------------------- setup */

/* Validate cfg, allocate the workspace on the current HIP device and bind
 * `stream` (a hipStream_t; NULL = the null stream).  *out receives the
 * context; on error *out is NULL. */
int swam_create(const swam_config* cfg, void* stream, swam_ctx** out);
int swam_destroy(swam_ctx* ctx);
/* Bind another stream (a hipStream_t; NULL = the null stream).  Later calls
 * run on it after everything already queued on the previous stream: the new
 * stream waits on an event recorded there (no host synchronisation).  Not
 * allowed while swam_step_graph captures (SWAM_E_STATE). */
int swam_set_stream(swam_ctx* ctx, void* stream);

/* Derived sizes; validates cfg exactly as swam_create does, without a GPU. */
int swam_plan(const swam_config* cfg, swam_plan_info* out);

const char* swam_status_str(int status);
/* Last error message of ctx (or of the last failed swam_create/swam_plan on
 * this thread when ctx is NULL).  Never NULL. */
const char* swam_last_error(const swam_ctx* ctx);

/* ------------------------------------------------------- (1) scoring */

/* Spatial scores of one layer for every sequence (App. A.2):
 *   S(f,j) = (1/N_h) sum_{i in I_f} sum_h alpha_{f,i}
 *            exp(q_h(i) . k_h(f,j) / sqrt(64) - lambda_h(i))
 * with I_f the f-th consecutive group of g action queries and alpha the
 * centre-weighted group weights (central half twice the outer quarters,
 * normalised; App. B.2).
 *   q_act : sequence b, action i, head h at
 *           q_act + b*q_seq_stride + i*q_row_stride + h*64   (elements)
 *   k_fut : sequence b, future token r = f*N_s + j at
 *           k_fut + b*k_seq_stride + r*k_row_stride + h*64
 *   lse_act (mode A, the paper's method): lambda_h(i) from the dense
 *           attention, float [B][H][N_h] contiguous.
 *   k_all (mode B, used iff lse_act == NULL): every visible key of the full
 *           sequence, row r at k_all + b*kall_seq_stride + r*k_row_stride;
 *           lambda is then computed over all l_full keys in-kernel.
 *   s_out : float [B][F][N_s].
 * Strides may point inside a fused QKV buffer (row stride 3d).  With
 * guidance pairs B here (and in swam_score_reduce, swam_select's v / a and
 * the score, Q, V, A exports) is the conditional half, batch / 2. */
int swam_score(swam_ctx* ctx,
               const void* q_act, int64_t q_seq_stride, int64_t q_row_stride,
               const void* k_fut, int64_t k_seq_stride, int64_t k_row_stride,
               const float* lse_act,
               const void* k_all, int64_t kall_seq_stride,
               float* s_out);

/* Layer quality and aggregated scores (Sec. 4.1; App. A.1):
 *   R_l = (1/F) sum_{f,j} S_l(f,j); E_l = normalised spatial entropy (0 log 0
 *   = 0); Q_l = R_l (1 - E_l); L_core = the min(K_layer, L) largest Q_l
 *   (compared as float32, lowest layer on ties); V = Q-weighted mean of S_l
 *   over L_core; V_all = the same over all layers; A_j = mu_j / (1 + c CV_j)
 *   with population std over frames (A_j = 0 when mu_j = 0).  A zero weight
 *   sum falls back to the unweighted mean.  Sums are accumulated in float64.
 *   s_all : float [B][n_blocks][F][N_s]
 *   q_out : float [B][n_blocks] (optional)     v_out : float [B][F][N_s]
 *   a_out : float [B][N_s]                      core_out: int32 [B][k_layer_eff] (optional)
 * Also stores V and A in the context (consumed by swam_select(ctx, NULL, NULL, ...)). */
int swam_score_reduce(swam_ctx* ctx, const float* s_all, float* q_out, float* v_out,
                      float* a_out, int32_t* core_out);

/* ----------------------------------------------------- (2) selection */

/* Pool, cores, anchors and retained sets (Sec. 4.1; App. A.1):
 *   P = TopK_j(max_f V(f,j), N_s - K_s); C_f = TopK_{j in P}(V(f,j), K_c);
 *   E = J minus union C_f; S = TopK_{j in E}(A_j, K_s); R_f = C_f u S.
 * TopK orders by score descending, then index ascending (deterministic).
 * v, a : float [B][F][N_s], [B][N_s]; NULL = the context's own V/A from the
 *        last swam_score_reduce.
 * Outputs (each optional, NULL = not copied out):
 *   keep_idx  int32 [B][F][k_max], R_f ascending, padded with -1
 *   keep_cnt  int32 [B][F]
 *   pack_pos  int32 [B*l_full], packed row of each full row or -1 if pruned
 *   gather    int32 [B*l_full], first T_pack entries = full row of each packed row
 *   cu_seqlens int32 [B+1] packed sequence offsets
 * The selection and its packing metadata are cached in the context for
 * swam_pack / swam_unpack / sparse steps.  In mass-threshold mode the packed
 * lengths are read back to the host (one stream synchronisation). */
int swam_select(swam_ctx* ctx, const float* v, const float* a, int32_t* keep_idx,
                int32_t* keep_cnt, int32_t* pack_pos, int32_t* gather,
                int32_t* cu_seqlens);

/* Selection without allocation, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid it): the pool / core / anchor selection and pack map of swam_select
 * for explicit sizes, with no context.  Its scratch (pool, core and keep
 * flags) is a static device array of SWAM_NOALLOC_SCRATCH_BYTES per GPU that
 * the library holds until the process ends; no call allocates or frees
 * anything and nothing is read back to the host.  Calls on one GPU share that
 * array, so calls that overlap on one GPU (different streams, or host
 * threads) race: serialise them.
 *   batch, n_frames, n_s, n_ctx, n_act : sizes as in swam_config (token
 *       layout of the header; l_full = n_ctx + n_frames * n_s + n_act);
 *   k_core, k_anchor, mass_threshold : budgets as in swam_config (the
 *       threshold's numerator is the integer nearest to 1000 x the value);
 *   v, a : float [batch][n_frames][n_s], [batch][n_s] device inputs;
 *   keep_idx int32 [batch][n_frames][k_max] (k_max = max(1, k_core +
 *       k_anchor), or n_s in mass-threshold mode), keep_cnt [batch][n_frames],
 *       pack_pos and gather [batch * l_full], cu_seqlens [batch + 1]: device
 *       outputs, all required, laid out as in swam_select;
 *   stream : the hipStream_t to enqueue on (NULL = the null stream).
 * Scratch need: align256(batch * n_s) + align256(batch * n_frames * n_s) +
 * 4 * batch * l_full bytes; above SWAM_NOALLOC_SCRATCH_BYTES the call returns
 * SWAM_E_SHAPE before launching anything.  Other invalid sizes or NULL
 * pointers give SWAM_E_INVALID / SWAM_E_SHAPE; the message is in
 * swam_last_error(NULL). */
#define SWAM_NOALLOC_SCRATCH_BYTES (1 << 20)
int swam_select_noalloc(int32_t batch, int32_t n_frames, int32_t n_s, int32_t n_ctx,
                        int32_t n_act, int32_t k_core, int32_t k_anchor, float mass_threshold,
                        const float* v, const float* a, int32_t* keep_idx, int32_t* keep_cnt,
                        int32_t* pack_pos, int32_t* gather, int32_t* cu_seqlens, void* stream);

/* Random-selection baseline (the component ablation compares the method
 * with tokens chosen at random at the same per-frame budget): per scored
 * sequence and frame, the K_c + K_s positions with the largest uniform keys
 * (ties to the lower index), i.e. a uniformly random subset drawn
 * independently per frame, no anchors.  The keys are the top 24 bits of word
 * 0 of Philox4x64-10 (Salmon et al., SC 2011) at counter
 * ((b * F + f) * N_s + j, 0, 0, 0) and key (seed, 0), times 2^-24; they
 * replace the context's V (A is cleared).  Outputs as in swam_select; the
 * selection is cached for sparse steps (with guidance pairs the partner
 * shares it).  SWAM_E_UNSUPPORTED in mass-threshold mode. */
int swam_select_random(swam_ctx* ctx, uint64_t seed, int32_t* keep_idx, int32_t* keep_cnt,
                       int32_t* pack_pos, int32_t* gather, int32_t* cu_seqlens);

/* Import a selection (int32 [B][F][k_max] ascending, -1 padded; counts
 * [B][F]; with guidance pairs B is the whole batch, partners included) and
 * rebuild the packing metadata.  Indices outside [0, N_s) are
 * ignored.  Synchronises once to read the packed lengths. */
int swam_set_selection(swam_ctx* ctx, const int32_t* keep_idx, const int32_t* keep_cnt);

/* Host value of the cached packed row count (sum over sequences). */
int swam_packed_rows(swam_ctx* ctx, int64_t* rows);

/* Copy cached state out (each pointer optional): the last refresh's scores
 * (float [B][n_blocks][F][N_s]), Q, V, A and the cached selection (layouts as
 * in swam_score_reduce / swam_select). */
int swam_export(swam_ctx* ctx, float* s_all, float* q, float* v, float* a,
                int32_t* keep_idx, int32_t* keep_cnt, int32_t* pack_pos,
                int32_t* gather, int32_t* cu_seqlens);

/* ---------------------------------------------- (3) pack, (5) unpack */

/* x_packed[r] = x_full[gather[r]] for r < T_pack (cached selection). */
int swam_pack(swam_ctx* ctx, const void* x_full, void* x_packed);

/* y_full[t] = y_packed[pack_pos[t]] where kept, x_full[t] where pruned.
 * If y_full == x_full only the retained rows are written (in place); pruned
 * rows are bit-identical to x_full either way. */
int swam_unpack(swam_ctx* ctx, const void* y_packed, const void* x_full, void* y_full);

/* ---------------------------------------------------------- (4) block */

/* One adaLN DiT block, in place on x [n_rows][d]:
 *   m = W_ada SiLU(temb) + b_ada -> (sh1, sc1, g1, sh2, sc2, g2)
 *   h = LN(x)(1+sc1)+sh1; [q|k|v] = h W_qkv^T + b_qkv
 *   o = softmax(q k^T / 8) v over the keys of the row's own sequence
 *   x += g1 (o W_o^T + b_o); h2 = LN(x)(1+sc2)+sh2
 *   x += g2 (GELU_tanh(h2 W_1^T + b_1) W_2^T + b_2)
 * With rope / qk_norm set, q and k are normalised / rotated after the
 * projection; a row's position is its index in its full sequence for the
 * dense layout (cu_seqlens == NULL) and its index inside its cu_seqlens
 * sequence otherwise (swam_step's sparse blocks use the original positions).
 * LN: biased variance, eps 1e-6, no affine.  temb: float [d_temb] (shared by
 * the batch).  cu_seqlens: device int32 [n_seqs+1] with cu[n_seqs] == n_rows,
 * or NULL for the dense layout (n_rows == B*l_full).  lse_out (optional):
 * float [n_rows][N_h] natural-log attention normalisers.  qkv_out (optional):
 * receives the [n_rows][3d] projection.  n_rows <= B*l_full. */
int swam_block(swam_ctx* ctx, const swam_block_weights* w, const float* temb, void* x,
               int64_t n_rows, const int32_t* cu_seqlens, int32_t n_seqs,
               float* lse_out, void* qkv_out);

/* ----------------------------------------------------------- step */

#define SWAM_STEP_FORCE_DENSE 1    /* dense step, no scoring, cache untouched */
#define SWAM_STEP_FORCE_REFRESH 2  /* refresh regardless of tau */

#define SWAM_KIND_DENSE 0
#define SWAM_KIND_REFRESH 1
#define SWAM_KIND_SPARSE 2

/* One denoising step x_full [B*l_full][d] -> y_full.  y_full is either
 * x_full itself (in place) or a buffer disjoint from it; a partial overlap
 * returns SWAM_E_INVALID.
 * Refresh (tau mod R == 0 or FORCE_REFRESH): dense blocks with scoring of
 * every layer, then score reduce, selection and packing metadata, cached.
 * Sparse: pack -> blocks on the packed sequences -> unpack; pruned rows of
 * y_full equal x_full bit for bit.  The pack runs inside the first block's
 * first LayerNorm kernel; in bf16 the unpack runs inside the last block's MLP
 * down projection, whose store writes each packed row straight to its row of
 * y_full (fp32: a separate scatter pass), so SWAM_T_UNPACK records no bf16
 * launch.  Returns SWAM_E_STATE for a sparse step
 * with no cached selection.  *kind_out (optional, host) receives SWAM_KIND_*. */
int swam_step(swam_ctx* ctx, const swam_model* model, const void* x_full,
              const float* temb, int32_t tau, void* y_full, int32_t flags,
              int32_t* kind_out);

/* As swam_step, but every distinct step -- same kind, x_full, y_full, temb,
 * weight pointers and packed length -- is captured once into a HIP graph on
 * the context stream and replayed afterwards, so the fixed-length step costs
 * one launch on the host (the paper's engine gains most from graph capture of
 * its fixed-length sparse step; Sec. 5 and App. B.4).  Needs a non-default
 * stream (SWAM_E_STATE otherwise).  Mass-threshold refresh steps read their
 * packed lengths back and run eagerly.  Graphs are cached (at most 64, oldest
 * evicted); the buffers they reference must stay valid while cached.  Timers
 * do not bracket captured work. */
int swam_step_graph(swam_ctx* ctx, const swam_model* model, const void* x_full,
                    const float* temb, int32_t tau, void* y_full, int32_t flags,
                    int32_t* kind_out);
/* Synchronise and free every cached graph of ctx. */
int swam_graph_clear(swam_ctx* ctx);

/* --------------------------------------------------- diagnostics */

/* Overlap of spatial distributions (App. C, attention-overlap eq.):
 *   out[m] = sum_i min(p_m[i] / sum_i p_m[i], q_m[i] / sum_i q_m[i])
 * for n_maps pairs of non-negative float maps of n values each, p and q
 * [n_maps][n] contiguous, out float [n_maps]; a map of zero mass gives 0.
 * Sums in float64.  E.g. cross-step overlap of V from two refreshes, or
 * cross-frame overlap of V(f) and V(f+1). */
int swam_overlap(swam_ctx* ctx, const float* p, const float* q, int64_t n_maps, int64_t n,
                 float* out);

/* ------------------------------------------ sampling update (Sec. 4.2) */

/* Latent read-in and read-out of the backbone (c = d_latent channels per
 * token, 1..64, with c * d_model * element size <= 64 KB; matrices
 * [out_features][in_features] row-major in the config dtype; weights, z,
 * x_full and y_full 16-byte aligned, else SWAM_E_INVALID).  Latent tensors -- z, velocities v, the velocity cache -- are float
 * [B][L_lat][c] with L_lat = F*N_s + H: the future tokens of each sequence
 * (frame-major, row-major in a frame) followed by its action tokens, i.e. the
 * full-layout rows n_ctx .. l_full-1 of every sequence.  With guidance pairs
 * z and the cache cover the P conditional sequences ([P][L_lat][c], one
 * state per pair) while v holds both branches ([B][L_lat][c], conditional
 * half first). */
typedef struct {
  int32_t d_latent;
  const void* w_in;  const void* b_in;     /* [d][c], [d]: token = z W_in^T + b_in */
  const void* w_v;   const void* b_v;      /* [c][d], [c]: v = LN(y) W_v^T + b_v   */
} swam_latent_io;

/* Tokens of the latent rows of x_full [B*l_full][d] from z (stored in the
 * config dtype); context rows are not touched.  With guidance pairs both
 * sequences of a pair get the tokens of the pair's latent state. */
int swam_embed(swam_ctx* ctx, const swam_latent_io* io, const float* z, void* x_full);

/* Velocity read-out v = LN(y) W_v^T + b_v (LayerNorm without affine, eps
 * 1e-6) of the latent rows of y_full.  retained_only != 0: only the rows of
 * the cached selection (retained future tokens and all action tokens; other
 * rows of v are left as they are; SWAM_E_STATE without a selection). */
int swam_velocity(swam_ctx* ctx, const swam_latent_io* io, const void* y_full,
                  int32_t retained_only, float* v);

/* One sampler update of z in place (c = d_latent channels), z <- z + dsigma * v~, where v~ is
 *   kind SWAM_KIND_DENSE  : v;
 *   kind SWAM_KIND_REFRESH: v, and the future-token rows of v are stored in
 *                           v_cache (the full step caches the visual velocity);
 *   kind SWAM_KIND_SPARSE : the paper's merge M v + (1 - M) v_cache over the
 *                           future tokens, M = the cached selection (Sec. 4.2,
 *                           cached visual prediction eq.); action rows take v.
 * (fp32 FMA per element.)  v_cache may be NULL for SWAM_KIND_DENSE.  With
 * guidance pairs "v" above is the guided v_u + guidance * (v_c - v_u) of the
 * two branch rows of v (one fp32 FMA), which is also what the cache holds. */
int swam_sample_update(swam_ctx* ctx, int32_t d_latent, const float* v, float* v_cache,
                       float* z, float dsigma, int32_t kind);

/* Noise levels of the sampler's flow schedule with a shift (the paper's
 * backbones use shift 5.0, App. B.2): sigma_i = shift s / (1 + (shift - 1) s)
 * with s = 1 - i / n_steps, for i = 0 .. n_steps, from 1 (pure noise) down to
 * 0; the model time of step i is 1000 sigma_i and its update uses
 * dsigma = sigma_{i+1} - sigma_i.  sigmas is a HOST array of n_steps + 1
 * doubles owned by the caller.  Pure host arithmetic: needs no context, no
 * GPU and no stream.  SWAM_E_INVALID for n_steps < 1, a shift that is not
 * finite and positive, or sigmas NULL. */
int swam_flow_sigmas(int32_t n_steps, double shift, double* sigmas);

/* One closed-loop sampling step: swam_embed(z -> x_full), swam_step(x_full ->
 * y_full), swam_velocity (all latent rows after a full step, the retained
 * rows after a sparse one) and swam_sample_update with the step's kind.
 * x_full must hold the context tokens in its context rows and must not
 * alias y_full (the context rows stay the conditioning of the next step).
 * dsigma = sigma_{tau+1} - sigma_tau of the caller's schedule (the paper's
 * backbones use a flow schedule with shift 5.0, App. B.2); temb encodes the
 * model time of step tau. */
int swam_sample_step(swam_ctx* ctx, const swam_model* model, const swam_latent_io* io,
                     float* z, float* v, float* v_cache, void* x_full, void* y_full,
                     const float* temb, int32_t tau, float dsigma, int32_t flags,
                     int32_t* kind_out);

/* --------------------------------------------------------- timers */

/* Kernel / phase classes for on-stream timing with HIP events. */
enum {
  SWAM_T_ADALN = 0, SWAM_T_LNMOD, SWAM_T_GEMM_QKV, SWAM_T_ATTN, SWAM_T_GEMM_OUT,
  SWAM_T_GEMM_UP, SWAM_T_GEMM_DOWN, SWAM_T_SCORE, SWAM_T_REDUCE, SWAM_T_SELECT,
  SWAM_T_PACK, SWAM_T_UNPACK, SWAM_T_COPY, SWAM_T_SAMPLE, SWAM_T_QK_POST, SWAM_T_COUNT
};

/* Bracket every launch (phase) of the classes in `mask` (bit i = class i)
 * with HIP events on the stream it runs on; mask 0 disables.  Enabling
 * allocates an event pool of `capacity` pairs (dropped beyond that) and
 * restarts the per-class launch counts of swam_timer_stride (the stride
 * itself is kept).  Each bracket costs the stream a few microseconds. */
int swam_timer_enable(swam_ctx* ctx, uint32_t mask, int32_t capacity);
/* Forget the recorded brackets and restart the launch counts. */
int swam_timer_reset(swam_ctx* ctx);
/* Bracket only launches whose ordinal within their class (0, 1, ... since
 * the last enable / reset / this call) is a multiple of `stride` (>= 1;
 * 1, the default, brackets every launch).  Synchronises the stream, drops
 * the recorded brackets; SWAM_E_INVALID for stride < 1.  With a stride
 * that divides a class's launches per step, every step contributes the
 * same launch positions. */
int swam_timer_stride(swam_ctx* ctx, int32_t stride);
/* Synchronise the stream and return the launch count and summed duration
 * of the bracketed launches of class `cls` since the last reset. */
int swam_timer_read(swam_ctx* ctx, int32_t cls, int64_t* launches, double* total_ms);

#define SWAM_KIND_NONE (-1)  /* launches outside swam_step / swam_sample_step */
#define SWAM_KIND_ANY (-2)   /* every launch (swam_timer_read) */

/* As swam_timer_read, restricted to the launches enqueued by steps of one
 * kind (SWAM_KIND_DENSE / _REFRESH / _SPARSE, from swam_step,
 * swam_sample_step and the eager path of swam_step_graph), by none
 * (SWAM_KIND_NONE: swam_block, swam_score, ...), or by any (SWAM_KIND_ANY).
 * SWAM_E_INVALID for another kind or class. */
int swam_timer_read_kind(swam_ctx* ctx, int32_t cls, int32_t kind, int64_t* launches,
                         double* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* SWAM_H */
