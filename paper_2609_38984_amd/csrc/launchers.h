// Host-side launchers of the libswam kernels (one per kernel family, all
// asynchronous on the given stream) and their argument structs.
#pragma once
#include "common.h"

namespace swam {

// ---------------------------------------------------------------------------
// launchers (host side), one per kernel family; all asynchronous on `st`
// ---------------------------------------------------------------------------
// EPI_PARTIAL is internal to the bf16 split-K path (fp32 partial sums);
// EPI_BIAS_QKPOST to launch_gemm_qkv
enum Epilogue { EPI_BIAS = 0, EPI_BIAS_GELU = 1, EPI_BIAS_GATED_RESIDUAL = 2, EPI_PARTIAL = 3,
                EPI_BIAS_QKPOST = 4 };

// QK-norm / rotary embedding of the q and k columns of a QKV projection
// (the arguments of launch_qk_post): d = model width (q columns [0, d), k
// columns [d, 2d)); pos_mode 0 = dense rows (position row % l_full), 1 =
// packed rows (gather[row] % l_full), 2 = index inside the cu_seqlens
// sequence; tab = rotary table [n_pos][32] (NULL: no rotation).
struct QkPost {
  int d = 0, pos_mode = 0, n_seqs = 0, l_full = 1, n_pos = 1, qk_norm = 0;
  const int32_t* gather = nullptr;
  const int32_t* cu = nullptr;
  const float2* tab = nullptr;
};

// The four projections of a block; the role fixes the epilogue:
// QKV bias, UP bias + tanh-GELU, OUT and DOWN bias + gated residual.
enum GemmRole { ROLE_QKV = 0, ROLE_OUT = 1, ROLE_UP = 2, ROLE_DOWN = 3 };

// C[M][N] = epi(A[M][K] . B[N][K]^T + bias[N]); for the gated residual
// C[m][n] = C[m][n] + gate[n] * (acc + bias[n]) (C read then written).
// ws / ws_floats: fp32 workspace the bf16 path may use to split K when the
// output tiles alone cannot fill the CUs (partial sums, then one reduce +
// epilogue pass); NULL or too small means no split.
// smap (bf16 OUT / DOWN only): row m of the result goes to Cs[smap[m]] (same
// ldc) instead of C[m]; the residual is still read from C[m].  The scatter of
// a packed sequence's rows back into the full latent rides on the last
// projection this way.
hipError_t launch_gemm(int dtype, int role, const void* A, int64_t lda, const void* B,
                       int64_t ldb, const void* bias, const float* gate, void* C,
                       int64_t ldc, int64_t M, int64_t N, int64_t K, hipStream_t st,
                       float* ws = nullptr, int64_t ws_floats = 0, void* Cs = nullptr,
                       const int32_t* smap = nullptr);

// QKV projection C = A . B^T + bias followed by the QK-norm / rotary
// embedding of qp on its q and k columns, with the same bf16 rounding of the
// projection as launch_gemm + launch_qk_post; fused into the GEMM's store
// for bf16 unless the shape splits K (then the two launches).
hipError_t launch_gemm_qkv(int dtype, const void* A, int64_t lda, const void* B, int64_t ldb,
                           const void* bias, void* C, int64_t ldc, int64_t M, int64_t N,
                           int64_t K, const QkPost& qp, hipStream_t st, float* ws = nullptr,
                           int64_t ws_floats = 0);

// mod[blk][6d] = W_ada[blk] SiLU(temb) + b_ada[blk] for n_blk blocks at once.
struct AdalnArgs {
  const void* w[64];
  const void* b[64];
};
hipError_t launch_adaln(int dtype, const AdalnArgs& a, int n_blk, const float* temb,
                        int d_temb, int d6, float* mod, hipStream_t st);

// h[r] = LN(x[r]) (1 + scale) + shift
hipError_t launch_ln_mod(int dtype, const void* x, void* h, const float* shift,
                         const float* scale, int64_t rows, int d, hipStream_t st);
// the same on gathered rows: xp[r] = x_full[gather[r]] (the gather-pack) and
// h[r] = LN(xp[r]) (1 + scale) + shift, in one pass
hipError_t launch_ln_mod_gather(int dtype, const void* x_full, const int32_t* gather, void* xp,
                                void* h, const float* shift, const float* scale, int64_t rows,
                                int d, hipStream_t st);

// backbone variants: rotary table and QK-norm / RoPE of the stored q and k
hipError_t launch_rope_table(float2* tab, int n_pos, hipStream_t st);
hipError_t launch_qk_post(int dtype, void* qkv, int64_t n_rows, int d, int pos_mode,
                          const int32_t* gather, const int32_t* cu, int n_seqs, int l_full,
                          const float2* tab, int n_pos, int qk_norm, hipStream_t st);

// o = softmax(q k^T / 8) v per head inside each sequence; lse (optional).
// Sequence bounds are clamped to [0, n_rows].
hipError_t launch_attention(int dtype, const void* qkv, void* o, float* lse,
                            const int32_t* cu_seqlens, int n_seqs, int64_t n_rows,
                            int n_heads, hipStream_t st);

// Score kernels (mode A with lse, mode B computes lse first into lse_ws).
struct ScoreArgs {
  const void* q; int64_t q_seq, q_row;
  const void* k; int64_t k_seq, k_row;
  const float* lse;           // sequence b, query i, head h at lse + b*lse_seq + i*N_h + h
  int64_t lse_seq;
  float* s_out;               // sequence b, frame f at s_out + b*s_seq + f*N_s
  int64_t s_seq;
  const float* alpha;         // [g] device
  int B, F, n_s, H, n_heads;
  int n_layers;               // layers scored by one launch (>= 1)
  int64_t q_lay, k_lay, lse_lay, s_lay;   // element strides between layers
};
hipError_t launch_score(int dtype, const ScoreArgs& a, hipStream_t st);
// MLP up projection (bias + GELU) of a refresh step with one layer's scores
// (ScoreArgs, bf16) computed by extra workgroups in the tail of its grid, on
// the CUs its last round of tiles leaves idle; gemm_up_scored_slots returns
// how many that is for a shape (0: not applicable, the caller scores
// separately), and launch_gemm_up_scored returns hipErrorNotSupported then.
int gemm_up_scored_slots(int64_t M, int64_t N, int64_t K, int64_t ws_floats);
hipError_t launch_gemm_up_scored(const void* A, int64_t lda, const void* B, int64_t ldb,
                                 const void* bias, void* C, int64_t ldc, int64_t M, int64_t N,
                                 int64_t K, const ScoreArgs& sa, hipStream_t st,
                                 int64_t ws_floats);
hipError_t launch_lse_all(int dtype, const void* q, int64_t q_seq, int64_t q_row,
                          const void* kall, int64_t k_seq, int64_t k_row, int64_t n_keys,
                          int B, int H, int n_heads, float* lse_out, float* part_ws,
                          hipStream_t st);

// Score reduction (layer quality, core layers, V, A).
struct ReduceArgs {
  const float* s_all;  // [B][L][F][N_s]
  double* frame_sum;   // ws [B][L][F]
  double* frame_ent;   // ws [B][L][F]
  float* q;            // [B][L]
  int32_t* core;       // [B][k_layer_eff]
  double* qd;          // ws [B][L] float64 quality
  float* v;            // [B][F][N_s]
  float* a;            // [B][N_s]
  double* vall;        // ws [B][F][N_s] float64 V_all
  int B, L, F, n_s, k_layer;
  float cv_penalty;
};
hipError_t launch_score_reduce(const ReduceArgs& a, hipStream_t st);

// Selection and packing metadata.
struct SelectArgs {
  const float* v;      // [B][F][N_s]
  const float* a;      // [B][N_s]
  uint8_t* pool;       // ws [B][N_s]
  uint8_t* core;       // ws [B][F][N_s]
  int32_t* keep_idx;   // [B][F][k_max]
  int32_t* keep_cnt;   // [B][F]
  int32_t* keep;       // ws [B*L_full] 0/1
  int B, F, n_s, k_core, k_anchor, k_max;
  int mass_num, mass_den;  // mass threshold as a fraction; den == 0: fixed K_c
  int n_ctx, n_act;
};
hipError_t launch_select(const SelectArgs& a, hipStream_t st);
// uniform keys in [0, 1) (top 24 bits of word 0 of Philox4x64-10 at counter
// (i, 0, 0, 0), key (seed, 0)) into v[i] for i < n, and zeros into a[n_a]
// (n_a <= n)
hipError_t launch_random_keys(float* v, int64_t n, float* a, int64_t n_a, uint64_t seed,
                              hipStream_t st);
// keep flags from an imported selection; rewrites keep_idx / keep_cnt ascending
hipError_t launch_keep_from_idx(const int32_t* in_idx, int32_t* keep_idx, int32_t* keep_cnt,
                                int32_t* keep, int B, int F, int n_s, int k_max, int n_ctx,
                                int n_act, hipStream_t st);
// exclusive scan of keep flags -> pack_pos, gather, cu_seqlens
hipError_t launch_packmap(const int32_t* keep, int32_t* pack_pos, int32_t* gather,
                          int32_t* cu, int B, int64_t l_full, hipStream_t st);
hipError_t launch_pack(const void* x_full, void* x_packed, const int32_t* gather,
                       int64_t rows, int64_t row_bytes, hipStream_t st);
hipError_t launch_unpack_scatter(const void* y_packed, void* y_full, const int32_t* gather,
                                 int64_t rows, int64_t row_bytes, hipStream_t st);
hipError_t launch_unpack_merge(const void* y_packed, const void* x_full, void* y_full,
                               const int32_t* pack_pos, int64_t rows, int64_t row_bytes,
                               hipStream_t st);
hipError_t launch_overlap(const float* p, const float* q, int64_t n_maps, int64_t n,
                          float* out, hipStream_t st);

// sampling update (k_sampler.hip)
// z_rows: latent rows of z; the latent rows of sequences past them (the
// unconditional partners of guidance pairs) read z row i - z_rows
hipError_t launch_embed(int dtype, const float* z, const void* w_in, const void* b_in, void* x,
                        int64_t n_lat_rows, int64_t z_rows, int l_lat, int l_full, int n_ctx,
                        int c, int d, hipStream_t st);
hipError_t launch_velocity(int dtype, const void* y, const int32_t* gather, int64_t n_items,
                           const void* w_v, const void* b_v, float* v, int l_lat, int l_full,
                           int n_ctx, int c, int d, hipStream_t st);
// pairs: v holds 2 * n_lat_rows rows (conditional, then unconditional) that
// are combined as v_u + guidance * (v_c - v_u) before the merge
hipError_t launch_sample_update(const float* v, float* v_cache, float* z, const int32_t* pack_pos,
                                float dsigma, int kind, int64_t n_lat_rows, int l_lat, int l_full,
                                int n_ctx, int n_fut, int c, int pairs, float guidance,
                                hipStream_t st);
hipError_t launch_copy(const void* src, void* dst, int64_t bytes, hipStream_t st);
// y_full row r = x_full row r where pack_pos[r] < 0 (the pruned rows)
hipError_t launch_copy_pruned(const void* x_full, void* y_full, const int32_t* pack_pos,
                              int64_t rows, int64_t row_bytes, hipStream_t st);

}  // namespace swam
