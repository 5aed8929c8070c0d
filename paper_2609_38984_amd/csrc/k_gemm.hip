// Dense projections of the DiT block: C = epi(A . B^T + bias).
//
// A [M][K] activations and B [N][K] weights are both K-contiguous, so every
// MFMA operand is eight consecutive bf16 of one row.  bf16 path: workgroup
// tile BM x BN x 64, waves arranged WM x WN, each wave a grid of 32x32x16
// MFMA tiles with fp32 accumulators; A/B tiles double-buffered in LDS with a
// 16-byte-chunk XOR swizzle (chunk ^ lds_swz(row)) so the column reads of the
// MFMA operand layout are spread over all banks.  Workgroup ids are remapped
// so that each XCD (dispatch round-robins over 8) receives a contiguous run
// of tiles, grouped GROUP_M tile-rows deep, to share its L2.
// Epilogues (bias, tanh-GELU, gated residual) are fused into the store.
// Split K: when the output tiles cannot fill the 256 CUs (few rows, or a
// narrow N), grid.y workgroups share a tile along K, store fp32 partial sums,
// and one memory-bound pass sums them and applies the epilogue.
#include "score_unit.h"

#include <algorithm>

namespace swam {

__device__ __forceinline__ float gelu_tanh(float u) {
  // 0.5 u (1 + tanh(z)) = u / (1 + exp(-2 z)), z = sqrt(2/pi) (u + 0.044715 u^3);
  // exp(-2z) = exp2(-2 log2(e) z) on the hardware exp2, then the hardware reciprocal
  // (both about 1 ulp: far below the bf16 rounding of the stored result)
  const float z2 = -2.0f * 1.4426950408889634f * 0.7978845608028654f *
                   (u + 0.044715f * u * u * u);
  return u * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z2));
}

template <int EPI>
__device__ __forceinline__ float epi_value(float acc, float bias, float gate, float resid) {
  if (EPI == EPI_BIAS) return acc + bias;
  if (EPI == EPI_BIAS_GELU) return gelu_tanh(acc + bias);
  return resid + gate * (acc + bias);
}

// Store of 8 consecutive QKV columns of one row with the QK-norm / rotary
// embedding of q and k heads applied (the steps of qk_post_kernel on the
// projection rounded to bf16).  The 8 lanes storing one row's 64 columns are
// consecutive and aligned, and a wave's 64 columns are one head, so the head
// norm is a 3-step exchange; every lane takes part (the store is guarded).
__device__ __forceinline__ void qkpost_store(const float* v, const bf16_t* __restrict__ bias,
                                             bf16_t* C, int64_t ldc, int row, int col, int col0,
                                             int M, int N, const QkPost& qp) {
  float x[8];
  {
    const float4 v0 = *reinterpret_cast<const float4*>(v);
    const float4 v1 = *reinterpret_cast<const float4*>(v + 4);
    const float a[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
    uint4 bw = make_uint4(0u, 0u, 0u, 0u);
    if (col < N) bw = *reinterpret_cast<const uint4*>(bias + col);
    const uint32_t bb[4] = {bw.x, bw.y, bw.z, bw.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      // the projection is stored (rounded to bf16) before the post-processing
      x[2 * e] = bf16_to_f32(f32_to_bf16(a[2 * e] + __uint_as_float(bb[e] << 16)));
      x[2 * e + 1] = bf16_to_f32(f32_to_bf16(a[2 * e + 1] + __uint_as_float(bb[e] & 0xFFFF0000u)));
    }
  }
  if (col0 < 2 * qp.d) {                      // q or k head (wave-uniform)
    if (qp.qk_norm) {
      float ss = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(x[e], x[e], ss);
      ss += __shfl_xor(ss, 1);
      ss += __shfl_xor(ss, 2);
      ss += __shfl_xor(ss, 4);
      const float r = rsqrtf(ss / 64.0f + 1e-6f);
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] *= r;
    }
    if (qp.tab != nullptr) {
      const int rr = min(row, M - 1);
      int pos;
      if (qp.pos_mode == 0) {
        pos = rr % qp.l_full;
      } else if (qp.pos_mode == 1) {
        pos = qp.gather[rr] % qp.l_full;
      } else {
        int b = 0;
        while (b + 1 < qp.n_seqs && qp.cu[b + 1] <= rr) ++b;
        pos = rr - qp.cu[b];
      }
      pos = min(max(pos, 0), qp.n_pos - 1);
      const float2* t = qp.tab + (int64_t)pos * 32 + ((col & 63) >> 1);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float2 cs = t[e];
        const float a = x[2 * e], b = x[2 * e + 1];
        x[2 * e] = a * cs.x - b * cs.y;
        x[2 * e + 1] = a * cs.y + b * cs.x;
      }
    }
  }
  if (row < M && col < N)
    *reinterpret_cast<uint4*>(C + (int64_t)row * ldc + col) =
        make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                   pack_bf16x2(x[6], x[7]));
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------
constexpr int GEMM_BK = 64;
constexpr int GROUP_M = 8;

__device__ __forceinline__ void tile_of(int pid, int nwg, int tiles_m, int tiles_n, int& tm,
                                        int& tn) {
  // XCD remap: ids with equal (pid % 8) run on one XCD; give them consecutive ids.
  const int xcd = pid & 7;
  const int per = nwg >> 3, rem = nwg & 7;
  const int id = xcd * per + min(xcd, rem) + (pid >> 3);
  const int in_group = GROUP_M * tiles_n;
  const int group = id / in_group;
  const int first_m = group * GROUP_M;
  const int gsz = min(tiles_m - first_m, GROUP_M);
  tm = first_m + (id % in_group) % gsz;
  tn = (id % in_group) / gsz;
}

typedef __attribute__((address_space(3))) void lds_void_t;

// dword 3 of a raw buffer descriptor on gfx9-family parts (32-bit data format)
constexpr int SWAM_BUF_DWORD3 = 0x00020000;

// per-lane offset + wave-uniform step, formed at the point of use: an asm add
// keeps the compiler from hoisting one live VGPR per slab out of the k loop
__device__ __forceinline__ int vadd_sgpr(int v, int s) {
  int r;
  asm volatile("v_add_u32 %0, %1, %2" : "=v"(r) : "s"(s), "v"(v));
  return r;
}

// one k-stage (64) of MFMAs from a staged A/B tile pair.  The operand
// fragments of k-step s + 1 are read from LDS while the MFMAs of k-step s
// run (two fragment sets), and the schedule interleaves one LDS read after
// each MFMA so the reads never queue behind a whole MFMA group.
template <int BM, int BN, int TM, int TN, int FM, int FN>
__device__ __forceinline__ void mma_stage(const uint4* __restrict__ as, const uint4* __restrict__ bs,
                                          int wm, int wn, int lane, f32x16 (&acc)[FM][FN]) {
  constexpr int KS = GEMM_BK / 16;
  // fragment reads of the next k-step paired with this k-step's MFMAs; with
  // fewer MFMAs than reads (the 96 x 32 wave tile) the rest follow as a group
  constexpr int PAIRS = FM * FN < FM + FN ? FM * FN : FM + FN;
  const int khalf = lane >> 5, r31 = lane & 31;
  const int sw = lds_swz(r31);   // rows differ from r31 by multiples of 32
  bf16x8 af[2][FM], bfr[2][FN];
  auto load = [&](int s, int buf) {
    const int chunk = (2 * s + khalf) ^ sw;
#pragma unroll
    for (int i = 0; i < FM; ++i)
      af[buf][i] = __builtin_bit_cast(bf16x8, as[(wm * TM + i * 32 + r31) * 8 + chunk]);
#pragma unroll
    for (int j = 0; j < FN; ++j)
      bfr[buf][j] = __builtin_bit_cast(bf16x8, bs[(wn * TN + j * 32 + r31) * 8 + chunk]);
  };
  load(0, 0);
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    if (s + 1 < KS) load(s + 1, (s + 1) & 1);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s & 1][i], bfr[s & 1][j], acc[i][j],
                                                            0, 0, 0);
  }
  // schedule: the first fragment set, then per k-step (MFMA, LDS read) pairs
  // for the next set followed by the remaining MFMAs; the last k-step's MFMAs
  __builtin_amdgcn_sched_group_barrier(0x100, FM + FN, 0);
#pragma unroll
  for (int s = 0; s + 1 < KS; ++s) {
#pragma unroll
    for (int r = 0; r < PAIRS; ++r) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    if constexpr (FM + FN > PAIRS)
      __builtin_amdgcn_sched_group_barrier(0x100, FM + FN - PAIRS, 0);
    if constexpr (FM * FN > PAIRS)
      __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - PAIRS, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);
}

// Stage loads go global -> LDS directly (no registers) as buffer loads: each
// instruction moves 8 rows x 128 bytes; lane i lands at slot i of the 1 KB
// slab, i.e. row lane >> 3 and physical chunk lane & 7, so it fetches logical
// chunk (lane & 7) ^ lds_swz(row) -- the swizzle is applied on the global
// side.  The descriptors start at the tile's first row and end at the last
// row of the operand, so the rows of a ragged last tile read as zeros (the
// hardware range check) and every offset stays below 2^31.  A wave's slabs
// are 8 rows apart; only bit 3 of the row enters the swizzle, so two
// per-lane offsets (even / odd slab) plus a wave-uniform step address them
// all.
// ROLE (a GemmRole) only names the instantiation after the block's
// projection, so a kernel trace tells the four projections apart.
// SC: workgroups past the tile count (the grid's tail) score one layer
// instead (scoring units of score_unit.h, two per 8-wave workgroup at a time),
// on the CUs that the last round of tiles leaves idle; sa / n_units describe
// that work.
template <int ROLE, int BM, int BN, int WM, int WN, int EPI, bool SC = false>
__global__ void __launch_bounds__(WM * WN * 64)
gemm_bf16_nt(const bf16_t* __restrict__ A, int64_t lda, const bf16_t* __restrict__ B,
             int64_t ldb, const bf16_t* __restrict__ bias, const float* __restrict__ gate,
             bf16_t* C, int64_t ldc, int M, int N, int K, int tiles_m, int tiles_n,
             float* __restrict__ part, const QkPost qp, const ScoreArgs sa, int n_units,
             bf16_t* Cs, const int32_t* __restrict__ smap) {
  constexpr int NW = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int A_INS = BM / 8 / NW, B_INS = BN / 8 / NW;
  static_assert(A_INS * 8 * NW == BM && B_INS * 8 * NW == BN, "tile/waves mismatch");
  __shared__ uint4 lds[2 * (BM + BN) * 8];   // [stage][A rows | B rows][8 chunks]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int n_tiles = tiles_m * tiles_n;
  if constexpr (SC) {
    static_assert(NW % 4 == 0, "scoring units take groups of four waves");
    if ((int)blockIdx.x >= n_tiles) {
      constexpr int G = NW / 4;
      const int group = wave >> 2;
      float (*sp)[16] = reinterpret_cast<float (*)[16]>(lds) + 4 * group;
      const int nsw = (int)gridDim.x - n_tiles;
      for (int base = ((int)blockIdx.x - n_tiles) * G; base < n_units; base += nsw * G) {
        __syncthreads();                 // the previous units' partial sums are consumed
        const int unit = base + group;
        score_unit_bf16(sa, unit, unit < n_units, wave & 3, lane, tid & 255, sp,
                        [] { __syncthreads(); });
      }
      return;
    }
  }
  int tm, tn;
  tile_of(blockIdx.x, n_tiles, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int wm = wave / WN, wn = wave % WN;
  const int lrow = lane >> 3;

  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(A + (int64_t)m0 * lda), (short)0,
      (int)min((int64_t)(M - m0) * lda * 2, (int64_t)0x7fffffff), SWAM_BUF_DWORD3);
  const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(B + (int64_t)n0 * ldb), (short)0,
      (int)min((int64_t)(N - n0) * ldb * 2, (int64_t)0x7fffffff), SWAM_BUF_DWORD3);
  // With an even slab count per wave, a wave's slabs start on a multiple of
  // 16 rows, so two offsets (even / odd slab) plus a 16-row step address them
  // all.  With an odd count bit 3 of a slab's first row alternates with the
  // wave, so every slab keeps its own offset.
  constexpr int NA = A_INS % 2 == 0 ? 2 : A_INS, NB = B_INS % 2 == 0 ? 2 : B_INS;
  int va[NA], vb[NB];
  if constexpr (A_INS % 2 == 0 && B_INS % 2 == 0) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int ch = (lane & 7) ^ lds_swz(8 * p + lrow);
      va[p] = (int)(((int64_t)(wave * A_INS * 8 + 8 * p + lrow) * lda + 8 * ch) * 2);
      vb[p] = (int)(((int64_t)(wave * B_INS * 8 + 8 * p + lrow) * ldb + 8 * ch) * 2);
    }
  } else {
#pragma unroll
    for (int p = 0; p < NA; ++p) {
      const int r = wave * A_INS * 8 + 8 * p + lrow;
      const int ch = (lane & 7) ^ lds_swz(A_INS % 2 == 0 ? 8 * p + lrow : r);
      va[p] = (int)(((int64_t)r * lda + 8 * ch) * 2);
    }
#pragma unroll
    for (int p = 0; p < NB; ++p) {
      const int r = wave * B_INS * 8 + 8 * p + lrow;
      const int ch = (lane & 7) ^ lds_swz(B_INS % 2 == 0 ? 8 * p + lrow : r);
      vb[p] = (int)(((int64_t)r * ldb + 8 * ch) * 2);
    }
  }
  const int step_a = (int)(16 * lda * 2), step_b = (int)(16 * ldb * 2);
  auto issue = [&](uint4* as, uint4* bs, int k0) {
#pragma unroll
    for (int j = 0; j < A_INS; ++j) {
      int off;
      if constexpr (A_INS % 2 == 0) off = vadd_sgpr(va[j & 1], (j >> 1) * step_a + k0 * 2);
      else off = vadd_sgpr(va[j], k0 * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void_t*)(as + (wave * A_INS + j) * 64), 16,
                                               off, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < B_INS; ++j) {
      int off;
      if constexpr (B_INS % 2 == 0) off = vadd_sgpr(vb[j & 1], (j >> 1) * step_b + k0 * 2);
      else off = vadd_sgpr(vb[j], k0 * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void_t*)(bs + (wave * B_INS + j) * 64), 16,
                                               off, 0, 0, 0);
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  constexpr int STAGE = (BM + BN) * 8;
  // k-stages of this workgroup: all of them, or split slice blockIdx.y of gridDim.y
  const int KT_all = K / GEMM_BK;
  const int kt0 = (int)((int64_t)KT_all * blockIdx.y / gridDim.y);
  const int KT = (int)((int64_t)KT_all * (blockIdx.y + 1) / gridDim.y);
  issue(lds, lds + BM * 8, kt0 * GEMM_BK);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  for (int kt = kt0; kt < KT; ++kt) {
    uint4* cur = lds + ((kt - kt0) & 1) * STAGE;
    uint4* nxt = lds + ((kt - kt0 + 1) & 1) * STAGE;
    // prefetch stage kt + 1 into the other buffer (released by the previous barrier)
    if (kt + 1 < KT) issue(nxt, nxt + BM * 8, (kt + 1) * GEMM_BK);
    mma_stage<BM, BN, TM, TN, FM, FN>(cur, cur + BM * 8, wm, wn, lane, acc);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }

  // Epilogue through LDS (the stage buffers are free after the last barrier):
  // each wave parks one 32-row slice of its tile as fp32, then every lane
  // handles 8 consecutive columns with 16-byte loads (bias, gate, residual) and
  // a 16-byte store, so each 8 lanes write one contiguous 128-byte row run.
  // A lane's column run is the same in every row it handles, so its bias and
  // gate are loaded once, and each slice's residual rows are requested one
  // slice ahead (one exposed memory latency per tile, not one per slice).
  constexpr int EP_LD = TN + 4;                       // fp32 row pitch of the staging slice
  constexpr int CPR = TN / 8;                         // 8-column runs per slice row
  constexpr int EP_IT = (32 * CPR + 63) / 64;         // runs per lane and slice
  static_assert((32 * CPR) % 64 == 0, "every lane handles whole runs");
  static_assert(EPI != EPI_BIAS_QKPOST || TN == 64, "a wave's columns must be one head");
  static_assert(NW * 32 * EP_LD * 4 <= (int)sizeof(lds), "epilogue staging exceeds LDS");
  float* stage = reinterpret_cast<float*>(lds) + wave * 32 * EP_LD;
  const int col0 = n0 + wn * TN;
  const int cl = (lane % CPR) * 8, col = col0 + cl;  // 64 is a multiple of CPR
  const bool col_ok = col < N;
  uint32_t bb[4] = {0u, 0u, 0u, 0u};
  float gg[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  uint4 res[2][EP_IT];                                // residual runs of slices i and i + 1
  auto load_res = [&](int i, uint4 (&r)[EP_IT]) {
#pragma unroll
    for (int it = 0; it < EP_IT; ++it) {
      const int row = m0 + wm * TM + i * 32 + (lane + 64 * it) / CPR;
      r[it] = (row < M && col_ok) ? *reinterpret_cast<const uint4*>(C + (int64_t)row * ldc + col)
                                  : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  if constexpr (EPI != EPI_PARTIAL && EPI != EPI_BIAS_QKPOST) {
    if (col_ok) {
      const uint4 bw = *reinterpret_cast<const uint4*>(bias + col);
      bb[0] = bw.x; bb[1] = bw.y; bb[2] = bw.z; bb[3] = bw.w;
      if constexpr (EPI == EPI_BIAS_GATED_RESIDUAL) {
        const float4 g0 = *reinterpret_cast<const float4*>(gate + col);
        const float4 g1 = *reinterpret_cast<const float4*>(gate + col + 4);
        gg[0] = g0.x; gg[1] = g0.y; gg[2] = g0.z; gg[3] = g0.w;
        gg[4] = g1.x; gg[5] = g1.y; gg[6] = g1.z; gg[7] = g1.w;
      }
    }
    if constexpr (EPI == EPI_BIAS_GATED_RESIDUAL) load_res(0, res[0]);
  }
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    // the next slice's residual rows are requested before this slice is parked
    if constexpr (EPI == EPI_BIAS_GATED_RESIDUAL)
      if (i + 1 < FM) load_res(i + 1, res[(i + 1) & 1]);
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stage[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * EP_LD + j * 32 + (lane & 31)] =
            acc[i][j][r];
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_s_waitcnt(0xc07f);                 // lgkmcnt(0): slice visible to the wave
    __builtin_amdgcn_wave_barrier();
    const int row0 = m0 + wm * TM + i * 32;
#pragma unroll
    for (int it = 0; it < EP_IT; ++it) {
      const int rl = (lane + 64 * it) / CPR;
      const int row = row0 + rl;
      if constexpr (EPI == EPI_BIAS_QKPOST) {
        qkpost_store(stage + rl * EP_LD + cl, bias, C, ldc, row, col, col0, M, N, qp);
        continue;
      }
      if (EPI == EPI_PARTIAL && row < M && col_ok) {
        // fp32 partial sums of this K slice: part[slice][M][N]
        float* q = part + ((int64_t)blockIdx.y * M + row) * N + col;
        reinterpret_cast<float4*>(q)[0] = *reinterpret_cast<const float4*>(stage + rl * EP_LD + cl);
        reinterpret_cast<float4*>(q)[1] = *reinterpret_cast<const float4*>(stage + rl * EP_LD + cl + 4);
      } else if (EPI != EPI_PARTIAL && row < M && col_ok) {
        const float4 v0 = *reinterpret_cast<const float4*>(stage + rl * EP_LD + cl);
        const float4 v1 = *reinterpret_cast<const float4*>(stage + rl * EP_LD + cl + 4);
        const float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
        uint32_t rr[4] = {0u, 0u, 0u, 0u};
        if constexpr (EPI == EPI_BIAS_GATED_RESIDUAL) {
          const uint4 rw = res[i & 1][it];
          rr[0] = rw.x; rr[1] = rw.y; rr[2] = rw.z; rr[3] = rw.w;
        }
        uint32_t out[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float b0 = __uint_as_float(bb[e] << 16), b1 = __uint_as_float(bb[e] & 0xFFFF0000u);
          const float x0 = __uint_as_float(rr[e] << 16), x1 = __uint_as_float(rr[e] & 0xFFFF0000u);
          out[e] = pack_bf16x2(epi_value<EPI>(v[2 * e], b0, gg[2 * e], x0),
                               epi_value<EPI>(v[2 * e + 1], b1, gg[2 * e + 1], x1));
        }
        bf16_t* dst = C + (int64_t)row * ldc + col;
        if constexpr (EPI == EPI_BIAS_GATED_RESIDUAL)
          if (smap != nullptr) dst = Cs + (int64_t)smap[row] * ldc + col;
        *reinterpret_cast<uint4*>(dst) = make_uint4(out[0], out[1], out[2], out[3]);
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// Sum of the split-K partials and the epilogue: one thread per 8 columns of
// a row (16-byte bias / residual loads and stores, 32-byte partial loads).
template <int ROLE, int EPI>
__global__ void __launch_bounds__(256)
splitk_epilogue(const float* __restrict__ part, int splits, int M, int N,
                const bf16_t* __restrict__ bias, const float* __restrict__ gate, bf16_t* C,
                int64_t ldc, bf16_t* Cs, const int32_t* __restrict__ smap) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int cpr = N / 8;
  if (id >= (int64_t)M * cpr) return;
  const int row = (int)(id / cpr), col = (int)(id % cpr) * 8;
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int z = 0; z < splits; ++z) {
    const float* q = part + ((int64_t)z * M + row) * N + col;
    const float4 a = reinterpret_cast<const float4*>(q)[0], b = reinterpret_cast<const float4*>(q)[1];
    v[0] += a.x; v[1] += a.y; v[2] += a.z; v[3] += a.w;
    v[4] += b.x; v[5] += b.y; v[6] += b.z; v[7] += b.w;
  }
  const uint4 bw = *reinterpret_cast<const uint4*>(bias + col);
  const uint32_t bb[4] = {bw.x, bw.y, bw.z, bw.w};
  bf16_t* p = C + (int64_t)row * ldc + col;
  uint32_t rr[4] = {0u, 0u, 0u, 0u};
  float gg[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (EPI == EPI_BIAS_GATED_RESIDUAL) {
    const uint4 rw = *reinterpret_cast<const uint4*>(p);
    rr[0] = rw.x; rr[1] = rw.y; rr[2] = rw.z; rr[3] = rw.w;
    const float4 g0 = *reinterpret_cast<const float4*>(gate + col);
    const float4 g1 = *reinterpret_cast<const float4*>(gate + col + 4);
    gg[0] = g0.x; gg[1] = g0.y; gg[2] = g0.z; gg[3] = g0.w;
    gg[4] = g1.x; gg[5] = g1.y; gg[6] = g1.z; gg[7] = g1.w;
  }
  uint32_t out[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float b0 = __uint_as_float(bb[e] << 16), b1 = __uint_as_float(bb[e] & 0xFFFF0000u);
    const float x0 = __uint_as_float(rr[e] << 16), x1 = __uint_as_float(rr[e] & 0xFFFF0000u);
    out[e] = pack_bf16x2(epi_value<EPI>(v[2 * e], b0, gg[2 * e], x0),
                         epi_value<EPI>(v[2 * e + 1], b1, gg[2 * e + 1], x1));
  }
  bf16_t* dst = p;
  if (EPI == EPI_BIAS_GATED_RESIDUAL && smap != nullptr) dst = Cs + (int64_t)smap[row] * ldc + col;
  *reinterpret_cast<uint4*>(dst) = make_uint4(out[0], out[1], out[2], out[3]);
}

// ---------------------------------------------------------------------------
// fp32 path (plain LDS-tiled FMA; used by the fp32 workload)
// ---------------------------------------------------------------------------
template <int EPI>
__global__ void __launch_bounds__(256)
gemm_f32_nt(const float* __restrict__ A, int64_t lda, const float* __restrict__ B, int64_t ldb,
            const float* __restrict__ bias, const float* __restrict__ gate, float* C,
            int64_t ldc, int M, int N, int K) {
  __shared__ float As[16][65];
  __shared__ float Bs[16][65];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int i = threadIdx.x; i < 64 * 16; i += 256) {
      const int r = i >> 4, kk = i & 15;
      const int gm = m0 + r, gn = n0 + r, gk = k0 + kk;
      As[kk][r] = (gm < M && gk < K) ? A[(int64_t)gm * lda + gk] : 0.0f;
      Bs[kk][r] = (gn < N && gk < K) ? B[(int64_t)gn * ldb + gk] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty + 16 * i;
    if (row >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx + 16 * j;
      if (col >= N) continue;
      float* p = C + (int64_t)row * ldc + col;
      const float resid = (EPI == EPI_BIAS_GATED_RESIDUAL) ? *p : 0.0f;
      const float gv = (EPI == EPI_BIAS_GATED_RESIDUAL) ? gate[col] : 0.0f;
      *p = epi_value<EPI>(acc[i][j], bias[col], gv, resid);
    }
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
template <int ROLE, int BM, int BN, int WM, int WN, int EPI>
static hipError_t run_bf16(const void* A, int64_t lda, const void* B, int64_t ldb,
                           const void* bias, const float* gate, void* C, int64_t ldc, int M,
                           int N, int K, int splits, float* part, hipStream_t st,
                           const QkPost& qp = QkPost{}, void* Cs = nullptr,
                           const int32_t* smap = nullptr) {
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  if (splits <= 1) {
    hipLaunchKernelGGL((gemm_bf16_nt<ROLE, BM, BN, WM, WN, EPI>), dim3(tiles_m * tiles_n),
                       dim3(WM * WN * 64), 0, st, (const bf16_t*)A, lda, (const bf16_t*)B, ldb,
                       (const bf16_t*)bias, gate, (bf16_t*)C, ldc, M, N, K, tiles_m, tiles_n,
                       (float*)nullptr, qp, ScoreArgs{}, 0, (bf16_t*)Cs, smap);
    return hipGetLastError();
  }
  if constexpr (EPI == EPI_BIAS_QKPOST) {
    return hipErrorNotSupported;             // no split-K store with the QK post-processing
  } else {
    hipLaunchKernelGGL((gemm_bf16_nt<ROLE, BM, BN, WM, WN, EPI_PARTIAL>), dim3(tiles_m * tiles_n, splits),
                       dim3(WM * WN * 64), 0, st, (const bf16_t*)A, lda, (const bf16_t*)B, ldb,
                       (const bf16_t*)bias, gate, (bf16_t*)C, ldc, M, N, K, tiles_m, tiles_n, part,
                       QkPost{}, ScoreArgs{}, 0, (bf16_t*)nullptr, (const int32_t*)nullptr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t n = (int64_t)M * (N / 8);
    hipLaunchKernelGGL((splitk_epilogue<ROLE, EPI>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                       part, splits, M, N, (const bf16_t*)bias, gate, (bf16_t*)C, ldc,
                       (bf16_t*)Cs, smap);
    return hipGetLastError();
  }
}

// Tile and K-split choice: modelled time = rounds * (per-CU MFMA work of one
// round / tile efficiency) + (split > 1) the partial-sum pass over HBM.  A
// round places `per_cu` workgroups on each of the 256 CUs (LDS-limited).  The
// 256x256 and 192x256 kernels fit one workgroup per CU and run in whole
// rounds; two 128x128 workgroups share a CU and start as soon as a slot
// frees, so their rounds count in halves once a grid spills past one slot per
// CU.  The efficiencies are the per-CU MFMA rates of the kernels measured on
// the block shapes of the d = 1536 and d = 2048 workloads, relative to the
// 256x256 kernel (whose rate, about 40% of the per-CU peak, is the base; the
// 192x256 tile, 8 waves of 96 x 64, runs at 0.85-0.92 of it and takes 0.85,
// which makes it the choice where its 3/4-size tiles fill whole rounds: the
// packed MLP up projection at 3,472 rows, the out and down projections at
// 17,472 rows); the pass moves splits * M * N fp32 partials plus the bf16
// output (and residual) at about 4 TB/s.  The 192x128 tile (8 waves of
// 96 x 32, two workgroups per CU) enters at 0.83, which selects it where
// half-rounds of its small tiles fill the CUs much better than the others:
// the packed out projection at 3,472 rows and the d = 1024 projections at
// 1,312 rows (measured 2-9% faster there).  At 0.84 it would also take the
// packed down projection at 3,472 rows without a K split, measured 11%
// slower than the three K slices.  (A 256x128 tile measured at 0.72 of the
// base rate never won at any block shape from d = 256 to 4096 and was
// dropped.)
struct GemmPlan { int tile, splits; };
constexpr int GEMM_TILES = 4;
static const int TILE_BM[GEMM_TILES] = {256, 128, 192, 192};
static const int TILE_BN[GEMM_TILES] = {256, 128, 256, 128};
static const int TILE_PER_CU[GEMM_TILES] = {1, 2, 1, 2};
// wide_only: only tiles whose waves span 64 columns (the QK post-processing
// store needs one head per wave)
static GemmPlan choose_gemm(int64_t M, int64_t N, int64_t K, int64_t ws_floats,
                            bool wide_only = false) {
  const double eff[GEMM_TILES] = {1.0, 0.80, 0.85, 0.83};
  const int split_opts[6] = {1, 2, 3, 4, 6, 8};
  const int64_t kt = K / GEMM_BK;
  const double cu_flops = 2.5e15 / 256.0 * 0.40;        // sustained MFMA rate per CU
  GemmPlan best{0, 1};
  double best_t = 1e30;
  for (int i = 0; i < GEMM_TILES; ++i) {
    if (wide_only && i == 3) continue;
    const int bm = TILE_BM[i], bn = TILE_BN[i], per_cu = TILE_PER_CU[i];
    const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
    for (int s : split_opts) {
      if (s > 1 && (kt / s < 4 || (int64_t)s * M * N > ws_floats)) continue;
      const int64_t wgs = tiles * s;
      double rounds;
      if (per_cu == 1) {
        rounds = (double)((wgs + 255) / 256);
      } else {
        // whole half-rounds while one slot per CU is not yet filled
        rounds = std::max((double)wgs / (256.0 * per_cu),
                          (double)((wgs + 255) / 256) / per_cu);
      }
      const double k_slice = (double)((kt + s - 1) / s) * GEMM_BK;
      double t = rounds * 2.0 * bm * bn * per_cu * k_slice /
                 (cu_flops * eff[i]);
      if (s > 1) t += ((double)s * M * N * 4.0 + 4.0 * M * N) / 4.0e12 + 3e-6;
      if (t < best_t) { best_t = t; best = {i, s}; }
    }
  }
  return best;
}

template <int ROLE, int EPI>
static hipError_t dispatch_bf16(const void* A, int64_t lda, const void* B, int64_t ldb,
                                const void* bias, const float* gate, void* C, int64_t ldc,
                                int M, int N, int K, float* ws, int64_t ws_floats,
                                hipStream_t st, void* Cs = nullptr,
                                const int32_t* smap = nullptr) {
  const GemmPlan p = choose_gemm(M, N, K, ws ? ws_floats : 0);
  if (p.tile == 0)
    return run_bf16<ROLE, 256, 256, 2, 4, EPI>(A, lda, B, ldb, bias, gate, C, ldc, M, N, K, p.splits, ws, st, QkPost{}, Cs, smap);
  if (p.tile == 2)
    return run_bf16<ROLE, 192, 256, 2, 4, EPI>(A, lda, B, ldb, bias, gate, C, ldc, M, N, K, p.splits, ws, st, QkPost{}, Cs, smap);
  if (p.tile == 3)
    return run_bf16<ROLE, 192, 128, 2, 4, EPI>(A, lda, B, ldb, bias, gate, C, ldc, M, N, K, p.splits, ws, st, QkPost{}, Cs, smap);
  return run_bf16<ROLE, 128, 128, 2, 2, EPI>(A, lda, B, ldb, bias, gate, C, ldc, M, N, K, p.splits, ws, st, QkPost{}, Cs, smap);
}

// The MLP up projection with one layer's scoring in the tail of its grid:
// the scoring workgroups are dispatched after every tile, i.e. into the last
// round, on the CUs its tiles leave idle there (at least 16 of them, or the
// caller scores on its side stream instead).
static int scored_idle_slots(const GemmPlan& p, int64_t M, int64_t N) {
  const int bm = TILE_BM[p.tile], bn = TILE_BN[p.tile];
  if (p.splits != 1) return 0;
  const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  const int64_t slots = 256 * TILE_PER_CU[p.tile];
  const int64_t idle = (slots - tiles % slots) % slots;
  return idle >= 16 ? (int)idle : 0;
}

int gemm_up_scored_slots(int64_t M, int64_t N, int64_t K, int64_t ws_floats) {
  if (M <= 0) return 0;
  return scored_idle_slots(choose_gemm(M, N, K, ws_floats), M, N);
}

template <int BM, int BN, int WM, int WN>
static hipError_t run_up_scored(const void* A, int64_t lda, const void* B, int64_t ldb,
                                const void* bias, void* C, int64_t ldc, int M, int N, int K,
                                const ScoreArgs& sa, int n_sw, hipStream_t st) {
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int ktiles = (sa.n_s + 15) / 16;
  const int n_units = (sa.n_layers < 1 ? 1 : sa.n_layers) * sa.B * sa.F * ktiles;
  constexpr int G = WM * WN / 4;
  n_sw = std::min(n_sw, (n_units + G - 1) / G);
  hipLaunchKernelGGL((gemm_bf16_nt<ROLE_UP, BM, BN, WM, WN, EPI_BIAS_GELU, true>),
                     dim3(tiles_m * tiles_n + n_sw), dim3(WM * WN * 64), 0, st, (const bf16_t*)A,
                     lda, (const bf16_t*)B, ldb, (const bf16_t*)bias, (const float*)nullptr,
                     (bf16_t*)C, ldc, M, N, K, tiles_m, tiles_n, (float*)nullptr, QkPost{}, sa,
                     n_units, (bf16_t*)nullptr, (const int32_t*)nullptr);
  return hipGetLastError();
}

hipError_t launch_gemm_up_scored(const void* A, int64_t lda, const void* B, int64_t ldb,
                                 const void* bias, void* C, int64_t ldc, int64_t M, int64_t N,
                                 int64_t K, const ScoreArgs& sa, hipStream_t st,
                                 int64_t ws_floats) {
  if (M <= 0) return hipSuccess;
  const GemmPlan p = choose_gemm(M, N, K, ws_floats);
  const int n_sw = scored_idle_slots(p, M, N);
  if (n_sw == 0) return hipErrorNotSupported;
  const int m = (int)M, n = (int)N, k = (int)K;
  if (p.tile == 0) return run_up_scored<256, 256, 2, 4>(A, lda, B, ldb, bias, C, ldc, m, n, k, sa, n_sw, st);
  if (p.tile == 2) return run_up_scored<192, 256, 2, 4>(A, lda, B, ldb, bias, C, ldc, m, n, k, sa, n_sw, st);
  if (p.tile == 3) return run_up_scored<192, 128, 2, 4>(A, lda, B, ldb, bias, C, ldc, m, n, k, sa, n_sw, st);
  return run_up_scored<128, 128, 2, 2>(A, lda, B, ldb, bias, C, ldc, m, n, k, sa, n_sw, st);
}

template <int EPI>
static hipError_t run_f32(const void* A, int64_t lda, const void* B, int64_t ldb,
                          const void* bias, const float* gate, void* C, int64_t ldc, int M,
                          int N, int K, hipStream_t st) {
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  hipLaunchKernelGGL(gemm_f32_nt<EPI>, grid, dim3(256), 0, st, (const float*)A, lda,
                     (const float*)B, ldb, (const float*)bias, gate, (float*)C, ldc, M, N, K);
  return hipGetLastError();
}

hipError_t launch_gemm(int dtype, int role, const void* A, int64_t lda, const void* B,
                       int64_t ldb, const void* bias, const float* gate, void* C,
                       int64_t ldc, int64_t M, int64_t N, int64_t K, hipStream_t st,
                       float* ws, int64_t ws_floats, void* Cs, const int32_t* smap) {
  if (M <= 0) return hipSuccess;
  const int m = (int)M, n = (int)N, k = (int)K;
  if (smap != nullptr && (dtype != 1 || (role != ROLE_OUT && role != ROLE_DOWN) || Cs == nullptr))
    return hipErrorNotSupported;             // row scatter: bf16 gated-residual stores only
  if (dtype == 1) {
    switch (role) {
      case ROLE_QKV: return dispatch_bf16<ROLE_QKV, EPI_BIAS>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, ws, ws_floats, st);
      case ROLE_UP: return dispatch_bf16<ROLE_UP, EPI_BIAS_GELU>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, ws, ws_floats, st);
      case ROLE_OUT: return dispatch_bf16<ROLE_OUT, EPI_BIAS_GATED_RESIDUAL>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, ws, ws_floats, st, Cs, smap);
      case ROLE_DOWN: return dispatch_bf16<ROLE_DOWN, EPI_BIAS_GATED_RESIDUAL>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, ws, ws_floats, st, Cs, smap);
      default: return hipErrorInvalidValue;
    }
  }
  switch (role) {
    case ROLE_QKV: return run_f32<EPI_BIAS>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, st);
    case ROLE_UP: return run_f32<EPI_BIAS_GELU>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, st);
    case ROLE_OUT:
    case ROLE_DOWN: return run_f32<EPI_BIAS_GATED_RESIDUAL>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_qkv(int dtype, const void* A, int64_t lda, const void* B, int64_t ldb,
                           const void* bias, void* C, int64_t ldc, int64_t M, int64_t N,
                           int64_t K, const QkPost& qp, hipStream_t st, float* ws,
                           int64_t ws_floats) {
  if (M <= 0) return hipSuccess;
  const bool post = qp.qk_norm || qp.tab != nullptr;
  if (dtype == 1 && post) {
    const GemmPlan p = choose_gemm(M, N, K, ws ? ws_floats : 0, true);
    if (p.splits <= 1) {
      const int m = (int)M, n = (int)N, k = (int)K;
      if (p.tile == 0)
        return run_bf16<ROLE_QKV, 256, 256, 2, 4, EPI_BIAS_QKPOST>(A, lda, B, ldb, bias, nullptr, C, ldc, m, n, k, 1, nullptr, st, qp);
      if (p.tile == 2)
        return run_bf16<ROLE_QKV, 192, 256, 2, 4, EPI_BIAS_QKPOST>(A, lda, B, ldb, bias, nullptr, C, ldc, m, n, k, 1, nullptr, st, qp);
      return run_bf16<ROLE_QKV, 128, 128, 2, 2, EPI_BIAS_QKPOST>(A, lda, B, ldb, bias, nullptr, C, ldc, m, n, k, 1, nullptr, st, qp);
    }
  }
  const hipError_t e = launch_gemm(dtype, ROLE_QKV, A, lda, B, ldb, bias, nullptr, C, ldc, M, N, K,
                                   st, ws, ws_floats);
  if (e != hipSuccess || !post) return e;
  return launch_qk_post(dtype, C, M, qp.d, qp.pos_mode, qp.gather, qp.cu, qp.n_seqs, qp.l_full,
                        qp.tab, qp.n_pos, qp.qk_norm, st);
}

}  // namespace swam
