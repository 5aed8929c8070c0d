// Softmax attention of the DiT block over the keys of each (dense or packed)
// sequence, writing O and the natural-log normaliser lambda of every query
// row and head (the normaliser the scorer reuses).
//
// bf16 path, one head per workgroup, 4 or 8 waves x 32 query rows:
//   S^T = K Q^T with 32x32x16 MFMA: K (64-key tile, LDS) is the A operand and
//   the wave's 32 query rows are the B operand held in registers, so the C
//   layout gives each lane ONE query (lane & 31) and 16 of every 32 keys;
//   the other 16 sit in lane ^ 32.  Row max / sum are in-lane plus one swap.
//   O^T = V^T P^T: P^T straight from the S^T accumulators is the B operand
//   (no shuffle); the V^T operand comes from transposed LDS reads of the
//   row-major V tile.  K and V tiles are DMA'd global -> LDS (no register
//   staging), double-buffered.  Online softmax in the log2 domain with the
//   1/8 scale folded into one FMA, tail-only masking and lazy rescaling.
// fp32 path: one wave per (query row, head), online softmax with shuffles.
#include "common.h"

#include <type_traits>

namespace swam {

constexpr int ATT_BK = 64;      // keys per tile

template <int BQ>
__device__ __forceinline__ bool find_tile(const int32_t* cu, int n_seqs, int n_rows, int t,
                                          int& s0, int& s1, int& q0) {
  for (int b = 0; b < n_seqs; ++b) {
    const int e = min(max(cu[b + 1], 0), n_rows);
    const int a = min(max(cu[b], 0), e);
    const int nt = (e - a + BQ - 1) / BQ;
    if (t < nt) { s0 = a; s1 = e; q0 = a + t * BQ; return true; }
    t -= nt;
  }
  return false;
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// NW waves x 32 query rows per workgroup; WPE = minimum waves per SIMD the
// register allocation must allow (4 caps it at 128 VGPRs); SUB 64-key tiles
// share one LDS stage, i.e. one barrier and one DMA wait.
template <int NW, int WPE, int SUB>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(WPE, 8)))
attn_fwd_bf16(const bf16_t* __restrict__ qkv, bf16_t* __restrict__ out, float* __restrict__ lse,
     const int32_t* __restrict__ cu, int n_seqs, int n_heads, int n_rows) {
  constexpr int S = 2;                           // LDS stages (K and V tiles)
  constexpr int SK = SUB * ATT_BK;               // keys per stage: SUB tiles per barrier
  __shared__ uint4 Ks[S][SK * 8];                 // [key][8 chunks], chunk ^ lds_swz(key)
  __shared__ uint4 Vs[S][SK * 8];
  const int nwg = gridDim.x, pid = blockIdx.x;
  const int xcd = pid & 7, per = nwg >> 3, rem = nwg & 7;
  const int id = xcd * per + min(xcd, rem) + (pid >> 3);
  const int slots = nwg / n_heads;
  const int h = id / slots;
  int s0, s1, q0;
  constexpr int BQ = 32 * NW;
  if (!find_tile<BQ>(cu, n_seqs, n_rows, id - h * slots, s0, s1, q0)) return;
  const int d = n_heads * 64;
  const int64_t ld = 3 * (int64_t)d;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5;
  const int qrow = q0 + wave * 32 + (lane & 31);
  const bool qvalid = qrow < s1;
  bf16x8 qf[4];
  {
    const bf16_t* qp = qkv + (int64_t)min(qrow, s1 - 1) * ld + h * 64;
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = __builtin_bit_cast(bf16x8, *(const uint4*)(qp + 8 * (2 * s + g)));
  }
  // K and V tiles go global -> LDS directly, row-major with the chunk swizzle
  // applied on the global side: each instruction moves an 8-row slab (1 KB),
  // lane i landing in row i >> 3, physical chunk i & 7.
  // (element offsets stay below 2^31: the launcher checks n_rows * 3d)
  const int lrow = lane >> 3;
  const int ld32 = 3 * d;
  const bf16_t* kbase = qkv + d + h * 64;
  const bf16_t* vbase = qkv + 2 * d + h * 64;
  constexpr int SLABS = SK / 8 / NW;             // 8-row slabs per wave and stage
  static_assert(SLABS * 8 * NW == SK, "every wave stages whole 8-row slabs");
  int lofs[SLABS];
#pragma unroll
  for (int j = 0; j < SLABS; ++j) {
    const int r0 = (SK / NW) * wave + 8 * j;
    lofs[j] = 8 * ((lane & 7) ^ lds_swz((r0 & 8) + lrow));
  }
  auto issue = [&](int buf, int kb) {
#pragma unroll
    for (int j = 0; j < SLABS; ++j) {
      const int r0 = (SK / NW) * wave + 8 * j;
      const int e = min(kb + r0 + lrow, s1 - 1) * ld32 + lofs[j];
      __builtin_amdgcn_global_load_lds((glb_void_t*)(kbase + e), (lds_void_t*)(&Ks[buf][r0 * 8]), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((glb_void_t*)(vbase + e), (lds_void_t*)(&Vs[buf][r0 * 8]), 16, 0, 0);
    }
  };
  // PV operand (V^T fragment) from transposed LDS reads: within each 16-lane
  // group, lane a addresses V[key0 + (a >> 2)][hd0 + 4 (a & 3)] and lane i
  // receives V[key0 .. key0+3][hd0 + i], i.e. four consecutive keys of one
  // head-dim column (the k order the P^T accumulators provide).
  const int a16 = lane & 15, G = lane >> 4;
  // loop-invariant part of those addresses: key 32t + 16u + rlo (+ 8 for the
  // second read), column hd = 32ht + 16 (G & 1) + 4 (a16 & 3); the swizzle
  // sees only key bits 1..3, i.e. rlo and the +8
  const int rlo = 4 * g + (a16 >> 2);
  int vofs[2][2];
#pragma unroll
  for (int ht = 0; ht < 2; ++ht)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int r = rlo + 8 * hf;
      const int hd = 32 * ht + 16 * (G & 1) + 4 * (a16 & 3);
      vofs[ht][hf] = r * 64 + 8 * ((hd >> 3) ^ lds_swz(r)) + (hd & 7);
    }
  // K fragment (logical chunk 2 s + g of key lane & 31) offsets in a tile
  int kofs[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
    kofs[s] = (lane & 31) * 8 + ((2 * s + g) ^ lds_swz(lane & 31));
  f32x16 o[2];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
  float m_run = -1e30f, l_run = 0.0f;
  const float sc = 1.4426950408889634f * 0.125f;
  const int nkt = (s1 - s0 + SK - 1) / SK;       // stages
#pragma unroll
  for (int p = 0; p < S - 1; ++p)
    if (p < nkt) issue(p, s0 + p * SK);
  // one 64-key tile of stage buffer `cur` at key offset sub * 64; full tiles
  // carry no masking code, the ragged last one runs a copy with the key mask
  auto tile = [&](int cur, int sub, int kb, auto masked) {
    const uint4* Kt = &Ks[cur][sub * ATT_BK * 8];
    auto scores = [&](f32x16 (&st)[2]) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int r = 0; r < 16; ++r) st[t][r] = 0.0f;
        // keys 32 t + (lane & 31): the swizzle sees the same row bits for both
        // halves, so the half is a constant offset of 32 rows
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          bf16x8 kf = __builtin_bit_cast(bf16x8, Kt[kofs[s] + t * 32 * 8]);
          st[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], st[t], 0, 0, 0);
        }
      }
      if constexpr (decltype(masked)::value) {
        const int nvalid = s1 - kb;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = 32 * t + 8 * (r >> 2) + 4 * g + (r & 3);
            if (key >= nvalid) st[t][r] = -INFINITY;
          }
      }
    };
    // probabilities against the running max.  Their row sum bounds every one
    // of them, so a sum above 2^8 is the only case in which the running max
    // must move (lazy rescaling: each p stays <= 2^8 otherwise); the scores
    // are then recomputed (K is still staged) and the tile is redone against
    // the new max.  The first tile of a row always takes that path (the
    // running max starts at -1e30).
    bf16x8 pf[2][2];
    float psum0, psum1;
    auto probs = [&](const f32x16 (&st)[2]) {
      psum0 = 0.0f; psum1 = 0.0f;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int mm = 0; mm < 8; mm += 2) {
            const float p0 = __builtin_amdgcn_exp2f(fmaf(st[t][8 * u + mm], sc, -m_run));
            const float p1 = __builtin_amdgcn_exp2f(fmaf(st[t][8 * u + mm + 1], sc, -m_run));
            // row sums from the fp32 probabilities (the exported normaliser)
            psum0 += p0; psum1 += p1;
            pf[t][u][mm] = (__bf16)p0; pf[t][u][mm + 1] = (__bf16)p1;
          }
    };
    {
      f32x16 st[2];
      scores(st);
      probs(st);
    }
    if (__any(!(psum0 + psum1 <= 256.0f))) {
      // re-read K from LDS rather than keeping the first pass's fragments live
      asm volatile("" ::: "memory");
      f32x16 st[2];
      scores(st);
      float mx = st[0][0];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, st[t][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx * sc);
      const float corr = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= corr;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] *= corr;
      probs(st);
    }
    l_run += psum0 + psum1;
    const unsigned short* vs = reinterpret_cast<const unsigned short*>(&Vs[cur][sub * ATT_BK * 8]);
#pragma unroll
    for (int ht = 0; ht < 2; ++ht) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int e1 = vofs[ht][0] + (32 * t + 16 * u) * 64;
          const int e2 = vofs[ht][1] + (32 * t + 16 * u) * 64;
          const v4i16 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(vs + e1));
          const v4i16 x2 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(vs + e2));
          const uint2 w1 = __builtin_bit_cast(uint2, x1), w2 = __builtin_bit_cast(uint2, x2);
          const bf16x8 vf = __builtin_bit_cast(bf16x8, make_uint4(w1.x, w1.y, w2.x, w2.y));
          o[ht] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[t][u], o[ht], 0, 0, 0);
        }
    }
  };
  auto stage = [&](int kt, auto masked) {
    const int cur = kt % S;
    const int kb = s0 + kt * SK;
    // stage kt has landed (own DMA done, then everyone's via the barrier); the
    // barrier also releases the stage the next prefetch overwrites
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (kt + S - 1 < nkt) issue((kt + S - 1) % S, kb + (S - 1) * SK);
#pragma unroll
    for (int sub = 0; sub < SUB; ++sub) {
      const int kbs = kb + sub * ATT_BK;
      if constexpr (decltype(masked)::value) {
        if (s1 > kbs) tile(cur, sub, kbs, std::true_type{});   // a no-op mask when full
      } else {
        tile(cur, sub, kbs, std::false_type{});
      }
    }
  };
  const int nfull = (s1 - s0) / SK;
  for (int kt = 0; kt < nfull; ++kt) stage(kt, std::false_type{});
  if (nfull < nkt) stage(nfull, std::true_type{});
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!qvalid) return;
  const float inv = 1.0f / l_tot;
  bf16_t* op = out + (int64_t)qrow * d + h * 64;
#pragma unroll
  for (int ht = 0; ht < 2; ++ht)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int hd = 32 * ht + 8 * q4 + 4 * g;
      uint2 w;
      w.x = pack_bf16x2(o[ht][4 * q4 + 0] * inv, o[ht][4 * q4 + 1] * inv);
      w.y = pack_bf16x2(o[ht][4 * q4 + 2] * inv, o[ht][4 * q4 + 3] * inv);
      *(uint2*)(op + hd) = w;
    }
  if (lse != nullptr && g == 0)
    lse[(int64_t)qrow * n_heads + h] = (m_run + log2f(l_tot)) * 0.6931471805599453f;
}

// fp32: one wave per (query row, head); lane = head-dim element.
__global__ void __launch_bounds__(64)
attn_fwd_f32(const float* __restrict__ qkv, float* __restrict__ out, float* __restrict__ lse,
             const int32_t* __restrict__ cu, int n_seqs, int n_heads, int64_t n_rows) {
  const int64_t row = blockIdx.x;
  const int h = blockIdx.y, lane = threadIdx.x;
  if (row >= n_rows) return;
  int s0 = 0, s1 = 0;
  for (int b = 0; b < n_seqs; ++b) {
    const int e = (int)min((int64_t)max(cu[b + 1], 0), n_rows);
    const int a = min(max(cu[b], 0), e);
    if (row >= a && row < e) { s0 = a; s1 = e; }
  }
  if (s1 <= s0) return;
  const int d = n_heads * 64;
  const int64_t ld = 3 * (int64_t)d;
  const float q = qkv[row * ld + h * 64 + lane] * 0.125f;
  float m = -INFINITY, l = 0.0f, acc = 0.0f;
  for (int j = s0; j < s1; ++j) {
    const float x = warp_sum(q * qkv[(int64_t)j * ld + d + h * 64 + lane]);
    const float mn = fmaxf(m, x);
    const float corr = expf(m - mn), p = expf(x - mn);
    l = l * corr + p;
    acc = acc * corr + p * qkv[(int64_t)j * ld + 2 * d + h * 64 + lane];
    m = mn;
  }
  out[row * d + h * 64 + lane] = acc / l;
  if (lse != nullptr && lane == 0) lse[row * n_heads + h] = m + logf(l);
}

hipError_t launch_attention(int dtype, const void* qkv, void* o, float* lse,
                            const int32_t* cu_seqlens, int n_seqs, int64_t n_rows,
                            int n_heads, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  if (dtype == 1) {
    if (n_rows * 3 * (int64_t)n_heads * 64 >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    // 8 waves (256 query rows) share each K/V tile when the grid gives the
    // CUs at least 1.75 such workgroups on average (measured: 3,744 packed
    // rows x 32 heads, 480 workgroups, run 11% faster than with 4 waves;
    // 3,472 x 24, 336 workgroups, 7% slower); otherwise 4 waves, with the
    // 4-waves/SIMD register cap only when enough workgroups exist to use it.
    const int slots8 = (int)((n_rows + 255) / 256) + n_seqs;
    const int slots4 = (int)((n_rows + 127) / 128) + n_seqs;
    const bf16_t* a = (const bf16_t*)qkv;
    bf16_t* ob = (bf16_t*)o;
    const int ni = (int)n_rows;
#define SWAM_ATT(NW_, WPE_, SUB_, SL_)                                                       \
  hipLaunchKernelGGL((attn_fwd_bf16<NW_, WPE_, SUB_>), dim3((SL_) * n_heads), dim3(NW_ * 64), 0, \
                     st, a, ob, lse, cu_seqlens, n_seqs, n_heads, ni)
    // the 8-wave kernel stages 128 keys per barrier (64 KB of LDS, two
    // workgroups per CU); the 4-wave ones keep 64 so four fit on a CU
    if ((int64_t)(slots8 - n_seqs) * n_heads >= 7 * 64)
      SWAM_ATT(8, 4, 2, slots8);
    else if ((int64_t)(slots4 - n_seqs) * n_heads >= 3 * 256)
      SWAM_ATT(4, 4, 1, slots4);
    else
      SWAM_ATT(4, 1, 1, slots4);
#undef SWAM_ATT
  } else {
    hipLaunchKernelGGL(attn_fwd_f32, dim3((unsigned)n_rows, n_heads), dim3(64), 0, st,
                       (const float*)qkv, (float*)o, lse, cu_seqlens, n_seqs, n_heads, n_rows);
  }
  return hipGetLastError();
}

}  // namespace swam
