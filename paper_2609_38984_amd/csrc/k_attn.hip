// Softmax attention of the DiT block over the keys of each (dense or packed)
// sequence, writing O and the natural-log normaliser lambda of every query
// row and head (the normaliser the scorer reuses).
//
// bf16 path, one head per workgroup, 4 waves x 32 query rows:
//   S^T = K Q^T with 32x32x16 MFMA: K (64-key tile, LDS) is the A operand and
//   the wave's 32 query rows are the B operand held in registers, so the C
//   layout gives each lane ONE query (lane & 31) and 16 of every 32 keys;
//   the other 16 sit in lane ^ 32.  Row max / sum are in-lane plus one swap.
//   O^T = V^T P^T: P^T straight from the S^T accumulators is the B operand
//   (no shuffle); V is staged transposed in LDS so the A operand reads are
//   8-byte row reads.  Online softmax in the log2 domain with the 1/8 scale
//   folded into the exponent.  K/V tiles are double-buffered.
// fp32 path: one wave per (query row, head), online softmax with shuffles.
#include "common.h"

namespace swam {

constexpr int ATT_BQ = 128;     // query rows per workgroup
constexpr int ATT_BK = 64;      // keys per tile
constexpr int VT_PITCH = 68;    // V^T row pitch in bf16 (64 keys + 4 pad) = 136 bytes

__device__ __forceinline__ bool find_tile(const int32_t* cu, int n_seqs, int n_rows, int t,
                                          int bq, int& s0, int& s1, int& q0) {
  for (int b = 0; b < n_seqs; ++b) {
    const int e = min(max(cu[b + 1], 0), n_rows);
    const int a = min(max(cu[b], 0), e);
    const int nt = (e - a + bq - 1) / bq;
    if (t < nt) {
      s0 = a; s1 = e; q0 = a + t * bq;
      return true;
    }
    t -= nt;
  }
  return false;
}

// WPE = minimum waves per SIMD the register allocation must allow: 4 caps the
// kernel at 128 VGPRs (no spills), which pays when enough workgroups exist to
// keep 4 waves on every SIMD; otherwise the unconstrained build (3) is used.
template <int WPE>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WPE, 8)))
attn_fwd_bf16(const bf16_t* __restrict__ qkv, bf16_t* __restrict__ out, float* __restrict__ lse,
              const int32_t* __restrict__ cu, int n_seqs, int n_heads, int n_rows) {
  __shared__ uint4 Ks[2][ATT_BK * 8];                 // [key][8 chunks], swizzled
  __shared__ uint32_t Vt[2][64 * VT_PITCH / 2];       // [hd][keys] bf16 pairs
  // XCD-aware order: dispatch deals workgroup ids round-robin over the 8 XCDs;
  // renumber so each XCD walks a contiguous run of (head, query tile) pairs and
  // its L2 holds the K/V of one or two heads at a time.
  const int nwg = gridDim.x, pid = blockIdx.x;
  const int xcd = pid & 7, per = nwg >> 3, rem = nwg & 7;
  const int id = xcd * per + min(xcd, rem) + (pid >> 3);
  const int slots = nwg / n_heads;
  const int h = id / slots;
  int s0, s1, q0;
  if (!find_tile(cu, n_seqs, n_rows, id - h * slots, ATT_BQ, s0, s1, q0)) return;
  const int d = n_heads * 64;
  const int64_t ld = 3 * (int64_t)d;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5;                            // half-wave
  const int qrow = q0 + wave * 32 + (lane & 31);
  const bool qvalid = qrow < s1;

  // Q^T B-operand fragments: query (lane & 31), hd chunk 2s + g
  bf16x8 qf[4];
  {
    const bf16_t* qp = qkv + (int64_t)min(qrow, s1 - 1) * ld + h * 64;
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = __builtin_bit_cast(bf16x8, *(const uint4*)(qp + 8 * (2 * s + g)));
  }

  // K / V staging: thread -> (chunk c, key pair kp)
  const int c = tid & 7, kp = tid >> 3;               // kp 0..31
  const bf16_t* kbase = qkv + d + h * 64 + 8 * c;
  const bf16_t* vbase = qkv + 2 * d + h * 64 + 8 * c;
  uint4 rk0, rk1, rv0, rv1;
#define SWAM_ATT_LOAD(t_)                                                         \
  {                                                                               \
    const int r0_ = s0 + (t_) * ATT_BK + 2 * kp;                                  \
    const int64_t k0_ = min(r0_, s1 - 1), k1_ = min(r0_ + 1, s1 - 1);            \
    rk0 = *(const uint4*)(kbase + k0_ * ld);                                      \
    rk1 = *(const uint4*)(kbase + k1_ * ld);                                      \
    rv0 = *(const uint4*)(vbase + k0_ * ld);                                      \
    rv1 = *(const uint4*)(vbase + k1_ * ld);                                      \
  }
  // K rows swizzled by 16-byte chunk; V transposed: Vt[8c + e][2kp .. 2kp+1], the
  // (key 2kp, key 2kp+1) pair of one head-dim column packed with one byte permute
#define SWAM_ATT_STORE(buf_)                                                      \
  {                                                                               \
    Ks[buf_][(2 * kp) * 8 + (c ^ ((2 * kp) & 7))] = rk0;                          \
    Ks[buf_][(2 * kp + 1) * 8 + (c ^ ((2 * kp + 1) & 7))] = rk1;                  \
    uint32_t* vt_ = &Vt[buf_][(8 * c) * (VT_PITCH / 2) + kp];                      \
    vt_[0 * (VT_PITCH / 2)] = __builtin_amdgcn_perm(rv1.x, rv0.x, 0x05040100u);   \
    vt_[1 * (VT_PITCH / 2)] = __builtin_amdgcn_perm(rv1.x, rv0.x, 0x07060302u);   \
    vt_[2 * (VT_PITCH / 2)] = __builtin_amdgcn_perm(rv1.y, rv0.y, 0x05040100u);   \
    vt_[3 * (VT_PITCH / 2)] = __builtin_amdgcn_perm(rv1.y, rv0.y, 0x07060302u);   \
    vt_[4 * (VT_PITCH / 2)] = __builtin_amdgcn_perm(rv1.z, rv0.z, 0x05040100u);   \
    vt_[5 * (VT_PITCH / 2)] = __builtin_amdgcn_perm(rv1.z, rv0.z, 0x07060302u);   \
    vt_[6 * (VT_PITCH / 2)] = __builtin_amdgcn_perm(rv1.w, rv0.w, 0x05040100u);   \
    vt_[7 * (VT_PITCH / 2)] = __builtin_amdgcn_perm(rv1.w, rv0.w, 0x07060302u);   \
  }

  f32x16 o[2];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
  float m_run = -1e30f, l_run = 0.0f;
  const float sc = 1.4426950408889634f * 0.125f;      // log2(e) / sqrt(64)

  const int nkt = (s1 - s0 + ATT_BK - 1) / ATT_BK;
  SWAM_ATT_LOAD(0);
  SWAM_ATT_STORE(0);
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int cur = kt & 1;
    const int kb = s0 + kt * ATT_BK;
    SWAM_ATT_LOAD(kt + 1 < nkt ? kt + 1 : kt);        // last iteration: harmless re-read

    // S^T tile: two 32-key halves
    f32x16 st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) st[t][r] = 0.0f;
      const int key = 32 * t + (lane & 31);
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int ch = 2 * s + g;
        bf16x8 kf = __builtin_bit_cast(bf16x8, Ks[cur][key * 8 + (ch ^ (key & 7))]);
        st[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], st[t], 0, 0, 0);
      }
    }
    // keys beyond the sequence exist only in the last tile (wave-uniform branch)
    const int nvalid = s1 - kb;
    if (nvalid < ATT_BK) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * t + 8 * (r >> 2) + 4 * g + (r & 3);
          if (key >= nvalid) st[t][r] = -INFINITY;
        }
    }
    // row max of the raw logits: 16 keys in-lane per half tile, the rest in lane ^ 32
    float mx = st[0][0];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, st[t][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    // lazy rescaling: the running max (log2 units) is only raised when some row of
    // the wave grew by more than 2^8; otherwise p <= 256 against the stale max
    const float m_tile = mx * sc;
    if (__any(m_tile > m_run + 8.0f)) {
      const float m_new = fmaxf(m_run, m_tile);
      const float corr = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= corr;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] *= corr;
    }
    // p = exp2(s * sc - m); P^T packed to bf16 pairs for the PV MFMA; the row sum
    // (and so lambda, which the scorer reuses) is accumulated from the fp32 values
    bf16x8 pf[2][2];
    float psum0 = 0.0f, psum1 = 0.0f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
#pragma unroll
        for (int mm = 0; mm < 8; mm += 2) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(st[t][8 * u + mm], sc, -m_run));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(st[t][8 * u + mm + 1], sc, -m_run));
          psum0 += p0;
          psum1 += p1;
          pf[t][u][mm] = (__bf16)p0;
          pf[t][u][mm + 1] = (__bf16)p1;
        }
      }
    const float psum = psum0 + psum1;
    l_run += psum;

    // O^T += V^T P^T; k-substep (t, u) covers keys 32t + 16u + {4g..4g+3, 8+4g..8+4g+3}
#pragma unroll
    for (int ht = 0; ht < 2; ++ht) {
      const int hd = 32 * ht + (lane & 31);
      const uint32_t* vrow = &Vt[cur][hd * (VT_PITCH / 2)];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int kb0 = 32 * t + 16 * u + 4 * g;          // keys kb0..kb0+3 and kb0+8..+11
          uint2 lo = *(const uint2*)(vrow + kb0 / 2);
          uint2 hi = *(const uint2*)(vrow + (kb0 + 8) / 2);
          uint4 w = make_uint4(lo.x, lo.y, hi.x, hi.y);
          bf16x8 vf = __builtin_bit_cast(bf16x8, w);
          o[ht] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[t][u], o[ht], 0, 0, 0);
        }
    }
    SWAM_ATT_STORE(cur ^ 1);                   // other stage released by the last barrier
    __syncthreads();
  }

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
#undef SWAM_ATT_LOAD
#undef SWAM_ATT_STORE
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
    const int slots = (int)((n_rows + ATT_BQ - 1) / ATT_BQ) + n_seqs;
    const bool dense_grid = (int64_t)(slots - n_seqs) * n_heads >= 3 * 256;
    if (dense_grid)
      hipLaunchKernelGGL(attn_fwd_bf16<4>, dim3(slots * n_heads), dim3(256), 0, st,
                         (const bf16_t*)qkv, (bf16_t*)o, lse, cu_seqlens, n_seqs, n_heads,
                         (int)n_rows);
    else
      hipLaunchKernelGGL(attn_fwd_bf16<1>, dim3(slots * n_heads), dim3(256), 0, st,
                         (const bf16_t*)qkv, (bf16_t*)o, lse, cu_seqlens, n_seqs, n_heads,
                         (int)n_rows);
  } else {
    hipLaunchKernelGGL(attn_fwd_f32, dim3((unsigned)n_rows, n_heads), dim3(64), 0, st,
                       (const float*)qkv, (float*)o, lse, cu_seqlens, n_seqs, n_heads, n_rows);
  }
  return hipGetLastError();
}

}  // namespace swam
