// One scoring unit of the reused-normaliser scorer (bf16): 16 future keys of
// one frame of one sequence (of one layer), scored against that frame's
// group of action queries:
//   S(f,j) = (1/N_h) sum_{i in I_f} sum_h alpha_i exp(q_h(i).k_h(f,j)/8 - lambda_h(i))
// Four waves take every 4th head: two 16x16x32 MFMAs per head with the keys
// as the A operand (lane -> key lane&15, 8 head dims at 8*(lane>>4)) and the
// group's queries as the B operand, so the accumulator gives each lane one
// query (lane & 15) and four keys.  exp2 of the scaled logit minus the
// query's normaliser is weighted by alpha (0 for padding queries), summed over
// the wave's heads in registers, reduced over queries with lane shuffles and
// over the four waves in LDS in a fixed order (deterministic: every caller
// gets the same bits).
//
// Used by the scoring kernel (one unit per workgroup) and by the MLP up
// projection of a refresh step, whose extra workgroups score a layer on the
// CUs that the projection's last round of tiles leaves idle.
#pragma once
#include "launchers.h"

namespace swam {

// unit -> (layer, sequence b, frame f, key tile kt), kt fastest
// wave4: this wave within its group of four; gtid: thread within the group;
// part: the group's 4 x 16 floats of LDS; sync(): a barrier over the group.
// active = false runs the barriers only (groups past the last unit).
template <class Sync>
__device__ __forceinline__ void score_unit_bf16(const ScoreArgs& a, int unit, bool active,
                                                int wave4, int lane, int gtid,
                                                float (*part)[16], Sync sync) {
  constexpr float kLog2e = 1.4426950408889634f;
  const int ktiles = (a.n_s + 15) >> 4;
  int bid = active ? unit : 0;
  const int kt = bid % ktiles;
  bid /= ktiles;
  const int f = bid % a.F;
  bid /= a.F;
  const int b = bid % a.B;
  const int layer = bid / a.B;
  const bf16_t* q = (const bf16_t*)a.q + layer * a.q_lay;
  const bf16_t* k = (const bf16_t*)a.k + layer * a.k_lay;
  const float* lse = a.lse + layer * a.lse_lay;
  float* s_out = a.s_out + layer * a.s_lay;
  const int g = a.H / a.F;
  const int j0 = kt * 16;
  const int key = min(j0 + (lane & 15), a.n_s - 1);
  const bf16_t* kp = k + b * a.k_seq + (int64_t)(f * a.n_s + key) * a.k_row + 8 * (lane >> 4);
  const int qi = lane & 15;                 // query slot within the group (C column)
  const int ql = min(qi, g - 1);            // loaded row (padding slots reuse a valid row)
  const float aw = qi < g ? a.alpha[qi] : 0.0f;
  const int qa = f * g + ql;
  const bf16_t* qp = q + b * a.q_seq + (int64_t)qa * a.q_row + 8 * (lane >> 4);
  const float* lp = lse + (int64_t)b * a.lse_seq + (int64_t)qa * a.n_heads;

  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  if (active) {
    for (int h = wave4; h < a.n_heads; h += 4) {
      const bf16x8 k0 = __builtin_bit_cast(bf16x8, *(const uint4*)(kp + h * 64));
      const bf16x8 k1 = __builtin_bit_cast(bf16x8, *(const uint4*)(kp + h * 64 + 32));
      const bf16x8 q0 = __builtin_bit_cast(bf16x8, *(const uint4*)(qp + h * 64));
      const bf16x8 q1 = __builtin_bit_cast(bf16x8, *(const uint4*)(qp + h * 64 + 32));
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, q0, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, q1, c, 0, 0, 0);
      const float lam = lp[h] * kLog2e;
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] += aw * exp2f(c[r] * (0.125f * kLog2e) - lam);
    }
  }
  // sum over the 16 query columns (lanes with equal lane >> 4)
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float v = acc[r];
    v += __shfl_xor(v, 8);
    v += __shfl_xor(v, 4);
    v += __shfl_xor(v, 2);
    v += __shfl_xor(v, 1);
    acc[r] = v;
  }
  if (active && (lane & 15) == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) part[wave4][4 * (lane >> 4) + r] = acc[r];
  }
  sync();
  if (active && gtid < 16) {
    const int j = j0 + gtid;
    if (j < a.n_s) {
      const float s = ((part[0][gtid] + part[1][gtid]) + (part[2][gtid] + part[3][gtid])) /
                      (float)a.n_heads;
      s_out[(int64_t)b * a.s_seq + (int64_t)f * a.n_s + j] = s;
    }
  }
}

}  // namespace swam
