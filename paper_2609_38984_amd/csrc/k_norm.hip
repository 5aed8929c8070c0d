// adaLN modulation vectors and the modulated LayerNorm of the DiT block.
//   mod = W_ada SiLU(t_emb) + b_ada        (all blocks of a step in one launch)
//   h   = LN(x) (1 + scale) + shift       (biased variance, eps 1e-6, no affine)
// One wavefront per output row (modulation) or per token row (LN); the row
// stays in registers between the mean and the variance pass.
#include "launchers.h"

namespace swam {

template <typename T>
__global__ void __launch_bounds__(256)
adaln_kernel(AdalnArgs args, const float* __restrict__ temb, int d_temb, int d6,
             float* __restrict__ mod) {
  const int blk = blockIdx.y;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= d6) return;
  const T* w = (const T*)args.w[blk] + (int64_t)row * d_temb;
  float acc = 0.0f;
  for (int k = lane; k < d_temb; k += 64) {
    const float t = temb[k];
    acc = fmaf(Elem<T>::load(w + k), t / (1.0f + expf(-t)), acc);
  }
  acc = warp_sum(acc);
  if (lane == 0) mod[(int64_t)blk * d6 + row] = acc + Elem<T>::load((const T*)args.b[blk] + row);
}

// bf16 weights, d_temb = 128: 16 lanes per output row (one 16-byte load of 8
// weights each), ADALN_RPG rows per 16-lane group (rows g, g + 16, ... of the
// workgroup's 16 * ADALN_RPG, so each round of loads reads 4 KB of
// consecutive rows), every load issued before the first reduction; SiLU(temb)
// once per lane instead of once per weight
constexpr int ADALN_RPG = 8;

__global__ void __launch_bounds__(256)
adaln_bf16_t128(AdalnArgs args, const float* __restrict__ temb, int d6,
                float* __restrict__ mod) {
  const int blk = blockIdx.y;
  const int g = threadIdx.x >> 4;
  const int row0 = blockIdx.x * (16 * ADALN_RPG) + g;
  const int k0 = (threadIdx.x & 15) * 8;
  const bf16_t* wb = (const bf16_t*)args.w[blk];
  uint4 w[ADALN_RPG];
#pragma unroll
  for (int j = 0; j < ADALN_RPG; ++j) {
    const int rr = min(row0 + 16 * j, d6 - 1);   // every lane joins the exchange
    w[j] = *reinterpret_cast<const uint4*>(wb + (int64_t)rr * 128 + k0);
  }
  float sl[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float t = temb[k0 + e];
    sl[e] = t / (1.0f + expf(-t));
  }
  const bf16_t* bb = (const bf16_t*)args.b[blk];
#pragma unroll
  for (int j = 0; j < ADALN_RPG; ++j) {
    const uint32_t p[4] = {w[j].x, w[j].y, w[j].z, w[j].w};
    float acc = 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc = fmaf(__uint_as_float(p[e] << 16), sl[2 * e], acc);
      acc = fmaf(__uint_as_float(p[e] & 0xFFFF0000u), sl[2 * e + 1], acc);
    }
    acc += __shfl_xor(acc, 1);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 4);
    acc += __shfl_xor(acc, 8);
    const int row = row0 + 16 * j;
    if ((threadIdx.x & 15) == 0 && row < d6)
      mod[(int64_t)blk * d6 + row] = acc + bf16_to_f32(bb[row]);
  }
}

hipError_t launch_adaln(int dtype, const AdalnArgs& a, int n_blk, const float* temb,
                        int d_temb, int d6, float* mod, hipStream_t st) {
  if (dtype == 1 && d_temb == 128) {
    hipLaunchKernelGGL(adaln_bf16_t128, dim3((d6 + 16 * ADALN_RPG - 1) / (16 * ADALN_RPG), n_blk),
                       dim3(256), 0, st, a, temb, d6, mod);
    return hipGetLastError();
  }
  dim3 grid((d6 + 3) / 4, n_blk);
  if (dtype == 1)
    hipLaunchKernelGGL(adaln_kernel<bf16_t>, grid, dim3(256), 0, st, a, temb, d_temb, d6, mod);
  else
    hipLaunchKernelGGL(adaln_kernel<float>, grid, dim3(256), 0, st, a, temb, d_temb, d6, mod);
  return hipGetLastError();
}

// bf16 rows: 16-byte chunks of 8 elements, up to CH chunks per lane (d <= 512 CH).
// GATHER: output row r reads input row gather[r] and also stores it unchanged
// to xp row r (the gather-pack of a sparse step fused into its first LN).
template <int CH, bool GATHER>
__global__ void __launch_bounds__(256)
ln_mod_bf16(const bf16_t* __restrict__ x, bf16_t* __restrict__ h,
            const float* __restrict__ shift, const float* __restrict__ scale, int64_t rows,
            int d, const int32_t* __restrict__ gather, bf16_t* __restrict__ xp) {
  const int64_t row =
      (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int nch = d >> 3;
  const int64_t src = GATHER ? (int64_t)gather[row] : row;
  const uint4* xr = (const uint4*)(x + src * d);
  float v[CH][8];
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int ci = lane + 64 * c;
    if (ci < nch) {
      const uint4 w = xr[ci];
      if (GATHER) ((uint4*)(xp + row * d))[ci] = w;
      const uint32_t p[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[c][2 * e] = __uint_as_float(p[e] << 16);
        v[c][2 * e + 1] = __uint_as_float(p[e] & 0xFFFF0000u);
        s += v[c][2 * e] + v[c][2 * e + 1];
      }
    }
  }
  const float mean = warp_sum(s) / d;
  float q = 0.0f;
#pragma unroll
  for (int c = 0; c < CH; ++c)
    if (lane + 64 * c < nch)
#pragma unroll
      for (int e = 0; e < 8; ++e) { const float t = v[c][e] - mean; q += t * t; }
  const float rstd = rsqrtf(warp_sum(q) / d + 1e-6f);
  uint4* hr = (uint4*)(h + row * d);
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int ci = lane + 64 * c;
    if (ci < nch) {
      const int col = ci * 8;
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        o[e] = (v[c][e] - mean) * rstd * (1.0f + scale[col + e]) + shift[col + e];
      uint4 w;
      w.x = pack_bf16x2(o[0], o[1]);
      w.y = pack_bf16x2(o[2], o[3]);
      w.z = pack_bf16x2(o[4], o[5]);
      w.w = pack_bf16x2(o[6], o[7]);
      hr[ci] = w;
    }
  }
}

// fp32 rows: two passes over global memory (rows are L1/L2 resident);
// gather != NULL: as the bf16 GATHER variant
__global__ void __launch_bounds__(256)
ln_mod_f32(const float* __restrict__ x, float* __restrict__ h, const float* __restrict__ shift,
           const float* __restrict__ scale, int64_t rows, int d,
           const int32_t* __restrict__ gather, float* __restrict__ xp) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* xr = x + (gather ? (int64_t)gather[row] : row) * d;
  float s = 0.0f;
  for (int c = lane; c < d; c += 64) {
    s += xr[c];
    if (gather) xp[row * d + c] = xr[c];
  }
  const float mean = warp_sum(s) / d;
  float q = 0.0f;
  for (int c = lane; c < d; c += 64) { const float t = xr[c] - mean; q += t * t; }
  const float rstd = 1.0f / sqrtf(warp_sum(q) / d + 1e-6f);
  for (int c = lane; c < d; c += 64)
    h[row * d + c] = (xr[c] - mean) * rstd * (1.0f + scale[c]) + shift[c];
}

template <bool GATHER>
static hipError_t ln_mod_any(int dtype, const void* x, void* h, const float* shift,
                             const float* scale, int64_t rows, int d, const int32_t* gather,
                             void* xp, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  dim3 grid((unsigned)((rows + 3) / 4));
  if (dtype == 1) {
    const bf16_t* xb = (const bf16_t*)x;
    bf16_t* hb = (bf16_t*)h;
    bf16_t* pb = (bf16_t*)xp;
    if (d <= 1024)
      hipLaunchKernelGGL((ln_mod_bf16<2, GATHER>), grid, dim3(256), 0, st, xb, hb, shift, scale,
                         rows, d, gather, pb);
    else if (d <= 2048)
      hipLaunchKernelGGL((ln_mod_bf16<4, GATHER>), grid, dim3(256), 0, st, xb, hb, shift, scale,
                         rows, d, gather, pb);
    else
      hipLaunchKernelGGL((ln_mod_bf16<8, GATHER>), grid, dim3(256), 0, st, xb, hb, shift, scale,
                         rows, d, gather, pb);
  } else {
    hipLaunchKernelGGL(ln_mod_f32, grid, dim3(256), 0, st, (const float*)x, (float*)h, shift,
                       scale, rows, d, GATHER ? gather : nullptr, (float*)xp);
  }
  return hipGetLastError();
}

hipError_t launch_ln_mod(int dtype, const void* x, void* h, const float* shift,
                         const float* scale, int64_t rows, int d, hipStream_t st) {
  return ln_mod_any<false>(dtype, x, h, shift, scale, rows, d, nullptr, nullptr, st);
}

hipError_t launch_ln_mod_gather(int dtype, const void* x_full, const int32_t* gather, void* xp,
                                void* h, const float* shift, const float* scale, int64_t rows,
                                int d, hipStream_t st) {
  return ln_mod_any<true>(dtype, x_full, h, shift, scale, rows, d, gather, xp, st);
}

// ---------------------------------------------------------------------------
// backbone variants on the stored q and k: QK-norm (unit-gain RMS per head),
// then the rotary embedding at each row's original position
// ---------------------------------------------------------------------------
// [l_full][32] (cos, sin) of pos * 10000^(-2i/64), evaluated in float64
// cos / sin of position * 10000^(-2i/64) for positions [0, n_pos), i < 32
__global__ void rope_table_kernel(float2* __restrict__ tab, int n_pos) {
  const int id = blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= n_pos * 32) return;
  const int pos = id >> 5, i = id & 31;
  const double ang = (double)pos * pow(10000.0, -2.0 * i / 64.0);
  tab[id] = make_float2((float)cos(ang), (float)sin(ang));
}

hipError_t launch_rope_table(float2* tab, int n_pos, hipStream_t st) {
  hipLaunchKernelGGL(rope_table_kernel, dim3((n_pos * 32 + 255) / 256), dim3(256), 0, st, tab,
                     n_pos);
  return hipGetLastError();
}

// one thread per 8 consecutive elements of q or k (a head is 8 threads, which
// are 8 consecutive lanes); pos_mode 0: row % l_full, 1: gather[row] % l_full,
// 2: row - cu[b] for the row's sequence b; positions are clamped to the
// table's n_pos rows
template <typename T>
__global__ void __launch_bounds__(256)
qk_post_kernel(T* __restrict__ qkv, int64_t n_rows, int d, int pos_mode,
               const int32_t* __restrict__ gather, const int32_t* __restrict__ cu, int n_seqs,
               int l_full, const float2* __restrict__ tab, int n_pos, int qk_norm) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int chunks = 2 * d / 8;               // q and k columns of a row
  const bool live = id < n_rows * chunks;
  const int64_t row = live ? id / chunks : 0;
  const int c8 = live ? (int)(id % chunks) * 8 : 0;
  T* p = qkv + row * 3 * d + c8;
  float x[8];
  if constexpr (sizeof(T) == 2) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(wv[e] << 16);
      x[2 * e + 1] = __uint_as_float(wv[e] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = p[e];
  }
  if (qk_norm) {
    // the 8 lanes of a head are consecutive and aligned (chunks per row and per
    // head are multiples of 8); every lane takes part in the exchange
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
  if (!live) return;
  if (tab != nullptr) {
    int pos;
    if (pos_mode == 0) {
      pos = (int)(row % l_full);
    } else if (pos_mode == 1) {
      pos = gather[row] % l_full;
    } else {
      int b = 0;
      while (b + 1 < n_seqs && cu[b + 1] <= row) ++b;
      pos = (int)(row - cu[b]);
    }
    pos = min(max(pos, 0), n_pos - 1);
    const float2* t = tab + (int64_t)pos * 32 + ((c8 & 63) >> 1);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float2 cs = t[e];
      const float a = x[2 * e], b = x[2 * e + 1];
      x[2 * e] = a * cs.x - b * cs.y;
      x[2 * e + 1] = a * cs.y + b * cs.x;
    }
  }
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<uint4*>(p) = make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]),
                                              pack_bf16x2(x[4], x[5]), pack_bf16x2(x[6], x[7]));
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) p[e] = x[e];
  }
}

hipError_t launch_qk_post(int dtype, void* qkv, int64_t n_rows, int d, int pos_mode,
                          const int32_t* gather, const int32_t* cu, int n_seqs, int l_full,
                          const float2* tab, int n_pos, int qk_norm, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  const int64_t n = n_rows * (2 * d / 8);
  const dim3 grid((unsigned)((n + 255) / 256));
  if (dtype == 1)
    hipLaunchKernelGGL(qk_post_kernel<bf16_t>, grid, dim3(256), 0, st, (bf16_t*)qkv, n_rows, d,
                       pos_mode, gather, cu, n_seqs, l_full, tab, n_pos, qk_norm);
  else
    hipLaunchKernelGGL(qk_post_kernel<float>, grid, dim3(256), 0, st, (float*)qkv, n_rows, d,
                       pos_mode, gather, cu, n_seqs, l_full, tab, n_pos, qk_norm);
  return hipGetLastError();
}

}  // namespace swam
