// Sampling update around the sparse step (Sec. 4.2, merge of current and
// cached visual velocities; App. B.2 schedule shift):
//   embed   : tokens of the latent rows (future frames, then actions) from the
//             fp32 latents, x = z W_in^T + b_in, stored in the config dtype;
//   velocity: v = LN(y) W_v^T + b_v for every latent row, or only for the rows
//             of the cached selection (retained future tokens and actions);
//             bf16 on the matrix cores (16 rows per wave), fp32 one row per
//             wave on the vector units;
//   update  : with guidance pairs the two branch velocities of a latent row
//             are first combined as v_u + g (v_c - v_u); a full step stores the
//             future velocities in the cache; a sparse step uses the current
//             velocity where the token was retained and the cached one
//             elsewhere (actions always current); then z <- z + dsigma * v
//             with one fp32 FMA.
// All three are memory-bound (c <= 64 latent channels against d >= 64 token
// channels); latents, velocities and the cache are fp32.
#include "launchers.h"

namespace swam {

// 8 consecutive elements of a T row as fp32 (one 16-byte load for bf16)
template <typename T>
__device__ __forceinline__ void load8(const T* p, float (&o)[8]) {
  if constexpr (sizeof(T) == 2) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[2 * e] = __uint_as_float(w[e] << 16);
      o[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  } else {
    const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w; o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
  }
}

// one thread per (latent row, 8 token columns): each output column reads its
// W_in row (c contiguous values) in 16-byte pieces; 16-byte stores of x.
// Needs c % 8 == 0 (the launcher falls back to scalar weight loads otherwise).
template <typename T, bool VEC>
__global__ void __launch_bounds__(256)
embed_kernel(const float* __restrict__ z, const T* __restrict__ w_in, const T* __restrict__ b_in,
             T* __restrict__ x, int64_t n_lat_rows, int64_t z_rows, int l_lat, int l_full, int n_ctx,
             int c, int d) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int chunks = d / 8;
  if (id >= n_lat_rows * chunks) return;
  const int64_t i = id / chunks;
  const int col = (int)(id % chunks) * 8;
  const int64_t b = i / l_lat;
  const int64_t row = b * l_full + n_ctx + (i - b * l_lat);
  const float* zr = z + (i < z_rows ? i : i - z_rows) * c;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
  if constexpr (VEC) {
    for (int k0 = 0; k0 < c; k0 += 8) {
      const float4 za = *reinterpret_cast<const float4*>(zr + k0);
      const float4 zb = *reinterpret_cast<const float4*>(zr + k0 + 4);
      const float zk[8] = {za.x, za.y, za.z, za.w, zb.x, zb.y, zb.z, zb.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float w[8];
        load8(w_in + (int64_t)(col + e) * c + k0, w);
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[e] = fmaf(zk[q], w[q], acc[e]);
      }
    }
  } else {
    for (int k = 0; k < c; ++k) {
      const float zk = zr[k];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = fmaf(zk, Elem<T>::load(w_in + (int64_t)(col + e) * c + k), acc[e]);
    }
  }
  float bb[8];
  load8(b_in + col, bb);
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] += bb[e];
  T* xo = x + row * d + col;
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<uint4*>(xo) = make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                                               pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7]));
  } else {
    reinterpret_cast<float4*>(xo)[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    reinterpret_cast<float4*>(xo)[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
  }
}

// c in {8, 16}: each thread keeps the W_in rows of its 8 columns in registers
// and walks EMB_ROWS consecutive latent rows, four at a time (the weights are
// read once per thread instead of once per row; the z row is the same address
// across the wave and 64 lanes store one contiguous kilobyte of x per row).
constexpr int EMB_ROWS = 16;
template <typename T, int C>
__global__ void __launch_bounds__(256)
embed_reg_kernel(const float* __restrict__ z, const T* __restrict__ w_in, const T* __restrict__ b_in,
                 T* __restrict__ x, int64_t n_lat_rows, int64_t z_rows, int l_lat, int l_full,
                 int n_ctx, int d) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int chunks = d / 8;
  const int64_t groups = (n_lat_rows + EMB_ROWS - 1) / EMB_ROWS;
  if (id >= groups * chunks) return;
  const int col = (int)(id % chunks) * 8;
  const int64_t i0 = (id / chunks) * EMB_ROWS;
  float w[8][C], bb[8];
#pragma unroll
  for (int e = 0; e < 8; ++e)
#pragma unroll
    for (int k0 = 0; k0 < C; k0 += 8) {
      float t[8];
      load8(w_in + (int64_t)(col + e) * C + k0, t);
#pragma unroll
      for (int q = 0; q < 8; ++q) w[e][k0 + q] = t[q];
    }
  load8(b_in + col, bb);
  const int64_t i1 = i0 + EMB_ROWS < n_lat_rows ? i0 + EMB_ROWS : n_lat_rows;
#pragma unroll 4
  for (int64_t i = i0; i < i1; ++i) {
    const int64_t b = i / l_lat;
    const int64_t row = b * l_full + n_ctx + (i - b * l_lat);
    float zk[C];
    const float* zr = z + (i < z_rows ? i : i - z_rows) * C;
#pragma unroll
    for (int k0 = 0; k0 < C; k0 += 4) {
      const float4 t = *reinterpret_cast<const float4*>(zr + k0);
      zk[k0] = t.x; zk[k0 + 1] = t.y; zk[k0 + 2] = t.z; zk[k0 + 3] = t.w;
    }
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      acc[e] = 0.0f;
#pragma unroll
      for (int k = 0; k < C; ++k) acc[e] = fmaf(zk[k], w[e][k], acc[e]);
      acc[e] += bb[e];
    }
    T* xo = x + row * d + col;
    if constexpr (sizeof(T) == 2) {
      *reinterpret_cast<uint4*>(xo) = make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                                                 pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7]));
    } else {
      reinterpret_cast<float4*>(xo)[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
      reinterpret_cast<float4*>(xo)[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
    }
  }
}

// one wave per latent row: each lane holds 8-element pieces of the row
// (16-byte loads, kept in registers across the mean, variance and head
// passes) and reads the matching 16-byte pieces of every W_v row.
constexpr int VEL_MAXP = 8;          // pieces per lane: d <= 64 * 8 * 8 = 4096
constexpr int VEL_LDS = 4096;        // uint4 slots: W_v staged in LDS when c * d * sizeof(T) <= 64 KB
template <typename T, int C>
__global__ void __launch_bounds__(256)
velocity_kernel(const T* __restrict__ y, const int32_t* __restrict__ gather, int64_t n_items,
                const T* __restrict__ w_v, const T* __restrict__ b_v, float* __restrict__ v,
                int l_lat, int l_full, int n_ctx, int c, int d) {
  __shared__ uint4 wl[VEL_LDS];
  const int lane = threadIdx.x & 63;
  // the whole head matrix into LDS once per workgroup (the launcher checks the size)
  const int n16 = c * d * (int)sizeof(T) / 16;
  for (int t = threadIdx.x; t < n16; t += blockDim.x) wl[t] = reinterpret_cast<const uint4*>(w_v)[t];
  __syncthreads();
  const T* wv = reinterpret_cast<const T*>(wl);
  const int np = (d + 511) / 512;                    // 8-element pieces per lane (uniform)
  const int items = (int)n_items;
  for (int item = blockIdx.x * 4 + (threadIdx.x >> 6); item < items; item += gridDim.x * 4) {
    // items are latent rows (gather == NULL) or packed rows of the cached selection
    int row, lat;
    if (gather == nullptr) {
      const int b = item / l_lat;
      lat = item;
      row = b * l_full + n_ctx + (item - b * l_lat);
    } else {
      row = gather[item];
      const int b = row / l_full, in_seq = row - b * l_full;
      if (in_seq < n_ctx) continue;                  // context rows carry no latent
      lat = b * l_lat + (in_seq - n_ctx);
    }
    const T* yr = y + (int64_t)row * d;
    float h[VEL_MAXP][8];
    float s = 0.0f;
#pragma unroll
    for (int p = 0; p < VEL_MAXP; ++p) {
      if (p < np) {
        const int k0 = 8 * lane + 512 * p;
        if (k0 < d) {
          load8(yr + k0, h[p]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) h[p][e] = 0.0f;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) s += h[p][e];
      }
    }
    const float mean = warp_sum(s) / (float)d;
    float q = 0.0f;
#pragma unroll
    for (int p = 0; p < VEL_MAXP; ++p) {
      if (p < np) {
        const bool live = 8 * lane + 512 * p < d;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          h[p][e] = live ? h[p][e] - mean : 0.0f;
          q = fmaf(h[p][e], h[p][e], q);
        }
      }
    }
    const float rstd = rsqrtf(warp_sum(q) / (float)d + 1e-6f);
    float acc[C];
#pragma unroll
    for (int j = 0; j < C; ++j) acc[j] = 0.0f;
#pragma unroll
    for (int p = 0; p < VEL_MAXP; ++p) {
      if (p < np) {
        // lanes past the end of the row read a valid piece of W_v and multiply it by 0
        const int k0 = min(8 * lane + 512 * p, d - 8);
#pragma unroll
        for (int j = 0; j < C; ++j) {
          if (j < c) {
            float w[8];
            load8(wv + j * d + k0, w);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[j] = fmaf(h[p][e], w[e], acc[j]);
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < C; ++j) {
      if (j < c) {
        const float t = warp_sum(acc[j]) * rstd;
        if (lane == 0) v[(int64_t)lat * c + j] = t + Elem<T>::load(b_v + j);
      }
    }
  }
}

// bf16 read-out on the matrix cores: one workgroup per 16 rows, 16x16 tiles
// of y . W_v^T by 16x16x32 MFMAs along d, the 32-column chunks of d dealt
// round-robin to the VEL_WAVES waves (lane l feeds row l & 15 and eight
// consecutive columns of its k-group l >> 4; W_v rows are the B operand,
// read straight from L2).  The row sums and sums of squares and the column
// sums of W_v come from the same fragments; the waves' partials are added
// in LDS in a fixed order and
//   v = rstd * (y . W_v^T - mean * sum_k W_v) + b_v,  rstd = 1/sqrt(var + eps)
// gives LN(y) W_v^T + b_v without a second pass over the row.
constexpr int VEL_WAVES = 4;
template <int NT>
__global__ void __launch_bounds__(64 * VEL_WAVES)
velocity_mfma_kernel(const bf16_t* __restrict__ y, const int32_t* __restrict__ gather, int n_items,
                     const bf16_t* __restrict__ w_v, const bf16_t* __restrict__ b_v,
                     float* __restrict__ v, int l_lat, int l_full, int n_ctx, int c, int d) {
  constexpr int NP = 5 * NT + 2;                 // partials per lane: acc, column sums, s1, s2
  __shared__ float red[VEL_WAVES - 1][NP][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, kg = lane >> 4;
  const int item = blockIdx.x * 16 + r;
  int row = 0, lat = -1;                         // lat < 0: nothing to write for this row
  if (item < n_items) {
    if (gather == nullptr) {
      const int b = item / l_lat;
      lat = item;
      row = b * l_full + n_ctx + (item - b * l_lat);
    } else {
      row = gather[item];
      const int b = row / l_full, in_seq = row - b * l_full;
      lat = in_seq < n_ctx ? -1 : b * l_lat + (in_seq - n_ctx);   // context rows carry no latent
    }
  }
  const bf16_t* yr = y + (int64_t)row * d + 8 * kg;
  f32x4 acc[NT];
  float cs[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    cs[t] = 0.f;
  }
  float s1 = 0.f, s2 = 0.f;
#pragma unroll 2
  for (int k0 = 32 * wave; k0 < d; k0 += 32 * VEL_WAVES) {
    const uint4 a = *reinterpret_cast<const uint4*>(yr + k0);
    const uint32_t aw[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = __uint_as_float(aw[e] << 16), hi = __uint_as_float(aw[e] & 0xFFFF0000u);
      s1 += lo + hi;
      s2 = fmaf(lo, lo, fmaf(hi, hi, s2));
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int n = t * 16 + r;
      uint4 w = make_uint4(0u, 0u, 0u, 0u);
      if (n < c) w = *reinterpret_cast<const uint4*>(w_v + (int64_t)n * d + k0 + 8 * kg);
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        cs[t] += __uint_as_float(ww[e] << 16) + __uint_as_float(ww[e] & 0xFFFF0000u);
      acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, w), acc[t], 0, 0, 0);
    }
  }
  // the waves' partial sums, added by wave 0 in wave order
  if (wave > 0) {
    float* q = &red[wave - 1][0][lane];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
      for (int i = 0; i < 4; ++i) q[(4 * t + i) * 64] = acc[t][i];
      q[(4 * NT + t) * 64] = cs[t];
    }
    q[(5 * NT) * 64] = s1;
    q[(5 * NT + 1) * 64] = s2;
  }
  __syncthreads();
  if (wave > 0) return;
  for (int w = 0; w < VEL_WAVES - 1; ++w) {
    const float* q = &red[w][0][lane];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[t][i] += q[(4 * t + i) * 64];
      cs[t] += q[(4 * NT + t) * 64];
    }
    s1 += q[(5 * NT) * 64];
    s2 += q[(5 * NT + 1) * 64];
  }
  // full-row statistics: the four k-groups of row r are lanes r, r+16, r+32, r+48
  s1 += __shfl_xor(s1, 16);
  s1 += __shfl_xor(s1, 32);
  s2 += __shfl_xor(s2, 16);
  s2 += __shfl_xor(s2, 32);
  const float mean = s1 / (float)d;
  const float rstd = rsqrtf(fmaxf(s2 / (float)d - mean * mean, 0.0f) + 1e-6f);
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    cs[t] += __shfl_xor(cs[t], 16);
    cs[t] += __shfl_xor(cs[t], 32);
  }
  // lane l holds output rows 4 kg + i (i < 4) of column r of every tile
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int src = 4 * kg + i;
    const float m_i = __shfl(mean, src), r_i = __shfl(rstd, src);
    const int lat_i = __shfl(lat, src);
    if (lat_i < 0) continue;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int n = t * 16 + r;
      if (n < c)
        v[(int64_t)lat_i * c + n] = r_i * (acc[t][i] - m_i * cs[t]) + Elem<bf16_t>::load(b_v + n);
    }
  }
}

// one thread per latent element (of the conditional half with pairs)
__global__ void __launch_bounds__(256)
update_kernel(const float* __restrict__ v, float* __restrict__ v_cache, float* __restrict__ z,
              const int32_t* __restrict__ pack_pos, float dsigma, int kind, int64_t n,
              int l_lat, int l_full, int n_ctx, int n_fut, int c, int pairs, float guidance) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= n) return;
  const int64_t i = id / c;
  const int64_t b = i / l_lat;
  const int r = (int)(i - b * l_lat);
  float vt = v[id];
  if (pairs) {
    const float vu = v[id + n];
    vt = fmaf(guidance, vt - vu, vu);
  }
  if (r < n_fut) {
    if (kind == 1) v_cache[id] = vt;
    else if (kind == 2 && pack_pos[b * l_full + n_ctx + r] < 0) vt = v_cache[id];
  }
  z[id] = fmaf(dsigma, vt, z[id]);
}

hipError_t launch_embed(int dtype, const float* z, const void* w_in, const void* b_in, void* x,
                        int64_t n_lat_rows, int64_t z_rows, int l_lat, int l_full, int n_ctx,
                        int c, int d, hipStream_t st) {
  if (n_lat_rows <= 0) return hipSuccess;
  const int64_t n = n_lat_rows * (d / 8);
  const dim3 grid((unsigned)((n + 255) / 256));
  if (c == 8 || c == 16) {
    const int64_t groups = (n_lat_rows + EMB_ROWS - 1) / EMB_ROWS;
    const dim3 g2((unsigned)((groups * (d / 8) + 255) / 256));
#define SWAM_EMBR(T_, C_)                                                                      \
  hipLaunchKernelGGL((embed_reg_kernel<T_, C_>), g2, dim3(256), 0, st, z, (const T_*)w_in,     \
                     (const T_*)b_in, (T_*)x, n_lat_rows, z_rows, l_lat, l_full, n_ctx, d)
    if (dtype == 1) {
      if (c == 8) SWAM_EMBR(bf16_t, 8); else SWAM_EMBR(bf16_t, 16);
    } else {
      if (c == 8) SWAM_EMBR(float, 8); else SWAM_EMBR(float, 16);
    }
#undef SWAM_EMBR
    return hipGetLastError();
  }
  const bool vec = c % 8 == 0;
#define SWAM_EMB(T_, V_)                                                                       \
  hipLaunchKernelGGL((embed_kernel<T_, V_>), grid, dim3(256), 0, st, z, (const T_*)w_in,       \
                     (const T_*)b_in, (T_*)x, n_lat_rows, z_rows, l_lat, l_full, n_ctx, c, d)
  if (dtype == 1) {
    if (vec) SWAM_EMB(bf16_t, true); else SWAM_EMB(bf16_t, false);
  } else {
    if (vec) SWAM_EMB(float, true); else SWAM_EMB(float, false);
  }
#undef SWAM_EMB
  return hipGetLastError();
}

template <typename T>
static hipError_t velocity_c(const void* y, const int32_t* gather, int64_t n_items, const void* w_v,
                             const void* b_v, float* v, int l_lat, int l_full, int n_ctx, int c,
                             int d, hipStream_t st) {
  if ((int64_t)c * d * (int64_t)sizeof(T) > (int64_t)VEL_LDS * 16 || d > 64 * 8 * VEL_MAXP)
    return hipErrorInvalidValue;                     // checked at the API: c * d * esz <= 64 KB
  const int64_t wgs = (n_items + 3) / 4;
  const dim3 grid((unsigned)(wgs < 1024 ? wgs : 1024));
#define SWAM_VEL(CB)                                                                              \
  hipLaunchKernelGGL((velocity_kernel<T, CB>), grid, dim3(256), 0, st, (const T*)y, gather,      \
                     n_items, (const T*)w_v, (const T*)b_v, v, l_lat, l_full, n_ctx, c, d)
  if (c <= 8) SWAM_VEL(8);
  else if (c <= 16) SWAM_VEL(16);
  else if (c <= 32) SWAM_VEL(32);
  else SWAM_VEL(64);
#undef SWAM_VEL
  return hipGetLastError();
}

hipError_t launch_velocity(int dtype, const void* y, const int32_t* gather, int64_t n_items,
                           const void* w_v, const void* b_v, float* v, int l_lat, int l_full,
                           int n_ctx, int c, int d, hipStream_t st) {
  if (n_items <= 0) return hipSuccess;
  if (dtype == 1 && d % 32 == 0 && c <= 64) {
    const dim3 grid((unsigned)((n_items + 15) / 16));
    const int ni = (int)n_items;
#define SWAM_VELM(NT_)                                                                        \
  hipLaunchKernelGGL((velocity_mfma_kernel<NT_>), grid, dim3(64 * VEL_WAVES), 0, st,          \
                     (const bf16_t*)y, gather, ni, (const bf16_t*)w_v, (const bf16_t*)b_v, v,   \
                     l_lat, l_full, n_ctx, c, d)
    if (c <= 16) SWAM_VELM(1);
    else if (c <= 32) SWAM_VELM(2);
    else if (c <= 48) SWAM_VELM(3);
    else SWAM_VELM(4);
#undef SWAM_VELM
    return hipGetLastError();
  }
  if (dtype == 1)
    return velocity_c<bf16_t>(y, gather, n_items, w_v, b_v, v, l_lat, l_full, n_ctx, c, d, st);
  return velocity_c<float>(y, gather, n_items, w_v, b_v, v, l_lat, l_full, n_ctx, c, d, st);
}

hipError_t launch_sample_update(const float* v, float* v_cache, float* z, const int32_t* pack_pos,
                                float dsigma, int kind, int64_t n_lat_rows, int l_lat, int l_full,
                                int n_ctx, int n_fut, int c, int pairs, float guidance,
                                hipStream_t st) {
  const int64_t n = n_lat_rows * c;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(update_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, v,
                     v_cache, z, pack_pos, dsigma, kind, n, l_lat, l_full, n_ctx, n_fut, c, pairs,
                     guidance);
  return hipGetLastError();
}

}  // namespace swam
