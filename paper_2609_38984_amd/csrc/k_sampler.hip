// Sampling update around the sparse step (Sec. 4.2, merge of current and
// cached visual velocities; App. B.2 schedule shift):
//   embed   : tokens of the latent rows (future frames, then actions) from the
//             fp32 latents, x = z W_in^T + b_in, stored in the config dtype;
//   velocity: v = LN(y) W_v^T + b_v for every latent row, or only for the rows
//             of the cached selection (retained future tokens and actions);
//   update  : a full step stores the future velocities in the cache; a sparse
//             step uses the current velocity where the token was retained and
//             the cached one elsewhere (actions always current); then
//             z <- z + dsigma * v with one fp32 FMA.
// All three are memory-bound (c <= 64 latent channels against d >= 64 token
// channels); latents, velocities and the cache are fp32.
#include "common.h"

namespace swam {

// one thread per (latent row, 8 token columns): 16-byte stores of x
template <typename T>
__global__ void __launch_bounds__(256)
embed_kernel(const float* __restrict__ z, const T* __restrict__ w_in, const T* __restrict__ b_in,
             T* __restrict__ x, int64_t n_lat_rows, int l_lat, int l_full, int n_ctx, int c, int d) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int chunks = d / 8;
  if (id >= n_lat_rows * chunks) return;
  const int64_t i = id / chunks;
  const int col = (int)(id % chunks) * 8;
  const int64_t b = i / l_lat;
  const int64_t row = b * l_full + n_ctx + (i - b * l_lat);
  const float* zr = z + i * c;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
  for (int k = 0; k < c; ++k) {
    const float zk = zr[k];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = fmaf(zk, Elem<T>::load(w_in + (int64_t)(col + e) * c + k), acc[e]);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] += Elem<T>::load(b_in + col + e);
  T* xo = x + row * d + col;
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<uint4*>(xo) = make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                                               pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7]));
  } else {
    reinterpret_cast<float4*>(xo)[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    reinterpret_cast<float4*>(xo)[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
  }
}

// one wave per latent row; C = compile-time bound on the latent channels
template <typename T, int C>
__global__ void __launch_bounds__(256)
velocity_kernel(const T* __restrict__ y, const int32_t* __restrict__ gather, int64_t n_items,
                const T* __restrict__ w_v, const T* __restrict__ b_v, float* __restrict__ v,
                int l_lat, int l_full, int n_ctx, int c, int d) {
  const int lane = threadIdx.x & 63;
  const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= n_items) return;
  // items are latent rows (gather == NULL) or packed rows of the cached selection
  int64_t row, lat;
  if (gather == nullptr) {
    const int64_t b = item / l_lat;
    lat = item;
    row = b * l_full + n_ctx + (item - b * l_lat);
  } else {
    row = gather[item];
    const int64_t b = row / l_full, in_seq = row - b * l_full;
    if (in_seq < n_ctx) return;                    // context rows carry no latent
    lat = b * l_lat + (in_seq - n_ctx);
  }
  const T* yr = y + row * d;
  float s = 0.0f;
  for (int k = lane; k < d; k += 64) s += Elem<T>::load(yr + k);
  const float mean = warp_sum(s) / (float)d;
  float q = 0.0f;
  for (int k = lane; k < d; k += 64) {
    const float t = Elem<T>::load(yr + k) - mean;
    q = fmaf(t, t, q);
  }
  const float rstd = rsqrtf(warp_sum(q) / (float)d + 1e-6f);
  float acc[C];
#pragma unroll
  for (int j = 0; j < C; ++j) acc[j] = 0.0f;
  for (int k = lane; k < d; k += 64) {
    const float h = (Elem<T>::load(yr + k) - mean) * rstd;
#pragma unroll
    for (int j = 0; j < C; ++j)
      if (j < c) acc[j] = fmaf(h, Elem<T>::load(w_v + (int64_t)j * d + k), acc[j]);
  }
#pragma unroll
  for (int j = 0; j < C; ++j) {
    if (j >= c) break;
    const float t = warp_sum(acc[j]);
    if (lane == 0) v[lat * c + j] = t + Elem<T>::load(b_v + j);
  }
}

// one thread per latent element
__global__ void __launch_bounds__(256)
update_kernel(const float* __restrict__ v, float* __restrict__ v_cache, float* __restrict__ z,
              const int32_t* __restrict__ pack_pos, float dsigma, int kind, int64_t n,
              int l_lat, int l_full, int n_ctx, int n_fut, int c) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= n) return;
  const int64_t i = id / c;
  const int64_t b = i / l_lat;
  const int r = (int)(i - b * l_lat);
  float vt = v[id];
  if (r < n_fut) {
    if (kind == 1) v_cache[id] = vt;
    else if (kind == 2 && pack_pos[b * l_full + n_ctx + r] < 0) vt = v_cache[id];
  }
  z[id] = fmaf(dsigma, vt, z[id]);
}

hipError_t launch_embed(int dtype, const float* z, const void* w_in, const void* b_in, void* x,
                        int64_t n_lat_rows, int l_lat, int l_full, int n_ctx, int c, int d,
                        hipStream_t st) {
  if (n_lat_rows <= 0) return hipSuccess;
  const int64_t n = n_lat_rows * (d / 8);
  const dim3 grid((unsigned)((n + 255) / 256));
  if (dtype == 1)
    hipLaunchKernelGGL(embed_kernel<bf16_t>, grid, dim3(256), 0, st, z, (const bf16_t*)w_in,
                       (const bf16_t*)b_in, (bf16_t*)x, n_lat_rows, l_lat, l_full, n_ctx, c, d);
  else
    hipLaunchKernelGGL(embed_kernel<float>, grid, dim3(256), 0, st, z, (const float*)w_in,
                       (const float*)b_in, (float*)x, n_lat_rows, l_lat, l_full, n_ctx, c, d);
  return hipGetLastError();
}

template <typename T>
static hipError_t velocity_c(const void* y, const int32_t* gather, int64_t n_items, const void* w_v,
                             const void* b_v, float* v, int l_lat, int l_full, int n_ctx, int c,
                             int d, hipStream_t st) {
  const dim3 grid((unsigned)((n_items + 3) / 4));
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
  if (dtype == 1)
    return velocity_c<bf16_t>(y, gather, n_items, w_v, b_v, v, l_lat, l_full, n_ctx, c, d, st);
  return velocity_c<float>(y, gather, n_items, w_v, b_v, v, l_lat, l_full, n_ctx, c, d, st);
}

hipError_t launch_sample_update(const float* v, float* v_cache, float* z, const int32_t* pack_pos,
                                float dsigma, int kind, int64_t n_lat_rows, int l_lat, int l_full,
                                int n_ctx, int n_fut, int c, hipStream_t st) {
  const int64_t n = n_lat_rows * c;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(update_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, v,
                     v_cache, z, pack_pos, dsigma, kind, n, l_lat, l_full, n_ctx, n_fut, c);
  return hipGetLastError();
}

}  // namespace swam
