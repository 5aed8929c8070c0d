// Action-to-future spatial scores of one layer (reused-normaliser scorer):
//   S(f,j) = (1/N_h) sum_{i in I_f} sum_h alpha_i exp(q_h(i).k_h(f,j)/8 - lambda_h(i))
// Only frame-f keys against frame-f's query group are formed; no attention
// matrix, no value product.  The work is a thin contraction (g <= 16 queries
// against a stream of keys), so it is bound by the single read of the future
// keys; MFMA only keeps the dot products off the VALU.
//
// One launch may score several layers (layer strides in ScoreArgs); a
// bf16 refresh step scores each layer inside that layer's MLP up projection
// launch (the same units, score_unit.h) and the last layer with this kernel.
//
// bf16: workgroup = 4 waves on 16 keys of one frame (score_unit.h); the MLP
// up projection of a refresh step can run the same units in extra
// workgroups of its own launch instead.
// fp32: one thread per key.
// Mode B normaliser: lambda over all keys of the sequence, per (query, head),
// as an online max/sum split over key chunks with wavefront-shuffle
// reductions, combined in a second pass.
#include "score_unit.h"

namespace swam {

// one 16-key unit per workgroup of four waves
__global__ void __launch_bounds__(256) score_bf16(const ScoreArgs a) {
  __shared__ float part[4][16];
  score_unit_bf16(a, (int)blockIdx.x, true, (int)(threadIdx.x >> 6), (int)(threadIdx.x & 63),
                  (int)threadIdx.x, part, [] { __syncthreads(); });
}

__global__ void __launch_bounds__(256)
score_f32(const float* __restrict__ q, int64_t q_seq, int64_t q_row,
          const float* __restrict__ k, int64_t k_seq, int64_t k_row,
          const float* __restrict__ lse, int64_t lse_seq, float* __restrict__ s_out,
          int64_t s_seq, const float* __restrict__ alpha, int B, int F, int n_s, int H,
          int n_heads, int n_layers, int64_t q_lay, int64_t k_lay, int64_t lse_lay,
          int64_t s_lay) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (int64_t)n_layers * B * F * n_s) return;
  const int j = id % n_s, f = (id / n_s) % F, b = (id / ((int64_t)n_s * F)) % B;
  const int layer = (int)(id / ((int64_t)n_s * F * B));
  q += layer * q_lay;
  k += layer * k_lay;
  lse += layer * lse_lay;
  s_out += layer * s_lay;
  const int g = H / F;
  const float* kr = k + b * k_seq + (int64_t)(f * n_s + j) * k_row;
  float s = 0.0f;
  for (int h = 0; h < n_heads; ++h) {
    for (int a = 0; a < g; ++a) {
      const int qa = f * g + a;
      const float* qr = q + b * q_seq + (int64_t)qa * q_row + h * 64;
      float x = 0.0f;
      for (int e = 0; e < 64; ++e) x = fmaf(qr[e], kr[h * 64 + e], x);
      s += alpha[a] * expf(x * 0.125f - lse[(int64_t)b * lse_seq + (int64_t)qa * n_heads + h]);
    }
  }
  s_out[(int64_t)b * s_seq + (int64_t)f * n_s + j] = s / (float)n_heads;
}

// ---------------------------------------------------------------------------
// mode B normaliser: partial (max, sum) per key chunk, then combine
// ---------------------------------------------------------------------------
constexpr int LSE_CHUNK = 256;

template <typename T>
__global__ void __launch_bounds__(256)
lse_partial(const T* __restrict__ q, int64_t q_seq, int64_t q_row, const T* __restrict__ k,
            int64_t k_seq, int64_t k_row, int64_t n_keys, int H, int n_heads,
            float* __restrict__ part) {
  // part layout [B][chunks][H][N_h][2]
  __shared__ float qs[64];
  __shared__ float red[2][4];
  const int chunks = (int)((n_keys + LSE_CHUNK - 1) / LSE_CHUNK);
  const int ch = blockIdx.x % chunks;
  const int i = (blockIdx.x / chunks) % H;
  const int b = blockIdx.x / (chunks * H);
  const int h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < 64) qs[tid] = Elem<T>::load(q + b * q_seq + (int64_t)i * q_row + h * 64 + tid);
  __syncthreads();
  const int64_t j = (int64_t)ch * LSE_CHUNK + tid;
  float x = -INFINITY;
  if (j < n_keys) {
    const T* kr = k + b * k_seq + j * k_row + h * 64;
    float acc = 0.0f;
    for (int e = 0; e < 64; ++e) acc = fmaf(qs[e], Elem<T>::load(kr + e), acc);
    x = acc * 0.125f;
  }
  float m = warp_max(x);
  if (lane == 0) red[0][wave] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
  float e = (j < n_keys) ? expf(x - m) : 0.0f;
  e = warp_sum(e);
  if (lane == 0) red[1][wave] = e;
  __syncthreads();
  if (tid == 0) {
    float* p = part + ((((int64_t)b * chunks + ch) * H + i) * n_heads + h) * 2;
    p[0] = m;
    p[1] = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
  }
}

__global__ void lse_combine(const float* __restrict__ part, int chunks, int B, int H,
                            int n_heads, float* __restrict__ lse) {
  const int id = blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= B * H * n_heads) return;
  const int h = id % n_heads, i = (id / n_heads) % H, b = id / (n_heads * H);
  float m = -INFINITY;
  for (int c = 0; c < chunks; ++c)
    m = fmaxf(m, part[((((int64_t)b * chunks + c) * H + i) * n_heads + h) * 2]);
  float s = 0.0f;
  for (int c = 0; c < chunks; ++c) {
    const float* p = part + ((((int64_t)b * chunks + c) * H + i) * n_heads + h) * 2;
    s += p[1] * expf(p[0] - m);
  }
  lse[id] = m + logf(s);
}

hipError_t launch_score(int dtype, const ScoreArgs& a, hipStream_t st) {
  const int nl = a.n_layers < 1 ? 1 : a.n_layers;
  if (dtype == 1) {
    const int ktiles = (a.n_s + 15) / 16;
    hipLaunchKernelGGL(score_bf16, dim3(nl * a.B * a.F * ktiles), dim3(256), 0, st, a);
  } else {
    const int64_t n = (int64_t)nl * a.B * a.F * a.n_s;
    hipLaunchKernelGGL(score_f32, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                       (const float*)a.q, a.q_seq, a.q_row, (const float*)a.k, a.k_seq,
                       a.k_row, a.lse, a.lse_seq, a.s_out, a.s_seq, a.alpha, a.B, a.F, a.n_s,
                       a.H, a.n_heads, nl, a.q_lay, a.k_lay, a.lse_lay, a.s_lay);
  }
  return hipGetLastError();
}

hipError_t launch_lse_all(int dtype, const void* q, int64_t q_seq, int64_t q_row,
                          const void* kall, int64_t k_seq, int64_t k_row, int64_t n_keys,
                          int B, int H, int n_heads, float* lse_out, float* part_ws,
                          hipStream_t st) {
  const int chunks = (int)((n_keys + LSE_CHUNK - 1) / LSE_CHUNK);
  dim3 grid(B * H * chunks, n_heads);
  if (dtype == 1)
    hipLaunchKernelGGL(lse_partial<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)q, q_seq,
                       q_row, (const bf16_t*)kall, k_seq, k_row, n_keys, H, n_heads, part_ws);
  else
    hipLaunchKernelGGL(lse_partial<float>, grid, dim3(256), 0, st, (const float*)q, q_seq,
                       q_row, (const float*)kall, k_seq, k_row, n_keys, H, n_heads, part_ws);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n = B * H * n_heads;
  hipLaunchKernelGGL(lse_combine, dim3((n + 255) / 256), dim3(256), 0, st, part_ws, chunks, B,
                     H, n_heads, lse_out);
  return hipGetLastError();
}

}  // namespace swam
