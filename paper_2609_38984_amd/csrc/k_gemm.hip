// Dense projections of the DiT block: C = epi(A . B^T + bias).
//
// A [M][K] activations and B [N][K] weights are both K-contiguous, so every
// MFMA operand is eight consecutive bf16 of one row.  bf16 path: workgroup
// tile BM x BN x 64, waves arranged WM x WN, each wave a grid of 32x32x16
// MFMA tiles with fp32 accumulators; A/B tiles double-buffered in LDS with a
// 16-byte-chunk XOR swizzle (chunk ^ (row & 7)) so the column reads of the
// MFMA operand layout are spread over all banks.  Workgroup ids are remapped
// so that each XCD (dispatch round-robins over 8) receives a contiguous run
// of tiles, grouped GROUP_M tile-rows deep, to share its L2.
// Epilogues (bias, tanh-GELU, gated residual) are fused into the store.
#include "common.h"

namespace swam {

__device__ __forceinline__ float gelu_tanh(float u) {
  // 0.5 u (1 + tanh(z)) = u / (1 + exp(-2 z)), z = sqrt(2/pi) (u + 0.044715 u^3)
  const float z = 0.7978845608028654f * (u + 0.044715f * u * u * u);
  return u / (1.0f + expf(-2.0f * z));
}

template <int EPI>
__device__ __forceinline__ float epi_value(float acc, float bias, float gate, float resid) {
  if (EPI == EPI_BIAS) return acc + bias;
  if (EPI == EPI_BIAS_GELU) return gelu_tanh(acc + bias);
  return resid + gate * (acc + bias);
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

template <int BM, int BN, int WM, int WN, int EPI>
__global__ void __launch_bounds__(WM * WN * 64)
gemm_bf16_nt(const bf16_t* __restrict__ A, int64_t lda, const bf16_t* __restrict__ B,
             int64_t ldb, const bf16_t* __restrict__ bias, const float* __restrict__ gate,
             bf16_t* C, int64_t ldc, int M, int N, int K, int tiles_m, int tiles_n) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int A_LD = BM * 8 / NT;   // 16-byte chunks per thread per stage
  constexpr int B_LD = BN * 8 / NT;
  static_assert(A_LD * NT == BM * 8 && B_LD * NT == BN * 8, "tile/threads mismatch");
  extern __shared__ uint4 lds[];
  uint4* As = lds;                    // [2][BM*8]
  uint4* Bs = lds + 2 * BM * 8;       // [2][BN*8]

  int tm, tn;
  tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // global -> register staging: thread owns chunk (tid & 7) of rows (tid >> 3) + i * NT / 8
  const int lc = tid & 7, lr = tid >> 3;
  const bf16_t* a_base = A + lc * 8;
  const bf16_t* b_base = B + lc * 8;
  auto a_ptr = [&](int i) {
    return a_base + (int64_t)min(m0 + lr + i * (NT / 8), M - 1) * lda;
  };
  auto b_ptr = [&](int i) {
    return b_base + (int64_t)min(n0 + lr + i * (NT / 8), N - 1) * ldb;
  };
  auto lds_slot = [&](int i) {
    const int row = lr + i * (NT / 8);
    return row * 8 + (lc ^ (row & 7));
  };
  uint4 ra[A_LD], rb[B_LD];

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int KT = K / GEMM_BK;
#pragma unroll
  for (int i = 0; i < A_LD; ++i) ra[i] = *(const uint4*)a_ptr(i);
#pragma unroll
  for (int i = 0; i < B_LD; ++i) rb[i] = *(const uint4*)b_ptr(i);
#pragma unroll
  for (int i = 0; i < A_LD; ++i) As[lds_slot(i)] = ra[i];
#pragma unroll
  for (int i = 0; i < B_LD; ++i) Bs[lds_slot(i)] = rb[i];
  __syncthreads();

  // per-lane operand row offsets inside the stage (rows are fixed per lane)
  int a_row[FM], b_row[FN];
#pragma unroll
  for (int i = 0; i < FM; ++i) a_row[i] = wm * TM + i * 32 + (lane & 31);
#pragma unroll
  for (int j = 0; j < FN; ++j) b_row[j] = wn * TN + j * 32 + (lane & 31);
  const int khalf = lane >> 5;

  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    {
      // prefetch the next stage (the last iteration re-reads a valid stage; unused)
      const int off = min(kt + 1, KT - 1) * GEMM_BK;
#pragma unroll
      for (int i = 0; i < A_LD; ++i) ra[i] = *(const uint4*)(a_ptr(i) + off);
#pragma unroll
      for (int i = 0; i < B_LD; ++i) rb[i] = *(const uint4*)(b_ptr(i) + off);
    }
    const uint4* as = As + cur * BM * 8;
    const uint4* bs = Bs + cur * BN * 8;
#pragma unroll
    for (int s = 0; s < GEMM_BK / 16; ++s) {
      const int chunk = 2 * s + khalf;
      bf16x8 af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        uint4 v = as[a_row[i] * 8 + (chunk ^ (a_row[i] & 7))];
        af[i] = __builtin_bit_cast(bf16x8, v);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        uint4 v = bs[b_row[j] * 8 + (chunk ^ (b_row[j] & 7))];
        bfr[j] = __builtin_bit_cast(bf16x8, v);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    {
      // the other stage was released by the barrier of the previous iteration
      uint4* an = As + (cur ^ 1) * BM * 8;
      uint4* bn = Bs + (cur ^ 1) * BN * 8;
#pragma unroll
      for (int i = 0; i < A_LD; ++i) an[lds_slot(i)] = ra[i];
#pragma unroll
      for (int i = 0; i < B_LD; ++i) bn[lds_slot(i)] = rb[i];
    }
    __syncthreads();
  }

  // epilogue: lane holds column (lane & 31) of rows 8*(r/4) + 4*(lane/32) + r%4
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int col = n0 + wn * TN + j * 32 + (lane & 31);
    if (col >= N) continue;
    const float bv = bf16_to_f32(bias[col]);
    const float gv = (EPI == EPI_BIAS_GATED_RESIDUAL) ? gate[col] : 0.0f;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int rbase = m0 + wm * TM + i * 32 + 4 * (lane >> 5);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = rbase + 8 * (r >> 2) + (r & 3);
        if (row < M) {
          bf16_t* p = C + (int64_t)row * ldc + col;
          const float resid = (EPI == EPI_BIAS_GATED_RESIDUAL) ? bf16_to_f32(*p) : 0.0f;
          *p = f32_to_bf16(epi_value<EPI>(acc[i][j][r], bv, gv, resid));
        }
      }
    }
  }
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
template <int BM, int BN, int WM, int WN, int EPI>
static hipError_t run_bf16(const void* A, int64_t lda, const void* B, int64_t ldb,
                           const void* bias, const float* gate, void* C, int64_t ldc, int M,
                           int N, int K, hipStream_t st) {
  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const size_t lds = (size_t)2 * (BM + BN) * 8 * sizeof(uint4);
  auto kern = gemm_bf16_nt<BM, BN, WM, WN, EPI>;
  static bool attr_set = false;  // per instantiation
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3(tiles_m * tiles_n), dim3(WM * WN * 64), lds, st,
                     (const bf16_t*)A, lda, (const bf16_t*)B, ldb, (const bf16_t*)bias, gate,
                     (bf16_t*)C, ldc, M, N, K, tiles_m, tiles_n);
  return hipGetLastError();
}

// Tile choice: fewest "rounds" of 256 CUs, weighted by per-tile efficiency.
static int choose_tile(int64_t M, int64_t N) {
  static int forced = -2;
  if (forced == -2) {
    const char* e = getenv("SWAM_GEMM_TILE");
    forced = e ? atoi(e) : -1;
  }
  if (forced >= 0 && forced <= 2) return forced;
  struct Cand { int bm, bn; double eff; };
  const Cand c[3] = {{256, 256, 1.0}, {256, 128, 0.85}, {128, 128, 0.7}};
  int best = 0;
  double best_t = 1e30;
  for (int i = 0; i < 3; ++i) {
    if (N % c[i].bn) continue;
    const int64_t tiles = ((M + c[i].bm - 1) / c[i].bm) * ((N + c[i].bn - 1) / c[i].bn);
    const int64_t rounds = (tiles + 255) / 256;
    const double t = (double)rounds * c[i].bm * c[i].bn / c[i].eff;
    if (t < best_t) { best_t = t; best = i; }
  }
  return best;
}

template <int EPI>
static hipError_t dispatch_bf16(const void* A, int64_t lda, const void* B, int64_t ldb,
                                const void* bias, const float* gate, void* C, int64_t ldc,
                                int M, int N, int K, hipStream_t st) {
  switch (choose_tile(M, N)) {
    case 0: return run_bf16<256, 256, 2, 2, EPI>(A, lda, B, ldb, bias, gate, C, ldc, M, N, K, st);
    case 1: return run_bf16<256, 128, 2, 2, EPI>(A, lda, B, ldb, bias, gate, C, ldc, M, N, K, st);
    default: return run_bf16<128, 128, 2, 2, EPI>(A, lda, B, ldb, bias, gate, C, ldc, M, N, K, st);
  }
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

hipError_t launch_gemm(int dtype, int epi, const void* A, int64_t lda, const void* B,
                       int64_t ldb, const void* bias, const float* gate, void* C,
                       int64_t ldc, int64_t M, int64_t N, int64_t K, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  const int m = (int)M, n = (int)N, k = (int)K;
  if (dtype == 1) {
    switch (epi) {
      case EPI_BIAS: return dispatch_bf16<EPI_BIAS>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, st);
      case EPI_BIAS_GELU: return dispatch_bf16<EPI_BIAS_GELU>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, st);
      default: return dispatch_bf16<EPI_BIAS_GATED_RESIDUAL>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, st);
    }
  }
  switch (epi) {
    case EPI_BIAS: return run_f32<EPI_BIAS>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, st);
    case EPI_BIAS_GELU: return run_f32<EPI_BIAS_GELU>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, st);
    default: return run_f32<EPI_BIAS_GATED_RESIDUAL>(A, lda, B, ldb, bias, gate, C, ldc, m, n, k, st);
  }
}

}  // namespace swam
