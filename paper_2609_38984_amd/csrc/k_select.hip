// Score reduction, selection, packing metadata, pack and unpack.
//
// Reduction (layer quality, core layers, core score V, anchor key A) sums in
// float64 in a fixed order and rounds once to float32.
// Selection orders positions by the composite key
//   key = (~ord(score) << 32) | index
// where ord() maps float bits to an order-preserving uint32 (signed zeros
// merged), so ascending keys are score-descending with the lowest index first
// on ties: every top-k is deterministic and bit-exact.  Fixed budgets take
// the first k keys by a radix select (8-bit digit histograms of ~ord in LDS,
// ties at the k-th value resolved lowest index first); the mass threshold,
// which walks the pool in that order, sorts the keys in LDS with a bitonic
// network and counts with exact integer codes floor(V 2^40) and a uint64
// prefix scan.
// Packing is an exclusive prefix sum of keep flags in original token order;
// pack is a coalesced 16-byte row gather, unpack the matching scatter.
#include "launchers.h"

namespace swam {

constexpr int SEL_THREADS = 1024;
constexpr int MASS_BITS = 40;

// ---------------------------------------------------------------------------
// block-wide helpers (blockDim.x == SEL_THREADS or 256)
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t float_order(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) == 0) u = 0;                  // -0 == +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ uint64_t sel_key(float score, int idx) {
  return ((uint64_t)(~float_order(score)) << 32) | (uint32_t)idx;
}

__device__ void bitonic_sort(uint64_t* s, int np) {
  for (int k = 2; k <= np; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < np; i += blockDim.x) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const uint64_t a = s[i], b = s[ixj];
          const bool up = (i & k) == 0;
          if ((a > b) == up) { s[i] = b; s[ixj] = a; }
        }
      }
      __syncthreads();
    }
  }
}

// exclusive scan of one int per thread; returns the exclusive prefix, *total
__device__ int block_excl_scan(int v, int* ws /* >= 32 ints */, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) ws[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < nw; ++w) { const int t = ws[w]; ws[w] = run; run += t; }
    ws[nw] = run;
  }
  __syncthreads();
  const int res = ws[wave] + x - v;
  *total = ws[nw];
  __syncthreads();
  return res;
}

__device__ uint64_t block_excl_scan_u64(uint64_t v, uint64_t* ws, uint64_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  uint64_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) ws[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t run = 0;
    for (int w = 0; w < nw; ++w) { const uint64_t t = ws[w]; ws[w] = run; run += t; }
    ws[nw] = run;
  }
  __syncthreads();
  const uint64_t res = ws[wave] + x - v;
  *total = ws[nw];
  __syncthreads();
  return res;
}

__device__ __forceinline__ int next_pow2(int n) {
  int p = 1;
  while (p < n) p <<= 1;
  return p;
}

// ---------------------------------------------------------------------------
// block-wide top-k by radix select (blockDim.x == SEL_THREADS)
// ---------------------------------------------------------------------------
constexpr int SEL_EPT = SWAM_SEL_MAXNP / SEL_THREADS;   // positions per thread

struct SelScratch {
  uint32_t hist[256];
  int ws[SEL_THREADS / 64 + 1];
  int pick[2];
};

// Thread t owns positions [t * SEL_EPT, (t + 1) * SEL_EPT).  Among the
// candidate positions, sel[] marks the k that come first in the order (ok
// ascending, then position ascending), where ok = ~float_order(score) puts
// higher scores first: the same set as sorting the composite keys
// (ok << 32 | j) and taking the first k.  Four passes of 8-bit digit
// histograms (LDS atomics) narrow down the ok value of the k-th key; its
// ties are then taken lowest position first by an exclusive scan in
// position order.
__device__ void block_topk(const uint32_t (&ok)[SEL_EPT], const bool (&cand)[SEL_EPT], int k,
                           bool (&sel)[SEL_EPT], SelScratch& sc) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int mine = 0;
#pragma unroll
  for (int e = 0; e < SEL_EPT; ++e) mine += cand[e];
  int total;
  block_excl_scan(mine, sc.ws, &total);
  if (k >= total || k <= 0) {
#pragma unroll
    for (int e = 0; e < SEL_EPT; ++e) sel[e] = k > 0 && cand[e];
    return;
  }
  uint32_t prefix = 0, pmask = 0;
  int need = k;                                 // keys still to take at or after `prefix`
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += blockDim.x) sc.hist[i] = 0;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < SEL_EPT; ++e)
      if (cand[e] && (ok[e] & pmask) == prefix) atomicAdd(&sc.hist[(ok[e] >> shift) & 255u], 1u);
    __syncthreads();
    if (wave == 0) {
      // the digit bucket that holds the need-th key: scan of the 256 counts
      uint32_t c[4], s = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) { c[q] = sc.hist[4 * lane + q]; s += c[q]; }
      uint32_t x = s;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(x, o);
        if (lane >= o) x += y;
      }
      const uint32_t before = x - s;
      if (before < (uint32_t)need && (uint32_t)need <= x) {
        uint32_t run = before;
        int q = 0;
        while (run + c[q] < (uint32_t)need) run += c[q++];
        sc.pick[0] = 4 * lane + q;
        sc.pick[1] = (int)run;
      }
    }
    __syncthreads();
    prefix |= (uint32_t)sc.pick[0] << shift;
    pmask |= 255u << shift;
    need -= sc.pick[1];
    __syncthreads();                            // pick is rewritten by the next pass
  }
  // prefix is now the k-th key's ok value; take `need` of its ties
  int t = 0;
#pragma unroll
  for (int e = 0; e < SEL_EPT; ++e) t += cand[e] && ok[e] == prefix;
  int tt;
  int rank = block_excl_scan(t, sc.ws, &tt);
#pragma unroll
  for (int e = 0; e < SEL_EPT; ++e) {
    const bool tie = cand[e] && ok[e] == prefix;
    sel[e] = cand[e] && (ok[e] < prefix || (tie && rank < need));
    rank += tie;
  }
}

// ---------------------------------------------------------------------------
// score reduction
// ---------------------------------------------------------------------------
// one block per (b, l, f): frame mass and entropy term (float64)
__global__ void __launch_bounds__(256)
reduce_frames(const float* __restrict__ s_all, int n_s, double* __restrict__ fsum,
              double* __restrict__ fent) {
  __shared__ double red[4];
  const float* row = s_all + (int64_t)blockIdx.x * n_s;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  double acc = 0.0;
  for (int j = threadIdx.x; j < n_s; j += 256) acc += (double)row[j];
  acc = warp_sum_d(acc);
  if (lane == 0) red[wave] = acc;
  __syncthreads();
  const double tot = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  double ent = 0.0;
  if (tot != 0.0) {
    for (int j = threadIdx.x; j < n_s; j += 256) {
      const double p = (double)row[j] / tot;
      if (p > 0.0) ent -= p * log(p);
    }
  }
  ent = warp_sum_d(ent);
  if (lane == 0) red[wave] = ent;
  __syncthreads();
  if (threadIdx.x == 0) {
    fsum[blockIdx.x] = tot;
    fent[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
  }
}

// one block (64 threads) per b: Q_l, core layers, weight sums
__global__ void __launch_bounds__(64)
reduce_layers(const double* __restrict__ fsum, const double* __restrict__ fent, int L, int F,
              int n_s, int k_eff, float* __restrict__ q_out, double* __restrict__ qd,
              int32_t* __restrict__ core, double* __restrict__ dens) {
  __shared__ float q32[64];
  __shared__ double qv[64];
  __shared__ int flag[64];
  const int b = blockIdx.x, l = threadIdx.x;
  if (l < L) {
    double tot = 0.0, ent = 0.0;
    for (int f = 0; f < F; ++f) {
      tot += fsum[((int64_t)b * L + l) * F + f];
      ent += fent[((int64_t)b * L + l) * F + f];
    }
    const double R = tot / F;
    const double E = ent / (F * log((double)n_s));
    const double Q = R * (1.0 - E);
    qv[l] = Q;
    q32[l] = (float)Q;
    qd[b * L + l] = Q;
    q_out[b * L + l] = (float)Q;
  }
  __syncthreads();
  if (l < L) {
    int rank = 0;
    for (int m = 0; m < L; ++m)
      rank += (q32[m] > q32[l]) || (q32[m] == q32[l] && m < l);
    flag[l] = rank < k_eff;
  }
  __syncthreads();
  if (l == 0) {
    int n = 0;
    double dc = 0.0, da = 0.0;
    for (int m = 0; m < L; ++m) {
      if (flag[m]) { core[b * k_eff + n++] = m; dc += qv[m]; }
      da += qv[m];
    }
    dens[2 * b] = dc;
    dens[2 * b + 1] = da;
  }
}

// one thread per (b, f, j): V over the core layers and V_all over all layers
// (float64 sums in layer order; V stored as float32, V_all kept in float64)
__global__ void __launch_bounds__(256)
reduce_positions(const float* __restrict__ s_all, const double* __restrict__ qd,
                 const int32_t* __restrict__ core, const double* __restrict__ dens, int L,
                 int F, int n_s, int k_eff, float* __restrict__ v_out,
                 double* __restrict__ vall) {
  const int bf = blockIdx.y;                 // b * F + f
  const int b = bf / F, f = bf - b * F;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= n_s) return;
  const double dc = dens[2 * b], da = dens[2 * b + 1];
  const float* sb = s_all + (int64_t)b * L * F * n_s + (int64_t)f * n_s + j;
  const int64_t ls = (int64_t)F * n_s;       // layer stride
  const double* q = qd + (int64_t)b * L;
  const int32_t* cl = core + b * k_eff;
  double acc = 0.0;
  if (dc != 0.0) {
    for (int c = 0; c < k_eff; ++c) {
      const int l = cl[c];
      acc += q[l] * (double)sb[l * ls];
    }
    acc /= dc;
  } else {
    for (int c = 0; c < k_eff; ++c) acc += (double)sb[cl[c] * ls];
    acc /= k_eff;
  }
  v_out[(int64_t)bf * n_s + j] = (float)acc;
  double all = 0.0;
  if (da != 0.0) {
    for (int l = 0; l < L; ++l) all += q[l] * (double)sb[l * ls];
    all /= da;
  } else {
    for (int l = 0; l < L; ++l) all += (double)sb[l * ls];
    all /= L;
  }
  vall[(int64_t)bf * n_s + j] = all;
}

// one thread per (b, j): mean and population std of V_all over frames, anchor key
__global__ void __launch_bounds__(256)
reduce_anchor(const double* __restrict__ vall, int F, int n_s, float cv, float* __restrict__ a_out) {
  const int b = blockIdx.y;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= n_s) return;
  const double* vb = vall + (int64_t)b * F * n_s + j;
  double mu = 0.0;
  for (int f = 0; f < F; ++f) mu += vb[(int64_t)f * n_s];
  mu /= F;
  double var = 0.0;
  for (int f = 0; f < F; ++f) {
    const double dv = vb[(int64_t)f * n_s] - mu;
    var += dv * dv;
  }
  const double sd = sqrt(var / F);
  a_out[(int64_t)b * n_s + j] = mu != 0.0 ? (float)(mu / (1.0 + (double)cv * (sd / mu))) : 0.0f;
}

// Overlap(P, Q) = sum_i min(P_i / sum P, Q_i / sum Q) per map (App. C
// attention-overlap eq.); one workgroup per map, float64 sums in a fixed
// order (per-thread strided partials, then a tree over the workgroup)
__device__ __forceinline__ double block_sum_d(double v, double* red) {
  v = warp_sum_d(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  double t = 0.0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += red[i];
  return t;
}

__global__ void __launch_bounds__(256)
overlap_kernel(const float* __restrict__ p, const float* __restrict__ q, int64_t n,
               float* __restrict__ out) {
  __shared__ double red[4];
  const float* pm = p + (int64_t)blockIdx.x * n;
  const float* qm = q + (int64_t)blockIdx.x * n;
  double sp = 0.0, sq = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
    sp += (double)pm[i];
    sq += (double)qm[i];
  }
  sp = block_sum_d(sp, red);
  sq = block_sum_d(sq, red);
  double acc = 0.0;
  if (sp > 0.0 && sq > 0.0)
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x)
      acc += fmin((double)pm[i] / sp, (double)qm[i] / sq);
  acc = block_sum_d(acc, red);
  if (threadIdx.x == 0) out[blockIdx.x] = (float)acc;
}

hipError_t launch_overlap(const float* p, const float* q, int64_t n_maps, int64_t n,
                          float* out, hipStream_t st) {
  if (n_maps <= 0) return hipSuccess;
  hipLaunchKernelGGL(overlap_kernel, dim3((unsigned)n_maps), dim3(256), 0, st, p, q, n, out);
  return hipGetLastError();
}

hipError_t launch_score_reduce(const ReduceArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(reduce_frames, dim3(a.B * a.L * a.F), dim3(256), 0, st, a.s_all, a.n_s,
                     a.frame_sum, a.frame_ent);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int k_eff = a.k_layer < a.L ? a.k_layer : a.L;
  double* dens = a.frame_sum + (int64_t)a.B * a.L * a.F;   // 2B doubles after the frame sums
  hipLaunchKernelGGL(reduce_layers, dim3(a.B), dim3(64), 0, st, a.frame_sum, a.frame_ent, a.L,
                     a.F, a.n_s, k_eff, a.q, a.qd, a.core, dens);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(reduce_positions, dim3((a.n_s + 255) / 256, a.B * a.F), dim3(256), 0, st,
                     a.s_all, a.qd, a.core, dens, a.L, a.F, a.n_s, k_eff, a.v, a.vall);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(reduce_anchor, dim3((a.n_s + 255) / 256, a.B), dim3(256), 0, st, a.vall,
                     a.F, a.n_s, a.cv_penalty, a.a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// selection
// ---------------------------------------------------------------------------
// pool: top (N_s - K_s) of max_f V(f, j); one block per b
__global__ void __launch_bounds__(SEL_THREADS)
select_pool(const float* __restrict__ v, int F, int n_s, int k_anchor,
            uint8_t* __restrict__ pool) {
  __shared__ SelScratch sc;
  const int b = blockIdx.x;
  const float* vb = v + (int64_t)b * F * n_s;
  uint32_t ok[SEL_EPT];
  bool cand[SEL_EPT], sel[SEL_EPT];
  const int j0 = threadIdx.x * SEL_EPT;
#pragma unroll
  for (int e = 0; e < SEL_EPT; ++e) {
    const int j = j0 + e;
    cand[e] = j < n_s;
    ok[e] = ~0u;
    if (cand[e]) {
      float m = vb[j];
      for (int f = 1; f < F; ++f) m = fmaxf(m, vb[(int64_t)f * n_s + j]);
      ok[e] = ~float_order(m);
    }
  }
  block_topk(ok, cand, n_s - k_anchor, sel, sc);
#pragma unroll
  for (int e = 0; e < SEL_EPT; ++e)
    if (j0 + e < n_s) pool[(int64_t)b * n_s + j0 + e] = sel[e];
}

__device__ __forceinline__ uint64_t mass_code(float x) {
  if (!(x > 0.0f)) return 0;
  if (x >= 1.0f) return 1ull << MASS_BITS;
  const uint32_t u = __float_as_uint(x);
  const int ex = (int)((u >> 23) & 0xFF);
  const uint64_t man = ex ? ((u & 0x7FFFFFu) | 0x800000u) : (u & 0x7FFFFFu);
  // x = man * 2^(e - 150) (normal) or man * 2^-149 (subnormal)
  const int sh = (ex ? ex - 150 : -149) + MASS_BITS;
  if (sh >= 0) return man << sh;
  if (sh <= -64) return 0;
  return man >> (-sh);
}

// cores: per (b, f), top K_c (or the mass-threshold count) of V(f, .) in P
__global__ void __launch_bounds__(SEL_THREADS)
select_core(const float* __restrict__ v, const uint8_t* __restrict__ pool, int F, int n_s,
            int k_core, int k_anchor, int mass_num, int mass_den, uint8_t* __restrict__ core,
            int32_t* __restrict__ kcount) {
  __shared__ uint64_t keys[SWAM_SEL_MAXNP];
  __shared__ uint64_t ws64[SEL_THREADS / 64 + 1];
  __shared__ int fails;
  __shared__ SelScratch sc;
  const int bf = blockIdx.x;               // b * F + f
  const int b = bf / F;
  const int np = next_pow2(n_s);
  const float* vr = v + (int64_t)bf * n_s;
  const uint8_t* pb = pool + (int64_t)b * n_s;
  uint8_t* cr = core + (int64_t)bf * n_s;
  if (mass_den == 0) {
    // fixed budget: the top K_c of the pool by radix select
    uint32_t ok[SEL_EPT];
    bool cand[SEL_EPT], sel[SEL_EPT];
    const int j0 = threadIdx.x * SEL_EPT;
#pragma unroll
    for (int e = 0; e < SEL_EPT; ++e) {
      const int j = j0 + e;
      cand[e] = j < n_s && pb[j];
      ok[e] = cand[e] ? ~float_order(vr[j]) : ~0u;
    }
    block_topk(ok, cand, k_core, sel, sc);
#pragma unroll
    for (int e = 0; e < SEL_EPT; ++e)
      if (j0 + e < n_s) cr[j0 + e] = sel[e];
    if (threadIdx.x == 0) kcount[bf] = min(k_core, n_s - k_anchor);
    return;
  }
  // mass threshold: the pool in TopK order (full sort), walked with the codes
  for (int j = threadIdx.x; j < np; j += blockDim.x) {
    uint64_t key = ~0ull;
    if (j < n_s) {
      if (pb[j]) key = sel_key(vr[j], j);
      cr[j] = 0;
    }
    keys[j] = key;
  }
  if (threadIdx.x == 0) fails = 0;
  __syncthreads();
  bitonic_sort(keys, np);
  const int psize = n_s - k_anchor;
  int kc = k_core;
  if (mass_den > 0) {
    // T = sum of codes over every position of the frame
    uint64_t part = 0;
    for (int j = threadIdx.x; j < n_s; j += blockDim.x) part += mass_code(vr[j]);
    uint64_t T;
    block_excl_scan_u64(part, ws64, &T);
    // inclusive prefix of codes in ranked order; each thread owns a contiguous run
    const int ept = (psize + blockDim.x - 1) / blockDim.x;
    const int r0 = threadIdx.x * ept;
    uint64_t local = 0;
    for (int r = r0; r < min(r0 + ept, psize); ++r)
      local += mass_code(vr[(int)(keys[r] & 0xFFFFFFFFu)]);
    uint64_t tot;
    uint64_t run = block_excl_scan_u64(local, ws64, &tot);
    int nf = 0;
    for (int r = r0; r < min(r0 + ept, psize); ++r) {
      run += mass_code(vr[(int)(keys[r] & 0xFFFFFFFFu)]);
      nf += ((uint64_t)mass_den * run < (uint64_t)mass_num * T);
    }
    if (nf) atomicAdd(&fails, nf);
    __syncthreads();
    kc = min(1 + fails, psize);
  }
  for (int r = threadIdx.x; r < kc; r += blockDim.x) cr[(int)(keys[r] & 0xFFFFFFFFu)] = 1;
  if (threadIdx.x == 0) kcount[bf] = kc;
}

// anchors + retained sets + keep flags; one block per b
__global__ void __launch_bounds__(SEL_THREADS)
select_anchor(const float* __restrict__ a, const uint8_t* __restrict__ core, int F, int n_s,
              int k_anchor, int k_max, int n_ctx, int n_act, int64_t l_full,
              int32_t* __restrict__ keep_idx, int32_t* __restrict__ keep_cnt,
              int32_t* __restrict__ keep) {
  __shared__ SelScratch sc;
  __shared__ uint8_t anchor[SWAM_MAX_NS_DEV];
  const int b = blockIdx.x;
  const uint8_t* cb = core + (int64_t)b * F * n_s;
  {
    // anchors: the top K_s of A over the positions no frame's core took
    uint32_t ok[SEL_EPT];
    bool cand[SEL_EPT], sel[SEL_EPT];
    const int j0 = threadIdx.x * SEL_EPT;
#pragma unroll
    for (int e = 0; e < SEL_EPT; ++e) {
      const int j = j0 + e;
      bool used = j >= n_s;
      for (int f = 0; f < F && !used; ++f) used |= cb[(int64_t)f * n_s + j] != 0;
      cand[e] = !used;
      ok[e] = cand[e] ? ~float_order(a[(int64_t)b * n_s + j]) : ~0u;
    }
    block_topk(ok, cand, k_anchor, sel, sc);
#pragma unroll
    for (int e = 0; e < SEL_EPT; ++e)
      if (j0 + e < n_s) anchor[j0 + e] = sel[e];
  }
  __syncthreads();
  int32_t* kb = keep + (int64_t)b * l_full;
  for (int64_t t = threadIdx.x; t < n_ctx; t += blockDim.x) kb[t] = 1;
  for (int64_t t = threadIdx.x; t < n_act; t += blockDim.x) kb[l_full - n_act + t] = 1;
  // retained set of each frame (core or anchor), in position order: one wave
  // per frame, 64 positions per round compacted by ballot + lane prefix count
  const int lane = threadIdx.x & 63, nw = blockDim.x >> 6;
  for (int f = threadIdx.x >> 6; f < F; f += nw) {
    const uint8_t* cf = cb + (int64_t)f * n_s;
    int32_t* out = keep_idx + ((int64_t)b * F + f) * k_max;
    int32_t* kf_out = kb + n_ctx + (int64_t)f * n_s;
    int total = 0;
    for (int j0 = 0; j0 < n_s; j0 += 64) {
      const int j = j0 + lane;
      const bool kf = j < n_s && (cf[j] | anchor[j]) != 0;
      if (j < n_s) kf_out[j] = kf;
      const uint64_t bal = __ballot(kf);
      if (kf) out[total + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                  __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u))] = j;
      total += __popcll(bal);
    }
    for (int r = total + lane; r < k_max; r += 64) out[r] = -1;
    if (lane == 0) keep_cnt[b * F + f] = total;
  }
}

hipError_t launch_select(const SelectArgs& s, hipStream_t st) {
  const int64_t l_full = s.n_ctx + (int64_t)s.F * s.n_s + s.n_act;
  hipLaunchKernelGGL(select_pool, dim3(s.B), dim3(SEL_THREADS), 0, st, s.v, s.F, s.n_s,
                     s.k_anchor, s.pool);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(select_core, dim3(s.B * s.F), dim3(SEL_THREADS), 0, st, s.v, s.pool, s.F,
                     s.n_s, s.k_core, s.k_anchor, s.mass_num, s.mass_den, s.core, s.keep_cnt);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(select_anchor, dim3(s.B), dim3(SEL_THREADS), 0, st, s.a, s.core, s.F,
                     s.n_s, s.k_anchor, s.k_max, s.n_ctx, s.n_act, l_full, s.keep_idx,
                     s.keep_cnt, s.keep);
  return hipGetLastError();
}

// imported selection -> keep flags, normalised keep_idx / keep_cnt (ascending, deduplicated)
__global__ void __launch_bounds__(SEL_THREADS)
keep_from_idx(const int32_t* __restrict__ in_idx, int32_t* __restrict__ keep_idx,
              int32_t* __restrict__ keep_cnt, int32_t* __restrict__ keep, int F, int n_s,
              int k_max, int n_ctx, int n_act, int64_t l_full) {
  __shared__ uint8_t flag[SWAM_MAX_NS_DEV];
  __shared__ int ws[SEL_THREADS / 64 + 1];
  const int b = blockIdx.x;
  int32_t* kb = keep + (int64_t)b * l_full;
  for (int64_t t = threadIdx.x; t < n_ctx; t += blockDim.x) kb[t] = 1;
  for (int64_t t = threadIdx.x; t < n_act; t += blockDim.x) kb[l_full - n_act + t] = 1;
  const int ept = (n_s + blockDim.x - 1) / blockDim.x;
  for (int f = 0; f < F; ++f) {
    for (int j = threadIdx.x; j < n_s; j += blockDim.x) flag[j] = 0;
    __syncthreads();
    const int32_t* src = in_idx + ((int64_t)b * F + f) * k_max;
    for (int r = threadIdx.x; r < k_max; r += blockDim.x) {
      const int j = src[r];
      if (j >= 0 && j < n_s) flag[j] = 1;
    }
    __syncthreads();
    const int j0 = threadIdx.x * ept;
    int cnt = 0;
    for (int j = j0; j < min(j0 + ept, n_s); ++j) cnt += flag[j];
    int total;
    int pos = block_excl_scan(cnt, ws, &total);
    int32_t* out = keep_idx + ((int64_t)b * F + f) * k_max;
    for (int j = j0; j < min(j0 + ept, n_s); ++j) {
      kb[n_ctx + (int64_t)f * n_s + j] = flag[j];
      if (flag[j]) out[pos++] = j;
    }
    for (int r = total + threadIdx.x; r < k_max; r += blockDim.x) out[r] = -1;
    if (threadIdx.x == 0) keep_cnt[b * F + f] = total;
    __syncthreads();
  }
}

hipError_t launch_keep_from_idx(const int32_t* in_idx, int32_t* keep_idx, int32_t* keep_cnt,
                                int32_t* keep, int B, int F, int n_s, int k_max, int n_ctx,
                                int n_act, hipStream_t st) {
  const int64_t l_full = n_ctx + (int64_t)F * n_s + n_act;
  hipLaunchKernelGGL(keep_from_idx, dim3(B), dim3(SEL_THREADS), 0, st, in_idx, keep_idx,
                     keep_cnt, keep, F, n_s, k_max, n_ctx, n_act, l_full);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// pack map: one block scans all B * L_full flags in original order
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(SEL_THREADS)
packmap_kernel(const int32_t* __restrict__ keep, int32_t* __restrict__ pack_pos,
               int32_t* __restrict__ gather, int32_t* __restrict__ cu, int B, int64_t l_full) {
  __shared__ int ws[SEL_THREADS / 64 + 1];
  const int64_t n = (int64_t)B * l_full;
  const int64_t ept = (n + blockDim.x - 1) / blockDim.x;
  const int64_t t0 = threadIdx.x * ept;
  const int64_t t1 = t0 + ept < n ? t0 + ept : n;
  int cnt = 0;
  for (int64_t t = t0; t < t1; ++t) cnt += keep[t] != 0;
  int total;
  int pos = block_excl_scan(cnt, ws, &total);
  for (int64_t t = t0; t < t1; ++t) {
    if (t % l_full == 0) cu[t / l_full] = pos;
    if (keep[t]) {
      pack_pos[t] = pos;
      gather[pos] = (int32_t)t;
      ++pos;
    } else {
      pack_pos[t] = -1;
    }
  }
  if (threadIdx.x == 0) cu[B] = total;
}

hipError_t launch_packmap(const int32_t* keep, int32_t* pack_pos, int32_t* gather,
                          int32_t* cu, int B, int64_t l_full, hipStream_t st) {
  hipLaunchKernelGGL(packmap_kernel, dim3(1), dim3(SEL_THREADS), 0, st, keep, pack_pos, gather,
                     cu, B, l_full);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// pack / unpack / copy: 16-byte chunks, one row per 64 x 16 B slice
// ---------------------------------------------------------------------------
// Row copies of pack / unpack: each wave moves ROWS rows (their source or
// target indices wave-uniform and read up front), every lane loading its
// 16-byte chunks of all of them before storing any, so one wave keeps
// ROWS x ceil(chunks / 64) x 16 B per lane in flight; four waves per
// 256-thread workgroup.  The copies are a few to a few tens of MB: what
// bounds them is how much is in flight, not the bandwidth.
constexpr int COPY_ROWS = 2;     // rows per wave
constexpr int COPY_CH = 4;       // 16-byte chunks per lane and row in flight per pass (4 KB rows)

// The row map gives the source and destination row pointers of row r.  Loads
// are unconditional (a row past the end repeats the last row, a chunk past
// the row end repeats the last chunk: always in bounds) so they all issue
// before the first store; only the stores are predicated.
template <typename RowMap>
__device__ __forceinline__ void copy_rows(const uint4* __restrict__ src_a,
                                          const uint4* __restrict__ src_b, uint4* __restrict__ dst,
                                          int64_t rows, int cpr, RowMap map) {
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int64_t r0 = ((int64_t)blockIdx.x * 4 + wave) * COPY_ROWS;
  if (r0 >= rows) return;
  const int lane = threadIdx.x & 63;
  const uint4* sp[COPY_ROWS];
  uint4* dp[COPY_ROWS];
#pragma unroll
  for (int i = 0; i < COPY_ROWS; ++i) map(min(r0 + i, rows - 1), src_a, src_b, dst, cpr, sp[i], dp[i]);
  for (int base = 0; base < cpr; base += 64 * COPY_CH) {
    const int c0 = base + lane;
    uint4 v[COPY_ROWS][COPY_CH];
#pragma unroll
    for (int i = 0; i < COPY_ROWS; ++i)
#pragma unroll
      for (int k = 0; k < COPY_CH; ++k) v[i][k] = sp[i][min(c0 + 64 * k, cpr - 1)];
    // keep every load ahead of the predicated stores (the compiler would
    // otherwise sink each load into its store's branch, one round trip each)
#pragma unroll
    for (int i = 0; i < COPY_ROWS; ++i)
#pragma unroll
      for (int k = 0; k < COPY_CH; ++k) {
        typedef int i32x4 __attribute__((ext_vector_type(4)));
        asm volatile("" ::"v"(__builtin_bit_cast(i32x4, v[i][k])));
      }
#pragma unroll
    for (int i = 0; i < COPY_ROWS; ++i)
#pragma unroll
      for (int k = 0; k < COPY_CH; ++k)
        if (r0 + i < rows && dp[i] && c0 + 64 * k < cpr) dp[i][c0 + 64 * k] = v[i][k];
  }
}

__global__ void __launch_bounds__(256)
pack_rows(const uint4* __restrict__ src, uint4* __restrict__ dst,
          const int32_t* __restrict__ gather, int64_t rows, int cpr) {
  copy_rows(src, nullptr, dst, rows, cpr,
            [gather](int64_t r, const uint4* a, const uint4*, uint4* d, int cpr_,
                     const uint4*& s_, uint4*& d_) {
              s_ = a + (int64_t)gather[r] * cpr_;
              d_ = d + r * cpr_;
            });
}

__global__ void __launch_bounds__(256)
unpack_scatter(const uint4* __restrict__ src, uint4* __restrict__ dst,
               const int32_t* __restrict__ gather, int64_t rows, int cpr) {
  copy_rows(src, nullptr, dst, rows, cpr,
            [gather](int64_t r, const uint4* a, const uint4*, uint4* d, int cpr_,
                     const uint4*& s_, uint4*& d_) {
              s_ = a + r * cpr_;
              d_ = d + (int64_t)gather[r] * cpr_;
            });
}

// y row r = packed row pack_pos[r] if retained, else x row r
__global__ void __launch_bounds__(256)
unpack_merge(const uint4* __restrict__ yp, const uint4* __restrict__ x, uint4* __restrict__ y,
             const int32_t* __restrict__ pack_pos, int64_t rows, int cpr) {
  copy_rows(yp, x, y, rows, cpr,
            [pack_pos](int64_t r, const uint4* a, const uint4* b, uint4* d, int cpr_,
                       const uint4*& s_, uint4*& d_) {
              const int32_t p = pack_pos[r];
              s_ = p >= 0 ? a + (int64_t)p * cpr_ : b + r * cpr_;
              d_ = d + r * cpr_;
            });
}

// y row r = x row r for the pruned rows (pack_pos[r] < 0) only
__global__ void __launch_bounds__(256)
copy_pruned_rows(const uint4* __restrict__ x, uint4* __restrict__ y,
                 const int32_t* __restrict__ pack_pos, int64_t rows, int cpr) {
  copy_rows(x, nullptr, y, rows, cpr,
            [pack_pos](int64_t r, const uint4* a, const uint4*, uint4* d, int cpr_,
                       const uint4*& s_, uint4*& d_) {
              // a retained row is loaded (in bounds) but not stored: its output
              // row comes from the scatter of the packed rows
              s_ = a + r * cpr_;
              d_ = pack_pos[r] < 0 ? d + r * cpr_ : nullptr;
            });
}

__global__ void __launch_bounds__(256)
copy_chunks(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    dst[i] = src[i];
}

static unsigned grid_for(int64_t chunks) {
  int64_t g = (chunks + 255) / 256;
  if (g > 8192) g = 8192;
  return (unsigned)(g < 1 ? 1 : g);
}

hipError_t launch_pack(const void* x_full, void* x_packed, const int32_t* gather, int64_t rows,
                       int64_t row_bytes, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const int cpr = (int)(row_bytes / 16);
  hipLaunchKernelGGL(pack_rows, dim3((unsigned)((rows + 4 * COPY_ROWS - 1) / (4 * COPY_ROWS))), dim3(256), 0, st,
                     (const uint4*)x_full, (uint4*)x_packed, gather, rows, cpr);
  return hipGetLastError();
}

hipError_t launch_unpack_scatter(const void* y_packed, void* y_full, const int32_t* gather,
                                 int64_t rows, int64_t row_bytes, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const int cpr = (int)(row_bytes / 16);
  hipLaunchKernelGGL(unpack_scatter, dim3((unsigned)((rows + 4 * COPY_ROWS - 1) / (4 * COPY_ROWS))), dim3(256), 0, st,
                     (const uint4*)y_packed, (uint4*)y_full, gather, rows, cpr);
  return hipGetLastError();
}

hipError_t launch_unpack_merge(const void* y_packed, const void* x_full, void* y_full,
                               const int32_t* pack_pos, int64_t rows, int64_t row_bytes,
                               hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const int cpr = (int)(row_bytes / 16);
  hipLaunchKernelGGL(unpack_merge, dim3((unsigned)((rows + 4 * COPY_ROWS - 1) / (4 * COPY_ROWS))), dim3(256), 0, st,
                     (const uint4*)y_packed, (const uint4*)x_full, (uint4*)y_full, pack_pos,
                     rows, cpr);
  return hipGetLastError();
}

hipError_t launch_copy_pruned(const void* x_full, void* y_full, const int32_t* pack_pos,
                              int64_t rows, int64_t row_bytes, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const int cpr = (int)(row_bytes / 16);
  hipLaunchKernelGGL(copy_pruned_rows, dim3((unsigned)((rows + 4 * COPY_ROWS - 1) / (4 * COPY_ROWS))),
                     dim3(256), 0, st, (const uint4*)x_full, (uint4*)y_full, pack_pos, rows, cpr);
  return hipGetLastError();
}

hipError_t launch_copy(const void* src, void* dst, int64_t bytes, hipStream_t st) {
  if (bytes <= 0 || src == dst) return hipSuccess;
  const int64_t n = bytes / 16;
  hipLaunchKernelGGL(copy_chunks, dim3(grid_for(n)), dim3(256), 0, st, (const uint4*)src,
                     (uint4*)dst, n);
  return hipGetLastError();
}

// Random-selection baseline: one Philox4x64-10 evaluation (Salmon et al.,
// SC 2011: ten rounds of two 64x64 -> 128-bit products crossed with the other
// two words and a Weyl-stepped key) per (sequence, frame, position); the
// selection then takes the largest keys per frame.  The same threads clear
// the n_a anchor keys (n_a <= n), so every anchor ties at zero.
__global__ void __launch_bounds__(256)
random_keys_kernel(float* __restrict__ v, int64_t n, float* __restrict__ a, int64_t n_a,
                   uint64_t seed) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= n) return;
  if (id < n_a) a[id] = 0.0f;
  uint64_t x0 = (uint64_t)id, x1 = 0, x2 = 0, x3 = 0, k0 = seed, k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t lo0 = 0xD2E7470EE14C6C93ull * x0, hi0 = __umul64hi(0xD2E7470EE14C6C93ull, x0);
    const uint64_t lo1 = 0xCA5A826395121157ull * x2, hi1 = __umul64hi(0xCA5A826395121157ull, x2);
    x0 = hi1 ^ x1 ^ k0;
    x1 = lo1;
    x2 = hi0 ^ x3 ^ k1;
    x3 = lo0;
    k0 += 0x9E3779B97F4A7C15ull;
    k1 += 0xBB67AE8584CAA73Bull;
  }
  v[id] = (float)(uint32_t)(x0 >> 40) * 0x1p-24f;
}

hipError_t launch_random_keys(float* v, int64_t n, float* a, int64_t n_a, uint64_t seed,
                              hipStream_t st) {
  if (n <= 0 || n_a > n) return n_a > n ? hipErrorInvalidValue : hipSuccess;
  hipLaunchKernelGGL(random_keys_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, v, n,
                     a, n_a, seed);
  return hipGetLastError();
}

}  // namespace swam
