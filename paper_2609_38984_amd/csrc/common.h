// Internal device helpers and types shared by the HIP sources of libswam
// (gfx950 only).  The host-side launcher declarations and their argument
// structs are in launchers.h.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define SWAM_SEL_MAXNP 4096   // selection sort capacity (next power of two >= N_s)
#define SWAM_MAX_NS_DEV 4096

namespace swam {

typedef uint16_t bf16_t;  // raw bf16 storage

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(bf16_t v) {
  return __uint_as_float(((uint32_t)v) << 16);
}

// Round to nearest even (inputs are finite in this library).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// Physical 16-byte chunk of logical chunk c in row r of an LDS tile with
// 128-byte rows is c ^ lds_swz(r).  The LDS serves a ds_read_b128 in phases
// of 16 lanes and a 64-bit read in phases of 32 lanes over 64 four-byte banks;
// with this swizzle 16 consecutive rows at one logical chunk (the MFMA operand
// reads) and the transposed 64-bit reads of 8 rows x 64 bytes both hit every
// bank once per phase.  Only row bits 1..3 matter.
__device__ __forceinline__ int lds_swz(int r) {
  return ((r >> 1) & 3) | ((((r >> 1) ^ (r >> 3)) & 1) << 2);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p) { return *p; }
  __device__ __forceinline__ static void store(float* p, float v) { *p = v; }
};
template <> struct Elem<bf16_t> {
  __device__ __forceinline__ static float load(const bf16_t* p) { return bf16_to_f32(*p); }
  __device__ __forceinline__ static void store(bf16_t* p, float v) { *p = f32_to_bf16(v); }
};

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ double warp_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

}  // namespace swam
