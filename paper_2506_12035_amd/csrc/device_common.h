// Device-side helpers shared by the HIP kernels of libmarche.so (gfx950,
// 64-lane wavefronts).
#pragma once

#include "marche_internal.h"

namespace marche {

// Native 16-byte vector (HIP's uint4 is a struct with a union, which keeps
// arrays of it from being promoted to registers).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Exact-erf GELU: z * Phi(z).
__device__ __forceinline__ float gelu_erf(float z) {
  return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));
}

template <typename T>
__device__ __forceinline__ T from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }  // RNE on gfx950

template <typename T>
__device__ __forceinline__ float to_f32(T v) { return (float)v; }

// XCD-aware reordering of a 1-D grid: the hardware deals consecutive
// workgroup ids round-robin over the 8 XCDs; this maps them so that each XCD
// receives a contiguous range of logical ids (neighbouring tiles then share
// that XCD's L2).  Identity when the grid is not a multiple of 8.
__device__ __forceinline__ int xcd_remap(int wg, int n_wg) {
  if (n_wg % 8 != 0) return wg;
  return (wg % 8) * (n_wg / 8) + wg / 8;
}

}  // namespace marche
