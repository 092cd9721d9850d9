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

// erf(u) for u >= 0 by the rational approximation of Abramowitz & Stegun
// 7.1.26 (after Hastings): erf(u) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5))))
// exp(-u^2) with t = 1 / (1 + p u), absolute error below 1.5e-7 for every
// u >= 0.  Branch-free: one reciprocal, one exp2, five FMAs.
__device__ __forceinline__ float erf_nonneg(float u) {
  constexpr float p = 0.3275911f, a1 = 0.254829592f, a2 = -0.284496736f, a3 = 1.421413741f,
                  a4 = -1.453152027f, a5 = 1.061405429f;
  const float t = __builtin_amdgcn_rcpf(fmaf(p, u, 1.0f));
  const float poly = t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, a5, a4), a3), a2), a1);
  const float e = __builtin_amdgcn_exp2f(-(u * u) * 1.4426950408889634f);
  return 1.0f - poly * e;
}

// Exact-erf GELU: z * Phi(z) = z (1 + erf(z / sqrt 2)) / 2, erf odd.
__device__ __forceinline__ float gelu_erf(float z) {
  const float e = erf_nonneg(fabsf(z) * 0.70710678118654752f);
  return 0.5f * z * (1.0f + copysignf(e, z));
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
