// Device-side helpers shared by the HIP kernels of libmarche.so (gfx950,
// 64-lane wavefronts).
#pragma once

#include <hip/hip_ext.h>

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

// Exact-erf GELU, z * Phi(z), written as max(z, 0) - |z| * Phi(-|z|) (the two
// agree for either sign of z), with the upper tail of the normal distribution
// from the rational approximation of Abramowitz & Stegun 7.1.26 (after
// Hastings): for a >= 0,
//   Phi(-a) = (1 - erf(a / sqrt 2)) / 2 = t (c1 + t (c2 + t (c3 + t (c4 + t c5)))) exp(-a^2 / 2),
//   t = 1 / (1 + p a / sqrt 2), c_i = a_i / 2,
// absolute error of erf below 1.5e-7.  Branch-free: one reciprocal, one exp2,
// about ten other operations.
__device__ __forceinline__ float gelu_erf(float z) {
  constexpr float p_s = 0.3275911f * 0.70710678118654752f;  // p / sqrt 2
  constexpr float c1 = 0.5f * 0.254829592f, c2 = 0.5f * -0.284496736f, c3 = 0.5f * 1.421413741f,
                  c4 = 0.5f * -1.453152027f, c5 = 0.5f * 1.061405429f;
  constexpr float h = -0.5f * 1.4426950408889634f;  // -log2(e) / 2
  const float a = fabsf(z);
  const float t = __builtin_amdgcn_rcpf(fmaf(p_s, a, 1.0f));
  const float poly = t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, c5, c4), c3), c2), c1);
  const float e = __builtin_amdgcn_exp2f(a * (a * h));
  return fmaf(-a, poly * e, fmaxf(z, 0.0f));
}

// SiLU z * sigmoid(z) = z / (1 + 2^(-z log2 e)); for z -> -inf the power
// overflows to +inf and the reciprocal to 0.
__device__ __forceinline__ float silu(float z) {
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
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

// Launch of a kernel of this library: when a timed call is in progress on
// this thread (kernel_events()), its events go with the dispatch of the
// call's first kernel.
template <typename... KArgs, typename... Args>
inline void launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, uint32_t lds,
                          hipStream_t s, Args... args) {
  KernelEvents *ev = kernel_events();
  if (ev && !ev->used) {
    ev->used = true;
    hipExtLaunchKernelGGL(kernel, grid, block, lds, s, ev->start, ev->stop, 0,
                          static_cast<KArgs>(args)...);
  } else {
    kernel<<<grid, block, lds, s>>>(static_cast<KArgs>(args)...);
  }
}

}  // namespace marche
