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
// agree for either sign of z).  The normal tail is Phi(-a) = 2^P(min(a, 6)),
// P(u) = c0 + c1 u + ... + c7 u^7 a polynomial fit to log2 Phi(-u) on [0, 6]
// (csrc/gelu_fit.py: Lawson-type reweighted least squares toward the minimax
// fit).  Evaluated in fp32 as here, Phi(-u) is within a relative 7e-6 of the
// exact tail on [0, 6], and the GELU within 6e-7 * max(1, |z|) of the exact
// one for every z (past |z| = 6 the tail term is below 1e-9 |z|).
// Branch-free: one exp2, seven FMAs and four other operations, against the
// reciprocal, exp2 and twelve operations of a rational erfc approximation.
__device__ __forceinline__ float gelu_erf(float z) {
  constexpr float c0 = -0.999995291f, c1 = -1.1512512f, c2 = -0.458464146f,
                  c3 = -0.0539602935f, c4 = 0.00850799028f, c5 = -0.000930548005f,
                  c6 = 6.16009856e-05f, c7 = -1.83493421e-06f;
  const float a = fabsf(z);
  const float u = fminf(a, 6.0f);
  float p = fmaf(c7, u, c6);
  p = fmaf(p, u, c5);
  p = fmaf(p, u, c4);
  p = fmaf(p, u, c3);
  p = fmaf(p, u, c2);
  p = fmaf(p, u, c1);
  p = fmaf(p, u, c0);
  return fmaf(-a, __builtin_amdgcn_exp2f(p), fmaxf(z, 0.0f));
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
