// Indexing, LayerNorm-gather and decoder-input kernels.
#include "device_common.h"

namespace marche {

// map[r] for every active row r: image, token and residual-stream row.
__global__ void row_map_kernel(RowMap *map, const int32_t *a_idx, const int32_t *a_off,
                               int32_t n_tokens) {
  const int b = blockIdx.x;
  const int r0 = a_off[b], r1 = a_off[b + 1];
  for (int r = r0 + threadIdx.x; r < r1; r += blockDim.x) {
    const int tok = a_idx[r];
    RowMap m;
    m.x_row = b * n_tokens + tok;
    m.b = b;
    m.tok = tok;
    m.pad = 0;
    map[r] = m;
  }
}

hipError_t launch_row_map(RowMap *map, const int32_t *a_idx, const int32_t *a_off, int32_t batch,
                          int32_t n_tokens, hipStream_t s) {
  launch_kernel(row_map_kernel, batch, 256, 0, s, map, a_idx, a_off, n_tokens);
  return hipGetLastError();
}

// Validation of the device-resident active lists (debug mode of the step):
// one workgroup per image.  report[0] receives the first failure as
// 1 + code * batch + image (0 = none); codes: 0 offsets (a_off[0] != 0,
// a_off[batch] != a_total, decreasing, or a list longer than a_max),
// 1 token outside [0, n_tokens), 2 a token listed twice for one image,
// 3 n_gen[b] outside [0, |A_b|] or above gen_max.  Every read stays inside
// a_off[0 .. batch] and a_idx[0 .. a_total), whatever the lists hold.
constexpr int kMaxTokens = 4096;  // the model check bounds n_tokens

__global__ void clear_word_kernel(int32_t *p) {
  if (threadIdx.x == 0) *p = 0;
}

__global__ __launch_bounds__(256) void check_active_kernel(
    const int32_t *a_idx, const int32_t *a_off, const int32_t *n_gen, int32_t batch,
    int32_t n_tokens, int32_t a_total, int32_t a_max, int32_t gen_max, int32_t *report) {
  __shared__ unsigned seen[kMaxTokens / 32];
  __shared__ int bad;
  const int b = blockIdx.x;
  auto fail = [&](int code) { atomicCAS(report, 0, 1 + code * batch + b); };
  for (int i = threadIdx.x; i < (n_tokens + 31) / 32; i += blockDim.x) seen[i] = 0u;
  if (threadIdx.x == 0) bad = 0;
  __syncthreads();
  const int lo = a_off[b], hi = a_off[b + 1];
  if (threadIdx.x == 0) {
    const bool first_ok = b > 0 || lo == 0;
    const bool last_ok = b + 1 < batch || hi == a_total;
    if (!first_ok || !last_ok || lo < 0 || hi < lo || hi > a_total || hi - lo > a_max) {
      fail(0);
      bad = 1;
    } else if (n_gen && (n_gen[b] < 0 || n_gen[b] > hi - lo || n_gen[b] > gen_max)) {
      fail(3);
    }
  }
  __syncthreads();
  if (bad) return;  // the list bounds are not trusted: read no index
  for (int r = lo + threadIdx.x; r < hi; r += blockDim.x) {
    const int tok = a_idx[r];
    if (tok < 0 || tok >= n_tokens) {
      fail(1);
      continue;
    }
    if (atomicOr(&seen[tok >> 5], 1u << (tok & 31)) & (1u << (tok & 31))) fail(2);
  }
}

hipError_t launch_check_active(const int32_t *a_idx, const int32_t *a_off, const int32_t *n_gen,
                               int32_t batch, int32_t n_tokens, int32_t a_total, int32_t a_max,
                               int32_t gen_max, int32_t *report, hipStream_t s) {
  launch_kernel(clear_word_kernel, 1, 64, 0, s, report);
  launch_kernel(check_active_kernel, batch, 256, 0, s, a_idx, a_off, n_gen, batch, n_tokens, a_total, a_max,
                                            gen_max, report);
  return hipGetLastError();
}

// u[r] = LN(x[map[r].x_row]) * g + b, one wavefront per active row.
// Each lane holds NV float4 chunks of the row (d_model = NV * 256).
// Statistics in float32: mean, then the population variance of the centred
// values; eps inside the square root.
template <typename OutT, int NV>
__global__ __launch_bounds__(256) void gather_ln_kernel(OutT *__restrict__ out,
                                                        const float *__restrict__ x,
                                                        const RowMap *__restrict__ map,
                                                        const float *__restrict__ g,
                                                        const float *__restrict__ bta, int rows,
                                                        float eps) {
  constexpr int D = NV * 256;
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const float4 *xr = reinterpret_cast<const float4 *>(x + (size_t)map[r].x_row * D);
  float4 v[NV];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    v[i] = xr[lane + 64 * i];
    s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
  }
  const float mean = wave_sum(s) * (1.0f / D);
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    v[i].x -= mean; v[i].y -= mean; v[i].z -= mean; v[i].w -= mean;
    ss += (v[i].x * v[i].x + v[i].y * v[i].y) + (v[i].z * v[i].z + v[i].w * v[i].w);
  }
  const float var = wave_sum(ss) * (1.0f / D);
  const float rstd = 1.0f / sqrtf(var + eps);
  const float4 *g4 = reinterpret_cast<const float4 *>(g);
  const float4 *b4 = reinterpret_cast<const float4 *>(bta);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c4 = lane + 64 * i;
    const float4 gg = g4[c4], bb = b4[c4];
    const float y0 = v[i].x * rstd * gg.x + bb.x;
    const float y1 = v[i].y * rstd * gg.y + bb.y;
    const float y2 = v[i].z * rstd * gg.z + bb.z;
    const float y3 = v[i].w * rstd * gg.w + bb.w;
    OutT *o = out + (size_t)r * D + 4 * c4;
    if constexpr (sizeof(OutT) == 4) {
      *reinterpret_cast<float4 *>(o) = make_float4(y0, y1, y2, y3);
    } else {
      bf16x4 pk = {(bf16)y0, (bf16)y1, (bf16)y2, (bf16)y3};
      *reinterpret_cast<bf16x4 *>(o) = pk;
    }
  }
}

template <typename OutT>
static hipError_t gather_ln_dispatch(OutT *out, const float *x, const RowMap *map, const float *g,
                                     const float *b, int rows, int d, float eps, hipStream_t s) {
  const int grid = (rows + 3) / 4;
  switch (d / 256) {
    case 1: launch_kernel(gather_ln_kernel<OutT, 1>, grid, 256, 0, s, out, x, map, g, b, rows, eps); break;
    case 2: launch_kernel(gather_ln_kernel<OutT, 2>, grid, 256, 0, s, out, x, map, g, b, rows, eps); break;
    case 3: launch_kernel(gather_ln_kernel<OutT, 3>, grid, 256, 0, s, out, x, map, g, b, rows, eps); break;
    case 4: launch_kernel(gather_ln_kernel<OutT, 4>, grid, 256, 0, s, out, x, map, g, b, rows, eps); break;
    case 5: launch_kernel(gather_ln_kernel<OutT, 5>, grid, 256, 0, s, out, x, map, g, b, rows, eps); break;
    case 6: launch_kernel(gather_ln_kernel<OutT, 6>, grid, 256, 0, s, out, x, map, g, b, rows, eps); break;
    case 7: launch_kernel(gather_ln_kernel<OutT, 7>, grid, 256, 0, s, out, x, map, g, b, rows, eps); break;
    case 8: launch_kernel(gather_ln_kernel<OutT, 8>, grid, 256, 0, s, out, x, map, g, b, rows, eps); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gather_ln(DType dt, void *out, const float *x, const RowMap *map, const float *g,
                            const float *b, int32_t rows, int32_t d_model, float eps,
                            hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (d_model % 256 != 0) return hipErrorInvalidValue;
  if (dt == DType::F32)
    return gather_ln_dispatch(static_cast<float *>(out), x, map, g, b, rows, d_model, eps, s);
  return gather_ln_dispatch(static_cast<bf16 *>(out), x, map, g, b, rows, d_model, eps, s);
}

// x[b][j] = pos[j] + (buffer token: cls[b] | generated: value[b][j-n_buf] | masked: mask).
__global__ __launch_bounds__(256) void decoder_input_kernel(
    float *__restrict__ x, const float *__restrict__ cls, const float *__restrict__ value,
    const float *__restrict__ mask, const float *__restrict__ pos, const int32_t *__restrict__ rank,
    int n_tokens, int n_buf, int d4, int n_known) {
  const int row = blockIdx.x;  // b * n_tokens + j
  const int b = row / n_tokens, j = row - b * n_tokens;
  const int n_img = n_tokens - n_buf;
  const float4 *src;
  if (j < n_buf) {
    src = reinterpret_cast<const float4 *>(cls + (size_t)b * d4 * 4);
  } else if (rank[(size_t)b * n_img + (j - n_buf)] < n_known) {
    src = reinterpret_cast<const float4 *>(value + ((size_t)b * n_img + (j - n_buf)) * d4 * 4);
  } else {
    src = reinterpret_cast<const float4 *>(mask);
  }
  const float4 *p = reinterpret_cast<const float4 *>(pos + (size_t)j * d4 * 4);
  float4 *o = reinterpret_cast<float4 *>(x + (size_t)row * d4 * 4);
  for (int c = threadIdx.x; c < d4; c += blockDim.x) {
    const float4 a = src[c], q = p[c];
    o[c] = make_float4(a.x + q.x, a.y + q.y, a.z + q.z, a.w + q.w);
  }
}

hipError_t launch_decoder_input(float *x, const float *cls, const float *value, const float *mask,
                                const float *pos, const int32_t *rank, int32_t batch,
                                int32_t n_tokens, int32_t n_buf, int32_t d_model, int32_t n_known,
                                hipStream_t s) {
  if (batch == 0) return hipSuccess;
  launch_kernel(decoder_input_kernel, batch * n_tokens, 256, 0, s, x, cls, value, mask, pos, rank, n_tokens,
                                                        n_buf, d_model / 4, n_known);
  return hipGetLastError();
}

__global__ void fill_zero_kernel(uint4 *dst, size_t n16, unsigned char *tail, size_t n_tail) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    dst[i] = make_uint4(0, 0, 0, 0);
  if (blockIdx.x == 0)
    for (size_t i = threadIdx.x; i < n_tail; i += blockDim.x) tail[i] = 0;
}

// Zero `bytes` bytes at a 16-byte aligned device pointer with plain vector stores.
hipError_t launch_fill_zero(void *dst, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  const size_t n16 = bytes / 16;
  unsigned char *tail = static_cast<unsigned char *>(dst) + n16 * 16;
  size_t grid = (n16 + 255) / 256;
  if (grid > 8192) grid = 8192;
  if (grid == 0) grid = 1;
  launch_kernel(fill_zero_kernel, (unsigned)grid, 256, 0, s, static_cast<uint4 *>(dst), n16, tail,
                                                  bytes - n16 * 16);
  return hipGetLastError();
}

}  // namespace marche
