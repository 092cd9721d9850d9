// The rest of a MAR step around the decoder: the encoder's input rows (Eq. 1),
// the decoder input's masked rows (Eq. 2), LayerNorm of gathered rows, and the
// kernels of the sampler of Eq. 3 between its GEMMs (time embedding table,
// condition SiLU, modulated LayerNorms, output projection + DDPM step).
//
// Row kernels run one wavefront per row, four rows per 256-thread workgroup;
// a row of width NV * 256 is NV float4 chunks per lane.  LayerNorm statistics
// are float32: the mean, then the population variance of the centred values,
// eps inside the square root.
#include "device_common.h"

namespace marche {

namespace {

template <typename T>
__device__ __forceinline__ void store_row4(T *p, float a, float b, float c, float d) {
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<float4 *>(p) = make_float4(a, b, c, d);
  } else {
    bf16x4 pk = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
    *reinterpret_cast<bf16x4 *>(p) = pk;
  }
}

template <typename T>
__device__ __forceinline__ float4 load_row4(const T *p) {
  if constexpr (sizeof(T) == 4) {
    return *reinterpret_cast<const float4 *>(p);
  } else {
    const bf16x4 v = *reinterpret_cast<const bf16x4 *>(p);
    return make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
  }
}

// Mean and reciprocal standard deviation of a row held as v[NV] (centres v).
template <int NV>
__device__ __forceinline__ float centre_rstd(float4 (&v)[NV], float eps) {
  constexpr float inv_d = 1.0f / (NV * 256);
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
  const float mean = wave_sum(s) * inv_d;
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    v[i].x -= mean; v[i].y -= mean; v[i].z -= mean; v[i].w -= mean;
    ss += (v[i].x * v[i].x + v[i].y * v[i].y) + (v[i].z * v[i].z + v[i].w * v[i].w);
  }
  return 1.0f / sqrtf(wave_sum(ss) * inv_d + eps);
}

}  // namespace

// ---- Eq. 1: encoder input rows -------------------------------------------
// Row i of image b (b = row / n_enc): i < n_buf -> cls[b] + pe[i]; else the
// known image token p = known[b][i - n_buf]: w_z . tok[b][p] + b_z + pe[n_buf + p].
template <int NV, int CM>
__global__ __launch_bounds__(256) void encoder_input_kernel(
    float *__restrict__ x, const float *__restrict__ cls, const float *__restrict__ tok,
    const float *__restrict__ w_z, const float *__restrict__ b_z, const float *__restrict__ pe,
    const int32_t *__restrict__ known, int rows, int n_enc, int n_buf, int n_img, int n_known,
    int C) {
  constexpr int D = NV * 256;
  __shared__ float tv[4][CM];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int row = blockIdx.x * 4 + w;
  if (row >= rows) return;  // no barrier below
  const int b = row / n_enc, i = row - b * n_enc;
  float4 *o = reinterpret_cast<float4 *>(x + (size_t)row * D);
  if (i < n_buf) {
    const float4 *c4 = reinterpret_cast<const float4 *>(cls + (size_t)b * D);
    const float4 *p4 = reinterpret_cast<const float4 *>(pe + (size_t)i * D);
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const float4 a = c4[lane + 64 * k], q = p4[lane + 64 * k];
      o[lane + 64 * k] = make_float4(a.x + q.x, a.y + q.y, a.z + q.z, a.w + q.w);
    }
    return;
  }
  const int p = known[(size_t)b * n_known + (i - n_buf)];
  // token value, zero-padded to CM channels
  if (lane < CM) tv[w][lane] = lane < C ? tok[((size_t)b * n_img + p) * C + lane] : 0.f;
  // the wavefront's own LDS writes are complete before its reads; no other
  // wavefront touches tv[w]
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
  __builtin_amdgcn_wave_barrier();
  const float4 *p4 = reinterpret_cast<const float4 *>(pe + (size_t)(n_buf + p) * D);
  const float4 *bz = reinterpret_cast<const float4 *>(b_z);
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int d0 = 4 * (lane + 64 * k);
    float acc[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float *wr = w_z + (size_t)(d0 + e) * C;
      float s = 0.f;
#pragma unroll 16
      for (int c = 0; c < CM; ++c) s = fmaf(wr[min(c, C - 1)], tv[w][c], s);
      acc[e] = s;
    }
    const float4 q = p4[lane + 64 * k], bb = bz[lane + 64 * k];
    o[lane + 64 * k] = make_float4(acc[0] + bb.x + q.x, acc[1] + bb.y + q.y, acc[2] + bb.z + q.z,
                                   acc[3] + bb.w + q.w);
  }
}

// ---- Eq. 2: masked rows of the decoder input ------------------------------
// x[b][n_buf + p] = mask + pe[n_buf + p] for every image token p with
// rank[b][p] >= n_known; known tokens and buffer rows are left to the
// embedding GEMM.
template <int NV>
__global__ __launch_bounds__(256) void mask_fill_kernel(float *__restrict__ x,
                                                        const float *__restrict__ mask,
                                                        const float *__restrict__ pe,
                                                        const int32_t *__restrict__ rank, int rows,
                                                        int n_tokens, int n_buf, int n_img,
                                                        int n_known) {
  constexpr int D = NV * 256;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);  // b * n_img + p
  if (row >= rows) return;
  if (rank[row] < n_known) return;
  const int b = row / n_img, j = n_buf + (row - b * n_img);
  const float4 *m4 = reinterpret_cast<const float4 *>(mask);
  const float4 *p4 = reinterpret_cast<const float4 *>(pe + (size_t)j * D);
  float4 *o = reinterpret_cast<float4 *>(x + ((size_t)b * n_tokens + j) * D);
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const float4 a = m4[lane + 64 * k], q = p4[lane + 64 * k];
    o[lane + 64 * k] = make_float4(a.x + q.x, a.y + q.y, a.z + q.z, a.w + q.w);
  }
}

// ---- LayerNorm of gathered rows -------------------------------------------
// out[r] = LN(x[src]) * g + b (+ add[tok - n_buf]), src = rows ? rows[r] : r,
// tok = src % n_tokens.  The encoder's final norm (rows = NULL, add = NULL)
// and the condition of Eq. 3 (decoder norm of the generating rows plus the
// head's positional embedding).
template <typename OutT, int NV>
__global__ __launch_bounds__(256) void ln_rows_kernel(OutT *__restrict__ out,
                                                      const float *__restrict__ x,
                                                      const int32_t *__restrict__ rows_idx,
                                                      const float *__restrict__ g,
                                                      const float *__restrict__ bta,
                                                      const float *__restrict__ add, int rows,
                                                      int n_tokens, int n_buf, float eps) {
  constexpr int D = NV * 256;
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int src = rows_idx ? rows_idx[r] : r;
  const float4 *xr = reinterpret_cast<const float4 *>(x + (size_t)src * D);
  float4 v[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = xr[lane + 64 * i];
  const float rstd = centre_rstd<NV>(v, eps);
  const float4 *g4 = reinterpret_cast<const float4 *>(g);
  const float4 *b4 = reinterpret_cast<const float4 *>(bta);
  const float4 *a4 =
      add ? reinterpret_cast<const float4 *>(add + (size_t)(src % n_tokens - n_buf) * D) : nullptr;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c4 = lane + 64 * i;
    const float4 gg = g4[c4], bb = b4[c4];
    float4 y = make_float4(v[i].x * rstd * gg.x + bb.x, v[i].y * rstd * gg.y + bb.y,
                           v[i].z * rstd * gg.z + bb.z, v[i].w * rstd * gg.w + bb.w);
    if (a4) {
      const float4 q = a4[c4];
      y.x += q.x; y.y += q.y; y.z += q.z; y.w += q.w;
    }
    store_row4(out + (size_t)r * D + 4 * c4, y.x, y.y, y.z, y.w);
  }
}

// ---- Eq. 3: sampler --------------------------------------------------------
// Sinusoidal embedding of timesteps 0..n_steps-1: out[i][f] = cos(i w_f) for
// f < F/2, sin(i w_{f - F/2}) otherwise, w_j = 10000^(-j / (F/2)).
template <typename OutT>
__global__ __launch_bounds__(256) void time_sinus_kernel(OutT *__restrict__ out, int n_steps, int F) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= n_steps * F) return;
  const int i = idx / F, f = idx - i * F, half = F / 2;
  const int j = f < half ? f : f - half;
  const float w = expf(-9.210340371976184f * (float)j / (float)half);  // ln 10000
  const float a = (float)i * w;
  out[idx] = (OutT)(f < half ? cosf(a) : sinf(a));
}

// sc[r][c] = SiLU(cond[r][c] + temb[c]) for one timestep's embedding row.
template <typename OutT>
__global__ __launch_bounds__(256) void silu_cond_kernel(OutT *__restrict__ sc,
                                                        const float *__restrict__ cond,
                                                        const float *__restrict__ temb, int rows,
                                                        int W) {
  const int w4 = W / 4;
  const int idx = blockIdx.x * 256 + threadIdx.x;  // float4 index
  if (idx >= rows * w4) return;
  const int c4 = idx % w4;
  const float4 a = reinterpret_cast<const float4 *>(cond)[idx];
  const float4 t = reinterpret_cast<const float4 *>(temb)[c4];
  store_row4(sc + (size_t)idx * 4, silu(a.x + t.x), silu(a.y + t.y), silu(a.z + t.z),
             silu(a.w + t.w));
}

// w_t[c][d] = w[d][c] for a [rows][cols] float32 matrix (the input
// projection, so that lanes over d read it coalesced).
__global__ __launch_bounds__(256) void transpose_f32_kernel(float *__restrict__ w_t,
                                                            const float *__restrict__ w, int rows,
                                                            int cols) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= rows * cols) return;
  const int d = idx / cols, c = idx - d * cols;
  w_t[(size_t)c * rows + d] = w[idx];
}

// Input projection of the noisy token and the first block's modulated norm:
// h[r] = w_in x[r] + b_in;  a[r] = LN(h[r]) * (1 + scale) + shift with
// (shift, scale) = mod[r][0 .. 2W) (block 0).  The projection is given
// transposed, w_in_t [C][W].
template <typename T, int NV, int CM>
__global__ __launch_bounds__(256) void head_in_mod_kernel(T *__restrict__ a_out,
                                                          float *__restrict__ h,
                                                          const float *__restrict__ x,
                                                          const float *__restrict__ w_in_t,
                                                          const float *__restrict__ b_in,
                                                          const T *__restrict__ mod, int mod_ld,
                                                          int rows, int C, float eps) {
  constexpr int W = NV * 256;
  __shared__ float tv[4][CM];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = blockIdx.x * 4 + w;
  if (r >= rows) return;
  if (lane < CM) tv[w][lane] = lane < C ? x[(size_t)r * C + lane] : 0.f;
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): own LDS writes done
  __builtin_amdgcn_wave_barrier();
  float4 v[NV];
  const float4 *bi = reinterpret_cast<const float4 *>(b_in);
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c4 = lane + 64 * k;
    float4 acc = bi[c4];
#pragma unroll 16
    for (int c = 0; c < CM; ++c) {  // channels past C have tv = 0 and repeat row C - 1
      const float4 wv = reinterpret_cast<const float4 *>(w_in_t + (size_t)min(c, C - 1) * W)[c4];
      const float xc = tv[w][c];
      acc.x = fmaf(wv.x, xc, acc.x);
      acc.y = fmaf(wv.y, xc, acc.y);
      acc.z = fmaf(wv.z, xc, acc.z);
      acc.w = fmaf(wv.w, xc, acc.w);
    }
    v[k] = acc;
    reinterpret_cast<float4 *>(h + (size_t)r * W)[lane + 64 * k] = v[k];
  }
  const float rstd = centre_rstd<NV>(v, eps);
  const T *mr = mod + (size_t)r * mod_ld;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c = 4 * (lane + 64 * k);
    const float4 sh = load_row4(mr + c), sc = load_row4(mr + W + c);
    store_row4(a_out + (size_t)r * W + c, v[k].x * rstd * (1.f + sc.x) + sh.x,
               v[k].y * rstd * (1.f + sc.y) + sh.y, v[k].z * rstd * (1.f + sc.z) + sh.z,
               v[k].w * rstd * (1.f + sc.w) + sh.w);
  }
}

// Gated residual of block k and the next modulated norm:
// h[r] += gate * t[r];  a[r] = LN(h[r]) * (1 + scale) + shift, where gate,
// shift and scale are W-wide slices of mod[r] at the given offsets.
template <typename T, int NV>
__global__ __launch_bounds__(256) void head_gate_mod_kernel(T *__restrict__ a_out,
                                                            float *__restrict__ h,
                                                            const float *__restrict__ t,
                                                            const T *__restrict__ mod, int mod_ld,
                                                            int gate_off, int shift_off,
                                                            int scale_off, int rows, float eps) {
  constexpr int W = NV * 256;
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const T *mr = mod + (size_t)r * mod_ld;
  float4 *hr = reinterpret_cast<float4 *>(h + (size_t)r * W);
  const float4 *tr = reinterpret_cast<const float4 *>(t + (size_t)r * W);
  float4 v[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c4 = lane + 64 * k;
    const float4 hv = hr[c4], tv = tr[c4], g = load_row4(mr + gate_off + 4 * c4);
    v[k] = make_float4(fmaf(g.x, tv.x, hv.x), fmaf(g.y, tv.y, hv.y), fmaf(g.z, tv.z, hv.z),
                       fmaf(g.w, tv.w, hv.w));
    hr[c4] = v[k];
  }
  const float rstd = centre_rstd<NV>(v, eps);
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c = 4 * (lane + 64 * k);
    const float4 sh = load_row4(mr + shift_off + c), sc = load_row4(mr + scale_off + c);
    store_row4(a_out + (size_t)r * W + c, v[k].x * rstd * (1.f + sc.x) + sh.x,
               v[k].y * rstd * (1.f + sc.y) + sh.y, v[k].z * rstd * (1.f + sc.z) + sh.z,
               v[k].w * rstd * (1.f + sc.w) + sh.w);
  }
}

// Output projection eps[r] = w_out a[r] + b_out (C values) and one DDPM step:
// x0 = sra x - srm1 eps;  x_next = c1 x0 + c2 x + sigma * noise, with x the
// current token value (x_cur) and sigma = tau * sqrt(posterior variance)
// (0 at the last step).  x_next may alias x_cur (each lane reads its own
// element before writing it).  On the last step the result also goes to
// tok_out[out_rows[r]].
template <typename T, int CM>
__global__ __launch_bounds__(256) void head_out_step_kernel(
    float *x_next, float *__restrict__ tok_out, const T *__restrict__ a,
    const float *__restrict__ w_out, const float *__restrict__ b_out, const float *x_cur,
    const float *__restrict__ noise, const int32_t *__restrict__ out_rows, int rows, int W, int C,
    float sra, float srm1, float c1, float c2, float sigma) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  float acc[CM];
#pragma unroll
  for (int c = 0; c < CM; ++c) acc[c] = 0.f;
  const T *ar = a + (size_t)r * W;
  for (int k0 = 4 * lane; k0 < W; k0 += 256) {
    const float4 av = load_row4(ar + k0);
    float4 wv[CM];  // all loads of this chunk first (rows past C repeat the last one)
#pragma unroll
    for (int c = 0; c < CM; ++c)
      wv[c] = *reinterpret_cast<const float4 *>(w_out + (size_t)min(c, C - 1) * W + k0);
#pragma unroll
    for (int c = 0; c < CM; ++c)
      acc[c] = fmaf(av.x, wv[c].x, fmaf(av.y, wv[c].y, fmaf(av.z, wv[c].z, fmaf(av.w, wv[c].w, acc[c]))));
  }
  float e = 0.f;
#pragma unroll
  for (int c = 0; c < CM; ++c) {
    const float s = wave_sum(acc[c]);
    if (lane == c) e = s;
  }
  if (lane < C) {
    const size_t idx = (size_t)r * C + lane;
    const float xv = x_cur[idx];
    const float eps_v = e + b_out[lane];
    const float x0 = sra * xv - srm1 * eps_v;
    float xn = c1 * x0 + c2 * xv;
    if (sigma != 0.f) xn = fmaf(sigma, noise[idx], xn);
    x_next[idx] = xn;
    if (tok_out) tok_out[(size_t)out_rows[r] * C + lane] = xn;
  }
}

// ------------------------------------------------------------------ launchers

#define MARCHE_NV_SWITCH(nv, CALL)        \
  switch (nv) {                           \
    case 1: CALL(1); break;               \
    case 2: CALL(2); break;               \
    case 3: CALL(3); break;               \
    case 4: CALL(4); break;               \
    case 5: CALL(5); break;               \
    case 6: CALL(6); break;               \
    case 7: CALL(7); break;               \
    case 8: CALL(8); break;               \
    case 9: CALL(9); break;               \
    case 10: CALL(10); break;             \
    case 11: CALL(11); break;             \
    case 12: CALL(12); break;             \
    case 13: CALL(13); break;             \
    case 14: CALL(14); break;             \
    case 15: CALL(15); break;             \
    case 16: CALL(16); break;             \
    default: return hipErrorInvalidValue; \
  }

// Token channels rounded up to 4, 8, 16, 32 or 64 (compile-time loops).
template <int NV>
static void encoder_input_dispatch(int grid, hipStream_t s, float *x, const float *cls,
                                   const float *tok, const float *w_z, const float *b_z,
                                   const float *pe, const int32_t *known, int rows, int n_enc,
                                   int n_buf, int n_img, int n_known, int c) {
#define E_(CM) launch_kernel(encoder_input_kernel<NV, CM>, grid, 256, 0, s, x, cls, tok, w_z, b_z, pe, known, \
                                                                rows, n_enc, n_buf, n_img, n_known, c)
  if (c <= 4) E_(4);
  else if (c <= 8) E_(8);
  else if (c <= 16) E_(16);
  else if (c <= 32) E_(32);
  else E_(64);
#undef E_
}

hipError_t launch_encoder_input(float *x, const float *cls, const float *tok, const float *w_z,
                                const float *b_z, const float *pe, const int32_t *known,
                                int32_t batch, int32_t n_buf, int32_t n_img, int32_t n_known,
                                int32_t d_model, int32_t c_tok, hipStream_t s) {
  const int n_enc = n_buf + n_known, rows = batch * n_enc;
  if (rows == 0) return hipSuccess;
  if (d_model % 256 != 0 || c_tok < 1 || c_tok > 64) return hipErrorInvalidValue;
  const int grid = (rows + 3) / 4;
#define L_(NV) encoder_input_dispatch<NV>(grid, s, x, cls, tok, w_z, b_z, pe, known, rows, n_enc, \
                                         n_buf, n_img, n_known, c_tok)
  MARCHE_NV_SWITCH(d_model / 256, L_)
#undef L_
  return hipGetLastError();
}

hipError_t launch_mask_fill(float *x, const float *mask, const float *pe, const int32_t *rank,
                            int32_t batch, int32_t n_tokens, int32_t n_buf, int32_t n_known,
                            int32_t d_model, hipStream_t s) {
  const int n_img = n_tokens - n_buf, rows = batch * n_img;
  if (rows == 0) return hipSuccess;
  if (d_model % 256 != 0) return hipErrorInvalidValue;
  const int grid = (rows + 3) / 4;
#define L_(NV)                                                                          \
  launch_kernel(mask_fill_kernel<NV>, grid, 256, 0, s, x, mask, pe, rank, rows, n_tokens, n_buf, n_img, \
                                            n_known)
  MARCHE_NV_SWITCH(d_model / 256, L_)
#undef L_
  return hipGetLastError();
}

hipError_t launch_ln_rows(DType dt, void *out, const float *x, const int32_t *rows_idx,
                          const float *g, const float *b, const float *add, int32_t rows,
                          int32_t n_tokens, int32_t n_buf, int32_t d_model, float eps,
                          hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (d_model % 256 != 0) return hipErrorInvalidValue;
  const int grid = (rows + 3) / 4;
  if (dt == DType::F32) {
#define L_(NV)                                                                                  \
  launch_kernel(ln_rows_kernel<float, NV>, grid, 256, 0, s, static_cast<float *>(out), x, rows_idx, g, b, add, \
                                                 rows, n_tokens, n_buf, eps)
    MARCHE_NV_SWITCH(d_model / 256, L_)
#undef L_
  } else {
#define L_(NV)                                                                                \
  launch_kernel(ln_rows_kernel<bf16, NV>, grid, 256, 0, s, static_cast<bf16 *>(out), x, rows_idx, g, b, add, \
                                                rows, n_tokens, n_buf, eps)
    MARCHE_NV_SWITCH(d_model / 256, L_)
#undef L_
  }
  return hipGetLastError();
}

hipError_t launch_time_sinus(DType dt, void *out, int32_t n_steps, int32_t freq, hipStream_t s) {
  const int n = n_steps * freq;
  if (n == 0) return hipSuccess;
  const int grid = (n + 255) / 256;
  if (dt == DType::F32)
    launch_kernel(time_sinus_kernel<float>, grid, 256, 0, s,
                  static_cast<float *>(out), n_steps, freq);
  else
    launch_kernel(time_sinus_kernel<bf16>, grid, 256, 0, s,
                  static_cast<bf16 *>(out), n_steps, freq);
  return hipGetLastError();
}

hipError_t launch_silu_cond(DType dt, void *sc, const float *cond, const float *temb, int32_t rows,
                            int32_t width, hipStream_t s) {
  const int n4 = rows * (width / 4);
  if (n4 == 0) return hipSuccess;
  if (width % 4 != 0) return hipErrorInvalidValue;
  const int grid = (n4 + 255) / 256;
  if (dt == DType::F32)
    launch_kernel(silu_cond_kernel<float>, grid, 256, 0, s,
                  static_cast<float *>(sc), cond, temb, rows, width);
  else
    launch_kernel(silu_cond_kernel<bf16>, grid, 256, 0, s,
                  static_cast<bf16 *>(sc), cond, temb, rows, width);
  return hipGetLastError();
}

template <typename T, int NV>
static void head_in_mod_dispatch(int grid, hipStream_t s, T *a, float *h, const float *x,
                                 const float *w_in_t, const float *b_in, const T *mod, int mod_ld,
                                 int rows, int c, float eps) {
#define E_(CM) launch_kernel(head_in_mod_kernel<T, NV, CM>, grid, 256, 0, s, a, h, x, w_in_t, b_in, mod, mod_ld, \
                                                                 rows, c, eps)
  if (c <= 4) E_(4);
  else if (c <= 8) E_(8);
  else if (c <= 16) E_(16);
  else if (c <= 32) E_(32);
  else E_(64);
#undef E_
}

hipError_t launch_transpose_f32(float *w_t, const float *w, int32_t rows, int32_t cols,
                                hipStream_t s) {
  const int n = rows * cols;
  if (n == 0) return hipSuccess;
  launch_kernel(transpose_f32_kernel, (n + 255) / 256, 256, 0, s, w_t, w, rows, cols);
  return hipGetLastError();
}

hipError_t launch_head_in_mod(DType dt, void *a, float *h, const float *x, const float *w_in_t,
                              const float *b_in, const void *mod, int32_t mod_ld, int32_t rows,
                              int32_t width, int32_t c_tok, float eps, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (width % 256 != 0 || c_tok < 1 || c_tok > 64) return hipErrorInvalidValue;
  const int grid = (rows + 3) / 4;
  if (dt == DType::F32) {
#define L_(NV)                                                                                \
  head_in_mod_dispatch<float, NV>(grid, s, static_cast<float *>(a), h, x, w_in_t, b_in,          \
                                  static_cast<const float *>(mod), mod_ld, rows, c_tok, eps)
    MARCHE_NV_SWITCH(width / 256, L_)
#undef L_
  } else {
#define L_(NV)                                                                              \
  head_in_mod_dispatch<bf16, NV>(grid, s, static_cast<bf16 *>(a), h, x, w_in_t, b_in,          \
                                 static_cast<const bf16 *>(mod), mod_ld, rows, c_tok, eps)
    MARCHE_NV_SWITCH(width / 256, L_)
#undef L_
  }
  return hipGetLastError();
}

hipError_t launch_head_gate_mod(DType dt, void *a, float *h, const float *t, const void *mod,
                                int32_t mod_ld, int32_t gate_off, int32_t shift_off,
                                int32_t scale_off, int32_t rows, int32_t width, float eps,
                                hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (width % 256 != 0) return hipErrorInvalidValue;
  const int grid = (rows + 3) / 4;
  if (dt == DType::F32) {
#define L_(NV)                                                                              \
  launch_kernel(head_gate_mod_kernel<float, NV>, grid, 256, 0, s, static_cast<float *>(a), h, t,          \
                                                       static_cast<const float *>(mod), mod_ld, \
                                                       gate_off, shift_off, scale_off, rows, eps)
    MARCHE_NV_SWITCH(width / 256, L_)
#undef L_
  } else {
#define L_(NV)                                                                            \
  launch_kernel(head_gate_mod_kernel<bf16, NV>, grid, 256, 0, s, static_cast<bf16 *>(a), h, t,          \
                                                      static_cast<const bf16 *>(mod), mod_ld, \
                                                      gate_off, shift_off, scale_off, rows, eps)
    MARCHE_NV_SWITCH(width / 256, L_)
#undef L_
  }
  return hipGetLastError();
}

template <typename T>
static void head_out_step_dispatch(int grid, hipStream_t s, float *x_next, float *tok_out,
                                   const T *a, const float *w_out, const float *b_out,
                                   const float *x_cur, const float *noise, const int32_t *out_rows,
                                   int rows, int W, int c, const HeadStep &st) {
#define E_(CM)                                                                                 \
  launch_kernel(head_out_step_kernel<T, CM>, grid, 256, 0, s, x_next, tok_out, a, w_out, b_out, x_cur, noise, \
                                                   out_rows, rows, W, c, st.sra, st.srm1, st.c1,   \
                                                   st.c2, st.sigma)
  if (c <= 4) E_(4);
  else if (c <= 8) E_(8);
  else if (c <= 16) E_(16);
  else if (c <= 32) E_(32);
  else E_(64);
#undef E_
}

hipError_t launch_head_out_step(DType dt, float *x_next, float *tok_out, const void *a,
                                const float *w_out, const float *b_out, const float *x_cur,
                                const float *noise, const int32_t *out_rows, int32_t rows,
                                int32_t width, int32_t c_tok, const HeadStep &st, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (width % 256 != 0 || c_tok < 1 || c_tok > 64) return hipErrorInvalidValue;
  const int grid = (rows + 3) / 4;
  if (dt == DType::F32)
    head_out_step_dispatch(grid, s, x_next, tok_out, static_cast<const float *>(a), w_out, b_out,
                           x_cur, noise, out_rows, rows, width, c_tok, st);
  else
    head_out_step_dispatch(grid, s, x_next, tok_out, static_cast<const bf16 *>(a), w_out, b_out,
                           x_cur, noise, out_rows, rows, width, c_tok, st);
  return hipGetLastError();
}

#undef MARCHE_NV_SWITCH

}  // namespace marche
