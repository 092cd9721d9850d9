// Internal declarations shared by the host API and the HIP kernels of
// libmarche.so.  Not part of the public ABI (include/marche.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace marche {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Where active row r of the packed activations lives: image b, token tok,
// and its row in the [batch][n_tokens][d_model] residual stream.
struct RowMap {
  int32_t x_row;  // b * n_tokens + tok
  int32_t b;
  int32_t tok;
  int32_t pad;
};

// Kernel timing of the library's profiling mode (marche_profile_*): while a
// timed call runs on a thread, the first kernel it launches through
// launch_kernel() (device_common.h) carries the call's two events on its
// dispatch (hipExtLaunchKernel), so they hold the kernel's own start and end,
// not the stream's dispatch gap before it.
struct KernelEvents {
  hipEvent_t start = nullptr, stop = nullptr;
  bool used = false;
};
// This thread's slot: the timed call in progress, or nullptr.
KernelEvents *&kernel_events();

// Element type of the packed activations, weights and KV cache.
enum class DType { F32 = 0, BF16 = 1 };

// ---- elementwise / indexing (k_elementwise.hip) ----
hipError_t launch_row_map(RowMap *map, const int32_t *a_idx, const int32_t *a_off, int32_t batch,
                          int32_t n_tokens, hipStream_t s);
hipError_t launch_gather_ln(DType dt, void *out, const float *x, const RowMap *map, const float *g,
                            const float *b, int32_t rows, int32_t d_model, float eps, hipStream_t s);
hipError_t launch_decoder_input(float *x, const float *cls, const float *value, const float *mask,
                                const float *pos, const int32_t *rank, int32_t batch,
                                int32_t n_tokens, int32_t n_buf, int32_t d_model, int32_t n_known,
                                hipStream_t s);
hipError_t launch_fill_zero(void *dst, size_t bytes, hipStream_t s);
// Debug-mode check of a step's active lists; report[0] = 0 or 1 + code*batch + image
// (codes: 0 offsets, 1 token range, 2 duplicate token, 3 n_gen).
hipError_t launch_check_active(const int32_t *a_idx, const int32_t *a_off, const int32_t *n_gen,
                               int32_t batch, int32_t n_tokens, int32_t a_total, int32_t a_max,
                               int32_t gen_max, int32_t *report, hipStream_t s);

// ---- the rest of a MAR step (k_mar.hip) ----
// Encoder input rows [batch][n_buf + n_known][d_model] (Eq. 1).
hipError_t launch_encoder_input(float *x, const float *cls, const float *tok, const float *w_z,
                                const float *b_z, const float *pe, const int32_t *known,
                                int32_t batch, int32_t n_buf, int32_t n_img, int32_t n_known,
                                int32_t d_model, int32_t c_tok, hipStream_t s);
// Masked rows of the decoder input (Eq. 2).
hipError_t launch_mask_fill(float *x, const float *mask, const float *pe, const int32_t *rank,
                           int32_t batch, int32_t n_tokens, int32_t n_buf, int32_t n_known,
                           int32_t d_model, hipStream_t s);
// out[r] = LN(x[rows ? rows[r] : r]) * g + b (+ add[src % n_tokens - n_buf]).
hipError_t launch_ln_rows(DType dt, void *out, const float *x, const int32_t *rows_idx,
                          const float *g, const float *b, const float *add, int32_t rows,
                          int32_t n_tokens, int32_t n_buf, int32_t d_model, float eps,
                          hipStream_t s);
// Sinusoidal time embedding table [n_steps][freq].
hipError_t launch_time_sinus(DType dt, void *out, int32_t n_steps, int32_t freq, hipStream_t s);
// sc = SiLU(cond + temb_row), [rows][width].
hipError_t launch_silu_cond(DType dt, void *sc, const float *cond, const float *temb, int32_t rows,
                            int32_t width, hipStream_t s);
// w_t = w^T for a [rows][cols] float32 matrix.
hipError_t launch_transpose_f32(float *w_t, const float *w, int32_t rows, int32_t cols,
                                hipStream_t s);
// h = w_in x + b_in (w_in given transposed, [C][W]); a = LN(h) (1 + scale) +
// shift with block 0's modulation.
hipError_t launch_head_in_mod(DType dt, void *a, float *h, const float *x, const float *w_in_t,
                              const float *b_in, const void *mod, int32_t mod_ld, int32_t rows,
                              int32_t width, int32_t c_tok, float eps, hipStream_t s);
// h += gate t; a = LN(h) (1 + scale) + shift (slices of mod at the offsets).
hipError_t launch_head_gate_mod(DType dt, void *a, float *h, const float *t, const void *mod,
                                int32_t mod_ld, int32_t gate_off, int32_t shift_off,
                                int32_t scale_off, int32_t rows, int32_t width, float eps,
                                hipStream_t s);
// Coefficients of one DDPM step (see head_out_step_kernel).
struct HeadStep {
  float sra, srm1, c1, c2, sigma;
};
hipError_t launch_head_out_step(DType dt, float *x_next, float *tok_out, const void *a,
                                const float *w_out, const float *b_out, const float *x_cur,
                                const float *noise, const int32_t *out_rows, int32_t rows,
                                int32_t width, int32_t c_tok, const HeadStep &st, hipStream_t s);

// ---- GEMMs with fused epilogues (k_gemm.hip) ----
// C[M][N] = A[M][K] . W[N][K]^T (+ bias) followed by one epilogue:
//   qkv:   columns [0,D) -> q [M][D]; [D,2D) -> K cache, [2D,3D) -> V cache
//          (scattered to [b][h][tok][d] of one layer's cache)
//   resid: x[map[r].x_row][c] += C + bias        (float32 residual stream)
//   gelu:  h[r][c] = GELU(C + bias)
struct QkvOut {
  void *q;
  void *k_cache;  // layer base
  void *v_cache;  // layer base
  int32_t d_model, head_dim, n_heads, n_tokens;
};
hipError_t launch_gemm_qkv(DType dt, const void *a, const void *w, const float *bias, int32_t m,
                           int32_t n, int32_t k, const RowMap *map, QkvOut out, hipStream_t s);
// tag: 0 = output projection, 1 = fc2 (separate kernel symbols)
hipError_t launch_gemm_resid(DType dt, const void *a, const void *w, const float *bias, int32_t m,
                             int32_t n, int32_t k, const RowMap *map, float *x, int32_t tag,
                             hipStream_t s);
hipError_t launch_gemm_gelu(DType dt, const void *a, const void *w, const float *bias, int32_t m,
                            int32_t n, int32_t k, void *h, hipStream_t s);
// Sampler GEMMs: out[r][c] = act(C + bias) as out_dt (row-major, ld = n), act
// SiLU or the identity; a float32 GEMM writes float32 only.
hipError_t launch_gemm_plain(DType dt, const void *a, const void *w, const float *bias, int32_t m,
                             int32_t n, int32_t k, void *out, DType out_dt, bool silu_act,
                             hipStream_t s);
// Decoder embedding of the encoder rows scattered to their sequence positions
// (n = d_model): x[b][j][c] = C + bias + pe[j][c], j the position encoder row
// r = b * n_enc + i holds (i < n_buf: i; else n_buf + known[b][i - n_buf]).
hipError_t launch_gemm_embed(DType dt, const void *a, const void *w, const float *bias, int32_t m,
                             int32_t n, int32_t k, float *x, const float *pe, const int32_t *known,
                             int32_t n_enc, int32_t n_buf, int32_t n_known, int32_t n_tokens,
                             hipStream_t s);
// bf16 GEMM workgroup tile for an M x N x K product: 128x256 (two workgroups
// per CU), 256x256 or 320x256 (one per CU), 128x128 (narrow products on a few
// thousand rows) or 64x128 (small products).
enum GemmTile {
  GEMM_TILE_128x256 = 0, GEMM_TILE_256 = 1, GEMM_TILE_64x128 = 2, GEMM_TILE_128 = 3,
  GEMM_TILE_320 = 4
};
int gemm_tile_kind(DType dt, int32_t m, int32_t n, int32_t k);
// Compute units of the current device (queried once per device, then cached).
int device_cu_count();

// ---- attention (k_attn.hip) ----
struct AttnArgs {
  const void *q;        // [a_total][D] packed queries
  const void *k_cache;  // layer base [B][H][N][dh] (keys 0..N-1; the first segment)
  const void *v_cache;
  void *o;              // [a_total][D]
  const int32_t *a_off; // CSR rows per image; NULL: image b owns rows [b*a_max, (b+1)*a_max)
  const RowMap *map;
  int32_t batch, n_heads, n_tokens, head_dim, d_model, a_total, a_max;
  // Optional second key/value segment [B][H][n2][dh], attended after the
  // first in the same online-softmax pass (bf16 attention only).
  const void *k2 = nullptr;
  const void *v2 = nullptr;
  int32_t n2 = 0;
  // Optional attention mass of the generating rows (the first n_gen[b] rows
  // of image b), scores[b][h][j], written by the same kernel where
  // attn_fuses_scores() holds (one key segment).
  const int32_t *n_gen = nullptr;
  float *scores = nullptr;
};
hipError_t launch_attention(DType dt, const AttnArgs &a, hipStream_t s);
// Whether bf16 attention with these sizes runs the resident-K/V kernel (one
// workgroup per (image, head)).
bool attn_resident(int32_t a_max, int32_t n_tokens, bool two_segments);
// Whether bf16 attention with these sizes runs the register-staged streaming
// kernel (head width 64, one key segment of whole tiles).
bool attn_streams(int32_t head_dim, int32_t n_tokens, bool two_segments);
// Whether bf16 attention with these sizes can write the score pass itself:
// the resident kernel (every key of a head in LDS), or the streaming kernel
// when the generating rows fit its first query chunk.
bool attn_fuses_scores(int32_t a_max, int32_t n_tokens, int32_t head_dim, int32_t gen_max);
// dst[b][h] = [a[b][h] (na rows) ; c[b][h] (nc rows)], rows of dh elements, for
// K and V: the concatenation of the active and cached segments.
hipError_t launch_concat_kv(DType dt, void *k_dst, void *v_dst, const void *k_a, const void *v_a,
                            const void *k_c, const void *v_c, int32_t bh, int32_t na, int32_t nc,
                            int32_t head_dim, hipStream_t s);
// scores[b][h][j] = sum over the first n_gen[b] active rows i of P_h[i][j]
hipError_t launch_attn_scores(DType dt, const AttnArgs &a, const int32_t *n_gen, int32_t gen_max,
                              float *scores, hipStream_t s);

// ---- selection (k_select.hip) ----
// lowest = false: highest scores first; true: lowest scores first.
hipError_t launch_select_topk(const float *scores, int32_t n_parts, const int32_t *excl_idx,
                              const int32_t *excl_off, int32_t batch, int32_t n_tokens, int32_t k,
                              int32_t *out_idx, const int32_t *out_off, bool lowest,
                              hipStream_t s);

}  // namespace marche
