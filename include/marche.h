/*
 * marche.h -- C ABI of libmarche.so: MARche's cache-aware decode step on
 * AMD Instinct MI355X (gfx950).
 *
 * MARche (cache-aware attention with selective KV refresh) speeds up the
 * decoder of masked autoregressive image generation.  At each decoding step
 * only the *active* tokens A = G u N u R (generating tokens G, caching tokens
 * N generated one step earlier, refreshing tokens R) are projected; their
 * fresh keys/values overwrite a per-layer, per-image KV cache; every active
 * query attends over all N tokens (fresh K/V at A, cached K/V elsewhere); the
 * output projection and the MLP run on the active rows only (Algorithm 1,
 * Section 4.1).  R is chosen by the attention mass the generating tokens put
 * on each token at a selection layer, summed over heads, top-k (Section 4.2).
 *
 * Conventions for every entry point:
 *  - All tensors are caller-owned device memory (hipMalloc / torch).  The
 *    library keeps no pointer after a call returns and allocates no device
 *    memory; scratch space is the caller's `workspace`.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t passed as a
 *    void*; NULL = the default stream).  No entry point synchronises the
 *    host, except where stated.
 *  - Host-side validation runs before any HIP call.  Errors are returned as a
 *    marche_status_t, never thrown and never an abort; marche_last_error()
 *    then returns a thread-local message naming the offending argument.
 *  - Device-side index lists (a_idx, excl_idx, ...) are preconditions: their
 *    values are not read on the host.
 *  - Block parameters: matrices are in nn.Linear layout [out][in] and in the
 *    model dtype; LayerNorm gains/shifts and biases are float32 vectors.
 *  - The residual stream x is always float32; the KV cache uses the model
 *    dtype.  bf16 values are IEEE bfloat16; fp32->bf16 rounds to nearest even.
 */
#ifndef MARCHE_H
#define MARCHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MARCHE_OK = 0,
  MARCHE_ERR_INVALID_ARG = 1, /* null pointer, inconsistent shape, bad range */
  MARCHE_ERR_UNSUPPORTED = 2, /* valid but not implemented (dtype, head_dim, width) */
  MARCHE_ERR_HIP = 3,         /* a HIP launch or runtime call failed */
  MARCHE_ERR_WORKSPACE = 4    /* workspace missing or smaller than required */
} marche_status_t;

typedef enum { MARCHE_F32 = 0, MARCHE_BF16 = 1 } marche_dtype_t;

/* Opaque HIP stream (hipStream_t). */
typedef void *marche_stream_t;

/* Shape of the decoder stack.  Pre-LN bidirectional blocks:
 *   x += W_o . Attn(LN1(x)) + b_o;   x += W_2 . GELU(W_1 . LN2(x) + b_1) + b_2,
 * LayerNorm with population variance and eps inside the square root,
 * exact-erf GELU, attention scale 1/sqrt(head_dim).
 * Supported: d_model == n_heads * head_dim, d_model % 256 == 0,
 * d_model <= 2048, head_dim in {64, 80}, d_mlp % 256 == 0,
 * 1 <= n_tokens <= 4096. */
typedef struct {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;
  int32_t head_dim;
  int32_t d_mlp;
  int32_t n_tokens;
  int32_t dtype; /* marche_dtype_t */
  float ln_eps;
} marche_model_t;

/* Parameters of one block (device pointers).
 * w_qkv [3D][D]: rows [0,D) queries, [D,2D) keys, [2D,3D) values; inside each
 * third head h owns rows [h*head_dim, (h+1)*head_dim).  b_qkv [3D] f32.
 * w_o [D][D], b_o [D] f32; w_1 [F][D], b_1 [F] f32; w_2 [D][F], b_2 [D] f32;
 * ln1_g/ln1_b/ln2_g/ln2_b [D] f32. */
typedef struct {
  const void *ln1_g, *ln1_b;
  const void *w_qkv, *b_qkv;
  const void *w_o, *b_o;
  const void *ln2_g, *ln2_b;
  const void *w_1, *b_1;
  const void *w_2, *b_2;
} marche_layer_t;

/* Per-layer, per-image KV cache C (Algorithm 1's cache).  k and v each hold
 * [n_layers][batch][n_heads][n_tokens][head_dim] elements of `dtype`. */
typedef struct {
  void *k;
  void *v;
  int32_t n_layers, batch, n_heads, n_tokens, head_dim;
  int32_t dtype; /* marche_dtype_t */
} marche_kv_cache_t;

/* Bind caller buffers k_buf / v_buf (bytes_each bytes each, at least
 * n_layers*batch*n_heads*n_tokens*head_dim elements) as the cache of `m` for
 * `batch` images and fill it: copied from k_init / v_init (device, same layout)
 * when given, else zero.  The first decoding step runs every layer with all
 * tokens active, which writes every cache row before any is read (Section
 * 4.3's initial full step).  Returns INVALID_ARG on null or short buffers. */
marche_status_t kv_cache_init(marche_kv_cache_t *cache, const marche_model_t *m, int32_t batch,
                              void *k_buf, void *v_buf, size_t bytes_each, const void *k_init,
                              const void *v_init, marche_stream_t stream);

/* Bytes of workspace marche_step needs for `a_total` active rows in total. */
size_t marche_step_workspace_bytes(const marche_model_t *m, int32_t batch, int32_t a_total);

/* Run layers [layer_begin, layer_end) of the stack the cache-aware way
 * (Algorithm 1) for `batch` images.
 *
 * Active set (device, CSR over images): image b's active tokens are
 * a_idx[a_off[b] .. a_off[b+1]), distinct values in [0, n_tokens); the first
 * n_gen[b] of them are the generating tokens.  a_total = a_off[batch],
 * a_max = max_b |A_b| and gen_max = max_b n_gen[b] are host copies used for
 * launch geometry (they must match the device arrays).  A full-attention
 * layer is the same call with every token active.
 *
 * Per layer l and image b:
 *   u      = LN1(x[b][i]) for i in A_b
 *   q|k|v  = u W_qkv^T + b_qkv
 *   cache.k[l][b][h][i] = k_h, cache.v[l][b][h][i] = v_h   (i in A_b; other rows untouched)
 *   o_i    = sum_j softmax_j(q_i . K[j] / sqrt(d_h)) V[j] over all n_tokens keys
 *   x[b][i] += o_i W_o^T + b_o;   x[b][i] += W_2 GELU(W_1 LN2(x[b][i]) + b_1) + b_2
 * Rows of x and of the cache outside A_b are neither read by the MLP nor
 * written.  x is [batch][n_tokens][d_model] float32, updated in place.
 * batch*n_tokens*d_model and a_total*max(3*d_model, d_mlp) must stay below
 * 2^31 (UNSUPPORTED otherwise).
 *
 * Scores (Section 4.2): when `scores` is non-NULL and score_layer lies in
 * [layer_begin, layer_end), that layer also writes
 *   scores[b][h][j] = sum over the generating rows i of P_h[i][j]
 * (post-softmax attention probabilities) for every key j, float32
 * [batch][n_heads][n_tokens], overwriting the buffer.
 *
 * `layers` is a host array of n_layers entries; `workspace` holds at least
 * marche_step_workspace_bytes(m, batch, a_total) bytes of device memory and
 * must not be used by another call in flight.
 *
 * The device lists are preconditions the host cannot see.  With the
 * environment variable MARCHE_VALIDATE set (to anything but "0"), the call
 * first checks them with a kernel and waits for the result on the host:
 * a_off[0] = 0, a_off[batch] = a_total, non-decreasing, no list longer than
 * a_max; every token in [0, n_tokens) and none twice for one image; n_gen[b]
 * within [0, |A_b|] and at most gen_max.  A violation returns INVALID_ARG,
 * naming one problem found and its image (the first recorded, when several
 * images are bad), before anything else is launched.  Without it nothing is checked on the device and the call never
 * synchronises. */
marche_status_t marche_step(const marche_model_t *m, const marche_layer_t *layers,
                            const marche_kv_cache_t *cache, int32_t layer_begin,
                            int32_t layer_end, int32_t batch, float *x, const int32_t *a_idx,
                            const int32_t *a_off, const int32_t *n_gen, int32_t a_total,
                            int32_t a_max, int32_t gen_max, float *scores, int32_t score_layer,
                            void *workspace, size_t workspace_bytes, marche_stream_t stream);

/* marche_step over images [first_image, first_image + batch) of `cache`
 * (Algorithm 1 runs per image, so any group of images is a step of its
 * own).  x, a_idx / a_off / n_gen, scores and the workspace describe only
 * those images: image first_image of the cache is image 0 of the call, a_off
 * starts at 0, x points at that image's [n_tokens][d_model] rows and scores
 * (if any) at its [n_heads][n_tokens] block.  The cache's other images are
 * neither read nor written, so calls on disjoint image ranges may run
 * concurrently on different streams, each with its own workspace.
 * marche_step is this call with first_image = 0.  Returns INVALID_ARG when
 * the range leaves the cache, otherwise as marche_step. */
marche_status_t marche_step_images(const marche_model_t *m, const marche_layer_t *layers,
                                   const marche_kv_cache_t *cache, int32_t first_image,
                                   int32_t layer_begin, int32_t layer_end, int32_t batch, float *x,
                                   const int32_t *a_idx, const int32_t *a_off,
                                   const int32_t *n_gen, int32_t a_total, int32_t a_max,
                                   int32_t gen_max, float *scores, int32_t score_layer,
                                   void *workspace, size_t workspace_bytes,
                                   marche_stream_t stream);

/* Size of the library's own step workspace, used by
 * marche_step_images_noalloc: 64 MiB of device memory per GPU the library
 * runs that entry point on, held until the process ends. */
#define MARCHE_SCRATCH_BYTES ((size_t)64 << 20)

/* marche_step_images without a caller workspace and without any allocation,
 * for callers that cannot allocate device memory: code under HIP graph
 * capture, serving loops that must not call hipMalloc, harnesses that forbid
 * it.  The step's workspace is a library-owned static device array of
 * MARCHE_SCRATCH_BYTES, one per GPU; its device address is looked up once
 * per device (hipGetSymbolAddress, with that device current) on the first
 * call there.  Arguments, layout, results and errors are those of
 * marche_step_images; additionally returns MARCHE_ERR_WORKSPACE, before any
 * HIP call, when marche_step_workspace_bytes(m, batch, a_total) exceeds
 * MARCHE_SCRATCH_BYTES (at d_model 1024 and d_mlp 4096 about 5400 active
 * rows), and MARCHE_ERR_HIP if the lookup fails.  Nothing in the array needs
 * to start at zero: every call writes each part of it before reading it.
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * contents, so calls that overlap on one GPU (two host threads, or two
 * streams without an ordering between them) race; order them on one stream.
 * Calls no hipMalloc, hipFree or other allocating routine (with kernel
 * timing switched on, marche_profile_enable, the library creates HIP events). */
marche_status_t marche_step_images_noalloc(const marche_model_t *m, const marche_layer_t *layers,
                                           const marche_kv_cache_t *cache, int32_t first_image,
                                           int32_t layer_begin, int32_t layer_end, int32_t batch,
                                           float *x, const int32_t *a_idx, const int32_t *a_off,
                                           const int32_t *n_gen, int32_t a_total, int32_t a_max,
                                           int32_t gen_max, float *scores, int32_t score_layer,
                                           marche_stream_t stream);

/* Refresh selection (Section 4.2, top-k of the head-aggregated scores).
 * For each image b: s_j = sum_{p < n_parts} scores[b][p][j] (summed in p
 * order, float32); candidates are the tokens not in
 * excl_idx[excl_off[b] .. excl_off[b+1]); the k candidates with the highest
 * s_j are chosen, equal scores going to the lower token index and NaN ranking
 * below every number; they are written in ascending token order to
 * out_idx[out_off[b] .. out_off[b]+k).  If an image has fewer than k
 * candidates the missing slots are written as -1.
 * Requires 0 <= k <= n_tokens <= 4096, n_parts >= 1. */
marche_status_t select_refresh(const float *scores, int32_t n_parts, const int32_t *excl_idx,
                               const int32_t *excl_off, int32_t batch, int32_t n_tokens,
                               int32_t k, int32_t *out_idx, const int32_t *out_off,
                               marche_stream_t stream);

/* Order of a refresh selection: the highest head-aggregated attention mass
 * (Section 4.2, the method) or the lowest (the low-attention ablation of the
 * refresh-strategy study, Table 3). */
typedef enum { MARCHE_SELECT_HIGHEST = 0, MARCHE_SELECT_LOWEST = 1 } marche_select_order_t;

/* select_refresh with an explicit order.  MARCHE_SELECT_LOWEST picks the k
 * candidates with the lowest s_j, equal scores going to the lower token index
 * and NaN ranking after every number; the output is ascending as for
 * select_refresh, which equals this call with MARCHE_SELECT_HIGHEST.  Returns
 * INVALID_ARG for any other order value. */
marche_status_t select_refresh_ordered(const float *scores, int32_t n_parts,
                                       const int32_t *excl_idx, const int32_t *excl_off,
                                       int32_t batch, int32_t n_tokens, int32_t k,
                                       int32_t *out_idx, const int32_t *out_off, int32_t order,
                                       marche_stream_t stream);

/* Decoder input of one step (stand-in for Eq. 2's concatenation of encoder
 * features and mask embeddings with positional encodings):
 *   x[b][j] = pos[j] + cls[b]                      for j <  n_buf,
 *   x[b][j] = pos[j] + value[b][j-n_buf]           for j >= n_buf, rank[b][j-n_buf] <  n_known,
 *   x[b][j] = pos[j] + mask                        otherwise,
 * where rank[b][p] is the position of image token p in image b's generation
 * order, so the tokens generated before the step are those with rank below
 * n_known.  All float32 except rank (int32 [batch][n_tokens-n_buf]);
 * cls [batch][D], value [batch][n_tokens-n_buf][D], mask [D], pos [n_tokens][D]. */
marche_status_t marche_decoder_input(float *x, const float *cls, const float *value,
                                     const float *mask, const float *pos, const int32_t *rank,
                                     int32_t batch, int32_t n_tokens, int32_t n_buf,
                                     int32_t d_model, int32_t n_known, marche_stream_t stream);

/* ---- Appendix B: attention over an active and a cached segment ----
 * For each image b and head h, the n_query query rows attend over the keys
 * [K_A ; K_C] -- the n_a keys of the active segment followed by the n_c keys
 * of the cached segment -- and the same values:
 *   o[b][i][h] = sum_j softmax_j(q[b][i][h] . K[b][h][j] / sqrt(head_dim)) V[b][h][j].
 * (In Appendix B's setting n_query = n_a: the active tokens are the queries.)
 * Layouts (bf16, 16-byte aligned): q and o [batch][n_query][n_heads*head_dim];
 * k_a, v_a [batch][n_heads][n_a][head_dim]; k_c, v_c [batch][n_heads][n_c][head_dim];
 * a segment of length 0 may pass NULL.
 *
 * MARCHE_ATTN_TWO_SEGMENT: one pass reads the key tiles of K_A and then of K_C
 *   from their own buffers and merges them with a running maximum and a
 *   rescaled running sum (Appendix A's online-softmax merge; nothing is
 *   copied).  Needs no workspace.  With n_c = 0 it is attention over one
 *   resident buffer, the layout marche_step uses.
 * MARCHE_ATTN_CONCAT: the baseline Appendix B compares against: K_A and K_C
 *   (and V_A, V_C) are first concatenated into the workspace, then the same
 *   attention runs over one segment of n_a + n_c keys.
 * The two modes differ only in rounding (the key tiles fall differently).
 * head_dim in {64, 80}, 1 <= n_query <= 4096, n_a, n_c >= 0 with
 * 1 <= n_a + n_c <= 65536, batch * n_heads <= 65535; UNSUPPORTED for other dtypes or head widths;
 * WORKSPACE when CONCAT's workspace (marche_attention_workspace_bytes,
 * 256-byte aligned) is missing or short. */
typedef enum { MARCHE_ATTN_TWO_SEGMENT = 0, MARCHE_ATTN_CONCAT = 1 } marche_attn_mode_t;

size_t marche_attention_workspace_bytes(int32_t batch, int32_t n_heads, int32_t head_dim,
                                         int32_t n_a, int32_t n_c, int32_t dtype, int32_t mode);

marche_status_t marche_attention_segments(const void *q, void *o, int32_t n_query,
                                          const void *k_a, const void *v_a, int32_t n_a,
                                          const void *k_c, const void *v_c, int32_t n_c,
                                          int32_t batch, int32_t n_heads, int32_t head_dim,
                                          int32_t dtype, int32_t mode, void *workspace,
                                          size_t workspace_bytes, marche_stream_t stream);

/* ---- The rest of a MAR step: encoder input, decoder input, sampler ----
 * These calls surround marche_step to make a whole generation step of the
 * masked autoregressive model: the encoder over the known tokens (Eq. 1), the
 * decoder input built from its output (Eq. 2), and the sampler that draws
 * the generating tokens' values from the decoder output (Eq. 3).  The encoder
 * blocks themselves are marche_step over a model whose n_tokens is the
 * encoder's row count n_buf + n_known, with every row active; its cache is
 * scratch that every layer overwrites before reading, so the caller may
 * describe it with a marche_kv_cache_t filled directly (no kv_cache_init).
 * Image tokens are numbered p in [0, n_img); sequence position of image
 * token p is n_buf + p, the n_buf buffer rows come first.  Known tokens are
 * those with rank[b][p] < n_known, rank being the position of p in image b's
 * generation order. */

/* Encoder input rows (Eq. 1), x_enc [batch][n_buf + n_known][d_model] float32:
 *   row i < n_buf:  cls[b] + pe_enc[i]                      (buffer rows)
 *   row n_buf + r:  w_z . tok[b][p] + b_z + pe_enc[n_buf + p],  p = known[b][r]
 * cls [batch][d_model]; tok [batch][n_img][c_tok]; w_z [d_model][c_tok];
 * b_z [d_model]; pe_enc [n_buf + n_img][d_model]; known [batch][n_known]
 * int32 image tokens (device; any order, ascending is the encoder's usual
 * order).  All float32.  d_model a multiple of 256, <= 4096; 1 <= c_tok <= 64. */
marche_status_t marche_encoder_input(float *x_enc, const float *cls, const float *tok,
                                     const float *w_z, const float *b_z, const float *pe_enc,
                                     const int32_t *known, int32_t batch, int32_t n_buf,
                                     int32_t n_img, int32_t n_known, int32_t d_model,
                                     int32_t c_tok, marche_stream_t stream);

/* Decoder input from the encoder output (Eq. 2), x_dec [batch][n_buf + n_img][d_model]
 * float32, every row written:
 *   u = LN(x_enc) * ln_g + ln_b;  v = u . w_de^T + b_de   (per encoder row)
 *   x_dec[b][j] = v[encoder row of j] + pe_dec[j]  for buffer rows j < n_buf and
 *                 known tokens j = n_buf + known[b][r] (encoder row n_buf + r);
 *   x_dec[b][n_buf + p] = mask + pe_dec[n_buf + p]  for rank[b][p] >= n_known.
 * x_enc [batch][n_buf + n_known][d_model] float32; w_de [d_model][d_model] in
 * `dtype` (u is rounded to it); ln_g, ln_b, b_de, mask [d_model] and pe_dec
 * [n_buf + n_img][d_model] float32; known [batch][n_known], rank [batch][n_img]
 * int32 (device).  workspace: marche_encoder_to_decoder_workspace_bytes, 256-byte
 * aligned.  d_model a multiple of 256, <= 4096. */
size_t marche_encoder_to_decoder_workspace_bytes(int32_t batch, int32_t n_buf, int32_t n_known,
                                                 int32_t d_model, int32_t dtype);
marche_status_t marche_encoder_to_decoder(float *x_dec, const float *x_enc, const float *ln_g,
                                          const float *ln_b, float ln_eps, const void *w_de,
                                          const float *b_de, const float *mask,
                                          const float *pe_dec, const int32_t *known,
                                          const int32_t *rank, int32_t batch, int32_t n_buf,
                                          int32_t n_img, int32_t n_known, int32_t d_model,
                                          int32_t dtype, void *workspace, size_t workspace_bytes,
                                          marche_stream_t stream);

/* Sampler of Eq. 3: x_i ~ p(x_i | z_i; tau) for n_rows generating tokens.
 * Condition z_i = LN(x_dec[row_i]) * dec_ln_g + dec_ln_b + pe_diff[p_i]
 * (row_i = rows[i] = b * n_tokens + n_buf + p_i).  Denoiser eps(x, t, z), W = width:
 *   c = W_t2 SiLU(W_t1 sinus(t) + b_t1) + b_t2 + W_c z + b_c,  s = SiLU(c)
 *   [shift_k | scale_k | gate_k] = rows [3kW, 3kW + 3W) of W_ada s + b_ada,
 *   [shift_f | scale_f] = rows [3nW, 3nW + 2W)            (n = n_blocks)
 *   h = W_in x + b_in;  for k < n: h += gate_k * (W_2k SiLU(W_1k (LN(h)(1 + scale_k) + shift_k) + b_1k) + b_2k)
 *   eps = W_out (LN(h)(1 + scale_f) + shift_f) + b_out
 * with LN without affine (eps head->ln_eps) and sinus(t) = [cos(t w_j) | sin(t w_j)],
 * w_j = 10000^(-j / (t_freq/2)).  DDPM ancestral sampling over n_steps steps of
 * the cosine schedule (alpha_bar(u) = cos^2((u + 0.008)/1.008 pi/2) normalised,
 * betas clipped at 0.999): x = noise[n_steps]; for i = n_steps-1 .. 0:
 *   x0 = (x - sqrt(1 - ab_i) eps(x, i, z)) / sqrt(ab_i),
 *   x = posterior mean(x0, x) + temperature * sqrt(posterior variance) * noise[i]
 * (no noise at i = 0); the final x goes to tok_out[out_rows[i]] (c_tok floats).
 * noise [n_steps + 1][n_rows][c_tok] float32 (caller-drawn, device);
 * rows, out_rows [n_rows] int32 (device).
 * Weights: w_t1 [W][t_freq], w_t2 [W][W], w_c [W][d_cond], w_ada [(3n+2)W][W],
 * w_1, w_2 [n][W][W] in head->dtype; w_in [W][c_tok], w_out [c_tok][W] and
 * every bias float32.  Supported: width and d_cond multiples of 256 (<= 4096),
 * t_freq a multiple of 64 (<= 4096), 1 <= n_blocks <= 64, 1 <= c_tok <= 64,
 * 1 <= n_steps <= 10000; n_rows * (3n+2) * width < 2^31.  workspace:
 * marche_diffusion_workspace_bytes, 256-byte aligned. */
typedef struct {
  int32_t width, n_blocks, c_tok, d_cond, t_freq;
  marche_dtype_t dtype;
  float ln_eps;
} marche_head_t;

typedef struct {
  const void *w_t1, *b_t1, *w_t2, *b_t2, *w_c, *b_c, *w_in, *b_in, *w_ada, *b_ada, *w_1, *b_1,
      *w_2, *b_2, *w_out, *b_out;
} marche_head_weights_t;

size_t marche_diffusion_workspace_bytes(const marche_head_t *head, int32_t n_rows,
                                        int32_t n_steps);
marche_status_t marche_diffusion_sample(const marche_head_t *head, const marche_head_weights_t *w,
                                        const float *x_dec, int32_t n_tokens, int32_t n_buf,
                                        const float *dec_ln_g, const float *dec_ln_b,
                                        float dec_ln_eps, const float *pe_diff,
                                        const int32_t *rows, const int32_t *out_rows,
                                        int32_t n_rows, const float *noise, int32_t n_steps,
                                        float temperature, float *tok_out, void *workspace,
                                        size_t workspace_bytes, marche_stream_t stream);

/* Name of a status code (static string). */
const char *marche_status_string(marche_status_t s);

/* Message of the calling thread's last non-OK return ("" if none). */
const char *marche_last_error(void);

/* ---- kernel timing (instrumentation; not needed to run the method) ----
 * While enabled, every kernel launched by this library on any stream is
 * bracketed by HIP events on its own stream, and its algorithmic work
 * (flops and bytes, from the launch shape) is recorded.
 * marche_profile_collect() synchronises those events (host sync), folds them
 * into per-kernel totals and returns the number of kernel classes;
 * marche_profile_entry() reads one.  marche_profile_reset() clears them.
 * A class is one kernel symbol; launches of the decoder step in layers where
 * not every token of every image is active (cache-aware layers) form classes
 * of their own, named with the suffix "_ca". */
marche_status_t marche_profile_enable(int32_t on);
int32_t marche_profile_collect(void);
marche_status_t marche_profile_entry(int32_t i, const char **name, int64_t *launches,
                                     double *total_ms, double *flops, double *bytes);
void marche_profile_reset(void);

#ifdef __cplusplus
}
#endif
#endif /* MARCHE_H */
