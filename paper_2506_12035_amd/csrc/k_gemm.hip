// GEMMs on the ragged active set with fused epilogues.
//
// C[M][N] = A[M][K] . W[N][K]^T: A is the packed activation of the active
// rows (M = active rows of all images, any value), W a weight in nn.Linear
// layout.  Both operands are K-contiguous, which is the layout MFMA wants for
// both sides.  The epilogue adds the bias and then either
//   - splits q|k|v: q to the packed query buffer, k and v scattered into the
//     layer's KV cache at [b][h][tok][d]           (QKV projection + cache write)
//   - adds into the float32 residual stream row     (output projection, fc2)
//   - applies exact GELU and stores the hidden row  (fc1)
//
// bf16 path (v_mfma_f32_32x32x16_bf16, fp32 accumulators): a 256x256 tile
// (one workgroup per CU; four wavefronts for K >= 2048, eight below) or a
// 320x256 tile (whole 320-token images per tile row, eight wavefronts) for
// shapes that fill the chip in whole waves, else a 128x256 tile of which two
// workgroups share a CU, or 128x128 / 64x128 tiles for narrow products.  All
// load operands straight from global memory into XOR-swizzled LDS stages and
// write back through LDS in row-major order.
//
// fp32 path: plain FMA, 64x64 tiles, 4x4 outputs per thread.
#include "device_common.h"

namespace marche {

// ------------------------------------------------------------------ epilogues
//
// Every epilogue works on four consecutive output columns col0..col0+3 of one
// row (col0 a multiple of 4), so each lane issues 8- or 16-byte stores.  Four
// consecutive columns never straddle a q|k|v third or a head (d_model and
// head_dim are multiples of 4).
//
// The write-back issues every load (row addressing data, biases, residual
// priors) before the stores it feeds: on this architecture the vector-memory
// counter also counts stores, so a load issued after a store would wait for
// the store's acknowledgement.

template <typename T>
__device__ __forceinline__ void store4(T *p, f32x4 v) {
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<f32x4 *>(p) = v;
  } else {
    bf16x4 pk = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
    *reinterpret_cast<bf16x4 *>(p) = pk;
  }
}

__device__ __forceinline__ f32x4 load_bias4(const float *bias, int col0) {
  return *reinterpret_cast<const f32x4 *>(bias + col0);
}

// Epilogue interface: row(r) per-row addressing data (may load the row map);
// col(c0) per-column addressing data for the four columns c0..c0+3, computed
// once per lane where the columns of a lane are fixed; bias4(c0); prior(row,
// col) the value the result is added to (residual epilogues); store(row, r,
// col, v) with v = acc + bias + prior.

template <typename T>
struct EpiQkv {
  static constexpr bool kPrior = false;
  T *q;
  T *kc;
  T *vc;
  const float *bias;
  const RowMap *map;
  int d_model, head_dim, n_heads, n_tokens;
  // 32-bit element offsets: the host limits every buffer to < 2^31 elements.
  // A row's offset in q and in a K/V cache layer, computed once per row when
  // the tile stages its row records, so the stores add instead of multiply.
  struct Row {
    uint32_t q_off;   // r * d_model
    uint32_t kv_off;  // (b * n_heads * n_tokens + tok) * head_dim
  };
  struct Col {
    T *base;       // q, or the K or V cache of the layer
    uint32_t off;  // column offset: c0 for q, h*n_tokens*head_dim + d for K/V
    bool is_q;
  };
  __device__ __forceinline__ Row row(int r) const {
    const RowMap m = map[r];
    return Row{(uint32_t)(r * d_model), (uint32_t)((m.b * n_heads * n_tokens + m.tok) * head_dim)};
  }
  // Which of q, K and V a column belongs to is decided once per wavefront:
  // every tile gives a wavefront a span of 64 or 128 columns aligned to its
  // width, and d_model is a multiple of 256, so no span crosses from one of
  // the three into the next.  The choice is then uniform (scalar) and the
  // stores take no divergent branches.
  __device__ __forceinline__ Col col(int c0) const {
    const int which = __builtin_amdgcn_readfirstlane(c0 < d_model ? 0 : c0 < 2 * d_model ? 1 : 2);
    if (which == 0) return Col{q, (uint32_t)c0, true};
    const int c = c0 - which * d_model;
    const int h = c / head_dim, d = c - h * head_dim;
    return Col{which == 1 ? kc : vc, (uint32_t)(h * n_tokens * head_dim + d), false};
  }
  __device__ __forceinline__ f32x4 bias4(int c0) const { return load_bias4(bias, c0); }
  __device__ __forceinline__ f32x4 prior(const Row &, const Col &) const { return f32x4{}; }
  __device__ __forceinline__ void store(const Row &m, int, const Col &c, f32x4 v) const {
    store4(c.base + (c.is_q ? m.q_off : m.kv_off) + c.off, v);
  }
};

// TAG only distinguishes the output projection (0) from fc2 (1) as kernel
// symbols, so per-kernel profiles can tell them apart.
template <int TAG>
struct EpiResid {
  static constexpr bool kPrior = true;
  float *x;
  const float *bias;
  const RowMap *map;
  int n;
  using Row = int32_t;  // element offset of the residual-stream row (< 2^31)
  using Col = int32_t;
  __device__ __forceinline__ Row row(int r) const { return map[r].x_row * n; }
  __device__ __forceinline__ Col col(int c0) const { return c0; }
  __device__ __forceinline__ f32x4 bias4(int c0) const { return load_bias4(bias, c0); }
  __device__ __forceinline__ f32x4 prior(const Row &xr, const Col &c) const {
    return *reinterpret_cast<const f32x4 *>(x + (uint32_t)(xr + c));
  }
  __device__ __forceinline__ void store(const Row &xr, int, const Col &c, f32x4 v) const {
    *reinterpret_cast<f32x4 *>(x + (uint32_t)(xr + c)) = v;
  }
};

template <typename T>
struct EpiGelu {
  static constexpr bool kPrior = false;
  T *h;
  const float *bias;
  int n;
  using Row = int32_t;
  using Col = int32_t;
  __device__ __forceinline__ Row row(int r) const { return r; }
  __device__ __forceinline__ Col col(int c0) const { return c0; }
  __device__ __forceinline__ f32x4 bias4(int c0) const { return load_bias4(bias, c0); }
  __device__ __forceinline__ f32x4 prior(const Row &, const Col &) const { return f32x4{}; }
  __device__ __forceinline__ void store(const Row &, int r, const Col &c, f32x4 v) const {
    f32x4 g = {gelu_erf(v[0]), gelu_erf(v[1]), gelu_erf(v[2]), gelu_erf(v[3])};
    store4(h + (uint32_t)(r * n + c), g);
  }
};

// Plain epilogue of the sampler's GEMMs: out[r][c] = act(C + bias) stored
// row-major as T (ld = n), act the identity or SiLU.
template <typename T, bool SILU>
struct EpiPlain {
  static constexpr bool kPrior = false;
  T *out;
  const float *bias;
  int n;
  using Row = int32_t;  // element offset of the output row (< 2^31, host-checked)
  using Col = int32_t;
  __device__ __forceinline__ Row row(int r) const { return r * n; }
  __device__ __forceinline__ Col col(int c0) const { return c0; }
  __device__ __forceinline__ f32x4 bias4(int c0) const { return load_bias4(bias, c0); }
  __device__ __forceinline__ f32x4 prior(const Row &, const Col &) const { return f32x4{}; }
  __device__ __forceinline__ void store(const Row &ro, int, const Col &c, f32x4 v) const {
    if constexpr (SILU) v = f32x4{silu(v[0]), silu(v[1]), silu(v[2]), silu(v[3])};
    store4(out + (uint32_t)(ro + c), v);
  }
};

// Decoder embedding of the encoder rows (Eq. 2): encoder row r of image
// b = r / n_enc holds buffer token i = r % n_enc (i < n_buf) or the known
// image token known[b][i - n_buf]; its result goes to that token's sequence
// position j in the float32 decoder input x [batch][n_tokens][n], plus the
// decoder's positional embedding pe[j].
struct EpiEmbed {
  static constexpr bool kPrior = true;
  float *x;
  const float *bias;
  const float *pe;
  const int32_t *known;
  int n, n_enc, n_buf, n_known, n_tokens;
  struct Row {
    int32_t x_off;   // (b * n_tokens + j) * n
    int32_t pe_off;  // j * n
  };
  using Col = int32_t;
  __device__ __forceinline__ Row row(int r) const {
    const int b = r / n_enc, i = r - b * n_enc;
    const int j = i < n_buf ? i : n_buf + known[b * n_known + (i - n_buf)];
    return Row{(b * n_tokens + j) * n, j * n};
  }
  __device__ __forceinline__ Col col(int c0) const { return c0; }
  __device__ __forceinline__ f32x4 bias4(int c0) const { return load_bias4(bias, c0); }
  __device__ __forceinline__ f32x4 prior(const Row &ro, const Col &c) const {
    return *reinterpret_cast<const f32x4 *>(pe + (uint32_t)(ro.pe_off + c));
  }
  __device__ __forceinline__ void store(const Row &ro, int, const Col &c, f32x4 v) const {
    *reinterpret_cast<f32x4 *>(x + (uint32_t)(ro.x_off + c)) = v;
  }
};

// Empty uses that pin loaded values to this point: without them the compiler
// sinks the loads into the row-guarded store blocks, one wait per block.
__device__ __forceinline__ void keep(const f32x4 &v) { asm volatile("" ::"v"(v)); }
__device__ __forceinline__ void keep(int32_t v) { asm volatile("" ::"v"(v)); }
__device__ __forceinline__ void keep(const RowMap &m) {
  asm volatile("" ::"v"(m.x_row), "v"(m.b), "v"(m.tok));
}

// ------------------------------------------------------------------ bf16 MFMA
//
// The MFMA A operand is a 32-row slice of W (output columns) and the B
// operand a 32-row slice of the activations (output rows), so each 32x32
// accumulator holds a block of C^T: lane l owns output row (l & 31) and, in
// register r, output column (r / 4) * 8 + (l / 32) * 4 + r % 4 -- four
// consecutive columns per group of four registers, which the epilogue stores
// together.

// Grouped tile order: GROUP consecutive tile rows sweep all tile columns
// together, so concurrently running workgroups share A rows and W columns.
template <int GROUP = 8>
__device__ __forceinline__ void tile_coords(int id, int tiles_m, int tiles_n, int &tm, int &tn) {
  const int per_group = GROUP * tiles_n;
  const int g = id / per_group;
  const int first_m = g * GROUP;
  const int gm = min(tiles_m - first_m, GROUP);
  const int in = id - g * per_group;
  tm = first_m + in % gm;
  tn = in / gm;
}

// ------------------------------------------------------------------ 256x256 tile
//
// For projections where every token is active: a 256x256x64 workgroup tile
// on four wavefronts of 128x128 (16 accumulators each, which live in the
// accumulation registers).  Operands go from global memory straight into LDS
// (global_load_lds_dwordx4: no staging registers, no LDS write instructions)
// as 32 KB stages of 256 rows x 64 k, 128-byte rows whose 16-byte chunks are
// permuted by an XOR with the row pair index, so the 16 rows one fragment
// read touches per chunk hit 16 distinct bank groups.  The activation rows,
// streamed from memory once per column tile, get three stages and are loaded
// two k-tiles ahead of use; the weight rows, shared by every tile and served
// from L2, get two and are loaded one k-tile ahead: all of the CU's 160 KB.
// Every MFMA is issued in a fixed slot with at most one memory operation
// beside it (sched_barrier): the eight fragment reads of the next k16 step,
// the sixteen loads of a k-tile and the barrier are spread over the 64 MFMAs
// of a k-tile.
namespace big {

constexpr int kStage = 32768;  // bytes per operand stage: 256 rows x 64 k
constexpr int kAStages = 3, kWStages = 2;
constexpr int kWBase = kAStages * kStage;               // weight stages start at 96 KB
constexpr int kSmem = (kAStages + kWStages) * kStage;   // 160 KB

struct Frag {
  bf16x8 x[4];  // activation rows (MFMA B operand)
  bf16x8 w[4];  // weight rows (MFMA A operand)
};

__device__ __forceinline__ void pin() { __builtin_amdgcn_sched_barrier(0); }

__device__ __forceinline__ int swz(int r, int kc) { return kc ^ ((r >> 1) & 7); }

// Load instruction q (0..31 per operand and k-tile, 8 per wavefront) moves
// 1 KB: rows 8q..8q+7 of the operand's 256-row block; lane l writes LDS bytes
// [16 l, 16 l + 16) of it, i.e. row 8q + l / 8 at physical chunk l % 8, which
// holds logical chunk swz(row, l % 8).  `stage` is the LDS byte address of the
// stage (wave-uniform, so M0 is set from a scalar register).  Activation rows
// past M repeat row M - 1 (their results are never stored).
__device__ __forceinline__ void load_lds(unsigned stage, int q, const bf16 *src, int rows, int K,
                                         int r0, int k0, int lane) {
  const int r = q * 8 + (lane >> 3), pc = lane & 7;
  const bf16 *g = src + (size_t)min(r0 + r, rows - 1) * K + k0 + swz(r, pc) * 8;
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(__builtin_amdgcn_readfirstlane(stage + q * 1024))
               : "memory", "m0");
}

// Fragment r of k16 step s, in the order the MFMAs need them: x0 w0 x1 x2 x3 w1 w2 w3.
__device__ __forceinline__ void read_frag(Frag &f, int r, const unsigned char *sa,
                                          const unsigned char *sw, int s, int wm, int wn,
                                          int lane) {
  const bool is_x = (r == 0 || r == 2 || r == 3 || r == 4);
  const int idx = r <= 1 ? 0 : (r <= 4 ? r - 1 : r - 4);
  const int kc = s * 2 + (lane >> 5);
  if (is_x) {
    const int row = wm * 128 + idx * 32 + (lane & 31);
    f.x[idx] = *reinterpret_cast<const bf16x8 *>(sa + row * 128 + swz(row, kc) * 16);
  } else {
    const int row = wn * 128 + idx * 32 + (lane & 31);
    f.w[idx] = *reinterpret_cast<const bf16x8 *>(sw + row * 128 + swz(row, kc) * 16);
  }
}

__device__ __forceinline__ void mfma(f32x16 (&acc)[4][4], const Frag &f, int q) {
  const int j = q >> 2, i = q & 3;
  acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.w[j], f.x[i], acc[j][i], 0, 0, 0);
}

// Own loads landed in LDS (all, or all but the last VM issued), own LDS reads
// done, then the workgroup barrier.
template <int VM>
__device__ __forceinline__ void barrier_vm() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(VM) : "memory");
}
__device__ __forceinline__ void barrier() { barrier_vm<0>(); }

}  // namespace big

// Write-back through LDS (free once the main loop is done).  In the
// accumulator layout a store instruction would write 16 bytes into each of
// 32 rows; instead each wavefront writes one 32-row block of its accumulators
// to LDS as fp32 and reads it back row-major, so one store instruction covers
// whole row segments (two rows of 128 columns, or four of 64).  Per-row
// addressing data of the tile were staged in LDS by the caller; residual
// priors of the next batch of rows are loaded before this batch's stores.
namespace big {
constexpr int kWbStride = 132;  // floats per staged row (128 + 4: no bank conflicts)
static_assert(4 * 32 * kWbStride * 4 <= kWBase, "staged write-back fits the activation stages");
}  // namespace big

// One wavefront's TM 32-row blocks of TN * 32 columns (accumulators acc[j][i]:
// column block j, row block i) starting at output row row0 and column col0.
// Each block goes through the wavefront's staging area `st` (32 rows of
// TN * 32 + 4 floats) and is read back with TN * 8 lanes per row, so lane l
// owns columns 4 (l % (8 TN)) .. + 3 of rows l / (8 TN) + (64 / (8 TN)) k.
// `rows` are the row records of rows row0.. (in LDS), `b` the bias of this
// lane's four columns.  Residual priors are loaded PB rows at a time, each
// batch before the stores of the previous one.
template <int TN, int TM, int PB, class Epi>
__device__ __forceinline__ void write_back_staged(const f32x16 (&acc)[TN][TM], const Epi &epi,
                                                  int row0, int col0, int M, int lane, float *st,
                                                  const typename Epi::Row *rows, f32x4 b) {
  constexpr int LPR = TN * 8;      // lanes per output row
  constexpr int RPP = 64 / LPR;    // rows per store instruction
  constexpr int KP = 32 / RPP;     // store instructions per 32-row block
  constexpr int STR = TN * 32 + 4; // staged row stride (floats): no bank conflicts
  static_assert(KP % PB == 0, "prior batches");
  constexpr int NB = KP / PB;      // batches per 32-row block
  const int c4 = (lane % LPR) * 4, rsub = lane / LPR, half = lane >> 5;
  const typename Epi::Col col = epi.col(col0 + c4);
  f32x4 pr[2][PB];  // residual priors; zero for epilogues without one
#pragma unroll
  for (int k = 0; k < PB; ++k) pr[0][k] = pr[1][k] = f32x4{};
  // batch u: block u / NB, rows rsub + RPP k for k in [(u % NB) PB, + PB)
  auto load_priors = [&](int u, f32x4 (&dst)[PB]) {
    const int i = u / NB, k0 = (u % NB) * PB;
#pragma unroll
    for (int k = 0; k < PB; ++k)
      dst[k] = Epi::kPrior ? epi.prior(rows[i * 32 + rsub + RPP * (k0 + k)], col) : f32x4{};
  };
  if constexpr (Epi::kPrior) load_priors(0, pr[0]);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    // block row i of the accumulators -> LDS rows 0..31 of this wavefront
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4 *>(st + (lane & 31) * STR + j * 32 + g * 8 + half * 4) =
            f32x4{acc[j][i][4 * g + 0], acc[j][i][4 * g + 1], acc[j][i][4 * g + 2],
                  acc[j][i][4 * g + 3]};
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    const int rbase = row0 + i * 32;
    const bool full = rbase + 32 <= M;  // the whole block exists: no per-row guard
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int u = i * NB + nb;
      f32x4 v[PB];
#pragma unroll
      for (int k = 0; k < PB; ++k)
        v[k] = *reinterpret_cast<const f32x4 *>(st + (rsub + RPP * (nb * PB + k)) * STR + c4);
      if constexpr (Epi::kPrior) {
        if (u + 1 < TM * NB) load_priors(u + 1, pr[(u + 1) & 1]);
#pragma unroll
        for (int k = 0; k < PB; ++k) keep(pr[u & 1][k]);
      }
      auto value = [&](int k) -> f32x4 {
        if constexpr (Epi::kPrior) return v[k] + b + pr[u & 1][k];
        else return v[k] + b;
      };
      if (full) {
#pragma unroll
        for (int k = 0; k < PB; ++k) {
          const int r = rsub + RPP * (nb * PB + k);
          epi.store(rows[i * 32 + r], rbase + r, col, value(k));
        }
      } else {
#pragma unroll
        for (int k = 0; k < PB; ++k) {
          const int r = rsub + RPP * (nb * PB + k);
          if (rbase + r < M) epi.store(rows[i * 32 + r], rbase + r, col, value(k));
        }
      }
    }
    // this block's reads of the staging rows are done before the next block
    // overwrites them
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
}

template <class Epi>
__global__ __launch_bounds__(256, 1) void gemm_bf16_big_kernel(const bf16 *A, const bf16 *W, int M,
                                                               int N, int K, Epi epi) {
  using namespace big;
  // activation stages at [0, 96K), weight stages at [96K, 160K); after the
  // main loop the write-back stages rows in [0, 66K) and keeps the tile's
  // biases and row records in the weight stage the last k-tile left free
  __shared__ __attribute__((aligned(1024))) unsigned char smem[kSmem];
  static_assert(1024 + 256 * sizeof(typename Epi::Row) <= kStage, "row records fit one stage");
  const int tiles_m = (M + 255) / 256, tiles_n = N / 256;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, gridDim.x), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * 256, n0 = tn * 256;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar address math
  const int wm = wave >> 1, wn = wave & 1;
  const int q0 = wave * 8;  // this wavefront's load instructions q0 .. q0 + 7 of each operand
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) void *)smem;
  f32x16 acc[4][4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[j][i] = f32x16{};
  const int nk = K / 64;
  auto load_a = [&](int sa, int kt, int p) {
    load_lds(lds0 + sa * kStage, q0 + p, A, M, K, m0, kt * 64, lane);
  };
  auto load_w = [&](int kt, int p) {
    load_lds(lds0 + kWBase + (kt & 1) * kStage, q0 + p, W, N, K, n0, kt * 64, lane);
  };

  // The write-back's bias (threads < 64, four columns each) and row record
  // (one row per thread), loaded first and kept in registers: they reach LDS
  // only after the main loop, so no wait on them holds up the pipeline.
  const typename Epi::Row rec = epi.row(min(m0 + tid, M - 1));
  const f32x4 bias = tid < 64 ? epi.bias4(n0 + tid * 4) : f32x4{};
  // k-tiles 0 and 1 of both operands, then wait for k-tile 0 only
#pragma unroll
  for (int p = 0; p < 8; ++p) load_a(0, 0, p);
#pragma unroll
  for (int p = 0; p < 8; ++p) load_w(0, p);
  if (nk > 1) {
#pragma unroll
    for (int p = 0; p < 8; ++p) load_a(1, 1, p);
#pragma unroll
    for (int p = 0; p < 8; ++p) load_w(1, p);
    barrier_vm<16>();
  } else {
    barrier();
  }
  Frag fa, fb;
#pragma unroll
  for (int r = 0; r < 8; ++r) read_frag(fa, r, smem, smem + kWBase, 0, wm, wn, lane);

  // activation stage of k-tiles kt, kt + 1, kt + 2 (kt mod 3, ...)
  int sa0 = 0, sa1 = 1, sa2 = 2;
  for (int kt = 0; kt + 1 < nk; ++kt) {
    const unsigned char *ac = smem + sa0 * kStage, *wc = smem + kWBase + (kt & 1) * kStage;
    const unsigned char *an = smem + sa1 * kStage, *wnx = smem + kWBase + ((kt + 1) & 1) * kStage;
    const bool a2 = kt + 2 < nk;  // k-tile kt+2 exists: its activation rows go out now
    // k16 steps 0..2: fragments of the next step; the second half of the
    // weight rows of k-tile kt+1 (the first went out at the end of k-tile
    // kt-1; k-tile 1 was loaded whole in the prologue), then the activation
    // rows of k-tile kt+2 into the stage k-tile kt-1 left
#pragma unroll
    for (int st = 0; st < 3; ++st) {
      Frag &fc = (st & 1) ? fb : fa;
      Frag &fn = (st & 1) ? fa : fb;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        mfma(acc, fc, q);
        if (q < 8) read_frag(fn, q, ac, wc, st + 1, wm, wn, lane);
        else if (st == 0 && q < 12 && kt > 0) load_w(kt + 1, 4 + (q - 8));
        else if (st == 0 && q >= 12 && a2) load_a(sa2, kt + 2, q - 12);
        else if (st == 1 && q < 12 && a2) load_a(sa2, kt + 2, 4 + (q - 8));
        pin();
      }
    }
    // k16 step 3: barrier (k-tile kt+1 complete -- only the activation loads
    // of k-tile kt+2 may still be in flight -- and every wavefront done with
    // k-tile kt), first fragments of k-tile kt+1, first half of the weight
    // rows of k-tile kt+2 into the weight stage of k-tile kt
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      mfma(acc, fb, q);
      pin();
    }
    if (a2) barrier_vm<8>();
    else barrier();
    pin();
#pragma unroll
    for (int q = 4; q < 12; ++q) {
      mfma(acc, fb, q);
      read_frag(fa, q - 4, an, wnx, 0, wm, wn, lane);
      pin();
    }
#pragma unroll
    for (int q = 12; q < 16; ++q) {
      mfma(acc, fb, q);
      if (a2) load_w(kt + 2, q - 12);
      pin();
    }
    const int t = sa0;
    sa0 = sa1;
    sa1 = sa2;
    sa2 = t;
  }
  {  // last k-tile: no loads in flight
    const unsigned char *ac = smem + sa0 * kStage, *wc = smem + kWBase + ((nk - 1) & 1) * kStage;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      Frag &fc = (st & 1) ? fb : fa;
      Frag &fn = (st & 1) ? fa : fb;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        mfma(acc, fc, q);
        if (st < 3 && q < 8) read_frag(fn, q, ac, wc, st + 1, wm, wn, lane);
        pin();
      }
    }
  }
  // the write-back's biases and row records into the weight stage that the
  // last k-tile does not read (no wavefront reads it after the last
  // k-tile's barrier); then every wavefront is done with the stages before
  // they hold the write-back's staging rows
  unsigned char *side = smem + kWBase + (nk & 1) * kStage;
  if (tid < 64) *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(side) + tid * 4) = bias;
  reinterpret_cast<typename Epi::Row *>(side + 1024)[tid] = rec;
  barrier();
  const f32x4 b = *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(side) +
                                                    wn * 128 + (lane & 31) * 4);
  write_back_staged<4, 4, 16>(acc, epi, m0 + wm * 128, n0 + wn * 128, M, lane,
                           reinterpret_cast<float *>(smem) + wave * 32 * kWbStride,
                           reinterpret_cast<const typename Epi::Row *>(side + 1024) + wm * 128, b);
}

// ------------------------------------------------------------------ 256x256 tile, eight wavefronts
//
// The 256x256x64 tile of gemm_bf16_big_kernel (same LDS stages, swizzle,
// direct-to-LDS loads and stage schedule) on eight wavefronts of 128x64 (8
// accumulator blocks, 128 accumulation registers each), two per SIMD: while
// one wavefront of a SIMD waits on a fragment read, a barrier or its
// write-back's LDS round trip, the other can issue MFMAs.  Per k16 step a
// wavefront reads 6 fragments for 8 MFMAs (4 activation and 2 weight
// fragments), 1.5 times the LDS reads per MFMA of the 128x128 wavefront tile.
namespace big8 {

struct Frag {
  bf16x8 x[4];  // activation rows (MFMA B operand)
  bf16x8 w[2];  // weight rows (MFMA A operand)
};

// Fragment r of k16 step s, in the order the MFMAs need them: x0 w0 x1 x2 x3 w1.
__device__ __forceinline__ void read_frag(Frag &f, int r, const unsigned char *sa,
                                          const unsigned char *sw, int s, int wm, int wn,
                                          int lane) {
  const int kc = s * 2 + (lane >> 5);
  if (r == 1 || r == 5) {
    const int idx = r == 1 ? 0 : 1;
    const int row = wn * 64 + idx * 32 + (lane & 31);
    f.w[idx] = *reinterpret_cast<const bf16x8 *>(sw + row * 128 + big::swz(row, kc) * 16);
  } else {
    const int idx = r == 0 ? 0 : r - 1;
    const int row = wm * 128 + idx * 32 + (lane & 31);
    f.x[idx] = *reinterpret_cast<const bf16x8 *>(sa + row * 128 + big::swz(row, kc) * 16);
  }
}

__device__ __forceinline__ void mfma(f32x16 (&acc)[2][4], const Frag &f, int q) {
  const int j = q >> 2, i = q & 3;
  acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.w[j], f.x[i], acc[j][i], 0, 0, 0);
}

}  // namespace big8

template <class Epi>
__global__ __launch_bounds__(512, 1) void gemm_bf16_big8_kernel(const bf16 *A, const bf16 *W,
                                                                int M, int N, int K, Epi epi) {
  using namespace big;
  // LDS as in gemm_bf16_big_kernel; the write-back stages 8 x 32 rows of 68
  // floats in [0, 70 KB)
  __shared__ __attribute__((aligned(1024))) unsigned char smem[kSmem];
  static_assert(1024 + 256 * sizeof(typename Epi::Row) <= kStage, "row records fit one stage");
  static_assert(8 * 32 * 68 * 4 <= kWBase, "staged write-back fits the activation stages");
  const int tiles_m = (M + 255) / 256, tiles_n = N / 256;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, gridDim.x), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * 256, n0 = tn * 256;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const int q0 = wave * 4;  // this wavefront's load instructions q0 .. q0 + 3 of each operand
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) void *)smem;
  f32x16 acc[2][4];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[j][i] = f32x16{};
  const int nk = K / 64;
  auto load_a = [&](int sa, int kt, int p) {
    load_lds(lds0 + sa * kStage, q0 + p, A, M, K, m0, kt * 64, lane);
  };
  auto load_w = [&](int kt, int p) {
    load_lds(lds0 + kWBase + (kt & 1) * kStage, q0 + p, W, N, K, n0, kt * 64, lane);
  };

  const typename Epi::Row rec = epi.row(min(m0 + (tid & 255), M - 1));
  const f32x4 bias = tid < 64 ? epi.bias4(n0 + tid * 4) : f32x4{};
  // k-tiles 0 and 1 of both operands, then wait for k-tile 0 only
#pragma unroll
  for (int p = 0; p < 4; ++p) load_a(0, 0, p);
#pragma unroll
  for (int p = 0; p < 4; ++p) load_w(0, p);
  if (nk > 1) {
#pragma unroll
    for (int p = 0; p < 4; ++p) load_a(1, 1, p);
#pragma unroll
    for (int p = 0; p < 4; ++p) load_w(1, p);
    barrier_vm<8>();
  } else {
    barrier();
  }
  big8::Frag fa, fb;
#pragma unroll
  for (int r = 0; r < 6; ++r) big8::read_frag(fa, r, smem, smem + kWBase, 0, wm, wn, lane);

  int sa0 = 0, sa1 = 1, sa2 = 2;
  for (int kt = 0; kt + 1 < nk; ++kt) {
    const unsigned char *ac = smem + sa0 * kStage, *wc = smem + kWBase + (kt & 1) * kStage;
    const unsigned char *an = smem + sa1 * kStage, *wnx = smem + kWBase + ((kt + 1) & 1) * kStage;
    const bool a2 = kt + 2 < nk;
    // k16 steps 0..2: the fragments of the next step, then two loads: the
    // second half of the weight rows of k-tile kt+1 (step 0; k-tile 1 was
    // loaded whole in the prologue), the activation rows of k-tile kt+2 into
    // the stage k-tile kt-1 left (steps 1 and 2)
#pragma unroll
    for (int st = 0; st < 3; ++st) {
      big8::Frag &fc = (st & 1) ? fb : fa;
      big8::Frag &fn = (st & 1) ? fa : fb;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        big8::mfma(acc, fc, q);
        if (q < 6) big8::read_frag(fn, q, ac, wc, st + 1, wm, wn, lane);
        else if (st == 0 && kt > 0) load_w(kt + 1, 2 + (q - 6));
        else if (st > 0 && a2) load_a(sa2, kt + 2, (st - 1) * 2 + (q - 6));
        pin();
      }
    }
    // k16 step 3: barrier (k-tile kt+1 complete -- only the activation loads
    // of k-tile kt+2 may still be in flight -- and every wavefront done with
    // k-tile kt), the first fragments of k-tile kt+1, the first half of the
    // weight rows of k-tile kt+2 into the weight stage of k-tile kt
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      big8::mfma(acc, fb, q);
      pin();
    }
    if (a2) barrier_vm<4>();
    else barrier();
    pin();
#pragma unroll
    for (int q = 2; q < 8; ++q) {
      big8::mfma(acc, fb, q);
      big8::read_frag(fa, q - 2, an, wnx, 0, wm, wn, lane);
      if (q >= 6 && a2) load_w(kt + 2, q - 6);
      pin();
    }
    const int t = sa0;
    sa0 = sa1;
    sa1 = sa2;
    sa2 = t;
  }
  {  // last k-tile: no loads in flight
    const unsigned char *ac = smem + sa0 * kStage, *wc = smem + kWBase + ((nk - 1) & 1) * kStage;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      big8::Frag &fc = (st & 1) ? fb : fa;
      big8::Frag &fn = (st & 1) ? fa : fb;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        big8::mfma(acc, fc, q);
        if (st < 3 && q < 6) big8::read_frag(fn, q, ac, wc, st + 1, wm, wn, lane);
        pin();
      }
    }
  }
  unsigned char *side = smem + kWBase + (nk & 1) * kStage;
  if (tid < 64) *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(side) + tid * 4) = bias;
  if (tid < 256) reinterpret_cast<typename Epi::Row *>(side + 1024)[tid] = rec;
  barrier();
  const f32x4 b = *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(side) +
                                                    wn * 64 + (lane & 15) * 4);
  write_back_staged<2, 4, 4>(acc, epi, m0 + wm * 128, n0 + wn * 64, M, lane,
                             reinterpret_cast<float *>(smem) + wave * 32 * 68,
                             reinterpret_cast<const typename Epi::Row *>(side + 1024) + wm * 128, b);
}

// ------------------------------------------------------------------ 320x256 tile, eight wavefronts
//
// A 320x256x64 workgroup tile for products over whole images of 320 tokens:
// one tile row is one image, so a range of b images has b tile rows and a
// product with N = 1024 runs b * 4 tiles -- exactly one wave of 256 compute
// units for a 64-image range, where 256x256 tiles make 320 (1.25 waves) --
// and N = 3072 / 4096 three / four whole waves.  Eight wavefronts of 160x64
// (2 x 5 accumulator blocks, 160 accumulation registers each; two wavefronts
// share a SIMD), the 256x256 tile's 128-byte swizzled rows and direct-to-LDS
// loads, two 40 KB activation stages and two 32 KB weight stages (144 KB).
// A k-tile's activation rows go out right after the barrier that frees their
// stage, one k-tile ahead of use; its weight rows, which the L2 serves, beside
// the first MFMAs of the next k-tile.  Per k16 step a wavefront reads 7 fragments for 10
// MFMAs (5 activation, 2 weight).  Accumulation is the same chain of k16
// steps in ascending order as every other tile, so results are bitwise
// those of the 256x256 tile.
namespace t320 {

constexpr int kBM = 320;
constexpr int kAStage = kBM * 128;      // 40 KB: 320 rows x 64 k
constexpr int kWStage = 256 * 128;      // 32 KB
constexpr int kWBase = 2 * kAStage;     // weight stages start at 80 KB
constexpr int kSmem = kWBase + 2 * kWStage;  // 144 KB
constexpr int kALoads = kBM / 8 / 8;    // 1 KB load instructions per wavefront per k-tile: 5
constexpr int kWLoads = 256 / 8 / 8;    // 4
constexpr int kLoads = kALoads + kWLoads;
constexpr int kWbStride = 68;           // floats per staged row (64 + 4)
static_assert(8 * 32 * kWbStride * 4 <= kWBase, "staged write-back fits the activation stages");

// One set of fragments, refilled as the MFMAs of a k16 step release them.
struct Frag {
  bf16x8 x[5];  // activation rows (MFMA B operand)
  bf16x8 w[2];  // weight rows (MFMA A operand)
};

// Fragment r (0..4: activation row block r; 5, 6: weight row block r - 5) of
// k16 step s from a stage pair.
__device__ __forceinline__ void read_frag(Frag &f, int r, const unsigned char *sa,
                                          const unsigned char *sw, int s, int wm, int wn,
                                          int lane) {
  const int kc = s * 2 + (lane >> 5);
  if (r >= 5) {
    const int row = wn * 64 + (r - 5) * 32 + (lane & 31);
    f.w[r - 5] = *reinterpret_cast<const bf16x8 *>(sw + row * 128 + big::swz(row, kc) * 16);
  } else {
    const int row = wm * 160 + r * 32 + (lane & 31);
    f.x[r] = *reinterpret_cast<const bf16x8 *>(sa + row * 128 + big::swz(row, kc) * 16);
  }
}

// MFMA q of a k16 step: column block q / 5, row block q % 5.
__device__ __forceinline__ void mfma(f32x16 (&acc)[2][5], const Frag &f, int q) {
  const int j = q / 5, i = q % 5;
  acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.w[j], f.x[i], acc[j][i], 0, 0, 0);
}

// 1 KB of an operand into LDS at `lds` (wave-uniform): the scalar base is the
// operand at the k-tile's first column, `off` the lane's byte offset from it
// (32-bit: the host keeps every operand below 2^31 elements).
__device__ __forceinline__ void load_lds(unsigned lds, const bf16 *base, uint32_t off) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(off), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory", "m0");
}

}  // namespace t320

template <class Epi>
__global__ __launch_bounds__(512, 1) void gemm_bf16_t320_kernel(const bf16 *A, const bf16 *W,
                                                                 int M, int N, int K, Epi epi) {
  using namespace t320;
  // activation stages at [0, 80K), weight stages at [80K, 144K); after the
  // main loop the write-back stages rows in [0, 68K) and keeps the tile's
  // biases and row records in the weight stage the last k-tile left free
  __shared__ __attribute__((aligned(1024))) unsigned char smem[kSmem];
  static_assert(1024 + kBM * sizeof(typename Epi::Row) <= kWStage, "row records fit one stage");
  const int tiles_m = (M + kBM - 1) / kBM, tiles_n = N / 256;
  int tm, tn;
  // groups of 4 tile rows: an XCD's 32 concurrent tiles cover 4 rows x 8
  // columns (QKV 117 -> 114.5 us per range against groups of 8, with about
  // the same L2 fetch bytes)
  tile_coords<4>(xcd_remap(blockIdx.x, gridDim.x), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * kBM, n0 = tn * 256;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) void *)smem;
  f32x16 acc[2][5];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 5; ++i) acc[j][i] = f32x16{};
  const int nk = K / 64;
  // This wavefront's load p of every k-tile: p < 5 moves activation rows
  // 8 q .. 8 q + 7 (q = 5 wave + p of the tile's 40 blocks), p >= 5 weight
  // rows (q = 4 wave + p - 5 of 32); lane l writes row 8 q + l / 8 at
  // physical chunk l % 8, which holds logical chunk swz(row, l % 8).
  // Activation rows past M repeat row M - 1 (their results are never stored).
  uint32_t off[kLoads];
#pragma unroll
  for (int p = 0; p < kLoads; ++p) {
    const bool is_a = p < kALoads;
    const int q = is_a ? wave * kALoads + p : wave * kWLoads + (p - kALoads);
    const int r = q * 8 + (lane >> 3);
    const int row = is_a ? min(m0 + r, M - 1) : n0 + r;
    off[p] = (uint32_t)(row * K + big::swz(r, lane & 7) * 8) * 2u;
  }
  auto load = [&](int kt, int p) {
    const int s = kt & 1;
    if (p < kALoads)
      load_lds(lds0 + s * kAStage + (wave * kALoads + p) * 1024, A + kt * 64, off[p]);
    else
      load_lds(lds0 + kWBase + s * kWStage + (wave * kWLoads + p - kALoads) * 1024, W + kt * 64,
               off[p]);
  };

  const typename Epi::Row rec = epi.row(min(m0 + min(tid, kBM - 1), M - 1));
  const f32x4 bias = tid < 64 ? epi.bias4(n0 + tid * 4) : f32x4{};
  // k-tiles 0 and 1, then wait for k-tile 0 only
#pragma unroll
  for (int p = 0; p < kLoads; ++p) load(0, p);
  if (nk > 1) {
#pragma unroll
    for (int p = 0; p < kLoads; ++p) load(1, p);
    big::barrier_vm<kLoads>();
  } else {
    big::barrier();
  }
  // Per k16 step: MFMA q uses weight block q / 5 and activation block q % 5.
  // The step's own x4 and w1 are read beside MFMAs 0 and 1 (their previous
  // values are last used by MFMA 9 of the step before); beside MFMAs 5..9
  // the next step's w0, x0, x1, x2, x3 replace the ones MFMAs 4..8 used last.
  Frag f;
  read_frag(f, 5, smem, smem + kWBase, 0, wm, wn, lane);
#pragma unroll
  for (int r = 0; r < 4; ++r) read_frag(f, r, smem, smem + kWBase, 0, wm, wn, lane);
  constexpr int kNext[5] = {5, 0, 1, 2, 3};  // fragment read beside MFMA 5 + i

  for (int kt = 0; kt + 1 < nk; ++kt) {
    const int c = kt & 1, n = c ^ 1;
    const unsigned char *ac = smem + c * kAStage, *wc = smem + kWBase + c * kWStage;
    const unsigned char *an = smem + n * kAStage, *wnx = smem + kWBase + n * kWStage;
    const bool more = kt + 2 < nk;  // k-tile kt+2 exists
#pragma unroll
    for (int st = 0; st < 4; ++st) {
#pragma unroll
      for (int q = 0; q < 10; ++q) {
        t320::mfma(acc, f, q);
        if (q == 0) read_frag(f, 4, ac, wc, st, wm, wn, lane);
        if (q == 1) read_frag(f, 6, ac, wc, st, wm, wn, lane);
        // loads 5..8 of k-tile kt+1 (loads 0..4 went out in the step 3 of
        // k-tile kt-1; k-tile 1 was loaded whole in the prologue)
        if (kt > 0 && st == 0 && q >= 2 && q <= 4) load(kt + 1, kALoads + q - 2);
        if (kt > 0 && st == 1 && q == 2) load(kt + 1, kLoads - 1);
        // step 3: barrier (k-tile kt+1 landed, every wavefront done with
        // k-tile kt), then the next k-tile's first fragments and loads 0..4
        // of k-tile kt+2 into the stages k-tile kt leaves
        if (st == 3 && q == 4) big::barrier();
        if (q >= 5) {
          if (st < 3) read_frag(f, kNext[q - 5], ac, wc, st + 1, wm, wn, lane);
          else read_frag(f, kNext[q - 5], an, wnx, 0, wm, wn, lane);
          if (st == 3 && more) load(kt + 2, q - 5);
        }
        big::pin();
      }
    }
  }
  {  // last k-tile: no loads in flight
    const int c = (nk - 1) & 1;
    const unsigned char *ac = smem + c * kAStage, *wc = smem + kWBase + c * kWStage;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
#pragma unroll
      for (int q = 0; q < 10; ++q) {
        t320::mfma(acc, f, q);
        if (q == 0) read_frag(f, 4, ac, wc, st, wm, wn, lane);
        if (q == 1) read_frag(f, 6, ac, wc, st, wm, wn, lane);
        if (st < 3 && q >= 5) read_frag(f, kNext[q - 5], ac, wc, st + 1, wm, wn, lane);
        big::pin();
      }
    }
  }
  unsigned char *side = smem + kWBase + (nk & 1) * kWStage;
  if (tid < 64) *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(side) + tid * 4) = bias;
  if (tid < kBM) reinterpret_cast<typename Epi::Row *>(side + 1024)[tid] = rec;
  big::barrier();
  const f32x4 b = *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(side) +
                                                    wn * 64 + (lane & 15) * 4);
  write_back_staged<2, 5, 4>(acc, epi, m0 + wm * 160, n0 + wn * 64, M, lane,
                             reinterpret_cast<float *>(smem) + wave * 32 * kWbStride,
                             reinterpret_cast<const typename Epi::Row *>(side + 1024) + wm * 160, b);
}

// ------------------------------------------------------------------ 128x256 tile, two per CU
//
// A 128x256x32 workgroup tile on four wavefronts of 64x128 (8 accumulators,
// 128 registers), budgeted so that two workgroups share a CU: while one
// writes its tile back (bias, GELU, residual read-modify-write, KV-cache
// scatter) the other keeps the matrix cores busy.  Three 24 KB stages of
// 64-byte rows (16-byte chunks permuted by an XOR with bits 2..3 of the row,
// so the 16 rows one fragment read touches per chunk hit 16 distinct bank
// groups), loaded straight from global memory; the loads of k-tile t+3 go out
// as soon as every wavefront is done with k-tile t, two k-tiles ahead of use.
namespace pair {

constexpr int kBM = 128, kBN = 256, kBK = 32;
constexpr int kWOff = kBM * kBK * 2;             // weight rows start 8 KB into a stage
constexpr int kStage = (kBM + kBN) * kBK * 2;    // 24 KB
constexpr int kLoads = kStage / 1024 / 4;        // load instructions per wavefront per k-tile
static_assert(kLoads == 6, "load schedule assumes six loads per wavefront");

__device__ __forceinline__ int swz(int r, int c) { return c ^ ((r >> 2) & 3); }

struct Frag {
  bf16x8 x[2];  // activation rows (MFMA B operand)
  bf16x8 w[4];  // weight rows (MFMA A operand)
};

// Load instruction q (0..23 per k-tile) moves 1 KB: q < 8 carries activation
// rows 16q..16q+15, q >= 8 weight rows 16(q-8)..; lane l writes LDS bytes
// [16 l, 16 l + 16) of the block: row 16 q' + l / 4 at physical chunk l % 4.
__device__ __forceinline__ void load_lds(unsigned stage, int q, const bf16 *A, const bf16 *W,
                                         int M, int K, int m0, int n0, int k0, int lane) {
  const int rr = lane >> 2, pc = lane & 3;
  const bf16 *g;
  if (q < 8) {
    const int r = q * 16 + rr;
    g = A + (size_t)min(m0 + r, M - 1) * K + k0 + swz(r, pc) * 8;
  } else {
    const int r = (q - 8) * 16 + rr;
    g = W + (size_t)(n0 + r) * K + k0 + swz(r, pc) * 8;
  }
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(__builtin_amdgcn_readfirstlane(stage + q * 1024))
               : "memory", "m0");
}

// Fragment r of k16 step s (0 or 1), in the order the MFMAs need them: x0 w0 x1 w1 w2 w3.
__device__ __forceinline__ void read_frag(Frag &f, int r, const unsigned char *stage, int s, int wm,
                                          int wn, int lane) {
  const int c = 2 * s + (lane >> 5);
  if (r == 0 || r == 2) {
    const int row = wm * 64 + (r >> 1) * 32 + (lane & 31);
    f.x[r >> 1] = *reinterpret_cast<const bf16x8 *>(stage + row * 64 + swz(row, c) * 16);
  } else {
    const int j = r == 1 ? 0 : r - 2;
    const int row = wn * 128 + j * 32 + (lane & 31);
    f.w[j] = *reinterpret_cast<const bf16x8 *>(stage + kWOff + row * 64 + swz(row, c) * 16);
  }
}

__device__ __forceinline__ void mfma(f32x16 (&acc)[4][2], const Frag &f, int q) {
  const int j = q >> 1, i = q & 1;
  acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.w[j], f.x[i], acc[j][i], 0, 0, 0);
}

// Wait until at most VM of this wavefront's loads are in flight and its LDS
// reads are done, then the workgroup barrier.
template <int VM>
__device__ __forceinline__ void barrier_vm() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(VM) : "memory");
}

// The same with the loads of n whole k-tiles (six per wavefront each) still
// in flight, n in [0, NS - 2].
template <int NS>
__device__ __forceinline__ void barrier_tiles(int n) {
  static_assert(NS >= 3 && NS <= 7, "stage count");
  if (NS > 6 && n >= 5) barrier_vm<30>();
  else if (NS > 5 && n >= 4) barrier_vm<24>();
  else if (NS > 4 && n >= 3) barrier_vm<18>();
  else if (NS > 3 && n >= 2) barrier_vm<12>();
  else if (n >= 1) barrier_vm<6>();
  else barrier_vm<0>();
}

}  // namespace pair

// NS stages of 24 KB: three when two workgroups share a CU; six for long
// reductions (K >= 2048) whose workgroups each have a CU to themselves, so
// that operands streamed from HBM (a cache-aware fc2's hidden rows, a
// layer's weights not touched since the previous step) have five k-tiles to
// land instead of two (measured: 82 -> 78 us for a cache-aware MAR-L fc2 with
// operands not in any cache; short reductions gain nothing).  The loads of
// k-tile t+NS go into the stage k-tile t leaves, issued once every wavefront
// is done with k-tile t.
template <class Epi, int NS>
__global__ __launch_bounds__(256, NS <= 3 ? 2 : 1) void gemm_bf16_pair_kernel(
    const bf16 *A, const bf16 *W, int M, int N, int K, Epi epi) {
  using namespace pair;
  using big::pin;
  using Row = typename Epi::Row;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[NS * kStage];
  __shared__ __attribute__((aligned(16))) Row rows_lds[kBM];
  static_assert(4 * 32 * big::kWbStride * 4 <= NS * kStage, "staged write-back fits the stages");
  const int tiles_m = (M + kBM - 1) / kBM, tiles_n = N / kBN;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, gridDim.x), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * kBM, n0 = tn * kBN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int q0 = wave * kLoads;
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) void *)smem;
  f32x16 acc[4][2];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 2; ++i) acc[j][i] = f32x16{};
  const int nk = K / kBK;
  auto stage = [&](int kt) { return lds0 + (unsigned)(kt % NS) * kStage; };

  // The write-back's row record (threads < 128) and bias (each lane's four
  // columns), loaded before the tile loads and kept in registers: they reach
  // LDS only after the main loop, so no wait on them holds up the pipeline.
  Row rec{};
  if (tid < kBM) rec = epi.row(min(m0 + tid, M - 1));
  const f32x4 bias = epi.bias4(n0 + wn * 128 + (lane & 31) * 4);

  // k-tiles 0 .. NS-2 and the first half of k-tile NS-1, then wait for k-tile 0
#pragma unroll
  for (int kt = 0; kt + 1 < NS; ++kt) {
    if (kt < nk) {
#pragma unroll
      for (int p = 0; p < kLoads; ++p)
        load_lds(lds0 + kt * kStage, q0 + p, A, W, M, K, m0, n0, kt * kBK, lane);
    }
  }
  if (nk >= NS) {
#pragma unroll
    for (int p = 0; p < 3; ++p)
      load_lds(lds0 + (NS - 1) * kStage, q0 + p, A, W, M, K, m0, n0, (NS - 1) * kBK, lane);
    barrier_vm<6 * (NS - 2) + 3>();
  } else {
    barrier_tiles<NS>(nk - 1);
  }
  Frag fa, fb;
  const unsigned char *smem_u = smem;
#pragma unroll
  for (int r = 0; r < 6; ++r) read_frag(fa, r, smem_u, 0, wm, wn, lane);

  for (int t = 0; t + 1 < nk; ++t) {
    // k-tile t+NS-1: its first half is in flight, the rest goes out now;
    // k-tile t+NS: into k-tile t's stage once every wavefront is done with it
    const int kl = t + NS - 1, kn = t + NS;
    const bool has_l = kl < nk, has_n = kn < nk;
    const unsigned sl = stage(kl), s_t = stage(t);
    const unsigned char *sc = smem_u + (s_t - lds0), *sn = smem_u + (stage(t + 1) - lds0);
    // k16 step 0: step-1 fragments; loads 3 and 4 of k-tile t+NS-1
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      mfma(acc, fa, q);
      if (q < 6) read_frag(fb, q, sc, 1, wm, wn, lane);
      else if (has_l) load_lds(sl, q0 + 3 + (q - 6), A, W, M, K, m0, n0, kl * kBK, lane);
      pin();
    }
    // k16 step 1: load 5 of k-tile t+NS-1; barrier (k-tile t+1 complete,
    // k-tile t read by all); step-0 fragments of k-tile t+1; first half of
    // k-tile t+NS into the stage k-tile t leaves
    mfma(acc, fb, 0);
    if (has_l) load_lds(sl, q0 + 5, A, W, M, K, m0, n0, kl * kBK, lane);
    pin();
    mfma(acc, fb, 1);
    pin();
    barrier_tiles<NS>(min(NS - 2, nk - t - 2));
    pin();
#pragma unroll
    for (int q = 2; q < 8; ++q) {
      mfma(acc, fb, q);
      read_frag(fa, q - 2, sn, 0, wm, wn, lane);
      if (q >= 5 && has_n) load_lds(s_t, q0 + (q - 5), A, W, M, K, m0, n0, kn * kBK, lane);
      pin();
    }
  }
  {  // last k-tile
    const unsigned char *sc = smem_u + (stage(nk - 1) - lds0);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      mfma(acc, fa, q);
      if (q < 6) read_frag(fb, q, sc, 1, wm, wn, lane);
      pin();
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      mfma(acc, fb, q);
      pin();
    }
  }
  if (tid < kBM) rows_lds[tid] = rec;
  // every wavefront is done with the stages before they hold the write-back's
  // staging rows, and the row records are in LDS
  barrier_vm<0>();
  write_back_staged<4, 2, 8>(acc, epi, m0 + wm * 64, n0 + wn * 128, M, lane,
                          reinterpret_cast<float *>(smem) + wave * 32 * big::kWbStride,
                          rows_lds + wm * 64, bias);
}

// ------------------------------------------------------------------ 128x128 tile
//
// For the narrow products of cache-aware layers (N = d_model: the output
// projection and fc2 on a few thousand active rows), where 256x256 tiles
// would occupy a few dozen compute units and the 64x128 tile moves more
// operand bytes per k-tile than its MFMAs take cycles (so it waits on the
// L2).  A 128x128x64 tile on four wavefronts of 64x64 (4 accumulator blocks)
// keeps one 64-row MFMA block per operand fragment and about as many load
// cycles per k-tile as MFMA cycles.  Operand stages use the 256x256 tile's
// 128-byte rows, XOR swizzle and direct-to-LDS loads (big::load_lds): NS
// stages of 32 KB, the loads of k-tile t + NS - 1 issued once every
// wavefront is done with k-tile t - 1, so NS - 1 k-tiles are in flight.
// No split of K: every output is one accumulation over all of K in
// ascending k16 steps, as in every other tile, so the result does not depend
// on which tile a shape gets.
namespace mid {

constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kStage = (kBM + kBN) * kBK * 2;  // 32 KB: activation rows, then weight rows
constexpr int kWOff = kBM * kBK * 2;           // weight rows 16 KB into a stage

struct Frag {
  bf16x8 x[2];  // activation rows (MFMA B operand)
  bf16x8 w[2];  // weight rows (MFMA A operand)
};

// Fragments of k16 step s (0..3) of a stage for wavefront (wm, wn).
__device__ __forceinline__ void read_frags(Frag &f, const unsigned char *stage, int s, int wm,
                                           int wn, int lane) {
  const int kc = s * 2 + (lane >> 5);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = wm * 64 + i * 32 + (lane & 31);
    f.x[i] = *reinterpret_cast<const bf16x8 *>(stage + row * 128 + big::swz(row, kc) * 16);
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = wn * 64 + j * 32 + (lane & 31);
    f.w[j] = *reinterpret_cast<const bf16x8 *>(stage + kWOff + row * 128 + big::swz(row, kc) * 16);
  }
}

__device__ __forceinline__ void mfma(f32x16 (&acc)[2][2], const Frag &f) {
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 2; ++i)
      acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.w[j], f.x[i], acc[j][i], 0, 0, 0);
}

}  // namespace mid

// Wait until at most n whole k-tiles (8 loads per wavefront each) of this
// wavefront's loads are in flight and its LDS reads are done, then the
// workgroup barrier; n in [0, 3].
__device__ __forceinline__ void mid_barrier(int n) {
  if (n >= 3) pair::barrier_vm<24>();
  else if (n == 2) pair::barrier_vm<16>();
  else if (n == 1) pair::barrier_vm<8>();
  else pair::barrier_vm<0>();
}

template <class Epi, int NS>
__global__ __launch_bounds__(256, 1) void gemm_bf16_mid_kernel(const bf16 *A, const bf16 *W, int M,
                                                               int N, int K, Epi epi) {
  using namespace mid;
  using big::pin;
  using Row = typename Epi::Row;
  static_assert(NS >= 3 && NS <= 5, "stage count (the staged write-back needs 3 stages)");
  // NS stages of 32 KB; after the main loop the write-back stages its rows in
  // [0, 66 KB) and the tile's row records sit at 96 KB (in the fourth stage,
  // or the third's second half)
  __shared__ __attribute__((aligned(1024))) unsigned char smem[NS * kStage];
  constexpr int kRowsOff = 96 * 1024 - (NS == 3 ? 16 * 1024 : 0);
  static_assert(4 * 32 * big::kWbStride * 4 <= kRowsOff, "staged write-back below the row records");
  static_assert(kRowsOff + kBM * sizeof(Row) <= NS * kStage, "row records fit the stages");
  const int tiles_m = (M + kBM - 1) / kBM, tiles_n = N / kBN;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, gridDim.x), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * kBM, n0 = tn * kBN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) void *)smem;
  const unsigned char *smem_u = smem;
  f32x16 acc[2][2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 2; ++i) acc[j][i] = f32x16{};
  const int nk = K / kBK;
  // k-tile t into stage st: 16 load instructions of 1 KB (8 rows) per operand,
  // four of each per wavefront
  auto load_tile = [&](int st, int t) {
    const unsigned sb = lds0 + (unsigned)st * kStage;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      big::load_lds(sb, wave * 4 + p, A, M, K, m0, t * kBK, lane);
      big::load_lds(sb + kWOff, wave * 4 + p, W, N, K, n0, t * kBK, lane);
    }
  };

  // the write-back's row record (threads < 128) and this lane's bias, kept in
  // registers until after the main loop
  Row rec{};
  if (tid < kBM) rec = epi.row(min(m0 + tid, M - 1));
  const f32x4 bias = epi.bias4(n0 + wn * 64 + (lane & 15) * 4);

  // k-tiles 0 .. NS-2 in flight, then wait for k-tile 0
  const int issued = min(NS - 1, nk);
#pragma unroll
  for (int t = 0; t < NS - 1; ++t)
    if (t < nk) load_tile(t, t);
  mid_barrier(issued - 1);
  Frag f[2];
  read_frags(f[0], smem_u, 0, wm, wn, lane);

  for (int t = 0; t < nk; ++t) {
    const unsigned char *sc = smem_u + (t % NS) * kStage;
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      read_frags(f[(s + 1) & 1], sc, s + 1, wm, wn, lane);
      mfma(acc, f[s & 1]);
      pin();
    }
    if (t + 1 < nk) {
      // k-tile t+1 landed and every wavefront is done with k-tile t-1's
      // stage.  Issued so far: k-tiles up to t + NS - 2, so the ones after
      // t + 1 that may stay in flight number min(NS - 3, nk - t - 2)
      mid_barrier(min(NS - 3, nk - t - 2));
      read_frags(f[0], smem_u + ((t + 1) % NS) * kStage, 0, wm, wn, lane);
      // k-tile t+NS-1 into the stage k-tile t-1 used (free: the barrier above)
      if (t + NS - 1 < nk) load_tile((t + NS - 1) % NS, t + NS - 1);
    }
    mfma(acc, f[1]);
    pin();
  }
  // every wavefront is done with the stages before the row records and the
  // staged rows overwrite them
  pair::barrier_vm<0>();
  Row *rows_lds = reinterpret_cast<Row *>(smem + kRowsOff);
  if (tid < kBM) rows_lds[tid] = rec;
  pair::barrier_vm<0>();
  write_back_staged<2, 2, 8>(acc, epi, m0 + wm * 64, n0 + wn * 64, M, lane,
                             reinterpret_cast<float *>(smem) + wave * 32 * big::kWbStride,
                             rows_lds + wm * 64, bias);
}

// ------------------------------------------------------------------ 64x128 tile
//
// For products too small to spread 128x256 tiles over the chip (the sampler's
// MLP on a few hundred rows, a shard of a few images): a 64x128x128 tile on
// four wavefronts of 32x64 (2 accumulator blocks).  With so little work per
// workgroup its time is the serial chain of k-tiles (barrier, LDS round trip,
// dependent MFMAs), not bandwidth, so the k-tile is long: three 48 KB stages
// of 256-byte rows (16-byte chunks XOR-permuted by the row's low four bits,
// so 16 rows read at one chunk hit 16 distinct bank groups), one barrier per
// 128 of K, the next k16 step's fragments read while the current one's MFMAs
// run, and the loads of k-tile t+3 issued once every wavefront is done with
// k-tile t.
namespace small {

constexpr int kBM = 64, kBN = 128, kBK = 128;
constexpr int kRow = kBK * 2;                  // 256-byte rows
constexpr int kWOff = kBM * kRow;              // weight rows start 16 KB into a stage
constexpr int kStage = (kBM + kBN) * kRow;     // 48 KB
constexpr int kLoads = kStage / 1024 / 4;      // load instructions per wavefront per k-tile
static_assert(kLoads == 12, "load count per wavefront");

__device__ __forceinline__ int swz(int r, int c) { return c ^ (r & 15); }

struct Frag {
  bf16x8 x;     // activation rows (MFMA B operand)
  bf16x8 w[2];  // weight rows (MFMA A operand)
};

// Load instruction q (0..47 per k-tile) moves 1 KB = four 256-byte rows:
// q < 16 carries activation rows 4q..4q+3, q >= 16 weight rows 4(q-16)..;
// lane l writes LDS bytes [16 l, 16 l + 16): row 4 q' + l / 16 at physical
// chunk l % 16.
__device__ __forceinline__ void load_lds(unsigned stage, int q, const bf16 *A, const bf16 *W,
                                         int M, int K, int m0, int n0, int k0, int lane) {
  const int rr = lane >> 4, pc = lane & 15;
  const bf16 *g;
  if (q < 16) {
    const int r = q * 4 + rr;
    g = A + (size_t)min(m0 + r, M - 1) * K + k0 + swz(r, pc) * 8;
  } else {
    const int r = (q - 16) * 4 + rr;
    g = W + (size_t)(n0 + r) * K + k0 + swz(r, pc) * 8;
  }
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(__builtin_amdgcn_readfirstlane(stage + q * 1024))
               : "memory", "m0");
}

// Fragments of k16 step s (0..7) of a stage.
__device__ __forceinline__ void read_frags(Frag &f, const unsigned char *stage, int s, int wm,
                                           int wn, int lane) {
  const int c = 2 * s + (lane >> 5);
  const int xr = wm * 32 + (lane & 31);
  f.x = *reinterpret_cast<const bf16x8 *>(stage + xr * kRow + swz(xr, c) * 16);
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int wr = wn * 64 + j * 32 + (lane & 31);
    f.w[j] = *reinterpret_cast<const bf16x8 *>(stage + kWOff + wr * kRow + swz(wr, c) * 16);
  }
}

__device__ __forceinline__ void mfma(f32x16 (&acc)[2][1], const Frag &f) {
#pragma unroll
  for (int j = 0; j < 2; ++j)
    acc[j][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.w[j], f.x, acc[j][0], 0, 0, 0);
}

}  // namespace small

template <class Epi>
__global__ __launch_bounds__(256) void gemm_bf16_small_kernel(const bf16 *A, const bf16 *W, int M,
                                                              int N, int K, Epi epi) {
  using namespace small;
  using pair::barrier_vm;
  using big::pin;
  using Row = typename Epi::Row;
  constexpr int kStr = 2 * 32 + 4;  // staged write-back row (floats)
  __shared__ __attribute__((aligned(1024))) unsigned char smem[3 * kStage];
  __shared__ __attribute__((aligned(16))) Row rows_lds[kBM];
  static_assert(4 * 32 * kStr * 4 <= 3 * kStage, "staged write-back fits the stages");
  const int tiles_m = (M + kBM - 1) / kBM, tiles_n = N / kBN;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, gridDim.x), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * kBM, n0 = tn * kBN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int q0 = wave * kLoads;
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) void *)smem;
  const unsigned char *smem_u = smem;
  f32x16 acc[2][1] = {{f32x16{}}, {f32x16{}}};
  const int nk = K / kBK;
  auto load_tile = [&](unsigned st, int t) {
#pragma unroll
    for (int p = 0; p < kLoads; ++p) load_lds(st, q0 + p, A, W, M, K, m0, n0, t * kBK, lane);
  };

  // the write-back's row record (threads < 64) and this lane's bias, kept in
  // registers until after the main loop
  Row rec{};
  if (tid < kBM) rec = epi.row(min(m0 + tid, M - 1));
  const f32x4 bias = epi.bias4(n0 + wn * 64 + (lane & 15) * 4);

  // k-tiles 0, 1 and 2 (as far as they exist)
  unsigned s0 = lds0, s1 = lds0 + kStage, s2 = lds0 + 2 * kStage;
  load_tile(s0, 0);
  if (nk > 1) load_tile(s1, 1);
  if (nk > 2) load_tile(s2, 2);
  if (nk > 2) barrier_vm<2 * kLoads>();
  else if (nk > 1) barrier_vm<kLoads>();
  else barrier_vm<0>();
  Frag f[2];
  read_frags(f[0], smem_u + (s0 - lds0), 0, wm, wn, lane);

  for (int t = 0; t < nk; ++t) {
    // s0: k-tile t (f[0] holds its step-0 fragments); s1, s2: k-tiles t+1, t+2
    const unsigned char *sc = smem_u + (s0 - lds0);
#pragma unroll
    for (int st = 0; st < 7; ++st) {
      read_frags(f[(st + 1) & 1], sc, st + 1, wm, wn, lane);
      mfma(acc, f[st & 1]);
      pin();
    }
    if (t + 1 < nk) {
      // k-tile t+1 complete (k-tile t+2 may still be in flight) and k-tile t
      // read by every wavefront
      if (t + 2 < nk) barrier_vm<kLoads>();
      else barrier_vm<0>();
      read_frags(f[0], smem_u + (s1 - lds0), 0, wm, wn, lane);
    }
    mfma(acc, f[1]);
    if (t + 3 < nk) load_tile(s0, t + 3);  // into the stage k-tile t left
    const unsigned s_old = s0;
    s0 = s1;
    s1 = s2;
    s2 = s_old;
  }
  if (tid < kBM) rows_lds[tid] = rec;
  barrier_vm<0>();
  write_back_staged<2, 1, 8>(acc, epi, m0 + wm * 32, n0 + wn * 64, M, lane,
                             reinterpret_cast<float *>(smem) + wave * 32 * kStr,
                             rows_lds + wm * 32, bias);
}

// Tile choice.  A large tile (one workgroup per CU) when 256x256 tiles fill
// at least 45% of their last wave over the compute units: a partly filled
// last wave runs at a higher clock under the chip's power limit, and beside
// another image range's kernels when the step runs as ranges on streams
// (which is why the bound is this low: with a single range, such a wave
// leaves the rest of the chip idle).  Of the two large tiles, the 320x256
// one when its waves cover no more rows than the 256x256 tile's.
// Otherwise the 128x256 tile, two workgroups per CU, whose write-backs
// overlap the other workgroup's main loop and whose finer steps fill the chip
// better; the 128x128 tile for narrow products it would spread too thinly;
// and when even 128x256 tiles would occupy fewer than half the compute units,
// the 64x128 tile (K a multiple of 128).  At MAR-L sizes, per 64-image range:
// every full-layer product takes the 320x256 tile (QKV 3, output projection
// and fc2 1, fc1 4 whole waves); the cache-aware fc1 and QKV take the 256x256
// tile when a range has more than 2304 active rows (10 tiles of rows), else
// the 128x256 tile; the cache-aware output projection and fc2 the 128x128
// tile; the sampler's per-block GEMMs (a few hundred rows) the 64x128 tile.
// Under sustained load the 128x256 tile runs at a lower clock (more operand
// traffic per flop), which is why it does not replace the large tiles.
int gemm_tile_kind(DType dt, int32_t m, int32_t n, int32_t k) {
  if (dt != DType::BF16 || m <= 0) return GEMM_TILE_128x256;
  const long cus = device_cu_count();
  const long tiles = (long)((m + 255) / 256) * (n / 256);
  const long waves = (tiles + cus - 1) / cus;
  const double fill = (double)tiles / (double)(waves * cus);
  if (fill >= 0.45) {
    // the 320x256 tile where its whole waves take no more time than the
    // 256x256 tile's, counting a wave as its tile area (whole 320-token
    // images at N = 1024 / 3072 / 4096: 1 wave against 1.25, 3 against
    // 3.75, 4 against 5 -- the tie, fc1, measured 176.8 against 180.8 us)
    const long tiles320 = (long)((m + t320::kBM - 1) / t320::kBM) * (n / 256);
    const long waves320 = (tiles320 + cus - 1) / cus;
    if (waves320 * t320::kBM <= waves * 256) return GEMM_TILE_320;
    return GEMM_TILE_256;
  }
  if (k % small::kBK == 0 && (long)((m + 127) / 128) * (n / 256) * 2 < cus) {
    // narrow products that 128x128 tiles still spread over half the compute
    // units or more take them (the cache-aware output projection and fc2 of
    // a 64-image MAR-L range: 39 vs 52 us for fc2, 13.5 vs 19.8 us for the
    // output projection, each alone); smaller ones the 64x128 tile
    if ((long)((m + mid::kBM - 1) / mid::kBM) * (n / mid::kBN) * 2 >= cus) return GEMM_TILE_128;
    return GEMM_TILE_64x128;
  }
  return GEMM_TILE_128x256;
}

// N a multiple of 256 and K of 64 (the host limits d_model and d_mlp to
// multiples of 256).
template <class Epi>
static hipError_t run_bf16(const void *a, const void *w, int m, int n, int k, const Epi &epi,
                           hipStream_t s) {
  if (m == 0) return hipSuccess;
  if (n % 256 != 0 || k % 64 != 0) return hipErrorInvalidValue;
  const bf16 *A = static_cast<const bf16 *>(a), *W = static_cast<const bf16 *>(w);
  switch (gemm_tile_kind(DType::BF16, m, n, k)) {
    case GEMM_TILE_256:
      // eight wavefronts where the write-back is a large share of a tile
      // (K < 2048: fc1, QKV, the output projection), four where the main
      // loop dominates and the fewer LDS reads per MFMA win (fc2)
      if (k < 2048)
        launch_kernel(gemm_bf16_big8_kernel<Epi>, ((m + 255) / 256) * (n / 256), 512, 0, s, A, W,
                      m, n, k, epi);
      else
        launch_kernel(gemm_bf16_big_kernel<Epi>, ((m + 255) / 256) * (n / 256), 256, 0, s, A, W,
                      m, n, k, epi);
      break;
    case GEMM_TILE_320:
      launch_kernel(gemm_bf16_t320_kernel<Epi>, ((m + t320::kBM - 1) / t320::kBM) * (n / 256), 512,
                    0, s, A, W, m, n, k, epi);
      break;
    case GEMM_TILE_64x128:
      launch_kernel(gemm_bf16_small_kernel<Epi>,
                    ((m + small::kBM - 1) / small::kBM) * (n / small::kBN), 256, 0, s, A, W, m, n,
                    k, epi);
      break;
    case GEMM_TILE_128:
      launch_kernel(gemm_bf16_mid_kernel<Epi, 4>,
                    ((m + mid::kBM - 1) / mid::kBM) * (n / mid::kBN), 256, 0, s, A, W, m, n, k,
                    epi);
      break;
    default: {
      const int tiles = ((m + pair::kBM - 1) / pair::kBM) * (n / pair::kBN);
      if (tiles <= device_cu_count() && k >= 2048)
        launch_kernel(gemm_bf16_pair_kernel<Epi, 6>, tiles, 256, 0, s, A, W, m, n, k, epi);
      else
        launch_kernel(gemm_bf16_pair_kernel<Epi, 3>, tiles, 256, 0, s, A, W, m, n, k, epi);
    }
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ fp32 FMA

template <class Epi>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float *__restrict__ A,
                                                       const float *__restrict__ W, int M, int N,
                                                       int K, Epi epi) {
  constexpr int T = 64, BK = 16;
  __shared__ float As[BK][T + 4];
  __shared__ float Ws[BK][T + 4];
  const int tiles_n = N / T;
  const int m0 = (blockIdx.x / tiles_n) * T, n0 = (blockIdx.x % tiles_n) * T;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int lr = tid >> 2, lc = (tid & 3) * 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += BK) {
    const float4 av =
        *reinterpret_cast<const float4 *>(A + (size_t)min(m0 + lr, M - 1) * K + k0 + lc);
    const float4 wv = *reinterpret_cast<const float4 *>(W + (size_t)(n0 + lr) * K + k0 + lc);
    As[lc + 0][lr] = av.x; As[lc + 1][lr] = av.y; As[lc + 2][lr] = av.z; As[lc + 3][lr] = av.w;
    Ws[lc + 0][lr] = wv.x; Ws[lc + 1][lr] = wv.y; Ws[lc + 2][lr] = wv.z; Ws[lc + 3][lr] = wv.w;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Ws[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  const f32x4 b = epi.bias4(n0 + tx * 4);
  const typename Epi::Col c = epi.col(n0 + tx * 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= M) continue;
    const typename Epi::Row r = epi.row(row);
    const f32x4 v = {acc[i][0], acc[i][1], acc[i][2], acc[i][3]};
    epi.store(r, row, c, v + b + (Epi::kPrior ? epi.prior(r, c) : f32x4{}));
  }
}

template <class Epi>
static hipError_t run_f32(const void *a, const void *w, int m, int n, int k, const Epi &epi,
                          hipStream_t s) {
  if (m == 0) return hipSuccess;
  if (n % 64 != 0 || k % 16 != 0) return hipErrorInvalidValue;
  const int grid = ((m + 63) / 64) * (n / 64);
  launch_kernel(gemm_f32_kernel<Epi>, grid, 256, 0, s, static_cast<const float *>(a),
                                            static_cast<const float *>(w), m, n, k, epi);
  return hipGetLastError();
}

// ------------------------------------------------------------------ launchers

hipError_t launch_gemm_qkv(DType dt, const void *a, const void *w, const float *bias, int32_t m,
                           int32_t n, int32_t k, const RowMap *map, QkvOut o, hipStream_t s) {
  if (dt == DType::F32) {
    EpiQkv<float> e{static_cast<float *>(o.q), static_cast<float *>(o.k_cache),
                    static_cast<float *>(o.v_cache), bias, map, o.d_model, o.head_dim,
                    o.n_heads, o.n_tokens};
    return run_f32(a, w, m, n, k, e, s);
  }
  EpiQkv<bf16> e{static_cast<bf16 *>(o.q), static_cast<bf16 *>(o.k_cache),
                 static_cast<bf16 *>(o.v_cache), bias, map, o.d_model, o.head_dim, o.n_heads,
                 o.n_tokens};
  return run_bf16(a, w, m, n, k, e, s);
}

hipError_t launch_gemm_resid(DType dt, const void *a, const void *w, const float *bias, int32_t m,
                             int32_t n, int32_t k, const RowMap *map, float *x, int32_t tag,
                             hipStream_t s) {
  if (tag == 0) {
    EpiResid<0> e{x, bias, map, n};
    return dt == DType::F32 ? run_f32(a, w, m, n, k, e, s) : run_bf16(a, w, m, n, k, e, s);
  }
  EpiResid<1> e{x, bias, map, n};
  return dt == DType::F32 ? run_f32(a, w, m, n, k, e, s) : run_bf16(a, w, m, n, k, e, s);
}

hipError_t launch_gemm_gelu(DType dt, const void *a, const void *w, const float *bias, int32_t m,
                            int32_t n, int32_t k, void *h, hipStream_t s) {
  if (dt == DType::F32) {
    EpiGelu<float> e{static_cast<float *>(h), bias, n};
    return run_f32(a, w, m, n, k, e, s);
  }
  EpiGelu<bf16> e{static_cast<bf16 *>(h), bias, n};
  return run_bf16(a, w, m, n, k, e, s);
}

}  // namespace marche

namespace marche {

hipError_t launch_gemm_plain(DType dt, const void *a, const void *w, const float *bias, int32_t m,
                             int32_t n, int32_t k, void *out, DType out_dt, bool silu_act,
                             hipStream_t s) {
  if (dt == DType::F32) {
    if (out_dt != DType::F32) return hipErrorInvalidValue;
    if (silu_act) return run_f32(a, w, m, n, k, EpiPlain<float, true>{static_cast<float *>(out), bias, n}, s);
    return run_f32(a, w, m, n, k, EpiPlain<float, false>{static_cast<float *>(out), bias, n}, s);
  }
  if (out_dt == DType::F32) {
    if (silu_act) return hipErrorInvalidValue;
    return run_bf16(a, w, m, n, k, EpiPlain<float, false>{static_cast<float *>(out), bias, n}, s);
  }
  if (silu_act) return run_bf16(a, w, m, n, k, EpiPlain<bf16, true>{static_cast<bf16 *>(out), bias, n}, s);
  return run_bf16(a, w, m, n, k, EpiPlain<bf16, false>{static_cast<bf16 *>(out), bias, n}, s);
}

hipError_t launch_gemm_embed(DType dt, const void *a, const void *w, const float *bias, int32_t m,
                             int32_t n, int32_t k, float *x, const float *pe, const int32_t *known,
                             int32_t n_enc, int32_t n_buf, int32_t n_known, int32_t n_tokens,
                             hipStream_t s) {
  EpiEmbed e{x, bias, pe, known, n, n_enc, n_buf, n_known, n_tokens};
  return dt == DType::F32 ? run_f32(a, w, m, n, k, e, s) : run_bf16(a, w, m, n, k, e, s);
}

}  // namespace marche
