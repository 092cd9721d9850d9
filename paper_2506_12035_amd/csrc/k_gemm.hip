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
// bf16 path: workgroup tile BM x BN x BK, a grid of wavefronts each owning a
// block of 32x32 MFMA tiles (v_mfma_f32_32x32x16_bf16, fp32 accumulators).
// Tiles are staged global -> registers -> LDS (double-buffered LDS, one or
// two k-tiles of register prefetch).  LDS rows are padded by 16 bytes, which
// makes the 16-byte MFMA operand reads (32 rows at one k offset) bank-conflict
// free.
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
  using Row = RowMap;
  // 32-bit element offsets: the host limits every buffer to < 2^31 elements.
  struct Col {
    T *base;       // q, or the K or V cache of the layer
    uint32_t off;  // column offset: c0 for q, h*n_tokens*head_dim + d for K/V
    bool is_q;
  };
  __device__ __forceinline__ Row row(int r) const { return map[r]; }
  __device__ __forceinline__ Col col(int c0) const {
    if (c0 < d_model) return Col{q, (uint32_t)c0, true};
    int c = c0 - d_model;
    T *dst = kc;
    if (c >= d_model) {
      c -= d_model;
      dst = vc;
    }
    const int h = c / head_dim, d = c - h * head_dim;
    return Col{dst, (uint32_t)(h * n_tokens * head_dim + d), false};
  }
  __device__ __forceinline__ f32x4 bias4(int c0) const { return load_bias4(bias, c0); }
  __device__ __forceinline__ f32x4 prior(const Row &, const Col &) const { return f32x4{}; }
  __device__ __forceinline__ void store(const Row &m, int r, const Col &c, f32x4 v) const {
    const uint32_t row_off = c.is_q ? (uint32_t)(r * d_model)
                                    : (uint32_t)((m.b * n_heads * n_tokens + m.tok) * head_dim);
    store4(c.base + row_off + c.off, v);
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

// Empty uses that pin loaded values to this point: without them the compiler
// sinks the loads into the row-guarded store blocks, one wait per block.
__device__ __forceinline__ void keep(const f32x4 &v) { asm volatile("" ::"v"(v)); }
__device__ __forceinline__ void keep(int32_t v) { asm volatile("" ::"v"(v)); }
__device__ __forceinline__ void keep(const RowMap &m) {
  asm volatile("" ::"v"(m.x_row), "v"(m.b), "v"(m.tok));
}

// Write-back of one wavefront's TM x TN block of 32x32 accumulators (C^T
// layout: lane l owns output row l & 31 of each block and, in register group g,
// columns g * 8 + (l / 32) * 4 .. + 3).  Rows at or beyond M are clamped for
// the loads and skipped for the stores.  Residual priors are loaded for IB
// block rows at a time (at most 16 four-column groups, 64 registers), each
// batch's loads issued before the previous batch's stores.
//
// With BIAS_LDS, the biases of the block's columns come from LDS
// (bias_lds[c - col_base] for column c; the caller staged them there), which
// keeps them out of registers and off the vector-memory counter.
template <int TM, int TN, bool BIAS_LDS = false, class Epi>
__device__ __forceinline__ void write_back(const f32x16 (&acc)[TN][TM], const Epi &epi, int row0,
                                           int col_base, int M, int lane,
                                           const float *bias_lds = nullptr) {
  typename Epi::Row rinfo[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) rinfo[i] = epi.row(min(row0 + i * 32 + (lane & 31), M - 1));
  f32x4 b[BIAS_LDS ? 1 : TN][4];
  if constexpr (!BIAS_LDS) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) b[j][g] = epi.bias4(col_base + j * 32 + g * 8 + (lane >> 5) * 4);
  }
  typename Epi::Col cinfo[TN][4];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) cinfo[j][g] = epi.col(col_base + j * 32 + g * 8 + (lane >> 5) * 4);
  auto bias_of = [&](int j, int g) -> f32x4 {
    if constexpr (BIAS_LDS)
      return *reinterpret_cast<const f32x4 *>(bias_lds + j * 32 + g * 8 + (lane >> 5) * 4);
    else
      return b[j][g];
  };
#pragma unroll
  for (int i = 0; i < TM; ++i) keep(rinfo[i]);
  constexpr int IB = (16 / (TN * 4)) < 1 ? 1 : ((16 / (TN * 4)) > TM ? TM : 16 / (TN * 4));
  constexpr int NB = TM / IB;
  static_assert(TM % IB == 0, "prior batches");
  f32x4 pr[2][IB][TN][4];
  auto load_priors = [&](int bi, f32x4 (&dst)[IB][TN][4]) {
#pragma unroll
    for (int ii = 0; ii < IB; ++ii)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          dst[ii][j][g] = Epi::kPrior ? epi.prior(rinfo[bi * IB + ii], cinfo[j][g]) : f32x4{};
  };
  load_priors(0, pr[0]);
#pragma unroll
  for (int bi = 0; bi < NB; ++bi) {
    // the next batch's loads go out before this batch's stores
    if (bi + 1 < NB) load_priors(bi + 1, pr[(bi + 1) & 1]);
    if constexpr (Epi::kPrior) {
#pragma unroll
      for (int ii = 0; ii < IB; ++ii)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) keep(pr[bi & 1][ii][j][g]);
    }
#pragma unroll
    for (int ii = 0; ii < IB; ++ii) {
      const int i = bi * IB + ii;
      const int row = row0 + i * 32 + (lane & 31);
      if (row >= M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 a = {acc[j][i][4 * g + 0], acc[j][i][4 * g + 1], acc[j][i][4 * g + 2],
                           acc[j][i][4 * g + 3]};
          epi.store(rinfo[i], row, cinfo[j][g], a + bias_of(j, g) + pr[bi & 1][ii][j][g]);
        }
    }
  }
}

// ------------------------------------------------------------------ bf16 MFMA
//
// The MFMA A operand is a 32-row slice of W (output columns) and the B
// operand a 32-row slice of the activations (output rows), so each 32x32
// accumulator holds a block of C^T: lane l owns output row (l & 31) and, in
// register r, output column (r / 4) * 8 + (l / 32) * 4 + r % 4 -- four
// consecutive columns per group of four registers, which the epilogue stores
// together.

template <int BM_, int BN_, int BK_, int WGM_, int WGN_, int PF_, int MINB_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_;
  static constexpr int WGM = WGM_, WGN = WGN_;  // wavefront grid
  static constexpr int PF = PF_;                // k-tiles staged in registers ahead
  static constexpr int MINB = MINB_;            // workgroups per CU to budget registers for
  static constexpr int NT = WGM * WGN * 64;
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int LS = BK + 8;             // LDS row stride (elements): +16 bytes
  static constexpr int CPR = BK / 8;            // 16-byte chunks per tile row
  static constexpr int A_CHUNKS = BM * CPR / NT;
  static constexpr int B_CHUNKS = BN * CPR / NT;
  static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile not divisible");
  static_assert(2 * (BM + BN) * LS * 2 <= 160 * 1024, "LDS budget");
};

// Grouped tile order: GROUP consecutive tile rows sweep all tile columns
// together, so concurrently running workgroups share A rows and W columns.
__device__ __forceinline__ void tile_coords(int id, int tiles_m, int tiles_n, int &tm, int &tn) {
  constexpr int GROUP = 8;
  const int per_group = GROUP * tiles_n;
  const int g = id / per_group;
  const int first_m = g * GROUP;
  const int gm = min(tiles_m - first_m, GROUP);
  const int in = id - g * per_group;
  tm = first_m + in % gm;
  tn = in / gm;
}

template <class C>
struct Stage {
  u32x4 a[C::A_CHUNKS];
  u32x4 b[C::B_CHUNKS];
};

template <class C>
__device__ __forceinline__ void stage_load(Stage<C> &st, const bf16 *__restrict__ A,
                                           const bf16 *__restrict__ W, int M, int K, int m0,
                                           int n0, int k0, int tid) {
#pragma unroll
  for (int i = 0; i < C::A_CHUNKS; ++i) {
    const int c = i * C::NT + tid, row = c / C::CPR, col = (c % C::CPR) * 8;
    st.a[i] = *reinterpret_cast<const u32x4 *>(A + (size_t)min(m0 + row, M - 1) * K + k0 + col);
  }
#pragma unroll
  for (int i = 0; i < C::B_CHUNKS; ++i) {
    const int c = i * C::NT + tid, row = c / C::CPR, col = (c % C::CPR) * 8;
    st.b[i] = *reinterpret_cast<const u32x4 *>(W + (size_t)(n0 + row) * K + k0 + col);
  }
}

template <class C>
__device__ __forceinline__ void stage_store(const Stage<C> &st, bf16 *As, bf16 *Bs, int tid) {
#pragma unroll
  for (int i = 0; i < C::A_CHUNKS; ++i) {
    const int c = i * C::NT + tid, row = c / C::CPR, col = (c % C::CPR) * 8;
    *reinterpret_cast<u32x4 *>(&As[row * C::LS + col]) = st.a[i];
  }
#pragma unroll
  for (int i = 0; i < C::B_CHUNKS; ++i) {
    const int c = i * C::NT + tid, row = c / C::CPR, col = (c % C::CPR) * 8;
    *reinterpret_cast<u32x4 *>(&Bs[row * C::LS + col]) = st.b[i];
  }
}

// One BK-deep slab of MFMAs for this wavefront's block of 32x32 tiles.
template <class C>
__device__ __forceinline__ void tile_mfma(f32x16 (&acc)[C::TN][C::TM], const bf16 *As,
                                          const bf16 *Bs, int wm, int wn, int lane) {
  const int lrow = lane & 31, lk = (lane >> 5) * 8;
#pragma unroll
  for (int kk = 0; kk < C::BK; kk += 16) {
    bf16x8 af[C::TM], bw[C::TN];
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
      af[i] = *reinterpret_cast<const bf16x8 *>(&As[(wm * C::WM + i * 32 + lrow) * C::LS + kk + lk]);
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
      bw[j] = *reinterpret_cast<const bf16x8 *>(&Bs[(wn * C::WN + j * 32 + lrow) * C::LS + kk + lk]);
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
        acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bw[j], af[i], acc[j][i], 0, 0, 0);
  }
}

template <class C, class Epi>
__global__ __launch_bounds__(C::NT, C::MINB) void gemm_bf16_kernel(const bf16 *__restrict__ A,
                                                                   const bf16 *__restrict__ W,
                                                                   int M, int N, int K, Epi epi) {
  __shared__ __attribute__((aligned(16))) bf16 As[2][C::BM * C::LS];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][C::BN * C::LS];
  const int tiles_m = (M + C::BM - 1) / C::BM, tiles_n = N / C::BN;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, gridDim.x), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * C::BM, n0 = tn * C::BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  f32x16 acc[C::TN][C::TM];
#pragma unroll
  for (int j = 0; j < C::TN; ++j)
#pragma unroll
    for (int i = 0; i < C::TM; ++i) acc[j][i] = f32x16{};

  const int nk = K / C::BK;
  if constexpr (C::PF == 1) {
    // k-tile t+1 is loaded into registers while k-tile t is multiplied, then
    // written to the other LDS buffer.
    Stage<C> st;
    stage_load<C>(st, A, W, M, K, m0, n0, 0, tid);
    stage_store<C>(st, As[0], Bs[0], tid);
    __syncthreads();
    for (int kt = 0; kt + 1 < nk; ++kt) {
      const int cur = kt & 1;
      stage_load<C>(st, A, W, M, K, m0, n0, (kt + 1) * C::BK, tid);
      tile_mfma<C>(acc, As[cur], Bs[cur], wm, wn, lane);
      stage_store<C>(st, As[cur ^ 1], Bs[cur ^ 1], tid);
      __syncthreads();
    }
    tile_mfma<C>(acc, As[(nk - 1) & 1], Bs[(nk - 1) & 1], wm, wn, lane);
  } else {
    // Two register stages: k-tile t+2 is loaded while k-tile t is multiplied
    // and k-tile t+1 (loaded one iteration earlier) goes to LDS after it, so
    // every load has two iterations to land.
    Stage<C> s0, s1;
    stage_load<C>(s0, A, W, M, K, m0, n0, 0, tid);
    if (nk > 1) stage_load<C>(s1, A, W, M, K, m0, n0, C::BK, tid);
    stage_store<C>(s0, As[0], Bs[0], tid);
    __syncthreads();
    int kt = 0;
    for (; kt + 2 < nk; kt += 2) {
      stage_load<C>(s0, A, W, M, K, m0, n0, (kt + 2) * C::BK, tid);
      tile_mfma<C>(acc, As[0], Bs[0], wm, wn, lane);
      stage_store<C>(s1, As[1], Bs[1], tid);
      __syncthreads();
      if (kt + 3 < nk) stage_load<C>(s1, A, W, M, K, m0, n0, (kt + 3) * C::BK, tid);
      tile_mfma<C>(acc, As[1], Bs[1], wm, wn, lane);
      stage_store<C>(s0, As[0], Bs[0], tid);
      __syncthreads();
    }
    if (kt + 1 < nk) {  // two k-tiles left: buffer 0 holds kt, s1 holds kt + 1
      tile_mfma<C>(acc, As[0], Bs[0], wm, wn, lane);
      stage_store<C>(s1, As[1], Bs[1], tid);
      __syncthreads();
      tile_mfma<C>(acc, As[1], Bs[1], wm, wn, lane);
    } else {
      tile_mfma<C>(acc, As[0], Bs[0], wm, wn, lane);
    }
  }

  write_back<C::TM, C::TN>(acc, epi, m0 + wm * C::WM, n0 + wn * C::WN, M, lane);
}

// 128x128 tile, 2x2 wavefronts of 64x64, two register stages, registers
// budgeted for two workgroups per CU.
using TileS = TileCfg<128, 128, 64, 2, 2, 2, 2>;

template <class C, class Epi>
static hipError_t launch_tile(const void *a, const void *w, int m, int n, int k, const Epi &epi,
                              hipStream_t s) {
  const int grid = ((m + C::BM - 1) / C::BM) * (n / C::BN);
  gemm_bf16_kernel<C, Epi><<<grid, C::NT, 0, s>>>(static_cast<const bf16 *>(a),
                                                  static_cast<const bf16 *>(w), m, n, k, epi);
  return hipGetLastError();
}

// ------------------------------------------------------------------ 256x256 tile
//
// For projections where every token is active: a 256x256x64 workgroup tile
// on four wavefronts of 128x128 (16 accumulators each, which live in the
// accumulation registers).  Operands go from global memory straight into LDS
// (global_load_lds_dwordx4: no staging registers, no LDS write instructions)
// through two 64 KB stages of 128-byte rows whose 16-byte chunks are permuted
// by an XOR with the row pair index, so the 16 rows one fragment read touches
// per chunk hit 16 distinct bank groups.  Every MFMA is issued in a fixed
// slot with at most one memory operation beside it (sched_barrier): the eight
// fragment reads of the next k16 step, the sixteen loads of the next k-tile
// and the barrier are spread over the 64 MFMAs of a k-tile, and the loads of
// k-tile t+1 have the whole of k-tile t to land.
namespace big {

constexpr int kStage = 65536;  // bytes per stage: activation rows [0, 32K), weight rows [32K, 64K)

struct Frag {
  bf16x8 x[4];  // activation rows (MFMA B operand)
  bf16x8 w[4];  // weight rows (MFMA A operand)
};

__device__ __forceinline__ void pin() { __builtin_amdgcn_sched_barrier(0); }

__device__ __forceinline__ int swz(int r, int kc) { return kc ^ ((r >> 1) & 7); }

// Load instruction q (0..63 per k-tile, 16 per wavefront) moves 1 KB: q < 32
// carries activation rows 8q..8q+7, q >= 32 weight rows 8(q-32)..; lane l
// writes LDS bytes [16 l, 16 l + 16) of the block, i.e. row 8q + l / 8 at
// physical chunk l % 8, which holds logical chunk swz(row, l % 8).
// `stage` is the LDS byte address of the stage (wave-uniform, so M0 is set
// from a scalar register).
__device__ __forceinline__ void load_lds(unsigned stage, int q, const bf16 *A, const bf16 *W,
                                         int M, int K, int m0, int n0, int k0, int lane) {
  const int rr = lane >> 3, pc = lane & 7;
  const bf16 *g;
  if (q < 32) {
    const int r = q * 8 + rr;
    g = A + (size_t)min(m0 + r, M - 1) * K + k0 + swz(r, pc) * 8;
  } else {
    const int r = (q - 32) * 8 + rr;
    g = W + (size_t)(n0 + r) * K + k0 + swz(r, pc) * 8;
  }
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(__builtin_amdgcn_readfirstlane(stage + q * 1024))
               : "memory", "m0");
}

// Fragment r of k16 step s, in the order the MFMAs need them: x0 w0 x1 x2 x3 w1 w2 w3.
__device__ __forceinline__ void read_frag(Frag &f, int r, const unsigned char *stage, int s, int wm,
                                          int wn, int lane) {
  const bool is_x = (r == 0 || r == 2 || r == 3 || r == 4);
  const int idx = r <= 1 ? 0 : (r <= 4 ? r - 1 : r - 4);
  const int kc = s * 2 + (lane >> 5);
  if (is_x) {
    const int row = wm * 128 + idx * 32 + (lane & 31);
    f.x[idx] = *reinterpret_cast<const bf16x8 *>(stage + row * 128 + swz(row, kc) * 16);
  } else {
    const int row = wn * 128 + idx * 32 + (lane & 31);
    f.w[idx] = *reinterpret_cast<const bf16x8 *>(stage + 32768 + row * 128 + swz(row, kc) * 16);
  }
}

__device__ __forceinline__ void mfma(f32x16 (&acc)[4][4], const Frag &f, int q) {
  const int j = q >> 2, i = q & 3;
  acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.w[j], f.x[i], acc[j][i], 0, 0, 0);
}

// Own loads landed in LDS, own LDS reads done, then the workgroup barrier.
__device__ __forceinline__ void barrier() {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace big

// Write-back of the 256x256 tile through LDS (free once the main loop is
// done).  In the accumulator layout a store instruction would write 16 bytes
// into each of 32 rows; instead each wavefront writes one 32-row block of its
// 128x128 accumulators to LDS as fp32 and reads it back row-major, so lane l
// owns columns 4 (l % 32) .. + 3 of rows l / 32 + 2k: one store instruction
// then covers two whole 128-column row segments.  Biases and per-row
// addressing data of the tile were staged in LDS by the caller; residual
// priors of the next block are loaded before this block's stores.
namespace big {
constexpr int kWbStride = 132;  // floats per staged row (128 + 4: no bank conflicts)
static_assert(4 * 32 * kWbStride * 4 <= 2 * kStage, "staged write-back fits the stages");
}  // namespace big

// `side` holds the tile's 256 biases (floats [0, 256)) followed by its 256 row
// records; both were loaded into LDS during the prologue.
template <class Epi>
__device__ __forceinline__ void write_back_staged(const f32x16 (&acc)[4][4], const Epi &epi, int m0,
                                                  int n0, int wm, int wn, int M, int lane, int wave,
                                                  unsigned char *smem, const unsigned char *side) {
  using namespace big;
  using Row = typename Epi::Row;
  float *st = reinterpret_cast<float *>(smem) + wave * 32 * kWbStride;
  const Row *rows = reinterpret_cast<const Row *>(side + 1024) + wm * 128;
  const int c4 = (lane & 31) * 4, half = lane >> 5;
  const typename Epi::Col col = epi.col(n0 + wn * 128 + c4);
  const f32x4 b = *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(side) +
                                                    wn * 128 + c4);
  f32x4 pr[2][16];  // residual priors; zero for epilogues without one
#pragma unroll
  for (int k = 0; k < 16; ++k) pr[0][k] = pr[1][k] = f32x4{};
  auto load_priors = [&](int i, f32x4 (&dst)[16]) {
#pragma unroll
    for (int k = 0; k < 16; ++k)
      dst[k] = Epi::kPrior ? epi.prior(rows[i * 32 + half + 2 * k], col) : f32x4{};
  };
  if constexpr (Epi::kPrior) load_priors(0, pr[0]);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // block row i of the accumulators -> LDS rows 0..31 of this wavefront
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4 *>(st + (lane & 31) * kWbStride + j * 32 + g * 8 + half * 4) =
            f32x4{acc[j][i][4 * g + 0], acc[j][i][4 * g + 1], acc[j][i][4 * g + 2],
                  acc[j][i][4 * g + 3]};
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    f32x4 v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k)
      v[k] = *reinterpret_cast<const f32x4 *>(st + (half + 2 * k) * kWbStride + c4);
    if constexpr (Epi::kPrior) {
      if (i + 1 < 4) load_priors(i + 1, pr[(i + 1) & 1]);
#pragma unroll
      for (int k = 0; k < 16; ++k) keep(pr[i & 1][k]);
    }
    const int rbase = m0 + wm * 128 + i * 32;
    auto value = [&](int k) -> f32x4 {
      if constexpr (Epi::kPrior) return v[k] + b + pr[i & 1][k];
      else return v[k] + b;
    };
    if (rbase + 32 <= M) {  // the whole block exists: no per-row guard
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int r = half + 2 * k;
        epi.store(rows[i * 32 + r], rbase + r, col, value(k));
      }
    } else {
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int r = half + 2 * k;
        if (rbase + r < M) epi.store(rows[i * 32 + r], rbase + r, col, value(k));
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
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * kStage];
  // biases and row records of the tile for the write-back (5 KB)
  __shared__ __attribute__((aligned(16))) unsigned char side[1024 + 256 * sizeof(typename Epi::Row)];
  const int tiles_m = (M + 255) / 256, tiles_n = N / 256;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, gridDim.x), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * 256, n0 = tn * 256;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar address math
  const int wm = wave >> 1, wn = wave & 1;
  const int q0 = wave * 16;  // this wavefront's load instructions q0 .. q0 + 15
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) void *)smem;
  const unsigned lds_stage[2] = {lds0, lds0 + kStage};
  f32x16 acc[4][4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[j][i] = f32x16{};
  const int nk = K / 64;

  // k-tile 0 into stage 0; the first quarter of k-tile 1 into stage 1
#pragma unroll
  for (int p = 0; p < 16; ++p) load_lds(lds_stage[0], q0 + p, A, W, M, K, m0, n0, 0, lane);
  // the write-back's biases and row records, loaded while the tile computes
  if (tid < 64)
    *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(side) + tid * 4) = epi.bias4(n0 + tid * 4);
  reinterpret_cast<typename Epi::Row *>(side + 1024)[tid] = epi.row(min(m0 + tid, M - 1));
  barrier();
  Frag fa, fb;
#pragma unroll
  for (int r = 0; r < 8; ++r) read_frag(fa, r, smem, 0, wm, wn, lane);
  {
    const int k1 = min(1, nk - 1) * 64;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      load_lds(lds_stage[1], q0 + p, A, W, M, K, m0, n0, k1, lane);
      pin();
    }
  }

  for (int kt = 0; kt + 1 < nk; ++kt) {
    const int cur = kt & 1;
    const unsigned char *sc = smem + cur * kStage;
    const unsigned char *sn = smem + (cur ^ 1) * kStage;
    const unsigned ln = lds_stage[cur ^ 1], lc = lds_stage[cur];
    const int k1 = (kt + 1) * 64, k2 = min(kt + 2, nk - 1) * 64;
    // k16 steps 0..2: fragments of the next step; the rest of k-tile kt+1
#pragma unroll
    for (int st = 0; st < 3; ++st) {
      Frag &fc = (st & 1) ? fb : fa;
      Frag &fn = (st & 1) ? fa : fb;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        mfma(acc, fc, q);
        if (q < 8) read_frag(fn, q, sc, st + 1, wm, wn, lane);
        else if (st == 0) load_lds(ln, q0 + 4 + (q - 8), A, W, M, K, m0, n0, k1, lane);
        else if (st == 1 && q < 12) load_lds(ln, q0 + 12 + (q - 8), A, W, M, K, m0, n0, k1, lane);
        pin();
      }
    }
    // k16 step 3: barrier (k-tile kt+1 complete, stage cur free), first
    // fragments of k-tile kt+1, first quarter of k-tile kt+2 into stage cur
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      mfma(acc, fb, q);
      pin();
    }
    barrier();
    pin();
#pragma unroll
    for (int q = 4; q < 12; ++q) {
      mfma(acc, fb, q);
      read_frag(fa, q - 4, sn, 0, wm, wn, lane);
      pin();
    }
#pragma unroll
    for (int q = 12; q < 16; ++q) {
      mfma(acc, fb, q);
      load_lds(lc, q0 + (q - 12), A, W, M, K, m0, n0, k2, lane);
      pin();
    }
  }
  {  // last k-tile
    const unsigned char *sc = smem + ((nk - 1) & 1) * kStage;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      Frag &fc = (st & 1) ? fb : fa;
      Frag &fn = (st & 1) ? fa : fb;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        mfma(acc, fc, q);
        if (st < 3 && q < 8) read_frag(fn, q, sc, st + 1, wm, wn, lane);
        pin();
      }
    }
  }
  // the last quarter-tile loads (a clamped repeat of the final k-tile) land
  // and every wavefront is done with the stages before they hold the
  // write-back's staging rows
  barrier();
  write_back_staged(acc, epi, m0, n0, wm, wn, M, lane, wave, smem, side);
}

// The 256x256 tile is chosen when its tiles fill the compute units in whole
// waves well enough: at least 90% of the last wave, or 80% when K >= 2048
// (the longer main loop amortises the tile's fixed start and write-back).
// Otherwise the 128x128 tile, two workgroups per CU, fills the chip in finer
// steps.  Measured at MAR-L sizes: full-step QKV, fc1 and fc2 and
// cache-aware QKV take the large tile; the output projection and the other
// cache-aware GEMMs the small one.
bool gemm_large_tile(DType dt, int32_t m, int32_t n, int32_t k) {
  if (dt != DType::BF16 || n % 256 != 0 || m <= 0) return false;
  const long tiles = (long)((m + 255) / 256) * (n / 256);
  const long cus = device_cu_count();
  const long waves = (tiles + cus - 1) / cus;
  const double fill = (double)tiles / (double)(waves * cus);
  return fill >= 0.9 || (fill >= 0.8 && k >= 2048);
}

template <class Epi>
static hipError_t run_bf16(const void *a, const void *w, int m, int n, int k, const Epi &epi,
                           hipStream_t s) {
  if (m == 0) return hipSuccess;
  if (n % TileS::BN != 0 || k % TileS::BK != 0) return hipErrorInvalidValue;
  if (gemm_large_tile(DType::BF16, m, n, k)) {
    const int grid = ((m + 255) / 256) * (n / 256);
    gemm_bf16_big_kernel<Epi><<<grid, 256, 0, s>>>(static_cast<const bf16 *>(a),
                                                    static_cast<const bf16 *>(w), m, n, k, epi);
    return hipGetLastError();
  }
  return launch_tile<TileS>(a, w, m, n, k, epi, s);
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
  gemm_f32_kernel<Epi><<<grid, 256, 0, s>>>(static_cast<const float *>(a),
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
