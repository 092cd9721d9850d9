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
// The write-back runs in three phases so that no load waits behind a store
// (on this architecture the vector-memory counter also counts stores):
//   row(r)            per-row addressing data (may load the row map),
//   bias(col0)        the bias of four columns,
//   prior(row, col0)  the value the result is added to (residual epilogues),
// all issued before the first store(row, r, col0, v), v = acc + bias + prior.

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
  __device__ __forceinline__ Row row(int r) const { return map[r]; }
  __device__ __forceinline__ f32x4 bias4(int col0) const { return load_bias4(bias, col0); }
  __device__ __forceinline__ f32x4 prior(const Row &, int) const { return f32x4{}; }
  __device__ __forceinline__ void store(const Row &m, int r, int col0, f32x4 v) const {
    if (col0 < d_model) {
      store4(q + (size_t)r * d_model + col0, v);
      return;
    }
    int c = col0 - d_model;
    T *dst = kc;
    if (c >= d_model) {
      c -= d_model;
      dst = vc;
    }
    const int h = c / head_dim, d = c - h * head_dim;
    store4(dst + ((size_t)(m.b * n_heads + h) * n_tokens + m.tok) * head_dim + d, v);
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
  using Row = int32_t;  // residual-stream row
  __device__ __forceinline__ Row row(int r) const { return map[r].x_row; }
  __device__ __forceinline__ f32x4 bias4(int col0) const { return load_bias4(bias, col0); }
  __device__ __forceinline__ f32x4 prior(const Row &xr, int col0) const {
    return *reinterpret_cast<const f32x4 *>(x + (size_t)xr * n + col0);
  }
  __device__ __forceinline__ void store(const Row &xr, int, int col0, f32x4 v) const {
    *reinterpret_cast<f32x4 *>(x + (size_t)xr * n + col0) = v;
  }
};

template <typename T>
struct EpiGelu {
  static constexpr bool kPrior = false;
  T *h;
  const float *bias;
  int n;
  using Row = int32_t;
  __device__ __forceinline__ Row row(int r) const { return r; }
  __device__ __forceinline__ f32x4 bias4(int col0) const { return load_bias4(bias, col0); }
  __device__ __forceinline__ f32x4 prior(const Row &, int) const { return f32x4{}; }
  __device__ __forceinline__ void store(const Row &, int r, int col0, f32x4 v) const {
    f32x4 g = {gelu_erf(v[0]), gelu_erf(v[1]), gelu_erf(v[2]), gelu_erf(v[3])};
    store4(h + (size_t)r * n + col0, g);
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
// block rows at a time, at most 16 four-column groups (64 registers).
template <int TM, int TN, class Epi>
__device__ __forceinline__ void write_back(const f32x16 (&acc)[TN][TM], const Epi &epi, int row0,
                                           int col_base, int M, int lane) {
  typename Epi::Row rinfo[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) rinfo[i] = epi.row(min(row0 + i * 32 + (lane & 31), M - 1));
  f32x4 b[TN][4];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) b[j][g] = epi.bias4(col_base + j * 32 + g * 8 + (lane >> 5) * 4);
#pragma unroll
  for (int i = 0; i < TM; ++i) keep(rinfo[i]);
  constexpr int IB = (16 / (TN * 4)) < 1 ? 1 : ((16 / (TN * 4)) > TM ? TM : 16 / (TN * 4));
#pragma unroll
  for (int i0 = 0; i0 < TM; i0 += IB) {
    f32x4 pr[IB][TN][4];
#pragma unroll
    for (int ii = 0; ii < IB; ++ii)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          pr[ii][j][g] = Epi::kPrior
                             ? epi.prior(rinfo[i0 + ii], col_base + j * 32 + g * 8 + (lane >> 5) * 4)
                             : f32x4{};
    if constexpr (Epi::kPrior) {
#pragma unroll
      for (int ii = 0; ii < IB; ++ii)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) keep(pr[ii][j][g]);
    }
#pragma unroll
    for (int ii = 0; ii < IB; ++ii) {
      const int i = i0 + ii;
      const int row = row0 + i * 32 + (lane & 31);
      if (row >= M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 a = {acc[j][i][4 * g + 0], acc[j][i][4 * g + 1], acc[j][i][4 * g + 2],
                           acc[j][i][4 * g + 3]};
          epi.store(rinfo[i], row, col_base + j * 32 + g * 8 + (lane >> 5) * 4,
                    a + b[j][g] + pr[ii][j][g]);
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
// 256x256 tile, 2x4 wavefronts of 128x64 (two per SIMD), one register stage:
// for large-M projections to wide outputs (measured faster there).
using TileL = TileCfg<256, 256, 64, 2, 4, 1, 1>;

template <class C, class Epi>
static hipError_t launch_tile(const void *a, const void *w, int m, int n, int k, const Epi &epi,
                              hipStream_t s) {
  const int grid = ((m + C::BM - 1) / C::BM) * (n / C::BN);
  gemm_bf16_kernel<C, Epi><<<grid, C::NT, 0, s>>>(static_cast<const bf16 *>(a),
                                                  static_cast<const bf16 *>(w), m, n, k, epi);
  return hipGetLastError();
}

bool gemm_large_tile(DType dt, int32_t m, int32_t n) {
  if (dt != DType::BF16) return false;
  const long large_tiles = (long)((m + TileL::BM - 1) / TileL::BM) * (n / TileL::BN);
  return n % TileL::BN == 0 && n >= 3072 && large_tiles >= 512;
}

template <class Epi>
static hipError_t run_bf16(const void *a, const void *w, int m, int n, int k, const Epi &epi,
                           hipStream_t s) {
  if (m == 0) return hipSuccess;
  if (n % TileS::BN != 0 || k % TileS::BK != 0) return hipErrorInvalidValue;
  if (gemm_large_tile(DType::BF16, m, n)) return launch_tile<TileL>(a, w, m, n, k, epi, s);
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
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= M) continue;
    const typename Epi::Row r = epi.row(row);
    const f32x4 v = {acc[i][0], acc[i][1], acc[i][2], acc[i][3]};
    epi.store(r, row, n0 + tx * 4, v + b + (Epi::kPrior ? epi.prior(r, n0 + tx * 4) : f32x4{}));
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
