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
// bf16 path: workgroup tile BM x BN x BK, 2x2 wavefronts, each wavefront a
// (BM/2) x (BN/2) block of 32x32 MFMA tiles (v_mfma_f32_32x32x16_bf16, fp32
// accumulators).  Tiles are staged global -> registers -> LDS with double
// buffering: the loads of k-tile t+1 are in flight while k-tile t is computed.
// LDS rows are padded by 16 bytes, which makes the 16-byte MFMA operand reads
// (32 rows at one k offset) bank-conflict free.
//
// fp32 path: plain FMA, 64x64 tiles, 4x4 outputs per thread.
#include "device_common.h"

namespace marche {

// ------------------------------------------------------------------ epilogues

template <typename T>
struct EpiQkv {
  T *q;
  T *kc;
  T *vc;
  const float *bias;
  const RowMap *map;
  int d_model, head_dim, n_heads, n_tokens;
  __device__ __forceinline__ void operator()(int row, int col, float v) const {
    v += bias[col];
    if (col < d_model) {
      q[(size_t)row * d_model + col] = from_f32<T>(v);
      return;
    }
    int c = col - d_model;
    T *dst = kc;
    if (c >= d_model) {
      c -= d_model;
      dst = vc;
    }
    const int h = c / head_dim, d = c - h * head_dim;
    const RowMap m = map[row];
    dst[((size_t)(m.b * n_heads + h) * n_tokens + m.tok) * head_dim + d] = from_f32<T>(v);
  }
};

// TAG only distinguishes the output projection (0) from fc2 (1) as kernel
// symbols, so per-kernel profiles can tell them apart.
template <int TAG>
struct EpiResid {
  float *x;
  const float *bias;
  const RowMap *map;
  int n;
  __device__ __forceinline__ void operator()(int row, int col, float v) const {
    float *p = x + (size_t)map[row].x_row * n + col;
    *p = *p + (v + bias[col]);
  }
};

template <typename T>
struct EpiGelu {
  T *h;
  const float *bias;
  int n;
  __device__ __forceinline__ void operator()(int row, int col, float v) const {
    h[(size_t)row * n + col] = from_f32<T>(gelu_erf(v + bias[col]));
  }
};

// ------------------------------------------------------------------ bf16 MFMA

template <int BM_, int BN_, int BK_, int WGM_, int WGN_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_;
  static constexpr int WGM = WGM_, WGN = WGN_;  // wavefront grid
  static constexpr int NT = WGM * WGN * 64;
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int LDS_STRIDE = BK + 8;    // elements; +16 bytes per row
  static constexpr int CPR = BK / 8;           // 16-byte chunks per tile row
  static constexpr int A_CHUNKS = BM * CPR / NT;
  static constexpr int B_CHUNKS = BN * CPR / NT;
  static constexpr int LDS_BYTES = 2 * (BM + BN) * LDS_STRIDE * 2;
  static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile not divisible");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
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

template <class Cfg>
struct Stage {
  u32x4 a[Cfg::A_CHUNKS];
  u32x4 b[Cfg::B_CHUNKS];
};

template <class Cfg>
__device__ __forceinline__ void stage_load(Stage<Cfg> &st, const bf16 *__restrict__ A,
                                           const bf16 *__restrict__ W, int M, int K, int m0,
                                           int n0, int k0, int tid) {
#pragma unroll
  for (int i = 0; i < Cfg::A_CHUNKS; ++i) {
    const int c = i * Cfg::NT + tid, row = c / Cfg::CPR, col = (c % Cfg::CPR) * 8;
    const int grow = min(m0 + row, M - 1);
    st.a[i] = *reinterpret_cast<const u32x4 *>(A + (size_t)grow * K + k0 + col);
  }
#pragma unroll
  for (int i = 0; i < Cfg::B_CHUNKS; ++i) {
    const int c = i * Cfg::NT + tid, row = c / Cfg::CPR, col = (c % Cfg::CPR) * 8;
    st.b[i] = *reinterpret_cast<const u32x4 *>(W + (size_t)(n0 + row) * K + k0 + col);
  }
}

template <class Cfg>
__device__ __forceinline__ void stage_store(const Stage<Cfg> &st, bf16 *As, bf16 *Bs, int tid) {
#pragma unroll
  for (int i = 0; i < Cfg::A_CHUNKS; ++i) {
    const int c = i * Cfg::NT + tid, row = c / Cfg::CPR, col = (c % Cfg::CPR) * 8;
    *reinterpret_cast<u32x4 *>(&As[row * Cfg::LDS_STRIDE + col]) = st.a[i];
  }
#pragma unroll
  for (int i = 0; i < Cfg::B_CHUNKS; ++i) {
    const int c = i * Cfg::NT + tid, row = c / Cfg::CPR, col = (c % Cfg::CPR) * 8;
    *reinterpret_cast<u32x4 *>(&Bs[row * Cfg::LDS_STRIDE + col]) = st.b[i];
  }
}

// One BK-deep slab of MFMAs for this wavefront's TM x TN block of 32x32 tiles.
template <class Cfg>
__device__ __forceinline__ void tile_mfma(f32x16 (&acc)[Cfg::TM][Cfg::TN], const bf16 *As,
                                          const bf16 *Bs, int wm, int wn, int lane) {
  constexpr int LS = Cfg::LDS_STRIDE;
  const int lrow = lane & 31, lk = (lane >> 5) * 8;
#pragma unroll
  for (int kk = 0; kk < Cfg::BK; kk += 16) {
    bf16x8 af[Cfg::TM], bw[Cfg::TN];
#pragma unroll
    for (int i = 0; i < Cfg::TM; ++i)
      af[i] = *reinterpret_cast<const bf16x8 *>(&As[(wm * Cfg::WM + i * 32 + lrow) * LS + kk + lk]);
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j)
      bw[j] = *reinterpret_cast<const bf16x8 *>(&Bs[(wn * Cfg::WN + j * 32 + lrow) * LS + kk + lk]);
#pragma unroll
    for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
      for (int j = 0; j < Cfg::TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bw[j], acc[i][j], 0, 0, 0);
  }
}

template <class Cfg, class Epi>
__global__ __launch_bounds__(Cfg::NT) void gemm_bf16_kernel(const bf16 *__restrict__ A,
                                                            const bf16 *__restrict__ W, int M,
                                                            int N, int K, Epi epi) {
  constexpr int BM = Cfg::BM, BN = Cfg::BN, BK = Cfg::BK, LS = Cfg::LDS_STRIDE;
  __shared__ __attribute__((aligned(16))) bf16 As[2][BM * LS];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * LS];

  const int tiles_m = (M + BM - 1) / BM, tiles_n = N / BN;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, gridDim.x), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / Cfg::WGN, wn = wave % Cfg::WGN;

  f32x16 acc[Cfg::TM][Cfg::TN];
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j) acc[i][j] = f32x16{};

  // Software pipeline: the global loads of k-tile t+1 are issued before the
  // MFMAs of k-tile t and land in the other LDS buffer after them.
  const int nk = K / BK;
  Stage<Cfg> st;
  stage_load<Cfg>(st, A, W, M, K, m0, n0, 0, tid);
  stage_store<Cfg>(st, As[0], Bs[0], tid);
  __syncthreads();
  for (int kt = 0; kt + 1 < nk; ++kt) {
    const int cur = kt & 1;
    stage_load<Cfg>(st, A, W, M, K, m0, n0, (kt + 1) * BK, tid);
    tile_mfma<Cfg>(acc, As[cur], Bs[cur], wm, wn, lane);
    stage_store<Cfg>(st, As[cur ^ 1], Bs[cur ^ 1], tid);
    __syncthreads();
  }
  tile_mfma<Cfg>(acc, As[(nk - 1) & 1], Bs[(nk - 1) & 1], wm, wn, lane);

  // 32x32 accumulator layout: lane -> column (lane & 31); register r ->
  // row (r / 4) * 8 + (lane / 32) * 4 + r % 4.
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = m0 + wm * Cfg::WM + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
      if (row >= M) continue;
#pragma unroll
      for (int j = 0; j < Cfg::TN; ++j) {
        const int col = n0 + wn * Cfg::WN + j * 32 + (lane & 31);
        epi(row, col, acc[i][j][r]);
      }
    }
  }
}

// 128x128 tile, 2x2 wavefronts of 64x64: two workgroups per CU; used when
// the 256x256 grid would leave CUs idle.
using TileS = TileCfg<128, 128, 64, 2, 2>;
// 256x256 tile, 2x2 wavefronts of 128x128 (accumulators in AGPRs): one
// workgroup per CU, four times the MFMA work per k-tile and per LDS byte.
using TileL = TileCfg<256, 256, 64, 2, 2>;

template <class C, class Epi>
static hipError_t launch_tile(const void *a, const void *w, int m, int n, int k, const Epi &epi,
                              hipStream_t s) {
  const int grid = ((m + C::BM - 1) / C::BM) * (n / C::BN);
  gemm_bf16_kernel<C, Epi><<<grid, C::NT, 0, s>>>(static_cast<const bf16 *>(a),
                                                  static_cast<const bf16 *>(w), m, n, k, epi);
  return hipGetLastError();
}

template <class Epi>
static hipError_t run_bf16(const void *a, const void *w, int m, int n, int k, const Epi &epi,
                           hipStream_t s) {
  if (m == 0) return hipSuccess;
  if (n % TileS::BN != 0 || k % TileS::BK != 0) return hipErrorInvalidValue;
  // 256 CUs: prefer the large tile when it still yields at least two
  // workgroups per CU.
  const long large_tiles = (long)((m + TileL::BM - 1) / TileL::BM) * (n / TileL::BN);
  if (n % TileL::BN == 0 && large_tiles >= 512) return launch_tile<TileL>(a, w, m, n, k, epi, s);
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
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) epi(row, n0 + tx * 4 + j, acc[i][j]);
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
