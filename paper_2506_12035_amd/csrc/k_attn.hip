// Cache-aware bidirectional attention (Algorithm 1 / Section 4.1) and the
// attention-mass score pass of the selection layer (Section 4.2).
//
// Because the fresh K/V of the active tokens were already written into the
// layer's cache by the QKV epilogue, the active segment K_A and the cached
// segment K_C are one resident buffer [b][h][N][d_h]: the online-softmax
// merge of the two segments (Appendix A) becomes the kernel's own loop over
// key tiles, with a running maximum and a rescaled running sum, and no K/V is
// ever concatenated or copied.
//
// bf16 kernel (gfx950 MFMA, v_mfma_f32_32x32x16_bf16), one workgroup per
// (image, head, chunk of NW*32 active queries), one wavefront per 32 queries:
//   - K and V tiles of 64 keys stream global -> registers -> LDS, double
//     buffered (the next tile's loads are in flight during this tile's math);
//   - S^T = K Q^T is formed so that lane l owns query (l & 31): the row
//     maximum and sum need one cross-half exchange, and the accumulator
//     rescale is a per-lane scalar;
//   - O^T = V^T P^T: P stays in registers (converted to bf16), V is stored
//     transposed in LDS with the keys of every 16-key group permuted to match
//     the accumulator layout of S^T, so each MFMA operand is one 16-byte read.
// Softmax runs in the log2 domain with fp32 statistics.
//
// The same kernel also takes the two segments as separate buffers (SEG2):
// key tiles of the first segment, then of the second, in one online-softmax
// pass -- Appendix A's merge without concatenation, as the stand-alone
// two-segment attention of Appendix B's comparison.
#include <type_traits>

#include "device_common.h"

namespace marche {

constexpr int TK = 64;  // keys per tile

// Position of key k (0..15) inside its 16-key group in the transposed V tile.
// S^T's accumulator gives lane half hf the keys {4hf..4hf+3, 8+4hf..8+4hf+3}
// of each 16-key group; this places exactly those at positions 8hf..8hf+7.
__device__ __forceinline__ int vperm16(int k) {
  return (k & 3) | (((k >> 3) & 1) << 2) | (((k >> 2) & 1) << 3);
}

// Element offsets inside one tile's K and V^T blocks.  Padded layout: rows of
// DH + 8 (K) and TK + 8 (V^T) elements.  Swizzled layout (DH = 64 only): rows
// of 64 elements whose 16-byte chunks are permuted by an XOR with the row
// pair index, so 16 consecutive rows read at one chunk hit distinct banks
// without padding (8 KB per tile for K and for V^T).
template <int DH, bool SWZ>
__device__ __forceinline__ int k_off(int key, int d) {
  if constexpr (SWZ) return key * 64 + ((((d >> 3) ^ (key >> 1)) & 7) << 3) + (d & 7);
  else return key * (DH + 8) + d;
}
template <int DH, bool SWZ>
__device__ __forceinline__ int vt_off(int row, int pos) {
  if constexpr (SWZ) return row * 64 + ((((pos >> 3) ^ (row >> 1)) & 7) << 3) + (pos & 7);
  else return row * (TK + 8) + pos;
}

// One 64-key tile of the online softmax for one wavefront's 32 queries.
// ks: the tile's K rows in LDS; vt: its transposed V (keys of each 16-key
// group permuted by vperm16); t0: the tile's first key within a segment of
// ns keys, MASK set when the tile runs past the segment's end.  Updates the
// running maximum, sum and the O^T accumulators in the log2 domain (sl2 =
// log2(e) / sqrt(d_h) > 0).  The maximum is taken over the raw logits: as
// rounding a product by a positive constant is monotone, fl(max * sl2) is
// the maximum of the scaled logits exactly, and the scale then folds into
// the exponent's argument as one FMA per logit.
template <int DH, bool SWZ = false, bool MASK = false>
__device__ __forceinline__ void attn_tile(const bf16 *ks, const bf16 *vt, const bf16x8 (&qf)[DH / 16],
                                          f32x16 (&acc)[(DH + 31) / 32], float &m_run, float &l_run,
                                          int t0, int ns, float sl2, int lane) {
  static_assert(!SWZ || DH == 64, "swizzled tiles hold 64-element rows");
  constexpr int QS = DH / 16, ODB = (DH + 31) / 32;
  // S^T for two 32-key blocks: lane -> query (lane & 31),
  // register r -> key (r / 4) * 8 + (lane / 32) * 4 + r % 4 of the block.
  f32x16 s[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    s[kb] = f32x16{};
#pragma unroll
    for (int st = 0; st < QS; ++st) {
      const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(
          &ks[k_off<DH, SWZ>(kb * 32 + (lane & 31), st * 16 + (lane >> 5) * 8)]);
      s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[st], s[kb], 0, 0, 0);
    }
  }
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if constexpr (MASK) {
        const int key = t0 + kb * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        if (key >= ns) s[kb][r] = -INFINITY;
      }
      mx = fmaxf(mx, s[kb][r]);
    }
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m_new = fmaxf(m_run, mx * sl2);
  const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
  float psum = 0.f;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float p = __builtin_amdgcn_exp2f(fmaf(s[kb][r], sl2, -m_new));
      s[kb][r] = p;
      psum += p;
    }
  l_run = l_run * alpha + psum;
  m_run = m_new;
#pragma unroll
  for (int d = 0; d < ODB; ++d) acc[d] *= alpha;

  // O^T += V^T P^T over the 64 keys of the tile, 16 keys per MFMA.
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      bf16x8 pb;
#pragma unroll
      for (int e = 0; e < 8; ++e) pb[e] = (bf16)s[kb][8 * u + e];
#pragma unroll
      for (int d = 0; d < ODB; ++d) {
        const bf16x8 va = *reinterpret_cast<const bf16x8 *>(
            &vt[vt_off<DH, SWZ>(d * 32 + (lane & 31), kb * 32 + 16 * u + (lane >> 5) * 8)]);
        acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, acc[d], 0, 0, 0);
      }
    }
}

// ALIGNED: every segment's length is a multiple of TK, so no key tile runs
// past its segment and only the unmasked tile step is compiled.
template <int DH, int NW, bool SEG2, bool ALIGNED>
__global__ __launch_bounds__(NW * 64) void attn_mfma_kernel(AttnArgs a, int chunks) {
  constexpr int NT = NW * 64;
  constexpr int KS = DH + 8;        // K tile row stride (elements)
  constexpr int ODB = (DH + 31) / 32;
  constexpr int DHV = ODB * 32;     // rows of the transposed V tile
  constexpr int VS = TK + 8;        // V^T tile row stride (elements)
  constexpr int CPR = DH / 8;       // 16-byte chunks per K/V row
  constexpr int TCH = TK * CPR;     // chunks per tile per matrix
  constexpr int LPT = (TCH + NT - 1) / NT;
  constexpr int QS = DH / 16;       // k-steps of the QK^T contraction
  __shared__ __attribute__((aligned(16))) bf16 Ks[2][TK * KS];
  __shared__ __attribute__((aligned(16))) bf16 Vt[2][DHV * VS];

  const int id = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = id / chunks, chunk = id - bh * chunks;
  const int b = bh / a.n_heads, h = bh - b * a.n_heads;
  const int r0 = a.a_off ? a.a_off[b] : b * a.a_max;
  const int na = a.a_off ? a.a_off[b + 1] - r0 : a.a_max;
  const int q0 = chunk * NW * 32;
  if (q0 >= na) return;  // uniform over the workgroup

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int N = a.n_tokens, D = a.d_model;
  const int N2 = SEG2 ? a.n2 : 0;
  const bf16 *kg = static_cast<const bf16 *>(a.k_cache) + (size_t)(b * a.n_heads + h) * N * DH;
  const bf16 *vg = static_cast<const bf16 *>(a.v_cache) + (size_t)(b * a.n_heads + h) * N * DH;
  const bf16 *kg2 = SEG2 ? static_cast<const bf16 *>(a.k2) + (size_t)(b * a.n_heads + h) * N2 * DH : kg;
  const bf16 *vg2 = SEG2 ? static_cast<const bf16 *>(a.v2) + (size_t)(b * a.n_heads + h) * N2 * DH : vg;
  const int nt1 = (N + TK - 1) / TK;
  // key tile t: first segment for t < nt1, else the second; its first key
  // within the segment and the segment's length
  auto seg_of = [&](int t, const bf16 *&kb, const bf16 *&vb, int &t0, int &ns) {
    if (!SEG2 || t < nt1) {
      kb = kg; vb = vg; t0 = t * TK; ns = N;
    } else {
      kb = kg2; vb = vg2; t0 = (t - nt1) * TK; ns = N2;
    }
  };

  // V^T rows beyond DH (padding up to a multiple of 32) hold zeros.
  if constexpr (DHV > DH) {
    for (int i = tid; i < 2 * (DHV - DH) * VS; i += NT) {
      const int buf = i / ((DHV - DH) * VS), rem = i % ((DHV - DH) * VS);
      Vt[buf][DH * VS + rem] = (bf16)0.0f;
    }
  }

  // This wavefront's queries as the B operand of S^T = K Q^T.
  const int wq0 = q0 + wave * 32;
  const int qi = wq0 + (lane & 31);
  const bf16 *qrow = static_cast<const bf16 *>(a.q) + (size_t)(r0 + min(qi, na - 1)) * D + h * DH;
  bf16x8 qf[QS];
#pragma unroll
  for (int s = 0; s < QS; ++s)
    qf[s] = *reinterpret_cast<const bf16x8 *>(qrow + s * 16 + (lane >> 5) * 8);

  // K tiles are staged as 16-byte chunks; V tiles as pairs of keys so that
  // the transposed write to LDS packs two keys into one 32-bit word (keys 2p
  // and 2p+1 are adjacent in the permuted layout).
  constexpr int VPCH = TCH / 2;
  constexpr int LPV = (VPCH + NT - 1) / NT;
  u32x4 rk[LPT], rv0[LPV], rv1[LPV];
  auto gload = [&](int t) {
    const bf16 *kb, *vb;
    int t0, ns;
    seg_of(t, kb, vb, t0, ns);
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      const int c = i * NT + tid;
      if (c < TCH) {
        const int key = min(t0 + c / CPR, ns - 1), d = (c % CPR) * 8;
        rk[i] = *reinterpret_cast<const u32x4 *>(kb + (size_t)key * DH + d);
      }
    }
#pragma unroll
    for (int i = 0; i < LPV; ++i) {
      const int c = i * NT + tid;
      if (c < VPCH) {
        const int kp = c / CPR, d = (c % CPR) * 8;
        const int k0 = min(t0 + 2 * kp, ns - 1), k1 = min(t0 + 2 * kp + 1, ns - 1);
        rv0[i] = *reinterpret_cast<const u32x4 *>(vb + (size_t)k0 * DH + d);
        rv1[i] = *reinterpret_cast<const u32x4 *>(vb + (size_t)k1 * DH + d);
      }
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      const int c = i * NT + tid;
      if (c < TCH) {
        const int key = c / CPR, d = (c % CPR) * 8;
        *reinterpret_cast<u32x4 *>(&Ks[buf][key * KS + d]) = rk[i];
      }
    }
#pragma unroll
    for (int i = 0; i < LPV; ++i) {
      const int c = i * NT + tid;
      if (c < VPCH) {
        const int kp = c / CPR, d = (c % CPR) * 8;
        const int pos = ((2 * kp) & ~15) | vperm16((2 * kp) & 15);
        unsigned *vt = reinterpret_cast<unsigned *>(&Vt[buf][d * VS + pos]);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const unsigned w0 = rv0[i][e >> 1], w1 = rv1[i][e >> 1];
          const unsigned lo = (e & 1) ? (w0 >> 16) : (w0 & 0xFFFFu);
          const unsigned hi = (e & 1) ? (w1 & 0xFFFF0000u) : (w1 << 16);
          vt[e * (VS / 2)] = lo | hi;
        }
      }
    }
  };

  const float sl2 = 1.4426950408889634f / sqrtf((float)DH);  // log2(e) / sqrt(d_h)
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 acc[ODB];
#pragma unroll
  for (int d = 0; d < ODB; ++d) acc[d] = f32x16{};

  const int ntiles = nt1 + (SEG2 ? (N2 + TK - 1) / TK : 0);
  gload(0);
  sstore(0);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int cur = t & 1;
    int t0 = t * TK, ns = N;
    if constexpr (SEG2) {
      const bf16 *kb, *vb;
      seg_of(t, kb, vb, t0, ns);
    }
    const bool more = t + 1 < ntiles;
    if (more) gload(t + 1);
    if (ALIGNED || t0 + TK <= ns)
      attn_tile<DH>(Ks[cur], Vt[cur], qf, acc, m_run, l_run, t0, ns, sl2, lane);
    else
      attn_tile<DH, false, true>(Ks[cur], Vt[cur], qf, acc, m_run, l_run, t0, ns, sl2, lane);
    if (more) sstore(cur ^ 1);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  if (qi < na) {
    bf16 *orow = static_cast<bf16 *>(a.o) + (size_t)(r0 + qi) * D + h * DH;
#pragma unroll
    for (int d = 0; d < ODB; ++d)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int dh0 = d * 32 + g * 8 + (lane >> 5) * 4;
        if (dh0 < DH) {
          bf16x4 pk = {(bf16)(acc[d][4 * g + 0] * inv), (bf16)(acc[d][4 * g + 1] * inv),
                       (bf16)(acc[d][4 * g + 2] * inv), (bf16)(acc[d][4 * g + 3] * inv)};
          *reinterpret_cast<bf16x4 *>(orow + dh0) = pk;
        }
      }
  }
}

// ------------------------------------------------------------ cache-aware kernel, head width 64
//
// Cache-aware layers at head width 64 with every key tile whole (N a multiple
// of 64): one workgroup per (image, head, chunk of QB*32 active queries), one
// wavefront per 32 queries over all keys.  Key tiles (64 keys of K and of V,
// 16 KB) go global -> registers -> one of two LDS slots, row-major: no
// transposition on the way.  The MFMA operand V^T (32 head dims x 16 keys per
// lane group) comes from the transposing LDS read of gfx950 (ds_read_tr16_b64:
// within 16 lanes, lane 4e + q names row e and four consecutive columns
// 4q..4q+3 of a 4 x 16 block, and lane i receives column i of the four rows).
// K and V tiles permute the 16-byte chunks of a row by an XOR with the
// bit-reversed row-pair index, so a K fragment read (16 rows at one chunk)
// and a V^T read (4 rows x 4 chunks per 32 lanes) each touch every bank group
// once.  Only registers stage the next tile, so a workgroup needs 32 KB of
// LDS and five fit on a compute unit: at MAR-L sizes every (image, head) of a
// call is resident at once, each with one tile in flight.
namespace strm {

constexpr int kSlotBytes = 16384;  // 64 keys x 64 dims x 2 bytes, K then V

// Chunk permutation of row r: the row-pair index (r >> 1) & 7, bit-reversed.
__device__ __forceinline__ int swz(int r) {
  const int x = (r >> 1) & 7;
  return ((x & 1) << 2) | (x & 2) | (x >> 2);
}

typedef short s16x4 __attribute__((ext_vector_type(4)));

// Transposing read of four consecutive keys for this lane's head dim (see above).
__device__ __forceinline__ s16x4 read_tr(const unsigned char *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (s16x4 __attribute__((address_space(3))) *)(
          (__attribute__((address_space(3))) unsigned char *)(uintptr_t)p));
}

// One 64-key tile of the online softmax for this wavefront's 32 queries
// (lane -> query lane & 31), in the log2 domain, as attn_tile does for the
// transposed-V layouts: S^T = K Q^T, running max over the raw logits, the
// scale folded into the exponent, O^T += V^T P^T.
__device__ __forceinline__ void tile(const unsigned char *slot, const bf16x8 (&qf)[4],
                                     f32x16 (&acc)[2], float &m_run, float &l_run, float sl2,
                                     int lane) {
  const unsigned char *kt = slot, *vt = slot + 8192;
  f32x16 s[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    s[kb] = f32x16{};
    const int row = kb * 32 + (lane & 31);
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const int c = st * 2 + (lane >> 5);
      const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(kt + row * 128 + ((c ^ swz(row)) << 4));
      s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[st], s[kb], 0, 0, 0);
    }
  }
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m_new = fmaxf(m_run, mx * sl2);
  const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
  float psum = 0.f;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float p = __builtin_amdgcn_exp2f(fmaf(s[kb][r], sl2, -m_new));
      s[kb][r] = p;
      psum += p;
    }
  l_run = l_run * alpha + psum;
  m_run = m_new;
  acc[0] *= alpha;
  acc[1] *= alpha;

  // V^T operand rows: lane group g = lane / 16 reads rows kbase + e (e = its
  // source lane's (lane & 15) / 4) at head dims d0 + 4 (lane & 3) .. + 3
  const int g = lane >> 4, e = (lane & 15) >> 2, q = lane & 3;
  const int hf = lane >> 5;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      // P^T: lane half hf holds keys 16u + 4hf + 0..3 and 16u + 8 + 4hf + 0..3
      // of the 32-key block in s[kb][8u .. 8u + 7]
      bf16x8 pb;
#pragma unroll
      for (int j = 0; j < 8; ++j) pb[j] = (bf16)s[kb][8 * u + j];
#pragma unroll
      for (int db = 0; db < 2; ++db) {
        const int c = db * 4 + (g & 1) * 2 + (q >> 1);  // logical 16-byte chunk
        s16x4 lo, hi;
        {
          const int row = kb * 32 + u * 16 + 4 * hf + e;
          lo = read_tr(vt + row * 128 + ((c ^ swz(row)) << 4) + (q & 1) * 8);
        }
        {
          const int row = kb * 32 + u * 16 + 8 + 4 * hf + e;
          hi = read_tr(vt + row * 128 + ((c ^ swz(row)) << 4) + (q & 1) * 8);
        }
        const s16x4 v8[2] = {lo, hi};
        const bf16x8 va = *reinterpret_cast<const bf16x8 *>(v8);
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, acc[db], 0, 0, 0);
      }
    }
}

}  // namespace strm

// SCORES (the selection layer, Section 4.2): the workgroup of query chunk 0,
// which holds the image's generating rows (its first n_gen[b] <= 16 QB rows),
// then writes the attention mass each key receives from them,
// a.scores[b][h][j].  Its wavefronts put the final row maximum and
// normaliser of those rows in LDS and stream the K tiles once more; wavefront
// w takes key block w % 2 of each tile for generating block w / 2: S = Q K^T
// (one lane per key), the probabilities with the final statistics, summed
// over the block's rows; the blocks' sums are added in block order.
template <int QB, bool SCORES = false>
__global__ __launch_bounds__(QB * 64) void attn_reg_kernel(AttnArgs a, int chunks) {
  using namespace strm;
  constexpr int NT = QB * 64;
  constexpr int CPL = 1024 / NT;  // 16-byte chunks per lane per tile (K and V)
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * kSlotBytes];

  const int id = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = id / chunks, chunk = id - bh * chunks;
  const int b = bh / a.n_heads, h = bh - b * a.n_heads;
  const int r0 = a.a_off ? a.a_off[b] : b * a.a_max;
  const int na = a.a_off ? a.a_off[b + 1] - r0 : a.a_max;
  const int q0 = chunk * QB * 32;
  if (q0 >= na) return;  // uniform over the workgroup

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int N = a.n_tokens, D = a.d_model, nt = N / TK;
  const bf16 *kg = static_cast<const bf16 *>(a.k_cache) + (size_t)bh * N * 64;
  const bf16 *vg = static_cast<const bf16 *>(a.v_cache) + (size_t)bh * N * 64;

  const int qi = q0 + wave * 32 + (lane & 31);
  const bf16 *qrow = static_cast<const bf16 *>(a.q) + (size_t)(r0 + min(qi, na - 1)) * D + h * 64;
  bf16x8 qf[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
    qf[s] = *reinterpret_cast<const bf16x8 *>(qrow + s * 16 + (lane >> 5) * 8);

  // Chunk j of a tile (j = i * NT + tid): matrix j / 512 (K, V), row (j % 512)
  // / 8, logical chunk j % 8; coalesced in global memory, permuted in LDS.
  // Every load is unconditional (a tile index past the last repeats the last
  // tile, which the L2 still holds), so the waits the compiler places count
  // exactly the loads issued after the ones a store needs.
  u32x4 rt[CPL];
  auto gload = [&](u32x4 (&r)[CPL], int t) {
    const size_t off = (size_t)min(t, nt - 1) * TK * 64;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int j = i * NT + tid;
      r[i] = *reinterpret_cast<const u32x4 *>((j < 512 ? kg : vg) + off + (j & 511) * 8);
    }
  };
  auto sstore = [&](const u32x4 (&r)[CPL], int buf) {
    unsigned char *slot = smem + buf * kSlotBytes;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int j = i * NT + tid;
      const int row = (j & 511) >> 3, c = j & 7;
      *reinterpret_cast<u32x4 *>(slot + (j >> 9) * 8192 + row * 128 + ((c ^ swz(row)) << 4)) = r[i];
    }
  };

  const float sl2 = 1.4426950408889634f / 8.0f;  // log2(e) / sqrt(64)
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 acc[2] = {f32x16{}, f32x16{}};
  gload(rt, 0);
  sstore(rt, 0);
  __syncthreads();
  // Tile t is in LDS slot t & 1 and the registers are free again: they take
  // tile t + 1 while tile t computes, then it goes into the other slot.  The
  // loop is unrolled by two so that each step's slot is a constant (its LDS
  // offsets fold into the reads' immediates).  The scheduling barriers keep
  // the stores of the next tile (and the waits for its loads) behind the
  // whole tile step, which would otherwise start them, and wait, in the
  // middle of it.
  // A wavefront whose 32 queries all lie past the active set (the last query
  // chunk of a long sequence) keeps loading, storing and meeting the
  // barriers but skips the tile step, leaving its SIMD to the others.
  const bool live = q0 + wave * 32 < na;  // uniform over the wavefront
  auto step = [&](int t, auto slot) {
    constexpr int SL = decltype(slot)::value;
    gload(rt, t + 1);
    __builtin_amdgcn_sched_barrier(0);
    if (live) tile(smem + SL * kSlotBytes, qf, acc, m_run, l_run, sl2, lane);
    __builtin_amdgcn_sched_barrier(0);
    sstore(rt, SL ^ 1);
    __syncthreads();
  };
  int t = 0;
  for (; t + 2 <= nt; t += 2) {
    step(t, std::integral_constant<int, 0>{});
    step(t + 1, std::integral_constant<int, 1>{});
  }
  if (t < nt) step(t, std::integral_constant<int, 0>{});

  const float inv = 1.0f / (l_run + __shfl_xor(l_run, 32, 64));
  if (qi < na) {
    bf16 *orow = static_cast<bf16 *>(a.o) + (size_t)(r0 + qi) * D + h * 64;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int dh0 = db * 32 + gq * 8 + (lane >> 5) * 4;
        bf16x4 pk = {(bf16)(acc[db][4 * gq + 0] * inv), (bf16)(acc[db][4 * gq + 1] * inv),
                     (bf16)(acc[db][4 * gq + 2] * inv), (bf16)(acc[db][4 * gq + 3] * inv)};
        *reinterpret_cast<bf16x4 *>(orow + dh0) = pk;
      }
  }
  if constexpr (SCORES) {
    if (chunk != 0) return;  // uniform over the workgroup
    constexpr int CPK = 512 / NT;  // K chunks per lane per tile
    const int n_gen = a.n_gen[b];
    const int gb_n = (n_gen + 31) / 32;
    // LDS: K tiles in the K halves of the two slots; the blocks' per-key sums
    // in slot 0's V half; the statistics in slot 1's V half
    float *part = reinterpret_cast<float *>(smem + 8192);
    float *st_mx = reinterpret_cast<float *>(smem + kSlotBytes + 8192);
    float *st_iv = st_mx + QB * 32;
    // (the main loop ended on a barrier: no wavefront reads the slots again)
    if (lane < 32) {
      const int row = wave * 32 + lane;            // query qi of this lane
      st_mx[row] = qi < n_gen ? m_run : INFINITY;  // rows past n_gen: probability 0
      st_iv[row] = qi < n_gen ? inv : 0.f;
    }
    const int kb = wave & 1, gb = wave >> 1, hf = lane >> 5;
    const bool active = gb < gb_n;
    bf16x8 qg[4];
    {
      const int row = r0 + min(gb * 32 + (lane & 31), na - 1);
      const bf16 *qr = static_cast<const bf16 *>(a.q) + (size_t)row * D + h * 64;
#pragma unroll
      for (int s2 = 0; s2 < 4; ++s2)
        qg[s2] = *reinterpret_cast<const bf16x8 *>(qr + s2 * 16 + hf * 8);
    }
    u32x4 rk[CPK];
    auto kload = [&](int tk) {
      const size_t off = (size_t)min(tk, nt - 1) * TK * 64;
#pragma unroll
      for (int i = 0; i < CPK; ++i)
        rk[i] = *reinterpret_cast<const u32x4 *>(kg + off + (i * NT + tid) * 8);
    };
    auto kstore = [&](int buf) {
      unsigned char *slot = smem + buf * kSlotBytes;
#pragma unroll
      for (int i = 0; i < CPK; ++i) {
        const int j = i * NT + tid, row = j >> 3, c = j & 7;
        *reinterpret_cast<u32x4 *>(slot + row * 128 + ((c ^ swz(row)) << 4)) = rk[i];
      }
    };
    __syncthreads();  // the statistics are in LDS
    f32x4 mx[4], iv[4];  // rows gb*32 + 8 g + 4 hf + 0..3 of the accumulator
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int r = min(gb, QB - 1) * 32 + 8 * g + 4 * hf;
      mx[g] = *reinterpret_cast<const f32x4 *>(st_mx + r);
      iv[g] = *reinterpret_cast<const f32x4 *>(st_iv + r);
    }
    kload(0);
    kstore(0);
    __syncthreads();
    for (int tk = 0; tk < nt; ++tk) {
      kload(tk + 1);
      __builtin_amdgcn_sched_barrier(0);
      if (active) {
        const unsigned char *kt = smem + (tk & 1) * kSlotBytes;
        const int row = kb * 32 + (lane & 31);
        f32x16 sc = f32x16{};
#pragma unroll
        for (int st = 0; st < 4; ++st) {
          const int c = st * 2 + hf;
          const bf16x8 ka =
              *reinterpret_cast<const bf16x8 *>(kt + row * 128 + ((c ^ swz(row)) << 4));
          sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qg[st], ka, sc, 0, 0, 0);
        }
        float p = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r)
          p += __builtin_amdgcn_exp2f(fmaf(sc[r], sl2, -mx[r >> 2][r & 3])) * iv[r >> 2][r & 3];
        p += __shfl_xor(p, 32, 64);
        if (lane < 32) part[gb * 64 + kb * 32 + lane] = p;
      }
      __syncthreads();
      if (wave == 0) {
        float tot = 0.f;
        for (int g2 = 0; g2 < gb_n; ++g2) tot += part[g2 * 64 + lane];
        a.scores[(size_t)bh * N + tk * TK + lane] = tot;
      }
      __builtin_amdgcn_sched_barrier(0);
      kstore((tk + 1) & 1);
      __syncthreads();
    }
  }
}

// Every query of an image in one workgroup and every key resident in LDS
// (layers where all N <= NTL * 64 tokens are active): one workgroup per
// (image, head); wavefront w owns the NQB 32-query blocks w, w + NW, ...  All
// K/V tiles are loaded at once (registers, then LDS: one memory latency per
// workgroup instead of one per tile) and read once per (image, head), after
// which each wavefront runs the online softmax over the resident tiles with
// no further loads or barriers.  With SWZ (head width 64) the tiles take
// 80 KB, so two workgroups share a CU and one's loads overlap the other's
// arithmetic.
//
// SCORES (the selection layer, Section 4.2): the kernel also writes the
// attention mass each key receives from the image's generating rows (its
// first n_gen[b] active rows), a.scores[b][h][j] = sum over those rows i of
// softmax_j(q_i . k_j / sqrt(d_h)), from the K tiles it holds.  Each
// wavefront keeps the final row maximum and normaliser of its generating
// rows; once every wavefront is done with the V tiles, those go to LDS in
// their place, and the wavefronts split the key tiles: for each key, S = Q
// K^T over the generating rows (one lane per key), the probabilities with
// the final statistics, summed over the rows in a fixed order.
template <int DH, int NW, int NTL, int NQB, bool SWZ, bool SCORES = false>
__global__ __launch_bounds__(NW * 64) void attn_resident_kernel(AttnArgs a) {
  constexpr int NT = NW * 64;
  constexpr int ODB = (DH + 31) / 32;
  constexpr int DHV = ODB * 32;
  constexpr int KT = SWZ ? TK * 64 : TK * (DH + 8);     // elements per K tile
  constexpr int VT = SWZ ? DHV * 64 : DHV * (TK + 8);   // elements per V^T tile
  constexpr int CPR = DH / 8;
  constexpr int TCH = TK * CPR;
  constexpr int LPT = (TCH + NT - 1) / NT;
  constexpr int VPCH = TCH / 2;
  constexpr int LPV = (VPCH + NT - 1) / NT;
  constexpr int QS = DH / 16;
  __shared__ __attribute__((aligned(16))) bf16 Ks[NTL][KT];
  __shared__ __attribute__((aligned(16))) bf16 Vt[NTL][VT];

  const int bh = xcd_remap(blockIdx.x, gridDim.x);
  const int b = bh / a.n_heads, h = bh - b * a.n_heads;
  const int r0 = a.a_off ? a.a_off[b] : b * a.a_max;
  const int na = a.a_off ? a.a_off[b + 1] - r0 : a.a_max;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int N = a.n_tokens, D = a.d_model;
  const int ntiles = (N + TK - 1) / TK;  // <= NTL (host-checked)
  const bf16 *kg = static_cast<const bf16 *>(a.k_cache) + (size_t)(b * a.n_heads + h) * N * DH;
  const bf16 *vg = static_cast<const bf16 *>(a.v_cache) + (size_t)(b * a.n_heads + h) * N * DH;

  if constexpr (DHV > DH) {  // V^T rows past DH (padding to a multiple of 32) hold zeros
    for (int i = tid; i < NTL * (DHV - DH) * (TK + 8); i += NT) {
      const int t = i / ((DHV - DH) * (TK + 8)), rem = i % ((DHV - DH) * (TK + 8));
      Vt[t][DH * (TK + 8) + rem] = (bf16)0.0f;
    }
  }
  // this wavefront's queries of every block it computes, issued first so
  // that their latency hides behind the K/V loads instead of stalling the
  // start of each block
  bf16x8 qall[NQB][QS];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const int wq0 = (qb * NW + wave) * 32;
    if (wq0 < na) {
      const int qi = wq0 + (lane & 31);
      const bf16 *qrow =
          static_cast<const bf16 *>(a.q) + (size_t)(r0 + min(qi, na - 1)) * D + h * DH;
#pragma unroll
      for (int st = 0; st < QS; ++st)
        qall[qb][st] = *reinterpret_cast<const bf16x8 *>(qrow + st * 16 + (lane >> 5) * 8);
    }
  }
  // all tiles' loads, then all LDS writes
  u32x4 rk[NTL][LPT], rv0[NTL][LPV], rv1[NTL][LPV];
#pragma unroll
  for (int t = 0; t < NTL; ++t) {
    if (t >= ntiles) break;
    const int t0 = t * TK;
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      const int c = i * NT + tid;
      if (c < TCH) {
        const int key = min(t0 + c / CPR, N - 1), d = (c % CPR) * 8;
        rk[t][i] = *reinterpret_cast<const u32x4 *>(kg + (size_t)key * DH + d);
      }
    }
#pragma unroll
    for (int i = 0; i < LPV; ++i) {
      const int c = i * NT + tid;
      if (c < VPCH) {
        const int kp = c / CPR, d = (c % CPR) * 8;
        const int k0 = min(t0 + 2 * kp, N - 1), k1 = min(t0 + 2 * kp + 1, N - 1);
        rv0[t][i] = *reinterpret_cast<const u32x4 *>(vg + (size_t)k0 * DH + d);
        rv1[t][i] = *reinterpret_cast<const u32x4 *>(vg + (size_t)k1 * DH + d);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < NTL; ++t) {
    if (t >= ntiles) break;
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      const int c = i * NT + tid;
      if (c < TCH) {
        const int key = c / CPR, d = (c % CPR) * 8;
        *reinterpret_cast<u32x4 *>(&Ks[t][k_off<DH, SWZ>(key, d)]) = rk[t][i];
      }
    }
#pragma unroll
    for (int i = 0; i < LPV; ++i) {
      const int c = i * NT + tid;
      if (c < VPCH) {
        const int kp = c / CPR, d = (c % CPR) * 8;
        const int pos = ((2 * kp) & ~15) | vperm16((2 * kp) & 15);  // even: a 32-bit pair
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const unsigned w0 = rv0[t][i][e >> 1], w1 = rv1[t][i][e >> 1];
          const unsigned lo = (e & 1) ? (w0 >> 16) : (w0 & 0xFFFFu);
          const unsigned hi = (e & 1) ? (w1 & 0xFFFF0000u) : (w1 << 16);
          *reinterpret_cast<unsigned *>(&Vt[t][vt_off<DH, SWZ>(d + e, pos)]) = lo | hi;
        }
      }
    }
  }
  __syncthreads();

  const float sl2 = 1.4426950408889634f / sqrtf((float)DH);
  const int n_gen = SCORES ? a.n_gen[b] : 0;
  // final statistics of this wavefront's blocks (generating rows only)
  float st_m[NQB], st_inv[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    st_m[qb] = INFINITY;
    st_inv[qb] = 0.f;
  }
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const int wq0 = (qb * NW + wave) * 32;
    if (wq0 >= na) break;  // uniform over the wavefront; no barrier inside the loop
    const int qi = wq0 + (lane & 31);
    const bf16x8 (&qf)[QS] = qall[qb];
    float m_run = -INFINITY, l_run = 0.f;
    f32x16 acc[ODB];
#pragma unroll
    for (int d = 0; d < ODB; ++d) acc[d] = f32x16{};
    for (int t = 0; t < N / TK; ++t)
      attn_tile<DH, SWZ>(Ks[t], Vt[t], qf, acc, m_run, l_run, t * TK, N, sl2, lane);
    if (N % TK)
      attn_tile<DH, SWZ, true>(Ks[N / TK], Vt[N / TK], qf, acc, m_run, l_run, (N / TK) * TK, N,
                               sl2, lane);

    const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
    const float inv = 1.0f / l_tot;
    if (SCORES && qi < n_gen) {
      st_m[qb] = m_run;
      st_inv[qb] = inv;
    }
    if (qi < na) {
      bf16 *orow = static_cast<bf16 *>(a.o) + (size_t)(r0 + qi) * D + h * DH;
#pragma unroll
      for (int d = 0; d < ODB; ++d)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int dh0 = d * 32 + g * 8 + (lane >> 5) * 4;
          if (dh0 < DH) {
            bf16x4 pk = {(bf16)(acc[d][4 * g + 0] * inv), (bf16)(acc[d][4 * g + 1] * inv),
                         (bf16)(acc[d][4 * g + 2] * inv), (bf16)(acc[d][4 * g + 3] * inv)};
            *reinterpret_cast<bf16x4 *>(orow + dh0) = pk;
          }
        }
    }
  }
  if constexpr (SCORES) {
    // statistics of generating row i at st_mx[i], st_iv[i], in the V tiles'
    // place; rows at or past n_gen read maximum +inf and normaliser 0, so
    // their probabilities are exactly 0
    const int gb_n = (n_gen + 31) / 32;  // blocks with generating rows
    float *st_mx = reinterpret_cast<float *>(&Vt[0][0]);
    float *st_iv = st_mx + NQB * NW * 32;
    static_assert(2 * NQB * NW * 32 * 4 <= (int)sizeof(Vt), "statistics fit the V tiles");
    __syncthreads();  // every wavefront is done with the V tiles
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      const int row = (qb * NW + wave) * 32 + (lane & 31);
      if (lane < 32 && row < gb_n * 32) {
        st_mx[row] = st_m[qb];
        st_iv[row] = st_inv[qb];
      }
    }
    __syncthreads();
    const int hf = lane >> 5;
    for (int t = wave; t < ntiles; t += NW) {
      float sc[2] = {0.f, 0.f};  // keys t*64 + kb*32 + (lane & 31), this lane's half of the rows
      for (int gb = 0; gb < gb_n; ++gb) {
        const int qi = gb * 32 + (lane & 31);
        const bf16 *qrow =
            static_cast<const bf16 *>(a.q) + (size_t)(r0 + min(qi, na - 1)) * D + h * DH;
        bf16x8 qf[QS];
#pragma unroll
        for (int st = 0; st < QS; ++st)
          qf[st] = *reinterpret_cast<const bf16x8 *>(qrow + st * 16 + hf * 8);
        // rows of register r: gb*32 + 8 (r / 4) + 4 hf + r % 4
        f32x4 mx[4], iv[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          mx[g] = *reinterpret_cast<const f32x4 *>(st_mx + gb * 32 + 8 * g + 4 * hf);
          iv[g] = *reinterpret_cast<const f32x4 *>(st_iv + gb * 32 + 8 * g + 4 * hf);
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          f32x16 s = f32x16{};
#pragma unroll
          for (int st = 0; st < QS; ++st) {
            const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(
                &Ks[t][k_off<DH, SWZ>(kb * 32 + (lane & 31), st * 16 + hf * 8)]);
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[st], ka, s, 0, 0, 0);
          }
          float part = 0.f;
#pragma unroll
          for (int r = 0; r < 16; ++r)
            part += __builtin_amdgcn_exp2f(fmaf(s[r], sl2, -mx[r >> 2][r & 3])) * iv[r >> 2][r & 3];
          sc[kb] += part;
        }
      }
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const float tot = sc[kb] + __shfl_xor(sc[kb], 32, 64);
        const int key = t * TK + kb * 32 + (lane & 31);
        if (lane < 32 && key < N) a.scores[(size_t)bh * N + key] = tot;
      }
    }
  }
}

constexpr int RES_NTL = 5;    // keys resident: 320
constexpr int RES_QMAX = 320; // queries per workgroup

// Host choice of the resident kernel: more than 64 active queries per image
// (where the streaming kernel needs several workgroups per (image, head)), all
// of them and all keys within one workgroup's reach, one key segment.
// Query blocks per workgroup of the streaming kernel for a_max rows.
static int reg_qb(int32_t a_max) {
  return a_max <= 32 ? 1 : a_max <= 64 ? 2 : a_max <= 128 ? 4 : 8;
}

bool attn_resident(int32_t a_max, int32_t n_tokens, bool two_segments) {
  return !two_segments && a_max > 64 && a_max <= RES_QMAX && n_tokens <= RES_NTL * TK;
}

bool attn_fuses_scores(int32_t a_max, int32_t n_tokens, int32_t head_dim, int32_t gen_max) {
  if (attn_resident(a_max, n_tokens, false)) return true;
  // streaming kernel: the generating rows within query chunk 0, and one
  // (key block, generating block) pair per wavefront
  return attn_streams(head_dim, n_tokens, false) && 2 * ((gen_max + 31) / 32) <= reg_qb(a_max);
}

template <int DH, int NW, bool SEG2>
static hipError_t run_attn_mfma(const AttnArgs &a, hipStream_t s) {
  const int chunks = (a.a_max + NW * 32 - 1) / (NW * 32);
  const int grid = a.batch * a.n_heads * chunks;
  const bool aligned = a.n_tokens % TK == 0 && (!SEG2 || a.n2 % TK == 0);
  if (aligned)
    launch_kernel(attn_mfma_kernel<DH, NW, SEG2, true>, grid, NW * 64, 0, s, a, chunks);
  else
    launch_kernel(attn_mfma_kernel<DH, NW, SEG2, false>, grid, NW * 64, 0, s, a, chunks);
  return hipGetLastError();
}

// The register-staged kernel of head width 64 for one key segment of whole
// tiles (at least three).
bool attn_streams(int32_t head_dim, int32_t n_tokens, bool two_segments) {
  return head_dim == 64 && !two_segments && n_tokens % TK == 0 && n_tokens >= 3 * TK;
}

template <int QB>
static hipError_t run_attn_reg(const AttnArgs &a, hipStream_t s) {
  const int chunks = (a.a_max + QB * 32 - 1) / (QB * 32);
  const int grid = a.batch * a.n_heads * chunks;
  if (a.scores)
    launch_kernel(attn_reg_kernel<QB, true>, grid, QB * 64, 0, s, a, chunks);
  else
    launch_kernel(attn_reg_kernel<QB>, grid, QB * 64, 0, s, a, chunks);
  return hipGetLastError();
}


template <int DH, bool SEG2>
static hipError_t attn_bf16_nw(const AttnArgs &a, hipStream_t s) {
  if (attn_streams(DH, a.n_tokens, SEG2)) {
    if (a.a_max <= 32) return run_attn_reg<1>(a, s);
    if (a.a_max <= 64) return run_attn_reg<2>(a, s);
    if (a.a_max <= 128) return run_attn_reg<4>(a, s);
    return run_attn_reg<8>(a, s);  // one pass over K/V per 256 queries
  }
  if (a.a_max <= 32) return run_attn_mfma<DH, 1, SEG2>(a, s);
  if (a.a_max <= 64) return run_attn_mfma<DH, 2, SEG2>(a, s);
  return run_attn_mfma<DH, 4, SEG2>(a, s);
}

template <int DH>
static hipError_t attn_bf16_dispatch(const AttnArgs &a, hipStream_t s) {
  if (a.k2) return attn_bf16_nw<DH, true>(a, s);
  if (attn_resident(a.a_max, a.n_tokens, a.k2 != nullptr)) {
    const int grid = a.batch * a.n_heads;
    if constexpr (DH == 64) {  // 80 KB of swizzled tiles: two workgroups per CU
      if (a.scores)
        launch_kernel(attn_resident_kernel<DH, 4, RES_NTL, 3, true, true>, grid, 4 * 64, 0, s, a);
      else
        launch_kernel(attn_resident_kernel<DH, 4, RES_NTL, 3, true>, grid, 4 * 64, 0, s, a);
    } else {
      if (a.scores)
        launch_kernel(attn_resident_kernel<DH, 10, RES_NTL, 1, false, true>, grid, 10 * 64, 0, s,
                      a);
      else
        launch_kernel(attn_resident_kernel<DH, 10, RES_NTL, 1, false>, grid, 10 * 64, 0, s, a);
    }
    return hipGetLastError();
  }
  return attn_bf16_nw<DH, false>(a, s);
}

// ------------------------------------------------------------ concatenation
//
// The baseline of Appendix B: K and V of the active segment and of the cached
// segment copied into one buffer per (image, head), active rows first.  Per
// (image, head) the destination is two contiguous copies, so chunk j (16
// bytes) of the destination block comes from chunk j of the active block
// (j < na * cpr) or chunk j - na * cpr of the cached block.  Each thread moves
// CPT chunks of K and of V, all loads issued before the stores.  Grid:
// (chunks of a destination block / (256 * CPT), image * head).
constexpr int CONCAT_CPT = 4;

__global__ __launch_bounds__(256) void concat_kv_kernel(u32x4 *__restrict__ kd, u32x4 *__restrict__ vd,
                                                        const u32x4 *__restrict__ ka,
                                                        const u32x4 *__restrict__ va,
                                                        const u32x4 *__restrict__ kc,
                                                        const u32x4 *__restrict__ vc, int a_chunks,
                                                        int c_chunks) {
  const int per = a_chunks + c_chunks;
  const size_t bh = blockIdx.y;
  const int j0 = blockIdx.x * 256 * CONCAT_CPT + threadIdx.x;
  u32x4 kv[CONCAT_CPT], vv[CONCAT_CPT];
#pragma unroll
  for (int u = 0; u < CONCAT_CPT; ++u) {
    const int j = j0 + u * 256;
    if (j < per) {
      const bool act = j < a_chunks;
      const size_t src = act ? bh * a_chunks + j : bh * c_chunks + (j - a_chunks);
      kv[u] = act ? ka[src] : kc[src];
      vv[u] = act ? va[src] : vc[src];
    }
  }
#pragma unroll
  for (int u = 0; u < CONCAT_CPT; ++u) {
    const int j = j0 + u * 256;
    if (j < per) {
      kd[bh * per + j] = kv[u];
      vd[bh * per + j] = vv[u];
    }
  }
}

hipError_t launch_concat_kv(DType dt, void *k_dst, void *v_dst, const void *k_a, const void *v_a,
                            const void *k_c, const void *v_c, int32_t bh, int32_t na, int32_t nc,
                            int32_t head_dim, hipStream_t s) {
  const int es = dt == DType::BF16 ? 2 : 4;
  if ((head_dim * es) % 16 != 0 || bh > 65535) return hipErrorInvalidValue;
  const int cpr = head_dim * es / 16;
  const int per = (na + nc) * cpr;
  if (bh == 0 || per == 0) return hipSuccess;
  const dim3 grid((per + 256 * CONCAT_CPT - 1) / (256 * CONCAT_CPT), bh);
  launch_kernel(concat_kv_kernel, grid, 256, 0, s, static_cast<u32x4 *>(k_dst), static_cast<u32x4 *>(v_dst), static_cast<const u32x4 *>(k_a),
      static_cast<const u32x4 *>(v_a), static_cast<const u32x4 *>(k_c),
      static_cast<const u32x4 *>(v_c), na * cpr, nc * cpr);
  return hipGetLastError();
}

// fp32 attention: one wavefront per (active row, head).  Logits are formed
// lane-per-key, then the output lane-per-dimension; exact expf.
template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  extern __shared__ float smem[];
  float *qs = smem;          // [DH]
  float *ps = smem + DH;     // [N]
  const int gw = blockIdx.x;
  const int row = gw / a.n_heads, h = gw - row * a.n_heads;
  const int lane = threadIdx.x;
  const int N = a.n_tokens, D = a.d_model;
  const RowMap m = a.map[row];
  const size_t head_base = (size_t)(m.b * a.n_heads + h) * N * DH;
  const float *kg = static_cast<const float *>(a.k_cache) + head_base;
  const float *vg = static_cast<const float *>(a.v_cache) + head_base;
  const float *qg = static_cast<const float *>(a.q) + (size_t)row * D + h * DH;
  for (int d = lane; d < DH; d += 64) qs[d] = qg[d];
  __syncthreads();
  const float scale = 1.0f / sqrtf((float)DH);
  float mx = -INFINITY;
  for (int j = lane; j < N; j += 64) {
    const float *kr = kg + (size_t)j * DH;
    float acc = 0.f;
#pragma unroll 8
    for (int d = 0; d < DH; ++d) acc = fmaf(qs[d], kr[d], acc);
    acc *= scale;
    ps[j] = acc;
    mx = fmaxf(mx, acc);
  }
  mx = wave_max(mx);
  float sum = 0.f;
  for (int j = lane; j < N; j += 64) {
    const float e = expf(ps[j] - mx);
    ps[j] = e;
    sum += e;
  }
  sum = wave_sum(sum);
  __syncthreads();
  const float inv = 1.0f / sum;
  float *og = static_cast<float *>(a.o) + (size_t)row * D + h * DH;
  for (int d = lane; d < DH; d += 64) {
    float acc = 0.f;
    for (int j = 0; j < N; ++j) acc = fmaf(ps[j], vg[(size_t)j * DH + d], acc);
    og[d] = acc * inv;
  }
}

template <int DH>
static hipError_t attn_f32_dispatch(const AttnArgs &a, hipStream_t s) {
  const size_t lds = (size_t)(DH + a.n_tokens) * sizeof(float);
  launch_kernel(attn_f32_kernel<DH>, a.a_total * a.n_heads, 64, lds, s, a);
  return hipGetLastError();
}

hipError_t launch_attention(DType dt, const AttnArgs &a, hipStream_t s) {
  if (a.a_total == 0) return hipSuccess;
  if (a.k2 && dt != DType::BF16) return hipErrorInvalidValue;
  if (dt == DType::BF16) {
    if (a.head_dim == 64) return attn_bf16_dispatch<64>(a, s);
    if (a.head_dim == 80) return attn_bf16_dispatch<80>(a, s);
  } else {
    if (a.head_dim == 64) return attn_f32_dispatch<64>(a, s);
    if (a.head_dim == 80) return attn_f32_dispatch<80>(a, s);
  }
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------- score pass
//
// scores[b][h][j] = sum over the generating rows i (the first n_gen[b] active
// rows of image b) of softmax_j(q_i . k_j / sqrt(d_h)) -- the post-softmax
// attention mass each key receives, one head at a time, with each row's
// maximum and normaliser taken over all N keys.  One workgroup per
// (image, head); thread t owns keys t, t+256, ...; generating rows are taken
// GQ at a time and their logits staged in LDS.  All sums run in a fixed
// order, so the result is deterministic.

constexpr int SC_THREADS = 256;
constexpr int SC_MAX_KPT = 16;  // keys per thread: n_tokens <= 4096

__device__ __forceinline__ float block_reduce(float v, bool is_max, float *red) {
  v = is_max ? wave_max(v) : wave_sum(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < SC_THREADS / 64; ++i) r = is_max ? fmaxf(r, red[i]) : r + red[i];
  return r;
}

// Eight consecutive elements as float (16- or 32-byte aligned source).
__device__ __forceinline__ void load8(const bf16 *p, float (&out)[8]) {
  const bf16x8 v = *reinterpret_cast<const bf16x8 *>(p);
#pragma unroll
  for (int e = 0; e < 8; ++e) out[e] = (float)v[e];
}
__device__ __forceinline__ void load8(const float *p, float (&out)[8]) {
  const f32x4 a = *reinterpret_cast<const f32x4 *>(p);
  const f32x4 b = *reinterpret_cast<const f32x4 *>(p + 4);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    out[e] = a[e];
    out[e + 4] = b[e];
  }
}

template <typename T, int DH>
__global__ __launch_bounds__(SC_THREADS) void attn_scores_kernel(AttnArgs a,
                                                                 const int32_t *__restrict__ n_gen,
                                                                 float *__restrict__ scores,
                                                                 int gq) {
  extern __shared__ float smem[];
  const int N = a.n_tokens, D = a.d_model;
  float *qs = smem;                 // [gq][DH]
  float *ss = smem + gq * DH;       // [gq][N]
  float *red = ss + gq * N;         // [4]
  const int b = blockIdx.x / a.n_heads, h = blockIdx.x - b * a.n_heads;
  const int tid = threadIdx.x;
  const int g = n_gen[b], r0 = a.a_off[b];
  const size_t head_base = (size_t)(b * a.n_heads + h) * N * DH;
  const T *kg = static_cast<const T *>(a.k_cache) + head_base;
  const T *qg = static_cast<const T *>(a.q);
  const float scale = 1.0f / sqrtf((float)DH);

  float acc[SC_MAX_KPT];
#pragma unroll
  for (int i = 0; i < SC_MAX_KPT; ++i) acc[i] = 0.f;

  for (int g0 = 0; g0 < g; g0 += gq) {
    const int nq = min(gq, g - g0);
    for (int i = tid; i < nq * DH; i += SC_THREADS) {
      const int qq = i / DH, d = i - qq * DH;
      qs[i] = to_f32(qg[(size_t)(r0 + g0 + qq) * D + h * DH + d]);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < SC_MAX_KPT; ++i) {
      const int j = tid + SC_THREADS * i;
      if (j >= N) break;
      float dot[8];
#pragma unroll
      for (int qq = 0; qq < 8; ++qq) dot[qq] = 0.f;
      const T *kr = kg + (size_t)j * DH;
#pragma unroll 2
      for (int d0 = 0; d0 < DH; d0 += 8) {
        float kv[8];
        load8(kr + d0, kv);
#pragma unroll
        for (int e = 0; e < 8; ++e)
#pragma unroll
          for (int qq = 0; qq < 8; ++qq)
            if (qq < nq) dot[qq] = fmaf(qs[qq * DH + d0 + e], kv[e], dot[qq]);
      }
#pragma unroll
      for (int qq = 0; qq < 8; ++qq)
        if (qq < nq) ss[qq * N + j] = dot[qq] * scale;
    }
    __syncthreads();
    for (int qq = 0; qq < nq; ++qq) {
      float mx = -INFINITY;
      for (int j = tid; j < N; j += SC_THREADS) mx = fmaxf(mx, ss[qq * N + j]);
      mx = block_reduce(mx, true, red);
      float sm = 0.f;
      for (int j = tid; j < N; j += SC_THREADS) sm += expf(ss[qq * N + j] - mx);
      sm = block_reduce(sm, false, red);
      const float inv = 1.0f / sm;
#pragma unroll
      for (int i = 0; i < SC_MAX_KPT; ++i) {
        const int j = tid + SC_THREADS * i;
        if (j >= N) break;
        acc[i] += expf(ss[qq * N + j] - mx) * inv;
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < SC_MAX_KPT; ++i) {
    const int j = tid + SC_THREADS * i;
    if (j >= N) break;
    scores[(size_t)(b * a.n_heads + h) * N + j] = acc[i];
  }
}

template <typename T, int DH>
static hipError_t scores_dispatch(const AttnArgs &a, const int32_t *n_gen, float *scores,
                                  hipStream_t s) {
  int gq = 12288 / a.n_tokens;
  gq = gq < 1 ? 1 : (gq > 8 ? 8 : gq);
  const size_t lds = (size_t)(gq * DH + gq * a.n_tokens + 4) * sizeof(float);
  launch_kernel(attn_scores_kernel<T, DH>, a.batch * a.n_heads, SC_THREADS, lds, s,
                a, n_gen, scores, gq);
  return hipGetLastError();
}

hipError_t launch_attn_scores(DType dt, const AttnArgs &a, const int32_t *n_gen, int32_t gen_max,
                              float *scores, hipStream_t s) {
  (void)gen_max;
  if (a.batch == 0) return hipSuccess;
  if (a.n_tokens > SC_THREADS * SC_MAX_KPT) return hipErrorInvalidValue;
  if (dt == DType::BF16) {
    if (a.head_dim == 64) return scores_dispatch<bf16, 64>(a, n_gen, scores, s);
    if (a.head_dim == 80) return scores_dispatch<bf16, 80>(a, n_gen, scores, s);
  } else {
    if (a.head_dim == 64) return scores_dispatch<float, 64>(a, n_gen, scores, s);
    if (a.head_dim == 80) return scores_dispatch<float, 80>(a, n_gen, scores, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace marche
