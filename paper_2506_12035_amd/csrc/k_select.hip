// Refresh selection (Section 4.2): head-aggregated attention mass, top-k.
//
// One workgroup per image, one thread per token (up to 1024 threads, two
// tokens per thread beyond that).  Each thread issues the loads of every
// head's score for its tokens at once (sixteen heads per batch), sums them in
// head order and stores an order-preserving 32-bit image of the sum in LDS: a
// larger score gives a larger value, NaN ranks after every number and -0.0
// ties +0.0; for the lowest-first order the bits are inverted.  The excluded
// tokens (generating and caching tokens), loaded beside the scores, then get
// 0, below every candidate.  One wavefront selects, with every value in its
// registers: the k-th largest value T by a 32-step descent over its bits
// (each step counts the values at or above a candidate with one ballot per 64
// tokens), then the tokens in ascending order, taking every value above T
// and, among the values equal to T, the lowest token indices until k are
// taken.  That is the first k tokens in the order (score, then lower index
// first), the order of the oracle's selection.  Everything is deterministic.
#include <algorithm>

#include "device_common.h"

namespace marche {

constexpr int SEL_MAX_THREADS = 1024;
constexpr int SEL_MAX_N = 4096;

// Order-preserving unsigned image of a float: larger float, larger key.
// NaN is placed after every number in the chosen order; -0.0 ties with +0.0.
__device__ __forceinline__ uint32_t order_bits(float f, bool lowest) {
  if (f != f) f = lowest ? INFINITY : -INFINITY;
  if (f == 0.0f) f = 0.0f;
  const uint32_t u = __float_as_uint(f);
  const uint32_t up = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  // lowest first: invert so that the smallest score gets the largest key;
  // (~up) is never 0 for a non-NaN float, so candidates stay above key 0
  return lowest ? ~up : up;
}

// KPL: keys per lane of the selecting wavefront (n_tokens <= 64 KPL).
template <int KPL>
__global__ __launch_bounds__(SEL_MAX_THREADS) void select_topk_kernel(
    const float *__restrict__ scores, int n_parts, const int32_t *__restrict__ excl_idx,
    const int32_t *__restrict__ excl_off, int n_tokens, int k, int32_t *__restrict__ out_idx,
    const int32_t *__restrict__ out_off, bool lowest) {
  __shared__ uint32_t key[64 * KPL];
  const int b = blockIdx.x, tid = threadIdx.x, nt = blockDim.x;
  const float *sb = scores + (size_t)b * n_parts * n_tokens;
  const int e0 = excl_off[b], e1 = excl_off[b + 1];
  const int ex = e0 + tid < e1 ? excl_idx[e0 + tid] : -1;  // in flight with the scores

  // head sums in head order; tokens tid and tid + nt together, sixteen heads'
  // loads of both in flight at a time.  The loads are unconditional (a head
  // or token past the end repeats the last one) and the sums skip them by
  // adding +0, which leaves every sum unchanged (it starts at +0, so it is
  // never -0).
  for (int j0 = tid; j0 < n_tokens; j0 += 2 * nt) {
    const int j1 = j0 + nt;
    const bool has1 = j1 < n_tokens;
    const int j1c = has1 ? j1 : j0;
    float s0 = 0.f, s1 = 0.f;
    for (int p0 = 0; p0 < n_parts; p0 += 16) {
      float v0[16], v1[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const size_t row = (size_t)min(p0 + u, n_parts - 1) * n_tokens;
        v0[u] = sb[row + j0];
        v1[u] = sb[row + j1c];
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const bool ok = p0 + u < n_parts;
        s0 += ok ? v0[u] : 0.f;
        s1 += ok ? v1[u] : 0.f;
      }
    }
    key[j0] = order_bits(s0, lowest);
    if (has1) key[j1] = order_bits(s1, lowest);
  }
  __syncthreads();
  if (ex >= 0 && ex < n_tokens) key[ex] = 0u;
  for (int e = e0 + nt + tid; e < e1; e += nt) {
    const int j = excl_idx[e];
    if (j >= 0 && j < n_tokens) key[j] = 0u;
  }
  __syncthreads();
  if (tid >= 64) return;  // the selection is one wavefront's
  const int lane = tid;
  uint32_t kr[KPL];  // token 64 i + lane; 0 past the last token
#pragma unroll
  for (int i = 0; i < KPL; ++i) kr[i] = 64 * i + lane < n_tokens ? key[64 * i + lane] : 0u;

  // number of tokens whose value is at least v (v >= 1: candidates only;
  // the zero keys past the last token never count, so no guard is needed)
  auto count_ge = [&](uint32_t v) {
    int c = 0;
#pragma unroll
    for (int i = 0; i < KPL; ++i) c += __popcll(__ballot(kr[i] >= v));
    return c;
  };
  // T: the largest value with at least k tokens at or above it (the k-th
  // largest value); with k or fewer candidates every candidate is taken
  uint32_t t_val = 1u;
  if (count_ge(1u) > k) {
    t_val = 0u;
    for (int bit = 31; bit >= 0; --bit) {
      const uint32_t cand = t_val | (1u << bit);
      if (count_ge(cand) >= k) t_val = cand;
    }
  }
  const int ties = k - (t_val == 0xFFFFFFFFu ? 0 : count_ge(t_val + 1u));  // values equal to T taken

  // ascending compaction
  int32_t *ob = out_idx + out_off[b];
  int base = 0, tie_base = 0;
  const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
  for (int i = 0; i < KPL; ++i) {
    const uint32_t v = kr[i];
    const unsigned long long tie = __ballot(v != 0u && v == t_val);
    const int tie_rank = tie_base + __popcll(tie & below);
    const bool take = v != 0u && (v > t_val || (v == t_val && tie_rank < ties));
    const unsigned long long sel = __ballot(take);
    if (take) ob[base + __popcll(sel & below)] = 64 * i + lane;
    base += __popcll(sel);
    tie_base += __popcll(tie);
  }
  // fewer than k candidates: pad with -1
  for (int i = base + lane; i < k; i += 64) ob[i] = -1;
}

hipError_t launch_select_topk(const float *scores, int32_t n_parts, const int32_t *excl_idx,
                              const int32_t *excl_off, int32_t batch, int32_t n_tokens, int32_t k,
                              int32_t *out_idx, const int32_t *out_off, bool lowest,
                              hipStream_t s) {
  if (batch == 0 || k == 0) return hipSuccess;
  if (n_tokens > SEL_MAX_N) return hipErrorInvalidValue;
  // one thread per token up to 1024 (whole wavefronts), two per thread beyond
  const int threads = std::min(SEL_MAX_THREADS, (n_tokens + 63) / 64 * 64);
  // the selecting wavefront's key registers: the fewest of these that hold
  // n_tokens (every step of the selection counts all of them)
  auto launch = [&](auto kernel) {
    launch_kernel(kernel, batch, threads, 0, s, scores, n_parts, excl_idx, excl_off, n_tokens, k,
                  out_idx, out_off, lowest);
  };
  if (n_tokens <= 64 * 5) launch(select_topk_kernel<5>);
  else if (n_tokens <= 64 * 8) launch(select_topk_kernel<8>);
  else if (n_tokens <= 64 * 17) launch(select_topk_kernel<17>);
  else if (n_tokens <= 64 * 32) launch(select_topk_kernel<32>);
  else launch(select_topk_kernel<64>);
  return hipGetLastError();
}

}  // namespace marche
