// Refresh selection (Section 4.2): head-aggregated attention mass, top-k.
//
// One workgroup per image.  Its four wavefronts sum each token's score over
// the heads (in head order) and store an order-preserving 32-bit image of it
// in LDS: a larger score gives a larger value, NaN ranks after every number
// and -0.0 ties +0.0; for the lowest-first order the bits are inverted.
// Excluded tokens (generating and caching tokens) get 0, below every
// candidate.  One wavefront then selects, with every value in its registers:
// the k-th largest value T by a 32-step descent over its bits (each step
// counts the values at or above a candidate with one ballot per 64 tokens),
// then the tokens in ascending order, taking every value above T and, among
// the values equal to T, the lowest token indices until k are taken.  That
// is the first k tokens in the order (score, then lower index first), the
// order of the oracle's selection.  Everything is deterministic.
#include "device_common.h"

namespace marche {

constexpr int SEL_THREADS = 256;
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
__global__ __launch_bounds__(SEL_THREADS) void select_topk_kernel(
    const float *__restrict__ scores, int n_parts, const int32_t *__restrict__ excl_idx,
    const int32_t *__restrict__ excl_off, int n_tokens, int k, int32_t *__restrict__ out_idx,
    const int32_t *__restrict__ out_off, bool lowest) {
  __shared__ uint32_t key[64 * KPL];
  const int b = blockIdx.x, tid = threadIdx.x;
  const float *sb = scores + (size_t)b * n_parts * n_tokens;

  // head sums in head order; eight heads' loads in flight at a time
  for (int j = tid; j < n_tokens; j += SEL_THREADS) {
    float s = 0.f;
    for (int p0 = 0; p0 < n_parts; p0 += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        v[u] = p0 + u < n_parts ? sb[(size_t)(p0 + u) * n_tokens + j] : 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (p0 + u < n_parts) s += v[u];
    }
    key[j] = order_bits(s, lowest);
  }
  __syncthreads();
  for (int e = excl_off[b] + tid; e < excl_off[b + 1]; e += SEL_THREADS) {
    const int j = excl_idx[e];
    if (j >= 0 && j < n_tokens) key[j] = 0u;
  }
  __syncthreads();
  if (tid >= 64) return;  // the selection is one wavefront's
  const int lane = tid;
  uint32_t kr[KPL];  // token 64 i + lane; 0 past the last token
#pragma unroll
  for (int i = 0; i < KPL; ++i) kr[i] = 64 * i + lane < n_tokens ? key[64 * i + lane] : 0u;

  // number of tokens whose value is at least v (v >= 1: candidates only)
  auto count_ge = [&](uint32_t v) {
    int c = 0;
#pragma unroll
    for (int i = 0; i < KPL; ++i)
      if (64 * i < n_tokens) c += __popcll(__ballot(kr[i] >= v));
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
    if (64 * i >= n_tokens) break;
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
  if (n_tokens <= 512)
    launch_kernel(select_topk_kernel<8>, batch, SEL_THREADS, 0, s, scores, n_parts, excl_idx, excl_off,
                                                        n_tokens, k, out_idx, out_off, lowest);
  else if (n_tokens <= 2048)
    launch_kernel(select_topk_kernel<32>, batch, SEL_THREADS, 0, s, scores, n_parts, excl_idx, excl_off,
                                                         n_tokens, k, out_idx, out_off, lowest);
  else
    launch_kernel(select_topk_kernel<64>, batch, SEL_THREADS, 0, s, scores, n_parts, excl_idx, excl_off,
                                                         n_tokens, k, out_idx, out_off, lowest);
  return hipGetLastError();
}

}  // namespace marche
