// Refresh selection (Section 4.2): head-aggregated attention mass, top-k.
//
// One workgroup per image.  Every token j gets a 64-bit key
//     (order-preserving bits of s_j) << 32  |  (0xFFFFFFFF - j)
// so that sorting keys in descending order ranks higher scores first and,
// among equal scores, lower token indices first; NaN is mapped to -inf and
// -0.0 to +0.0 before encoding.  For the lowest-first order the score bits are
// inverted (and NaN mapped to +inf).  Excluded tokens (generating and caching
// tokens) get key 0, below every candidate.  A bitonic sort in LDS orders the
// keys; the first k are flagged and written out in ascending token order with
// a block-wide prefix count.  Everything is deterministic.
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

__global__ __launch_bounds__(SEL_THREADS) void select_topk_kernel(
    const float *__restrict__ scores, int n_parts, const int32_t *__restrict__ excl_idx,
    const int32_t *__restrict__ excl_off, int n_tokens, int np2, int k,
    int32_t *__restrict__ out_idx, const int32_t *__restrict__ out_off, bool lowest) {
  extern __shared__ unsigned long long keys[];  // [np2], then int flags[n_tokens]
  int *flags = reinterpret_cast<int *>(keys + np2);
  __shared__ int part[SEL_THREADS];
  const int b = blockIdx.x, tid = threadIdx.x;
  const float *sb = scores + (size_t)b * n_parts * n_tokens;

  for (int j = tid; j < np2; j += SEL_THREADS) {
    unsigned long long key = 0ull;
    if (j < n_tokens) {
      float s = 0.f;
      for (int p = 0; p < n_parts; ++p) s += sb[(size_t)p * n_tokens + j];
      key = ((unsigned long long)order_bits(s, lowest) << 32) | (0xFFFFFFFFu - (uint32_t)j);
      flags[j] = 0;
    }
    keys[j] = key;
  }
  __syncthreads();
  for (int e = excl_off[b] + tid; e < excl_off[b + 1]; e += SEL_THREADS) {
    const int j = excl_idx[e];
    if (j >= 0 && j < n_tokens) keys[j] = 0ull;
  }
  __syncthreads();

  // bitonic sort, descending
  for (int size = 2; size <= np2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < (np2 >> 1); i += SEL_THREADS) {
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool desc = (lo & size) == 0;
        const unsigned long long x = keys[lo], y = keys[hi];
        if ((x < y) == desc) {
          keys[lo] = y;
          keys[hi] = x;
        }
      }
      __syncthreads();
    }
  }

  for (int i = tid; i < k && i < np2; i += SEL_THREADS) {
    const unsigned long long key = keys[i];
    if (key != 0ull) flags[0xFFFFFFFFu - (uint32_t)(key & 0xFFFFFFFFull)] = 1;
  }
  __syncthreads();

  // ascending compaction: thread t owns a contiguous run of tokens
  const int per = (n_tokens + SEL_THREADS - 1) / SEL_THREADS;
  const int j0 = tid * per, j1 = min(j0 + per, n_tokens);
  int cnt = 0;
  for (int j = j0; j < j1; ++j) cnt += flags[j];
  part[tid] = cnt;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int t = 0; t < SEL_THREADS; ++t) {
      const int c = part[t];
      part[t] = run;
      run += c;
    }
  }
  __syncthreads();
  int pos = part[tid];
  int32_t *ob = out_idx + out_off[b];
  for (int j = j0; j < j1; ++j)
    if (flags[j]) ob[pos++] = j;
  // Fewer than k candidates: pad with -1.  The last thread's run ends at the
  // last token, so its final write position is the number selected.
  if (tid == SEL_THREADS - 1)
    for (int i = pos; i < k; ++i) ob[i] = -1;
}

hipError_t launch_select_topk(const float *scores, int32_t n_parts, const int32_t *excl_idx,
                              const int32_t *excl_off, int32_t batch, int32_t n_tokens, int32_t k,
                              int32_t *out_idx, const int32_t *out_off, bool lowest,
                              hipStream_t s) {
  if (batch == 0 || k == 0) return hipSuccess;
  if (n_tokens > SEL_MAX_N) return hipErrorInvalidValue;
  int np2 = 1;
  while (np2 < n_tokens) np2 <<= 1;
  if (np2 < 2) np2 = 2;
  const size_t lds = (size_t)np2 * sizeof(unsigned long long) + (size_t)n_tokens * sizeof(int);
  select_topk_kernel<<<batch, SEL_THREADS, lds, s>>>(scores, n_parts, excl_idx, excl_off, n_tokens,
                                                     np2, k, out_idx, out_off, lowest);
  return hipGetLastError();
}

}  // namespace marche
