// Exact (score, expert) ordering and the small sorting networks of the top-K
// selection (Section 2.3; Appendix D's stable top-K): a pair packs the
// order-preserving image of the fp32 score above the complemented expert
// index, so the unsigned pair order is score descending, then expert
// ascending (equal scores go to the lower expert), with no score perturbed.
// Shared by the routing kernels and the router GEMM's fused epilogue.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace smoe {

// Order-preserving integer image of an fp32 score (+0 and -0 map to one key).
// Comparisons go through it so the selection order is total even for NaN
// scores (a NaN never compares greater or smaller as a float, which would let
// the lanes of a wave disagree on the winner and pick an expert twice).
__device__ __forceinline__ uint32_t topk_key(float x) {
  uint32_t b = __float_as_uint(x);
  if (b == 0x80000000u) b = 0;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
// inverse of topk_key (-0 comes back as +0)
__device__ __forceinline__ float topk_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// (score, expert) pair; 0 ranks below every real pair
__device__ __forceinline__ uint64_t topk_pair(float score, int expert) {
  return ((uint64_t)topk_key(score) << 32) | (uint32_t)~(uint32_t)expert;
}

// a >= b afterwards.  The swap selects the 32-bit halves on one 64-bit
// comparison; written as a 64-bit select pair it becomes an unsigned max and
// min, i.e. two comparisons.
template <int KM>
__device__ __forceinline__ void topk_cex(uint64_t& a, uint64_t& b) {
  const bool sw = b > a;
  const uint32_t al = (uint32_t)a, ah = (uint32_t)(a >> 32), bl = (uint32_t)b, bh = (uint32_t)(b >> 32);
  const uint32_t xl = sw ? bl : al, xh = sw ? bh : ah, yl = sw ? al : bl, yh = sw ? ah : bh;
  a = ((uint64_t)xh << 32) | xl;
  b = ((uint64_t)yh << 32) | yl;
}
// sort of KM pairs, largest first (KM a power of two): for KM = 8 Batcher's
// odd-even merge sort (19 compare-exchanges: pairs, then odd-even merges of
// 2 + 2 and 4 + 4), otherwise a bitonic sort
template <int KM>
__device__ __forceinline__ void topk_sort(uint64_t (&v)[KM]) {
  if constexpr (KM == 8) {
    constexpr int kNet[19][2] = {{0, 1}, {2, 3}, {4, 5}, {6, 7},                  // sorted pairs
                                 {0, 2}, {1, 3}, {1, 2}, {4, 6}, {5, 7}, {5, 6},  // sorted quadruples
                                 {0, 4}, {1, 5}, {2, 6}, {3, 7}, {2, 4}, {3, 5}, {1, 2}, {3, 4}, {5, 6}};
#pragma unroll
    for (int c = 0; c < 19; ++c) topk_cex<KM>(v[kNet[c][0]], v[kNet[c][1]]);
    return;
  }
#pragma unroll
  for (int k = 2; k <= KM; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < KM; ++i) {
        const int l = i ^ j;
        if (l > i) {
          if ((i & k) == 0)
            topk_cex<KM>(v[i], v[l]);
          else
            topk_cex<KM>(v[l], v[i]);
        }
      }
}
template <int KM>
__device__ __forceinline__ void topk_merge(uint64_t (&a)[KM], const uint64_t (&b)[KM]) {
#pragma unroll
  for (int i = 0; i < KM; ++i) a[i] = a[i] > b[KM - 1 - i] ? a[i] : b[KM - 1 - i];
#pragma unroll
  for (int h = KM / 2; h >= 1; h >>= 1)
#pragma unroll
    for (int i = 0; i < KM; ++i)
      if ((i & h) == 0) topk_cex<KM>(a[i], a[i + h]);
}

}  // namespace smoe
