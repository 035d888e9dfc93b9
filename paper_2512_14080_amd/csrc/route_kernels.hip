// Routing kernels: softmax + top-K selection, the per-expert membership
// bitmap, and the routing metadata built from it (counts, offsets,
// expert-major rows and the token-major CSR view).
//
// Top-K follows the token-choice rule of Section 2.3 with the stable order of
// the top-K kernel in Appendix D (equal scores go to the lower expert index).
// Unlike that kernel, the expert index is not packed into the low mantissa
// bits: the comparison uses the exact (score, index) pair, so no score is
// perturbed.  One wave64 handles one token; the K winners are found by K
// rounds of a wave-wide arg-max over (score desc, index asc).
#include "device_common.h"
#include "launch.h"

namespace smoe {

template <int EPL>
// `in` and `scores` may alias (logits overwritten in place by the scores).
__global__ __launch_bounds__(256) void softmax_topk_kernel(const float* in, float* scores,
                                                           float* __restrict__ scores_t, int32_t* __restrict__ topk_idx,
                                                           float* __restrict__ topk_w, int T, int E, int K,
                                                           int do_softmax) {
  const int wave = threadIdx.x >> 6;
  const int lane = lane_id();
  const int t = blockIdx.x * 4 + wave;
  if (t >= T) return;
  const float* row = in + (size_t)t * E;
  float v[EPL];
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const int e = lane + 64 * j;
    v[j] = e < E ? row[e] : -INFINITY;
  }
  if (do_softmax) {
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < EPL; ++j) m = fmaxf(m, v[j]);
    m = wave_max(m);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + 64 * j;
      v[j] = e < E ? expf(v[j] - m) : 0.f;
      s += v[j];
    }
    s = wave_sum(s);
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + 64 * j;
      if (e < E) {
        v[j] = v[j] / s;
        scores[(size_t)t * E + e] = v[j];
      }
    }
  }
  if (scores_t) {
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + 64 * j;
      if (e < E) scores_t[(size_t)e * T + t] = v[j];
    }
  }
  // K rounds of wave arg-max over (value desc, expert asc)
  uint32_t taken = 0;
  int sel_e[16];
  float sel_v[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    sel_e[k] = 0;
    sel_v[k] = 0.f;
    if (k < K) {
      float bv = -INFINITY;
      int be = 0x7fffffff;
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
        const int e = lane + 64 * j;
        if (e < E && !((taken >> j) & 1u)) {
          if (be == 0x7fffffff || v[j] > bv || (v[j] == bv && e < be)) {
            bv = v[j];
            be = e;
          }
        }
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const float ov = __shfl_xor(bv, o, kWave);
        const int oe = __shfl_xor(be, o, kWave);
        // candidates without a valid expert carry index INT_MAX and lose
        const bool better = (oe != 0x7fffffff) && (be == 0x7fffffff || ov > bv || (ov == bv && oe < be));
        if (better) {
          bv = ov;
          be = oe;
        }
      }
      if ((be & 63) == lane) taken |= 1u << (be >> 6);
      sel_e[k] = be;
      sel_v[k] = bv;
    }
  }
  // renormalisation denominator: selected scores summed in ascending expert order
  float denom = 0.f;
  int last = -1;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    if (r < K) {
      int nxt = 0x7fffffff;
      float nv = 0.f;
#pragma unroll
      for (int k = 0; k < 16; ++k)
        if (k < K && sel_e[k] > last && sel_e[k] < nxt) {
          nxt = sel_e[k];
          nv = sel_v[k];
        }
      denom += nv;
      last = nxt;
    }
  }
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    if (k < K && lane == k) {
      topk_idx[(size_t)t * K + k] = sel_e[k];
      if (topk_w) topk_w[(size_t)t * K + k] = sel_v[k] / denom;
    }
  }
}

// One wave per 64-token word: bit (t % 64) of mask[e][t / 64] is set iff
// expert e is among token t's selected experts.
__global__ __launch_bounds__(256) void build_mask_kernel(const int32_t* __restrict__ topk_idx,
                                                         uint64_t* __restrict__ mask, int T, int E, int K, int W) {
  const int wave = threadIdx.x >> 6;
  const int lane = lane_id();
  const int w = blockIdx.x * 4 + wave;
  if (w >= W) return;
  const int t = w * 64 + lane;
  int ex[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) ex[k] = (k < K && t < T) ? topk_idx[(size_t)t * K + k] : -1;
  for (int e0 = 0; e0 < E; e0 += 64) {
    uint64_t mine = 0;
    const int lim = min(64, E - e0);
    for (int i = 0; i < lim; ++i) {
      const int e = e0 + i;
      bool hit = false;
#pragma unroll
      for (int k = 0; k < 16; ++k) hit |= (ex[k] == e);
      const uint64_t b = __ballot(hit);
      if (lane == i) mine = b;
    }
    if (lane < lim) mask[(size_t)(e0 + lane) * W + w] = mine;
  }
}

// Per expert: popcount prefix over its mask words and its count f_e.
__global__ __launch_bounds__(256) void expert_scan_kernel(const uint64_t* __restrict__ mask,
                                                          int32_t* __restrict__ prefix, int32_t* __restrict__ counts,
                                                          int W) {
  __shared__ int lds[16];
  const int e = blockIdx.x;
  const uint64_t* m = mask + (size_t)e * W;
  int32_t* p = prefix + (size_t)e * W;
  int running = 0;
  for (int c0 = 0; c0 < W; c0 += 256) {
    const int w = c0 + threadIdx.x;
    const int pc = w < W ? __popcll(m[w]) : 0;
    int total;
    const int ex = block_excl_scan<256>(pc, &total, lds);
    if (w < W) p[w] = running + ex;
    running += total;
  }
  if (threadIdx.x == 0) counts[e] = running;
}

// offsets[0..n] = exclusive scan of cnt[0..n-1] (one block of 1024 threads).
__global__ __launch_bounds__(1024) void scan_kernel(const int32_t* __restrict__ cnt, int32_t* __restrict__ out,
                                                    int n) {
  __shared__ int lds[16];
  int running = 0;
  for (int c0 = 0; c0 < n; c0 += 1024) {
    const int i = c0 + threadIdx.x;
    const int v = i < n ? cnt[i] : 0;
    int total;
    const int ex = block_excl_scan<1024>(v, &total, lds);
    if (i < n) out[i] = running + ex;
    running += total;
  }
  if (threadIdx.x == 0) out[n] = running;
}

// Per token: number of selected experts and the renormalisation denominator
// (selected scores summed in ascending expert order, fp32).
__global__ __launch_bounds__(256) void token_count_kernel(const uint64_t* __restrict__ mask,
                                                          const float* __restrict__ scores, int32_t* __restrict__ cnt,
                                                          float* __restrict__ denom, int T, int E, int W) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  const int w = t >> 6, b = t & 63;
  int c = 0;
  float s = 0.f;
  for (int e = 0; e < E; ++e) {
    const uint64_t word = mask[(size_t)e * W + w];
    if ((word >> b) & 1ull) {
      ++c;
      s += scores[(size_t)t * E + e];
    }
  }
  cnt[t] = c;
  denom[t] = s;
}

// Per token: place its rows (expert-major index of each pair), the
// token-major list and the renormalised weights.
__global__ __launch_bounds__(256) void token_place_kernel(
    const uint64_t* __restrict__ mask, const int32_t* __restrict__ prefix, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ tok_offsets, const float* __restrict__ scores, const float* __restrict__ denom,
    int32_t* __restrict__ tok_rows, int32_t* __restrict__ row_token, int32_t* __restrict__ row_expert,
    float* __restrict__ row_w, int T, int E, int W) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  const int w = t >> 6, b = t & 63;
  const uint64_t below = b ? (~0ull >> (64 - b)) : 0ull;
  int j = tok_offsets[t];
  const float dn = denom[t];
  for (int e = 0; e < E; ++e) {
    const uint64_t word = mask[(size_t)e * W + w];
    if ((word >> b) & 1ull) {
      const int r = offsets[e] + prefix[(size_t)e * W + w] + __popcll(word & below);
      tok_rows[j++] = r;
      row_token[r] = t;
      row_expert[r] = e;
      row_w[r] = scores[(size_t)t * E + e] / dn;
    }
  }
}

// ---------------------------------------------------------------- launchers

hipError_t launch_softmax_topk(const float* in, float* scores, float* scores_t, int32_t* topk_idx, float* topk_w,
                               int T, int E, int K, int do_softmax, hipStream_t s) {
  const dim3 grid((T + 3) / 4), block(256);
  const int epl = (E + 63) / 64;
#define SMOE_TOPK(N)                                                                                    \
  if (epl <= N) {                                                                                       \
    softmax_topk_kernel<N><<<grid, block, 0, s>>>(in, scores, scores_t, topk_idx, topk_w, T, E, K, do_softmax); \
    return hipGetLastError();                                                                           \
  }
  SMOE_TOPK(1)
  SMOE_TOPK(2)
  SMOE_TOPK(4)
  SMOE_TOPK(8)
  SMOE_TOPK(16)
  SMOE_TOPK(32)
  SMOE_TOPK(64)
#undef SMOE_TOPK
  return hipErrorInvalidValue;
}

hipError_t launch_build_mask(const int32_t* topk_idx, uint64_t* mask, int T, int E, int K, int W, hipStream_t s) {
  build_mask_kernel<<<dim3((W + 3) / 4), dim3(256), 0, s>>>(topk_idx, mask, T, E, K, W);
  return hipGetLastError();
}

hipError_t launch_metadata(const moe_routing& r, const float* scores, int T, int E, hipStream_t s) {
  const int W = r.words;
  expert_scan_kernel<<<dim3(E), dim3(256), 0, s>>>(r.mask, r.mask_prefix, r.counts, W);
  scan_kernel<<<dim3(1), dim3(1024), 0, s>>>(r.counts, r.offsets, E);
  const dim3 tg((T + 255) / 256), tb(256);
  token_count_kernel<<<tg, tb, 0, s>>>(r.mask, scores, r.tok_count, r.tok_denom, T, E, W);
  scan_kernel<<<dim3(1), dim3(1024), 0, s>>>(r.tok_count, r.tok_offsets, T);
  token_place_kernel<<<tg, tb, 0, s>>>(r.mask, r.mask_prefix, r.offsets, r.tok_offsets, scores, r.tok_denom,
                                       r.tok_rows, r.row_token, r.row_expert, r.row_w, T, E, W);
  return hipGetLastError();
}

}  // namespace smoe
