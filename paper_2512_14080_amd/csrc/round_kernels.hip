// Token rounding (Section 5.2): per-expert rounding decision and the
// selection of the dropped TC tokens or the padded non-TC tokens.
//
// The paper describes the method as a two-step sort (TC top-K, then a sort of
// each expert's tokens by router score with TC tokens preferred).  Only the
// last tile changes, so instead of sorting all T tokens per expert this code
// selects the at most m_tile-1 tokens that change with a 4-pass 8-bit radix
// select on an order-preserving integer image of the fp32 score, then breaks
// ties on the threshold value by token index.  The result is the same set the
// full sort would give.
#include "device_common.h"
#include "launch.h"

namespace smoe {

// Decide f^TR_e for every expert; writes round_dir[e] and the number of
// tokens to change, need[e] = |f^TR_e - f_e|.
__global__ __launch_bounds__(256) void tr_decide_kernel(const int32_t* __restrict__ counts, const float* __restrict__ u,
                                                        int32_t* __restrict__ round_dir, int32_t* __restrict__ need,
                                                        int T, int E, int M, int mode) {
  if (mode == MOE_ROUND_BALANCE) {
    // running residual over experts in index order: sequential by definition
    if (threadIdx.x != 0) return;
    long z = 0;
    for (int e = 0; e < E; ++e) {
      const int f = counts[e];
      const int lo = (f / M) * M;
      const int hi = lo + ((f % M) ? M : 0);
      const long r_up = hi - f, r_dn = lo - f;
      const long a = r_up + z < 0 ? -(r_up + z) : r_up + z;
      const long b = r_dn + z < 0 ? -(r_dn + z) : r_dn + z;
      const bool pad = (a < b) && (hi <= T);
      z += pad ? r_up : r_dn;
      const int ftr = pad ? hi : lo;
      round_dir[e] = ftr > f ? 1 : (ftr < f ? -1 : 0);
      need[e] = ftr > f ? ftr - f : f - ftr;
    }
    return;
  }
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    const int f = counts[e];
    const int lo = (f / M) * M;
    const int hi = lo + ((f % M) ? M : 0);
    bool pad;
    if (mode == MOE_ROUND_NEAREST)
      pad = (hi - f) < (f - lo);
    else if (mode == MOE_ROUND_UP)
      pad = hi > f;
    else if (mode == MOE_ROUND_DOWN)
      pad = false;
    else  // stochastic: Bernoulli((f - lo)/M) from the supplied uniform
      pad = (u[e] * (float)M) < (float)(f - lo);
    pad = pad && (hi <= T);
    const int ftr = pad ? hi : lo;
    round_dir[e] = ftr > f ? 1 : (ftr < f ? -1 : 0);
    need[e] = ftr > f ? ftr - f : f - ftr;
  }
}

// order-preserving image of an fp32 score (+0 and -0 map to the same key)
__device__ __forceinline__ uint32_t score_key(float x) {
  uint32_t b = __float_as_uint(x);
  if (b == 0x80000000u) b = 0;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

constexpr int kSelThreads = 1024;

// One block per expert.  Copies the TC mask row of expert e into the rounded
// mask and flips the `need` selected bits:
//   pad  (dir > 0): the need best non-TC tokens by (score desc, token asc);
//   drop (dir < 0): the need worst TC tokens by (score asc, token desc).
// Both become "the need largest keys" with key = score_key for pads and
// ~score_key for drops, ties preferring low tokens for pads, high for drops.
__global__ __launch_bounds__(kSelThreads) void tr_select_kernel(const uint64_t* __restrict__ tc_mask,
                                                                uint64_t* __restrict__ tr_mask,
                                                                const float* __restrict__ scores_t,
                                                                const int32_t* __restrict__ round_dir,
                                                                const int32_t* __restrict__ need_arr, int T, int W) {
  __shared__ int hist[256];
  __shared__ int sh[4];
  __shared__ int lds[16];
  const int e = blockIdx.x;
  const uint64_t* src = tc_mask + (size_t)e * W;
  uint64_t* dst = tr_mask + (size_t)e * W;
  const int dir = round_dir[e];
  const int need = need_arr[e];
  if (dir == 0 || need == 0) {
    for (int w = threadIdx.x; w < W; w += kSelThreads) dst[w] = src[w];
    return;
  }
  const float* S = scores_t + (size_t)e * T;
  const bool want_set = dir < 0;  // candidates: TC tokens for drops, non-TC for pads
  uint32_t prefix = 0;
  int remaining = need;
  for (int pass = 3; pass >= 0; --pass) {
    for (int i = threadIdx.x; i < 256; i += kSelThreads) hist[i] = 0;
    __syncthreads();
    const int sh_hi = 8 * (pass + 1);
    for (int t = threadIdx.x; t < T; t += kSelThreads) {
      const bool in_tc = (src[t >> 6] >> (t & 63)) & 1ull;
      if (in_tc != want_set) continue;
      uint32_t k = score_key(S[t]);
      if (dir < 0) k = ~k;
      if (pass == 3 || (k >> sh_hi) == prefix) atomicAdd(&hist[(k >> (8 * pass)) & 255], 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int cum = 0, dsel = 0;
      for (int dgt = 255; dgt >= 0; --dgt) {
        if (cum + hist[dgt] >= remaining) {
          dsel = dgt;
          break;
        }
        cum += hist[dgt];
      }
      sh[0] = dsel;
      sh[1] = remaining - cum;
    }
    __syncthreads();
    prefix = (prefix << 8) | (uint32_t)sh[0];
    remaining = sh[1];
    __syncthreads();
  }
  const uint32_t tau = prefix;
  // marking pass over words, in preferred token order (ascending for pads,
  // descending for drops); ties on tau are taken until `remaining` are used
  int carry = 0;
  for (int c0 = 0; c0 < W; c0 += kSelThreads) {
    const int idx = c0 + threadIdx.x;
    const int w = dir > 0 ? idx : W - 1 - idx;
    uint64_t word = 0;
    int ties = 0;
    const bool valid = idx < W;
    if (valid) {
      word = src[w];
      for (int b = 0; b < 64; ++b) {
        const int t = w * 64 + b;
        if (t >= T) break;
        const bool in_tc = (word >> b) & 1ull;
        if (in_tc != want_set) continue;
        uint32_t k = score_key(S[t]);
        if (dir < 0) k = ~k;
        ties += (k == tau);
      }
    }
    int total;
    const int before = carry + block_excl_scan<kSelThreads>(ties, &total, lds);
    if (valid) {
      uint64_t out = word;
      int rank = before;
      for (int bb = 0; bb < 64; ++bb) {
        const int b = dir > 0 ? bb : 63 - bb;
        const int t = w * 64 + b;
        if (t >= T) continue;
        const bool in_tc = (word >> b) & 1ull;
        if (in_tc != want_set) continue;
        uint32_t k = score_key(S[t]);
        if (dir < 0) k = ~k;
        bool flip = k > tau;
        if (k == tau) {
          flip = rank < remaining;
          ++rank;
        }
        if (flip) out ^= (1ull << b);
      }
      dst[w] = out;
    }
    carry += total;
  }
}

hipError_t launch_round(const moe_routing& tc, moe_routing& tr, const float* u, int T, int E, int M, int mode,
                        hipStream_t s) {
  int32_t* need = tr.scratch;
  tr_decide_kernel<<<dim3(1), dim3(256), 0, s>>>(tc.counts, u, tr.round_dir, need, T, E, M, mode);
  tr_select_kernel<<<dim3(E), dim3(kSelThreads), 0, s>>>(tc.mask, tr.mask, tc.scores_t, tr.round_dir, need, T,
                                                         tr.words);
  return hipGetLastError();
}

}  // namespace smoe
