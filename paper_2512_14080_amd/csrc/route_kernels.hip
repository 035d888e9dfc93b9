// Routing kernels: softmax + top-K selection, the per-expert membership
// bitmap, and the routing metadata built from it (counts, offsets,
// expert-major rows and the token-major CSR view).
//
// Top-K follows the token-choice rule of Section 2.3 with the stable order of
// the top-K kernel in Appendix D (equal scores go to the lower expert index).
// Unlike that kernel, the expert index is not packed into the low mantissa
// bits: the comparison uses the exact (score, index) pair, so no score is
// perturbed.  One wave64 handles one token at a time; the K winners are found
// by K rounds of a wave-wide arg-max over (score desc, index asc).  A
// workgroup owns 64 consecutive tokens, i.e. one 64-bit word of every
// expert's membership bitmap, which it assembles in LDS.
#include "device_common.h"
#include "launch.h"
#include "topk_net.h"

namespace smoe {

constexpr int kTopkWaves = 16;

// Workgroup = 64 tokens (one membership word).  `in` and `scores` may alias
// (logits overwritten in place by the scores).  With STASH every output of the
// workgroup's 64 tokens is staged in LDS and written at the end: the scores
// (token-major and transposed, scores_t[e][t] in 64-token runs) and the top-K
// lists.  With no global store pending while the token loop runs, the wait
// for the next token's row (requested one token ahead) covers only loads.
constexpr int kStashPitch = 65;  // floats per expert row of the stash (bank-conflict-free both ways)
template <int EPL, bool STASH>
__global__ __launch_bounds__(1024) void topk_route_kernel(const float* in, float* scores, float* __restrict__ scores_t,
                                                         int32_t* __restrict__ topk_idx, float* __restrict__ topk_w,
                                                         uint64_t* __restrict__ mask, int T, int E, int K, int W,
                                                         int do_softmax) {
  static_assert(EPL >= 1 && EPL <= 64, "the taken mask holds one bit per value of a lane");
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  unsigned long long* mword = (unsigned long long*)dyn;                  // [E]
  float* st = (float*)(dyn + ((E * 8 + 15) & ~15));                       // STASH: [E][kStashPitch]
  int* sidx = (int*)(st + (STASH ? E * kStashPitch : 0));                 // STASH: [64][K]
  float* sw = (float*)(sidx + (STASH ? 64 * K : 0));                      // STASH: [64][K]
  const int w = blockIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = lane_id();
  for (int e = threadIdx.x; e < E; e += kTopkWaves * 64) mword[e] = 0ull;
  __syncthreads();
  auto load_row = [&](int i, float (&v)[EPL]) {
    const int t = w * 64 + i;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + 64 * j;
      v[j] = (t < T && e < E) ? in[(size_t)t * E + e] : -INFINITY;
    }
  };
  float vn[EPL];
  load_row(wave, vn);
  for (int i = wave; i < 64; i += kTopkWaves) {
    const int t = w * 64 + i;
    if (t >= T) break;
    float v[EPL];
#pragma unroll
    for (int j = 0; j < EPL; ++j) v[j] = vn[j];
    if (i + kTopkWaves < 64) load_row(i + kTopkWaves, vn);  // the wave's next token, in flight meanwhile
    if (do_softmax) {
      float m = -INFINITY;
#pragma unroll
      for (int j = 0; j < EPL; ++j) m = fmaxf(m, v[j]);
      m = dpp_reduce(m, [](float a, float b) { return fmaxf(a, b); });
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
        const int e = lane + 64 * j;
        v[j] = e < E ? expf(v[j] - m) : 0.f;
        s += v[j];
      }
      s = dpp_reduce(s, [](float a, float b) { return a + b; });
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
        const int e = lane + 64 * j;
        if (e < E) {
          v[j] = v[j] / s;
          if (!STASH) scores[(size_t)t * E + e] = v[j];
        }
      }
    }
    if (STASH || scores_t) {
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
        const int e = lane + 64 * j;
        if (e < E) {
          if (STASH)
            st[e * kStashPitch + i] = v[j];
          else
            scores_t[(size_t)e * T + t] = v[j];
        }
      }
    }
    // K rounds of wave arg-max over (value desc, expert asc): the wave maximum
    // of the 32-bit keys (a DPP max), then the lowest expert holding it from
    // ballots (expert 64j + l is value j of lane l: lowest j, then lowest lane)
    uint64_t taken = 0;  // bit j: value j of this lane is selected (EPL <= 64)
    int sel_e[16];
    float sel_v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      sel_e[k] = 0;
      sel_v[k] = 0.f;
      if (k < K) {
        uint32_t best = 0;
        int bj = -1;  // j of this lane's best candidate (the lowest j on equal keys)
#pragma unroll
        for (int j = 0; j < EPL; ++j) {
          const int e = lane + 64 * j;
          if (e < E && !((taken >> j) & 1ull)) {
            const uint32_t c = topk_key(v[j]);
            if (bj < 0 || c > best) {
              best = c;
              bj = j;
            }
          }
        }
        const uint32_t m = dpp_reduce(bj >= 0 ? best : 0u, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
        int be = 0x7fffffff;
#pragma unroll
        for (int j = 0; j < EPL; ++j) {
          const uint64_t hit = __ballot(bj == j && best == m);
          if (hit && be == 0x7fffffff) be = __ffsll((unsigned long long)hit) - 1 + 64 * j;
        }
        if (be != 0x7fffffff && (be & 63) == lane) taken |= 1ull << (be >> 6);
        sel_e[k] = be;
        sel_v[k] = topk_value(m);
      }
    }
    // renormalisation denominator: selected scores summed in ascending expert
    // order (expert 64j + l is value j of lane l; ballots list them in order)
    float denom = 0.f;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      uint64_t sel = __ballot((taken >> j) & 1ull);
      while (sel) {
        const int l = __ffsll((unsigned long long)sel) - 1;
        denom += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v[j]), l));
        sel &= sel - 1;
      }
    }
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      if (k < K && lane == k) {
        if (STASH) {
          sidx[i * K + k] = sel_e[k];
          sw[i * K + k] = sel_v[k] / denom;
        } else {
          topk_idx[(size_t)t * K + k] = sel_e[k];
          topk_w[(size_t)t * K + k] = sel_v[k] / denom;
        }
        atomicOr(&mword[sel_e[k]], 1ull << i);
      }
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += kTopkWaves * 64) mask[(size_t)e * W + w] = mword[e];
  if (STASH) {
    const int nt = min(64, T - w * 64);  // tokens of this workgroup
    if (do_softmax)
      for (int idx = threadIdx.x; idx < nt * E; idx += kTopkWaves * 64) {
        const int i = idx / E, e = idx % E;
        scores[(size_t)(w * 64 + i) * E + e] = st[e * kStashPitch + i];
      }
    if (scores_t)
      for (int idx = threadIdx.x; idx < E * 64; idx += kTopkWaves * 64) {
        const int e = idx >> 6, i = idx & 63;
        if (i < nt) scores_t[(size_t)e * T + w * 64 + i] = st[e * kStashPitch + i];
      }
    for (int idx = threadIdx.x; idx < nt * K; idx += kTopkWaves * 64) {
      topk_idx[(size_t)w * 64 * K + idx] = sidx[idx];
      topk_w[(size_t)w * 64 * K + idx] = sw[idx];
    }
  }
}

// Lane-per-token selection (K <= KM <= 16; E a multiple of 4 * NW, E <= 256).
// A workgroup owns the 64 tokens of one membership word, lane l token 64w + l,
// and its NW waves split the experts into NW contiguous slices, so the
// per-token work is ordinary per-lane arithmetic instead of wave-wide
// reductions.  Each wave keeps its slice of the token's row in LDS as
// [slice/4][64] float4 (lane l's column: conflict-free in every pass):
//   1. row max (the row loads are issued 16 float4 at a time), combined
//      across the slices;
//   2. exp(x - max) and the slice sums, combined in slice order;
//   3. scores = exp * (1 / sum) (written token-major and, coalesced across lanes,
//      transposed), and a KM-slot insertion network over the (key, expert)
//      pairs of the slice: an element moves down past every slot whose pair
//      it exceeds; the network runs only when some lane's element beats its
//      last slot.  The slices' lists are then merged (top-KM of two sorted
//      lists: pairwise maxima of one list against the other reversed, then a
//      bitonic clean-up), every wave doing the same merge;
//   4. membership: expert e is selected iff its pair ranks at or above the
//      K-th slot; a ballot per expert is the membership word.  The selected
//      scores are summed in ascending expert order for the renormalisation
//      denominator (each slice lists its selected scores in order in LDS,
//      the first wave adds the lists slice by slice).
// The (score, index) pairs are compared exactly, as in the wave-per-token
// kernel above: equal keys order by the lower expert.
template <int KM, int NW>
__global__ __launch_bounds__(64 * NW) void topk_lane_kernel(const float* in, float* scores, float* __restrict__ scores_t,
                                                            int32_t* __restrict__ topk_idx, float* __restrict__ topk_w,
                                                            uint64_t* __restrict__ mask, int T, int E, int K, int W,
                                                            int do_softmax) {
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  const int w = blockIdx.x;
  const int q = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = lane_id();
  const int t = w * 64 + lane;
  const bool live = t < T;
  const int Eq = E / NW, Gq = Eq >> 2, e0 = q * Eq;
  f32x4* cols = (f32x4*)dyn + (size_t)q * Gq * 64;      // [Gq][64]
  float* xmax = (float*)(dyn + (size_t)E * 256);           // [NW][64]
  float* xsum = xmax + NW * 64;                            // [NW][64]
  uint64_t* lists = (uint64_t*)(xsum + NW * 64);           // [NW][KM][64]
  float* sv = (float*)(lists + NW * KM * 64);              // [NW][KM][64] selected scores, expert order
  int* nsel = (int*)(sv + NW * KM * 64);                   // [NW][64]
  // a lane past T reads token 0's row and discards it
  const f32x4* row = (const f32x4*)(in + (size_t)(live ? t : 0) * E + e0);
  const f32x4 ninf = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
  float m = -INFINITY;
#pragma unroll 16
  for (int g = 0; g < Gq; ++g) {
    const f32x4 x0 = row[g];
    const f32x4 x = live ? x0 : ninf;
    cols[g * 64 + lane] = x;
    m = fmaxf(m, fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
  }
  float s = 1.f;
  if (do_softmax) {
    if constexpr (NW > 1) {
      xmax[q * 64 + lane] = m;
      __syncthreads();
#pragma unroll
      for (int p = 0; p < NW; ++p) m = fmaxf(m, xmax[p * 64 + lane]);
    }
    s = 0.f;
#pragma unroll 4
    for (int g = 0; g < Gq; ++g) {
      f32x4 x = cols[g * 64 + lane];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        x[c] = __expf(x[c] - m);  // v_exp_f32 of (x - m) log2(e): a few ulp for |x - m| < 100
        s += x[c];
      }
      cols[g * 64 + lane] = x;
    }
    if constexpr (NW > 1) {
      xsum[q * 64 + lane] = s;
      __syncthreads();
      s = xsum[lane];
#pragma unroll
      for (int p = 1; p < NW; ++p) s += xsum[p * 64 + lane];
    }
  }
  const float rs = 1.f / s;  // scores = exp * (1 / sum): within an ulp of the quotient
  uint64_t top[KM];
#pragma unroll
  for (int k = 0; k < KM; ++k) top[k] = 0;  // below every (key, ~expert) pair
  // Pairs are taken in groups of KM: each group is sorted by a bitonic network
  // and merged into the running top-KM list, i.e. independent compare-exchanges
  // instead of a serial insertion chain per pair.  One step covers G2 float4s
  // (KM = 8: two); slots past the slice and lanes past T hold 0, below every
  // real pair.
  constexpr int G2 = KM >= 4 ? KM / 4 : 1;
  for (int g0 = 0; g0 < Gq; g0 += G2) {
    uint64_t pr[4 * G2];
#pragma unroll
    for (int gg = 0; gg < G2; ++gg) {
      const int g = g0 + gg;
      if (g < Gq) {
        f32x4 p = cols[g * 64 + lane];
        const int eg = e0 + 4 * g;
        if (do_softmax) {
#pragma unroll
          for (int c = 0; c < 4; ++c) p[c] = p[c] * rs;
          cols[g * 64 + lane] = p;
          if (live) *(f32x4*)(scores + (size_t)t * E + eg) = p;
        }
        if (scores_t && live) {
#pragma unroll
          for (int c = 0; c < 4; ++c) scores_t[(size_t)(eg + c) * T + t] = p[c];
        }
#pragma unroll
        for (int c = 0; c < 4; ++c)
          pr[4 * gg + c] = live ? topk_pair(p[c], eg + c) : 0ull;
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) pr[4 * gg + c] = 0ull;
      }
    }
#pragma unroll
    for (int h = 0; h < 4 * G2; h += KM) {
      uint64_t grp[KM];
#pragma unroll
      for (int k = 0; k < KM; ++k) grp[k] = pr[h + k];
      topk_sort<KM>(grp);
      topk_merge<KM>(top, grp);
    }
  }
  if constexpr (NW > 1) {
#pragma unroll
    for (int k = 0; k < KM; ++k) lists[(q * KM + k) * 64 + lane] = top[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < KM; ++k) top[k] = lists[k * 64 + lane];
#pragma unroll
    for (int p = 1; p < NW; ++p) {
      uint64_t b[KM];
#pragma unroll
      for (int k = 0; k < KM; ++k) b[k] = lists[(p * KM + k) * 64 + lane];
      topk_merge<KM>(top, b);
    }
  }
  uint64_t thr = top[0];
#pragma unroll
  for (int k = 1; k < KM; ++k)
    if (k == K - 1) thr = top[k];
  // membership words of this wave's experts (expert e0 + 64 r + lane in mw[r])
  constexpr int kWords = NW > 1 ? 1 : 4;
  float den = 0.f;
  int ns = 0;
  uint64_t mw[kWords];
#pragma unroll
  for (int r = 0; r < kWords; ++r) mw[r] = 0ull;
#pragma unroll
  for (int r = 0; r < kWords; ++r) {
    const int g1 = min(Gq, 16 * r + 16);
    for (int g = 16 * r; g < g1; ++g) {
      const f32x4 p = cols[g * 64 + lane];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int el = 4 * g + c;  // expert e0 + el
        const uint64_t x = topk_pair(p[c], e0 + el);
        const bool sel = live && x >= thr;
        const uint64_t word = __ballot(sel);
        if (lane == (el & 63)) mw[r] = word;
        if constexpr (NW > 1) {
          if (sel) sv[(q * KM + ns) * 64 + lane] = p[c];
          ns += sel;
        } else {
          den += sel ? p[c] : 0.f;  // +0 for the others leaves the sum unchanged
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < kWords; ++r)
    if (64 * r + lane < Eq) mask[(size_t)(e0 + 64 * r + lane) * W + w] = mw[r];
  if constexpr (NW > 1) {
    nsel[q * 64 + lane] = ns;
    __syncthreads();
    if (q != 0) return;
    // selected scores in ascending expert order: slice by slice
    for (int p = 0; p < NW; ++p) {
      const int np = nsel[p * 64 + lane];
      for (int j = 0; j < np; ++j) den += sv[(p * KM + j) * 64 + lane];
    }
  }
  if (live) {
#pragma unroll
    for (int k = 0; k < KM; ++k)
      if (k < K) {
        topk_idx[(size_t)t * K + k] = (int32_t)~(uint32_t)top[k];
        topk_w[(size_t)t * K + k] = topk_value((uint32_t)(top[k] >> 32)) / den;
      }
  }
}

static size_t topk_lane_lds(int E, int KM, int NW) {
  return (size_t)E * 256 + (NW > 1 ? (size_t)NW * 64 * (4 + 4 + 8 * KM + 4 * KM + 4) : 0);
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

// out[0..n] = exclusive scan of cnt[0..n-1] (one block of 1024 threads, four
// values per thread per pass).
__global__ __launch_bounds__(1024) void scan_kernel(const int32_t* __restrict__ cnt, int32_t* __restrict__ out,
                                                    int n, int32_t* __restrict__ status) {
  __shared__ int lds[16];
  if (status && threadIdx.x == 0) *status = 0;  // cleared before the placement that may flag it
  int running = 0;
  for (int c0 = 0; c0 < n; c0 += 4096) {
    const int i0 = c0 + threadIdx.x * 4;
    int v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = i0 + q < n ? cnt[i0 + q] : 0;
    const int sum = v[0] + v[1] + v[2] + v[3];
    int total;
    int ex = block_excl_scan<1024>(sum, &total, lds) + running;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (i0 + q < n) out[i0 + q] = ex;
      ex += v[q];
    }
    running += total;
  }
  if (threadIdx.x == 0) out[n] = running;
}

__device__ __forceinline__ int expert_row(const uint64_t* __restrict__ mask, const int32_t* __restrict__ prefix,
                                          const int32_t* __restrict__ offsets, int e, int W, int w, uint64_t below) {
  const uint64_t word = mask[(size_t)e * W + w];
  return offsets[e] + prefix[(size_t)e * W + w] + __popcll(word & below);
}

// Token-choice placement: every token has exactly K rows, so the token-major
// offsets are t*K.  Each token's experts are visited in ascending order.
__global__ __launch_bounds__(256) void tc_place_kernel(const int32_t* __restrict__ topk_idx,
                                                       const float* __restrict__ topk_w,
                                                       const uint64_t* __restrict__ mask,
                                                       const int32_t* __restrict__ prefix,
                                                       const int32_t* __restrict__ offsets,
                                                       int32_t* __restrict__ tok_offsets, int32_t* __restrict__ tok_count,
                                                       int32_t* __restrict__ tok_rows, int32_t* __restrict__ row_token,
                                                       int32_t* __restrict__ row_expert, float* __restrict__ row_w, int T,
                                                       int K, int W, int32_t* __restrict__ status) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  const int w = t >> 6, b = t & 63;
  const uint64_t below = b ? (~0ull >> (64 - b)) : 0ull;
  int ex[16];
  float wt[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    ex[k] = k < K ? topk_idx[(size_t)t * K + k] : 0x7fffffff;
    wt[k] = k < K ? topk_w[(size_t)t * K + k] : 0.f;
  }
  int last = -1;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    if (r < K) {
      int e = 0x7fffffff;
      float wv = 0.f;
#pragma unroll
      for (int k = 0; k < 16; ++k)
        if (ex[k] > last && ex[k] < e) {
          e = ex[k];
          wv = wt[k];
        }
      last = e;
      if (e == 0x7fffffff) {
        // Fewer than K distinct experts in topk_idx (never from moe_route's
        // top-K).  The mask then holds fewer rows than T*K: flag the routing
        // as invalid and point the token's remaining slots at row 0, so a
        // later kernel that ignores the flag still reads in bounds.
        atomicOr(status, MOE_STATUS_DUPLICATE_EXPERT);
        tok_rows[(size_t)t * K + r] = 0;
        continue;
      }
      const int row = expert_row(mask, prefix, offsets, e, W, w, below);
      tok_rows[(size_t)t * K + r] = row;
      row_token[row] = t;
      row_expert[row] = e;
      row_w[row] = wv;
    }
  }
  tok_offsets[t] = t * K;
  tok_count[t] = K;
  if (t == T - 1) tok_offsets[T] = T * K;
}

// 64-bit value of lane (lane ^ s), and of lane src (any per-lane index).
__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int s) {
  const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, s, kWave);
  const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), s, kWave);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src, kWave);
  const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), src, kWave);
  return ((uint64_t)hi << 32) | lo;
}
// 64 x 64 bit transpose across a wave: lane i holds row i on entry; on exit
// lane j holds column j (bit i of lane j's result = bit j of lane i's input).
// Six butterfly stages, each exchanging the off-diagonal s x s blocks of
// every 2s x 2s block between lanes i and i ^ s.
__device__ __forceinline__ uint64_t wave_transpose64(uint64_t x, int lane) {
  constexpr uint64_t kLow[6] = {0x00000000FFFFFFFFull, 0x0000FFFF0000FFFFull, 0x00FF00FF00FF00FFull,
                                0x0F0F0F0F0F0F0F0Full, 0x3333333333333333ull, 0x5555555555555555ull};
#pragma unroll
  for (int k = 0; k < 6; ++k) {
    const int s = 32 >> k;
    const uint64_t m = kLow[k];  // bit positions j with (j & s) == 0
    const uint64_t y = shfl_xor_u64(x, s);
    x = (lane & s) ? (((y >> s) & m) | (x & ~m)) : ((x & m) | ((y & m) << s));
  }
  return x;
}

// General placement (any membership, e.g. after token rounding), one wave per
// 64-token word.  Pass 1: per-token expert count and renormalisation
// denominator (selected scores summed in ascending expert order, fp32).
// The wave loads the mask words of 64 experts (lane i: expert c0 + i) and
// transposes them, so that lane l holds token l's membership bits of those
// experts; it then walks its own set bits, lowest expert first, issuing the
// score loads of kMetaBatch experts before summing them.
constexpr int kMetaBatch = 8;
constexpr int kMetaChunks = 4;  // 64-expert chunks whose mask words are loaded together

__global__ __launch_bounds__(64) void token_count_kernel(const uint64_t* __restrict__ mask,
                                                         const float* __restrict__ scores_t, int32_t* __restrict__ cnt,
                                                         float* __restrict__ denom, int32_t* __restrict__ word_sum,
                                                         const int32_t* __restrict__ counts,
                                                         int32_t* __restrict__ offsets, int T, int E, int W,
                                                         int32_t* __restrict__ status) {
  const int w = blockIdx.x;
  const int lane = lane_id();
  if (w == W) {
    if (lane == 0) *status = 0;  // membership from the bitmap: always consistent
    // the extra workgroup: offsets = exclusive scan of the expert counts
    int running = 0;
    for (int e0 = 0; e0 < E; e0 += 64) {
      const int v = e0 + lane < E ? counts[e0 + lane] : 0;
      const int inc = wave_incl_scan(v);
      if (e0 + lane < E) offsets[e0 + lane] = running + inc - v;
      running += __shfl(inc, 63, kWave);
    }
    if (lane == 0) offsets[E] = running;
    return;
  }
  const int t = w * 64 + lane;
  const bool live = t < T;
  int c = 0;
  float s = 0.f;
  for (int cb = 0; cb < E; cb += 64 * kMetaChunks) {
    uint64_t words[kMetaChunks];
#pragma unroll
    for (int h = 0; h < kMetaChunks; ++h) {
      const int e = cb + 64 * h + lane;
      words[h] = e < E ? mask[(size_t)e * W + w] : 0ull;
    }
#pragma unroll
    for (int h = 0; h < kMetaChunks; ++h) {
      const int c0 = cb + 64 * h;
      if (c0 >= E) break;
      uint64_t bits = wave_transpose64(words[h], lane);
      if (!live) bits = 0;
      c += __popcll(bits);
      while (__ballot(bits != 0)) {
        float v[kMetaBatch];
#pragma unroll
        for (int u = 0; u < kMetaBatch; ++u) {
          const bool has = bits != 0;
          const int i = has ? __ffsll((unsigned long long)bits) - 1 : 0;
          v[u] = has ? scores_t[(size_t)(c0 + i) * T + t] : 0.f;
          bits &= bits - 1;
        }
        // adding +0 for a miss leaves the sum unchanged (it is never -0)
#pragma unroll
        for (int u = 0; u < kMetaBatch; ++u) s += v[u];
      }
    }
  }
  if (live) {
    cnt[t] = c;
    denom[t] = s;
  }
  const int total = wave_sum(live ? c : 0);
  if (lane == 0) word_sum[w] = total;  // rows of the word's 64 tokens
}

// Pass 2: rows of every token (expert ascending), renormalised weights.  The
// kPlaceWaves waves of a workgroup share one word: wave q places experts
// [q*Ew, (q+1)*Ew); it first counts its experts per token, and the counts of
// the lower ranges (exchanged through LDS) give each token's first slot.  As
// in pass 1, each lane walks its own token's set bits (from the transposed
// mask words); the expert's mask word and row base come from the lane that
// loaded them.
constexpr int kPlaceWaves = 4;
constexpr int kPlaceSumWords = 4096;  // T <= 262144

__global__ __launch_bounds__(64 * kPlaceWaves) void token_place_kernel(
    const uint64_t* __restrict__ mask, const int32_t* __restrict__ prefix, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ tok_count, const int32_t* __restrict__ word_base,
    const int32_t* __restrict__ word_sum, int32_t* __restrict__ tok_offsets,
    const float* __restrict__ scores_t, const float* __restrict__ denom, int32_t* __restrict__ tok_rows,
    int32_t* __restrict__ row_token, int32_t* __restrict__ row_expert, float* __restrict__ row_w, int T, int E,
    int W) {
  __shared__ int cnt[kPlaceWaves][64];
  const int w = blockIdx.x;
  const int lane = lane_id();
  const int q = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int t = w * 64 + lane;
  const bool live = t < T;
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  const int ew = (E + kPlaceWaves - 1) / kPlaceWaves;
  const int e_lo = min(E, q * ew), e_hi = min(E, e_lo + ew);
  // independent loads first: they overlap the count pass and the barrier
  const int ct = live ? tok_count[t] : 0;
  const float dn = live ? denom[t] : 1.f;
  // the first chunk's words and row bases stay in registers for pass 2
  const int el0 = e_lo + lane;
  const uint64_t words0 = el0 < e_hi ? mask[(size_t)el0 * W + w] : 0ull;
  const int bases0 = el0 < e_hi ? offsets[el0] + prefix[(size_t)el0 * W + w] : 0;
  uint64_t bits0 = wave_transpose64(words0, lane);
  if (!live) bits0 = 0;
  int c = __popcll(bits0);
  for (int c0 = e_lo + 64; c0 < e_hi; c0 += 64) {
    const int el = c0 + lane;
    const uint64_t words = el < e_hi ? mask[(size_t)el * W + w] : 0ull;
    const uint64_t bits = wave_transpose64(words, lane);
    c += live ? __popcll(bits) : 0;
  }
  cnt[q][lane] = c;
  // the word's base: given (word_base), or summed here from the word sums
  __shared__ int wsum[kPlaceWaves];
  int base;
  if (word_base) {
    base = word_base[w];
  } else {
    int part = 0;
    for (int i = threadIdx.x; i < w; i += 64 * kPlaceWaves) part += word_sum[i];
    part = wave_sum(part);
    if (lane == 0) wsum[q] = part;
  }
  __syncthreads();
  if (!word_base) {
    base = 0;
#pragma unroll
    for (int p = 0; p < kPlaceWaves; ++p) base += wsum[p];
  }
  // token t's first row: the word's base plus the rows of the word's earlier
  // tokens; wave 0 also writes tok_offsets
  const int tok_first = base + wave_incl_scan(ct) - ct;
  if (q == 0) {
    if (live) tok_offsets[t] = tok_first;
    if (w == W - 1 && lane == 63) tok_offsets[T] = tok_first + ct;
  }
  int j = tok_first;
  for (int p = 0; p < q; ++p) j += cnt[p][lane];
  for (int c0 = e_lo; c0 < e_hi; c0 += 64) {
    uint64_t words = words0, bits = bits0;
    int bases = bases0;
    if (c0 != e_lo) {
      const int el = c0 + lane;
      words = el < e_hi ? mask[(size_t)el * W + w] : 0ull;
      bases = el < e_hi ? offsets[el] + prefix[(size_t)el * W + w] : 0;
      bits = wave_transpose64(words, lane);
      if (!live) bits = 0;
    }
    while (__ballot(bits != 0)) {
      float v[kMetaBatch];
      int r[kMetaBatch], ex[kMetaBatch];
      bool hit[kMetaBatch];
#pragma unroll
      for (int u = 0; u < kMetaBatch; ++u) {
        hit[u] = bits != 0;
        const int i = hit[u] ? __ffsll((unsigned long long)bits) - 1 : 0;
        bits &= bits - 1;
        const uint64_t word = shfl_u64(words, i);  // expert c0 + i's mask word
        r[u] = __shfl(bases, i, kWave) + __popcll(word & below);
        ex[u] = c0 + i;
        v[u] = hit[u] ? scores_t[(size_t)(c0 + i) * T + t] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kMetaBatch; ++u) {
        if (hit[u]) {
          tok_rows[j++] = r[u];
          row_token[r[u]] = t;
          row_expert[r[u]] = ex[u];
          row_w[r[u]] = v[u] / dn;
        }
      }
    }
  }
}

// ---------------------------------------------------------------- launchers

static size_t topk_lds_bytes(int E, int K, bool stash) {
  return ((E * 8 + 15) & ~15) + (stash ? (size_t)E * kStashPitch * 4 + 64 * (size_t)K * 8 : 0);
}

hipError_t launch_topk_route(const float* in, float* scores, float* scores_t, int32_t* topk_idx, float* topk_w,
                             uint64_t* mask, int T, int E, int K, int W, int do_softmax, hipStream_t s) {
  if (E % 4 == 0 && E <= 256 && K <= 16 && K <= E) {
    // LDS beyond the default 64 KB of dynamic LDS is granted per kernel
#define SMOE_TOPK_LANE(KM, NW)                                                                                    \
  do {                                                                                                            \
    const size_t lds = topk_lane_lds(E, KM, NW);                                                                  \
    if (lds > 65536) {                                                                                            \
      const hipError_t e = hipFuncSetAttribute((const void*)topk_lane_kernel<KM, NW>,                             \
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);            \
      if (e != hipSuccess) return e;                                                                              \
    }                                                                                                             \
    topk_lane_kernel<KM, NW><<<dim3(W), dim3(64 * NW), lds, s>>>(in, scores, scores_t, topk_idx, topk_w, mask, T, \
                                                                 E, K, W, do_softmax);                            \
  } while (0)
    // four waves per word when the experts split into four slices of whole float4s
    const bool four = E % 16 == 0;
    if (K <= 2) {
      if (four) SMOE_TOPK_LANE(2, 4); else SMOE_TOPK_LANE(2, 1);
    } else if (K <= 4) {
      if (four) SMOE_TOPK_LANE(4, 4); else SMOE_TOPK_LANE(4, 1);
    } else if (K <= 8) {
      if (four) SMOE_TOPK_LANE(8, 4); else SMOE_TOPK_LANE(8, 1);
    } else {
      if (four) SMOE_TOPK_LANE(16, 4); else SMOE_TOPK_LANE(16, 1);
    }
#undef SMOE_TOPK_LANE
    return hipGetLastError();
  }
  const dim3 grid(W), block(kTopkWaves * 64);
  const int epl = (E + 63) / 64;
  // the stash must fit the default 64 KB of dynamic LDS
  const bool stash = topk_lds_bytes(E, K, true) <= 65536;
#define SMOE_TOPK(N)                                                                                               \
  if (epl <= N) {                                                                                                  \
    if (stash)                                                                                                     \
      topk_route_kernel<N, true><<<grid, block, topk_lds_bytes(E, K, true), s>>>(in, scores, scores_t, topk_idx,      \
                                                                               topk_w, mask, T, E, K, W, do_softmax); \
    else                                                                                                           \
      topk_route_kernel<N, false><<<grid, block, topk_lds_bytes(E, K, false), s>>>(in, scores, scores_t, topk_idx,    \
                                                                                 topk_w, mask, T, E, K, W, do_softmax); \
    return hipGetLastError();                                                                                      \
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

hipError_t launch_tc_metadata(const moe_routing& r, int T, int E, int K, bool counts_only, hipStream_t s) {
  const int W = r.words;
  expert_scan_kernel<<<dim3(E), dim3(256), 0, s>>>(r.mask, r.mask_prefix, r.counts, W);
  if (counts_only) return hipGetLastError();
  scan_kernel<<<dim3(1), dim3(1024), 0, s>>>(r.counts, r.offsets, E, r.status);
  tc_place_kernel<<<dim3((T + 255) / 256), dim3(256), 0, s>>>(r.topk_idx, r.topk_w, r.mask, r.mask_prefix, r.offsets,
                                                              r.tok_offsets, r.tok_count, r.tok_rows, r.row_token,
                                                              r.row_expert, r.row_w, T, K, W, r.status);
  return hipGetLastError();
}

hipError_t launch_metadata(const moe_routing& r, const float* scores_t, int T, int E, bool counted, hipStream_t s) {
  const int W = r.words;
  int32_t* word_sum = r.scratch + E + 64;  // [W]
  int32_t* word_base = word_sum + W + 1;   // [W + 1]
  if (!counted) expert_scan_kernel<<<dim3(E), dim3(256), 0, s>>>(r.mask, r.mask_prefix, r.counts, W);
  // one extra workgroup turns the expert counts into offsets
  token_count_kernel<<<dim3(W + 1), dim3(64), 0, s>>>(r.mask, scores_t, r.tok_count, r.tok_denom, word_sum, r.counts,
                                                      r.offsets, T, E, W, r.status);
  // up to kPlaceSumWords words every placement workgroup sums the word sums
  // before it itself; beyond that a scan kernel provides the bases
  const bool scan_words = W > kPlaceSumWords;
  if (scan_words) scan_kernel<<<dim3(1), dim3(1024), 0, s>>>(word_sum, word_base, W, nullptr);
  token_place_kernel<<<dim3(W), dim3(64 * kPlaceWaves), 0, s>>>(r.mask, r.mask_prefix, r.offsets, r.tok_count,
                                                                scan_words ? word_base : nullptr, word_sum,
                                                                r.tok_offsets, scores_t, r.tok_denom, r.tok_rows,
                                                                r.row_token, r.row_expert, r.row_w, T, E, W);
  return hipGetLastError();
}

}  // namespace smoe
