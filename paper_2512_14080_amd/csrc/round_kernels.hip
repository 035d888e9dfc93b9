// Token rounding (Section 5.2): per-expert rounding decision and the
// selection of the dropped TC tokens or the padded non-TC tokens.
//
// The paper describes the method as a two-step sort (TC top-K, then a sort of
// each expert's tokens by router score with TC tokens preferred).  Only the
// last tile changes, so instead of sorting all T tokens per expert this code
// selects the at most m_tile-1 tokens that change with a bitwise (32-pass)
// select on an order-preserving integer image of the fp32 score, then breaks
// ties on the threshold value by token index.  The result is the same set the
// full sort would give.
#include "device_common.h"
#include "launch.h"

namespace smoe {

// The per-expert rounding decision of the independent subroutines (all but
// Balance-f): direction of f^TR_e - f_e and its size.
__device__ __forceinline__ void tr_decide_one(int f, float u_e, int T, int M, int mode, int* dir, int* need) {
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
    pad = (u_e * (float)M) < (float)(f - lo);
  pad = pad && (hi <= T);
  const int ftr = pad ? hi : lo;
  *dir = ftr > f ? 1 : (ftr < f ? -1 : 0);
  *need = ftr > f ? ftr - f : f - ftr;
}

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
    int dir, nd;
    tr_decide_one(counts[e], mode == MOE_ROUND_STOCHASTIC ? u[e] : 0.f, T, M, mode, &dir, &nd);
    round_dir[e] = dir;
    need[e] = nd;
  }
}

// order-preserving image of an fp32 score (+0 and -0 map to the same key)
__device__ __forceinline__ uint32_t score_key(float x) {
  uint32_t b = __float_as_uint(x);
  if (b == 0x80000000u) b = 0;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

constexpr int kSelThreads = 1024;

// 32 x 32 bit transpose in registers by recursive block swaps (the published
// bit-matrix transpose, H. S. Warren, "Hacker's Delight", section 7-3):
// afterwards A[b] bit i = bit b of the original A[i].
__device__ __forceinline__ void transpose32(uint32_t (&A)[32]) {
  uint32_t m = 0x0000FFFFu;
#pragma unroll
  for (int j = 16; j != 0; j >>= 1, m ^= m << j) {
#pragma unroll
    for (int k = 0; k < 32; k = (k + j + 1) & ~j) {
      const uint32_t t = ((A[k] >> j) ^ A[k + j]) & m;
      A[k + j] ^= t;
      A[k] ^= t << j;
    }
  }
}

// One block per expert.  Copies the TC mask row of expert e into the rounded
// mask and flips the `need` selected bits:
//   pad  (dir > 0): the need best non-TC tokens by (score desc, token asc);
//   drop (dir < 0): the need worst TC tokens by (score asc, token desc).
// Both become "the need largest keys" with key = score_key for pads and
// ~score_key for drops, ties preferring low tokens for pads, high for drops.
//
// Token t is owned by thread t % 1024 as its slot t / 1024.  With KPT > 0 the
// block holds all T <= 1024*KPT keys in registers (read once; KPT <= 32 keeps
// them within the 128 VGPRs a 1024-thread block allows); KPT == 0 is the
// any-T form that re-reads the scores from memory on every pass.
template <int KPT>
__global__ __launch_bounds__(kSelThreads) void tr_select_kernel(const uint64_t* __restrict__ tc_mask,
                                                                uint64_t* __restrict__ tr_mask,
                                                                const float* __restrict__ scores_t,
                                                                int32_t* __restrict__ round_dir,
                                                                const int32_t* __restrict__ need_arr,
                                                                const int32_t* __restrict__ counts,
                                                                const float* __restrict__ u, int M, int mode, int T,
                                                                int W, int32_t* __restrict__ prefix_out,
                                                                int32_t* __restrict__ counts_out) {
  constexpr int kWaves = kSelThreads / 64;
  __shared__ int lds[kWaves];
  __shared__ int cnt_lds[2][kWaves];  // per-wave counts of a pass, double-buffered by pass parity
  const int e = blockIdx.x;
  const uint64_t* src = tc_mask + (size_t)e * W;
  uint64_t* dst = tr_mask + (size_t)e * W;
  // the decision: taken here unless a Balance-f pass (sequential over
  // experts) made it already (need_arr non-null)
  int dir, need;
  if (need_arr) {
    dir = round_dir[e];
    need = need_arr[e];
  } else {
    tr_decide_one(counts[e], mode == MOE_ROUND_STOCHASTIC ? u[e] : 0.f, T, M, mode, &dir, &need);
    if (threadIdx.x == 0) round_dir[e] = dir;
  }
  // With KPT > 0 (W <= 16 * KPT <= 1024 words) the block also writes the
  // rounded row's word prefix counts and the expert's row count, which are
  // otherwise a pass of their own.
  auto write_prefix = [&](int pc) {
    int total;
    const int ex = block_excl_scan<kSelThreads>(pc, &total, lds);
    if ((int)threadIdx.x < W) prefix_out[(size_t)e * W + threadIdx.x] = ex;
    if (threadIdx.x == 0) counts_out[e] = total;
  };
  if (dir == 0 || need == 0) {
    if constexpr (KPT > 0) {
      const uint64_t v = (int)threadIdx.x < W ? src[threadIdx.x] : 0ull;
      if ((int)threadIdx.x < W) dst[threadIdx.x] = v;
      write_prefix(__popcll(v));
    } else {
      for (int w = threadIdx.x; w < W; w += kSelThreads) dst[w] = src[w];
    }
    return;
  }
  const float* S = scores_t + (size_t)e * T;
  const bool want_set = dir < 0;  // candidates: TC tokens for drops, non-TC for pads
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int slots = (T + kSelThreads - 1) / kSelThreads;

  // key of slot i of this thread; cand tells whether the token is a candidate
  auto load_key = [&](int i, bool& cand) -> uint32_t {
    const int t = i * kSelThreads + threadIdx.x;
    cand = false;
    if (t >= T) return 0u;
    cand = (((src[t >> 6] >> (t & 63)) & 1ull) != 0) == want_set;
    if (!cand) return 0u;
    const uint32_t k = score_key(S[t]);
    return dir < 0 ? ~k : k;
  };
  uint32_t keys[KPT > 0 ? KPT : 1];
  uint64_t cmask = 0;
  if constexpr (KPT > 0) {
    // scores and mask words are requested 16 slots at a time before any is used
    constexpr int kBatch = KPT < 16 ? KPT : 16;
#pragma unroll
    for (int i0 = 0; i0 < KPT; i0 += kBatch) {
      uint64_t words[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = i0 + u;
        const int t = i * kSelThreads + threadIdx.x;
        const int w = __builtin_amdgcn_readfirstlane(i * kWaves + wave);  // the wave's word: a scalar load
        keys[i] = t < T ? __float_as_uint(S[t]) : 0u;
        words[u] = w < W ? src[w] : 0ull;
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = i0 + u;
        const int t = i * kSelThreads + threadIdx.x;
        const bool c = t < T && ((((words[u] >> lane) & 1ull) != 0) == want_set);
        const uint32_t k = score_key(__uint_as_float(keys[i]));
        keys[i] = c ? (dir < 0 ? ~k : k) : 0u;
        cmask |= (uint64_t)c << i;
      }
      asm volatile("" ::: "memory");  // keep the next batch's loads after this one
    }
  }
  // number of candidates in the block whose key k has (k >> sh) == v.  One
  // barrier per call: the counts of consecutive calls go to alternating slots,
  // and a slot is only rewritten after the next call's barrier, which every
  // wave reaches after reading it.
  int parity = 0;
  auto count_eq = [&](uint32_t v, int sh) -> int {
    int cnt = 0;
    if constexpr (KPT > 0) {
#pragma unroll
      for (int i = 0; i < KPT; ++i) cnt += __popcll(__ballot(((cmask >> i) & 1ull) && (keys[i] >> sh) == v));
    } else {
      for (int i = 0; i < slots; ++i) {
        bool c;
        const uint32_t k = load_key(i, c);
        cnt += __popcll(__ballot(c && (k >> sh) == v));
      }
    }
    if (lane == 0) cnt_lds[parity][wave] = cnt;
    __syncthreads();
    int total = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) total += cnt_lds[parity][q];
    parity ^= 1;
    return total;
  };

  // Bitwise select (MSB first) of tau, the need-th largest candidate key:
  // keep a bit set when the candidates extending the prefix with a 1 still
  // hold `remaining` keys, else count them as taken and clear it.
  uint32_t prefix = 0;
  int remaining = need;
  int nties;
  uint32_t gt_mask = 0, tie_mask = 0;  // register form: candidates with key > tau / == tau
  if constexpr (KPT > 0) {
    // Register form: bit i of `alive` marks key i as a candidate that still
    // matches the prefix.  The keys are first transposed into bit planes
    // (plane[b] bit i = bit b of key i), so a pass costs a few mask
    // operations and popcounts per lane instead of a ballot per key.
    uint32_t alive = (uint32_t)cmask;
    uint32_t plane[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) plane[i] = i < KPT ? keys[i] : 0u;
    transpose32(plane);
    auto block_total = [&](int cnt) {
      if (lane == 0) cnt_lds[parity][wave] = cnt;
      __syncthreads();
      int total = 0;
#pragma unroll
      for (int q = 0; q < kWaves; ++q) total += cnt_lds[parity][q];
      parity ^= 1;
      return total;
    };
    auto wave_sum_u = [&](uint32_t x) { return dpp_reduce(x, [](uint32_t a, uint32_t b) { return a + b; }); };
    // two bits per pass: block counts of the alive keys whose next digit is
    // 3, 2 and 1 decide the digit of tau (16 passes, one barrier each)
    // per-wave counts of a pass: digit 1, and digits 3 (low half) and 2 (high
    // half) packed (block totals stay below 2^16), read back four waves at a time
    __shared__ __attribute__((aligned(16))) uint32_t cnt3_lds[2][2][kWaves];
#pragma unroll
    for (int sh = 30; sh >= 0; sh -= 2) {
      const uint32_t hi = plane[sh + 1], lo = plane[sh];
      const uint32_t a3 = alive & hi & lo, a2 = alive & hi & ~lo, a1 = alive & ~hi & lo;
      // per-wave counts (each <= 64 * 32): digits 3 and 2 share one word
      const uint32_t c32 = wave_sum_u((uint32_t)__popc(a3) | ((uint32_t)__popc(a2) << 16));
      const uint32_t c1 = wave_sum_u((uint32_t)__popc(a1));
      if (lane == 0) {
        cnt3_lds[parity][0][wave] = c1;
        cnt3_lds[parity][1][wave] = c32;
      }
      __syncthreads();
      uint32_t s1 = 0, s32 = 0;
#pragma unroll
      for (int q = 0; q < kWaves; q += 4) {
        const u32x4 x = *(const u32x4*)&cnt3_lds[parity][0][q];
        const u32x4 y = *(const u32x4*)&cnt3_lds[parity][1][q];
        s1 += (x[0] + x[1]) + (x[2] + x[3]);
        s32 += (y[0] + y[1]) + (y[2] + y[3]);
      }
      const int t1 = (int)s1, t2 = (int)(s32 >> 16), t3 = (int)(s32 & 0xffffu);
      parity ^= 1;
      if (t3 >= remaining) {
        prefix |= 3u << sh;
        alive = a3;
      } else if (t3 + t2 >= remaining) {
        prefix |= 2u << sh;
        remaining -= t3;
        alive = a2;
      } else if (t3 + t2 + t1 >= remaining) {
        prefix |= 1u << sh;
        remaining -= t3 + t2;
        alive = a1;
      } else {
        remaining -= t3 + t2 + t1;
        alive &= ~(hi | lo);
      }
    }
    // the survivors are exactly the candidate keys equal to tau
    nties = block_total((int)wave_sum_u((uint32_t)__popc(alive)));
    tie_mask = alive;
    // key > tau from the planes (most significant bit first, tau uniform)
    uint32_t eq = 0xffffffffu;
#pragma unroll
    for (int b = 31; b >= 0; --b) {
      const uint32_t tb = ((prefix >> b) & 1u) ? 0xffffffffu : 0u;
      gt_mask |= eq & plane[b] & ~tb;
      eq &= ~(plane[b] ^ tb);
    }
    gt_mask &= (uint32_t)cmask;
  } else {
    for (int bit = 31; bit >= 0; --bit) {
      const int total = count_eq((prefix >> bit) | 1u, bit);
      if (total >= remaining)
        prefix |= 1u << bit;
      else
        remaining -= total;
    }
    nties = count_eq(prefix, 0);
  }
  const uint32_t tau = prefix;

  // Marking pass in ascending token order: slot i of wave w is word 16i + w.
  // Every candidate with key > tau flips; of the nties ties on tau, the
  // `remaining` first ones flip for pads and the last ones for drops.  A
  // tie's ascending rank comes from ballots, a scan over the waves and a
  // carry over slots.
  const int first_tie = dir > 0 ? 0 : nties - remaining;
  const int last_tie = dir > 0 ? remaining : nties;  // flip ranks in [first_tie, last_tie)
  int carry = 0;
  auto mark = [&](int i, bool cand, uint32_t k) {
    const int w = i * kWaves + wave;
    const bool gt = cand && k > tau;
    const bool tie = cand && k == tau;
    const uint64_t ties = __ballot(tie);
    if (lane == 0) lds[wave] = __popcll(ties);
    __syncthreads();
    int base = carry, total = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) {
      const int c = lds[q];
      if (q < wave) base += c;
      total += c;
    }
    const int rank = base + __popcll(ties & lanemask_lt());
    const bool flip = gt || (tie && rank >= first_tie && rank < last_tie);
    const uint64_t flips = __ballot(flip);
    if (w < W && lane == 0) dst[w] = src[w] ^ flips;
    carry += total;
    __syncthreads();
  };
  if constexpr (KPT > 0) {
    // Register form: all tie counts first (flat index slot * waves + wave),
    // one block scan for every tie's rank base, then all flips.
    __shared__ int tie_base[KPT * kWaves];
    __shared__ int word_pc[KPT * kWaves];
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const uint64_t ties = __ballot((tie_mask >> i) & 1u);
      if (lane == 0) tie_base[i * kWaves + wave] = __popcll(ties);
    }
    __syncthreads();
    const int cnt = threadIdx.x < KPT * kWaves ? tie_base[threadIdx.x] : 0;
    int all_ties;
    const int ex = block_excl_scan<kSelThreads>(cnt, &all_ties, lds);
    if (threadIdx.x < KPT * kWaves) tie_base[threadIdx.x] = ex;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      if (i >= slots) break;
      const int w = i * kWaves + wave;
      const bool gt = (gt_mask >> i) & 1u;
      const bool tie = (tie_mask >> i) & 1u;
      const uint64_t ties = __ballot(tie);
      const int rank = tie_base[w] + __popcll(ties & lanemask_lt());
      const bool flip = gt || (tie && rank >= first_tie && rank < last_tie);
      const uint64_t flips = __ballot(flip);
      if (w < W && lane == 0) {
        const uint64_t v = src[w] ^ flips;
        dst[w] = v;
        word_pc[w] = __popcll(v);
      }
    }
    __syncthreads();
    write_prefix((int)threadIdx.x < W ? word_pc[threadIdx.x] : 0);
  } else {
    for (int i = 0; i < slots; ++i) {
      bool c;
      const uint32_t k = load_key(i, c);
      mark(i, c, k);
    }
  }
}

hipError_t launch_round(const moe_routing& tc, moe_routing& tr, const float* u, int T, int E, int M, int mode,
                        bool* counted, hipStream_t s) {
  // Balance-f is sequential over experts: its own pass decides; the other
  // subroutines are decided inside the selection workgroups
  int32_t* need = nullptr;
  if (mode == MOE_ROUND_BALANCE) {
    need = tr.scratch;
    tr_decide_kernel<<<dim3(1), dim3(256), 0, s>>>(tc.counts, u, tr.round_dir, need, T, E, M, mode);
  }
  const int slots = (T + kSelThreads - 1) / kSelThreads;
  auto select = [&](auto kernel) {
    kernel<<<dim3(E), dim3(kSelThreads), 0, s>>>(tc.mask, tr.mask, tc.scores_t, tr.round_dir, need, tc.counts, u, M,
                                                 mode, T, tr.words, tr.mask_prefix, tr.counts);
  };
  *counted = slots <= 32;
  if (slots <= 4)
    select(tr_select_kernel<4>);
  else if (slots <= 16)
    select(tr_select_kernel<16>);
  else if (slots <= 32)
    select(tr_select_kernel<32>);
  else
    select(tr_select_kernel<0>);
  return hipGetLastError();
}

}  // namespace smoe
