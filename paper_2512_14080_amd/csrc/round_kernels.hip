// Token rounding (Section 5.2): per-expert rounding decision and the
// selection of the dropped TC tokens or the padded non-TC tokens.
//
// The paper describes the method as a two-step sort (TC top-K, then a sort of
// each expert's tokens by router score with TC tokens preferred).  Only the
// last tile changes, so instead of sorting all T tokens per expert this code
// selects the at most m_tile-1 tokens that change with a bitwise select on an
// order-preserving integer image of the fp32 score, ties on the threshold
// value broken by token index.  The result is the same set the full sort
// would give.  The select runs in levels: per 2048-token chunk, then over
// the chunks' picks.
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

// ------------------------------------------------ selection in levels
// The need largest candidate keys of an expert, with ties on the key broken by
// token (low first for pads, high first for drops), form a strict total order
// on the candidates.  Under a strict order the global top-need set lies in the
// union of the top-need sets of any partition of the candidates: an element of
// the global set outranks all but fewer than need candidates, so also within
// its own part.  Level 1 gives every kTrChunk tokens of an expert one wave,
// which selects its chunk's top-need with wave reductions only (no workgroup
// barrier) and lists the chosen (key, token) pairs in token order, M entries
// per chunk.  While an expert's lists hold more than kTrMergeMax entries, a
// reduce level selects again per kTrChunk entries (positions keep token
// order).  The final level selects the top-need of the remaining entries per
// expert with one wave and writes the rounded mask row, its word prefixes and
// the count.  The selection work of an expert is spread over T / kTrChunk
// waves instead of one CU.
constexpr int kTrChunk = 2048;     // tokens (or list entries) per wave: 32 slots x 64 lanes
constexpr int kTrMergeMax = 4096;  // list entries the final wave holds (64 slots per lane)
constexpr int kTrRowWords = 1024;  // mask words per pass of the final level's LDS row

// entries of an expert's lists after a level that starts from n entries
__host__ __device__ inline int64_t tr_level_entries(int64_t n, int M) { return (n + kTrChunk - 1) / kTrChunk * M; }

// List space: two alternating list buffers sized for m_tile = 256 (level 1
// lists in the first, the first reduce level's in the second).
size_t round_scratch_bytes(int T, int E) {
  const int64_t l1 = tr_level_entries(T, 256), l2 = tr_level_entries(l1, 256);
  return (size_t)E * (size_t)(l1 + l2) * 8;
}

// Packed digit counts of a pass: each lane holds three 10-bit counts; the
// sum over a group of 16 / G lanes stays below 1024 per field (at most
// 32 G keys per lane).  DPP adds form the group sums in every lane; the
// groups' sums are read out and added per field on the scalar unit.
template <int G>
__device__ __forceinline__ void wave_counts3(uint32_t x, int* f0, int* f1, int* f2) {
  auto add = [](uint32_t a, uint32_t b) { return a + b; };
  x = add(x, dpp_mov<0xB1, 0xf>(x));  // quad_perm [1,0,3,2]
  x = add(x, dpp_mov<0x4E, 0xf>(x));  // quad_perm [2,3,0,1]
  x = add(x, dpp_mov<0x141, 0xf>(x));  // row_half_mirror: 8-lane sums
  if constexpr (G == 1) x = add(x, dpp_mov<0x140, 0xf>(x));  // row_mirror: 16-lane sums
  constexpr int kStep = 16 / G;
  int a = 0, b = 0, c = 0;
#pragma unroll
  for (int l = 0; l < 64; l += kStep) {
    const uint32_t v = (uint32_t)__builtin_amdgcn_readlane((int)x, l);
    a += (int)(v & 1023u);
    b += (int)((v >> 10) & 1023u);
    c += (int)(v >> 20);
  }
  *f0 = a;
  *f1 = b;
  *f2 = c;
}

// Wave-local selection of the `need` largest candidate keys.  Key (g, i) of
// lane l sits at position p = (32 g + i) * 64 + l; ties on the key go to the
// lower positions first when low_first, else to the higher ones.  cm[g] bit i
// marks a candidate; keys[g][i] is its key (destroyed: the keys become bit
// planes).  Returns the selected candidates as sel[g] bits.
//
// Bitwise select over the planes, two bits per pass, MSB first: `alive`
// holds the candidates that still match the selected prefix, `taken` those
// already known to be selected (a higher digit at some pass).  Once the alive
// keys are exactly as many as are still to take, all of them are taken and
// the remaining bits are not looked at.
template <int G>
__device__ __forceinline__ void wave_select(uint32_t (&keys)[G][32], const uint32_t (&cm)[G], int need,
                                            bool low_first, uint32_t (&sel)[G]) {
  uint32_t c = 0;
#pragma unroll
  for (int g = 0; g < G; ++g) c += (uint32_t)__popc(cm[g]);
  int nalive, unused0, unused1;
  wave_counts3<G>(c, &nalive, &unused0, &unused1);
  if (nalive <= need) {
#pragma unroll
    for (int g = 0; g < G; ++g) sel[g] = cm[g];
    return;
  }
#pragma unroll
  for (int g = 0; g < G; ++g) transpose32(keys[g]);  // keys[g][b] bit i = bit b of key i
  uint32_t alive[G], taken[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    alive[g] = cm[g];
    taken[g] = 0u;
  }
  int remaining = need;
#pragma unroll
  for (int sh = 30; sh >= 0; sh -= 2) {
    uint32_t a3[G], a2[G], a1[G], cnt = 0;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint32_t hi = keys[g][sh + 1], lo = keys[g][sh];
      a3[g] = alive[g] & hi & lo;
      a2[g] = alive[g] & hi & ~lo;
      a1[g] = alive[g] & ~hi & lo;
      cnt += (uint32_t)__popc(a3[g]) | ((uint32_t)__popc(a2[g]) << 10) | ((uint32_t)__popc(a1[g]) << 20);
    }
    int t3, t2, t1;
    wave_counts3<G>(cnt, &t3, &t2, &t1);
    if (t3 >= remaining) {
      nalive = t3;
#pragma unroll
      for (int g = 0; g < G; ++g) alive[g] = a3[g];
    } else if (t3 + t2 >= remaining) {
      remaining -= t3;
      nalive = t2;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        taken[g] |= a3[g];
        alive[g] = a2[g];
      }
    } else if (t3 + t2 + t1 >= remaining) {
      remaining -= t3 + t2;
      nalive = t1;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        taken[g] |= a3[g] | a2[g];
        alive[g] = a1[g];
      }
    } else {
      remaining -= t3 + t2 + t1;
      nalive -= t3 + t2 + t1;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        taken[g] |= a3[g] | a2[g] | a1[g];
        alive[g] &= ~(a3[g] | a2[g] | a1[g]);
      }
    }
    if (nalive == remaining) break;
  }
  if (nalive == remaining) {
#pragma unroll
    for (int g = 0; g < G; ++g) sel[g] = taken[g] | alive[g];
    return;
  }
  // every bit decided: alive holds the nalive keys equal to the threshold,
  // of which `remaining` are taken by position.  A tie's rank: the ties of
  // the earlier slots, then of the lower lanes of its own slot.
  const int lo_rank = low_first ? 0 : nalive - remaining, hi_rank = low_first ? remaining : nalive;
  int base = 0;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    uint32_t take = 0;
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const bool tie = (alive[g] >> i) & 1u;
      const uint64_t b = __ballot(tie);
      const int rank = base + __popcll(b & lanemask_lt());
      take |= (uint32_t)(tie && rank >= lo_rank && rank < hi_rank) << i;
      base += __popcll(b);
    }
    sel[g] = taken[g] | take;
  }
}

// The rounding decision of expert e (both levels take it the same way).
__device__ __forceinline__ void tr_decision(int e, const int32_t* round_dir, const int32_t* need_arr,
                                            const int32_t* counts, const float* u, int T, int M, int mode, int* dir,
                                            int* need) {
  if (need_arr) {
    *dir = round_dir[e];
    *need = need_arr[e];
  } else {
    tr_decide_one(counts[e], mode == MOE_ROUND_STOCHASTIC ? u[e] : 0.f, T, M, mode, dir, need);
  }
}

// Level 1: wave (e, c) selects the top-need candidates among tokens
// [c * kTrChunk, (c + 1) * kTrChunk) of expert e and writes the M list
// entries of its chunk at list[(e * nch + c) * M]: the chosen ones in token
// order as (key << 32) | (token << 1) | 1, then zeros (entry bit 0 marks a
// pick).  Token 64 i + l of the chunk is slot i of lane l (slot i is mask
// word 32 c + i).
__global__ __launch_bounds__(256) void tr_local_kernel(const uint64_t* __restrict__ tc_mask,
                                                       const float* __restrict__ scores_t,
                                                       const int32_t* __restrict__ round_dir,
                                                       const int32_t* __restrict__ need_arr,
                                                       const int32_t* __restrict__ counts, const float* __restrict__ u,
                                                       int M, int mode, int T, int E, int W, int nch,
                                                       uint64_t* __restrict__ list) {
  const int gw = __builtin_amdgcn_readfirstlane((int)(blockIdx.x * 4 + (threadIdx.x >> 6)));
  const int e = gw / nch, c = gw - e * nch;
  if (e >= E) return;
  int dir, need;
  tr_decision(e, round_dir, need_arr, counts, u, T, M, mode, &dir, &need);
  if (dir == 0 || need == 0) return;  // level 2 reads no list for this expert
  const int lane = lane_id();
  const bool want_set = dir < 0;  // candidates: TC tokens for drops, non-TC for pads
  const float* S = scores_t + (size_t)e * T;
  const uint64_t* src = tc_mask + (size_t)e * W;
  uint32_t keys[1][32];
  uint64_t words[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const int t = c * kTrChunk + 64 * i + lane;
    const int w = c * 32 + i;  // wave-uniform: a scalar load
    words[i] = w < W ? src[w] : 0ull;
    keys[0][i] = t < T ? __float_as_uint(S[t]) : 0u;
  }
  uint32_t cm[1] = {0u}, kept[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const int t = c * kTrChunk + 64 * i + lane;
    const bool cnd = t < T && ((((words[i] >> lane) & 1ull) != 0) == want_set);
    const uint32_t k = score_key(__uint_as_float(keys[0][i]));
    keys[0][i] = kept[i] = cnd ? (dir < 0 ? ~k : k) : 0u;
    cm[0] |= (uint32_t)cnd << i;
  }
  uint32_t sel[1];
  wave_select<1>(keys, cm, need, dir > 0, sel);
  uint64_t* out = list + (size_t)gw * M;
  int n = 0;
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const bool s = (sel[0] >> i) & 1u;
    const uint64_t b = __ballot(s);
    if (s)
      out[n + __popcll(b & lanemask_lt())] =
          ((uint64_t)kept[i] << 32) | ((uint32_t)(c * kTrChunk + 64 * i + lane) << 1) | 1u;
    n += __popcll(b);
  }
  for (int q = n + lane; q < M; q += 64) out[q] = 0ull;
}

// Reduce level: wave (e, c) selects the top-need entries among positions
// [c * kTrChunk, (c + 1) * kTrChunk) of expert e's nin input entries and
// writes M output entries at out[(e * ngroups + c) * M], in position order.
__global__ __launch_bounds__(256) void tr_reduce_kernel(const int32_t* __restrict__ round_dir,
                                                        const int32_t* __restrict__ need_arr,
                                                        const int32_t* __restrict__ counts,
                                                        const float* __restrict__ u, int M, int mode, int T, int E,
                                                        int64_t nin, int ngroups, const uint64_t* __restrict__ in,
                                                        uint64_t* __restrict__ out) {
  const int gw = __builtin_amdgcn_readfirstlane((int)(blockIdx.x * 4 + (threadIdx.x >> 6)));
  const int e = gw / ngroups, c = gw - e * ngroups;
  if (e >= E) return;
  int dir, need;
  tr_decision(e, round_dir, need_arr, counts, u, T, M, mode, &dir, &need);
  if (dir == 0 || need == 0) return;
  const int lane = lane_id();
  const uint64_t* lst = in + (size_t)e * nin;
  uint32_t keys[1][32], cm[1] = {0u};
  uint64_t ent[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const int64_t p = (int64_t)c * kTrChunk + 64 * i + lane;
    ent[i] = p < nin ? lst[p] : 0ull;
    keys[0][i] = (uint32_t)(ent[i] >> 32);
    cm[0] |= (uint32_t)(ent[i] & 1u) << i;
  }
  uint32_t sel[1];
  wave_select<1>(keys, cm, need, dir > 0, sel);
  uint64_t* o = out + (size_t)gw * M;
  int n = 0;
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const bool s = (sel[0] >> i) & 1u;
    const uint64_t b = __ballot(s);
    if (s) o[n + __popcll(b & lanemask_lt())] = ent[i];
    n += __popcll(b);
  }
  for (int q = n + lane; q < M; q += 64) o[q] = 0ull;
}

// Final level, one workgroup of 4 waves per expert.  Wave 0 selects the
// top-need of the expert's nin <= 64 * 32 G remaining entries (position order
// is token order); then the TC mask row is copied through LDS kTrRowWords
// words at a time, the chosen tokens' bits are flipped there, and the rounded
// row goes out with its word prefixes and count.
template <int G>
__global__ __launch_bounds__(256) void tr_merge_kernel(const uint64_t* __restrict__ tc_mask,
                                                       uint64_t* __restrict__ tr_mask,
                                                       int32_t* __restrict__ round_dir,
                                                       const int32_t* __restrict__ need_arr,
                                                       const int32_t* __restrict__ counts, const float* __restrict__ u,
                                                       int M, int mode, int T, int W, int nin,
                                                       const uint64_t* __restrict__ list,
                                                       int32_t* __restrict__ prefix_out,
                                                       int32_t* __restrict__ counts_out) {
  __shared__ uint64_t row[kTrRowWords];
  __shared__ int scan_lds[4];
  const int e = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = lane_id();
  int dir, need;
  tr_decision(e, round_dir, need_arr, counts, u, T, M, mode, &dir, &need);
  if (!need_arr && threadIdx.x == 0) round_dir[e] = dir;
  const uint64_t* src = tc_mask + (size_t)e * W;
  uint64_t* dst = tr_mask + (size_t)e * W;
  const bool select = dir != 0 && need != 0;
  // the first pass's row words are requested before the selection, so that
  // their loads overlap it (wave 0's otherwise wait until it has selected)
  constexpr int kPre = kTrRowWords / 256;
  uint64_t pre[kPre];
  {
    const int nw0 = min(kTrRowWords, W);
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      const int w = threadIdx.x + 256 * i;
      pre[i] = w < nw0 ? src[w] : 0ull;
    }
  }
  uint32_t sel[G];
  int tok[G][32];
  if (select && wave == 0) {
    const uint64_t* lst = list + (size_t)e * nin;
    uint32_t keys[G][32], cm[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      cm[g] = 0u;
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        const int p = (32 * g + i) * 64 + lane;
        const uint64_t v = p < nin ? lst[p] : 0ull;
        tok[g][i] = (int)((uint32_t)v >> 1);
        keys[g][i] = (uint32_t)(v >> 32);
        cm[g] |= (uint32_t)(v & 1u) << i;
      }
    }
    wave_select<G>(keys, cm, need, dir > 0, sel);
  }
  int carry = 0;
  for (int w0 = 0; w0 < W; w0 += kTrRowWords) {
    const int nw = min(kTrRowWords, W - w0);
    if (w0 == 0) {
#pragma unroll
      for (int i = 0; i < kPre; ++i)
        if (threadIdx.x + 256 * i < nw) row[threadIdx.x + 256 * i] = pre[i];
    } else {
      for (int w = threadIdx.x; w < nw; w += 256) row[w] = src[w0 + w];
    }
    __syncthreads();
    if (select && wave == 0) {
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int i = 0; i < 32; ++i) {
          const int w = (tok[g][i] >> 6) - w0;
          if (((sel[g] >> i) & 1u) && w >= 0 && w < nw)
            atomicXor((unsigned long long*)&row[w], 1ull << (tok[g][i] & 63));
        }
    }
    __syncthreads();
    // four consecutive words per thread
    const int q0 = 4 * threadIdx.x;
    int pc[4], sum = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint64_t v = q0 + k < nw ? row[q0 + k] : 0ull;
      if (q0 + k < nw) dst[w0 + q0 + k] = v;
      pc[k] = __popcll(v);
      sum += pc[k];
    }
    int total;
    int ex = carry + block_excl_scan<256>(sum, &total, scan_lds);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (q0 + k < nw) prefix_out[(size_t)e * W + w0 + q0 + k] = ex;
      ex += pc[k];
    }
    carry += total;  // block_excl_scan ends with a barrier: row may be refilled
  }
  if (threadIdx.x == 0) counts_out[e] = carry;
}

hipError_t launch_round(const moe_routing& tc, moe_routing& tr, const float* u, int T, int E, int M, int mode,
                        uint64_t* list, bool* counted, hipStream_t s) {
  // Balance-f is sequential over experts: its own pass decides; the other
  // subroutines are decided inside the selection workgroups
  int32_t* need = nullptr;
  if (mode == MOE_ROUND_BALANCE) {
    need = tr.scratch;
    tr_decide_kernel<<<dim3(1), dim3(256), 0, s>>>(tc.counts, u, tr.round_dir, need, T, E, M, mode);
  }
  if (list == nullptr) return hipErrorInvalidValue;
  const int nch = (T + kTrChunk - 1) / kTrChunk;
  tr_local_kernel<<<dim3(((int64_t)E * nch + 3) / 4), dim3(256), 0, s>>>(tc.mask, tc.scores_t, tr.round_dir, need,
                                                                         tc.counts, u, M, mode, T, E, tr.words, nch,
                                                                         list);
  // reduce levels while the lists exceed what the final wave holds; the
  // lists alternate between the two buffers
  uint64_t* buf[2] = {list, list + (size_t)E * tr_level_entries(T, 256)};
  int cur = 0;
  int64_t nin = (int64_t)nch * M;
  while (nin > kTrMergeMax) {
    const int ngroups = (int)((nin + kTrChunk - 1) / kTrChunk);
    tr_reduce_kernel<<<dim3(((int64_t)E * ngroups + 3) / 4), dim3(256), 0, s>>>(tr.round_dir, need, tc.counts, u, M,
                                                                                mode, T, E, nin, ngroups, buf[cur],
                                                                                buf[cur ^ 1]);
    cur ^= 1;
    nin = (int64_t)ngroups * M;
  }
  if (nin <= kTrMergeMax / 2)
    tr_merge_kernel<1><<<dim3(E), dim3(256), 0, s>>>(tc.mask, tr.mask, tr.round_dir, need, tc.counts, u, M, mode, T,
                                                     tr.words, (int)nin, buf[cur], tr.mask_prefix, tr.counts);
  else
    tr_merge_kernel<2><<<dim3(E), dim3(256), 0, s>>>(tc.mask, tr.mask, tr.round_dir, need, tc.counts, u, M, mode, T,
                                                     tr.words, (int)nin, buf[cur], tr.mask_prefix, tr.counts);
  *counted = true;
  return hipGetLastError();
}

}  // namespace smoe
