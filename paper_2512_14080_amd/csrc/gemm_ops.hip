// The eight GEMMs of the MoE layer on the shared grouped-GEMM core:
//   router     logits = X W_r (+ bias)                              (routing)
//   up         H = gather(X) W1_e, A = SwiGLU(H)      up-proj A kernel   (forward, Section 3)
//   down       Y = A W2_e                             down-proj Y kernel (forward)
//   dh         dA' = gather(dO) W2_e^T; dS, dH, A'    dH kernel          (down-proj backward)
//   dw2        dW2_e = A'^T gather(dO)   (varlen-K)   dW2 kernel         (down-proj backward)
//   dxt        dX~ = dH W1_e^T                        dX~ kernel         (up-proj backward, Appendix E)
//   dw1        dW1_e = gather(X)^T dH    (varlen-K)   dW1 kernel         (up-proj backward)
//   dwr        dW_r = X^T dL             (split-K)    router weight gradient
// varlen-M GEMMs schedule (expert, m-tile) pairs from the device-side expert
// offsets, so no host synchronisation is needed for the ragged row counts.
#include <algorithm>

#include "gemm_core.h"
#include "launch.h"
#include "topk_net.h"

namespace smoe {

__device__ __forceinline__ float silu_sig(float g, float* sig) {
  const float s = fast_sigmoid(g);
  *sig = s;
  return g * s;
}


// One 32-column accumulator block of a row, as bf16: v[g] holds columns
// 8g + 4*(lane/32) + [0, 4) (the MFMA output layout).  One lane-pair swap per
// dword (v_permlane32_swap exchanges the upper half of its first operand with
// the lower half of its second) leaves every lane with 8 consecutive
// columns, so each lane stores 16 bytes: lane < 32 columns 8g .. 8g+7 and
// lane >= 32 columns 8g+8 .. 8g+15, for g = 0, 2.
__device__ __forceinline__ void store_block_bf16(uint16_t* row_block, const u32x2 (&v)[4]) {
  const int hi = (threadIdx.x >> 5) & 1;
#pragma unroll
  for (int g = 0; g < 4; g += 2) {
    const auto a = __builtin_amdgcn_permlane32_swap(v[g][0], v[g + 1][0], false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(v[g][1], v[g + 1][1], false, false);
    *(u32x4*)(row_block + 8 * g + 8 * hi) = u32x4{a[0], b[0], a[1], b[1]};
  }
}

// The inverse: 16-byte loads of a 32-column block, returned in the
// accumulator layout of store_block_bf16 (the swap is its own inverse).
__device__ __forceinline__ void load_block_bf16(const uint16_t* row_block, u32x2 (&v)[4]) {
  const int hi = (threadIdx.x >> 5) & 1;
#pragma unroll
  for (int g = 0; g < 4; g += 2) {
    const u32x4 x = *(const u32x4*)(row_block + 8 * g + 8 * hi);
    const auto a = __builtin_amdgcn_permlane32_swap(x[0], x[2], false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(x[1], x[3], false, false);
    v[g] = u32x2{a[0], b[0]};
    v[g + 1] = u32x2{a[1], b[1]};
  }
}

__device__ __forceinline__ u32x2 pack_bf16x4(float a, float b, float c, float d) {
  return u32x2{pack_bf2(a, b), pack_bf2(c, d)};
}


// ---------------------------------------------------------------- scheduling
// ---------------------------------------------------------------- m-tile list
// The varlen-M m-tiles (BM = kMTile rows) as a list, built on the device from
// the expert offsets: int32 header {all m-tiles, partial m-tiles, 0, 0}, then
// one {expert, m0, rows, first global row} entry per m-tile, the full tiles
// of every expert in expert order first and the partial last tiles after
// them.  A GEMM workgroup reads its tile's entry with one scalar load.
constexpr int kMTile = 256;
typedef int i32x4 __attribute__((ext_vector_type(4)));
#define SMOE_CONST __attribute__((address_space(4)))

size_t mtiles_bytes(int64_t capacity, int E) { return 16 * (size_t)(1 + capacity / kMTile + E); }

constexpr int kMTilesThreads = 1024;
// pf, pp: LDS [4097] each (per-expert exclusive prefix of full / partial m-tiles)
__device__ __forceinline__ void mtiles_body(const int32_t* __restrict__ offsets, int E, int32_t* __restrict__ out,
                                            int* pf, int* pp, int* scan_lds) {
  const int tid = threadIdx.x;
  // thread t owns experts 4t .. 4t+3 (E <= 4096)
  int nf[4], np[4], sf = 0, sp = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = 4 * tid + q;
    const int cnt = e < E ? offsets[e + 1] - offsets[e] : 0;
    nf[q] = cnt / kMTile;
    np[q] = cnt % kMTile != 0;
    sf += nf[q];
    sp += np[q];
  }
  int F, H;
  int bf = block_excl_scan<kMTilesThreads>(sf, &F, scan_lds);
  int bp = block_excl_scan<kMTilesThreads>(sp, &H, scan_lds);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = 4 * tid + q;
    if (e < E) {
      pf[e] = bf;
      pp[e] = bp;
    }
    bf += nf[q];
    bp += np[q];
  }
  if (tid == 0) {
    pf[E] = F;
    pp[E] = H;
  }
  __syncthreads();
  if (tid == 0) *(i32x4*)out = i32x4{F + H, H, 0, 0};
  for (int t = tid; t < F + H; t += kMTilesThreads) {
    const bool part = t >= F;
    const int key = part ? t - F : t;
    const int* pre = part ? pp : pf;
    // the expert e with pre[e] <= key < pre[e + 1]
    int lo = 0, hi = E;  // pre[lo] <= key < pre[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (pre[mid] <= key) lo = mid; else hi = mid;
    }
    const int off = offsets[lo], cnt = offsets[lo + 1] - off;
    const int m0 = part ? (cnt / kMTile) * kMTile : (key - pre[lo]) * kMTile;
    *(i32x4*)(out + 4 + 4 * t) = i32x4{lo, m0, min(kMTile, cnt - m0), off + m0};
  }
}

__global__ __launch_bounds__(kMTilesThreads) void mtiles_kernel(const int32_t* __restrict__ offsets, int E,
                                                               int32_t* __restrict__ out) {
  __shared__ int pf[4097], pp[4097];
  __shared__ int scan_lds[kMTilesThreads / 64];
  mtiles_body(offsets, E, out, pf, pp, scan_lds);
}

hipError_t launch_mtiles(const int32_t* offsets, int E, int32_t* out, hipStream_t s) {
  if (E > 4096) return hipErrorInvalidValue;
  mtiles_kernel<<<1, kMTilesThreads, 0, s>>>(offsets, E, out);
  return hipGetLastError();
}

// ------------------------------------------------------------ k-chunk list
// The weight gradients reduce over an expert's rows (varlen K).  With skewed
// routing a few experts own most rows, and their tiles would run for the
// whole kernel on a handful of CUs.  The k-chunk list cuts every expert with
// more than Kc rows into Kc-row chunks (Kc = max(kKcMin, 2P / slabs), so the
// chunks need at most `slabs` fp32 partial slabs); a split expert's chunks
// write fp32 partials that dw_reduce_kernel sums in chunk order, the others
// store bf16 directly.  The entries (chunks and unsplit experts) are sorted
// by length, longest first (a counting sort on k steps), and dealt round-robin
// to the 8 XCDs; each XCD's entries are contiguous in the list, so its 32
// workgroups take its tiles (entry-major, longest first) round-robin.  Which
// CU computes a tile does not change any value.
// Layout (int32): header[16] = {entries, split experts, Kc, tiles,
// xcd_start[0..8] (tiles)}; entries at 16 (int4 {e, k_begin, k_len, slot or
// -1}); unsorted entries at 16 + 4 (E + kDwSlabs); split experts at
// 16 + 8 (E + kDwSlabs) (int4 {e, first slot, chunks, 0}).
constexpr int kKcMin = 2048;
constexpr int kKChunksThreads = 1024;
constexpr int kLenBins = 1024;  // counting-sort bins: k steps of 64 rows, the last bin open-ended

size_t kchunks_bytes(int E) { return 4 * (16 + 8 * (size_t)(E + kDwSlabs) + 4 * (kDwSlabs / 2 + 1)); }
__host__ __device__ inline int kchunks_split_off(int E) { return 16 + 8 * (E + kDwSlabs); }

// bins: LDS [kLenBins]
__device__ __forceinline__ void kchunks_body(const int32_t* __restrict__ offsets, int E, int tpe, int slabs,
                                             int32_t* __restrict__ out, int* bins, int* scan_lds, int* sh_kc) {
  static_assert(kLenBins == kKChunksThreads, "one bin per thread");
  const int tid = threadIdx.x;
  if (tid == 0) {
    const int P = offsets[E];
    int kc = 0x7fffffff;  // no slabs: nothing is split
    if (slabs > 0) {
      const int64_t q = (2 * (int64_t)P + slabs - 1) / slabs;
      kc = (int)max((int64_t)kKcMin, (q + 63) / 64 * 64);
    }
    *sh_kc = kc;
  }
  bins[tid] = 0;
  __syncthreads();
  const int Kc = *sh_kc;
  // thread t owns experts 4t .. 4t+3 (E <= 4096)
  int f[4], nc[4], sc = 0, su = 0, sx = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = 4 * tid + q;
    f[q] = e < E ? offsets[e + 1] - offsets[e] : 0;
    nc[q] = (e < E && f[q] > Kc) ? (f[q] + Kc - 1) / Kc : 0;  // chunks of a split expert
    sc += nc[q];
    su += (e < E && nc[q] == 0);
    sx += nc[q] > 0;
  }
  int S, U, X;
  int bc = block_excl_scan<kKChunksThreads>(sc, &S, scan_lds);
  int bu = block_excl_scan<kKChunksThreads>(su, &U, scan_lds);
  int bx = block_excl_scan<kKChunksThreads>(sx, &X, scan_lds);
  i32x4* ent = (i32x4*)(out + 16);
  i32x4* raw = (i32x4*)(out + 16 + 4 * (E + kDwSlabs));
  i32x4* spl = (i32x4*)(out + kchunks_split_off(E));
  auto bin_of = [](int k_len) { return min(kLenBins - 1, (k_len + 63) / 64); };
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = 4 * tid + q;
    if (e >= E) continue;
    const int k0 = offsets[e];
    if (nc[q] > 0) {
      for (int c = 0; c < nc[q]; ++c) {
        const int kb = c * Kc, kl = min(Kc, f[q] - kb);
        raw[bc + c] = i32x4{e, k0 + kb, kl, bc + c};  // slot = chunk position
        atomicAdd(&bins[bin_of(kl)], 1);
      }
      spl[bx] = i32x4{e, bc, nc[q], 0};
      bc += nc[q];
      ++bx;
    } else {
      raw[S + bu] = i32x4{e, k0, f[q], -1};
      atomicAdd(&bins[bin_of(f[q])], 1);
      ++bu;
    }
  }
  const int N = S + U;
  __syncthreads();  // raw entries and bin counts complete
  // first sorted position of each bin, longest bins first (thread t: bin kLenBins-1-t)
  const int b = kLenBins - 1 - tid;
  int total;
  const int first = block_excl_scan<kKChunksThreads>(bins[b], &total, scan_lds);
  bins[b] = first;  // from here on: the bin's next free position
  __syncthreads();
  // sorted position s -> XCD s % 8, place s / 8 within that XCD's contiguous range
  auto xcd_base = [N](int x) {  // entries of the XCDs before x
    int base = 0;
    for (int y = 0; y < x; ++y) base += (N + 7 - y) / 8;
    return base;
  };
  for (int i = tid; i < N; i += kKChunksThreads) {
    const i32x4 r = raw[i];
    const int s2 = atomicAdd(&bins[bin_of(r[2])], 1);
    ent[xcd_base(s2 % 8) + s2 / 8] = r;
  }
  if (tid == 0) {
    out[0] = N;
    out[1] = X;
    out[2] = Kc;
    out[3] = N * tpe;
  }
  if (tid <= 8) out[4 + tid] = xcd_base(tid) * tpe;
}

// The backward's tile lists in one launch: workgroup 0 the m-tile list,
// 1 and 2 the k-chunk lists of dW2 and dW1.
static_assert(kMTilesThreads == kKChunksThreads, "one workgroup size");
__global__ __launch_bounds__(kMTilesThreads) void bwd_lists_kernel(const int32_t* __restrict__ offsets, int E,
                                                                  int32_t* __restrict__ mtiles, int tpe2, int slabs2,
                                                                  int32_t* __restrict__ klist2, int tpe1, int slabs1,
                                                                  int32_t* __restrict__ klist1,
                                                                  const uint16_t* __restrict__ Wr,
                                                                  uint16_t* __restrict__ WrT, int d) {
  __shared__ int lds[2 * 4097];
  __shared__ int scan_lds[kMTilesThreads / 64];
  __shared__ int sh_kc;
  if (blockIdx.x == 0) {
    mtiles_body(offsets, E, mtiles, lds, lds + 4097, scan_lds);
  } else if (blockIdx.x == 1) {
    kchunks_body(offsets, E, tpe2, slabs2, klist2, lds, scan_lds, &sh_kc);
  } else if (blockIdx.x == 2) {
    kchunks_body(offsets, E, tpe1, slabs1, klist1, lds, scan_lds, &sh_kc);
  } else {  // W_r transpose, one element per thread
    const int idx = (blockIdx.x - 3) * kMTilesThreads + threadIdx.x;
    if (idx < d * E) {
      const int e = idx / d, i = idx % d;
      WrT[idx] = Wr[(size_t)i * E + e];
    }
  }
}

// partials of split experts -> bf16 dW: chunk slabs summed in chunk order
// workgroup (bx, by) of a gx x gy grid
__device__ __forceinline__ void dw_reduce_body(const int32_t* __restrict__ klist, const float* __restrict__ part,
                                               uint16_t* __restrict__ dW, int E, int64_t MN, int bx, int by, int gx,
                                               int gy) {
  const SMOE_CONST int32_t* h = (const SMOE_CONST int32_t*)klist;
  const SMOE_CONST i32x4* spl = (const SMOE_CONST i32x4*)(klist + kchunks_split_off(E));
  for (int si = by; si < h[1]; si += gy) {
    const i32x4 sp = spl[si];
    const int e = sp[0], first = sp[1], nc = sp[2];
    for (int64_t i = 4 * ((int64_t)bx * 256 + threadIdx.x); i < MN; i += 4 * (int64_t)gx * 256) {
      f32x4 a = *(const f32x4*)(part + (size_t)first * MN + i);
      for (int c = 1; c < nc; ++c) {
        const f32x4 b = *(const f32x4*)(part + (size_t)(first + c) * MN + i);
        a[0] += b[0];
        a[1] += b[1];
        a[2] += b[2];
        a[3] += b[3];
      }
      *(u32x2*)(dW + (size_t)e * MN + i) = u32x2{pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3])};
    }
  }
}

__global__ __launch_bounds__(256) void dw_reduce_kernel(const int32_t* __restrict__ klist, const float* __restrict__ part,
                                                        uint16_t* __restrict__ dW, int E, int64_t MN) {
  dw_reduce_body(klist, part, dW, E, MN, blockIdx.x, blockIdx.y, gridDim.x, gridDim.y);
}

static void dw_reduce_grid(int64_t MN, int slabs, int* gx, int* gy) {
  *gx = (int)std::min<int64_t>((MN / 4 + 255) / 256, 64);
  // split experts are looped over: most calls have none, and a grid sized for
  // every possible one would mostly launch workgroups that exit at once
  *gy = slabs > 0 ? std::min(slabs / 2, 8) : 0;
}

// The backward's last reductions in one launch: workgroups [0, nd) sum the
// dW1 chunk slabs of split experts (as dw_reduce_kernel), the next nr the dW_r
// split-K partials (fixed split order), the last ne the dbias chunk sums of
// one expert each (fixed tree).
__global__ __launch_bounds__(256) void bwd_final_reduce_kernel(const int32_t* __restrict__ klist1,
                                                               const float* __restrict__ part1,
                                                               uint16_t* __restrict__ dW1, int64_t MN1, int gx1,
                                                               int gy1, const float* __restrict__ dwr_part,
                                                               float* __restrict__ dWr, int n, int splits, int nr,
                                                               const float* __restrict__ cs_part,
                                                               float* __restrict__ dbias, int chunks, int E) {
  const int nd = gx1 * gy1;
  int b = blockIdx.x;
  if (b < nd) {
    dw_reduce_body(klist1, part1, dW1, E, MN1, b % gx1, b / gx1, gx1, gy1);
    return;
  }
  b -= nd;
  if (b < nr) {
    const int i = b * 256 + threadIdx.x;
    if (i >= n) return;
    float s = 0.f;
    for (int k = 0; k < splits; ++k) s += dwr_part[(size_t)k * n + i];
    dWr[i] = s;
    return;
  }
  __shared__ float red[4];
  const int e = b - nr;
  float s = 0.f;
  for (int i = threadIdx.x; i < chunks; i += 256) s += cs_part[(size_t)i * E + e];
  s = wave_sum(s);
  if (lane_id() == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) dbias[e] = (red[0] + red[1]) + (red[2] + red[3]);
}

hipError_t launch_dw_reduce(const int32_t* klist, const float* part, uint16_t* dW, int E, int64_t MN, int slabs,
                            hipStream_t s) {
  if (slabs <= 0) return hipSuccess;
  int gx, gy;
  dw_reduce_grid(MN, slabs, &gx, &gy);
  dw_reduce_kernel<<<dim3(gx, gy), dim3(256), 0, s>>>(klist, part, dW, E, MN);
  return hipGetLastError();
}

// A varlen-K tile from the k-chunk list: entry = id / (tiles per entry).
template <int BM, int BN>
__device__ __forceinline__ bool tile_kchunk(const int32_t* klist, int E, int M, int N, int id, TileInfo& ti) {
  const int mtn = M / BM, ntn = N / BN;
  const SMOE_CONST i32x4* ent = (const SMOE_CONST i32x4*)(klist + 16);
  const i32x4 t = ent[id / (mtn * ntn)];
  const int rem = id % (mtn * ntn);
  ti.e = t[0];
  ti.m0 = (rem / ntn) * BM;
  ti.n0 = (rem % ntn) * BN;
  ti.mrows = BM;
  ti.row_base = t[3];  // partial slab, or -1
  ti.k_begin = t[1];
  ti.k_len = t[2];
  return true;
}
__device__ __forceinline__ void kchunk_xcd_range(const int32_t* klist, int x, int* begin, int* count) {
  const SMOE_CONST int32_t* h = (const SMOE_CONST int32_t*)klist;
  *begin = h[4 + x];
  *count = h[5 + x] - h[4 + x];
}

// fp32 tile of a partial slab [M][ld]
template <class Cfg>
__device__ __forceinline__ void store_part_f32(float* out, int64_t ld, int m0, int n0, Acc<Cfg>& t) {
#pragma unroll
  for (int i = 0; i < Cfg::RM; ++i) {
    float* o = out + (size_t)(m0 + t.m_of(i)) * ld + n0;
#pragma unroll
    for (int j = 0; j < Cfg::RN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 v;
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = t.acc[i][j][4 * g + q];
        *(f32x4*)(o + t.n_of(j, g)) = v;
      }
  }
}

// Logical tile ids are m-tile-major within their class (full m-tiles, then
// the partial ones): id = mt * (N / BN) + nt, so neighbouring ids share the
// rows of one m-tile and the weights of one expert.  The list entry is
// read with a scalar load (the id is workgroup-uniform).
template <int BM, int BN>
__device__ __forceinline__ bool tile_varlen_m(const int32_t* mtiles, int N, int K, int id, TileInfo& ti) {
  static_assert(BM == kMTile, "varlen-M tiles are the m-tile list's tiles");
  const int nnt = N / BN;
  const bool partial = (id & kPartialTile) != 0;
  id &= kPartialTile - 1;
  const int mt = id / nnt, nt = id % nnt;
  const SMOE_CONST i32x4* list = (const SMOE_CONST i32x4*)mtiles;
  const i32x4 h = list[0];
  const int idx = partial ? h[0] - h[1] + mt : mt;
  if (idx >= h[0]) return false;
  const i32x4 t = list[1 + idx];
  ti.e = t[0];
  ti.m0 = t[1];
  ti.mrows = t[2];
  ti.row_base = t[3];
  ti.n0 = nt * BN;
  ti.k_begin = 0;
  ti.k_len = K;
  return true;
}

template <int BN>
__device__ __forceinline__ int count_varlen_m(const int32_t* mtiles, int N) {
  return ((const SMOE_CONST i32x4*)mtiles)[0][0] * (N / BN);
}
// tiles of the tail class (partial m-tiles)
template <int BN>
__device__ __forceinline__ int count_varlen_m_tail(const int32_t* mtiles, int N) {
  return ((const SMOE_CONST i32x4*)mtiles)[0][1] * (N / BN);
}

template <int BM, int BN>
__device__ __forceinline__ bool tile_plain_m(int M, int N, int K, int id, TileInfo& ti) {
  const int nnt = (N + BN - 1) / BN;
  const int mt = id / nnt, nt = id % nnt;
  ti.e = 0;
  ti.m0 = mt * BM;
  if (ti.m0 >= M) return false;
  ti.mrows = min(BM, M - ti.m0);
  ti.row_base = ti.m0;
  ti.n0 = nt * BN;
  ti.k_begin = 0;
  ti.k_len = K;
  return true;
}

struct ColOffset {
  int c0;
  __device__ __forceinline__ int operator()(int c) const { return c0 + c; }
};

// Adds bias[colmap(c)] to every accumulator of tile-local column c (the
// expert biases of the projections).  A lane's accumulator block (j, g) holds
// four consecutive columns, which colmap keeps consecutive.
template <class Cfg, class ColMap>
__device__ __forceinline__ void add_col_bias(Acc<Cfg>& t, const float* bias, ColMap colmap) {
#pragma unroll
  for (int j = 0; j < Cfg::RN; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 b = *(const f32x4*)(bias + colmap(t.n_of(j, g)));
#pragma unroll
      for (int i = 0; i < Cfg::RM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) t.acc[i][j][4 * g + r] += b[r];
    }
}

// ================================================================== router
template <class Cfg_>
struct OpRouter {
  using Cfg = Cfg_;
  static constexpr int M_MODE = ROWS, N_MODE = KOUTER;
  static constexpr int EPI_LDS = 0;
  struct Params { RouterGemmArgs a; };
  static __device__ int count(const Params& p, int*) {
    return ((p.a.T + Cfg::BM - 1) / Cfg::BM) * ((p.a.E + Cfg::BN - 1) / Cfg::BN);
  }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int*) {
    return tile_plain_m<Cfg::BM, Cfg::BN>(p.a.T, p.a.E, p.a.d, id, ti);
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, RowsSide<Cfg::BM, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.X, p.a.d, nullptr, ti.row_base, ti.mrows);
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BN, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.Wr, p.a.E, nullptr, 0, p.a.d, p.a.E, ColOffset{ti.n0});
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char*) {
#pragma unroll
    for (int i = 0; i < Cfg::RM; ++i) {
      const int m = t.m_of(i);
      if (m >= ti.mrows) continue;
      float* out = p.a.logits + (size_t)(ti.row_base + m) * p.a.E;
#pragma unroll
      for (int j = 0; j < Cfg::RN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = ti.n0 + t.n_of(j, g);
          if (col >= p.a.E) continue;
          f32x4 v;
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = t.acc[i][j][4 * g + q] + (p.a.bias ? p.a.bias[col + q] : 0.f);
          *(f32x4*)(out + col) = v;
        }
    }
  }
};

// ======================================================= router + softmax/top-K
// The router GEMM with the routing of Section 2.3 / Appendix D in its
// epilogue, for E <= BN (one N tile holds every logit of its 128 tokens).  A
// token's row is spread over WN waves and two lanes per wave (the MFMA layout:
// lane l and l + 32 hold alternate groups of four columns), NV = 16 RN values
// per lane.  The epilogue:
//   1. logits = acc (+ bias), written when asked for; row maximum and then the
//      sum of exp(x - max) over the lane, its partner lane, and the WN waves
//      (through LDS, in wave order, so every holder of the row agrees);
//   2. scores = exp * (1 / sum), written token-major and expert-major;
//   3. each lane sorts its NV (score, expert) pairs in groups of KM and merges
//      them into a top-KM list, merges that with its partner lane's list and
//      then with the other waves' lists (LDS): all holders of the row end with
//      the row's sorted top-KM;
//   4. membership: a pair at or above the K-th is selected; one ballot per
//      (column group) gives 32 rows of two columns, parked in LDS per 32-row
//      block, then written as the 64-bit words of the expert-major bitmap;
//   5. the weights: the K selected scores summed in ascending expert order
//      (the order the separate top-K kernel uses, so the two agree bit for bit
//      on the same scores), then score / sum.
// A wave with two 32-row blocks (128 x 256 tiles) runs steps 1-5 for each
// block in turn; the membership words go out once both are parked.
// The results match launch_topk_route on these scores exactly; the scores
// themselves differ from its own softmax of the same logits only in the
// rounding of the sum.
template <class Cfg_, int KM, bool FULL_N>
struct OpRouterTopk {
  using Cfg = Cfg_;
  static constexpr int M_MODE = ROWS, N_MODE = KOUTER;
  static constexpr int BM = Cfg::BM, BN = Cfg::BN, WN = Cfg::WN, NV = Cfg::RN * 16;
  static_assert(Cfg::RM <= 2, "one or two 32-row blocks per wave");
  static_assert(NV % KM == 0, "pairs per lane in groups of KM");
  // LDS: row maxima, row sums [WN][BM] f32; top lists [WN][KM][BM] u64;
  // membership pieces [BM / 32][BN] u32
  static constexpr int kSumOff = WN * BM * 4, kListOff = 2 * WN * BM * 4;
  static constexpr int kBitsOff = kListOff + WN * KM * BM * 8;
  static constexpr int EPI_LDS = kBitsOff + (BM / 32) * BN * 4;
  struct Params { RouterTopkArgs a; };
  static __device__ int count(const Params& p, int*) { return (p.a.T + BM - 1) / BM; }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int*) {
    return tile_plain_m<BM, BN>(p.a.T, p.a.E, p.a.d, id, ti);
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, RowsSide<BM, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.X, p.a.d, nullptr, ti.row_base, ti.mrows);
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, KOuterSide<BN, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.Wr, p.a.E, nullptr, 0, p.a.d, p.a.E, ColOffset{ti.n0});
  }
  static __device__ uint64_t xor32(uint64_t v) {
    const uint32_t lo = __shfl_xor((uint32_t)v, 32, kWave), hi = __shfl_xor((uint32_t)(v >> 32), 32, kWave);
    return ((uint64_t)hi << 32) | lo;
  }
  // row block I of the wave (rows 32 I .. 32 I + 31 of its BM / WM)
  template <int I>
  static __device__ void row_block(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char* lds) {
    const RouterTopkArgs& a = p.a;
    // lane-dependent coordinates from an opaque lane read: computed here, not
    // hoisted out of the tile loop as constants that stay live through it
    const int lane = volatile_lane(), wave = threadIdx.x >> 6;
    const int wn = Cfg::wave_n(wave), wm = Cfg::wave_m(wave), h = lane >> 5, u = lane & 31;
    const int m = wm * (BM / Cfg::WM) + 32 * I + u;
    // column of value 4 (4 j + g) + q: the MFMA output layout (Acc::n_of)
    const int c0 = wn * (BN / WN) + 4 * h;
    auto col_of = [&](int k) { return c0 + 32 * (k >> 4) + 8 * ((k >> 2) & 3) + (k & 3); };
    // E a multiple of 8: a group of four columns is wholly inside or outside
    auto col_ok = [&](int k) { return FULL_N || col_of(k) < a.E; };
    const bool live = m < ti.mrows;
    const size_t row = (size_t)(ti.row_base + m);
    float* rmax = (float*)lds;
    float* rsum = (float*)(lds + kSumOff);
    uint64_t* lists = (uint64_t*)(lds + kListOff);
    uint32_t* bits = (uint32_t*)(lds + kBitsOff);
    float v[NV];
    float mx = -INFINITY;
#pragma unroll
    for (int k0 = 0; k0 < NV; k0 += 4) {
      const int col = col_of(k0);
      f32x4 x;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        x[q] = t.acc[I][k0 >> 4][(k0 & 15) + q];
        if (a.bias) x[q] += col_ok(k0) ? a.bias[col + q] : 0.f;
        v[k0 + q] = col_ok(k0) ? x[q] : -INFINITY;
        mx = fmaxf(mx, v[k0 + q]);
      }
      if (a.logits && live && col_ok(k0)) *(f32x4*)(a.logits + row * a.E + col) = x;
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    if (h == 0) rmax[wn * BM + m] = mx;
    barrier_lds();
    mx = rmax[m];
#pragma unroll
    for (int w = 1; w < WN; ++w) mx = fmaxf(mx, rmax[w * BM + m]);
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      v[k] = __expf(v[k] - mx);  // 0 for the columns past E
      sum += v[k];
    }
    sum += __shfl_xor(sum, 32, kWave);  // the same value in both lanes
    if (h == 0) rsum[wn * BM + m] = sum;
    barrier_lds();
    sum = rsum[m];
#pragma unroll
    for (int w = 1; w < WN; ++w) sum += rsum[w * BM + m];
    const float rs = 1.f / sum;
#pragma unroll
    for (int k0 = 0; k0 < NV; k0 += 4) {
      const int col = col_of(k0);
      f32x4 x;
#pragma unroll
      for (int q = 0; q < 4; ++q) x[q] = v[k0 + q] = v[k0 + q] * rs;
      if (live && col_ok(k0)) {
        *(f32x4*)(a.scores + row * a.E + col) = x;
        if (a.scores_t) {
#pragma unroll
          for (int q = 0; q < 4; ++q) a.scores_t[(size_t)(col + q) * a.T + row] = x[q];
        }
      }
    }
    // (score, expert) pair of value k, 0 for a row past T or a column past E
    // (masked, not branched around)
    const uint64_t live_mask = live ? ~0ull : 0ull;
    auto pair = [&](int k) -> uint64_t {
      const uint64_t pk = topk_pair(v[k], col_of(k)) & live_mask;
      if constexpr (FULL_N) return pk;
      return col_ok(k) ? pk : 0ull;
    };
    uint64_t top[KM];
#pragma unroll
    for (int k = 0; k < KM; ++k) top[k] = pair(k);
    topk_sort<KM>(top);
#pragma unroll
    for (int g0 = KM; g0 < NV; g0 += KM) {
      uint64_t grp[KM];
#pragma unroll
      for (int k = 0; k < KM; ++k) grp[k] = pair(g0 + k);
      topk_sort<KM>(grp);
      topk_merge<KM>(top, grp);
    }
    {
      uint64_t o[KM];
#pragma unroll
      for (int k = 0; k < KM; ++k) o[k] = xor32(top[k]);
      topk_merge<KM>(top, o);  // the row's pairs are distinct: both lanes get the same list
    }
    if (h == 0) {
#pragma unroll
      for (int k = 0; k < KM; ++k) lists[(wn * KM + k) * BM + m] = top[k];
    }
    barrier_lds();
#pragma unroll
    for (int w = 0; w < WN; ++w) {
      if (w == wn) continue;
      uint64_t o[KM];
#pragma unroll
      for (int k = 0; k < KM; ++k) o[k] = lists[(w * KM + k) * BM + m];
      topk_merge<KM>(top, o);
    }
    uint64_t thr = top[0];
#pragma unroll
    for (int k = 1; k < KM; ++k)
      if (k == a.K - 1) thr = top[k];
    // membership: ballot k holds rows 0..31 of the wave for column col_of(k)
    // of the lanes below 32 (low half) and of the lanes above (high half);
    // lane u + 32 h keeps half h of ballots u, u + 32, ..., i.e. its own
    // columns col_of(u), col_of(u + 32), ...
    constexpr int kMine = (NV + 31) / 32;  // ballots kept per lane
    uint32_t mine[kMine];
#pragma unroll
    for (int r = 0; r < kMine; ++r) mine[r] = 0;
#pragma unroll
    for (int k = 0; k < NV; ++k) asm volatile("" : "+v"(v[k]));  // recompute the pairs, do not keep them
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const uint64_t pk = pair(k);
      const uint64_t b = __ballot(pk != 0ull && pk >= thr);
      mine[k >> 5] = u == (k & 31) ? (uint32_t)(b >> (32 * h)) : mine[k >> 5];
    }
#pragma unroll
    for (int r = 0; r < kMine; ++r)
      if (32 * r + u < NV) bits[(wm * Cfg::RM + I) * BN + col_of(32 * r + u)] = mine[r];
    if (live && wn == 0 && h == 0) {
      // the selected scores in ascending expert order: (expert, score) halves
      // swapped, so the descending sort puts the lowest expert first
      uint64_t byx[KM];
#pragma unroll
      for (int k = 0; k < KM; ++k) byx[k] = k < a.K ? (top[k] << 32) | (top[k] >> 32) : 0ull;
      topk_sort<KM>(byx);
      float den = 0.f;
#pragma unroll
      for (int k = 0; k < KM; ++k)
        if (k < a.K) den += topk_value((uint32_t)byx[k]);
#pragma unroll
      for (int k = 0; k < KM; ++k)
        if (k < a.K) {
          a.topk_idx[row * a.K + k] = (int32_t)~(uint32_t)top[k];
          a.topk_w[row * a.K + k] = topk_value((uint32_t)(top[k] >> 32)) / den;
        }
    }
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char* lds) {
    row_block<0>(p, ti, t, lds);
    if constexpr (Cfg::RM > 1) row_block<1>(p, ti, t, lds);
    // the membership words: 64 tile rows (two 32-row pieces) per word
    const RouterTopkArgs& a = p.a;
    const uint32_t* bits = (const uint32_t*)(lds + kBitsOff);
    barrier_lds();
    const int w0 = ti.row_base / 64;
    for (int i = threadIdx.x; i < (BM / 64) * a.E; i += Cfg::THREADS) {
      const int e = i / (BM / 64), ww = i % (BM / 64);
      if (w0 + ww < a.W)
        a.mask[(size_t)e * a.W + w0 + ww] = bits[2 * ww * BN + e] | ((uint64_t)bits[(2 * ww + 1) * BN + e] << 32);
    }
  }
};

// Row-contiguous stores of a wave's output: the two 32-column accumulator
// blocks j, j+1 of one 32-row block (64 columns, 128 bytes of a bf16 row) go
// through the wave's own 2 KB of LDS, 16 rows at a time, and come back so
// that 8 lanes hold one 128-byte row segment.  Each store instruction then
// writes 8 whole cache lines instead of 32-byte pieces of 32 rows.  The LDS
// operations of one wave complete in order, so no barrier is needed; the
// 16-byte chunk c of staged row r sits at chunk c ^ ((r >> 1) & 7), which
// keeps both the writes (one chunk of 16 rows) and the reads (two whole
// rows per 16 lanes) free of bank conflicts.  The stores are nontemporal:
// these outputs (H and A, Y, dH and A', dX~, the weight gradients) are
// consumed by a later kernel that streams them once, and left in the cache
// as dirty lines they only add write-back traffic at the end of the
// producing kernel (plain stores measured slower for up and no better for dH).
constexpr int kStageBytesPerWave = 16 * 128;
template <class Cfg>
constexpr bool kStagedStores = Cfg::RN % 2 == 0 && Cfg::LDS_BYTES + Cfg::NW * kStageBytesPerWave + 256 <= 160 * 1024;
// store instructions per wave of store_rows_bf16_any on a full tile: staged
// (through the idle last stage or the epilogue area), four per 64-column row
// block; direct, two per 32 columns
template <class Cfg>
constexpr int kStoresPerFullTile =
    Cfg::RN % 2 == 0 && (Cfg::STAGE_BYTES >= Cfg::NW * 4096 || kStagedStores<Cfg>) ? Cfg::RM * (Cfg::RN / 2) * 4
                                                                                   : Cfg::RM * Cfg::RN * 2;
// Epilogue address arithmetic uses the lane index from a volatile asm, so
// it stays in the epilogue instead of being hoisted out of the tile loop.
__device__ __forceinline__ int epilogue_lane() { return volatile_lane(); }

__device__ __forceinline__ void store_rows64_staged(char* wl, uint16_t* blk, int64_t ld, int rows_valid,
                                                    const u32x2 (&v0)[4], const u32x2 (&v1)[4]) {
  const int lane = epilogue_lane();
  const int r = lane & 31, hi = lane >> 5;
  u32x4 c[2][2];  // [block][g/2]: 16 bytes, chunk 4*block + g + hi of row r
#pragma unroll
  for (int g = 0; g < 4; g += 2) {
    {
      const auto a = __builtin_amdgcn_permlane32_swap(v0[g][0], v0[g + 1][0], false, false);
      const auto b = __builtin_amdgcn_permlane32_swap(v0[g][1], v0[g + 1][1], false, false);
      c[0][g / 2] = u32x4{a[0], b[0], a[1], b[1]};
    }
    {
      const auto a = __builtin_amdgcn_permlane32_swap(v1[g][0], v1[g + 1][0], false, false);
      const auto b = __builtin_amdgcn_permlane32_swap(v1[g][1], v1[g + 1][1], false, false);
      c[1][g / 2] = u32x4{a[0], b[0], a[1], b[1]};
    }
  }
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    if ((r >> 4) == q) {
      const int rr = r & 15;
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int g = 0; g < 4; g += 2) {
          const int ch = 4 * b + g + hi;
          *(u32x4*)(wl + rr * 128 + ((ch ^ ((rr >> 1) & 7)) << 4)) = c[b][g / 2];
        }
    }
    // other lanes' data is read back: keep the compiler from reordering or
    // forwarding across this point (the hardware keeps one wave's LDS
    // operations in order)
    asm volatile("" ::: "memory");
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int R = 8 * t + (lane >> 3), C = lane & 7;
      const u32x4 x = *(const u32x4*)(wl + R * 128 + ((C ^ ((R >> 1) & 7)) << 4));
      const int row = 16 * q + R;
      if (row < rows_valid) __builtin_nontemporal_store(x, (u32x4*)(blk + (row * (int)ld + 8 * C)));
    }
    asm volatile("" ::: "memory");  // reads of this round before the next round's writes
  }
}

// Two-step form of the staging above for 32 rows at once, used where an
// output's two 32-column blocks are produced one after the other: each block
// is written into a wave-private 4 KB area as soon as it is computed (chunk
// 4 * jj + g + hi of row r, same swizzle), and the 32 rows are then stored as
// whole lines.  The area must not be touched by other waves in between.
__device__ __forceinline__ void stage_block32(char* wl, int jj, const u32x2 (&v)[4]) {
  const int lane = epilogue_lane();
  const int r = lane & 31, hi = lane >> 5;
#pragma unroll
  for (int g = 0; g < 4; g += 2) {
    const auto a = __builtin_amdgcn_permlane32_swap(v[g][0], v[g + 1][0], false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(v[g][1], v[g + 1][1], false, false);
    const int ch = 4 * jj + g + hi;
    *(u32x4*)(wl + r * 128 + ((ch ^ ((r >> 1) & 7)) << 4)) = u32x4{a[0], b[0], a[1], b[1]};
  }
}

__device__ __forceinline__ void store_staged32(const char* wl, uint16_t* blk, int64_t ld, int rows_valid) {
  asm volatile("" ::: "memory");  // the staged writes of every lane precede these reads
  const int lane = epilogue_lane();
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int R = 8 * t + (lane >> 3), C = lane & 7;
    const u32x4 x = *(const u32x4*)(wl + R * 128 + ((C ^ ((R >> 1) & 7)) << 4));
    if (R < rows_valid) __builtin_nontemporal_store(x, (u32x4*)(blk + (R * (int)ld + 8 * C)));
  }
  asm volatile("" ::: "memory");  // and precede the next writes to the area
}

// The same with every row sent to its own destination row dst[R] of out
// (columns col .. col + 63): the scatter-fused store of the aggregation
// ablation.
__device__ __forceinline__ void store_staged32_scatter(const char* wl, uint16_t* out, int64_t ld, int col,
                                                       const int32_t* dst, int rows_valid) {
  asm volatile("" ::: "memory");
  const int lane = epilogue_lane();
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int R = 8 * t + (lane >> 3), C = lane & 7;
    const u32x4 x = *(const u32x4*)(wl + R * 128 + ((C ^ ((R >> 1) & 7)) << 4));
    if (R < rows_valid)
      __builtin_nontemporal_store(x, (u32x4*)(out + (size_t)dst[R] * ld + col + 8 * C));
  }
  asm volatile("" ::: "memory");
}

// The same for an output whose first block is held in a 2 KB half-row area
// (32 rows x 64 bytes, chunk c of row r at r * 64 + ((c ^ ((r >> 1) & 3)) <<
// 4)) and whose second block is in chunks 4..7 of a 4 KB area as above.
__device__ __forceinline__ void stage_half32(char* wh, const u32x2 (&v)[4]) {
  const int lane = epilogue_lane();
  const int r = lane & 31, hi = lane >> 5;
#pragma unroll
  for (int g = 0; g < 4; g += 2) {
    const auto a = __builtin_amdgcn_permlane32_swap(v[g][0], v[g + 1][0], false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(v[g][1], v[g + 1][1], false, false);
    const int ch = g + hi;
    *(u32x4*)(wh + r * 64 + ((ch ^ ((r >> 1) & 3)) << 4)) = u32x4{a[0], b[0], a[1], b[1]};
  }
}

__device__ __forceinline__ void store_staged32_split(const char* wh, const char* wl, uint16_t* blk, int64_t ld,
                                                     int rows_valid) {
  asm volatile("" ::: "memory");
  const int lane = epilogue_lane();
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int R = 8 * t + (lane >> 3), C = lane & 7;
    const char* src = C < 4 ? wh + R * 64 + ((C ^ ((R >> 1) & 3)) << 4) : wl + R * 128 + ((C ^ ((R >> 1) & 7)) << 4);
    const u32x4 x = *(const u32x4*)src;
    if (R < rows_valid) __builtin_nontemporal_store(x, (u32x4*)(blk + (R * (int)ld + 8 * C)));
  }
  asm volatile("" ::: "memory");
}

template <class Cfg>
__device__ __forceinline__ void store_rows_bf16(uint16_t* out, int64_t ld, int row_base, int mrows, int n0,
                                                Acc<Cfg>& t, char* epi) {
  if constexpr (!kStagedStores<Cfg>) {
#pragma unroll
    for (int i = 0; i < Cfg::RM; ++i) {
      const int m = t.m_of(i);
      if (m >= mrows) continue;
      uint16_t* y = out + (size_t)(row_base + m) * ld + n0;
#pragma unroll
      for (int j = 0; j < Cfg::RN; ++j) {
        u32x2 v[4];
#pragma unroll
        for (int g = 0; g < 4; ++g)
          v[g] = pack_bf16x4(t.acc[i][j][4 * g], t.acc[i][j][4 * g + 1], t.acc[i][j][4 * g + 2], t.acc[i][j][4 * g + 3]);
        store_block_bf16(y + t.n_of(j, 0) - 4 * ((threadIdx.x >> 5) & 1), v);
      }
    }
    return;
  }
  char* wl = epi + (threadIdx.x >> 6) * kStageBytesPerWave;
  const int wm0 = t.m_of(0) - (threadIdx.x & 31);
#pragma unroll
  for (int i = 0; i < Cfg::RM; ++i) {
    const int m0 = wm0 + 32 * i;  // first tile row of the block
    if (m0 >= mrows) continue;
#pragma unroll
    for (int j = 0; j + 1 < Cfg::RN; j += 2) {
      u32x2 v0[4], v1[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        v0[g] = pack_bf16x4(t.acc[i][j][4 * g], t.acc[i][j][4 * g + 1], t.acc[i][j][4 * g + 2], t.acc[i][j][4 * g + 3]);
        v1[g] = pack_bf16x4(t.acc[i][j + 1][4 * g], t.acc[i][j + 1][4 * g + 1], t.acc[i][j + 1][4 * g + 2],
                            t.acc[i][j + 1][4 * g + 3]);
      }
      const int col = n0 + t.n_of(j, 0) - 4 * ((threadIdx.x >> 5) & 1);
      store_rows64_staged(wl, out + (size_t)(row_base + m0) * ld + col, ld, mrows - m0, v0, v1);
    }
  }
}

// ================================================================== up-proj
// N tile: BN/2 gate columns starting at j0 = nt * BN/2 and the matching up
// columns.  Wave column group wn owns Wn = BN/WN tile columns: its first
// Wn/2 are gate columns j0 + wn*Wn/2 + [0, Wn/2) (accumulator blocks
// j < RN/2) and its last Wn/2 the matching up columns (blocks j >= RN/2).

template <class Cfg_>
struct OpUp {
  using Cfg = Cfg_;
  static constexpr int M_MODE = ROWS, N_MODE = KOUTER;
  static constexpr int Wn = Cfg::BN / Cfg::WN;
  static_assert(Cfg::RN % 2 == 0, "gate and up blocks in one wave");
  struct Params { UpArgs a; };
  struct ColMap {
    int j0, n;
    __device__ __forceinline__ int operator()(int c) const {
      const int wn = c / Wn, q = c % Wn;
      return q < Wn / 2 ? j0 + wn * (Wn / 2) + q : n + j0 + wn * (Wn / 2) + (q - Wn / 2);
    }
  };
  static constexpr int IDX_LDS = Cfg::NW * Cfg::QM * 256;  // gathered X rows of the next tile
  // with 64 gate and 64 up columns per wave, H and A leave as whole 128-byte
  // lines through store_rows64_staged
  static constexpr bool STAGED =
      Cfg::RN % 4 == 0 && Cfg::LDS_BYTES + Cfg::NW * kStageBytesPerWave + IDX_LDS <= 160 * 1024;
  static constexpr int EPI_LDS = STAGED ? Cfg::NW * kStageBytesPerWave : 0;
  // full tile: staged, per row block and 64-column pair, H gate, H up and A,
  // four stores each; direct, per 32-column block, two stores each
  static constexpr int EPI_STORES = STAGED ? Cfg::RM * (Cfg::RN / 4) * 12 : Cfg::RM * (Cfg::RN / 2) * 6;
  static __device__ int count(const Params& p, int* sh) {
    return count_varlen_m<Cfg::BN>(p.a.mtiles, 2 * p.a.n);
  }
  static __device__ int count_tail(const Params& p, const int* sh) {
    return count_varlen_m_tail<Cfg::BN>(p.a.mtiles, 2 * p.a.n);
  }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int* sh) {
    return tile_varlen_m<Cfg::BM, Cfg::BN>(p.a.mtiles, 2 * p.a.n, p.a.d, id, ti);
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, RowsSide<Cfg::BM, Cfg::BK, Cfg::NW, true>& s) {
    s.init(p.a.X, p.a.d, p.a.row_token, ti.row_base, ti.mrows);
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BN, Cfg::BK, Cfg::NW>& s) {
    const uint16_t* w = p.a.W1 + (size_t)ti.e * p.a.d * (2 * p.a.n);
    s.init(w, 2 * p.a.n, nullptr, 0, p.a.d, 2 * p.a.n, ColMap{(ti.n0 / Cfg::BN) * (Cfg::BN / 2), p.a.n});
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char* epi) {
    constexpr int RN = Cfg::RN;
    const int n = p.a.n;
    const int j0 = (ti.n0 / Cfg::BN) * (Cfg::BN / 2);
    const int wn = t.wave_n();
    if (p.a.b1) add_col_bias<Cfg>(t, p.a.b1 + (size_t)ti.e * (2 * n), ColMap{j0, n});
    if constexpr (STAGED) {
      char* wl = epi + (threadIdx.x >> 6) * kStageBytesPerWave;
      const int wm0 = t.m_of(0) - (threadIdx.x & 31);
#pragma unroll
      for (int i = 0; i < Cfg::RM; ++i) {
        const int m0 = wm0 + 32 * i;
        if (m0 >= ti.mrows) continue;
        const size_t r0 = (size_t)(ti.row_base + m0);
#pragma unroll
        for (int j = 0; j < RN / 2; j += 2) {
          const int col = j0 + wn * (Wn / 2) + 32 * j;  // first column of the 64-column pair
          u32x2 hg[2][4], hu[2][4], ha[2][4];
#pragma unroll
          for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              float gv[4], uv[4], av[4];
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                gv[r] = t.acc[i][j + q][4 * g + r];
                uv[r] = t.acc[i][j + q + RN / 2][4 * g + r];
                float sg;
                av[r] = silu_sig(gv[r], &sg) * uv[r];
              }
              hg[q][g] = pack_bf16x4(gv[0], gv[1], gv[2], gv[3]);
              hu[q][g] = pack_bf16x4(uv[0], uv[1], uv[2], uv[3]);
              ha[q][g] = pack_bf16x4(av[0], av[1], av[2], av[3]);
            }
          const int rv = ti.mrows - m0;
          if constexpr (Cfg::STAGE_BYTES >= Cfg::NW * 8192) {
            // one round per output through the wave's 8 KB of the idle last stage buffer
            char* st = epi - Cfg::STAGE_BYTES + (threadIdx.x >> 6) * 8192;
            stage_block32(st, 0, hg[0]);
            stage_block32(st, 1, hg[1]);
            store_staged32(st, p.a.H + r0 * (2 * n) + col, 2 * n, rv);
            stage_block32(st + 4096, 0, hu[0]);
            stage_block32(st + 4096, 1, hu[1]);
            store_staged32(st + 4096, p.a.H + r0 * (2 * n) + n + col, 2 * n, rv);
            stage_block32(st, 0, ha[0]);
            stage_block32(st, 1, ha[1]);
            store_staged32(st, p.a.A + r0 * n + col, n, rv);
          } else {
            store_rows64_staged(wl, p.a.H + r0 * (2 * n) + col, 2 * n, rv, hg[0], hg[1]);
            store_rows64_staged(wl, p.a.H + r0 * (2 * n) + n + col, 2 * n, rv, hu[0], hu[1]);
            store_rows64_staged(wl, p.a.A + r0 * n + col, n, rv, ha[0], ha[1]);
          }
        }
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < Cfg::RM; ++i) {
      const int m = t.m_of(i);
      if (m >= ti.mrows) continue;
      const size_t row = (size_t)(ti.row_base + m);
      uint16_t* h = p.a.H + row * (2 * n);
      uint16_t* a = p.a.A + row * n;
#pragma unroll
      for (int j = 0; j < RN / 2; ++j) {
        const int col = j0 + wn * (Wn / 2) + 32 * j;  // first column of the 32-column block
        u32x2 hg[4], hu[4], ha[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float gv[4], uv[4], av[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            gv[r] = t.acc[i][j][4 * g + r];
            uv[r] = t.acc[i][j + RN / 2][4 * g + r];
            float sg;
            av[r] = silu_sig(gv[r], &sg) * uv[r];
          }
          hg[g] = pack_bf16x4(gv[0], gv[1], gv[2], gv[3]);
          hu[g] = pack_bf16x4(uv[0], uv[1], uv[2], uv[3]);
          ha[g] = pack_bf16x4(av[0], av[1], av[2], av[3]);
        }
        store_block_bf16(h + col, hg);
        store_block_bf16(h + n + col, hu);
        store_block_bf16(a + col, ha);
      }
    }
  }
};

// As store_rows_bf16, for ops whose last stage buffer is idle during the
// epilogue (no DMA writes it before the next tile's first barrier): each 32 x
// 64 block pair goes through the wave's 4 KB share of it in one round
// (stage_block32 twice, then store_staged32) instead of two 16-row rounds
// through the 2 KB epilogue area.
template <class Cfg>
__device__ __forceinline__ void store_rows_bf16_stage(uint16_t* out, int64_t ld, int row_base, int mrows, int n0,
                                                      Acc<Cfg>& t, char* epi) {
  static_assert(Cfg::RN % 2 == 0 && Cfg::STAGE_BYTES >= Cfg::NW * 4096, "a 4 KB share of the last stage per wave");
  char* st = epi - Cfg::STAGE_BYTES + (threadIdx.x >> 6) * 4096;
  const int wm0 = t.m_of(0) - (threadIdx.x & 31);
#pragma unroll
  for (int i = 0; i < Cfg::RM; ++i) {
    const int m0 = wm0 + 32 * i;  // first tile row of the block
    if (m0 >= mrows) continue;
#pragma unroll
    for (int j = 0; j + 1 < Cfg::RN; j += 2) {
      u32x2 v0[4], v1[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        v0[g] = pack_bf16x4(t.acc[i][j][4 * g], t.acc[i][j][4 * g + 1], t.acc[i][j][4 * g + 2], t.acc[i][j][4 * g + 3]);
        v1[g] = pack_bf16x4(t.acc[i][j + 1][4 * g], t.acc[i][j + 1][4 * g + 1], t.acc[i][j + 1][4 * g + 2],
                            t.acc[i][j + 1][4 * g + 3]);
      }
      const int col = n0 + t.n_of(j, 0) - 4 * ((threadIdx.x >> 5) & 1);
      stage_block32(st, 0, v0);
      stage_block32(st, 1, v1);
      store_staged32(st, out + (size_t)(row_base + m0) * ld + col, ld, mrows - m0);
    }
  }
}

// the one-round form where the last stage buffer allows it
template <class Cfg>
__device__ __forceinline__ void store_rows_bf16_any(uint16_t* out, int64_t ld, int row_base, int mrows, int n0,
                                                    Acc<Cfg>& t, char* epi) {
  if constexpr (Cfg::RN % 2 == 0 && Cfg::STAGE_BYTES >= Cfg::NW * 4096)
    store_rows_bf16_stage<Cfg>(out, ld, row_base, mrows, n0, t, epi);
  else
    store_rows_bf16<Cfg>(out, ld, row_base, mrows, n0, t, epi);
}

// ================================================================== down-proj
// AGG selects how Y meets the aggregation (the paper's comparison of
// expert-aggregation strategies): kAggGather stores Y expert-major for the
// gather-and-sum O kernel (the layer's path); kAggScatter stores each row at
// its token-major position (a.dst[row]) for a contiguous sum; kAggAtomic adds
// s * Y into an fp32 O with atomics (a.O32, a.row_token, a.row_w) and
// stores no Y.  The last two exist for the ablation only.
enum { kAggGather = 0, kAggScatter = 1, kAggAtomic = 2 };
template <class Cfg_, int AGG = kAggGather>
struct OpDown {
  using Cfg = Cfg_;
  static constexpr int M_MODE = ROWS, N_MODE = KOUTER;
  struct Params { DownArgs a; };
  static constexpr int EPI_LDS = kStagedStores<Cfg> ? Cfg::NW * kStageBytesPerWave : 0;
  static constexpr int EPI_STORES = kStoresPerFullTile<Cfg>;
  static __device__ int count(const Params& p, int* sh) {
    return count_varlen_m<Cfg::BN>(p.a.mtiles, p.a.d);
  }
  static __device__ int count_tail(const Params& p, const int* sh) {
    return count_varlen_m_tail<Cfg::BN>(p.a.mtiles, p.a.d);
  }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int* sh) {
    return tile_varlen_m<Cfg::BM, Cfg::BN>(p.a.mtiles, p.a.d, p.a.n, id, ti);
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, RowsSide<Cfg::BM, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.A, p.a.n, nullptr, ti.row_base, ti.mrows);
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BN, Cfg::BK, Cfg::NW>& s) {
    const uint16_t* w = p.a.W2 + (size_t)ti.e * p.a.n * p.a.d;
    s.init(w, p.a.d, nullptr, 0, p.a.n, p.a.d, ColOffset{ti.n0});
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char* epi) {
    if (p.a.b2) add_col_bias<Cfg>(t, p.a.b2 + (size_t)ti.e * p.a.d, ColOffset{ti.n0});
    if constexpr (AGG == kAggGather) {
      store_rows_bf16_any<Cfg>(p.a.Y, p.a.d, ti.row_base, ti.mrows, ti.n0, t, epi);
    } else if constexpr (AGG == kAggScatter) {
      static_assert(Cfg::RN % 2 == 0 && Cfg::STAGE_BYTES >= Cfg::NW * 4096, "staged rows");
      char* st = epi - Cfg::STAGE_BYTES + (threadIdx.x >> 6) * 4096;
      const int wm0 = t.m_of(0) - (threadIdx.x & 31);
#pragma unroll
      for (int i = 0; i < Cfg::RM; ++i) {
        const int m0 = wm0 + 32 * i;
        if (m0 >= ti.mrows) continue;
#pragma unroll
        for (int j = 0; j + 1 < Cfg::RN; j += 2) {
          u32x2 v0[4], v1[4];
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            v0[g] = pack_bf16x4(t.acc[i][j][4 * g], t.acc[i][j][4 * g + 1], t.acc[i][j][4 * g + 2],
                                t.acc[i][j][4 * g + 3]);
            v1[g] = pack_bf16x4(t.acc[i][j + 1][4 * g], t.acc[i][j + 1][4 * g + 1], t.acc[i][j + 1][4 * g + 2],
                                t.acc[i][j + 1][4 * g + 3]);
          }
          const int col = ti.n0 + t.n_of(j, 0) - 4 * ((threadIdx.x >> 5) & 1);
          stage_block32(st, 0, v0);
          stage_block32(st, 1, v1);
          store_staged32_scatter(st, p.a.Y, p.a.d, col, p.a.dst + ti.row_base + m0, ti.mrows - m0);
        }
      }
    } else {
      // fp32 atomics: O32[t][c] += s * bf16(Y) (Y rounded as the stored Y would be)
#pragma unroll
      for (int i = 0; i < Cfg::RM; ++i) {
        const int m = t.m_of(i);
        if (m >= ti.mrows) continue;
        const int row = ti.row_base + m;
        const float w = p.a.row_w[row];
        float* o = p.a.O32 + (size_t)p.a.row_token[row] * p.a.d + ti.n0;
#pragma unroll
        for (int j = 0; j < Cfg::RN; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float y = bf2f(f2bf(t.acc[i][j][4 * g + r]));
              unsafeAtomicAdd(o + t.n_of(j, g) + r, w * y);
            }
      }
    }
  }
};

// ================================================================== dH
// Epilogue (down-proj backward): with A recomputed from the cached H,
// dS = <dA', A> (reduced over this tile's n columns), dA = s dA',
// dH = dSwiGLU(dA, H), A' = s A.
template <class Cfg_>
struct OpDH {
  using Cfg = Cfg_;
  static constexpr int M_MODE = ROWS, N_MODE = ROWS;
  struct Params { DHArgs a; };
  static constexpr int RED_LDS = Cfg::BM * Cfg::WN * 4;  // dS partial sums [BM][WN]
  static constexpr int IDX_LDS = Cfg::NW * Cfg::QM * 256;  // gathered dO rows of the next tile
  // dH gate, dH up and A' leave as whole 128-byte lines through
  // wave-private LDS staging where the LDS allows it
  static constexpr bool STAGED = Cfg::RN % 2 == 0 && Cfg::STAGE_BYTES >= Cfg::NW * 8192 &&
                                 Cfg::LDS_BYTES + RED_LDS + Cfg::NW * kStageBytesPerWave + IDX_LDS <= 160 * 1024;
  static constexpr int EPI_LDS = RED_LDS + (STAGED ? Cfg::NW * kStageBytesPerWave : 0);
  // full tile: staged, four stores per output and 64-column row block;
  // direct, two per output and 32 x 32 block
  static constexpr int EPI_STORES = STAGED ? Cfg::RM * (Cfg::RN / 2) * 12 : Cfg::RM * Cfg::RN * 6;
  static __device__ int count(const Params& p, int* sh) {
    return count_varlen_m<Cfg::BN>(p.a.mtiles, p.a.n);
  }
  static __device__ int count_tail(const Params& p, const int* sh) {
    return count_varlen_m_tail<Cfg::BN>(p.a.mtiles, p.a.n);
  }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int* sh) {
    return tile_varlen_m<Cfg::BM, Cfg::BN>(p.a.mtiles, p.a.n, p.a.d, id, ti);
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, RowsSide<Cfg::BM, Cfg::BK, Cfg::NW, true>& s) {
    s.init(p.a.dO, p.a.d, p.a.row_token, ti.row_base, ti.mrows);
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, RowsSide<Cfg::BN, Cfg::BK, Cfg::NW>& s) {
    // rows of W2_e [n][d] are the n columns of dA', with d contiguous
    s.init(p.a.W2 + (size_t)ti.e * p.a.n * p.a.d, p.a.d, nullptr, ti.n0, Cfg::BN);
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char* smem) {
    constexpr int RM = Cfg::RM, RN = Cfg::RN;
    const int n = p.a.n;
    const int lane = epilogue_lane();
    const int wn = t.wave_n();
    const int wm0 = Cfg::wave_m(threadIdx.x >> 6) * (Cfg::BM / Cfg::WM);
    auto m_of = [&](int i) { return wm0 + 32 * i + (lane & 31); };
    // first column of accumulator block j
    auto col_of = [&](int j) { return ti.n0 + wn * (Cfg::BN / Cfg::WN) + 32 * j; };
    float* red = (float*)smem;  // [BM][WN], the epilogue's own LDS
    // H values (gate and up halves) of one 32 x 32 accumulator block,
    // double-buffered over the blocks in (i, j) order: the loads of the next
    // block are in flight while this one is computed and stored.
    float swr[RM];
#pragma unroll
    for (int i = 0; i < RM; ++i) {
      const int m = m_of(i);
      swr[i] = m < ti.mrows ? p.a.row_w[(size_t)(ti.row_base + m)] : 0.f;
    }
    u32x2 hg[2][4], hu[2][4];
    auto load_block = [&](int blk, int b) {
      const int i = blk / RN, j = blk % RN;
      const int m = m_of(i);
      const size_t row = (size_t)(ti.row_base + (m < ti.mrows ? m : 0));
      const uint16_t* h = p.a.H + row * (2 * n);
      const int col = col_of(j);
      load_block_bf16(h + col, hg[b]);
      load_block_bf16(h + n + col, hu[b]);
    };
    load_block(0, 0);
    float part = 0.f;
#pragma unroll
    for (int blk = 0; blk < RM * RN; ++blk) {
      const int i = blk / RN, j = blk % RN, b = blk & 1;
      if (blk + 1 < RM * RN) load_block(blk + 1, b ^ 1);
      const int m = m_of(i);
      const bool valid = m < ti.mrows;
      const size_t row = (size_t)(ti.row_base + (valid ? m : 0));
      const float s = swr[i];
      if (j == 0) part = 0.f;
      if constexpr (STAGED) {
        // dH gate and up of block j go to the wave's 8 KB of the last stage
        // buffer at once (no DMA writes it before the next tile's first
        // barrier); A' of the even block waits in the wave's 2 KB of the
        // epilogue area, the odd one in the gate area once that is stored.
        const int m0 = wm0 + 32 * i;
        if (m0 < ti.mrows) {
          u32x2 vg[4], vu[4], va[4];
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const float gv[4] = {bf_lo(hg[b][g][0]), bf_hi(hg[b][g][0]), bf_lo(hg[b][g][1]), bf_hi(hg[b][g][1])};
            const float uv[4] = {bf_lo(hu[b][g][0]), bf_hi(hu[b][g][0]), bf_lo(hu[b][g][1]), bf_hi(hu[b][g][1])};
            float dg[4], du[4], apv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float dap = t.acc[i][j][4 * g + r];
              float sg;
              const float sl = silu_sig(gv[r], &sg);
              const float av = sl * uv[r];
              part += dap * av;
              const float da = s * dap;
              dg[r] = da * uv[r] * sg * (1.f + gv[r] * (1.f - sg));
              du[r] = da * sl;
              apv[r] = s * av;
            }
            vg[g] = pack_bf16x4(dg[0], dg[1], dg[2], dg[3]);
            vu[g] = pack_bf16x4(du[0], du[1], du[2], du[3]);
            va[g] = pack_bf16x4(apv[0], apv[1], apv[2], apv[3]);
          }
          char* st = smem - Cfg::STAGE_BYTES + (threadIdx.x >> 6) * 8192;
          char* wh = smem + RED_LDS + (threadIdx.x >> 6) * kStageBytesPerWave;
          stage_block32(st, j % 2, vg);
          stage_block32(st + 4096, j % 2, vu);
          if (j % 2 == 0) {
            stage_half32(wh, va);
          } else {
            const size_t r0 = (size_t)(ti.row_base + m0);
            const int col = col_of(j - 1), rv = ti.mrows - m0;
            store_staged32(st, p.a.dH + r0 * (2 * n) + col, 2 * n, rv);
            store_staged32(st + 4096, p.a.dH + r0 * (2 * n) + n + col, 2 * n, rv);
            // the gate area is free again: A' of this block joins the even one
            stage_block32(st, 1, va);
            store_staged32_split(wh, st, p.a.Ap + r0 * n + col, n, rv);
          }
        }
      } else if (valid) {
        uint16_t* dh = p.a.dH + row * (2 * n);
        uint16_t* ap = p.a.Ap + row * n;
        const int col = col_of(j);
        u32x2 vg[4], vu[4], va[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float gv[4] = {bf_lo(hg[b][g][0]), bf_hi(hg[b][g][0]), bf_lo(hg[b][g][1]), bf_hi(hg[b][g][1])};
          const float uv[4] = {bf_lo(hu[b][g][0]), bf_hi(hu[b][g][0]), bf_lo(hu[b][g][1]), bf_hi(hu[b][g][1])};
          float dg[4], du[4], apv[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float dap = t.acc[i][j][4 * g + r];
            float sg;
            const float sl = silu_sig(gv[r], &sg);
            const float av = sl * uv[r];
            part += dap * av;
            const float da = s * dap;
            dg[r] = da * uv[r] * sg * (1.f + gv[r] * (1.f - sg));
            du[r] = da * sl;
            apv[r] = s * av;
          }
          vg[g] = pack_bf16x4(dg[0], dg[1], dg[2], dg[3]);
          vu[g] = pack_bf16x4(du[0], du[1], du[2], du[3]);
          va[g] = pack_bf16x4(apv[0], apv[1], apv[2], apv[3]);
        }
        store_block_bf16(dh + col, vg);
        store_block_bf16(dh + n + col, vu);
        store_block_bf16(ap + col, va);
      }
      if (j == RN - 1) {
        float q = part + __shfl_xor(part, 32, kWave);
        if (lane < 32) red[m * Cfg::WN + wn] = q;
      }
    }
    barrier_lds();
    const int nnt = n / Cfg::BN;
    const int nt = ti.n0 / Cfg::BN;
    for (int m = threadIdx.x; m < ti.mrows; m += Cfg::THREADS) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < Cfg::WN; ++w) v += red[m * Cfg::WN + w];
      const size_t row = (size_t)(ti.row_base + m);
      if (p.a.bq && nt == 0) {
        // + <dO_t, b2_e> (expert bias of the down-projection), high part then low part
        const float* q = p.a.bq + (size_t)p.a.row_token[row] * (2 * p.a.E);
        v += q[ti.e] + q[p.a.E + ti.e];
      }
      if (nnt == 1)
        p.a.dS[row] = v;
      else
        p.a.dS_part[row * nnt + nt] = v;
    }
  }
};

// ================================================================== dX~
template <class Cfg_>
struct OpDXt {
  using Cfg = Cfg_;
  static constexpr int M_MODE = ROWS, N_MODE = ROWS;
  struct Params { DXtArgs a; };
  static constexpr int EPI_LDS = kStagedStores<Cfg> ? Cfg::NW * kStageBytesPerWave : 0;
  static constexpr int EPI_STORES = kStoresPerFullTile<Cfg>;
  static __device__ int count(const Params& p, int* sh) {
    return count_varlen_m<Cfg::BN>(p.a.mtiles, p.a.d);
  }
  static __device__ int count_tail(const Params& p, const int* sh) {
    return count_varlen_m_tail<Cfg::BN>(p.a.mtiles, p.a.d);
  }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int* sh) {
    return tile_varlen_m<Cfg::BM, Cfg::BN>(p.a.mtiles, p.a.d, 2 * p.a.n, id, ti);
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, RowsSide<Cfg::BM, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.dH, 2 * p.a.n, nullptr, ti.row_base, ti.mrows);
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, RowsSide<Cfg::BN, Cfg::BK, Cfg::NW>& s) {
    // rows of W1_e [d][2n] are the d columns of dX~, with 2n contiguous
    s.init(p.a.W1 + (size_t)ti.e * p.a.d * (2 * p.a.n), 2 * p.a.n, nullptr, ti.n0, Cfg::BN);
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char* epi) {
    store_rows_bf16_any<Cfg>(p.a.dXt, p.a.d, ti.row_base, ti.mrows, ti.n0, t, epi);
  }
};

// ================================================================== weight gradients (varlen-K)
// dW2_e[n,d] = A'_e^T gather(dO): M = n (A' columns), N = d (dO columns)
template <class Cfg_>
struct OpDW2 {
  using Cfg = Cfg_;
  static constexpr int M_MODE = KOUTER, N_MODE = KOUTER;
  struct Params { DW2Args a; };
  static constexpr int EPI_LDS = kStagedStores<Cfg> ? Cfg::NW * kStageBytesPerWave : 0;
  static __device__ int count(const Params& p, int*) { return ((const SMOE_CONST int32_t*)p.a.klist)[3]; }
  static __device__ void xcd_range(const Params& p, int x, int* begin, int* cnt) {
    kchunk_xcd_range(p.a.klist, x, begin, cnt);
  }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int*) {
    return tile_kchunk<Cfg::BM, Cfg::BN>(p.a.klist, p.a.E, p.a.n, p.a.d, id, ti);
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BM, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.Ap, p.a.n, nullptr, ti.k_begin, ti.k_len, p.a.n, ColOffset{ti.m0});
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BN, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.dO, p.a.d, p.a.row_token, ti.k_begin, ti.k_len, p.a.d, ColOffset{ti.n0});
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char* epi) {
    if (ti.row_base >= 0)
      store_part_f32<Cfg>(p.a.part + (size_t)ti.row_base * p.a.n * p.a.d, p.a.d, ti.m0, ti.n0, t);
    else
      store_rows_bf16_any<Cfg>(p.a.dW2 + (size_t)ti.e * p.a.n * p.a.d, p.a.d, ti.m0, Cfg::BM, ti.n0, t, epi);
  }
};

// dW1_e[d,2n] = gather(X)_e^T dH_e: M = d (X columns), N = 2n (dH columns)
template <class Cfg_>
struct OpDW1 {
  using Cfg = Cfg_;
  static constexpr int M_MODE = KOUTER, N_MODE = KOUTER;
  struct Params { DW1Args a; };
  static constexpr int EPI_LDS = kStagedStores<Cfg> ? Cfg::NW * kStageBytesPerWave : 0;
  static __device__ int count(const Params& p, int*) { return ((const SMOE_CONST int32_t*)p.a.klist)[3]; }
  static __device__ void xcd_range(const Params& p, int x, int* begin, int* cnt) {
    kchunk_xcd_range(p.a.klist, x, begin, cnt);
  }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int*) {
    return tile_kchunk<Cfg::BM, Cfg::BN>(p.a.klist, p.a.E, p.a.d, 2 * p.a.n, id, ti);
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BM, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.X, p.a.d, p.a.row_token, ti.k_begin, ti.k_len, p.a.d, ColOffset{ti.m0});
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BN, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.dH, 2 * p.a.n, nullptr, ti.k_begin, ti.k_len, 2 * p.a.n, ColOffset{ti.n0});
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char* epi) {
    if (ti.row_base >= 0)
      store_part_f32<Cfg>(p.a.part + (size_t)ti.row_base * p.a.d * (2 * p.a.n), 2 * p.a.n, ti.m0, ti.n0, t);
    else
      store_rows_bf16_any<Cfg>(p.a.dW1 + (size_t)ti.e * p.a.d * (2 * p.a.n), 2 * p.a.n, ti.m0, Cfg::BM, ti.n0, t, epi);
  }
};

// dW_r[d,E] = X^T dL, split over token chunks into fp32 partials
template <class Cfg_>
struct OpDWr {
  using Cfg = Cfg_;
  static constexpr int M_MODE = KOUTER, N_MODE = KOUTER;
  static constexpr int EPI_LDS = 0;
  struct Params { DWrArgs a; };
  static __device__ int count(const Params& p, int*) {
    return p.a.splits * (p.a.d / Cfg::BM) * ((p.a.E + Cfg::BN - 1) / Cfg::BN);
  }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int*) {
    const int mtn = p.a.d / Cfg::BM, ntn = (p.a.E + Cfg::BN - 1) / Cfg::BN;
    const int split = id / (mtn * ntn), rem = id % (mtn * ntn);
    ti.e = split;
    ti.m0 = (rem / ntn) * Cfg::BM;
    ti.n0 = (rem % ntn) * Cfg::BN;
    ti.mrows = Cfg::BM;
    ti.row_base = 0;
    const int chunk = (((p.a.T + p.a.splits - 1) / p.a.splits) + Cfg::BK - 1) / Cfg::BK * Cfg::BK;
    ti.k_begin = split * chunk;
    ti.k_len = max(0, min(chunk, p.a.T - ti.k_begin));
    return true;
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BM, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.X, p.a.d, nullptr, ti.k_begin, ti.k_len, p.a.d, ColOffset{ti.m0});
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BN, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.dL, p.a.E, nullptr, ti.k_begin, ti.k_len, p.a.E, ColOffset{ti.n0});
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char*) {
    float* out = p.a.part + (size_t)ti.e * p.a.d * p.a.E;
#pragma unroll
    for (int i = 0; i < Cfg::RM; ++i) {
      const int m = t.m_of(i);
      float* o = out + (size_t)(ti.m0 + m) * p.a.E;
#pragma unroll
      for (int j = 0; j < Cfg::RN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = ti.n0 + t.n_of(j, g);
          if (col >= p.a.E) continue;
          f32x4 v;
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = t.acc[i][j][4 * g + q];
          *(f32x4*)(o + col) = v;
        }
    }
  }
};

// ================================================================== launchers
// One persistent workgroup per CU (the grid is a multiple of 8 for the XCD
// split), fewer when there are fewer tiles than CUs.
static int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

template <class Op>
static hipError_t run(const typename Op::Params& p, int tiles_bound, hipStream_t s) {
  if (tiles_bound <= 0) return hipSuccess;
  using Cfg = typename Op::Cfg;
  const int grid = (std::min(tiles_bound, cu_count() * Cfg::OCC) + 7) & ~7;
  grouped_gemm_kernel<Op><<<dim3(grid), dim3(Cfg::THREADS), 0, s>>>(p);
  return hipGetLastError();
}

static int pad8(int g) { return (g + 7) & ~7; }
// upper bound of sum_e ceil(count_e / BM) given sum_e count_e <= capacity
static int mtiles_bound(int capacity, int E, int BM) { return capacity / BM + E; }

// tile configurations <BM, BN, WM, WN, STAGES>; varlen-M GEMMs use BM = 256
using C256x256 = GemmCfg<256, 256, 2, 4, 2>;
using C256x256w = GemmCfg<256, 256, 4, 2, 2>;  // 64 x 128 per wave (up, dH, dX~: measured faster)
// the split ring (M rows two steps ahead) for the GEMMs that gather nothing
using C256x256s = GemmCfg<256, 256, 2, 4, 2, kBK, 1, true>;
using C256x256ws = GemmCfg<256, 256, 4, 2, 2, kBK, 1, true>;
using C256x128 = GemmCfg<256, 128, 4, 2, 3>;
using C256x64 = GemmCfg<256, 64, 8, 1, 3>;
using C128x256 = GemmCfg<128, 256, 2, 4, 3>;
// the router and router-gradient GEMMs stream X once (no operand reuse across
// tiles): four 64-deep stages keep three in flight (router 31 -> 28 us, dW_r
// 31 -> 27 us at 7B against three stages)
using C128x128 = GemmCfg<128, 128, 4, 2, 4>;
using C128x64 = GemmCfg<128, 64, 4, 2, 4>;

hipError_t launch_router_gemm(const RouterGemmArgs& a, hipStream_t s) {
  const int mt = (a.T + 255) / 256;
  if (a.E <= 64 && mt < cu_count()) return run<OpRouter<C128x64>>({a}, (a.T + 127) / 128, s);
  if (a.E <= 64) return run<OpRouter<C256x64>>({a}, mt, s);
  // 128-row tiles while 256-row tiles would leave CUs idle
  if (a.E <= 128 && mt < 2 * cu_count()) return run<OpRouter<C128x128>>({a}, (a.T + 127) / 128, s);
  if (a.E <= 128) return run<OpRouter<C256x128>>({a}, mt, s);
  if (mt * ((a.E + 255) / 256) < cu_count())
    return run<OpRouter<C128x256>>({a}, (a.T + 127) / 128 * ((a.E + 255) / 256), s);
  return run<OpRouter<C256x256>>({a}, mt * ((a.E + 255) / 256), s);
}

bool router_topk_fusable(int E, int K) { return E % 8 == 0 && E <= 256 && K <= 8; }

// 128 x 256 tiles for E in (128, 256]: 64 rows x 64 columns per wave (two
// row blocks of 32 values per lane, handled one after the other), two stages
// (the epilogue's LDS does not fit a third)
using C128x256r = GemmCfg<128, 256, 2, 4, 2>;

hipError_t launch_router_topk(const RouterTopkArgs& a, hipStream_t s) {
  if (!router_topk_fusable(a.E, a.K)) return hipErrorInvalidValue;
  const int tiles = (a.T + 127) / 128;
  if (a.E == 64) return run<OpRouterTopk<C128x64, 8, true>>({a}, tiles, s);
  if (a.E < 64) return run<OpRouterTopk<C128x64, 8, false>>({a}, tiles, s);
  if (a.E == 128) return run<OpRouterTopk<C128x128, 8, true>>({a}, tiles, s);
  if (a.E < 128) return run<OpRouterTopk<C128x128, 8, false>>({a}, tiles, s);
  if (a.E == 256) return run<OpRouterTopk<C128x256r, 8, true>>({a}, tiles, s);
  return run<OpRouterTopk<C128x256r, 8, false>>({a}, tiles, s);
}

hipError_t launch_up(const UpArgs& a, hipStream_t s) {
  const int N = 2 * a.n;
  if (a.n % 128 == 0) return run<OpUp<C256x256w>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (N / 256)), s);
  return run<OpUp<C256x128>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (N / 128)), s);  // n % 64
}

hipError_t launch_down(const DownArgs& a, hipStream_t s) {
  if (a.d % 256 == 0) return run<OpDown<C256x256s>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (a.d / 256)), s);
  return run<OpDown<C256x128>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (a.d / 128)), s);
}

hipError_t launch_down_ablation(const DownArgs& a, int strategy, hipStream_t s) {
  const int g256 = pad8(mtiles_bound(a.capacity, a.E, 256) * (a.d / 256));
  const int g128 = pad8(mtiles_bound(a.capacity, a.E, 256) * (a.d / 128));
  if (strategy == kAggScatter) {
    if (a.d % 256 == 0) return run<OpDown<C256x256, kAggScatter>>({a}, g256, s);
    return run<OpDown<C256x128, kAggScatter>>({a}, g128, s);
  }
  if (strategy == kAggAtomic) {
    if (a.d % 256 == 0) return run<OpDown<C256x256, kAggAtomic>>({a}, g256, s);
    return run<OpDown<C256x128, kAggAtomic>>({a}, g128, s);
  }
  return launch_down(a, s);
}

static int dh_bn(int n) { return n % 256 == 0 ? 256 : (n % 128 == 0 ? 128 : 64); }
int dh_n_tiles(int n) { return n / dh_bn(n); }

hipError_t launch_dh(const DHArgs& a, hipStream_t s) {
  const int grid = pad8(mtiles_bound(a.capacity, a.E, 256) * dh_n_tiles(a.n));
  switch (dh_bn(a.n)) {
    case 256: return run<OpDH<C256x256w>>({a}, grid, s);
    case 128: return run<OpDH<C256x128>>({a}, grid, s);
    default: return run<OpDH<C256x64>>({a}, grid, s);
  }
}

hipError_t launch_dxt(const DXtArgs& a, hipStream_t s) {
  if (a.d % 256 == 0) return run<OpDXt<C256x256ws>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (a.d / 256)), s);
  return run<OpDXt<C256x128>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (a.d / 128)), s);
}

// varlen-K GEMMs gather their k rows: two stages (the row indices of the next
// stage are fetched one step ahead into registers)
using W256x256 = GemmCfg<256, 256, 2, 4, 2>;
using W128x256 = GemmCfg<128, 256, 2, 4, 2>;
using W64x256 = GemmCfg<64, 256, 2, 4, 2>;
using W128x128 = GemmCfg<128, 128, 4, 2, 2>;
using W64x128 = GemmCfg<64, 128, 2, 4, 2>;

// slabs of one weight-gradient GEMM: at most kDwSlabs, within kDwSlabBytes
int dw_slabs(int64_t mn) {
  const int64_t b = kDwSlabBytes / (mn * 4);
  return (int)std::min<int64_t>(kDwSlabs, b) & ~1;
}
size_t dw_part_bytes(int d, int n) {
  const int64_t mn = (int64_t)d * n;
  return (size_t)std::max<int64_t>(dw_slabs(2 * mn) * 2 * mn, dw_slabs(mn) * mn) * 4;
}

// tile shapes of the weight-gradient GEMMs (their k-chunk lists are built
// for these shapes); dW2: M = n, N = d; dW1: M = d, N = 2n
static void dw2_tile(int d, int n, int* bm, int* bn) {
  *bn = d % 256 == 0 ? 256 : 128;
  *bm = (*bn == 256 && n % 256 == 0) ? 256 : (n % 128 == 0 ? 128 : 64);
}
static void dw1_tile(int d, int n, int* bm, int* bn) {
  *bm = *bn = (d % 256 == 0 && (2 * n) % 256 == 0) ? 256 : 128;
}

hipError_t launch_bwd_lists(const int32_t* offsets, int E, int d, int n, int32_t* mtiles, int32_t* klist2,
                            int32_t* klist1, const uint16_t* Wr, uint16_t* WrT, hipStream_t s) {
  if (E > 4096) return hipErrorInvalidValue;
  int bm2, bn2, bm1, bn1;
  dw2_tile(d, n, &bm2, &bn2);
  dw1_tile(d, n, &bm1, &bn1);
  const int tpe2 = (n / bm2) * (d / bn2), tpe1 = (d / bm1) * (2 * n / bn1);
  const int tr_blocks = Wr ? (d * E + kMTilesThreads - 1) / kMTilesThreads : 0;
  bwd_lists_kernel<<<3 + tr_blocks, kMTilesThreads, 0, s>>>(offsets, E, mtiles, tpe2, dw_slabs((int64_t)n * d), klist2,
                                                           tpe1, dw_slabs((int64_t)d * 2 * n), klist1, Wr, WrT, d);
  return hipGetLastError();
}

// the GEMM over the k-chunk list, then (if reduce) the partials of split experts
template <class Op, class Args>
static hipError_t run_dw(const Args& a, int M, int N, uint16_t* dW, bool reduce, hipStream_t s) {
  using Cfg = typename Op::Cfg;
  const int tpe = (M / Cfg::BM) * (N / Cfg::BN);
  const int slabs = dw_slabs((int64_t)M * N);
  hipError_t err = run<Op>({a}, pad8((a.E + slabs) * tpe), s);
  if (err != hipSuccess || !reduce) return err;
  return launch_dw_reduce(a.klist, a.part, dW, a.E, (int64_t)M * N, slabs, s);
}

hipError_t launch_dw2(const DW2Args& a, hipStream_t s) {
  int bm, bn;
  dw2_tile(a.d, a.n, &bm, &bn);
  if (bn == 256) {
    if (bm == 256) return run_dw<OpDW2<W256x256>>(a, a.n, a.d, a.dW2, true, s);
    if (bm == 128) return run_dw<OpDW2<W128x256>>(a, a.n, a.d, a.dW2, true, s);
    return run_dw<OpDW2<W64x256>>(a, a.n, a.d, a.dW2, true, s);
  }
  if (bm == 128) return run_dw<OpDW2<W128x128>>(a, a.n, a.d, a.dW2, true, s);
  return run_dw<OpDW2<W64x128>>(a, a.n, a.d, a.dW2, true, s);
}

hipError_t launch_dw1(const DW1Args& a, hipStream_t s) {
  int bm, bn;
  dw1_tile(a.d, a.n, &bm, &bn);
  // its split experts are summed by launch_bwd_final_reduce
  if (bm == 256) return run_dw<OpDW1<W256x256>>(a, a.d, 2 * a.n, a.dW1, false, s);
  return run_dw<OpDW1<W128x128>>(a, a.d, 2 * a.n, a.dW1, false, s);
}

hipError_t launch_bwd_final_reduce(const int32_t* klist1, const float* part1, uint16_t* dW1, int d, int n,
                                   const float* dwr_part, float* dWr, int splits, const float* cs_part, float* dbias,
                                   int T, int E, hipStream_t s) {
  const int64_t MN1 = (int64_t)d * 2 * n;
  int gx1, gy1;
  dw_reduce_grid(MN1, dw_slabs(MN1), &gx1, &gy1);
  const int nr = dWr ? (d * E + 255) / 256 : 0, ne = dbias ? E : 0;
  const int blocks = gx1 * gy1 + nr + ne;
  if (blocks == 0) return hipSuccess;
  bwd_final_reduce_kernel<<<dim3(blocks), dim3(256), 0, s>>>(klist1, part1, dW1, MN1, gx1, gy1, dwr_part, dWr, d * E,
                                                             splits, nr, cs_part, dbias, colsum_chunks(T), E);
  return hipGetLastError();
}

int dwr_splits(int T, int d, int E) {
  // the output tiles of launch_dwr's configuration: 128 x 64, 128 x 128 or 128 x 256
  const int tiles = (d / 128) * (E <= 128 ? 1 : (E + 255) / 256);
  int s = 256 / tiles;  // at most one tile per CU: a second round would double the time
  const int max_s = (T + 255) / 256;  // at least 256 tokens per split
  if (s > max_s) s = max_s;
  return s < 1 ? 1 : s;
}

hipError_t launch_dwr(const DWrArgs& a, hipStream_t s) {
  hipError_t err;
  const int mtn = a.d / 128;
  if (a.E <= 64)
    err = run<OpDWr<C128x64>>({a}, a.splits * mtn, s);
  else if (a.E <= 128)
    err = run<OpDWr<C128x128>>({a}, a.splits * mtn, s);
  else
    err = run<OpDWr<C128x256>>({a}, a.splits * mtn * ((a.E + 255) / 256), s);
  return err;  // the partials are summed by launch_bwd_final_reduce
}

}  // namespace smoe
