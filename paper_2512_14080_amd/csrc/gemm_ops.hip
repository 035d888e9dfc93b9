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
__global__ __launch_bounds__(kMTilesThreads) void mtiles_kernel(const int32_t* __restrict__ offsets, int E,
                                                               int32_t* __restrict__ out) {
  __shared__ int pf[4097], pp[4097];  // per-expert exclusive prefix of full / partial m-tiles
  __shared__ int scan_lds[kMTilesThreads / 64];
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

hipError_t launch_mtiles(const int32_t* offsets, int E, int32_t* out, hipStream_t s) {
  if (E > 4096) return hipErrorInvalidValue;
  mtiles_kernel<<<1, kMTilesThreads, 0, s>>>(offsets, E, out);
  return hipGetLastError();
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

// varlen-K: one tile per (expert, m-tile, n-tile); k = the expert's rows
template <int BM, int BN>
__device__ __forceinline__ bool tile_varlen_k(const int32_t* offsets, int M, int N, int id, TileInfo& ti) {
  const int mtn = M / BM, ntn = N / BN;
  ti.e = id / (mtn * ntn);
  const int rem = id % (mtn * ntn);
  ti.m0 = (rem / ntn) * BM;
  ti.n0 = (rem % ntn) * BN;
  ti.mrows = BM;
  ti.row_base = 0;
  ti.k_begin = offsets[ti.e];
  ti.k_len = offsets[ti.e + 1] - ti.k_begin;
  return true;
}

struct ColOffset {
  int c0;
  __device__ __forceinline__ int operator()(int c) const { return c0 + c; }
};

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
  static constexpr int EPI_LDS = 0;
  static constexpr int IDX_LDS = Cfg::NW * Cfg::QM * 256;  // gathered X rows of the next tile
  // full tile: per row block, H gate, H up and A, two stores each
  static constexpr int EPI_STORES = Cfg::RM * (Cfg::RN / 2) * 6;
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
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char*) {
    constexpr int RN = Cfg::RN;
    const int n = p.a.n;
    const int j0 = (ti.n0 / Cfg::BN) * (Cfg::BN / 2);
    const int wn = t.wave_n();
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

// Row-contiguous stores of a wave's output: the two 32-column accumulator
// blocks j, j+1 of one 32-row block (64 columns, 128 bytes of a bf16 row) go
// through the wave's own 2 KB of LDS, 16 rows at a time, and come back so
// that 8 lanes hold one 128-byte row segment.  Each store instruction then
// writes 8 whole cache lines instead of 32-byte pieces of 32 rows.  The LDS
// operations of one wave complete in order, so no barrier is needed; the
// 16-byte chunk c of staged row r sits at chunk c ^ ((r >> 1) & 7), which
// keeps both the writes (one chunk of 16 rows) and the reads (two whole
// rows per 16 lanes) free of bank conflicts.  The stores are nontemporal:
// these outputs (Y, dX~, the weight gradients) are consumed by a later
// kernel that streams them once, and left in the cache as dirty lines they
// only add write-back traffic at the end of the producing kernel.
constexpr int kStageBytesPerWave = 16 * 128;
template <class Cfg>
constexpr bool kStagedStores = Cfg::RN % 2 == 0 && Cfg::LDS_BYTES + Cfg::NW * kStageBytesPerWave + 256 <= 160 * 1024;
// store instructions per wave of store_rows_bf16 on a full tile: staged, four
// per 64-column row block (two rounds of two); direct, two per 32 columns
template <class Cfg>
constexpr int kStoresPerFullTile = kStagedStores<Cfg> ? Cfg::RM * (Cfg::RN / 2) * 4 : Cfg::RM * Cfg::RN * 2;
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

// ================================================================== down-proj
template <class Cfg_>
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
    store_rows_bf16<Cfg>(p.a.Y, p.a.d, ti.row_base, ti.mrows, ti.n0, t, epi);
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
  static constexpr int EPI_LDS = Cfg::BM * Cfg::WN * 4;  // dS partial sums [BM][WN]
  static constexpr int IDX_LDS = Cfg::NW * Cfg::QM * 256;  // gathered dO rows of the next tile
  // full tile: per 32 x 32 block, dH gate, dH up and A', two stores each
  static constexpr int EPI_STORES = Cfg::RM * Cfg::RN * 6;
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
      if (valid) {
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
    store_rows_bf16<Cfg>(p.a.dXt, p.a.d, ti.row_base, ti.mrows, ti.n0, t, epi);
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
  static __device__ int count(const Params& p, int*) { return p.a.E * (p.a.n / Cfg::BM) * (p.a.d / Cfg::BN); }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int*) {
    return tile_varlen_k<Cfg::BM, Cfg::BN>(p.a.offsets, p.a.n, p.a.d, id, ti);
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BM, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.Ap, p.a.n, nullptr, ti.k_begin, ti.k_len, p.a.n, ColOffset{ti.m0});
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BN, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.dO, p.a.d, p.a.row_token, ti.k_begin, ti.k_len, p.a.d, ColOffset{ti.n0});
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char* epi) {
    store_rows_bf16<Cfg>(p.a.dW2 + (size_t)ti.e * p.a.n * p.a.d, p.a.d, ti.m0, Cfg::BM, ti.n0, t, epi);
  }
};

// dW1_e[d,2n] = gather(X)_e^T dH_e: M = d (X columns), N = 2n (dH columns)
template <class Cfg_>
struct OpDW1 {
  using Cfg = Cfg_;
  static constexpr int M_MODE = KOUTER, N_MODE = KOUTER;
  struct Params { DW1Args a; };
  static constexpr int EPI_LDS = kStagedStores<Cfg> ? Cfg::NW * kStageBytesPerWave : 0;
  static __device__ int count(const Params& p, int*) { return p.a.E * (p.a.d / Cfg::BM) * (2 * p.a.n / Cfg::BN); }
  static __device__ bool tile(const Params& p, int id, TileInfo& ti, int*) {
    return tile_varlen_k<Cfg::BM, Cfg::BN>(p.a.offsets, p.a.d, 2 * p.a.n, id, ti);
  }
  static __device__ void init_m(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BM, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.X, p.a.d, p.a.row_token, ti.k_begin, ti.k_len, p.a.d, ColOffset{ti.m0});
  }
  static __device__ void init_n(const Params& p, const TileInfo& ti, KOuterSide<Cfg::BN, Cfg::BK, Cfg::NW>& s) {
    s.init(p.a.dH, 2 * p.a.n, nullptr, ti.k_begin, ti.k_len, 2 * p.a.n, ColOffset{ti.n0});
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, Acc<Cfg>& t, char* epi) {
    store_rows_bf16<Cfg>(p.a.dW1 + (size_t)ti.e * p.a.d * (2 * p.a.n), 2 * p.a.n, ti.m0, Cfg::BM, ti.n0, t, epi);
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
using C256x128 = GemmCfg<256, 128, 4, 2, 3>;
using C256x64 = GemmCfg<256, 64, 8, 1, 3>;
using C128x256 = GemmCfg<128, 256, 2, 4, 3>;
using C128x128 = GemmCfg<128, 128, 4, 2, 3>;
using C128x64 = GemmCfg<128, 64, 4, 2, 3>;

hipError_t launch_router_gemm(const RouterGemmArgs& a, hipStream_t s) {
  const int mt = (a.T + 255) / 256;
  if (a.E <= 64) return run<OpRouter<C256x64>>({a}, mt, s);
  // 128-row tiles while 256-row tiles would leave CUs idle
  if (a.E <= 128 && mt < 2 * cu_count()) return run<OpRouter<C128x128>>({a}, (a.T + 127) / 128, s);
  if (a.E <= 128) return run<OpRouter<C256x128>>({a}, mt, s);
  return run<OpRouter<C256x256>>({a}, mt * ((a.E + 255) / 256), s);
}

hipError_t launch_up(const UpArgs& a, hipStream_t s) {
  const int N = 2 * a.n;
  if (a.n % 128 == 0) return run<OpUp<C256x256>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (N / 256)), s);
  return run<OpUp<C256x128>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (N / 128)), s);  // n % 64
}

hipError_t launch_down(const DownArgs& a, hipStream_t s) {
  if (a.d % 256 == 0) return run<OpDown<C256x256>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (a.d / 256)), s);
  return run<OpDown<C256x128>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (a.d / 128)), s);
}

static int dh_bn(int n) { return n % 256 == 0 ? 256 : (n % 128 == 0 ? 128 : 64); }
int dh_n_tiles(int n) { return n / dh_bn(n); }

hipError_t launch_dh(const DHArgs& a, hipStream_t s) {
  const int grid = pad8(mtiles_bound(a.capacity, a.E, 256) * dh_n_tiles(a.n));
  switch (dh_bn(a.n)) {
    case 256: return run<OpDH<C256x256>>({a}, grid, s);
    case 128: return run<OpDH<C256x128>>({a}, grid, s);
    default: return run<OpDH<C256x64>>({a}, grid, s);
  }
}

hipError_t launch_dxt(const DXtArgs& a, hipStream_t s) {
  if (a.d % 256 == 0) return run<OpDXt<C256x256>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (a.d / 256)), s);
  return run<OpDXt<C256x128>>({a}, pad8(mtiles_bound(a.capacity, a.E, 256) * (a.d / 128)), s);
}

// varlen-K GEMMs gather their k rows: two stages (the row indices of the next
// stage are fetched one step ahead into registers)
using W256x256 = GemmCfg<256, 256, 2, 4, 2>;
using W128x256 = GemmCfg<128, 256, 2, 4, 2>;
using W64x256 = GemmCfg<64, 256, 2, 4, 2>;
using W128x128 = GemmCfg<128, 128, 4, 2, 2>;
using W64x128 = GemmCfg<64, 128, 2, 4, 2>;

hipError_t launch_dw2(const DW2Args& a, hipStream_t s) {
  // M = n, N = d
  if (a.d % 256 == 0) {
    if (a.n % 256 == 0) return run<OpDW2<W256x256>>({a}, pad8(a.E * (a.n / 256) * (a.d / 256)), s);
    if (a.n % 128 == 0) return run<OpDW2<W128x256>>({a}, pad8(a.E * (a.n / 128) * (a.d / 256)), s);
    return run<OpDW2<W64x256>>({a}, pad8(a.E * (a.n / 64) * (a.d / 256)), s);
  }
  if (a.n % 128 == 0) return run<OpDW2<W128x128>>({a}, pad8(a.E * (a.n / 128) * (a.d / 128)), s);
  return run<OpDW2<W64x128>>({a}, pad8(a.E * (a.n / 64) * (a.d / 128)), s);
}

hipError_t launch_dw1(const DW1Args& a, hipStream_t s) {
  // M = d, N = 2n
  if (a.d % 256 == 0 && (2 * a.n) % 256 == 0)
    return run<OpDW1<W256x256>>({a}, pad8(a.E * (a.d / 256) * (2 * a.n / 256)), s);
  return run<OpDW1<W128x128>>({a}, pad8(a.E * (a.d / 128) * (2 * a.n / 128)), s);
}

int dwr_splits(int T, int d, int E) {
  const int tiles = (d / 128) * ((E + 127) / 128);
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
  if (err != hipSuccess) return err;
  return launch_reduce_rows(a.part, a.dWr, a.d * a.E, a.splits, s);
}

}  // namespace smoe
