// Grouped GEMM core for gfx950: bf16 MFMA (v_mfma_f32_32x32x16_bf16) with
// fp32 accumulation, LDS double buffering and gather-fused operand loads.
//
// The paper builds its whole MoE computation from one grouped GEMM with
// modular fusion plus an aggregation kernel (Section 3.1).  This core is that
// grouped GEMM, written for CDNA4: a 256-thread workgroup (4 wave64, 2 x 2)
// computes a BM x BN tile of C[M,N] = sum_k Mside[m,k] * Nside[n,k].
//
// Both operands are staged in LDS as [rows][64 k] bf16 tiles, k contiguous,
// with the 16-byte chunk index XOR-swizzled by (row & 7) so the fragment reads
// of 32 consecutive rows hit distinct banks.  Operands are fetched in one of
// two source layouts:
//   ROWS   : operand rows with k contiguous in memory (X, dO, A, dH, weight
//            rows of W1/W2 read transposed); rows may be gathered through an
//            index list (the token gather of Section 4.1.1 fused into the load)
//   KOUTER : k is the outer (row) index in memory and the operand's m/n index
//            is contiguous (W1/W2 in the forward, all operands of the weight
//            gradients); a thread loads an 8(k) x 8(m) block with 16-byte
//            loads, transposes it in registers and writes 8 k-contiguous
//            16-byte rows to LDS.  k rows may be gathered (varlen-K weight
//            gradients over an expert's tokens) and are zero-filled past the
//            end of the reduction.
//
// The MFMA is issued as D = Nfrag x Mfrag, so a lane's accumulator holds one
// m (lane % 32) and 16 n values in four runs of 4 consecutive columns; row
// reductions (dS) stay mostly in-lane and stores are 8-byte runs per row.
#pragma once
#include "device_common.h"

namespace smoe {

constexpr int kBK = 64;          // k per LDS stage
constexpr int kRowBytes = 128;   // one LDS tile row: 64 bf16

enum SrcMode { ROWS = 0, KOUTER = 1 };

struct TileInfo {
  int e;        // expert (group)
  int m0;       // first m of the tile inside the group
  int mrows;    // valid m rows in the tile (<= BM)
  int n0;       // first n of the tile
  int row_base; // global row of m = 0 for varlen-M (expert offset + m0)
  int k_begin;  // first k (global row index for varlen-K)
  int k_len;    // reduction length
};

__device__ __forceinline__ int lds_off(int row, int chunk) { return row * kRowBytes + ((chunk ^ (row & 7)) << 4); }

// 8x8 transpose of bf16: in[j] holds 8 consecutive m of k-row j; out[c] holds
// 8 consecutive k of m-column c.
__device__ __forceinline__ void transpose8x8(const u32x4 (&in)[8], u32x4 (&out)[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t a = in[2 * q][c >> 1];
      const uint32_t b = in[2 * q + 1][c >> 1];
      out[c][q] = (c & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
    }
  }
}

// ---------------------------------------------------------------------------
// ROWS loader: R rows x 64 k per stage; thread -> (row = tid/8 + 32p, chunk = tid%8)
template <int R>
struct RowsLoader {
  static constexpr int P = R / 32;
  const char* ptr[P];  // byte pointer to the row start (k = 0)
  u32x4 buf[P];

  __device__ __forceinline__ void stage_load(int k0) {
    const int chunk = threadIdx.x & 7;
#pragma unroll
    for (int p = 0; p < P; ++p) buf[p] = *(const u32x4*)(ptr[p] + (size_t)(k0 + chunk * 8) * 2);
  }
  __device__ __forceinline__ void stage_store(char* lds) const {
    const int chunk = threadIdx.x & 7;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int row = (threadIdx.x >> 3) + 32 * p;
      *(u32x4*)(lds + lds_off(row, chunk)) = buf[p];
    }
  }
};

// KOUTER loader: R (m) x 64 k per stage from a [k][ld] matrix.
// thread -> kb = tid%8 (k rows 8kb..8kb+7), rb = tid/8 (m cols 8rb..8rb+7)
template <int R>
struct KOuterLoader {
  static constexpr bool kActive = true;
  const char* colptr;  // byte pointer to element (k row 0 of the matrix, this thread's m col block), or null
  int64_t ld_bytes;
  const int32_t* gidx; // gathered k rows (index into the matrix rows), or null
  int k_begin, k_len;
  bool active;         // this thread owns an m block inside R and inside the valid columns
  u32x4 raw[8];

  __device__ __forceinline__ void stage_load(int k0) {
    const int kb = threadIdx.x & 7;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = k0 + kb * 8 + j;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (active && k < k_len) {
        const int64_t row = gidx ? (int64_t)gidx[k_begin + k] : (int64_t)(k_begin + k);
        v = *(const u32x4*)(colptr + row * ld_bytes);
      }
      raw[j] = v;
    }
  }
  __device__ __forceinline__ void stage_store(char* lds) const {
    const int kb = threadIdx.x & 7;
    const int r0 = (threadIdx.x >> 3) * 8;
    if (r0 >= R) return;
    u32x4 t[8];
    transpose8x8(raw, t);
#pragma unroll
    for (int c = 0; c < 8; ++c) *(u32x4*)(lds + (r0 + c) * kRowBytes + ((kb ^ c) << 4)) = t[c];
  }
};

template <int BM, int BN>
struct MfmaTile {
  static constexpr int RM = BM / 64;
  static constexpr int RN = BN / 64;
  f32x16 acc[RM][RN];

  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < RM; ++i)
#pragma unroll
      for (int j = 0; j < RN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  }

  // one 64-wide k stage from LDS tiles lm [BM][64] and ln [BN][64]
  __device__ __forceinline__ void compute(const char* lm, const char* ln) {
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int wm = wave & 1, wn = wave >> 1;
    const int r32 = lane & 31, hi = lane >> 5;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int chunk = 2 * s + hi;
      bf16x8 fm[RM], fn[RN];
#pragma unroll
      for (int i = 0; i < RM; ++i) {
        const int row = wm * (BM / 2) + i * 32 + r32;
        fm[i] = *(const bf16x8*)(lm + lds_off(row, chunk));
      }
#pragma unroll
      for (int j = 0; j < RN; ++j) {
        const int row = wn * (BN / 2) + j * 32 + r32;
        fn[j] = *(const bf16x8*)(ln + lds_off(row, chunk));
      }
#pragma unroll
      for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int j = 0; j < RN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fn[j], fm[i], acc[i][j], 0, 0, 0);
    }
  }

  // coordinates of accumulator element (i, j, v) for this lane, tile-local
  __device__ __forceinline__ static int m_of(int i) {
    const int wave = threadIdx.x >> 6;
    return (wave & 1) * (BM / 2) + i * 32 + (threadIdx.x & 31);
  }
  // first of the 4 consecutive columns of group g (v = 4g..4g+3) in block j
  __device__ __forceinline__ static int n_of(int j, int g) {
    const int wave = threadIdx.x >> 6;
    return (wave >> 1) * (BN / 2) + j * 32 + 8 * g + 4 * ((threadIdx.x >> 5) & 1);
  }
};

// XCD-aware remap of the flat workgroup id: workgroups are dispatched to the
// 8 XCDs round-robin, so consecutive logical tiles are handed to the same XCD
// (and share its L2) by mapping id -> (id % 8) * (G / 8) + id / 8.
__device__ __forceinline__ int xcd_remap(int id, int G) {
  if ((G & 7) != 0) return id;
  return (id & 7) * (G >> 3) + (id >> 3);
}

// For varlen-M scheduling: find the expert e and its local m-tile for the
// global m-tile index mt, where expert e owns ceil(count_e / BM) tiles.
// Runs on wave 0; result broadcast through LDS.  Returns false if mt is past
// the last tile.
template <int BM>
__device__ __forceinline__ bool find_m_tile(const int32_t* __restrict__ offsets, int E, int mt, int* sh, TileInfo& ti) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    int base = 0;
    int found_e = -1, found_m0 = 0, found_cnt = 0, found_off = 0;
    for (int e0 = 0; e0 < E; e0 += 64) {
      const int e = e0 + lane;
      int off = 0, cnt = 0;
      if (e < E) {
        off = offsets[e];
        cnt = offsets[e + 1] - off;
      }
      const int nt = (cnt + BM - 1) / BM;
      const int inc = wave_incl_scan(nt);
      const int start = base + inc - nt;
      const bool hit = (e < E) && (mt >= start) && (mt < start + nt);
      const uint64_t b = __ballot(hit);
      if (b) {
        const int src = __ffsll((unsigned long long)b) - 1;
        found_e = __shfl(e, src, kWave);
        found_m0 = (mt - __shfl(start, src, kWave)) * BM;
        found_cnt = __shfl(cnt, src, kWave);
        found_off = __shfl(off, src, kWave);
        break;
      }
      base += __shfl(inc, 63, kWave);
    }
    if (lane == 0) {
      sh[0] = found_e;
      sh[1] = found_m0;
      sh[2] = found_cnt;
      sh[3] = found_off;
    }
  }
  __syncthreads();
  ti.e = sh[0];
  if (ti.e < 0) return false;
  ti.m0 = sh[1];
  ti.mrows = min(BM, sh[2] - sh[1]);
  ti.row_base = sh[3] + sh[1];
  return true;
}

// The main loop shared by every GEMM.  Op supplies:
//   Op::BM, Op::BN, Op::kMinBlocks
//   bool tile(const Params&, TileInfo&, int* sh)     -- scheduling
//   MLoader / NLoader types with stage_load/stage_store, built by
//   make_m(p, ti) / make_n(p, ti)
//   void epilogue(const Params&, const TileInfo&, MfmaTile&, char* smem)
template <class Op>
__global__ __launch_bounds__(256, Op::kMinBlocks) void grouped_gemm_kernel(const typename Op::Params p) {
  constexpr int BM = Op::BM, BN = Op::BN;
  constexpr int kStage = (BM + BN) * kRowBytes;
  __shared__ __attribute__((aligned(16))) char smem[2 * kStage];
  __shared__ int sh[8];
  TileInfo ti;
  if (!Op::tile(p, ti, sh)) return;
  auto ml = Op::make_m(p, ti);
  auto nl = Op::make_n(p, ti);
  MfmaTile<BM, BN> mt;
  mt.zero();
  const int nk = (ti.k_len + kBK - 1) / kBK;
  if (nk > 0) {
    ml.stage_load(0);
    nl.stage_load(0);
    ml.stage_store(smem);
    nl.stage_store(smem + BM * kRowBytes);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      char* cur = smem + (kt & 1) * kStage;
      char* nxt = smem + ((kt + 1) & 1) * kStage;
      const bool more = kt + 1 < nk;
      if (more) {
        ml.stage_load((kt + 1) * kBK);
        nl.stage_load((kt + 1) * kBK);
      }
      mt.compute(cur, cur + BM * kRowBytes);
      if (more) {
        ml.stage_store(nxt);
        nl.stage_store(nxt + BM * kRowBytes);
      }
      __syncthreads();
    }
  }
  Op::epilogue(p, ti, mt, smem);
}

}  // namespace smoe
