// Grouped GEMM core for gfx950: bf16 MFMA (v_mfma_f32_32x32x16_bf16) with
// fp32 accumulation, operands streamed HBM -> LDS by direct (LDS-DMA) loads.
//
// The paper builds its whole MoE computation from one grouped GEMM with
// modular fusion plus an aggregation kernel (Section 3.1).  This core is that
// grouped GEMM written for CDNA4.  A workgroup of 4 or 8 wave64 computes a
// BM x BN tile of C[M,N] = sum_k Mside[m,k] * Nside[n,k]; with 4 waves two
// workgroups share a CU, so one's epilogue overlaps the other's k loop.
//
// Operands never pass through registers on their way to LDS:
// global_load_lds_dwordx4 writes 16 bytes per lane straight into LDS.  The
// LDS layout of a stage is chosen per operand:
//   ROWS   : operand rows with k contiguous in memory (X, dO, A, dH, W rows).
//            LDS tile [rows][BK k], 16-byte chunk index XOR-swizzled by the
//            row so fragment reads are bank-conflict free.  Rows may be gathered through an index
//            list -- the token gather of Section 4.1.1 fused into the load.
//            MFMA fragments are read with ds_read_b128.
//   KOUTER : k is the outer index in memory, m/n contiguous (W1/W2 in the
//            forward, every operand of the weight gradients).  LDS tile
//            [BK k][R], stored as in memory with a 16-byte chunk XOR swizzle
//            on the k row.  MFMA fragments (8 consecutive k of one column)
//            are read with the CDNA4 transposing load ds_read_b64_tr_b16, so
//            no register transpose is needed.  k rows may be gathered
//            (varlen-K weight gradients over an expert's tokens) and rows past
//            the end of the reduction read a zero page.
//
// The k loop keeps STAGES LDS buffers of BK (32 or 64) k each; each step
// waits for its own stage (s_waitcnt vmcnt + s_barrier), then issues the DMA
// for the stage STAGES-1 ahead, then runs the MFMAs, so up to STAGES-1 stages
// of loads are in flight behind the compute, with one barrier per step.  The DMA and the wait are inline
// assembly so the compiler's conservative LDS-DMA tracking does not serialise
// the pipeline; every wait that orders DMA data is explicit here.
//
// The MFMA is issued as D = Nfrag x Mfrag, so a lane's accumulator holds one
// m (lane % 32) and 16 n values in four runs of 4 consecutive columns; row
// reductions (dS) stay mostly in-lane; epilogues regroup the runs for
// 16-byte (or, staged through LDS, whole-row) stores.
#pragma once
#include <type_traits>

#include "device_common.h"

namespace smoe {

constexpr int kBK = 64;  // default k depth of a stage

enum SrcMode { ROWS = 0, KOUTER = 1 };

typedef short v4i16 __attribute__((ext_vector_type(4)));
#define SMOE_LDS __attribute__((address_space(3)))

// read-only zero page for masked k rows / columns of KOUTER operands
__device__ __attribute__((aligned(4096))) uint32_t g_zero_page[1024];

struct TileInfo {
  int e;        // expert (group)
  int m0;       // first m of the tile inside the group
  int mrows;    // valid m rows in the tile (<= BM)
  int n0;       // first n of the tile
  int row_base; // global row of m = 0 for varlen-M (expert offset + m0)
  int k_begin;  // first k (global row index for varlen-K)
  int k_len;    // reduction length
};

// One 16-byte-per-lane LDS DMA.  lds_byte must be wave-uniform: it is the
// instruction's M0 operand, which the "{m0}" constraint has the compiler
// load itself (so M0 is an input it knows about, never a hidden clobber).
__device__ __forceinline__ void dma16(const void* g, uint32_t lds_byte) {
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(lds_byte) : "memory");
}
// The lane index from a volatile asm: per-lane address arithmetic derived
// from it is recomputed where it is used instead of being hoisted out of the
// persistent tile loop, where it would hold registers across the k loop.
__device__ __forceinline__ int volatile_lane() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}
// One 4-byte-per-lane LDS DMA (lane l's dword lands at lds_byte + 4 l).
__device__ __forceinline__ void dma4(const void* g, uint32_t lds_byte) {
  asm volatile("global_load_lds_dword %0, off" ::"v"(g), "{m0}"(lds_byte) : "memory");
}
// Wait until at most N of this wave's vector-memory ops are outstanding, then
// workgroup barrier.  LDS reads of the previous step are complete as well.
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}
__device__ __forceinline__ void barrier_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// BM x BN tile, WM x WN waves (each BM/WM x BN/WN), STAGES LDS buffers of BK
// k, OCC workgroups per CU.  SPLIT: the M side gets one buffer more than the N
// side (STAGES = 2: three M buffers, two N buffers), so its rows are requested
// two steps ahead while the N side (weights, mostly L2 hits) stays one step
// ahead.  Buffer order A0 A1 B0 A2 B1: the last STAGE_BYTES (A2, B1) are the
// ones idle during an epilogue, as the last stage is in the plain layout.
template <int BM_, int BN_, int WM_, int WN_, int STAGES_, int BK_ = kBK, int OCC_ = 1, bool SPLIT_ = false>
struct GemmCfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, STAGES = STAGES_, BK = BK_, OCC = OCC_;
  static constexpr bool SPLIT = SPLIT_;
  static constexpr int NW = WM * WN, THREADS = NW * 64;
  static constexpr int RM = BM / WM / 32, RN = BN / WN / 32;
  static constexpr int SUB = BK / 16;  // MFMA k steps per stage
  static constexpr int M_BYTES = BM * BK * 2, N_BYTES = BN * BK * 2;
  static constexpr int STAGE_BYTES = M_BYTES + N_BYTES;
  static constexpr int A_STAGES = STAGES + (SPLIT ? 1 : 0);
  static constexpr int LDS_BYTES = A_STAGES * M_BYTES + STAGES * N_BYTES;
  static_assert(!SPLIT || STAGES == 2, "the split ring is three M buffers and two N buffers");
  // byte offsets of M buffer st (st < A_STAGES) and N buffer st (st < STAGES)
  static constexpr int a_off(int st) {
    return SPLIT ? (st < 2 ? st * M_BYTES : 2 * M_BYTES + N_BYTES) : st * STAGE_BYTES;
  }
  static constexpr int b_off(int st) {
    return SPLIT ? (st == 0 ? 2 * M_BYTES : 3 * M_BYTES + N_BYTES) : st * STAGE_BYTES + M_BYTES;
  }
  static constexpr int QM = BM * BK / (NW * 512), QN = BN * BK / (NW * 512);  // DMA instructions per wave per stage
  static_assert(BK == 32 || BK == 64, "stage depth");
  static_assert(STAGES >= 2 && STAGES <= 4, "stages");
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
  static_assert(OCC * LDS_BYTES <= 160 * 1024, "LDS of the co-resident workgroups");
  static_assert(RM >= 1 && RN >= 1 && BM % (WM * 32) == 0 && BN % (WN * 32) == 0, "wave tile");
  static_assert(BM % 64 == 0 && BN % 64 == 0, "tile multiple of 64");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");
  // wave w owns rows wave_m(w) * BM/WM .. and columns wave_n(w) * BN/WN ..;
  // waves w and w + 4 share a SIMD and sit in different row blocks, so a
  // tile with only its first rows valid still keeps every SIMD busy
  static __device__ __forceinline__ int wave_m(int w) { return w / WN; }
  static __device__ __forceinline__ int wave_n(int w) { return w % WN; }
};

// ---------------------------------------------------------------- ROWS side
// LDS: [R][BK] bf16, C = BK/8 chunks of 16 bytes per row; chunk c of row r at
// r*2BK + ((c ^ swz(r)) << 4) with swz(r) = (r >> 1) & 7 for BK = 64 and
// (r >> 2) & 3 for BK = 32.  A fragment read (32 rows, one chunk each) is
// served 16 lanes at a time; with this swizzle those 16 lanes hit 16
// different 16-byte bank groups.
// DMA instruction q covers rows (64/C)q .. (64/C)q + 64/C - 1; lane l -> row
// (64/C)q + l/C, physical chunk l%C, logical chunk (l%C) ^ swz(row).
template <int R, int BK, int NW, bool AI = false>
struct RowsSide {
  static constexpr int C = BK / 8;              // chunks per row
  static constexpr int RPI = 64 / C;            // rows per DMA instruction
  static constexpr int Q = R * BK / (NW * 512);  // instructions per wave
  static_assert(Q >= 1 && Q * NW * 512 == R * BK, "rows x k of a stage must be whole DMA instructions per wave");
  static __device__ __forceinline__ int swz(int r) { return BK == 64 ? ((r >> 1) & 7) : ((r >> 2) & 3); }
  const char* ptr[Q];  // row start (k = 0) of the row this lane loads, per instruction (after commit)
  const uint16_t* base_;
  int64_t ld_;
  int32_t row_[Q];     // the row this lane loads, per instruction
  // AI (always-gathered sides): LDS bytes (NW * Q * 256) that receive the
  // tile's row indices by DMA
  uint32_t idx_lds = 0;
  // The rows of a tile: gathered rows are looked up in idx here, but the row
  // pointers are only formed in commit().  With AI the index loads are LDS
  // DMA issued in program order with the stage DMA (inline asm the compiler
  // cannot move), so a next tile's lookups are in flight behind the current
  // tile's stages and land before its last full drain; loaded into registers,
  // the compiler is free to sink them to their use after the k loop, where
  // they would be waited for on the critical path.  With AI, idx must not be
  // null.
  __device__ __forceinline__ void init(const uint16_t* base, int64_t ld, const int32_t* idx, int row_base, int nrows) {
    const int wave = threadIdx.x >> 6, lane = AI ? volatile_lane() : threadIdx.x & 63;
    base_ = base;
    ld_ = ld;
    const uint32_t w = __builtin_amdgcn_readfirstlane(wave);
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      const int lrow = RPI * (wave + NW * j) + lane / C;
      const int r = min(lrow, nrows - 1);
      if constexpr (AI) {
        dma4(idx + row_base + r, idx_lds + (w * Q + j) * 256);
        row_[j] = 0;  // read from LDS in commit()
      } else {
        row_[j] = idx ? idx[row_base + r] : row_base + r;
      }
    }
  }
  // Called where the index loads are known to be complete (after a full
  // drain); the empty asm keeps the pointer arithmetic after that point.
  __device__ __forceinline__ void commit() {
    const int wave = threadIdx.x >> 6, lane = AI ? volatile_lane() : threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      if constexpr (AI) row_[j] = *(const SMOE_LDS int32_t*)(uintptr_t)(idx_lds + (wave * Q + j) * 256 + lane * 4);
      asm volatile("" : "+v"(row_[j]));
      const int lrow = RPI * (wave + NW * j) + lane / C;
      const int logical = (lane % C) ^ swz(lrow);
      ptr[j] = (const char*)(base_ + (int64_t)row_[j] * ld_) + logical * 16;
    }
  }
  // instructions j with j % parts == part (so a stage can be issued in pieces)
  __device__ __forceinline__ void issue(uint32_t lds_side, int k0, int part = 0, int parts = 1) const {
    const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int j = 0; j < Q; ++j)
      if (j % parts == part) dma16(ptr[j] + k0 * 2, lds_side + (w + NW * j) * 1024);
  }
  static __device__ __forceinline__ bf16x8 frag(const char* lds_side, int r0, int s) {
    const int lane = threadIdx.x & 63;
    const int row = r0 + (lane & 31);
    const int c = (2 * s + (lane >> 5)) ^ swz(row);
    return *(const bf16x8*)(lds_side + row * (2 * BK) + c * 16);
  }
};

// --------------------------------------------------------------- KOUTER side
// LDS: [BK k][R] bf16 (2R bytes per k row, L = R/8 chunks), chunk c of row k
// at k*2R + ((c ^ x(k)) << 4) with x(k) = 4*(k%4) for L >= 16 and
// 4*((k/2)%2) for L = 8; with it, the 8 k rows x 64 bytes one transposing
// read touches spread over all banks.
template <int R, int BK, int NW>
struct KOuterSide {
  static constexpr int L = R / 8;
  static constexpr int RPI = 512 / R;            // k rows per DMA instruction
  static constexpr int Q = R * BK / (NW * 512);  // instructions per wave
  static_assert(L >= 8, "R >= 64");
  static_assert(Q >= 1 && Q * NW * 512 == R * BK, "k x columns of a stage must be whole DMA instructions per wave");
  static __device__ __forceinline__ int swz(int k) { return L >= 16 ? 4 * (k & 3) : 4 * ((k >> 1) & 1); }

  const char* base;      // matrix base (bytes)
  int64_t ld_bytes;
  const int32_t* gidx;   // gathered k rows, or null
  int k_begin, k_len;
  int krow[Q];           // tile-local k row this lane loads, per instruction
  int colb[Q];           // byte offset of this lane's 16 bytes within the stored row (or -1: masked column)
  int gnext[Q];          // gathered row index for the next stage to issue

  // colmap(local_col) -> global column of tile-local column local_col (multiple of 8)
  template <class ColMap>
  __device__ __forceinline__ void init(const uint16_t* b, int64_t ld, const int32_t* g, int kb, int kl, int cvalid,
                                       ColMap colmap) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    base = (const char*)b;
    ld_bytes = ld * 2;
    gidx = g;
    k_begin = kb;
    k_len = kl;
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      const int q = wave + NW * j;
      const int row = q * RPI + lane / L;
      const int phys = lane % L;
      const int logical = phys ^ swz(row);
      const int gc = colmap(8 * logical);
      krow[j] = row;
      colb[j] = gc < cvalid ? gc * 2 : -1;
    }
  }
  __device__ __forceinline__ void commit() {}
  // gathered operands: fetch the row indices of the stage at k0 (registers)
  __device__ __forceinline__ void prefetch_idx(int k0) {
    if (!gidx) return;
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      const int k = k0 + krow[j];
      gnext[j] = k < k_len ? gidx[k_begin + k] : 0;
    }
  }
  // Called where the index loads are known to be complete (after a
  // vmcnt(0) wait).  The empty asm redefines the registers, so the compiler
  // sees no pending load behind them later on; otherwise it places its own
  // vmcnt(0) before every use, which also waits for the DMA (invisible to
  // it) issued in between.
  __device__ __forceinline__ void idx_commit() {
#pragma unroll
    for (int j = 0; j < Q; ++j) asm volatile("" : "+v"(gnext[j]));
  }
  // The source address is formed without branches: row and leading
  // dimension are below 2^31 and 2^32, so one 32 x 32 -> 64-bit multiply-add
  // gives the byte offset, and k rows past the reduction (or masked columns)
  // select the zero page instead.
  __device__ __forceinline__ void issue(uint32_t lds_side, int k0, int part = 0, int parts = 1) const {
    const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const uint32_t ld32 = (uint32_t)ld_bytes;
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      if (j % parts != part) continue;
      const int k = k0 + krow[j];
      const uint32_t row = gidx ? (uint32_t)gnext[j] : (uint32_t)(k_begin + k);
      const uint64_t off = (uint64_t)row * ld32 + (uint32_t)colb[j];
      const bool ok = k < k_len && colb[j] >= 0;
      const char* src = ok ? base + off : (const char*)g_zero_page + lane * 16;
      dma16(src, lds_side + (w + NW * j) * 1024);
    }
  }
  static __device__ __forceinline__ bf16x8 frag(const char* lds_side, int c0, int s) {
    // 32 columns c0..c0+31, 8 k (16s + 8*(lane/32) ..) per lane, two transposing reads
    const int lane = threadIdx.x & 63;
    const int g = lane >> 4, i = lane & 15;
    const int m = c0 + 16 * (g & 1) + 4 * (i & 3);
    // this lane's first k row within a sub-step; its rows kb + 16 s and kb + 16 s + 4
    // have the same chunk swizzle (swz depends on bits 0-1 of k, which 16 s and the
    // carry-free + 4 leave alone), so one per-lane offset serves every read and the
    // sub-step and second-read steps are constants
    const int kb = 8 * (g >> 1) + (i >> 2);
    const char* p = lds_side + kb * (2 * R) + (((m >> 3) ^ swz(kb)) << 4) + (m & 7) * 2 + 16 * s * (2 * R);
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SMOE_LDS v4i16*)p);
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SMOE_LDS v4i16*)(p + 4 * (2 * R)));
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
  }
};

template <int MODE, int R, int BK, int NW, bool AI = false>
struct SideT;
template <int R, int BK, int NW, bool AI>
struct SideT<ROWS, R, BK, NW, AI> {
  using type = RowsSide<R, BK, NW, AI>;
};
template <int R, int BK, int NW, bool AI>
struct SideT<KOUTER, R, BK, NW, AI> {
  using type = KOuterSide<R, BK, NW>;
};

template <class Cfg>
struct Acc {
  static constexpr int RM = Cfg::RM, RN = Cfg::RN;
  f32x16 acc[RM][RN];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < RM; ++i)
#pragma unroll
      for (int j = 0; j < RN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  }
  // tile-local coordinates of accumulator element (i, j, 4g..4g+3) of this lane
  __device__ __forceinline__ static int m_of(int i) {
    const int wave = threadIdx.x >> 6;
    return Cfg::wave_m(wave) * (Cfg::BM / Cfg::WM) + i * 32 + (threadIdx.x & 31);
  }
  __device__ __forceinline__ static int n_of(int j, int g) {
    const int wave = threadIdx.x >> 6;
    return Cfg::wave_n(wave) * (Cfg::BN / Cfg::WN) + j * 32 + 8 * g + 4 * ((threadIdx.x >> 5) & 1);
  }
  __device__ __forceinline__ static int wave_n() { return Cfg::wave_n(threadIdx.x >> 6); }
};

// Varlen-M tiles come in two classes: the full m-tiles of every expert
// (floor(count_e / BM) each, expert-major) and the partial last m-tile of
// each expert with count_e % BM != 0.  The schedule runs the partial tiles
// last: with their idle row blocks skipped they are the cheapest tiles, so
// the final, ragged round of a launch is short.  The m-tile list itself is
// built once per forward / backward call (mtiles_kernel).
constexpr int kPartialTile = 1 << 30;  // flag on a tile id: index among the partial tiles

// Persistent schedule.  The grid holds one workgroup per CU, a multiple of 8,
// and workgroup b runs on XCD b % 8 (round-robin dispatch).  Tiles come in a
// main class [0, nmain) and a tail class [nmain, ntiles) (the partial
// varlen-M tiles; empty for other GEMMs).  Each class is cut into 8
// contiguous ranges, one per XCD; XCD x runs its main range, then its tail
// range, and its G/8 workgroups take that sequence round-robin.  Tiles that
// run at the same time on one XCD are then neighbours in the logical order
// (same expert, shared operand rows in that XCD's L2), every XCD gets the
// same amount of work, and the tail tiles form the last rounds.  id() returns
// main tiles as their index and tail tiles as kPartialTile | index in class.
struct Sched {
  int nmain, ntail, cm, ct, fx, hx, gx, x, slot, base;
  __device__ __forceinline__ void init(int ntiles, int tail) {
    ntail = tail;
    nmain = ntiles - tail;
    cm = (nmain + 7) >> 3;
    ct = (ntail + 7) >> 3;
    gx = gridDim.x >> 3;
    x = blockIdx.x & 7;
    slot = blockIdx.x >> 3;
    fx = max(0, min(cm, nmain - x * cm));
    hx = max(0, min(ct, ntail - x * ct));
    base = x * cm;
  }
  // the op gives each XCD its own range [begin, begin + count) (no tail class)
  __device__ __forceinline__ void init_range(int begin, int count) {
    ntail = ct = hx = 0;
    gx = gridDim.x >> 3;
    x = blockIdx.x & 7;
    slot = blockIdx.x >> 3;
    nmain = fx = cm = count;
    base = begin;
  }
  // logical id of this workgroup's k-th tile, or -1 when it has no more
  __device__ __forceinline__ int id(int k) const {
    const int l = slot + k * gx;
    if (l < fx) return base + l;
    if (l < fx + hx) return kPartialTile | (x * ct + (l - fx));
    return -1;
  }
};

// Ops that place their tiles on the XCDs themselves define
//   void xcd_range(const Params&, int xcd, int* begin, int* count)
template <class Op, class = void>
struct HasXcdRange : std::false_type {};
template <class Op>
struct HasXcdRange<Op, std::void_t<decltype(&Op::xcd_range)>> : std::true_type {};

// Ops with a tail class define  int count_tail(const Params&, const int* sh)
// (called after count() with the same sh).
// Ops whose M side gathers rows define  static constexpr int IDX_LDS  (bytes
// for the next tile's row indices, loaded by DMA).
template <class Op, class = void>
struct IdxLds : std::integral_constant<int, 0> {};
template <class Op>
struct IdxLds<Op, std::void_t<decltype(Op::IDX_LDS)>> : std::integral_constant<int, Op::IDX_LDS> {};

// Ops define  static constexpr int EPI_STORES : a lower bound on the vector
// memory instructions each wave issues in the epilogue of a full tile (all
// BM rows valid).  A wave's vector memory operations retire in issue order,
// loads and stores alike, so a wait for stage 0 of a tile only has to leave
// outstanding the operations issued after it: the other prologue stages and
// the previous tile's epilogue stores.
template <class Op, class = void>
struct EpiStores : std::integral_constant<int, 0> {};
template <class Op>
struct EpiStores<Op, std::void_t<decltype(Op::EPI_STORES)>> : std::integral_constant<int, Op::EPI_STORES> {};

template <class Op, class = void>
struct HasCountTail : std::false_type {};
template <class Op>
struct HasCountTail<Op, std::void_t<decltype(&Op::count_tail)>> : std::true_type {};

// The main loop shared by every GEMM.  Op supplies:
//   using Cfg = GemmCfg<...>;  static constexpr int M_MODE, N_MODE, EPI_LDS;
//   int  count(const Params&, int* sh)                     -- number of tiles
//   bool tile(const Params&, int id, TileInfo&, int* sh)   -- tile id -> TileInfo
//   void init_m(const Params&, const TileInfo&, Side&)      -- operand sides
//   void init_n(const Params&, const TileInfo&, Side&)
//   void epilogue(const Params&, const TileInfo&, Acc<Cfg>&, char* epi_lds)
// Each workgroup is persistent over its tiles.  For tile k it looks up tile
// k+1 and sets up its operand sides while tile k's first stages are in
// flight; after tile k's k loop it issues tile k+1's prologue DMA and only
// then runs tile k's epilogue, so the epilogue's stores and arithmetic
// overlap the next tile's first loads.  The epilogue gets its own LDS
// (EPI_LDS bytes) since the stage buffers are being refilled meanwhile.
template <class Op>
__global__ __launch_bounds__(Op::Cfg::THREADS, Op::Cfg::OCC) void grouped_gemm_kernel(const typename Op::Params p) {
  using Cfg = typename Op::Cfg;
  // an M side with IDX_LDS always gathers its rows: indices by LDS DMA
  using MSide = typename SideT<Op::M_MODE, Cfg::BM, Cfg::BK, Cfg::NW, (IdxLds<Op>::value > 0)>::type;
  using NSide = typename SideT<Op::N_MODE, Cfg::BN, Cfg::BK, Cfg::NW>::type;
  constexpr int BM = Cfg::BM, BN = Cfg::BN, S = Cfg::STAGES, BK = Cfg::BK, SUB = Cfg::SUB;
  constexpr int kEpiBytes = (Op::EPI_LDS > 0 ? (Op::EPI_LDS + 255) / 256 * 256 : 256);
  constexpr int kIdxLds = IdxLds<Op>::value;
  // The split ring fills all 160 KB with stage buffers: no epilogue area (the
  // epilogue stages its stores in the idle A2 and B1 buffers), no index area
  // and no shared tile-lookup words (its ops' count() and tile() read the
  // m-tile list directly and get a null pointer).
  constexpr bool kSplit = Cfg::SPLIT;
  // (its ops gather nothing: row-major M side, N side without k-row indices)
  static_assert(!kSplit || (Op::M_MODE == ROWS && kIdxLds == 0 && Op::EPI_LDS == 0), "split-ring ops");
  constexpr int kSmem = kSplit ? Cfg::LDS_BYTES : Cfg::LDS_BYTES + kEpiBytes + kIdxLds;
  static_assert(kSmem <= 160 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) char smem[kSmem];
  int* sh = nullptr;  // [0..3], [4..7]: tile lookups of even / odd k; [8..9]: tile counts
  if constexpr (!kSplit) {
    __shared__ int sh_words[16];
    sh = sh_words;
  }
  Sched sched;
  if constexpr (HasXcdRange<Op>::value) {
    int b, c;
    Op::xcd_range(p, blockIdx.x & 7, &b, &c);
    sched.init_range(b, c);
  } else {
    const int ntiles = Op::count(p, kSplit ? nullptr : sh + 8);
    int tail = 0;
    if constexpr (HasCountTail<Op>::value) tail = Op::count_tail(p, kSplit ? nullptr : sh + 8);
    sched.init(ntiles, tail);
  }
  const int id = sched.id(0);
  TileInfo ti;
  // tile() may synchronise the workgroup: ids are workgroup-uniform
  if (id < 0 || !Op::tile(p, id, ti, sh)) return;
  const uint32_t lds0 = (uint32_t)(uintptr_t)smem;
  MSide ms, ms_next;
  NSide ns, ns_next;
  if constexpr (kIdxLds > 0) ms.idx_lds = ms_next.idx_lds = lds0 + Cfg::LDS_BYTES + kEpiBytes;
  Op::init_m(p, ti, ms);
  Op::init_n(p, ti, ns);
  if constexpr (kIdxLds > 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the first tile's index DMA
  ms.commit();
  ns.commit();
  const int wave = threadIdx.x >> 6;
  const int wm0 = Cfg::wave_m(wave) * (BM / Cfg::WM);
  const int wn0 = Cfg::wave_n(wave) * (BN / Cfg::WN);
  constexpr int kPerStage = Cfg::QM + Cfg::QN;  // DMA ops per wave per stage
  // The next stage's DMA is interleaved with the MFMAs: instruction d goes
  // just before MFMA number kDmaStride * d of the step.  A wave cannot issue
  // past a DMA instruction until the CU's texture path accepts it, so a burst
  // of a whole stage at the top of the step keeps every wave from issuing
  // MFMAs meanwhile; one instruction every few MFMAs lets the other wave of
  // the SIMD keep the matrix pipe busy while one waits.  Every 2nd MFMA puts
  // the whole stage in the first half of the step, so it still has half a
  // step to land from the Infinity Cache or HBM.
  constexpr int kMfmaPerStep = Cfg::SUB * Cfg::RM * Cfg::RN;
  constexpr int kDmaStride = kMfmaPerStep >= 2 * kPerStage ? 2 : 1;
  // The weight-gradient GEMMs (k outer on both sides, gathered k rows) set up
  // the next tile's sides after the k loop: that is plain arithmetic, and its
  // registers would otherwise be held across the loop (with the interleaved
  // DMA the 256x256 loop then spilled).
  constexpr bool kLateSides = Op::M_MODE == KOUTER && Op::N_MODE == KOUTER;
  // The two-stage schedule with its barrier before the last sub-step (below)
  // needs a stage's instructions to fit every second MFMA of one sub-step.
  // It holds fragment addresses for both stage buffers across the step, and
  // only the weight-gradient GEMMs stay spill-free with it (dW1 -4%, dW2 -2%;
  // up, down and dH spilled 3-7 VGPRs and lost 2-7%, dX~ was unchanged).
  constexpr bool kMidBarrier =
      kLateSides && S == 2 && SUB >= 2 && Cfg::RM * Cfg::RN >= kPerStage && kPerStage % 2 == 0;
  static_assert(kDmaStride * (kPerStage - 1) < kMfmaPerStep, "every DMA instruction has an MFMA after it");

  // stages 0 .. S-2 of a tile, and the row indices of stage S-1 (gathered k)
  auto prologue = [&](const TileInfo& t, MSide& a, NSide& b) {
    const int nk = (t.k_len + BK - 1) / BK;
    if constexpr (kSplit) {
      // A0, B0, A1 (in this order: the waits count on it)
      if (nk > 0) {
        a.issue(lds0 + Cfg::a_off(0), 0);
        b.issue(lds0 + Cfg::b_off(0), 0);
      }
      if (nk > 1) a.issue(lds0 + Cfg::a_off(1), BK);
      return;
    }
#pragma unroll
    for (int st = 0; st < S - 1; ++st) {
      if (st < nk) {
        if constexpr (Op::M_MODE == KOUTER) a.prefetch_idx(st * BK);
        if constexpr (Op::N_MODE == KOUTER) b.prefetch_idx(st * BK);
        if constexpr (Op::M_MODE == KOUTER || Op::N_MODE == KOUTER) {
          // gathered k rows: this stage's row indices must have arrived
          bool g = false;
          if constexpr (Op::M_MODE == KOUTER) g = g || a.gidx != nullptr;
          if constexpr (Op::N_MODE == KOUTER) g = g || b.gidx != nullptr;
          if (g) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
          if constexpr (Op::M_MODE == KOUTER) a.idx_commit();
          if constexpr (Op::N_MODE == KOUTER) b.idx_commit();
        }
        a.issue(lds0 + st * Cfg::STAGE_BYTES, st * BK);
        b.issue(lds0 + st * Cfg::STAGE_BYTES + Cfg::M_BYTES, st * BK);
      }
    }
    if constexpr (Op::M_MODE == KOUTER) a.prefetch_idx((S - 1) * BK);
    if constexpr (Op::N_MODE == KOUTER) b.prefetch_idx((S - 1) * BK);
  };

  Acc<Cfg> acc;
  acc.zero();
  prologue(ti, ms, ns);
  bool prev_full = false;  // the epilogue just issued was a full tile's
  for (int k = 0;; ++k) {
    // next tile: lookup and side setup overlap this tile's first DMA
    int idn = sched.id(k + 1);
    TileInfo tn;
    if (idn >= 0 && !Op::tile(p, idn, tn, kSplit ? nullptr : sh + 4 * ((k + 1) & 1))) idn = -1;
    // Sides that gather rows by index DMA set up here, so those loads overlap
    // this tile's k loop; the weight-gradient sides (plain arithmetic) set up
    // after it, so their registers are free during the k loop.
    if (idn >= 0 && !kLateSides) {
      Op::init_m(p, tn, ms_next);
      Op::init_n(p, tn, ns_next);
    }
    const int nk = (ti.k_len + BK - 1) / BK;
    // a wave whose rows all lie past the tile's valid rows skips its MFMAs
    // (it still issues its share of the DMA and joins every barrier); the
    // weight-gradient GEMMs (k outer on both sides) always have full tiles
    const bool active = wm0 < ti.mrows;
    // gathered k rows: their index loads are younger than the DMA, so only a
    // full drain covers them
    bool gathered = false;
    if constexpr (Op::M_MODE == KOUTER) gathered = gathered || ms.gidx != nullptr;
    if constexpr (Op::N_MODE == KOUTER) gathered = gathered || ns.gidx != nullptr;
    if constexpr (kSplit) {
      // Split ring: step kt reads A(kt) from M buffer kt % 3 and B(kt) from N
      // buffer kt % 2, and requests B(kt+1) and then A(kt+2) (interleaved with
      // its MFMAs, B first).  At the top of step kt the only requests younger
      // than B(kt) are A(kt+1)'s QM (from the prologue or step kt-1) and, at
      // kt = 0, the previous epilogue's stores.  Leaving QM outstanding is
      // therefore always enough (whatever the youngest QM are, B(kt) is
      // older), and after a full tile QM plus its exact store count is.  The
      // barrier after the wait also certifies that step kt-1's buffers, which
      // this step refills, are no longer read.
      constexpr int QM = Cfg::QM, QN = Cfg::QN;
      constexpr int kEpi = EpiStores<Op>::value;
      static_assert(QM + kEpi <= 63, "vmcnt range");
      for (int kt = 0; kt < nk; ++kt) {
        const bool a_ahead = kt + 1 < nk;  // A(kt+1) was requested after B(kt)
        if (kt == 0 && prev_full) {
          if (a_ahead)
            wait_vm_barrier<QM + kEpi>();
          else
            wait_vm_barrier<kEpi>();
        } else if (a_ahead) {
          wait_vm_barrier<QM>();
        } else {
          wait_vm_barrier<0>();  // (at kt = 0 after a partial tile: its store count is not known)
        }
        const int kb = kt + 1, ka = kt + 2;
        const bool issue_b = kb < nk, issue_a = ka < nk;
        const uint32_t bdst = lds0 + Cfg::b_off(kb & 1), adst = lds0 + Cfg::a_off(ka % 3);
        const char* lm = smem + Cfg::a_off(kt % 3);
        const char* ln = smem + Cfg::b_off(kt & 1);
        auto issue_one = [&](int d) {
          if (d < QN) {
            if (issue_b) ns.issue(bdst, kb * BK, d, QN);
          } else if (issue_a) {
            ms.issue(adst, ka * BK, d - QN, QM);
          }
        };
        if (active) {
          bf16x8 fm[Cfg::RM], fn[Cfg::RN];
#pragma unroll
          for (int i = 0; i < Cfg::RM; ++i) fm[i] = MSide::frag(lm, wm0 + 32 * i, 0);
#pragma unroll
          for (int j = 0; j < Cfg::RN; ++j) fn[j] = NSide::frag(ln, wn0 + 32 * j, 0);
#pragma unroll
          for (int s = 0; s < SUB; ++s)
#pragma unroll
            for (int i = 0; i < Cfg::RM; ++i)
#pragma unroll
              for (int j = 0; j < Cfg::RN; ++j) {
                const int c = (s * Cfg::RM + i) * Cfg::RN + j;
                if (c % kDmaStride == 0 && c / kDmaStride < kPerStage) {
                  __builtin_amdgcn_sched_barrier(0);
                  issue_one(c / kDmaStride);
                  __builtin_amdgcn_sched_barrier(0);
                }
                acc.acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fn[j], fm[i], acc.acc[i][j], 0, 0, 0);
                if (s + 1 < SUB) {
                  if (j == Cfg::RN - 1) fm[i] = MSide::frag(lm, wm0 + 32 * i, s + 1);
                  if (i == Cfg::RM - 1) fn[j] = NSide::frag(ln, wn0 + 32 * j, s + 1);
                }
              }
        } else {
          if (issue_b) ns.issue(bdst, kb * BK);
          if (issue_a) ms.issue(adst, ka * BK);
        }
      }
    } else if constexpr (kMidBarrier) {
      // Two stages, one barrier per step, placed before the last sub-step.
      // By then every wave holds that sub-step's fragments in registers and
      // has waited for its share of stage kt+1, so the barrier certifies both
      // that stage kt's buffer is no longer read and that stage kt+1 is
      // complete: stage kt+2's DMA (into stage kt's buffer) starts during the
      // last sub-step, and the first fragments of step kt+1 are read while
      // its MFMAs issue instead of after a barrier at the top of the step.
      // A stage goes out in two halves, every second MFMA: the first in the
      // last sub-step of the step before, the second in sub-step 0 (all of it
      // in sub-step 0 of a tile's first step).
      constexpr int kHalf = kPerStage / 2;
      // stage 0 (the prologue's) is complete, and every wave is past the
      // previous epilogue, whose stores may stay outstanding
      if (!gathered && prev_full)
        wait_vm_barrier<(EpiStores<Op>::value < 63 ? EpiStores<Op>::value : 63)>();
      else
        wait_vm_barrier<0>();
      if constexpr (Op::M_MODE == KOUTER) ms.idx_commit();
      if constexpr (Op::N_MODE == KOUTER) ns.idx_commit();
      // DMA instruction d of stage st (buffer st & 1)
      auto issue_one = [&](int st, int d) {
        const uint32_t dst = lds0 + (st & 1) * Cfg::STAGE_BYTES;
        if (d < Cfg::QM)
          ms.issue(dst, st * BK, d, Cfg::QM);
        else
          ns.issue(dst + Cfg::M_BYTES, st * BK, d - Cfg::QM, Cfg::QN);
      };
      auto dma_at = [&](int st, int d) {
        __builtin_amdgcn_sched_barrier(0);
        issue_one(st, d);
        __builtin_amdgcn_sched_barrier(0);
      };
      bf16x8 fm[Cfg::RM], fn[Cfg::RN];
      auto k_loop = [&](auto active_c) {
        constexpr bool ACT = decltype(active_c)::value;
        if constexpr (ACT) {
#pragma unroll
          for (int i = 0; i < Cfg::RM; ++i) fm[i] = MSide::frag(smem, wm0 + 32 * i, 0);
#pragma unroll
          for (int j = 0; j < Cfg::RN; ++j) fn[j] = NSide::frag(smem + Cfg::M_BYTES, wn0 + 32 * j, 0);
        }
        for (int kt = 0; kt < nk; ++kt) {
          const char* cur = smem + (kt & 1) * Cfg::STAGE_BYTES;
          const char* nxt = smem + ((kt + 1) & 1) * Cfg::STAGE_BYTES;
          const bool has1 = kt + 1 < nk, has2 = kt + 2 < nk;
#pragma unroll
          for (int s = 0; s < SUB; ++s)
#pragma unroll
            for (int i = 0; i < Cfg::RM; ++i)
#pragma unroll
              for (int j = 0; j < Cfg::RN; ++j) {
                const int cs = i * Cfg::RN + j;  // MFMA number within the sub-step
                if (s == 0 && has1) {
                  if (kt == 0) {
                    if (cs < kPerStage) dma_at(kt + 1, cs);
                  } else if (cs % 2 == 0 && kHalf + cs / 2 < kPerStage) {
                    dma_at(kt + 1, kHalf + cs / 2);
                  }
                }
                if (s == 1 && cs == 0 && has2) {
                  // gathered k rows of stage kt+2: stage kt+1 no longer needs the index registers
                  if constexpr (Op::M_MODE == KOUTER) ms.prefetch_idx((kt + 2) * BK);
                  if constexpr (Op::N_MODE == KOUTER) ns.prefetch_idx((kt + 2) * BK);
                }
                if (s == SUB - 1 && cs == 0) {
                  wait_vm_barrier<0>();
                  if constexpr (Op::M_MODE == KOUTER) ms.idx_commit();
                  if constexpr (Op::N_MODE == KOUTER) ns.idx_commit();
                }
                if (s == SUB - 1 && has2 && cs % 2 == 0 && cs / 2 < kHalf) dma_at(kt + 2, cs / 2);
                if constexpr (ACT) {
                  acc.acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fn[j], fm[i], acc.acc[i][j], 0, 0, 0);
                  // each fragment is re-read right after its last use: the next
                  // sub-step's from this stage, or sub-step 0 of the next step
                  if (s + 1 < SUB || has1) {
                    const char* b = s + 1 < SUB ? cur : nxt;
                    const int sn = s + 1 < SUB ? s + 1 : 0;
                    if (j == Cfg::RN - 1) fm[i] = MSide::frag(b, wm0 + 32 * i, sn);
                    if (i == Cfg::RM - 1) fn[j] = NSide::frag(b + Cfg::M_BYTES, wn0 + 32 * j, sn);
                  }
                }
              }
        }
      };
      if (active)
        k_loop(std::true_type{});
      else
        k_loop(std::false_type{});
    } else {
      for (int kt = 0; kt < nk; ++kt) {
        // stage kt is complete when at most (stages issued after it) * kPerStage
        // ops remain.  At kt = 0 the previous epilogue's stores are younger than
        // stage 0, and gathered index loads are younger than the DMA: full drain.
        const int ahead = (kt == 0 || gathered) ? 0 : min(S - 2, nk - 1 - kt);
        // stage 0: the younger prologue stages and epilogue stores may stay outstanding
        constexpr int kYoung = (S - 2) * kPerStage;
        constexpr int kYoungEpi = kYoung + EpiStores<Op>::value < 63 ? kYoung + EpiStores<Op>::value : 63;
        if (kt == 0 && !gathered && nk >= S - 1 && (kYoung > 0 || prev_full)) {
          if (prev_full)
            wait_vm_barrier<kYoungEpi>();
          else
            wait_vm_barrier<kYoung>();
        } else if (ahead >= 2)
          wait_vm_barrier<(S >= 4 ? 2 : 0) * kPerStage>();
        else if (ahead == 1)
          wait_vm_barrier<(S >= 3 ? 1 : 0) * kPerStage>();
        else
          wait_vm_barrier<0>();
        // with gathered k rows the wait above was a full drain, index loads included
        if constexpr (Op::M_MODE == KOUTER) ms.idx_commit();
        if constexpr (Op::N_MODE == KOUTER) ns.idx_commit();
        const int knext = kt + S - 1;
        const bool issue_next = knext < nk;
        const uint32_t st_next = lds0 + (knext % S) * Cfg::STAGE_BYTES;
        const char* cur = smem + (kt % S) * Cfg::STAGE_BYTES;
        const char* lm = cur;
        const char* ln = cur + Cfg::M_BYTES;
        // DMA instruction d of this wave's share of the next stage
        auto issue_one = [&](int d) {
          if (d < Cfg::QM)
            ms.issue(st_next, knext * BK, d, Cfg::QM);
          else
            ns.issue(st_next + Cfg::M_BYTES, knext * BK, d - Cfg::QM, Cfg::QN);
        };
        if (active) {
          // One set of fragments: each is re-read for sub-step s+1 right after
          // the last MFMA of sub-step s that uses it (A fragment i after MFMA
          // (i, RN-1), B fragment j after MFMA (RM-1, j)), so its read has the
          // rest of the sub-step to land and no second set of registers is
          // needed.
          bf16x8 fm[Cfg::RM], fn[Cfg::RN];
  #pragma unroll
          for (int i = 0; i < Cfg::RM; ++i) fm[i] = MSide::frag(lm, wm0 + 32 * i, 0);
  #pragma unroll
          for (int j = 0; j < Cfg::RN; ++j) fn[j] = NSide::frag(ln, wn0 + 32 * j, 0);
  #pragma unroll
          for (int s = 0; s < SUB; ++s)
  #pragma unroll
            for (int i = 0; i < Cfg::RM; ++i)
  #pragma unroll
              for (int j = 0; j < Cfg::RN; ++j) {
                const int c = (s * Cfg::RM + i) * Cfg::RN + j;  // MFMA number within the step
                if (c % kDmaStride == 0 && c / kDmaStride < kPerStage) {
                  // the scheduling barriers keep the instruction between these MFMAs
                  __builtin_amdgcn_sched_barrier(0);
                  if (issue_next) issue_one(c / kDmaStride);
                  __builtin_amdgcn_sched_barrier(0);
                }
                acc.acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fn[j], fm[i], acc.acc[i][j], 0, 0, 0);
                if (s + 1 < SUB) {
                  if (j == Cfg::RN - 1) fm[i] = MSide::frag(lm, wm0 + 32 * i, s + 1);
                  if (i == Cfg::RM - 1) fn[j] = NSide::frag(ln, wn0 + 32 * j, s + 1);
                }
              }
        } else if (issue_next) {
          // a wave without valid rows only requests its share of the stage
          ms.issue(st_next, knext * BK);
          ns.issue(st_next + Cfg::M_BYTES, knext * BK);
        }
        if (issue_next) {
          if constexpr (Op::M_MODE == KOUTER) ms.prefetch_idx((knext + 1) * BK);
          if constexpr (Op::N_MODE == KOUTER) ns.prefetch_idx((knext + 1) * BK);
        }
      }
    }
    barrier_lds();  // every wave is done with the stage buffers
    if (idn >= 0) {
      if constexpr (kLateSides) {
        Op::init_m(p, tn, ms_next);
        Op::init_n(p, tn, ns_next);
      }
      // the last step's full drain covered the next tile's index loads
      ms_next.commit();
      ns_next.commit();
      ms = ms_next;
      ns = ns_next;
      prologue(tn, ms, ns);
    }
    Op::epilogue(p, ti, acc, smem + Cfg::LDS_BYTES);
    prev_full = ti.mrows == BM;
    if (idn < 0) break;
    ti = tn;
    acc.zero();
  }
}

}  // namespace smoe
