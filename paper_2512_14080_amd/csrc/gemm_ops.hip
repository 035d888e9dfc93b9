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
#include "gemm_core.h"
#include "launch.h"

namespace smoe {

__device__ __forceinline__ float silu_sig(float g, float* sig) {
  const float s = 1.f / (1.f + __expf(-g));
  *sig = s;
  return g * s;
}

__device__ __forceinline__ void store_bf16x4(uint16_t* dst, float a, float b, float c, float d) {
  u32x2 v;
  v[0] = pack_bf2(a, b);
  v[1] = pack_bf2(c, d);
  *(u32x2*)dst = v;
}

__device__ __forceinline__ void load_bf16x4(const uint16_t* src, float* out) {
  const u32x2 v = *(const u32x2*)src;
  out[0] = bf_lo(v[0]);
  out[1] = bf_hi(v[0]);
  out[2] = bf_lo(v[1]);
  out[3] = bf_hi(v[1]);
}

// ---------------------------------------------------------------- scheduling
template <int BM, int BN>
__device__ __forceinline__ bool tile_varlen_m(const int32_t* offsets, int E, int N, int K, int* sh, TileInfo& ti) {
  const int nnt = N / BN;
  const int id = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = id / nnt, nt = id % nnt;
  if (!find_m_tile<BM>(offsets, E, mt, sh, ti)) return false;
  ti.n0 = nt * BN;
  ti.k_begin = 0;
  ti.k_len = K;
  return true;
}

template <int BM, int BN>
__device__ __forceinline__ bool tile_plain_m(int M, int N, int K, TileInfo& ti) {
  const int nnt = (N + BN - 1) / BN;
  const int id = blockIdx.x;
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
__device__ __forceinline__ bool tile_varlen_k(const int32_t* offsets, int M, int N, TileInfo& ti) {
  const int mtn = M / BM, ntn = N / BN;
  const int id = xcd_remap(blockIdx.x, gridDim.x);
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

// ROWS loader over rows [row_base, row_base + mrows) of a [*, ld] bf16 matrix,
// optionally gathered through idx.  Rows past mrows are clamped to the last
// valid row; their results are never stored.
template <int R>
__device__ __forceinline__ RowsLoader<R> rows_loader(const uint16_t* base, int64_t ld, const int32_t* idx, int row_base,
                                                     int mrows) {
  RowsLoader<R> L;
#pragma unroll
  for (int p = 0; p < R / 32; ++p) {
    const int m = min((threadIdx.x >> 3) + 32 * p, mrows - 1);
    const int64_t row = idx ? (int64_t)idx[row_base + m] : (int64_t)(row_base + m);
    L.ptr[p] = (const char*)(base + row * ld);
  }
  return L;
}

// KOUTER loader: columns [c0 + 8rb, +8) of a [*, ld] matrix, k rows
// k_begin.. (optionally gathered), valid columns < cvalid.
template <int R>
__device__ __forceinline__ KOuterLoader<R> kouter_loader(const uint16_t* base, int64_t ld, int c0, int cvalid,
                                                         const int32_t* gidx, int k_begin, int k_len) {
  KOuterLoader<R> L;
  const int r0 = (threadIdx.x >> 3) * 8;
  L.active = (r0 < R) && (c0 + r0 < cvalid);
  L.colptr = (const char*)(base + c0 + r0);
  L.ld_bytes = ld * 2;
  L.gidx = gidx;
  L.k_begin = k_begin;
  L.k_len = k_len;
  return L;
}

// ================================================================== router
template <int BN_>
struct OpRouter {
  static constexpr int BM = 128, BN = BN_, kMinBlocks = BN_ >= 256 ? 1 : 2;
  struct Params { RouterGemmArgs a; };
  static __device__ bool tile(const Params& p, TileInfo& ti, int*) { return tile_plain_m<BM, BN>(p.a.T, p.a.E, p.a.d, ti); }
  static __device__ RowsLoader<BM> make_m(const Params& p, const TileInfo& ti) {
    return rows_loader<BM>(p.a.X, p.a.d, nullptr, ti.row_base, ti.mrows);
  }
  static __device__ KOuterLoader<BN> make_n(const Params& p, const TileInfo& ti) {
    return kouter_loader<BN>(p.a.Wr, p.a.E, ti.n0, p.a.E, nullptr, 0, p.a.d);
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, MfmaTile<BM, BN>& t, char*) {
#pragma unroll
    for (int i = 0; i < t.RM; ++i) {
      const int m = t.m_of(i);
      if (m >= ti.mrows) continue;
      float* out = p.a.logits + (size_t)(ti.row_base + m) * p.a.E;
#pragma unroll
      for (int j = 0; j < t.RN; ++j)
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
// N tile: BN/2 gate columns [j0, j0 + BN/2) and the matching up columns.
// Wave half wn owns gate columns j0 + wn*BN/4 + [0, BN/4) in its first RN/2
// accumulator blocks and the matching up columns in the last RN/2 blocks.
template <int BM_, int BN_>
struct OpUp {
  static constexpr int BM = BM_, BN = BN_, kMinBlocks = 1;
  struct Params { UpArgs a; };
  static __device__ bool tile(const Params& p, TileInfo& ti, int* sh) {
    return tile_varlen_m<BM, BN>(p.a.offsets, p.a.E, 2 * p.a.n, p.a.d, sh, ti);
  }
  static __device__ RowsLoader<BM> make_m(const Params& p, const TileInfo& ti) {
    return rows_loader<BM>(p.a.X, p.a.d, p.a.row_token, ti.row_base, ti.mrows);
  }
  static __device__ __forceinline__ int w1_col(const Params& p, const TileInfo& ti, int r) {
    const int j0 = (ti.n0 / BN) * (BN / 2);
    const int wn = r / (BN / 2), q = r % (BN / 2);
    return q < BN / 4 ? j0 + wn * (BN / 4) + q : p.a.n + j0 + wn * (BN / 4) + (q - BN / 4);
  }
  static __device__ KOuterLoader<BN> make_n(const Params& p, const TileInfo& ti) {
    const int r0 = (threadIdx.x >> 3) * 8;
    const uint16_t* w = p.a.W1 + (size_t)ti.e * p.a.d * (2 * p.a.n);
    KOuterLoader<BN> L = kouter_loader<BN>(w, 2 * p.a.n, 0, 1 << 30, nullptr, 0, p.a.d);
    L.colptr = (const char*)(w + (r0 < BN ? w1_col(p, ti, r0) : 0));
    return L;
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, MfmaTile<BM, BN>& t, char*) {
    constexpr int RN = MfmaTile<BM, BN>::RN;
    const int n = p.a.n;
    const int j0 = (ti.n0 / BN) * (BN / 2);
    const int wn = (threadIdx.x >> 6) >> 1;
#pragma unroll
    for (int i = 0; i < t.RM; ++i) {
      const int m = t.m_of(i);
      if (m >= ti.mrows) continue;
      const size_t row = (size_t)(ti.row_base + m);
      uint16_t* h = p.a.H + row * (2 * n);
      uint16_t* a = p.a.A + row * n;
#pragma unroll
      for (int j = 0; j < RN / 2; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int q = t.n_of(j, g) - wn * (BN / 2);
          const int col = j0 + wn * (BN / 4) + q;
          float gv[4], uv[4], av[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            gv[r] = t.acc[i][j][4 * g + r];
            uv[r] = t.acc[i][j + RN / 2][4 * g + r];
            float sg;
            av[r] = silu_sig(gv[r], &sg) * uv[r];
          }
          store_bf16x4(h + col, gv[0], gv[1], gv[2], gv[3]);
          store_bf16x4(h + n + col, uv[0], uv[1], uv[2], uv[3]);
          store_bf16x4(a + col, av[0], av[1], av[2], av[3]);
        }
    }
  }
};

// ================================================================== down-proj
template <int BM_, int BN_>
struct OpDown {
  static constexpr int BM = BM_, BN = BN_, kMinBlocks = 1;
  struct Params { DownArgs a; };
  static __device__ bool tile(const Params& p, TileInfo& ti, int* sh) {
    return tile_varlen_m<BM, BN>(p.a.offsets, p.a.E, p.a.d, p.a.n, sh, ti);
  }
  static __device__ RowsLoader<BM> make_m(const Params& p, const TileInfo& ti) {
    return rows_loader<BM>(p.a.A, p.a.n, nullptr, ti.row_base, ti.mrows);
  }
  static __device__ KOuterLoader<BN> make_n(const Params& p, const TileInfo& ti) {
    const uint16_t* w = p.a.W2 + (size_t)ti.e * p.a.n * p.a.d;
    return kouter_loader<BN>(w, p.a.d, ti.n0, p.a.d, nullptr, 0, p.a.n);
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, MfmaTile<BM, BN>& t, char*) {
#pragma unroll
    for (int i = 0; i < t.RM; ++i) {
      const int m = t.m_of(i);
      if (m >= ti.mrows) continue;
      uint16_t* y = p.a.Y + (size_t)(ti.row_base + m) * p.a.d + ti.n0;
#pragma unroll
      for (int j = 0; j < t.RN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int c = t.n_of(j, g);
          store_bf16x4(y + c, t.acc[i][j][4 * g], t.acc[i][j][4 * g + 1], t.acc[i][j][4 * g + 2], t.acc[i][j][4 * g + 3]);
        }
    }
  }
};

// ================================================================== dH
// Epilogue (down-proj backward): with A recomputed from the cached H,
// dS = <dA', A> (reduced over this tile's n columns), dA = s dA',
// dH = dSwiGLU(dA, H), A' = s A.
template <int BM_, int BN_>
struct OpDH {
  static constexpr int BM = BM_, BN = BN_, kMinBlocks = 1;
  struct Params { DHArgs a; };
  static __device__ bool tile(const Params& p, TileInfo& ti, int* sh) {
    return tile_varlen_m<BM, BN>(p.a.offsets, p.a.E, p.a.n, p.a.d, sh, ti);
  }
  static __device__ RowsLoader<BM> make_m(const Params& p, const TileInfo& ti) {
    return rows_loader<BM>(p.a.dO, p.a.d, p.a.row_token, ti.row_base, ti.mrows);
  }
  static __device__ RowsLoader<BN> make_n(const Params& p, const TileInfo& ti) {
    // rows of W2_e [n][d] are the n columns of dA', with d contiguous
    const uint16_t* w = p.a.W2 + (size_t)ti.e * p.a.n * p.a.d;
    return rows_loader<BN>(w, p.a.d, nullptr, ti.n0, BN);
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, MfmaTile<BM, BN>& t, char* smem) {
    const int n = p.a.n;
    const int lane = threadIdx.x & 63;
    const int wn = (threadIdx.x >> 6) >> 1;
    float* red = (float*)smem;  // [BM][2]
#pragma unroll
    for (int i = 0; i < t.RM; ++i) {
      const int m = t.m_of(i);
      const bool valid = m < ti.mrows;
      const size_t row = (size_t)(ti.row_base + (valid ? m : 0));
      const float s = valid ? p.a.row_w[row] : 0.f;
      const uint16_t* h = p.a.H + row * (2 * n);
      uint16_t* dh = p.a.dH + row * (2 * n);
      uint16_t* ap = p.a.Ap + row * n;
      float part = 0.f;
#pragma unroll
      for (int j = 0; j < t.RN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          if (!valid) continue;
          const int col = ti.n0 + t.n_of(j, g);
          float gv[4], uv[4], dg[4], du[4], apv[4];
          load_bf16x4(h + col, gv);
          load_bf16x4(h + n + col, uv);
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
          store_bf16x4(dh + col, dg[0], dg[1], dg[2], dg[3]);
          store_bf16x4(dh + n + col, du[0], du[1], du[2], du[3]);
          store_bf16x4(ap + col, apv[0], apv[1], apv[2], apv[3]);
        }
      part += __shfl_xor(part, 32, kWave);
      if (lane < 32) red[m * 2 + wn] = part;
    }
    __syncthreads();
    const int nnt = n / BN;
    const int nt = ti.n0 / BN;
    for (int m = threadIdx.x; m < ti.mrows; m += 256) {
      const float v = red[m * 2] + red[m * 2 + 1];
      const size_t row = (size_t)(ti.row_base + m);
      if (nnt == 1)
        p.a.dS[row] = v;
      else
        p.a.dS_part[row * nnt + nt] = v;
    }
  }
};

// ================================================================== dX~
template <int BM_, int BN_>
struct OpDXt {
  static constexpr int BM = BM_, BN = BN_, kMinBlocks = 1;
  struct Params { DXtArgs a; };
  static __device__ bool tile(const Params& p, TileInfo& ti, int* sh) {
    return tile_varlen_m<BM, BN>(p.a.offsets, p.a.E, p.a.d, 2 * p.a.n, sh, ti);
  }
  static __device__ RowsLoader<BM> make_m(const Params& p, const TileInfo& ti) {
    return rows_loader<BM>(p.a.dH, 2 * p.a.n, nullptr, ti.row_base, ti.mrows);
  }
  static __device__ RowsLoader<BN> make_n(const Params& p, const TileInfo& ti) {
    // rows of W1_e [d][2n] are the d columns of dX~, with 2n contiguous
    const uint16_t* w = p.a.W1 + (size_t)ti.e * p.a.d * (2 * p.a.n);
    return rows_loader<BN>(w, 2 * p.a.n, nullptr, ti.n0, BN);
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, MfmaTile<BM, BN>& t, char*) {
#pragma unroll
    for (int i = 0; i < t.RM; ++i) {
      const int m = t.m_of(i);
      if (m >= ti.mrows) continue;
      uint16_t* y = p.a.dXt + (size_t)(ti.row_base + m) * p.a.d + ti.n0;
#pragma unroll
      for (int j = 0; j < t.RN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int c = t.n_of(j, g);
          store_bf16x4(y + c, t.acc[i][j][4 * g], t.acc[i][j][4 * g + 1], t.acc[i][j][4 * g + 2], t.acc[i][j][4 * g + 3]);
        }
    }
  }
};

// ================================================================== weight gradients (varlen-K)
template <int BM, int BN>
__device__ __forceinline__ void store_weight_tile(uint16_t* out, int64_t ld, const TileInfo& ti, MfmaTile<BM, BN>& t) {
#pragma unroll
  for (int i = 0; i < t.RM; ++i) {
    const int m = t.m_of(i);
    uint16_t* y = out + (size_t)(ti.m0 + m) * ld + ti.n0;
#pragma unroll
    for (int j = 0; j < t.RN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c = t.n_of(j, g);
        store_bf16x4(y + c, t.acc[i][j][4 * g], t.acc[i][j][4 * g + 1], t.acc[i][j][4 * g + 2], t.acc[i][j][4 * g + 3]);
      }
  }
}

// dW2_e[n,d] = A'_e^T gather(dO): M = n (A' columns), N = d (dO columns)
template <int BM_, int BN_>
struct OpDW2 {
  static constexpr int BM = BM_, BN = BN_, kMinBlocks = 1;
  struct Params { DW2Args a; };
  static __device__ bool tile(const Params& p, TileInfo& ti, int*) { return tile_varlen_k<BM, BN>(p.a.offsets, p.a.n, p.a.d, ti); }
  static __device__ KOuterLoader<BM> make_m(const Params& p, const TileInfo& ti) {
    return kouter_loader<BM>(p.a.Ap, p.a.n, ti.m0, p.a.n, nullptr, ti.k_begin, ti.k_len);
  }
  static __device__ KOuterLoader<BN> make_n(const Params& p, const TileInfo& ti) {
    return kouter_loader<BN>(p.a.dO, p.a.d, ti.n0, p.a.d, p.a.row_token, ti.k_begin, ti.k_len);
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, MfmaTile<BM, BN>& t, char*) {
    store_weight_tile<BM, BN>(p.a.dW2 + (size_t)ti.e * p.a.n * p.a.d, p.a.d, ti, t);
  }
};

// dW1_e[d,2n] = gather(X)_e^T dH_e: M = d (X columns), N = 2n (dH columns)
template <int BM_, int BN_>
struct OpDW1 {
  static constexpr int BM = BM_, BN = BN_, kMinBlocks = 1;
  struct Params { DW1Args a; };
  static __device__ bool tile(const Params& p, TileInfo& ti, int*) { return tile_varlen_k<BM, BN>(p.a.offsets, p.a.d, 2 * p.a.n, ti); }
  static __device__ KOuterLoader<BM> make_m(const Params& p, const TileInfo& ti) {
    return kouter_loader<BM>(p.a.X, p.a.d, ti.m0, p.a.d, p.a.row_token, ti.k_begin, ti.k_len);
  }
  static __device__ KOuterLoader<BN> make_n(const Params& p, const TileInfo& ti) {
    return kouter_loader<BN>(p.a.dH, 2 * p.a.n, ti.n0, 2 * p.a.n, nullptr, ti.k_begin, ti.k_len);
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, MfmaTile<BM, BN>& t, char*) {
    store_weight_tile<BM, BN>(p.a.dW1 + (size_t)ti.e * p.a.d * (2 * p.a.n), 2 * p.a.n, ti, t);
  }
};

// dW_r[d,E] = X^T dL, split over token chunks into fp32 partials
template <int BN_>
struct OpDWr {
  static constexpr int BM = 128, BN = BN_, kMinBlocks = BN_ >= 256 ? 1 : 2;
  struct Params { DWrArgs a; };
  static __device__ bool tile(const Params& p, TileInfo& ti, int*) {
    const int mtn = p.a.d / BM, ntn = (p.a.E + BN - 1) / BN;
    const int id = blockIdx.x;
    const int split = id / (mtn * ntn), rem = id % (mtn * ntn);
    ti.e = split;
    ti.m0 = (rem / ntn) * BM;
    ti.n0 = (rem % ntn) * BN;
    ti.mrows = BM;
    ti.row_base = 0;
    const int chunk = (((p.a.T + p.a.splits - 1) / p.a.splits) + kBK - 1) / kBK * kBK;
    ti.k_begin = split * chunk;
    ti.k_len = max(0, min(chunk, p.a.T - ti.k_begin));
    return true;
  }
  static __device__ KOuterLoader<BM> make_m(const Params& p, const TileInfo& ti) {
    return kouter_loader<BM>(p.a.X, p.a.d, ti.m0, p.a.d, nullptr, ti.k_begin, ti.k_len);
  }
  static __device__ KOuterLoader<BN> make_n(const Params& p, const TileInfo& ti) {
    return kouter_loader<BN>(p.a.dL, p.a.E, ti.n0, p.a.E, nullptr, ti.k_begin, ti.k_len);
  }
  static __device__ void epilogue(const Params& p, const TileInfo& ti, MfmaTile<BM, BN>& t, char*) {
    float* out = p.a.part + (size_t)ti.e * p.a.d * p.a.E;
#pragma unroll
    for (int i = 0; i < t.RM; ++i) {
      const int m = t.m_of(i);
      float* o = out + (size_t)(ti.m0 + m) * p.a.E;
#pragma unroll
      for (int j = 0; j < t.RN; ++j)
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
template <class Op>
static hipError_t run(const typename Op::Params& p, int grid, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  grouped_gemm_kernel<Op><<<dim3(grid), dim3(256), 0, s>>>(p);
  return hipGetLastError();
}

static int pad8(int g) { return (g + 7) & ~7; }
// upper bound of sum_e ceil(count_e / BM) given sum_e count_e <= capacity
static int mtiles_bound(int capacity, int E, int BM) { return capacity / BM + E; }

hipError_t launch_router_gemm(const RouterGemmArgs& a, hipStream_t s) {
  const int mt = (a.T + 127) / 128;
  if (a.E <= 64) return run<OpRouter<64>>({a}, mt, s);
  if (a.E <= 128) return run<OpRouter<128>>({a}, mt, s);
  return run<OpRouter<256>>({a}, mt * ((a.E + 255) / 256), s);
}

hipError_t launch_up(const UpArgs& a, hipStream_t s) {
  const int N = 2 * a.n;
  if (a.n % 128 == 0) {
    constexpr int BM = 256, BN = 256;
    return run<OpUp<BM, BN>>({a}, pad8(mtiles_bound(a.capacity, a.E, BM) * (N / BN)), s);
  }
  constexpr int BM = 128, BN = 128;  // n = 64
  return run<OpUp<BM, BN>>({a}, pad8(mtiles_bound(a.capacity, a.E, BM) * (N / BN)), s);
}

hipError_t launch_down(const DownArgs& a, hipStream_t s) {
  if (a.d % 256 == 0) {
    constexpr int BM = 256, BN = 256;
    return run<OpDown<BM, BN>>({a}, pad8(mtiles_bound(a.capacity, a.E, BM) * (a.d / BN)), s);
  }
  constexpr int BM = 128, BN = 128;
  return run<OpDown<BM, BN>>({a}, pad8(mtiles_bound(a.capacity, a.E, BM) * (a.d / BN)), s);
}

static int dh_bn(int n) { return n % 256 == 0 ? 256 : (n % 128 == 0 ? 128 : 64); }
int dh_n_tiles(int n) { return n / dh_bn(n); }

hipError_t launch_dh(const DHArgs& a, hipStream_t s) {
  constexpr int BM = 128;
  const int grid = pad8(mtiles_bound(a.capacity, a.E, BM) * dh_n_tiles(a.n));
  switch (dh_bn(a.n)) {
    case 256: return run<OpDH<BM, 256>>({a}, grid, s);
    case 128: return run<OpDH<BM, 128>>({a}, grid, s);
    default: return run<OpDH<BM, 64>>({a}, grid, s);
  }
}

hipError_t launch_dxt(const DXtArgs& a, hipStream_t s) {
  if (a.d % 256 == 0) {
    constexpr int BM = 256, BN = 256;
    return run<OpDXt<BM, BN>>({a}, pad8(mtiles_bound(a.capacity, a.E, BM) * (a.d / BN)), s);
  }
  constexpr int BM = 128, BN = 128;
  return run<OpDXt<BM, BN>>({a}, pad8(mtiles_bound(a.capacity, a.E, BM) * (a.d / BN)), s);
}

hipError_t launch_dw2(const DW2Args& a, hipStream_t s) {
  // M = n, N = d
  if (a.n % 128 == 0 && a.d % 256 == 0) {
    constexpr int BM = 128, BN = 256;
    return run<OpDW2<BM, BN>>({a}, pad8(a.E * (a.n / BM) * (a.d / BN)), s);
  }
  constexpr int BM = 64, BN = 128;
  return run<OpDW2<BM, BN>>({a}, pad8(a.E * (a.n / BM) * (a.d / BN)), s);
}

hipError_t launch_dw1(const DW1Args& a, hipStream_t s) {
  // M = d, N = 2n
  if (a.d % 256 == 0 && (2 * a.n) % 256 == 0) {
    constexpr int BM = 256, BN = 256;
    return run<OpDW1<BM, BN>>({a}, pad8(a.E * (a.d / BM) * (2 * a.n / BN)), s);
  }
  constexpr int BM = 128, BN = 128;
  return run<OpDW1<BM, BN>>({a}, pad8(a.E * (a.d / BM) * (2 * a.n / BN)), s);
}

int dwr_splits(int T, int d, int E) {
  const int tiles = (d / 128) * ((E + 127) / 128);
  int s = (512 + tiles - 1) / tiles;  // aim for ~512 workgroups
  const int max_s = (T + 255) / 256;  // at least 256 tokens per split
  if (s > max_s) s = max_s;
  return s < 1 ? 1 : s;
}

hipError_t launch_dwr(const DWrArgs& a, hipStream_t s) {
  hipError_t err;
  const int mtn = a.d / 128;
  if (a.E <= 64)
    err = run<OpDWr<64>>({a}, a.splits * mtn, s);
  else if (a.E <= 128)
    err = run<OpDWr<128>>({a}, a.splits * mtn, s);
  else
    err = run<OpDWr<256>>({a}, a.splits * mtn * ((a.E + 255) / 256), s);
  if (err != hipSuccess) return err;
  return launch_reduce_rows(a.part, a.dWr, a.d * a.E, a.splits, s);
}

}  // namespace smoe
