// Expert aggregation (gather-and-sum) and the small helper kernels.
//
// Forward O kernel (Section 3, forward algorithm): every token gathers its
// experts' Y rows and sums them weighted by the routing scores.  Backward dX
// kernel (Appendix E, up-projection backward): the same gather-and-sum over
// dX~ rows, with the router's gradient term fused in.  Each token is owned by
// one wave, so the sum order is fixed and no atomics are used (the paper's
// gather-and-sum choice keeps the result deterministic).
#include "device_common.h"
#include "launch.h"

namespace smoe {

constexpr int kAggBatch = 8;  // rows whose loads are in flight together
constexpr int kColRows = 32;  // tokens per chunk of the dbias column sum
constexpr int kDLPerLane = 4;  // router-gradient row entries per lane collected in registers (E <= 256)
static_assert(kAggBatch == 8, "lane & 7 picks a batch slot");

__device__ __forceinline__ int bcast_i(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ float bcast_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// One wave per token; lanes cover 8 consecutive bf16 (16 bytes) of the row,
// in NC chunks of 512 columns starting at column c0.  The token's rows are taken kAggBatch at a time
// without branches: lanes 0..7 fetch the batch's row indices and weights
// (padding slots clamped to the token's last row, weight 0) and broadcast
// them, then the row loads of every chunk are issued before any is
// accumulated, so a lane keeps NC * kAggBatch HBM reads in flight.  Every Y
// row is read exactly once and O is not read again here: both go through the
// caches as nontemporal accesses.
// CONTIG (the aggregation ablation's scatter + sum): Y holds the rows in
// token-major order, so the token's rows are Y[j0 .. j1) themselves.
template <int NC, bool CONTIG = false>
__global__ __launch_bounds__(256) void agg_o_kernel(const uint16_t* __restrict__ Y, const int32_t* __restrict__ tok_offsets,
                                                    const int32_t* __restrict__ tok_rows, const float* __restrict__ row_w,
                                                    uint16_t* __restrict__ O, int T, int d, int c0) {
  // wave-uniform token: row indices and weights become scalar loads
  const int t = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (t >= T) return;
  const int lane = lane_id();
  const int j0 = tok_offsets[t], j1 = tok_offsets[t + 1];
  float acc[NC][8];
#pragma unroll
  for (int ci = 0; ci < NC; ++ci)
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[ci][q] = 0.f;
  for (int jb = j0; jb < j1; jb += kAggBatch) {
    const int slot = jb + (lane & 7);
    const int rl = tok_rows[min(slot, j1 - 1)];
    const float wl = slot < j1 ? row_w[rl] : 0.f;
    int r[kAggBatch];
    float w[kAggBatch];
#pragma unroll
    for (int u = 0; u < kAggBatch; ++u) {
      r[u] = CONTIG ? min(jb + u, j1 - 1) : bcast_i(rl, u);
      w[u] = bcast_f(wl, u);
    }
    u32x4 v[NC][kAggBatch];
#pragma unroll
    for (int ci = 0; ci < NC; ++ci) {
      const int c = min(c0 + lane * 8 + 512 * ci, d - 8);  // lanes past the row end re-read its last chunk
#pragma unroll
      for (int u = 0; u < kAggBatch; ++u) v[ci][u] = __builtin_nontemporal_load((const u32x4*)(Y + (size_t)r[u] * d + c));
    }
#pragma unroll
    for (int ci = 0; ci < NC; ++ci)
#pragma unroll
      for (int u = 0; u < kAggBatch; ++u)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[ci][2 * q] += w[u] * bf_lo(v[ci][u][q]);
          acc[ci][2 * q + 1] += w[u] * bf_hi(v[ci][u][q]);
        }
  }
#pragma unroll
  for (int ci = 0; ci < NC; ++ci) {
    const int c = c0 + lane * 8 + 512 * ci;
    if (c < d) {
      u32x4 o;
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = pack_bf2(acc[ci][2 * q], acc[ci][2 * q + 1]);
      __builtin_nontemporal_store(o, (u32x4*)(O + (size_t)t * d + c));
    }
  }
}

// dX_t = sum over the token's rows of dX~ + sum_j dl_j W_r[:, e_j], with the
// router gradient on the token's selected set dl_j = s_j (dS_j - sum_k s_k dS_k).
// Also writes the dense router-logit gradient row dL[t, :] (bf16) for dW_r
// (when dL is given; the launch for column slice 0 does it).
// W_r^T [E][d] is a bf16 copy (exact: W_r is bf16), so each row term is one
// 16-byte load per lane.  As in the forward kernel, a batch's dX~ rows are
// requested for every column chunk before any is accumulated; the W_r^T rows
// (a few hundred KB, cache resident) follow chunk by chunk.
template <int NC>
__global__ __launch_bounds__(256) void agg_dx_kernel(const uint16_t* __restrict__ dXt, const float* __restrict__ dS,
                                                     const uint16_t* __restrict__ WrT,
                                                     const int32_t* __restrict__ tok_offsets,
                                                     const int32_t* __restrict__ tok_rows,
                                                     const int32_t* __restrict__ row_expert,
                                                     const float* __restrict__ row_w, uint16_t* __restrict__ dX,
                                                     uint16_t* __restrict__ dL, int T, int d, int E, int c0) {
  // wave-uniform token: row indices and weights become scalar loads
  const int t = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (t >= T) return;
  const int lane = lane_id();
  const int j0 = tok_offsets[t], j1 = tok_offsets[t + 1];
  // g = sum_k s_k dS_k in row order; lanes 0..7 fetch a batch's terms.  A
  // token whose rows fit one batch (every token-choice token with K <= 8,
  // most rounded ones) forms g in the main loop's only iteration instead, from
  // the weights and dS values that iteration loads anyway: one round trip of
  // dependent loads fewer before its dX~ rows are requested.
  const bool one_batch = j1 - j0 <= kAggBatch;
  float g = 0.f;
  if (WrT && !one_batch)
    for (int jb = j0; jb < j1; jb += kAggBatch) {
      const int slot = jb + (lane & 7);
      const int rl = tok_rows[min(slot, j1 - 1)];
      const float pl = slot < j1 ? row_w[rl] * dS[rl] : 0.f;
#pragma unroll
      for (int u = 0; u < kAggBatch; ++u) g += bcast_f(pl, u);
    }
  // dL[t, e] for e = lane + 64 q (q < kDLPerLane), collected from the batches
  const bool dl_fast = dL != nullptr && E <= 64 * kDLPerLane;
  float dlv[kDLPerLane] = {0.f, 0.f, 0.f, 0.f};
  float acc[NC][8];
#pragma unroll
  for (int ci = 0; ci < NC; ++ci)
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[ci][q] = 0.f;
  for (int jb = j0; jb < j1; jb += kAggBatch) {
    // slot lane&7 of the batch: one vector load per level, then broadcast
    const int slot = jb + (lane & 7);
    const int rl = tok_rows[min(slot, j1 - 1)];
    const int el = WrT ? row_expert[rl] : 0;
    if (WrT && one_batch) {
      const float pl = slot < j1 ? row_w[rl] * dS[rl] : 0.f;
#pragma unroll
      for (int u = 0; u < kAggBatch; ++u) g += bcast_f(pl, u);
    }
    const float dll = (WrT && slot < j1) ? row_w[rl] * (dS[rl] - g) : 0.f;
    int r[kAggBatch];
#pragma unroll
    for (int u = 0; u < kAggBatch; ++u) r[u] = bcast_i(rl, u);
    u32x4 v[NC][kAggBatch];
#pragma unroll
    for (int ci = 0; ci < NC; ++ci) {
      const int c = min(c0 + lane * 8 + 512 * ci, d - 8);  // lanes past the row end re-read its last chunk
#pragma unroll
      for (int u = 0; u < kAggBatch; ++u) v[ci][u] = __builtin_nontemporal_load((const u32x4*)(dXt + (size_t)r[u] * d + c));
    }
    float keep[kAggBatch];
#pragma unroll
    for (int u = 0; u < kAggBatch; ++u) keep[u] = jb + u < j1 ? 1.f : 0.f;  // padding slots re-read the last row
#pragma unroll
    for (int ci = 0; ci < NC; ++ci)
#pragma unroll
      for (int u = 0; u < kAggBatch; ++u)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[ci][2 * q] += keep[u] * bf_lo(v[ci][u][q]);
          acc[ci][2 * q + 1] += keep[u] * bf_hi(v[ci][u][q]);
        }
    if (WrT) {
#pragma unroll
      for (int ci = 0; ci < NC; ++ci) {
        const int c = min(c0 + lane * 8 + 512 * ci, d - 8);
        u32x4 wv[kAggBatch];
#pragma unroll
        for (int u = 0; u < kAggBatch; ++u) wv[u] = *(const u32x4*)(WrT + (size_t)bcast_i(el, u) * d + c);
#pragma unroll
        for (int u = 0; u < kAggBatch; ++u) {
          const float dl = bcast_f(dll, u);  // 0 for padding slots
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            acc[ci][2 * q] += dl * bf_lo(wv[u][q]);
            acc[ci][2 * q + 1] += dl * bf_hi(wv[u][q]);
          }
        }
      }
      if (dl_fast)
#pragma unroll
        for (int u = 0; u < kAggBatch; ++u) {
          const int e = bcast_i(el, u);
          const float dl = bcast_f(dll, u);
#pragma unroll
          for (int q = 0; q < kDLPerLane; ++q)
            if (jb + u < j1 && e == lane + 64 * q) dlv[q] = dl;
        }
    }
  }
#pragma unroll
  for (int ci = 0; ci < NC; ++ci) {
    const int c = c0 + lane * 8 + 512 * ci;
    if (c < d) {
      u32x4 o;
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = pack_bf2(acc[ci][2 * q], acc[ci][2 * q + 1]);
      __builtin_nontemporal_store(o, (u32x4*)(dX + (size_t)t * d + c));
    }
  }
  if (dl_fast) {
#pragma unroll
    for (int q = 0; q < kDLPerLane; ++q)
      if (lane + 64 * q < E) dL[(size_t)t * E + lane + 64 * q] = f2bf(dlv[q]);
  } else if (dL) {
    for (int e = lane; e < E; e += 64) {
      float v = 0.f;
      for (int j = j0; j < j1; ++j) {
        const int r = tok_rows[j];
        if (row_expert[r] == e) v = row_w[r] * (dS[r] - g);
      }
      dL[(size_t)t * E + e] = f2bf(v);
    }
  }
}

// out[i] = sum_k part[i * parts + k] (fixed order)
__global__ __launch_bounds__(256) void reduce_rowparts_kernel(const float* __restrict__ part, float* __restrict__ out,
                                                              int n, int parts) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int k = 0; k < parts; ++k) s += part[(size_t)i * parts + k];
  out[i] = s;
}

// dbias[e] = sum_t dL[t][e] in two fixed-order passes: per chunk of
// kColRows tokens a column sum (reads of a row are contiguous across the
// block), then one block per expert reduces the chunk sums with a fixed tree
// (in bwd_final_reduce_kernel).
__global__ __launch_bounds__(128) void colsum_rows_kernel(const uint16_t* __restrict__ dL, float* __restrict__ part,
                                                          int T, int E) {
  const int r0 = blockIdx.x * kColRows, r1 = min(T, r0 + kColRows);
  for (int c = threadIdx.x; c < E; c += 128) {
    float s = 0.f;
#pragma unroll 8
    for (int r = r0; r < r1; ++r) s += bf2f(dL[(size_t)r * E + c]);
    part[(size_t)blockIdx.x * E + c] = s;
  }
}

// ---------------------------------------------------------------- expert biases
// B2s[k][e] = hi(b2[e][k]) and B2s[k][E + e] = bf16(b2[e][k] - hi), hi = the
// round-to-nearest bf16 of b2[e][k]: the layout of W_r [d][E'] with E' = 2E,
// so the router GEMM forms dO B2s, i.e. <dO_t, hi_e> and <dO_t, lo_e>.
__global__ __launch_bounds__(256) void bias_split_kernel(const float* __restrict__ b2, int E, int d,
                                                         uint16_t* __restrict__ B2s) {
  const int i = blockIdx.x * 256 + threadIdx.x;  // over d x E, e fastest
  if (i >= d * E) return;
  const int k = i / E, e = i % E;
  const float v = b2[(size_t)e * d + k];
  const uint16_t hi = f2bf(v);
  B2s[(size_t)k * 2 * E + e] = hi;
  B2s[(size_t)k * 2 * E + E + e] = f2bf(v - bf2f(hi));
}

// One workgroup per (expert, 512-column chunk).  Wave w sums the expert's
// rows w, w + 4, w + 8, ... (four rows' loads in flight per step), lane l owns
// columns 8l .. 8l + 7 of the chunk; the four wave sums are added in wave
// order through LDS, so the result does not depend on timing.
constexpr int kColsumWaves = 4;
__global__ __launch_bounds__(64 * kColsumWaves) void expert_colsum_kernel(
    const uint16_t* __restrict__ src, int64_t ld, int cols, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ row_token, const float* __restrict__ row_w, float* __restrict__ out) {
  __shared__ float red[kColsumWaves][512];
  const int e = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = lane_id();
  const int c = blockIdx.y * 512 + lane * 8;
  const bool live = c < cols;
  const int r0 = offsets[e], r1 = offsets[e + 1];
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  constexpr int kU = 4;
  for (int rb = r0 + wave; rb < r1; rb += kColsumWaves * kU) {
    u32x4 v[kU];
    float w[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int r = rb + u * kColsumWaves;
      const bool ok = r < r1 && live;
      const int g = ok ? (row_token ? row_token[r] : r) : 0;
      w[u] = ok ? (row_w ? row_w[r] : 1.f) : 0.f;
      v[u] = ok ? *(const u32x4*)(src + (size_t)g * ld + c) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[2 * q] += w[u] * bf_lo(v[u][q]);
        acc[2 * q + 1] += w[u] * bf_hi(v[u][q]);
      }
  }
#pragma unroll
  for (int q = 0; q < 8; ++q) red[wave][lane * 8 + q] = acc[q];
  __syncthreads();
  for (int i = threadIdx.x; i < 512; i += 64 * kColsumWaves) {
    const int cc = blockIdx.y * 512 + i;
    if (cc >= cols) continue;
    float t = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < kColsumWaves; ++w2) t += red[w2][i];
    out[(size_t)e * cols + cc] = t;
  }
}

hipError_t launch_bias_split(const float* b2, int E, int d, uint16_t* B2s, hipStream_t s) {
  bias_split_kernel<<<dim3((d * E + 255) / 256), dim3(256), 0, s>>>(b2, E, d, B2s);
  return hipGetLastError();
}

hipError_t launch_expert_colsum(const uint16_t* src, int64_t ld, int cols, const int32_t* offsets,
                                const int32_t* row_token, const float* row_w, int E, float* out, hipStream_t s) {
  if (cols % 8) return hipErrorInvalidValue;  // 16-byte column groups
  expert_colsum_kernel<<<dim3(E, (cols + 511) / 512), dim3(64 * kColsumWaves), 0, s>>>(src, ld, cols, offsets,
                                                                                        row_token, row_w, out);
  return hipGetLastError();
}

hipError_t launch_agg_o(const uint16_t* Y, const moe_routing& r, uint16_t* O, int T, int d, hipStream_t s) {
  const dim3 grid((T + 3) / 4), block(256);
  const int nc = (d + 511) / 512;
  if (nc <= 1) agg_o_kernel<1><<<grid, block, 0, s>>>(Y, r.tok_offsets, r.tok_rows, r.row_w, O, T, d, 0);
  else if (nc == 2) agg_o_kernel<2><<<grid, block, 0, s>>>(Y, r.tok_offsets, r.tok_rows, r.row_w, O, T, d, 0);
  else if (nc == 3) agg_o_kernel<3><<<grid, block, 0, s>>>(Y, r.tok_offsets, r.tok_rows, r.row_w, O, T, d, 0);
  else  // rows wider than 1536: 2048-column slices, one launch each
    for (int c0 = 0; c0 < d; c0 += 2048)
      agg_o_kernel<4><<<grid, block, 0, s>>>(Y, r.tok_offsets, r.tok_rows, r.row_w, O, T, d, c0);
  return hipGetLastError();
}

hipError_t launch_agg_o_contig(const uint16_t* Yt, const moe_routing& r, uint16_t* O, int T, int d, hipStream_t s) {
  const dim3 grid((T + 3) / 4), block(256);
  const int nc = (d + 511) / 512;
  if (nc <= 1) agg_o_kernel<1, true><<<grid, block, 0, s>>>(Yt, r.tok_offsets, r.tok_rows, r.row_w, O, T, d, 0);
  else if (nc == 2) agg_o_kernel<2, true><<<grid, block, 0, s>>>(Yt, r.tok_offsets, r.tok_rows, r.row_w, O, T, d, 0);
  else if (nc == 3) agg_o_kernel<3, true><<<grid, block, 0, s>>>(Yt, r.tok_offsets, r.tok_rows, r.row_w, O, T, d, 0);
  else
    for (int c0 = 0; c0 < d; c0 += 2048)
      agg_o_kernel<4, true><<<grid, block, 0, s>>>(Yt, r.tok_offsets, r.tok_rows, r.row_w, O, T, d, c0);
  return hipGetLastError();
}

// dst[tok_rows[j]] = j for the j < tok_offsets[T] (token-major slot of each row)
__global__ __launch_bounds__(256) void tok_slots_kernel(const int32_t* __restrict__ tok_offsets,
                                                        const int32_t* __restrict__ tok_rows, int T, int n,
                                                        int32_t* __restrict__ dst) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j < n && j < tok_offsets[T]) dst[tok_rows[j]] = j;
}

__global__ __launch_bounds__(256) void fill_f32_kernel(float* __restrict__ p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) p[i] = 0.f;
}

__global__ __launch_bounds__(256) void f32_to_bf16_kernel(const float* __restrict__ in, uint16_t* __restrict__ out,
                                                          size_t n) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) out[i] = f2bf(in[i]);
}

hipError_t launch_tok_slots(const moe_routing& r, int T, int P_bound, int32_t* dst, hipStream_t s) {
  if (P_bound > 0) tok_slots_kernel<<<dim3((P_bound + 255) / 256), dim3(256), 0, s>>>(r.tok_offsets, r.tok_rows, T,
                                                                                     P_bound, dst);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, size_t n, hipStream_t s) {
  fill_f32_kernel<<<dim3(2048), dim3(256), 0, s>>>(p, n);
  return hipGetLastError();
}

hipError_t launch_f32_to_bf16(const float* in, uint16_t* out, size_t n, hipStream_t s) {
  f32_to_bf16_kernel<<<dim3(2048), dim3(256), 0, s>>>(in, out, n);
  return hipGetLastError();
}

hipError_t launch_agg_dx(const uint16_t* dXt, const float* dS, const uint16_t* WrT, const moe_routing& r, uint16_t* dX,
                         uint16_t* dL, int T, int d, int E, hipStream_t s) {
  const dim3 grid((T + 3) / 4), block(256);
  const int nc = (d + 511) / 512;
  if (nc <= 1)
    agg_dx_kernel<1><<<grid, block, 0, s>>>(dXt, dS, WrT, r.tok_offsets, r.tok_rows, r.row_expert, r.row_w, dX, dL, T,
                                            d, E, 0);
  else if (nc == 2)
    agg_dx_kernel<2><<<grid, block, 0, s>>>(dXt, dS, WrT, r.tok_offsets, r.tok_rows, r.row_expert, r.row_w, dX, dL, T,
                                            d, E, 0);
  else if (nc == 3)
    agg_dx_kernel<3><<<grid, block, 0, s>>>(dXt, dS, WrT, r.tok_offsets, r.tok_rows, r.row_expert, r.row_w, dX, dL, T,
                                            d, E, 0);
  else  // rows wider than 1536: 2048-column slices, one launch each; the first writes dL
    for (int c0 = 0; c0 < d; c0 += 2048)
      agg_dx_kernel<4><<<grid, block, 0, s>>>(dXt, dS, WrT, r.tok_offsets, r.tok_rows, r.row_expert, r.row_w, dX,
                                              c0 == 0 ? dL : nullptr, T, d, E, c0);
  return hipGetLastError();
}

hipError_t launch_reduce_rowparts(const float* part, float* out, int rows, int parts, hipStream_t s) {
  reduce_rowparts_kernel<<<dim3((rows + 255) / 256), dim3(256), 0, s>>>(part, out, rows, parts);
  return hipGetLastError();
}

int colsum_chunks(int T) { return (T + kColRows - 1) / kColRows; }

hipError_t launch_colsum_rows(const uint16_t* dL, float* part, int T, int E, hipStream_t s) {
  const int chunks = colsum_chunks(T);
  if (chunks > 0) colsum_rows_kernel<<<dim3(chunks), dim3(128), 0, s>>>(dL, part, T, E);
  return hipGetLastError();
}


}  // namespace smoe
