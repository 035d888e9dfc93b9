// Internal launchers of the HIP kernels (host side, C++).  The C ABI in
// moe_abi.cpp validates arguments, carves workspaces and calls these.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sonicmoe.h"

namespace smoe {

// routing
hipError_t launch_topk_route(const float* in, float* scores, float* scores_t, int32_t* topk_idx, float* topk_w,
                             uint64_t* mask, int T, int E, int K, int W, int do_softmax, hipStream_t s);
hipError_t launch_tc_metadata(const moe_routing& r, int T, int E, int K, bool counts_only, hipStream_t s);
// counted: r.mask_prefix and r.counts are already written (by launch_round)
hipError_t launch_metadata(const moe_routing& r, const float* scores_t, int T, int E, bool counted, hipStream_t s);
// list: round_scratch_bytes(T, E) bytes (8-byte aligned) for the selection's
// lists
size_t round_scratch_bytes(int T, int E);
hipError_t launch_round(const moe_routing& tc, moe_routing& tr, const float* u, int T, int E, int M, int mode,
                        uint64_t* list, bool* counted, hipStream_t s);

// GEMMs (all bf16 in, fp32 accumulation)
struct RouterGemmArgs {
  const uint16_t* X; const uint16_t* Wr; const float* bias; float* logits; int T, d, E;
};
hipError_t launch_router_gemm(const RouterGemmArgs& a, hipStream_t s);
// The router GEMM with softmax and top-K fused into its epilogue (one tile
// spans every expert): the outputs of launch_topk_route with do_softmax = 1,
// and the logits too when logits is not null.
struct RouterTopkArgs {
  const uint16_t* X; const uint16_t* Wr; const float* bias;
  float* logits; float* scores; float* scores_t; int32_t* topk_idx; float* topk_w; uint64_t* mask;
  int T, d, E, K, W;
};
bool router_topk_fusable(int E, int K);
hipError_t launch_router_topk(const RouterTopkArgs& a, hipStream_t s);

// The varlen-M m-tile list (mtiles_kernel): built from the expert offsets
// once per forward / backward call, read by the up, down, dH and dX~ GEMMs.
size_t mtiles_bytes(int64_t capacity, int E);
hipError_t launch_mtiles(const int32_t* offsets, int E, int32_t* out, hipStream_t s);

struct UpArgs {
  const uint16_t* X; const uint16_t* W1; const int32_t* offsets; const int32_t* row_token;
  uint16_t* H; uint16_t* A; int d, n, E, capacity; const int32_t* mtiles;
  const float* b1;  // [E,2n] expert bias added to H, or null
};
hipError_t launch_up(const UpArgs& a, hipStream_t s);

struct DownArgs {
  const uint16_t* A; const uint16_t* W2; const int32_t* offsets; uint16_t* Y; int d, n, E, capacity;
  const int32_t* mtiles;
  const float* b2;  // [E,d] expert bias added to Y, or null
  // aggregation ablation only: token-major destination row of each row
  // (scatter), or the fp32 output and the row tokens / weights (atomics)
  const int32_t* dst = nullptr; float* O32 = nullptr; const int32_t* row_token = nullptr;
  const float* row_w = nullptr;
};
hipError_t launch_down(const DownArgs& a, hipStream_t s);
// strategy 0: as launch_down; 1: Y rows scattered to a.dst[row]; 2: fp32
// atomic accumulation of s * Y into a.O32 (no Y stored)
hipError_t launch_down_ablation(const DownArgs& a, int strategy, hipStream_t s);

struct DHArgs {
  const uint16_t* dO; const uint16_t* W2; const uint16_t* H; const int32_t* offsets; const int32_t* row_token;
  const float* row_w; uint16_t* dH; uint16_t* Ap; float* dS; float* dS_part; int d, n, E, capacity;
  const int32_t* mtiles;
  // <dO_t, b2_e> of the expert-bias dS term as two fp32 halves [T][2E]
  // (columns e and E + e; see launch_bias_split), or null
  const float* bq;
};
int dh_n_tiles(int n);
hipError_t launch_dh(const DHArgs& a, hipStream_t s);

struct DXtArgs {
  const uint16_t* dH; const uint16_t* W1; const int32_t* offsets; uint16_t* dXt; int d, n, E, capacity;
  const int32_t* mtiles;
};
hipError_t launch_dxt(const DXtArgs& a, hipStream_t s);

// Weight gradients (varlen K over each expert's rows).  klist: the GEMM's
// k-chunk list (kchunks_bytes(E) bytes, written by launch_bwd_lists); part:
// dw_part_bytes(d, n) bytes of fp32 partials for experts split into row
// chunks.
constexpr int kDwSlabs = 128;                                // partial slabs per GEMM at most
constexpr int64_t kDwSlabBytes = (int64_t)256 << 20;         // and at most this many bytes
size_t kchunks_bytes(int E);
size_t dw_part_bytes(int d, int n);
int dw_slabs(int64_t mn);
// the backward's m-tile list (as launch_mtiles) and the k-chunk lists of dW2
// and dW1, in one launch; with Wr non-null the same launch writes WrT[e][i] =
// Wr[i][e] (the dX aggregation's router term reads W_r by expert)
hipError_t launch_bwd_lists(const int32_t* offsets, int E, int d, int n, int32_t* mtiles, int32_t* klist2,
                            int32_t* klist1, const uint16_t* Wr, uint16_t* WrT, hipStream_t s);

struct DW2Args {
  const uint16_t* Ap; const uint16_t* dO; const int32_t* offsets; const int32_t* row_token; uint16_t* dW2;
  int d, n, E;
  int32_t* klist; float* part;
};
hipError_t launch_dw2(const DW2Args& a, hipStream_t s);

struct DW1Args {
  const uint16_t* X; const uint16_t* dH; const int32_t* offsets; const int32_t* row_token; uint16_t* dW1;
  int d, n, E;
  int32_t* klist; float* part;
};
hipError_t launch_dw1(const DW1Args& a, hipStream_t s);

struct DWrArgs {
  const uint16_t* X; const uint16_t* dL; float* part; float* dWr; int T, d, E, splits;
};
int dwr_splits(int T, int d, int E);
hipError_t launch_dwr(const DWrArgs& a, hipStream_t s);

// Expert biases.  The down-projection bias term of dS, <dO_t, b2_e> for every
// (t, e), is one GEMM dO [T,d] x B2s [d,2E] on the router GEMM's path: B2s
// holds b2^T split into bf16 high and low parts (columns e and E + e), whose
// products with the bf16 dO are exact in the fp32 accumulation, so the term
// keeps about 16 bits of b2.  launch_bias_split writes B2s.
hipError_t launch_bias_split(const float* b2, int E, int d, uint16_t* B2s, hipStream_t s);
// out[e][c] = sum over the rows r of expert e of w_r * src[g(r)][c], with
// g(r) = row_token[r] (or r when row_token is null) and w_r = row_w[r] (or 1);
// fixed summation order, fp32.
hipError_t launch_expert_colsum(const uint16_t* src, int64_t ld, int cols, const int32_t* offsets,
                                const int32_t* row_token, const float* row_w, int E, float* out, hipStream_t s);

// aggregation and small kernels
hipError_t launch_agg_o(const uint16_t* Y, const moe_routing& r, uint16_t* O, int T, int d, hipStream_t s);
// aggregation ablation: dst[tok_rows[j]] = j (token-major slot of each row);
// O from token-major (contiguous) Y rows; fp32 buffer fill and fp32 -> bf16
hipError_t launch_tok_slots(const moe_routing& r, int T, int P_bound, int32_t* dst, hipStream_t s);
hipError_t launch_agg_o_contig(const uint16_t* Yt, const moe_routing& r, uint16_t* O, int T, int d, hipStream_t s);
hipError_t launch_fill_f32(float* p, size_t n, hipStream_t s);
hipError_t launch_f32_to_bf16(const float* in, uint16_t* out, size_t n, hipStream_t s);
hipError_t launch_agg_dx(const uint16_t* dXt, const float* dS, const uint16_t* WrT, const moe_routing& r, uint16_t* dX,
                         uint16_t* dL, int T, int d, int E, hipStream_t s);
hipError_t launch_reduce_rowparts(const float* part, float* out, int rows, int parts, hipStream_t s);
// dbias = column sums of dL [T][E]: per-chunk sums into part (colsum_chunks(T)
// * E floats), then launch_bwd_final_reduce sums them.  That launch also sums
// the dW1 chunk slabs of split experts (launch_dw1 leaves them) and the dW_r
// split-K partials (dwr_part: splits x d x E floats); dWr and dbias may be null.
int colsum_chunks(int T);
hipError_t launch_colsum_rows(const uint16_t* dL, float* part, int T, int E, hipStream_t s);
hipError_t launch_bwd_final_reduce(const int32_t* klist1, const float* part1, uint16_t* dW1, int d, int n,
                                   const float* dwr_part, float* dWr, int splits, const float* cs_part, float* dbias,
                                   int T, int E, hipStream_t s);

// timing hooks (moe_abi.cpp)
void prof_begin(int kernel_class, hipStream_t s);
void prof_end(int kernel_class, hipStream_t s);

}  // namespace smoe
