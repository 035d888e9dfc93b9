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
hipError_t launch_round(const moe_routing& tc, moe_routing& tr, const float* u, int T, int E, int M, int mode,
                        bool* counted, hipStream_t s);

// GEMMs (all bf16 in, fp32 accumulation)
struct RouterGemmArgs {
  const uint16_t* X; const uint16_t* Wr; const float* bias; float* logits; int T, d, E;
};
hipError_t launch_router_gemm(const RouterGemmArgs& a, hipStream_t s);

// The varlen-M m-tile list (mtiles_kernel): built from the expert offsets
// once per forward / backward call, read by the up, down, dH and dX~ GEMMs.
size_t mtiles_bytes(int64_t capacity, int E);
hipError_t launch_mtiles(const int32_t* offsets, int E, int32_t* out, hipStream_t s);

struct UpArgs {
  const uint16_t* X; const uint16_t* W1; const int32_t* offsets; const int32_t* row_token;
  uint16_t* H; uint16_t* A; int d, n, E, capacity; const int32_t* mtiles;
};
hipError_t launch_up(const UpArgs& a, hipStream_t s);

struct DownArgs {
  const uint16_t* A; const uint16_t* W2; const int32_t* offsets; uint16_t* Y; int d, n, E, capacity;
  const int32_t* mtiles;
};
hipError_t launch_down(const DownArgs& a, hipStream_t s);

struct DHArgs {
  const uint16_t* dO; const uint16_t* W2; const uint16_t* H; const int32_t* offsets; const int32_t* row_token;
  const float* row_w; uint16_t* dH; uint16_t* Ap; float* dS; float* dS_part; int d, n, E, capacity;
  const int32_t* mtiles;
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

// aggregation and small kernels
hipError_t launch_agg_o(const uint16_t* Y, const moe_routing& r, uint16_t* O, int T, int d, hipStream_t s);
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
