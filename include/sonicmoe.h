/*
 * sonicmoe.h -- C ABI of an MI355X (gfx950) implementation of the SonicMoE
 * layer: "SonicMoE: Accelerating MoE with IO and Tile-aware Optimizations"
 * (arXiv 2512.14080).
 *
 * The layer follows the paper's problem statement (Appendix A, notation table):
 *   X[T,d]            token embeddings
 *   W_r[d,E]          router weights (token-choice top-K, Section 2.3)
 *   W1[E,d,2n]        expert up-projections; columns [0,n) are the SwiGLU gate,
 *                     columns [n,2n) the up branch
 *   W2[E,n,d]         expert down-projections
 *   K                 experts per token
 *
 * Conventions for every entry point:
 *   - bf16 tensors are raw IEEE bfloat16 bit patterns (uint16_t).
 *   - Every pointer is a DEVICE pointer unless stated otherwise, caller-owned,
 *     row-major and contiguous.  The library never allocates device memory,
 *     never synchronises the stream and keeps no pointer after it returns.
 *   - `stream` is a hipStream_t (NULL = the default stream); all work is
 *     enqueued asynchronously on it.
 *   - Arguments are validated on the host before anything is enqueued; on a
 *     validation error nothing is enqueued and a negative MOE_ERR_* code is
 *     returned.  moe_last_error() returns a thread-local description of the
 *     last failure.  A HIP launch failure returns MOE_ERR_HIP.
 *   - Outputs are overwritten, never accumulated into.
 */
#ifndef SONICMOE_H
#define SONICMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t moe_bf16;

typedef struct {
  int32_t T; /* tokens in the microbatch, >= 1 */
  int32_t d; /* model dimension, multiple of 128 */
  int32_t n; /* expert intermediate dimension, multiple of 64 */
  int32_t E; /* experts, multiple of 8, <= 4096 */
  int32_t K; /* experts per token, 1 <= K <= min(E, 16) */
} moe_dims;

/* Error codes. */
enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = -1, /* null pointer, bad size, misaligned pointer   */
  MOE_ERR_UNSUPPORTED = -2, /* a shape outside the supported range          */
  MOE_ERR_CAPACITY = -3,    /* routing capacity below the worst-case rows   */
  MOE_ERR_WORKSPACE = -4,   /* workspace smaller than moe_workspace_bytes() */
  MOE_ERR_HIP = -5          /* a HIP runtime call or kernel launch failed   */
};

/*
 * Routing metadata of one routing matrix pi in {0,1}^{T x E} (Appendix A) and
 * its softmax scores.  "Rows" are routed (token, expert) pairs; P = sum_e f_e
 * of them exist after routing (P = T*K for token choice).  All arrays live in
 * one caller-allocated device buffer laid out by moe_routing_init().
 *
 * Integer results are a deterministic function of the fp32 scores:
 *   - experts are selected by (score descending, expert index ascending);
 *   - expert-major rows are ordered by (expert ascending, token ascending);
 *   - each token's rows are listed by expert ascending.
 */
typedef struct {
  int32_t capacity;      /* rows the row_* / tok_rows arrays can hold          */
  int32_t words;         /* W = ceil(T/64), 64-bit words per expert in mask    */
  int32_t state;         /* host-side build state, MOE_ROUTING_STATE_*: set by
                            moe_routing_init / moe_route / moe_round_tokens
                            (what has been enqueued), checked by the consumers */
  int32_t reserved;      /* zero                                               */
  float *logits;         /* [T,E] router logits (nullable: MOE_ROUTING_LOGITS)  */
  float *scores;         /* [T,E] S_full = softmax over all E experts          */
  float *scores_t;       /* [E,T] transposed S_full (nullable: MOE_ROUTING_SCORES_T;
                            required by moe_round_tokens on the TC routing)    */
  int32_t *topk_idx;     /* [T,K] TC selection, (score desc, expert asc)       */
  float *topk_w;         /* [T,K] renormalised weights of topk_idx             */
  uint64_t *mask;        /* [E,W] membership bitmap: bit t%64 of word t/64     */
  int32_t *mask_prefix;  /* [E,W] set bits of expert e before each word        */
  int32_t *counts;       /* [E]   f_e, rows per expert                         */
  int32_t *offsets;      /* [E+1] exclusive scan of counts; offsets[E] = P     */
  int32_t *row_token;    /* [capacity] token of each expert-major row (gather) */
  int32_t *row_expert;   /* [capacity] expert of each row                      */
  float *row_w;          /* [capacity] weight s_{t,e} of each row              */
  int32_t *tok_offsets;  /* [T+1] CSR offsets of the token-major view          */
  int32_t *tok_rows;     /* [capacity] rows of each token, expert ascending    */
  int32_t *tok_count;    /* [T]   experts of each token                        */
  float *tok_denom;      /* [T]   sum of the token's selected scores           */
  int32_t *round_dir;    /* [E]   -1 dropped / 0 kept / +1 padded (rounding)   */
  int32_t *scratch;      /* internal: scans and the rounding select's lists    */
  int32_t *status;       /* [1]   device word: 0 once the metadata kernels have
                            run on a consistent selection; otherwise the OR of
                            MOE_STATUS_* bits, and the rows are not valid
                            (every index written is still in bounds)        */
} moe_routing;

/* moe_routing.state */
enum {
  MOE_ROUTING_STATE_EMPTY = 0,  /* laid out by moe_routing_init; nothing written  */
  MOE_ROUTING_STATE_COUNTS = 1, /* mask, mask_prefix, counts (MOE_ROUTE_COUNTS_ONLY) */
  MOE_ROUTING_STATE_BUILT = 2   /* complete metadata: moe_fwd / moe_bwd accept it */
};

/* bits of the device status word */
enum {
  MOE_STATUS_DUPLICATE_EXPERT = 1 /* a token's topk_idx lists an expert twice   */
};

enum {
  MOE_ROUTING_LOGITS = 1,   /* carve the logits array                 */
  MOE_ROUTING_SCORES_T = 2  /* carve the transposed-scores array      */
};

/* Bytes of the routing buffer for `capacity` rows; 0 if the dims are invalid. */
size_t moe_routing_bytes(moe_dims dims, int32_t capacity, int flags);

/* Lays out the routing arrays inside `buf` (device, 256-byte aligned, at least
 * moe_routing_bytes() bytes) and fills `*r` (host struct, state
 * MOE_ROUTING_STATE_EMPTY).  Enqueues nothing. */
int moe_routing_init(moe_dims dims, int32_t capacity, int flags, void *buf, size_t bytes,
                     moe_routing *r);

/* Smallest capacity that token rounding to multiples of m_tile may need:
 * min(T*E, T*K + E*(m_tile-1)); -1 for invalid dims or an m_tile outside
 * the powers of two in [8, 256]. */
int32_t moe_round_capacity(moe_dims dims, int32_t m_tile);

/* moe_route flags */
enum {
  MOE_ROUTE_SCORES_IN = 1,     /* skip the router GEMM and softmax; r->scores is
                                  an input holding S_full                      */
  MOE_ROUTE_WRITE_LOGITS = 2,  /* keep the logits in r->logits                 */
  MOE_ROUTE_WRITE_SCORES_T = 4, /* also write r->scores_t                      */
  MOE_ROUTE_COUNTS_ONLY = 8,    /* metadata stops at mask, mask_prefix and
                                   counts: enough for moe_round_tokens, which
                                   builds the rounded routing's own metadata;
                                   offsets and the row lists are not written,
                                   and r->state becomes MOE_ROUTING_STATE_COUNTS,
                                   which moe_fwd and moe_bwd refuse          */
  MOE_ROUTE_SEPARATE_TOPK = 16  /* run the router GEMM and softmax/top-K as two
                                   launches even where they fuse (the logits
                                   then pass through r->logits or r->scores) */
};

/*
 * Token-choice top-K routing (Section 2.3; top-K selection of Appendix D).
 *   logits = X W_r (+ bias)  fp32 accumulation of bf16 inputs
 *   S_full = softmax over E  (row maximum subtracted)
 *   sel(t) = first K experts by (S_full desc, expert asc)
 *   s_{t,e} = S_full[t,e] / sum_{e' in sel(t)} S_full[t,e']   (denominator
 *             summed over selected experts in ascending index order)
 * then the metadata of the routing matrix: mask, counts, offsets, expert-major
 * rows (row_token, row_expert, row_w), token-major CSR (tok_offsets, tok_rows).
 *   X     [T,d] bf16;  Wr [d,E] bf16 (unused with MOE_ROUTE_SCORES_IN)
 *   bias  [E] fp32, nullable
 * r->capacity must be >= T*K.  On success r->state is MOE_ROUTING_STATE_BUILT
 * (MOE_ROUTING_STATE_COUNTS with MOE_ROUTE_COUNTS_ONLY) and the device word
 * r->status is cleared by the metadata kernels.
 * With E <= 256 and K <= 8 the softmax and top-K run in the
 * router GEMM's epilogue (one launch; the logits are written only with
 * MOE_ROUTE_WRITE_LOGITS).  Its scores may differ from the two-launch path's
 * in the last bits (the order of the softmax sum); selection, mask and weights
 * are those the two-launch path derives from the scores it writes.
 * Scores are compared through the order-preserving image of their fp32 bit
 * pattern, which is the float order for numbers (+0 = -0) and extends it to
 * NaN (sign clear: above +Inf; sign set: below -Inf), so non-finite scores
 * still select K distinct experts per token (their weights are then not
 * finite).  Token rounding orders scores the same way.
 */
int moe_route(moe_dims dims, const moe_bf16 *X, const moe_bf16 *Wr, const float *bias, int flags,
              moe_routing *r, void *stream);

/* rounding subroutines (Section 5.2 and the appendix ablation on rounding) */
enum {
  MOE_ROUND_NEAREST = 0,   /* NR-f: pad iff ceil - f < f - floor (default)        */
  MOE_ROUND_UP = 1,        /* always pad                                          */
  MOE_ROUND_DOWN = 2,      /* always drop (TC token dropping)                     */
  MOE_ROUND_BALANCE = 3,   /* Balance-f: running residual over experts in order   */
  MOE_ROUND_STOCHASTIC = 4 /* SR-f: pad iff u_e * m_tile < f - floor               */
};

/*
 * Token rounding (Section 5.2): rounds every expert's TC frequency f_e to a
 * multiple of m_tile.  Per expert, tokens are ordered by (TC first, score
 * descending, token ascending) and the first f^TR_e are kept, so a rounded-down
 * expert drops its lowest-scored TC tokens and a rounded-up expert adds the
 * highest-scored non-TC tokens; |f^TR_e - f_e| < m_tile.  An expert whose
 * ceiling exceeds T is rounded down.  Weights are renormalised over each
 * token's new expert set.
 *   tc     routing written by moe_route (state at least
 *          MOE_ROUTING_STATE_COUNTS; needs tc->scores_t written, i.e.
 *          MOE_ROUTE_WRITE_SCORES_T)
 *   tr     output routing; tr->capacity >= moe_round_capacity(dims, m_tile);
 *          tr->scores may alias tc->scores (it is read, not written); on
 *          success tr->state is MOE_ROUTING_STATE_BUILT
 *   m_tile power of two in [8, 256] (otherwise MOE_ERR_INVALID_ARG)
 *   u      [E] fp32 uniforms in [0,1), device, required by MOE_ROUND_STOCHASTIC
 */
int moe_round_tokens(moe_dims dims, int32_t m_tile, int mode, const float *u, const moe_routing *tc,
                     moe_routing *tr, void *stream);

/*
 * Optional per-expert biases of the two projections (the expert-bias footnote
 * of the "Gradient computation" appendix).  With them the expert computes
 *   h = x W1_e + b1_e,  y = SwiGLU(h) W2_e + b2_e,
 * and the score gradient dS_{t,e} = <dO_t, y> becomes <dA', A> + <dO_t, b2_e>.
 * Every pointer is a device pointer, fp32, 16-byte aligned, and nullable:
 *   b1   [E,2n] up-projection bias (gate columns first, as W1)
 *   b2   [E,d]  down-projection bias
 *   db1  [E,2n] out of moe_bwd: column sums of dH over the expert's rows
 *   db2  [E,d]  out of moe_bwd: column sums of s * dO_t over the expert's rows
 * Experts without rows get zero bias gradients.  moe_fwd reads b1 and b2;
 * moe_bwd reads b2 (for dS) and writes db1 and db2 where they are given.
 */
typedef struct {
  const float *b1;
  const float *b2;
  float *db1;
  float *db2;
} moe_expert_bias;

/* Workspace bytes for moe_fwd (which = 1), moe_bwd (which = 2) and
 * moe_fwd_aggregation_ablation (which = 3). */
enum { MOE_WS_FWD = 1, MOE_WS_BWD = 2, MOE_WS_FWD_AGG_ABLATION = 3 };
size_t moe_workspace_bytes(moe_dims dims, int32_t capacity, int which);

/*
 * Forward (Section 3, forward algorithm: up-proj A kernel, down-proj Y kernel,
 * expert aggregation O kernel):
 *   H = gather(X) W1_e (+ b1_e)   -> H [capacity,2n] bf16 (cached for backward;
 *                                    the first P rows are written)
 *   A = SiLU(H_gate) * H_up       (workspace)
 *   Y = A W2_e (+ b2_e)           (workspace)
 *   O_t = sum_{rows of t} s * Y   -> O [T,d] bf16 (zero for a token without experts)
 *   eb  expert biases, nullable (b1 and b2 are read; see moe_expert_bias)
 *   r   routing in state MOE_ROUTING_STATE_BUILT (otherwise MOE_ERR_INVALID_ARG)
 *   ws  device workspace of moe_workspace_bytes(dims, r->capacity, MOE_WS_FWD)
 */
int moe_fwd(moe_dims dims, const moe_bf16 *X, const moe_bf16 *W1, const moe_bf16 *W2,
            const moe_expert_bias *eb, const moe_routing *r, moe_bf16 *H, moe_bf16 *O, void *ws,
            size_t ws_bytes, void *stream);

/*
 * Backward (down-projection backward algorithm of Section 3; up-projection
 * backward algorithm of Appendix E; dS identity of the "Gradient computation"
 * appendix), recomputing A from the cached H:
 *   dA' = gather(dO) W2_e^T, dS = <dA', A>, dA = s dA', dH = dSwiGLU(dA, H),
 *   A' = s A, dW2_e = A'^T gather(dO), dX~ = dH W1_e^T, dW1_e = gather(X)^T dH,
 *   dX_t = sum_{rows of t} dX~ + dL_t W_r^T,
 * where the router gradient on each token's selected set is
 *   dl_j = s_j (dS_j - sum_k s_k dS_k)  (softmax over the selected logits),
 *   dW_r = X^T dL, dbias = column sums of dL.
 *   eb   expert biases, nullable: b2 adds <dO_t, b2_e> to dS; db1 and db2 are
 *        written where given (see moe_expert_bias)
 *   r    routing in state MOE_ROUTING_STATE_BUILT (otherwise MOE_ERR_INVALID_ARG)
 *   dO   [T,d] bf16           H [capacity,2n] bf16 from moe_fwd
 *   Wr   [d,E] bf16, nullable: then no router gradient is formed and dX holds
 *        only the expert part
 *   dX   [T,d] bf16 out;  dW1 [E,d,2n] bf16 out;  dW2 [E,n,d] bf16 out
 *        (experts without rows get zero weight gradients)
 *   dWr  [d,E] fp32 out, nullable;  dbias [E] fp32 out, nullable
 *   dS   [capacity] fp32 out, nullable (dS of each expert-major row)
 *   ws   device workspace of moe_workspace_bytes(dims, r->capacity, MOE_WS_BWD)
 */
int moe_bwd(moe_dims dims, const moe_bf16 *dO, const moe_bf16 *X, const moe_bf16 *H,
            const moe_bf16 *W1, const moe_bf16 *W2, const moe_expert_bias *eb, const moe_bf16 *Wr,
            const moe_routing *r,
            moe_bf16 *dX, moe_bf16 *dW1, moe_bf16 *dW2, float *dWr, float *dbias, float *dS, void *ws,
            size_t ws_bytes, void *stream);

/*
 * moe_fwd for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same forward, with its workspace (A, Y and the m-tile list) in a static
 * device array of moe_fwd_static_max_bytes() = 64 MiB that the library holds
 * on every GPU it runs on until the process ends.  No allocation happens in
 * the call.  A routing whose forward workspace
 * (moe_workspace_bytes(dims, r->capacity, MOE_WS_FWD)) exceeds the array is
 * refused with MOE_ERR_WORKSPACE before anything is enqueued.  Every call on
 * one GPU uses that GPU's one array: calls that overlap on a GPU (on
 * different streams, or from different threads without ordering) race.  The
 * array belongs to the current device (hipGetDevice), which must be the
 * stream's.  Other arguments as moe_fwd.
 */
size_t moe_fwd_static_max_bytes(void);
int moe_fwd_static(moe_dims dims, const moe_bf16 *X, const moe_bf16 *W1, const moe_bf16 *W2,
                   const moe_expert_bias *eb, const moe_routing *r, moe_bf16 *H, moe_bf16 *O, void *stream);

/*
 * Expert-aggregation ablation (Appendix F.3 and the expert-aggregation
 * figure of the "Referenced tables" appendix): the forward of moe_fwd with
 * the down-projection and the aggregation done by one of three strategies.
 * Not on the layer's path; it exists to measure the choice.
 *   MOE_AGG_GATHER_SUM   Y stored expert-major, each token gathers and sums
 *                        its rows (what moe_fwd does; deterministic)
 *   MOE_AGG_SCATTER_SUM  the down-projection epilogue scatters each Y row to
 *                        its token-major slot, then a contiguous weighted sum
 *   MOE_AGG_ATOMIC_F32   the epilogue adds s * bf16(Y) into an fp32 O with
 *                        atomics (order-dependent rounding), then O -> bf16
 * No expert biases.  ws: moe_workspace_bytes(dims, r->capacity,
 * MOE_WS_FWD_AGG_ABLATION) bytes; other arguments as moe_fwd.
 */
enum { MOE_AGG_GATHER_SUM = 0, MOE_AGG_SCATTER_SUM = 1, MOE_AGG_ATOMIC_F32 = 2 };
int moe_fwd_aggregation_ablation(moe_dims dims, const moe_bf16 *X, const moe_bf16 *W1, const moe_bf16 *W2,
                                 const moe_routing *r, moe_bf16 *H, moe_bf16 *O, int strategy, void *ws,
                                 size_t ws_bytes, void *stream);

/* Static description of an error code. */
const char *moe_strerror(int code);
/* Thread-local description of the last error returned on this thread. */
const char *moe_last_error(void);

/*
 * Kernel timing (measurement support).  moe_prof_select(k) brackets every
 * later launch of kernel class k with HIP events on the launch stream
 * (k = -1 disables); moe_prof_read() synchronises those events and returns the
 * summed milliseconds and the number of launches since the last reset.
 */
enum {
  MOE_KC_ROUTER_GEMM = 0, MOE_KC_TOPK, MOE_KC_META, MOE_KC_ROUND,
  MOE_KC_UP, MOE_KC_DOWN, MOE_KC_AGG_O,
  MOE_KC_DH, MOE_KC_DW2, MOE_KC_DXT, MOE_KC_DW1, MOE_KC_AGG_DX, MOE_KC_DWR,
  MOE_KC_ROUTER_TOPK, /* the router GEMM with fused softmax/top-K */
  MOE_KC_COUNT
};
int moe_prof_select(int kernel_class);
int moe_prof_read(double *ms, int32_t *launches);
const char *moe_kernel_class_name(int kernel_class);

#ifdef __cplusplus
}
#endif
#endif /* SONICMOE_H */
