// C ABI of the MoE layer: host-side validation, routing/workspace layout and
// the launch sequence of each entry point.  No entry point allocates device
// memory or synchronises the stream.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "launch.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int hip_fail(hipError_t e, const char* where) {
  return fail(MOE_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int check_dims(const moe_dims& m) {
  if (m.T < 1) return fail(MOE_ERR_INVALID_ARG, "T must be >= 1 (got %d)", m.T);
  if (m.d < 128 || m.d % 128) return fail(MOE_ERR_UNSUPPORTED, "d must be a positive multiple of 128 (got %d)", m.d);
  if (m.n < 64 || m.n % 64) return fail(MOE_ERR_UNSUPPORTED, "n must be a positive multiple of 64 (got %d)", m.n);
  if (m.E < 8 || m.E % 8 || m.E > 4096)
    return fail(MOE_ERR_UNSUPPORTED, "E must be a multiple of 8 in [8, 4096] (got %d)", m.E);
  if (m.K < 1 || m.K > 16 || m.K > m.E)
    return fail(MOE_ERR_UNSUPPORTED, "K must be in [1, min(E, 16)] (got K=%d, E=%d)", m.K, m.E);
  if ((int64_t)m.T * m.E > (int64_t)INT32_MAX)
    return fail(MOE_ERR_UNSUPPORTED, "T*E must fit in int32 (got %lld)", (long long)m.T * m.E);
  return MOE_OK;
}

#define CHECK_PTR(p, a)                                                                                   \
  do {                                                                                                    \
    if (!(p)) return fail(MOE_ERR_INVALID_ARG, "%s must not be null", #p);                                \
    if (!aligned((p), (a))) return fail(MOE_ERR_INVALID_ARG, "%s must be %d-byte aligned", #p, (int)(a)); \
  } while (0)

int check_routing(const moe_dims& m, const moe_routing* r, int64_t min_capacity, const char* name) {
  if (!r) return fail(MOE_ERR_INVALID_ARG, "%s must not be null", name);
  if (r->words != (m.T + 63) / 64)
    return fail(MOE_ERR_INVALID_ARG, "%s->words must be ceil(T/64) = %d (got %d)", name, (m.T + 63) / 64, r->words);
  if ((int64_t)r->capacity < min_capacity)
    return fail(MOE_ERR_CAPACITY, "%s->capacity %d < required %lld", name, r->capacity, (long long)min_capacity);
  const void* req[] = {r->scores, r->mask, r->mask_prefix, r->counts, r->offsets, r->row_token, r->row_expert,
                       r->row_w, r->tok_offsets, r->tok_rows, r->tok_count, r->tok_denom, r->round_dir, r->scratch,
                       r->status};
  for (const void* p : req)
    if (!p) return fail(MOE_ERR_INVALID_ARG, "%s has a null array (initialise it with moe_routing_init)", name);
  return MOE_OK;
}

// the consumers of a routing (moe_fwd, moe_bwd) need its complete metadata
int check_built(const moe_routing* r, const char* name) {
  if (r->state != MOE_ROUTING_STATE_BUILT)
    return fail(MOE_ERR_INVALID_ARG,
                "%s is not a complete routing (state %d; moe_route without MOE_ROUTE_COUNTS_ONLY or "
                "moe_round_tokens builds one)",
                name, r->state);
  return MOE_OK;
}

bool valid_m_tile(int m) { return m >= 8 && m <= 256 && (m & (m - 1)) == 0; }

// ---------------------------------------------------------------- static workspace
// The forward workspace of moe_fwd_static: a file-scope device array that
// each GPU holds from the library's load to the end of the process.  In host
// code `scratch` only names the host-side stand-in of the symbol; its device
// address comes from hipGetSymbolAddress, once per device, with that device
// current, and only that address is ever handed to a kernel.
constexpr size_t kStaticWsBytes = (size_t)64 << 20;
static __device__ __align__(256) char scratch[kStaticWsBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int static_ws(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(MOE_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(MOE_ERR_HIP, "hipGetSymbolAddress(scratch) returned null");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MOE_OK;
}

// ---------------------------------------------------------------- timing
std::mutex g_prof_mu;
int g_prof_class = -1;
std::vector<std::pair<hipEvent_t, hipEvent_t>> g_prof_events;  // recorded pairs
std::vector<std::pair<hipEvent_t, hipEvent_t>> g_prof_pool;     // free pairs

// ---------------------------------------------------------------- workspaces
struct FwdWs {
  uint16_t* A;
  uint16_t* Y;
  int32_t* mtiles;
};
struct BwdWs {
  int32_t* mtiles;
  uint16_t* dH;
  uint16_t* Ap;
  uint16_t* dXt;
  float* dS;
  float* dS_part;
  uint16_t* dL;
  uint16_t* WrT;
  float* dWr_part;
  float* dbias_part;
  int32_t* klist2;  // k-chunk lists of the weight gradients
  int32_t* klist1;
  float* dw_part;   // fp32 partials of row-chunked experts
  uint16_t* b2s;    // expert-bias dS term: b2^T as bf16 high/low parts [d][2E]
  float* bq;        // and <dO_t, b2_e> in those two parts [T][2E]
};

size_t carve(char* base, size_t off, size_t bytes, void** out) {
  if (out) *out = base ? base + off : nullptr;
  return align_up(off + bytes);
}

size_t fwd_layout(const moe_dims& m, int64_t cap, char* base, FwdWs* w) {
  size_t off = 0;
  off = carve(base, off, (size_t)cap * m.n * 2, w ? (void**)&w->A : nullptr);
  off = carve(base, off, (size_t)cap * m.d * 2, w ? (void**)&w->Y : nullptr);
  off = carve(base, off, smoe::mtiles_bytes(cap, m.E), w ? (void**)&w->mtiles : nullptr);
  return off;
}

// the aggregation ablation: the forward workspace, then the token-major slot
// of every row and an fp32 O
size_t abl_layout(const moe_dims& m, int64_t cap, char* base, FwdWs* w, int32_t** dst, float** O32) {
  size_t off = fwd_layout(m, cap, base, w);
  off = carve(base, off, (size_t)cap * 4, (void**)dst);
  off = carve(base, off, (size_t)m.T * m.d * 4, (void**)O32);
  return off;
}

size_t bwd_layout(const moe_dims& m, int64_t cap, char* base, BwdWs* w) {
  const int nnt = smoe::dh_n_tiles(m.n);
  const int splits = smoe::dwr_splits(m.T, m.d, m.E);
  size_t off = 0;
  off = carve(base, off, smoe::mtiles_bytes(cap, m.E), w ? (void**)&w->mtiles : nullptr);
  off = carve(base, off, (size_t)cap * 2 * m.n * 2, w ? (void**)&w->dH : nullptr);
  off = carve(base, off, (size_t)cap * m.n * 2, w ? (void**)&w->Ap : nullptr);
  off = carve(base, off, (size_t)cap * m.d * 2, w ? (void**)&w->dXt : nullptr);
  off = carve(base, off, (size_t)cap * 4, w ? (void**)&w->dS : nullptr);
  off = carve(base, off, nnt > 1 ? (size_t)cap * nnt * 4 : 0, w ? (void**)&w->dS_part : nullptr);
  off = carve(base, off, (size_t)m.T * m.E * 2, w ? (void**)&w->dL : nullptr);
  off = carve(base, off, (size_t)m.E * m.d * 2, w ? (void**)&w->WrT : nullptr);
  off = carve(base, off, (size_t)splits * m.d * m.E * 4, w ? (void**)&w->dWr_part : nullptr);
  off = carve(base, off, (size_t)smoe::colsum_chunks(m.T) * m.E * 4, w ? (void**)&w->dbias_part : nullptr);
  off = carve(base, off, smoe::kchunks_bytes(m.E), w ? (void**)&w->klist2 : nullptr);
  off = carve(base, off, smoe::kchunks_bytes(m.E), w ? (void**)&w->klist1 : nullptr);
  off = carve(base, off, smoe::dw_part_bytes(m.d, m.n), w ? (void**)&w->dw_part : nullptr);
  off = carve(base, off, (size_t)m.d * 2 * m.E * 2, w ? (void**)&w->b2s : nullptr);
  off = carve(base, off, (size_t)m.T * 2 * m.E * 4, w ? (void**)&w->bq : nullptr);
  return off;
}

// byte offset of the rounding selection's lists in the routing scratch
size_t round_lists_offset(const moe_dims& m) {
  const int W = (m.T + 63) / 64;
  return ((size_t)(m.E + 64 + 2 * (W + 1)) * 4 + 255) / 256 * 256;
}

size_t routing_layout(const moe_dims& m, int64_t cap, int flags, char* base, moe_routing* r) {
  const int W = (m.T + 63) / 64;
  const size_t TE = (size_t)m.T * m.E, EW = (size_t)m.E * W, TK = (size_t)m.T * m.K;
  moe_routing tmp;
  moe_routing* o = r ? r : &tmp;
  size_t off = 0;
  auto take = [&](size_t bytes, void** p) { off = carve(base, off, bytes, p); };
  void* p;
  take((flags & MOE_ROUTING_LOGITS) ? TE * 4 : 0, &p);
  o->logits = (flags & MOE_ROUTING_LOGITS) ? (float*)p : nullptr;
  take(TE * 4, &p);
  o->scores = (float*)p;
  take((flags & MOE_ROUTING_SCORES_T) ? TE * 4 : 0, &p);
  o->scores_t = (flags & MOE_ROUTING_SCORES_T) ? (float*)p : nullptr;
  take(TK * 4, &p);
  o->topk_idx = (int32_t*)p;
  take(TK * 4, &p);
  o->topk_w = (float*)p;
  take(EW * 8, &p);
  o->mask = (uint64_t*)p;
  take(EW * 4, &p);
  o->mask_prefix = (int32_t*)p;
  take((size_t)m.E * 4, &p);
  o->counts = (int32_t*)p;
  take((size_t)(m.E + 1) * 4, &p);
  o->offsets = (int32_t*)p;
  take((size_t)cap * 4, &p);
  o->row_token = (int32_t*)p;
  take((size_t)cap * 4, &p);
  o->row_expert = (int32_t*)p;
  take((size_t)cap * 4, &p);
  o->row_w = (float*)p;
  take((size_t)(m.T + 1) * 4, &p);
  o->tok_offsets = (int32_t*)p;
  take((size_t)cap * 4, &p);
  o->tok_rows = (int32_t*)p;
  take((size_t)m.T * 4, &p);
  o->tok_count = (int32_t*)p;
  take((size_t)m.T * 4, &p);
  o->tok_denom = (float*)p;
  take((size_t)m.E * 4, &p);
  o->round_dir = (int32_t*)p;
  // rounding needs [E], then per-word token sums and bases, then the
  // selection's lists
  take(round_lists_offset(m) + smoe::round_scratch_bytes(m.T, m.E), &p);
  o->scratch = (int32_t*)p;
  take(4, &p);
  o->status = (int32_t*)p;
  o->capacity = (int32_t)cap;
  o->words = W;
  o->state = MOE_ROUTING_STATE_EMPTY;
  o->reserved = 0;
  return off;
}

#define HIP_TRY(expr, where)                          \
  do {                                                \
    hipError_t _e = (expr);                           \
    if (_e != hipSuccess) return hip_fail(_e, where); \
  } while (0)

#define LAUNCH(kc, expr, where)          \
  do {                                   \
    smoe::prof_begin((kc), stream);      \
    hipError_t _e = (expr);              \
    smoe::prof_end((kc), stream);        \
    if (_e != hipSuccess) return hip_fail(_e, where); \
  } while (0)

}  // namespace

namespace smoe {

void prof_begin(int kc, hipStream_t s) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (kc != g_prof_class) return;
  std::pair<hipEvent_t, hipEvent_t> ev;
  if (!g_prof_pool.empty()) {
    ev = g_prof_pool.back();
    g_prof_pool.pop_back();
  } else {
    if (hipEventCreate(&ev.first) != hipSuccess || hipEventCreate(&ev.second) != hipSuccess) return;
  }
  (void)hipEventRecord(ev.first, s);
  g_prof_events.push_back(ev);
}

void prof_end(int kc, hipStream_t s) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (kc != g_prof_class || g_prof_events.empty()) return;
  (void)hipEventRecord(g_prof_events.back().second, s);
}

}  // namespace smoe

extern "C" {

const char* moe_strerror(int code) {
  switch (code) {
    case MOE_OK: return "success";
    case MOE_ERR_INVALID_ARG: return "invalid argument";
    case MOE_ERR_UNSUPPORTED: return "unsupported shape";
    case MOE_ERR_CAPACITY: return "routing capacity too small";
    case MOE_ERR_WORKSPACE: return "workspace too small";
    case MOE_ERR_HIP: return "HIP runtime error";
    default: return "unknown error";
  }
}

const char* moe_last_error(void) { return g_last_error.c_str(); }

size_t moe_routing_bytes(moe_dims dims, int32_t capacity, int flags) {
  if (check_dims(dims) != MOE_OK || capacity < 0) return 0;
  return routing_layout(dims, capacity, flags, nullptr, nullptr);
}

int moe_routing_init(moe_dims dims, int32_t capacity, int flags, void* buf, size_t bytes, moe_routing* r) {
  int rc = check_dims(dims);
  if (rc) return rc;
  if (!r) return fail(MOE_ERR_INVALID_ARG, "r must not be null");
  CHECK_PTR(buf, kAlign);
  if (capacity < dims.T * dims.K)
    return fail(MOE_ERR_CAPACITY, "capacity %d < T*K = %d", capacity, dims.T * dims.K);
  const size_t need = routing_layout(dims, capacity, flags, nullptr, nullptr);
  if (bytes < need) return fail(MOE_ERR_INVALID_ARG, "routing buffer of %zu bytes < required %zu", bytes, need);
  routing_layout(dims, capacity, flags, (char*)buf, r);
  return MOE_OK;
}

int32_t moe_round_capacity(moe_dims dims, int32_t m_tile) {
  if (check_dims(dims) != MOE_OK || !valid_m_tile(m_tile)) return -1;
  const int64_t a = (int64_t)dims.T * dims.E;
  const int64_t b = (int64_t)dims.T * dims.K + (int64_t)dims.E * (m_tile - 1);
  const int64_t c = a < b ? a : b;
  return c > INT32_MAX ? -1 : (int32_t)c;
}

size_t moe_workspace_bytes(moe_dims dims, int32_t capacity, int which) {
  if (check_dims(dims) != MOE_OK || capacity < 0) return 0;
  if (which == MOE_WS_FWD) return fwd_layout(dims, capacity, nullptr, nullptr);
  if (which == MOE_WS_BWD) return bwd_layout(dims, capacity, nullptr, nullptr);
  if (which == MOE_WS_FWD_AGG_ABLATION) {
    int32_t* dst;
    float* o32;
    return abl_layout(dims, capacity, nullptr, nullptr, &dst, &o32);
  }
  return 0;
}

int moe_route(moe_dims m, const moe_bf16* X, const moe_bf16* Wr, const float* bias, int flags, moe_routing* r,
              void* stream_) {
  int rc = check_dims(m);
  if (rc) return rc;
  rc = check_routing(m, r, (int64_t)m.T * m.K, "r");
  if (rc) return rc;
  if (!r->topk_idx || !r->topk_w) return fail(MOE_ERR_INVALID_ARG, "r->topk_idx and r->topk_w must not be null");
  const bool scores_in = flags & MOE_ROUTE_SCORES_IN;
  if (!scores_in) {
    CHECK_PTR(X, 16);
    CHECK_PTR(Wr, 16);
  }
  if (bias && !aligned(bias, 4)) return fail(MOE_ERR_INVALID_ARG, "bias must be 4-byte aligned");
  if ((flags & MOE_ROUTE_WRITE_LOGITS) && !r->logits)
    return fail(MOE_ERR_INVALID_ARG, "MOE_ROUTE_WRITE_LOGITS needs r->logits");
  if ((flags & MOE_ROUTE_WRITE_SCORES_T) && !r->scores_t)
    return fail(MOE_ERR_INVALID_ARG, "MOE_ROUTE_WRITE_SCORES_T needs r->scores_t");
  if (flags & ~(MOE_ROUTE_SCORES_IN | MOE_ROUTE_WRITE_LOGITS | MOE_ROUTE_WRITE_SCORES_T | MOE_ROUTE_COUNTS_ONLY |
                MOE_ROUTE_SEPARATE_TOPK))
    return fail(MOE_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
  hipStream_t stream = (hipStream_t)stream_;
  float* scores_t = (flags & MOE_ROUTE_WRITE_SCORES_T) ? r->scores_t : nullptr;
  const float* in = r->scores;
  if (!scores_in && !(flags & MOE_ROUTE_SEPARATE_TOPK) && smoe::router_topk_fusable(m.E, m.K)) {
    float* logits = (flags & MOE_ROUTE_WRITE_LOGITS) ? r->logits : nullptr;
    smoe::RouterTopkArgs a{X, Wr, bias, logits, r->scores, scores_t, r->topk_idx, r->topk_w, r->mask,
                           m.T, m.d, m.E, m.K, r->words};
    LAUNCH(MOE_KC_ROUTER_TOPK, smoe::launch_router_topk(a, stream), "router gemm with softmax/top-K");
  } else {
    if (!scores_in) {
      float* logits = (flags & MOE_ROUTE_WRITE_LOGITS) ? r->logits : r->scores;
      smoe::RouterGemmArgs a{X, Wr, bias, logits, m.T, m.d, m.E};
      LAUNCH(MOE_KC_ROUTER_GEMM, smoe::launch_router_gemm(a, stream), "router gemm");
      in = logits;
    }
    LAUNCH(MOE_KC_TOPK,
           smoe::launch_topk_route(in, r->scores, scores_t, r->topk_idx, r->topk_w, r->mask, m.T, m.E, m.K,
                                   r->words, scores_in ? 0 : 1, stream),
           "softmax/top-K");
  }
  const bool counts_only = (flags & MOE_ROUTE_COUNTS_ONLY) != 0;
  r->state = MOE_ROUTING_STATE_EMPTY;  // until the metadata launch is enqueued
  LAUNCH(MOE_KC_META, smoe::launch_tc_metadata(*r, m.T, m.E, m.K, counts_only, stream), "routing metadata");
  r->state = counts_only ? MOE_ROUTING_STATE_COUNTS : MOE_ROUTING_STATE_BUILT;
  return MOE_OK;
}

int moe_round_tokens(moe_dims m, int32_t m_tile, int mode, const float* u, const moe_routing* tc, moe_routing* tr,
                     void* stream_) {
  int rc = check_dims(m);
  if (rc) return rc;
  if (!valid_m_tile(m_tile))
    return fail(MOE_ERR_INVALID_ARG, "m_tile must be a power of two in [8, 256] (got %d)", m_tile);
  if (mode < MOE_ROUND_NEAREST || mode > MOE_ROUND_STOCHASTIC)
    return fail(MOE_ERR_INVALID_ARG, "unknown rounding mode %d", mode);
  if (mode == MOE_ROUND_STOCHASTIC) CHECK_PTR(u, 4);
  rc = check_routing(m, tc, (int64_t)m.T * m.K, "tc");
  if (rc) return rc;
  if (!tc->scores_t) return fail(MOE_ERR_INVALID_ARG, "tc->scores_t must be written (MOE_ROUTE_WRITE_SCORES_T)");
  if (tc->state < MOE_ROUTING_STATE_COUNTS)
    return fail(MOE_ERR_INVALID_ARG, "tc has no counts yet (state %d): run moe_route on it first", tc->state);
  rc = check_routing(m, tr, moe_round_capacity(m, m_tile), "tr");
  if (rc) return rc;
  if (tr == tc || tr->mask == tc->mask) return fail(MOE_ERR_INVALID_ARG, "tr must not alias tc");
  hipStream_t stream = (hipStream_t)stream_;
  tr->state = MOE_ROUTING_STATE_EMPTY;
  smoe::prof_begin(MOE_KC_ROUND, stream);
  bool counted = false;
  uint64_t* list = (uint64_t*)((char*)tr->scratch + round_lists_offset(m));
  hipError_t e = smoe::launch_round(*tc, *tr, u, m.T, m.E, m_tile, mode, list, &counted, stream);
  if (e == hipSuccess) e = smoe::launch_metadata(*tr, tc->scores_t, m.T, m.E, counted, stream);
  smoe::prof_end(MOE_KC_ROUND, stream);
  if (e != hipSuccess) return hip_fail(e, "token rounding");
  tr->state = MOE_ROUTING_STATE_BUILT;
  return MOE_OK;
}

int check_expert_bias(const moe_expert_bias* eb) {
  if (!eb) return MOE_OK;
  const void* p[] = {eb->b1, eb->b2, eb->db1, eb->db2};
  const char* name[] = {"eb->b1", "eb->b2", "eb->db1", "eb->db2"};
  for (int i = 0; i < 4; ++i)
    if (p[i] && !aligned(p[i], 16)) return fail(MOE_ERR_INVALID_ARG, "%s must be 16-byte aligned", name[i]);
  return MOE_OK;
}

int moe_fwd(moe_dims m, const moe_bf16* X, const moe_bf16* W1, const moe_bf16* W2, const moe_expert_bias* eb,
            const moe_routing* r, moe_bf16* H, moe_bf16* O, void* ws, size_t ws_bytes, void* stream_) {
  int rc = check_dims(m);
  if (rc) return rc;
  rc = check_routing(m, r, 1, "r");
  if (rc) return rc;
  rc = check_built(r, "r");
  if (rc) return rc;
  CHECK_PTR(X, 16);
  CHECK_PTR(W1, 16);
  CHECK_PTR(W2, 16);
  CHECK_PTR(H, 16);
  CHECK_PTR(O, 16);
  rc = check_expert_bias(eb);
  if (rc) return rc;
  const float* b1 = eb ? eb->b1 : nullptr;
  const float* b2 = eb ? eb->b2 : nullptr;
  const size_t need = fwd_layout(m, r->capacity, nullptr, nullptr);
  if (ws_bytes < need) return fail(MOE_ERR_WORKSPACE, "forward workspace %zu < required %zu", ws_bytes, need);
  CHECK_PTR(ws, kAlign);
  FwdWs w;
  fwd_layout(m, r->capacity, (char*)ws, &w);
  hipStream_t stream = (hipStream_t)stream_;
  HIP_TRY(smoe::launch_mtiles(r->offsets, m.E, w.mtiles, stream), "m-tile list");
  LAUNCH(MOE_KC_UP,
         smoe::launch_up({X, W1, r->offsets, r->row_token, H, w.A, m.d, m.n, m.E, r->capacity, w.mtiles, b1}, stream),
         "up-proj");
  LAUNCH(MOE_KC_DOWN, smoe::launch_down({w.A, W2, r->offsets, w.Y, m.d, m.n, m.E, r->capacity, w.mtiles, b2}, stream),
         "down-proj");
  LAUNCH(MOE_KC_AGG_O, smoe::launch_agg_o(w.Y, *r, O, m.T, m.d, stream), "aggregation");
  return MOE_OK;
}

size_t moe_fwd_static_max_bytes(void) { return kStaticWsBytes; }

int moe_fwd_static(moe_dims m, const moe_bf16* X, const moe_bf16* W1, const moe_bf16* W2, const moe_expert_bias* eb,
                   const moe_routing* r, moe_bf16* H, moe_bf16* O, void* stream) {
  int rc = check_dims(m);
  if (rc) return rc;
  rc = check_routing(m, r, 1, "r");
  if (rc) return rc;
  const size_t need = fwd_layout(m, r->capacity, nullptr, nullptr);
  if (need > kStaticWsBytes)
    return fail(MOE_ERR_WORKSPACE,
                "the forward workspace for capacity %d (%zu bytes) exceeds the static workspace of %zu bytes; "
                "use moe_fwd with a caller workspace",
                r->capacity, need, kStaticWsBytes);
  void* ws = nullptr;
  rc = static_ws(&ws);
  if (rc) return rc;
  return moe_fwd(m, X, W1, W2, eb, r, H, O, ws, kStaticWsBytes, stream);
}

int moe_fwd_aggregation_ablation(moe_dims m, const moe_bf16* X, const moe_bf16* W1, const moe_bf16* W2,
                                 const moe_routing* r, moe_bf16* H, moe_bf16* O, int strategy, void* ws,
                                 size_t ws_bytes, void* stream_) {
  int rc = check_dims(m);
  if (rc) return rc;
  rc = check_routing(m, r, 1, "r");
  if (rc) return rc;
  rc = check_built(r, "r");
  if (rc) return rc;
  CHECK_PTR(X, 16);
  CHECK_PTR(W1, 16);
  CHECK_PTR(W2, 16);
  CHECK_PTR(H, 16);
  CHECK_PTR(O, 16);
  if (strategy < MOE_AGG_GATHER_SUM || strategy > MOE_AGG_ATOMIC_F32)
    return fail(MOE_ERR_INVALID_ARG, "unknown aggregation strategy %d", strategy);
  int32_t* dst = nullptr;
  float* o32 = nullptr;
  const size_t need = abl_layout(m, r->capacity, nullptr, nullptr, &dst, &o32);
  if (ws_bytes < need) return fail(MOE_ERR_WORKSPACE, "ablation workspace %zu < required %zu", ws_bytes, need);
  CHECK_PTR(ws, kAlign);
  FwdWs w;
  abl_layout(m, r->capacity, (char*)ws, &w, &dst, &o32);
  hipStream_t stream = (hipStream_t)stream_;
  HIP_TRY(smoe::launch_mtiles(r->offsets, m.E, w.mtiles, stream), "m-tile list");
  LAUNCH(MOE_KC_UP,
         smoe::launch_up({X, W1, r->offsets, r->row_token, H, w.A, m.d, m.n, m.E, r->capacity, w.mtiles, nullptr},
                         stream),
         "up-proj");
  smoe::DownArgs da{w.A, W2, r->offsets, w.Y, m.d, m.n, m.E, r->capacity, w.mtiles, nullptr};
  if (strategy == MOE_AGG_GATHER_SUM) {
    LAUNCH(MOE_KC_DOWN, smoe::launch_down(da, stream), "down-proj");
    LAUNCH(MOE_KC_AGG_O, smoe::launch_agg_o(w.Y, *r, O, m.T, m.d, stream), "aggregation");
  } else if (strategy == MOE_AGG_SCATTER_SUM) {
    da.dst = dst;
    LAUNCH(MOE_KC_DOWN,
           [&]() {
             hipError_t e = smoe::launch_tok_slots(*r, m.T, r->capacity, dst, stream);
             return e == hipSuccess ? smoe::launch_down_ablation(da, 1, stream) : e;
           }(),
           "down-proj (scatter)");
    LAUNCH(MOE_KC_AGG_O, smoe::launch_agg_o_contig(w.Y, *r, O, m.T, m.d, stream), "contiguous sum");
  } else {
    da.O32 = o32;
    da.row_token = r->row_token;
    da.row_w = r->row_w;
    const size_t td = (size_t)m.T * m.d;
    LAUNCH(MOE_KC_DOWN,
           [&]() {
             hipError_t e = smoe::launch_fill_f32(o32, td, stream);
             return e == hipSuccess ? smoe::launch_down_ablation(da, 2, stream) : e;
           }(),
           "down-proj (fp32 atomics)");
    LAUNCH(MOE_KC_AGG_O, smoe::launch_f32_to_bf16(o32, O, td, stream), "fp32 -> bf16");
  }
  return MOE_OK;
}

int moe_bwd(moe_dims m, const moe_bf16* dO, const moe_bf16* X, const moe_bf16* H, const moe_bf16* W1,
            const moe_bf16* W2, const moe_expert_bias* eb, const moe_bf16* Wr, const moe_routing* r, moe_bf16* dX, moe_bf16* dW1, moe_bf16* dW2,
            float* dWr, float* dbias, float* dS, void* ws, size_t ws_bytes, void* stream_) {
  int rc = check_dims(m);
  if (rc) return rc;
  rc = check_routing(m, r, 1, "r");
  if (rc) return rc;
  rc = check_built(r, "r");
  if (rc) return rc;
  CHECK_PTR(dO, 16);
  CHECK_PTR(X, 16);
  CHECK_PTR(H, 16);
  CHECK_PTR(W1, 16);
  CHECK_PTR(W2, 16);
  CHECK_PTR(dX, 16);
  CHECK_PTR(dW1, 16);
  CHECK_PTR(dW2, 16);
  if (Wr && !aligned(Wr, 16)) return fail(MOE_ERR_INVALID_ARG, "Wr must be 16-byte aligned");
  if (!Wr && (dWr || dbias)) return fail(MOE_ERR_INVALID_ARG, "dWr/dbias need Wr");
  if (dWr && !aligned(dWr, 16)) return fail(MOE_ERR_INVALID_ARG, "dWr must be 16-byte aligned");
  if (dbias && !aligned(dbias, 4)) return fail(MOE_ERR_INVALID_ARG, "dbias must be 4-byte aligned");
  if (dS && !aligned(dS, 4)) return fail(MOE_ERR_INVALID_ARG, "dS must be 4-byte aligned");
  rc = check_expert_bias(eb);
  if (rc) return rc;
  const float* b2 = eb ? eb->b2 : nullptr;
  const size_t need = bwd_layout(m, r->capacity, nullptr, nullptr);
  if (ws_bytes < need) return fail(MOE_ERR_WORKSPACE, "backward workspace %zu < required %zu", ws_bytes, need);
  CHECK_PTR(ws, kAlign);
  BwdWs w;
  bwd_layout(m, r->capacity, (char*)ws, &w);
  hipStream_t stream = (hipStream_t)stream_;
  float* dS_out = dS ? dS : w.dS;
  const int nnt = smoe::dh_n_tiles(m.n);
  HIP_TRY(smoe::launch_bwd_lists(r->offsets, m.E, m.d, m.n, w.mtiles, w.klist2, w.klist1, Wr, Wr ? w.WrT : nullptr,
                                 stream),
          "tile lists and W_r transpose");
  if (b2) {
    // <dO_t, b2_e> for every (t, e): dO times b2^T split into bf16 high and low parts
    HIP_TRY(smoe::launch_bias_split(b2, m.E, m.d, w.b2s, stream), "expert-bias split");
    HIP_TRY(smoe::launch_router_gemm({dO, w.b2s, nullptr, w.bq, m.T, m.d, 2 * m.E}, stream), "expert-bias dS term");
  }
  LAUNCH(MOE_KC_DH,
         smoe::launch_dh({dO, W2, H, r->offsets, r->row_token, r->row_w, w.dH, w.Ap, dS_out, w.dS_part, m.d, m.n, m.E,
                          r->capacity, w.mtiles, b2 ? w.bq : nullptr},
                         stream),
         "dH");
  if (nnt > 1) HIP_TRY(smoe::launch_reduce_rowparts(w.dS_part, dS_out, r->capacity, nnt, stream), "dS reduce");
  LAUNCH(MOE_KC_DW2, smoe::launch_dw2({w.Ap, dO, r->offsets, r->row_token, dW2, m.d, m.n, m.E, w.klist2, w.dw_part}, stream), "dW2");
  LAUNCH(MOE_KC_DXT, smoe::launch_dxt({w.dH, W1, r->offsets, w.dXt, m.d, m.n, m.E, r->capacity, w.mtiles}, stream),
         "dX~");
  LAUNCH(MOE_KC_DW1, smoe::launch_dw1({X, w.dH, r->offsets, r->row_token, dW1, m.d, m.n, m.E, w.klist1, w.dw_part}, stream), "dW1");
  LAUNCH(MOE_KC_AGG_DX,
         smoe::launch_agg_dx(w.dXt, dS_out, Wr ? w.WrT : nullptr, *r, dX, Wr ? w.dL : nullptr, m.T, m.d, m.E, stream),
         "dX aggregation");
  const int splits = smoe::dwr_splits(m.T, m.d, m.E);
  if (dWr) LAUNCH(MOE_KC_DWR, smoe::launch_dwr({X, w.dL, w.dWr_part, dWr, m.T, m.d, m.E, splits}, stream), "dW_r");
  if (dbias) HIP_TRY(smoe::launch_colsum_rows(w.dL, w.dbias_part, m.T, m.E, stream), "dbias");
  HIP_TRY(smoe::launch_bwd_final_reduce(w.klist1, w.dw_part, dW1, m.d, m.n, w.dWr_part, dWr, splits, w.dbias_part,
                                        dbias, m.T, m.E, stream),
          "final reductions (dW1 split experts, dW_r, dbias)");
  if (eb && eb->db1)
    HIP_TRY(smoe::launch_expert_colsum(w.dH, 2 * m.n, 2 * m.n, r->offsets, nullptr, nullptr, m.E, eb->db1, stream),
            "expert-bias gradient db1");
  if (eb && eb->db2)
    HIP_TRY(smoe::launch_expert_colsum(dO, m.d, m.d, r->offsets, r->row_token, r->row_w, m.E, eb->db2, stream),
            "expert-bias gradient db2");
  return MOE_OK;
}

int moe_prof_select(int kc) {
  if (kc < -1 || kc >= MOE_KC_COUNT) return fail(MOE_ERR_INVALID_ARG, "unknown kernel class %d", kc);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_class = kc;
  return MOE_OK;
}

int moe_prof_read(double* ms, int32_t* launches) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  double total = 0.0;
  int32_t count = 0;
  for (auto& ev : g_prof_events) {
    hipError_t e = hipEventSynchronize(ev.second);
    if (e != hipSuccess) return hip_fail(e, "prof event");
    float t = 0.f;
    e = hipEventElapsedTime(&t, ev.first, ev.second);
    if (e != hipSuccess) return hip_fail(e, "prof elapsed");
    total += t;
    ++count;
    g_prof_pool.push_back(ev);
  }
  g_prof_events.clear();
  if (ms) *ms = total;
  if (launches) *launches = count;
  return MOE_OK;
}

const char* moe_kernel_class_name(int kc) {
  static const char* names[MOE_KC_COUNT] = {"router_gemm", "topk", "routing_meta", "token_round", "up_proj",
                                            "down_proj", "aggregate_O", "dH", "dW2", "dXtilde",
                                            "dW1", "aggregate_dX", "dWr", "router_topk"};
  return (kc >= 0 && kc < MOE_KC_COUNT) ? names[kc] : "unknown";
}

}  // extern "C"
