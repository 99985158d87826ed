// Host side of libeta: argument validation, split planning, workspace
// carve-up, optional kernel timing, and the extern "C" entry points declared
// in include/eta.h.  Every entry point validates all arguments before it
// enqueues anything, and never throws across the ABI.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "eta.h"
#include "eta_internal.h"

namespace eta {
namespace {

thread_local std::string g_err;

eta_status_t fail(eta_status_t code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

eta_status_t ok() {
  g_err.clear();
  return ETA_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int elem_bytes(int dt) { return dt == ETA_DT_F32 ? 4 : 2; }

bool valid_dtype(int dt) { return dt == ETA_DT_F32 || dt == ETA_DT_BF16; }

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Geometry checks shared by every entry point that takes an eta_kv_desc_t.
eta_status_t check_kv(const eta_kv_desc_t* kv, Geom* g) {
  if (kv == nullptr) return fail(ETA_ERR_INVALID_ARG, "kv descriptor is NULL");
  if (kv->batch < 1) return fail(ETA_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", kv->batch);
  if (kv->num_q_heads < 1 || kv->num_kv_heads < 1)
    return fail(ETA_ERR_INVALID_ARG, "head counts must be >= 1 (q %d, kv %d)", kv->num_q_heads,
                kv->num_kv_heads);
  if (kv->num_q_heads % kv->num_kv_heads != 0)
    return fail(ETA_ERR_INVALID_ARG, "num_q_heads (%d) is not a multiple of num_kv_heads (%d)",
                kv->num_q_heads, kv->num_kv_heads);
  if (kv->head_dim < 1 || kv->block_size < 1)
    return fail(ETA_ERR_INVALID_ARG, "head_dim and block_size must be >= 1");
  if (kv->capacity_tokens < 1)
    return fail(ETA_ERR_INVALID_ARG, "capacity_tokens must be >= 1 (got %lld)",
                (long long)kv->capacity_tokens);
  if (!valid_dtype(kv->kv_dtype)) return fail(ETA_ERR_INVALID_ARG, "kv_dtype %d is not an eta_dtype_t", kv->kv_dtype);
  const int G = kv->num_q_heads / kv->num_kv_heads;
  if (kv->head_dim != 64 && kv->head_dim != 128)
    return fail(ETA_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", kv->head_dim);
  if (kv->block_size != 64 && kv->block_size != 128)
    return fail(ETA_ERR_UNSUPPORTED, "block_size %d unsupported (64 or 128)", kv->block_size);
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(ETA_ERR_UNSUPPORTED, "GQA group size %d unsupported (1, 2, 4 or 8)", G);
  if (kv->num_q_heads > 256) return fail(ETA_ERR_UNSUPPORTED, "num_q_heads > 256 unsupported");
  const int64_t eb = elem_bytes(kv->kv_dtype);
  if (kv->stride_t < kv->head_dim)
    return fail(ETA_ERR_INVALID_ARG, "stride_t (%lld) < head_dim (%d)", (long long)kv->stride_t,
                kv->head_dim);
  if (kv->stride_h < 0 || kv->stride_b < 0)
    return fail(ETA_ERR_INVALID_ARG, "negative stride");
  if ((kv->stride_t * eb) % 16 || (kv->stride_h * eb) % 16 || (kv->stride_b * eb) % 16)
    return fail(ETA_ERR_INVALID_ARG, "K/V strides must keep token rows 16-byte aligned");
  g->B = kv->batch;
  g->Hq = kv->num_q_heads;
  g->Hkv = kv->num_kv_heads;
  g->D = kv->head_dim;
  g->BS = kv->block_size;
  g->G = G;
  g->kv_dtype = kv->kv_dtype;
  g->stat_dtype = ETA_DT_F32;
  g->cap = kv->capacity_tokens;
  g->sb = kv->stride_b;
  g->sh = kv->stride_h;
  g->st = kv->stride_t;
  g->ncap = kv->capacity_tokens / kv->block_size;
  g->n_tiles = (int)((g->ncap + kScreenTile - 1) / kScreenTile);
  if (g->n_tiles < 1) g->n_tiles = 1;
  return ETA_OK;
}

// The block capacity of the summary a call reads: the stride of the summary and
// mask arrays, and what the decode workspace is laid out for (its id lists and
// tile counts), so the workspace query and the decode take it from here alike.
eta_status_t set_blk_cap(int64_t n_blk_cap, Geom* g) {
  if (n_blk_cap < 1) return fail(ETA_ERR_INVALID_ARG, "n_blk_cap must be >= 1 (got %lld)", (long long)n_blk_cap);
  if (n_blk_cap < g->cap / g->BS)
    return fail(ETA_ERR_INVALID_ARG, "n_blk_cap (%lld) < capacity_tokens / block_size (%lld)",
                (long long)n_blk_cap, (long long)(g->cap / g->BS));
  g->ncap = n_blk_cap;
  g->n_tiles = (int)((g->ncap + kScreenTile - 1) / kScreenTile);
  if (g->n_tiles < 1) g->n_tiles = 1;
  if (g->n_tiles > kMaxTiles || n_blk_cap >= kMaxBlocks)
    return fail(ETA_ERR_UNSUPPORTED, "n_blk_cap %lld exceeds %d screening tiles of %d blocks",
                (long long)n_blk_cap, kMaxTiles, kScreenTile);
  return ETA_OK;
}

eta_status_t check_summary(const eta_summary_t* s, Geom* g) {
  if (s == nullptr) return fail(ETA_ERR_INVALID_ARG, "summary descriptor is NULL");
  if (!s->mu || !s->sigma || !s->max_norm)
    return fail(ETA_ERR_INVALID_ARG, "summary buffers must be non-NULL");
  if (!aligned16(s->mu) || !aligned16(s->sigma) || !aligned16(s->max_norm))
    return fail(ETA_ERR_INVALID_ARG, "summary buffers must be 16-byte aligned");
  if (s->stat_dtype != ETA_DT_F32 && s->stat_dtype != ETA_DT_F16 && s->stat_dtype != ETA_DT_FP8)
    return fail(ETA_ERR_INVALID_ARG,
                "stat_dtype %d: summaries are ETA_DT_F32, ETA_DT_F16 or ETA_DT_FP8", s->stat_dtype);
  g->stat_dtype = s->stat_dtype;
  return set_blk_cap(s->n_blk_cap, g);
}

eta_status_t check_params(const eta_decode_params_t* p) {
  if (p == nullptr) return fail(ETA_ERR_INVALID_ARG, "params is NULL");
  if (!std::isfinite(p->beta) || p->beta < 0.f)
    return fail(ETA_ERR_INVALID_ARG, "beta must be finite and >= 0");
  if (!std::isfinite(p->z) || p->z < 0.f) return fail(ETA_ERR_INVALID_ARG, "z must be finite and >= 0");
  if (!std::isfinite(p->offset_a)) return fail(ETA_ERR_INVALID_ARG, "offset_a must be finite");
  if (p->rescue_window_blocks < 0) return fail(ETA_ERR_INVALID_ARG, "rescue_window_blocks < 0");
  if (p->rescue_window_blocks > kMaxRescueWindow)
    return fail(ETA_ERR_UNSUPPORTED, "rescue_window_blocks > %d unsupported", kMaxRescueWindow);
  if (p->pin_recent_blocks < 0) return fail(ETA_ERR_INVALID_ARG, "pin_recent_blocks < 0");
  if (p->num_splits < 0 || p->num_splits > kMaxSplits)
    return fail(ETA_ERR_INVALID_ARG, "num_splits must be in [0, %d]", kMaxSplits);
  return ETA_OK;
}

// ------------------------------------------------------------- kernel timer

struct Profiler {
  std::mutex mu;
  bool on = false;
  std::vector<hipEvent_t> pool;       // pairs: [2i] start, [2i+1] end
  std::vector<int> kinds;
  size_t used = 0;
  static constexpr size_t kMaxPairs = 65536;
};
Profiler& prof() {
  static Profiler p;
  return p;
}

void hook_fn(int kind, hipStream_t st, bool after) {
  Profiler& P = prof();
  std::lock_guard<std::mutex> lk(P.mu);
  if (!P.on) return;
  if (!after) {
    if (P.used >= Profiler::kMaxPairs) return;
    if (2 * P.used + 2 > P.pool.size()) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess) return;
      if (hipEventCreate(&b) != hipSuccess) { (void)hipEventDestroy(a); return; }
      P.pool.push_back(a);
      P.pool.push_back(b);
    }
    (void)hipEventRecord(P.pool[2 * P.used], st);
    P.kinds.push_back(kind);
  } else {
    if (P.kinds.size() != P.used + 1) return;
    (void)hipEventRecord(P.pool[2 * P.used + 1], st);
    ++P.used;
  }
}

LaunchHook active_hook() {
  Profiler& P = prof();
  std::lock_guard<std::mutex> lk(P.mu);
  return P.on ? hook_fn : nullptr;
}

}  // namespace

int default_splits(const Geom& g) {
  // One sequence: one workgroup per compute unit (256 in all) -- a split
  // streams as fast with four wavefronts per compute unit as with eight, and
  // fewer splits mean fewer partials for the combine.  Several sequences:
  // about 4096 workgroups, i.e. several rounds that the dispatcher balances
  // over ragged lengths and unions (32 ragged 16K-64K sequences: 5-13% faster
  // than one round of 512, within 1-2% of 24 or 32 splits per kv head), but no
  // split covering less than 32 blocks of capacity: a sparse union would leave
  // such splits a few tiles each behind their prologue (8 x 128K at 18.6%
  // union: 116.5 us per step at 64 splits vs 131.8 at 128).
  const int64_t groups = (int64_t)g.B * g.Hkv;
  const int64_t target = g.B == 1 ? 256 : 4096;
  int64_t S = (target + groups - 1) / groups;
  if (S > 256) S = 256;
  const int64_t floor_cap = g.B == 1 ? g.ncap / 2 : g.ncap / 32;
  const int64_t cap = floor_cap > 0 ? floor_cap : 1;
  if (S > cap) S = cap;
  if (S < 1) S = 1;
  return (int)S;
}

// Split layout of a decode call.  One sequence (or a tile count table too large
// for the split kernel's LDS): S splits per kv head, num_splits or the default
// (one workgroup per compute unit for one sequence).  Several sequences: W =
// num_splits x B x Hkv workgroups (num_splits 0: see below) dealt to the
// (sequence, kv head) groups in proportion to their unions, so ragged lengths
// and unequal unions finish together; num_splits is then the average per group
// (8 x 128K at 18.6% union: 106 us per step at 512 in all against 143 with 64
// uniform splits per group; 32 ragged 16K-64K sequences: 849 us at 2048 in all,
// 1139 at 512).
constexpr int kPropSplits = 512;
constexpr int kPropMaxSplits = 4096;

SplitPlan plan_splits(const Geom& g, int num_splits) {
  const int64_t BG = (int64_t)g.B * g.Hkv;
  if (g.B > 1 && BG <= kPropMaxGroups && BG * g.n_tiles <= kPropMaxCounts) {
    // default: at least 8 per group on average (coarser shares leave some groups
    // with one workgroup for up to twice the average work), at least 512 in all
    // (2 per compute unit), at most 4096
    int64_t W = 8 * BG;
    W = W < kPropSplits ? kPropSplits : (W > kPropMaxSplits ? kPropMaxSplits : W);
    if (W < BG) W = BG;
    if (num_splits > 0) W = num_splits * BG;
    return SplitPlan{0, (int)W};
  }
  const int S = num_splits > 0 ? num_splits : default_splits(g);
  return SplitPlan{S, (int)(S * BG)};
}

size_t decode_ws_bytes(const Geom& g, const SplitPlan& sp, DecodeWs* c, void* base) {
  const size_t nb = (size_t)g.B * g.Hkv * g.ncap;
  const size_t BG = (size_t)g.B * g.Hkv, BH = (size_t)g.B * g.Hq;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  const size_t o_ids = take(nb * 4);
  const size_t o_tc = take(BG * g.n_tiles * 4);
  const size_t o_hc = take(BH * g.n_tiles * 4);
  const size_t o_ml = take((size_t)sp.W * g.G * 8);
  const size_t o_acc = take((size_t)sp.W * g.G * g.D * 4);
  const size_t o_tau = take(BH * 4);
  const size_t o_rb = take(BH * kRescueTiles * 4);
  const size_t o_ri = take(BH * kRescueTiles * 4);
  const size_t o_wb = take(BG * kMaxRescueWindow);
  const size_t o_ro = take(BH * 4);
  const size_t o_xu = take(BG * 4);
  const size_t o_pl = take(BG * 8);
  if (c && base) {
    char* p = static_cast<char*>(base);
    c->tau = reinterpret_cast<float*>(p + o_tau);
    c->ids = reinterpret_cast<int32_t*>(p + o_ids);
    c->tile_cnt = reinterpret_cast<int32_t*>(p + o_tc);
    c->head_cnt = reinterpret_cast<int32_t*>(p + o_hc);
    c->part_ml = reinterpret_cast<float2*>(p + o_ml);
    c->part_acc = reinterpret_cast<float*>(p + o_acc);
    c->resc_best = reinterpret_cast<float*>(p + o_rb);
    c->resc_info = reinterpret_cast<int32_t*>(p + o_ri);
    c->wbits = reinterpret_cast<uint8_t*>(p + o_wb);
    c->resc_out = reinterpret_cast<int32_t*>(p + o_ro);
    c->extra_union = reinterpret_cast<int32_t*>(p + o_xu);
    c->plan = reinterpret_cast<int2*>(p + o_pl);
  }
  return off;
}

size_t dense_ws_bytes(const Geom& g, int S, DecodeWs* c, void* base) {
  size_t off = 0;
  const size_t o_ml = off;
  off = align256(off + (size_t)g.B * g.Hq * S * 8);
  const size_t o_acc = off;
  off = align256(off + (size_t)g.B * g.Hq * S * g.D * 4);
  if (c && base) {
    char* p = static_cast<char*>(base);
    *c = DecodeWs{};
    c->part_ml = reinterpret_cast<float2*>(p + o_ml);
    c->part_acc = reinterpret_cast<float*>(p + o_acc);
  }
  return off;
}

}  // namespace eta

using namespace eta;

static_assert(kScratchBytes == ETA_DECODE_NOALLOC_SCRATCH_BYTES,
              "the header states the library scratch size");

extern "C" {

const char* eta_last_error_string(void) { return g_err.c_str(); }

int32_t eta_abi_version(void) { return 5; }

static eta_status_t summaries_impl(const eta_kv_desc_t* kv, const void* k,
                                   const int32_t* prev_lens, const int32_t* seq_lens,
                                   int32_t max_new_blocks, int32_t sub_block,
                                   const eta_summary_t* out, void* stream) {
  Geom g;
  eta_status_t st = check_kv(kv, &g);
  if (st) return st;
  if (!k || !seq_lens) return fail(ETA_ERR_INVALID_ARG, "k and seq_lens must be non-NULL");
  if (!aligned16(k) || !aligned16(seq_lens) || (prev_lens && !aligned16(prev_lens)))
    return fail(ETA_ERR_INVALID_ARG, "k / seq_lens / prev_lens must be 16-byte aligned");
  if (sub_block < 0 || sub_block > g.BS || (sub_block & (sub_block - 1)) != 0)
    return fail(ETA_ERR_INVALID_ARG, "sub_block must be 0 or a power of two in [1, block_size = %d]", g.BS);
  if ((st = check_summary(out, &g))) return st;
  hipError_t e = launch_summaries(g, k, seq_lens, prev_lens, max_new_blocks, sub_block, *out,
                                  (hipStream_t)stream, active_hook());
  if (e != hipSuccess) return fail(ETA_ERR_HIP, "summaries launch failed: %s", hipGetErrorString(e));
  return ok();
}

eta_status_t eta_build_block_summaries(const eta_kv_desc_t* kv, const void* k,
                                       const int32_t* seq_lens, const eta_summary_t* out,
                                       void* stream) {
  return summaries_impl(kv, k, nullptr, seq_lens, 0, 0, out, stream);
}

eta_status_t eta_build_block_summaries_envelope(const eta_kv_desc_t* kv, const void* k,
                                                const int32_t* seq_lens, int32_t sub_block,
                                                const eta_summary_t* out, void* stream) {
  return summaries_impl(kv, k, nullptr, seq_lens, 0, sub_block, out, stream);
}

eta_status_t eta_update_block_summaries(const eta_kv_desc_t* kv, const void* k,
                                        const int32_t* prev_lens, const int32_t* seq_lens,
                                        int32_t max_new_blocks, int32_t sub_block,
                                        const eta_summary_t* out, void* stream) {
  if (!prev_lens) return fail(ETA_ERR_INVALID_ARG, "prev_lens must be non-NULL");
  if (max_new_blocks < 0) return fail(ETA_ERR_INVALID_ARG, "max_new_blocks must be >= 0");
  if (kv && kv->block_size > 0 && max_new_blocks > kv->capacity_tokens / kv->block_size)
    max_new_blocks = (int32_t)(kv->capacity_tokens / kv->block_size);
  return summaries_impl(kv, k, prev_lens, seq_lens, max_new_blocks, sub_block, out, stream);
}

eta_status_t eta_predict_threshold(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                                   int32_t q_dtype, const void* q, const float* W,
                                   const float* bias, float* tau_out, void* stream) {
  if (batch < 1 || num_q_heads < 1 || head_dim < 1)
    return fail(ETA_ERR_INVALID_ARG, "batch, num_q_heads and head_dim must be >= 1");
  if (num_q_heads > 256) return fail(ETA_ERR_UNSUPPORTED, "num_q_heads > 256 unsupported");
  if (head_dim > 1024) return fail(ETA_ERR_UNSUPPORTED, "head_dim > 1024 unsupported");
  if (!valid_dtype(q_dtype)) return fail(ETA_ERR_INVALID_ARG, "q_dtype %d is not an eta_dtype_t", q_dtype);
  if (!q || !bias || !tau_out) return fail(ETA_ERR_INVALID_ARG, "q, bias and tau_out must be non-NULL");
  if (!aligned16(q) || !aligned16(bias) || !aligned16(tau_out) || (W && !aligned16(W)))
    return fail(ETA_ERR_INVALID_ARG, "q, W, bias and tau_out must be 16-byte aligned");
  hipError_t e = launch_predict(batch, num_q_heads, head_dim, q_dtype, q, W, bias, tau_out,
                                (hipStream_t)stream, active_hook());
  if (e != hipSuccess) return fail(ETA_ERR_HIP, "predictor launch failed: %s", hipGetErrorString(e));
  return ok();
}

eta_status_t eta_decode_workspace_size(const eta_kv_desc_t* kv, int64_t n_blk_cap,
                                       const eta_decode_params_t* p, size_t* bytes) {
  Geom g;
  eta_status_t st = check_kv(kv, &g);
  if (st) return st;
  if ((st = set_blk_cap(n_blk_cap, &g))) return st;
  if ((st = check_params(p))) return st;
  if (!bytes) return fail(ETA_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = decode_ws_bytes(g, plan_splits(g, p->num_splits), nullptr, nullptr);
  return ok();
}

static eta_status_t decode_impl(const eta_kv_desc_t* kv, int32_t q_dtype, const void* q,
                                const void* k, const void* v, const int32_t* seq_lens,
                                const eta_summary_t* summ, const float* tau, const float* W,
                                const float* bias, float* tau_out,
                                const eta_decode_params_t* p, void* out, uint8_t* block_mask,
                                int32_t* head_token_counts, int32_t* union_counts,
                                void* workspace, size_t workspace_bytes, void* stream,
                                bool library_scratch = false) {
  Geom g;
  eta_status_t st = check_kv(kv, &g);
  if (st) return st;
  if ((st = check_params(p))) return st;
  if (!valid_dtype(q_dtype)) return fail(ETA_ERR_INVALID_ARG, "q_dtype %d is not an eta_dtype_t", q_dtype);
  if (!q || !k || !v || !seq_lens || !out || !block_mask)
    return fail(ETA_ERR_INVALID_ARG, "q, k, v, seq_lens, out and block_mask must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(seq_lens) ||
      !aligned16(out) || !aligned16(block_mask) ||
      (head_token_counts && !aligned16(head_token_counts)) ||
      (union_counts && !aligned16(union_counts)) || (tau && !aligned16(tau)) ||
      (W && !aligned16(W)) || (bias && !aligned16(bias)) || (tau_out && !aligned16(tau_out)))
    return fail(ETA_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  // the mask and the workspace are laid out with the summary capacity
  if ((st = check_summary(summ, &g))) return st;
  const SplitPlan plan = plan_splits(g, p->num_splits);
  if (library_scratch) {
    // every check above is on the host; the scratch is looked up only for a valid call
    const size_t need = decode_ws_bytes(g, plan, nullptr, nullptr);
    if (need > kScratchBytes)
      return fail(ETA_ERR_WORKSPACE,
                  "this call needs %zu bytes of scratch; the library's scratch holds %zu "
                  "(use eta_decode_predicted with a workspace)", need, kScratchBytes);
    hipError_t e = scratch_address((hipStream_t)stream, &workspace);
    if (e != hipSuccess)
      return fail(ETA_ERR_HIP, "library scratch lookup failed: %s", hipGetErrorString(e));
    workspace_bytes = kScratchBytes;
  }
  if (!workspace) return fail(ETA_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(ETA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  DecodeWs ws;
  const size_t need = decode_ws_bytes(g, plan, &ws, workspace);
  if (workspace_bytes < need)
    return fail(ETA_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
  DecodeCfg c{p->beta, p->z, p->offset_a, p->rescue_window_blocks, p->pin_recent_blocks,
              p->self_ungated ? 1 : 0, p->screen_all ? 1 : 0, plan};
  hipError_t e = launch_decode(g, c, q_dtype, q, k, v, seq_lens, *summ, tau, W, bias, tau_out,
                               out, block_mask, head_token_counts, union_counts, ws,
                               (hipStream_t)stream, active_hook());
  if (e != hipSuccess) return fail(ETA_ERR_HIP, "decode launch failed: %s", hipGetErrorString(e));
  return ok();
}

eta_status_t eta_decode(const eta_kv_desc_t* kv, int32_t q_dtype, const void* q, const void* k,
                        const void* v, const int32_t* seq_lens, const eta_summary_t* summ,
                        const float* tau, const eta_decode_params_t* p, void* out,
                        uint8_t* block_mask, int32_t* head_token_counts, int32_t* union_counts,
                        void* workspace, size_t workspace_bytes, void* stream) {
  if (!tau) return fail(ETA_ERR_INVALID_ARG, "tau must be non-NULL");
  return decode_impl(kv, q_dtype, q, k, v, seq_lens, summ, tau, nullptr, nullptr, nullptr, p, out,
                     block_mask, head_token_counts, union_counts, workspace, workspace_bytes,
                     stream);
}

eta_status_t eta_decode_predicted(const eta_kv_desc_t* kv, int32_t q_dtype, const void* q,
                                  const void* k, const void* v, const int32_t* seq_lens,
                                  const eta_summary_t* summ, const float* W, const float* bias,
                                  const eta_decode_params_t* p, void* out, uint8_t* block_mask,
                                  int32_t* head_token_counts, int32_t* union_counts,
                                  float* tau_out, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  if (!bias) return fail(ETA_ERR_INVALID_ARG, "bias must be non-NULL");
  return decode_impl(kv, q_dtype, q, k, v, seq_lens, summ, nullptr, W, bias, tau_out, p, out,
                     block_mask, head_token_counts, union_counts, workspace, workspace_bytes,
                     stream);
}

eta_status_t eta_decode_predicted_noalloc(const eta_kv_desc_t* kv, int32_t q_dtype,
                                          const void* q, const void* k, const void* v,
                                          const int32_t* seq_lens, const eta_summary_t* summ,
                                          const float* W, const float* bias,
                                          const eta_decode_params_t* p, void* out,
                                          uint8_t* block_mask, int32_t* head_token_counts,
                                          int32_t* union_counts, float* tau_out, void* stream) {
  if (!bias) return fail(ETA_ERR_INVALID_ARG, "bias must be non-NULL");
  return decode_impl(kv, q_dtype, q, k, v, seq_lens, summ, nullptr, W, bias, tau_out, p, out,
                     block_mask, head_token_counts, union_counts, nullptr, 0, stream, true);
}

static eta_status_t check_calib(const eta_calib_desc_t* cd, const eta_calib_state_t* st) {
  if (!cd || !st) return fail(ETA_ERR_INVALID_ARG, "calibration descriptor or state is NULL");
  if (cd->num_seqs < 1 || cd->num_seqs > 65535 || cd->seq_len < 1)
    return fail(ETA_ERR_INVALID_ARG, "num_seqs must be in [1, 65535] and seq_len >= 1");
  if (cd->num_q_heads < 1 || cd->num_kv_heads < 1 || cd->num_q_heads % cd->num_kv_heads != 0)
    return fail(ETA_ERR_INVALID_ARG, "num_q_heads must be a positive multiple of num_kv_heads");
  const int G = cd->num_q_heads / cd->num_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(ETA_ERR_UNSUPPORTED, "GQA group size %d unsupported (1, 2, 4 or 8)", G);
  if (cd->num_q_heads > 256) return fail(ETA_ERR_UNSUPPORTED, "num_q_heads > 256 unsupported");
  if (cd->head_dim != 64 && cd->head_dim != 128)
    return fail(ETA_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", cd->head_dim);
  if (cd->dtype != ETA_DT_BF16)
    return fail(ETA_ERR_UNSUPPORTED, "calibration takes bf16 q and K (dtype %d)", cd->dtype);
  if (!std::isfinite(cd->beta) || cd->beta <= 0.f)
    return fail(ETA_ERR_INVALID_ARG, "beta must be finite and > 0");
  if (!std::isfinite(cd->lo) || !std::isfinite(cd->hi) || !(cd->lo < cd->hi))
    return fail(ETA_ERR_INVALID_ARG, "histogram range must be finite with lo < hi");
  if (cd->num_bins < 1 || cd->num_bins > kCalibBinsMax)
    return fail(ETA_ERR_INVALID_ARG, "num_bins must be in [1, %d]", kCalibBinsMax);
  if ((int64_t)cd->num_seqs * cd->seq_len >= (int64_t(1) << 23))
    return fail(ETA_ERR_INVALID_ARG, "num_seqs x seq_len must stay below 2^23 (fixed-point range)");
  if (!st->hist || !st->density) return fail(ETA_ERR_INVALID_ARG, "accumulators must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(st->hist) | reinterpret_cast<uintptr_t>(st->density)) & 7u)
    return fail(ETA_ERR_INVALID_ARG, "accumulators must be 8-byte aligned");
  return ETA_OK;
}

eta_status_t eta_calib_accumulate(const eta_calib_desc_t* cd, const void* q, const void* k,
                                  const float* tau, const eta_calib_state_t* st, void* stream) {
  eta_status_t s = check_calib(cd, st);
  if (s) return s;
  if (!q || !k || !tau) return fail(ETA_ERR_INVALID_ARG, "q, k and tau must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(tau))
    return fail(ETA_ERR_INVALID_ARG, "q, k and tau must be 16-byte aligned");
  hipError_t e = launch_calib(*cd, q, k, tau, *st, (hipStream_t)stream, active_hook());
  if (e != hipSuccess) return fail(ETA_ERR_HIP, "calibration launch failed: %s", hipGetErrorString(e));
  return ok();
}

eta_status_t eta_calib_solve(const eta_calib_desc_t* cd, const eta_calib_state_t* st, float* c_out,
                             double* target_out, void* stream) {
  eta_status_t s = check_calib(cd, st);
  if (s) return s;
  if (!c_out) return fail(ETA_ERR_INVALID_ARG, "c_out must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(c_out) & 3u) || (reinterpret_cast<uintptr_t>(target_out) & 7u))
    return fail(ETA_ERR_INVALID_ARG, "c_out / target_out misaligned");
  hipError_t e = launch_calib_solve(*cd, *st, c_out, target_out, (hipStream_t)stream, active_hook());
  if (e != hipSuccess) return fail(ETA_ERR_HIP, "calibration solve launch failed: %s", hipGetErrorString(e));
  return ok();
}

eta_status_t eta_gated_prefill(const eta_prefill_desc_t* pd, const void* q, const void* k,
                               const void* v, const float* tau, const int32_t* seq_lens,
                               void* out, float* R, float* L, void* stream) {
  if (!pd) return fail(ETA_ERR_INVALID_ARG, "prefill descriptor is NULL");
  if (pd->batch < 1 || pd->batch > 65535 || pd->capacity_tokens < 1)
    return fail(ETA_ERR_INVALID_ARG, "batch must be in [1, 65535] and capacity_tokens >= 1");
  if (pd->num_q_heads < 1 || pd->num_kv_heads < 1 || pd->num_q_heads % pd->num_kv_heads != 0)
    return fail(ETA_ERR_INVALID_ARG, "num_q_heads must be a positive multiple of num_kv_heads");
  const int G = pd->num_q_heads / pd->num_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(ETA_ERR_UNSUPPORTED, "GQA group size %d unsupported (1, 2, 4 or 8)", G);
  if (pd->num_q_heads > 256) return fail(ETA_ERR_UNSUPPORTED, "num_q_heads > 256 unsupported");
  if (pd->head_dim != 64 && pd->head_dim != 128)
    return fail(ETA_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", pd->head_dim);
  if (pd->dtype != ETA_DT_BF16) return fail(ETA_ERR_UNSUPPORTED, "prefill takes bf16 q, k, v");
  if (!std::isfinite(pd->beta) || pd->beta < 0.f)
    return fail(ETA_ERR_INVALID_ARG, "beta must be finite and >= 0");
  if (pd->additive != 0 && pd->additive != 1) return fail(ETA_ERR_INVALID_ARG, "additive must be 0 or 1");
  if (pd->additive && !std::isfinite(pd->C)) return fail(ETA_ERR_INVALID_ARG, "C must be finite");
  if (!q || !k || !v || !tau || !seq_lens || !out || !R || !L)
    return fail(ETA_ERR_INVALID_ARG, "q, k, v, tau, seq_lens, out, R and L must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) ||
      (reinterpret_cast<uintptr_t>(tau) | reinterpret_cast<uintptr_t>(R) |
       reinterpret_cast<uintptr_t>(L) | reinterpret_cast<uintptr_t>(seq_lens)) & 3u)
    return fail(ETA_ERR_INVALID_ARG, "q, k, v, out must be 16-byte and tau, R, L, seq_lens 4-byte aligned");
  hipError_t e = launch_prefill(*pd, q, k, v, tau, seq_lens, out, R, L, (hipStream_t)stream,
                                active_hook());
  if (e != hipSuccess) return fail(ETA_ERR_HIP, "prefill launch failed: %s", hipGetErrorString(e));
  return ok();
}

eta_status_t eta_block_bounds(const eta_kv_desc_t* kv, int32_t q_dtype, const void* q,
                              const int32_t* seq_lens, const eta_summary_t* summ, float z,
                              float* bounds, void* stream) {
  Geom g;
  eta_status_t st = check_kv(kv, &g);
  if (st) return st;
  if (!valid_dtype(q_dtype)) return fail(ETA_ERR_INVALID_ARG, "q_dtype %d is not an eta_dtype_t", q_dtype);
  if (!std::isfinite(z) || z < 0.f) return fail(ETA_ERR_INVALID_ARG, "z must be finite and >= 0");
  if (!q || !seq_lens || !bounds) return fail(ETA_ERR_INVALID_ARG, "q, seq_lens and bounds must be non-NULL");
  if (!aligned16(q) || !aligned16(seq_lens) || !aligned16(bounds))
    return fail(ETA_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  if ((st = check_summary(summ, &g))) return st;
  hipError_t e = launch_bounds(g, q_dtype, q, seq_lens, *summ, z, bounds, (hipStream_t)stream,
                               active_hook());
  if (e != hipSuccess) return fail(ETA_ERR_HIP, "bounds launch failed: %s", hipGetErrorString(e));
  return ok();
}

eta_status_t eta_dense_workspace_size(const eta_kv_desc_t* kv, int32_t num_splits, size_t* bytes) {
  Geom g;
  eta_status_t st = check_kv(kv, &g);
  if (st) return st;
  if (num_splits < 0 || num_splits > kMaxSplits)
    return fail(ETA_ERR_INVALID_ARG, "num_splits must be in [0, %d]", kMaxSplits);
  if (!bytes) return fail(ETA_ERR_INVALID_ARG, "bytes is NULL");
  const int S = num_splits > 0 ? num_splits : default_splits(g);
  *bytes = dense_ws_bytes(g, S, nullptr, nullptr);
  return ok();
}

eta_status_t eta_dense_decode(const eta_kv_desc_t* kv, int32_t q_dtype, const void* q,
                              const void* k, const void* v, const int32_t* seq_lens, void* out,
                              int32_t num_splits, void* workspace, size_t workspace_bytes,
                              void* stream) {
  Geom g;
  eta_status_t st = check_kv(kv, &g);
  if (st) return st;
  if (!valid_dtype(q_dtype)) return fail(ETA_ERR_INVALID_ARG, "q_dtype %d is not an eta_dtype_t", q_dtype);
  if (num_splits < 0 || num_splits > kMaxSplits)
    return fail(ETA_ERR_INVALID_ARG, "num_splits must be in [0, %d]", kMaxSplits);
  if (!q || !k || !v || !seq_lens || !out)
    return fail(ETA_ERR_INVALID_ARG, "q, k, v, seq_lens and out must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(seq_lens) || !aligned16(out))
    return fail(ETA_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  const int S = num_splits > 0 ? num_splits : default_splits(g);
  if (!workspace) return fail(ETA_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(ETA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  DecodeWs ws;
  const size_t need = dense_ws_bytes(g, S, &ws, workspace);
  if (workspace_bytes < need)
    return fail(ETA_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
  hipError_t e = launch_dense(g, S, q_dtype, q, k, v, seq_lens, out, ws, (hipStream_t)stream,
                              active_hook());
  if (e != hipSuccess) return fail(ETA_ERR_HIP, "dense launch failed: %s", hipGetErrorString(e));
  return ok();
}

eta_status_t eta_profile_begin(void) {
  Profiler& P = prof();
  std::lock_guard<std::mutex> lk(P.mu);
  P.on = true;
  P.used = 0;
  P.kinds.clear();
  return ok();
}

eta_status_t eta_profile_end(eta_kernel_time_t* out) {
  Profiler& P = prof();
  std::lock_guard<std::mutex> lk(P.mu);
  if (!out) return fail(ETA_ERR_INVALID_ARG, "out is NULL");
  for (int i = 0; i < ETA_KERNEL_KINDS; ++i) out[i] = eta_kernel_time_t{0.0, 0};
  P.on = false;
  for (size_t i = 0; i < P.used; ++i) {
    hipError_t e = hipEventSynchronize(P.pool[2 * i + 1]);
    if (e != hipSuccess) return fail(ETA_ERR_HIP, "event synchronize failed: %s", hipGetErrorString(e));
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, P.pool[2 * i], P.pool[2 * i + 1]);
    if (e != hipSuccess) return fail(ETA_ERR_HIP, "event elapsed time failed: %s", hipGetErrorString(e));
    const int k = P.kinds[i];
    if (k >= 0 && k < ETA_KERNEL_KINDS) {
      out[k].ms_total += ms;
      out[k].launches += 1;
    }
  }
  P.used = 0;
  P.kinds.clear();
  return ok();
}

}  // extern "C"
