// Host side of libeta (eta_api.cpp: argument validation, split planning,
// workspace carve-up) built with the address and undefined-behaviour sanitizers
// against stub launchers that check what they are handed instead of launching.
// The decode stubs write to every workspace region the carve-up hands out, at
// both ends of the size its layout defines, inside a workspace
// allocated at exactly eta_decode_workspace_size() bytes: a region reaching past
// the workspace is a heap overflow the sanitizer reports, and every region is
// also checked against the workspace's extent and the other regions.  Exit
// status 0 when all hold.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "eta.h"
#include "eta_internal.h"

static int failures = 0;
static int launches = 0;
#define CHECK(c, ...)                                                 \
  do {                                                                \
    if (!(c)) {                                                       \
      ++failures;                                                     \
      if (failures < 30) {                                            \
        std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__);     \
        std::fprintf(stderr, __VA_ARGS__);                            \
        std::fprintf(stderr, "\n");                                   \
      }                                                               \
    }                                                                 \
  } while (0)

struct Region {
  void* p;
  size_t bytes;
};

static const unsigned char* g_ws = nullptr;   // the workspace of the call under test
static size_t g_ws_bytes = 0;

// Each region inside [g_ws, g_ws + g_ws_bytes), 16-byte aligned, no two
// overlapping; its first and last 4 KiB are written (the sanitizer reports a
// write past the allocation, whatever the explicit check says).
static void fill_and_check(const std::vector<Region>& rs, const char* what) {
  for (size_t r = 0; r < rs.size(); ++r) {
    const unsigned char* p = static_cast<const unsigned char*>(rs[r].p);
    CHECK(p >= g_ws && p + rs[r].bytes <= g_ws + g_ws_bytes,
          "%s: region %zu [%td, +%zu) outside the %zu-byte workspace", what, r, p - g_ws,
          rs[r].bytes, g_ws_bytes);
    CHECK(reinterpret_cast<uintptr_t>(p) % 16 == 0, "%s: region %zu not 16-byte aligned", what, r);
    for (size_t o = 0; o < r; ++o) {
      const unsigned char* q = static_cast<const unsigned char*>(rs[o].p);
      const bool apart = p + rs[r].bytes <= q || q + rs[o].bytes <= p;
      CHECK(apart || rs[r].bytes == 0 || rs[o].bytes == 0, "%s: regions %zu and %zu overlap", what,
            o, r);
    }
    const size_t edge = rs[r].bytes < 8192 ? rs[r].bytes : 4096;
    std::memset(rs[r].p, (int)(r + 1), edge);
    std::memset(static_cast<unsigned char*>(rs[r].p) + rs[r].bytes - edge, (int)(r + 1), edge);
  }
}

// The real launchers bracket each kernel with the hook; the stubs do the same
// so the kernel timer sees one launch per call.
static void bracket(eta::LaunchHook hook, int kind, hipStream_t st) {
  if (hook) {
    hook(kind, st, false);
    hook(kind, st, true);
  }
}

// ------------------------------------------------------------------ HIP stubs
extern "C" {
// The library keeps its timer's events until the process ends: hand out
// addresses inside a static pool rather than heap objects.
static char g_events[1 << 18];
static size_t g_next_event = 0;
hipError_t hipEventCreate(hipEvent_t* e) {
  *e = reinterpret_cast<hipEvent_t>(g_events + (g_next_event++ % sizeof(g_events)));
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t) { return hipSuccess; }
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) {
  *ms = 1.0f;
  return hipSuccess;
}
const char* hipGetErrorString(hipError_t) { return "stub"; }
}

// ------------------------------------------------------------------ launcher stubs
namespace eta {

static void* g_scratch = nullptr;

hipError_t scratch_address(hipStream_t, void** out) {
  if (!g_scratch) g_scratch = std::aligned_alloc(256, kScratchBytes);
  *out = g_scratch;
  return hipSuccess;
}

hipError_t launch_summaries(const Geom& g, const void*, const int32_t*, const int32_t*, int, int,
                            const eta_summary_t& s, hipStream_t stream, LaunchHook hook) {
  ++launches;
  bracket(hook, ETA_KERNEL_SUMMARIES, stream);
  CHECK(s.n_blk_cap >= g.cap / g.BS, "summary capacity");
  return hipSuccess;
}
hipError_t launch_predict(int B, int Hq, int D, int, const void*, const float*, const float*, float*,
                          hipStream_t stream, LaunchHook hook) {
  ++launches;
  bracket(hook, ETA_KERNEL_PREDICT, stream);
  CHECK(B >= 1 && Hq >= 1 && Hq <= 256 && D >= 1 && D <= 1024, "predict geometry");
  return hipSuccess;
}

hipError_t launch_decode(const Geom& g, const DecodeCfg& c, int, const void*, const void*,
                         const void*, const int32_t*, const eta_summary_t&, const float*,
                         const float*, const float*, float*, void*, uint8_t*, int32_t*, int32_t*,
                         const DecodeWs& ws, hipStream_t stream, LaunchHook hook) {
  ++launches;
  bracket(hook, ETA_KERNEL_SCREEN, stream);
  const size_t B = g.B, Hq = g.Hq, Hkv = g.Hkv, BG = B * Hkv, W = (size_t)c.plan.W;
  if (c.plan.S > 0) {
    CHECK((size_t)c.plan.S * BG == W, "uniform plan: W %zu != S %d x %zu groups", W, c.plan.S, BG);
    CHECK(c.plan.S <= kMaxSplits, "S %d", c.plan.S);
  } else {
    // proportional: the split kernel keeps every tile count and group in LDS
    CHECK(g.B > 1 && BG <= (size_t)kPropMaxGroups && BG * g.n_tiles <= (size_t)kPropMaxCounts,
          "proportional plan outside the kernel's LDS tables (%zu groups, %d tiles)", BG, g.n_tiles);
    CHECK(W >= BG, "proportional plan: %zu workgroups for %zu groups", W, BG);
  }
  CHECK(g.n_tiles >= 1 && g.n_tiles <= kMaxTiles && g.n_tiles * (int64_t)kScreenTile >= g.ncap,
        "n_tiles %d for %lld blocks", g.n_tiles, (long long)g.ncap);
  std::vector<Region> rs = {
      {ws.ids, BG * g.ncap * 4},           {ws.tile_cnt, BG * g.n_tiles * 4},
      {ws.head_cnt, B * Hq * g.n_tiles * 4}, {ws.part_ml, W * g.G * 8},
      {ws.part_acc, W * g.G * g.D * 4},    {ws.tau, B * Hq * 4},
      {ws.resc_best, B * Hq * kRescueTiles * 4}, {ws.resc_info, B * Hq * kRescueTiles * 4},
      {ws.wbits, BG * kMaxRescueWindow},   {ws.resc_out, B * Hq * 4},
      {ws.extra_union, BG * 4},            {ws.plan, BG * 8}};
  fill_and_check(rs, "decode");
  return hipSuccess;
}

hipError_t launch_bounds(const Geom&, int, const void*, const int32_t*, const eta_summary_t&, float,
                         float*, hipStream_t stream, LaunchHook hook) {
  ++launches;
  bracket(hook, ETA_KERNEL_BOUNDS, stream);
  return hipSuccess;
}
hipError_t launch_calib(const eta_calib_desc_t&, const void*, const void*, const float*,
                        const eta_calib_state_t&, hipStream_t stream, LaunchHook hook) {
  ++launches;
  bracket(hook, ETA_KERNEL_CALIB_ACCUMULATE, stream);
  return hipSuccess;
}
hipError_t launch_calib_solve(const eta_calib_desc_t&, const eta_calib_state_t&, float*, double*,
                              hipStream_t stream, LaunchHook hook) {
  ++launches;
  bracket(hook, ETA_KERNEL_CALIB_SOLVE, stream);
  return hipSuccess;
}
hipError_t launch_prefill(const eta_prefill_desc_t&, const void*, const void*, const void*,
                          const float*, const int32_t*, void*, float*, float*, hipStream_t stream,
                          LaunchHook hook) {
  ++launches;
  bracket(hook, ETA_KERNEL_PREFILL, stream);
  return hipSuccess;
}
hipError_t launch_dense(const Geom& g, int S, int, const void*, const void*, const void*,
                        const int32_t*, void*, const DecodeWs& ws, hipStream_t stream, LaunchHook hook) {
  ++launches;
  bracket(hook, ETA_KERNEL_DENSE_SPLIT, stream);
  const size_t BH = (size_t)g.B * g.Hq;
  std::vector<Region> rs = {{ws.part_ml, BH * S * 8}, {ws.part_acc, BH * S * g.D * 4}};
  fill_and_check(rs, "dense");
  return hipSuccess;
}

}  // namespace eta

// ------------------------------------------------------------------ driver
static void* const FAKE = reinterpret_cast<void*>(0x10000);   // aligned, never dereferenced

static eta_kv_desc_t desc(int B, int Hq, int Hkv, int d, int b, int64_t cap, int dt = ETA_DT_BF16) {
  eta_kv_desc_t k{};
  k.batch = B;
  k.num_q_heads = Hq;
  k.num_kv_heads = Hkv;
  k.head_dim = d;
  k.block_size = b;
  k.kv_dtype = dt;
  k.capacity_tokens = cap;
  k.stride_t = d;
  k.stride_h = cap * d;
  k.stride_b = (int64_t)Hkv * cap * d;
  return k;
}

static eta_decode_params_t params(int splits = 0) {
  eta_decode_params_t p{};
  p.beta = 4.0f;
  p.z = 1.0f;
  p.rescue_window_blocks = 128;
  p.num_splits = splits;
  return p;
}

static eta_summary_t summ(const eta_kv_desc_t& k, int st = ETA_DT_F32) {
  eta_summary_t s{};
  s.mu = FAKE;
  s.sigma = FAKE;
  s.max_norm = reinterpret_cast<float*>(FAKE);
  s.n_blk_cap = k.capacity_tokens / k.block_size;
  if (s.n_blk_cap < 1) s.n_blk_cap = 1;
  s.stat_dtype = st;
  return s;
}

// blk_extra: a summary holding that many blocks more than capacity_tokens /
// block_size (n_blk_cap only has a lower bound).
static void decode_geometry(int B, int Hq, int Hkv, int d, int b, int64_t cap, int splits,
                            int64_t blk_extra = 0) {
  eta_kv_desc_t k = desc(B, Hq, Hkv, d, b, cap);
  eta_decode_params_t p = params(splits);
  eta_summary_t s = summ(k);
  s.n_blk_cap += blk_extra;
  size_t need = 0;
  eta_status_t st = eta_decode_workspace_size(&k, s.n_blk_cap, &p, &need);
  CHECK(st == ETA_OK, "workspace size: %s", eta_last_error_string());
  if (st != ETA_OK) return;
  void* ws = std::aligned_alloc(256, (need + 255) / 256 * 256);
  g_ws = static_cast<const unsigned char*>(ws);
  g_ws_bytes = need;
  const int before = launches;
  st = eta_decode(&k, ETA_DT_BF16, FAKE, FAKE, FAKE, (const int32_t*)FAKE, &s, (const float*)FAKE,
                  &p, FAKE, (uint8_t*)FAKE, nullptr, nullptr, ws, need, nullptr);
  CHECK(st == ETA_OK && launches == before + 1,
        "decode B=%d %d/%d d=%d b=%d cap=%lld +%lld blocks S=%d: %s", B, Hq, Hkv, d, b,
        (long long)cap, (long long)blk_extra, splits, eta_last_error_string());
  st = eta_decode_predicted(&k, ETA_DT_BF16, FAKE, FAKE, FAKE, (const int32_t*)FAKE, &s,
                            (const float*)FAKE, (const float*)FAKE, &p, FAKE, (uint8_t*)FAKE,
                            nullptr, nullptr, nullptr, ws, need, nullptr);
  CHECK(st == ETA_OK, "decode_predicted: %s", eta_last_error_string());
  // one byte short of the requirement is refused before any launch
  const int mid = launches;
  st = eta_decode(&k, ETA_DT_BF16, FAKE, FAKE, FAKE, (const int32_t*)FAKE, &s, (const float*)FAKE,
                  &p, FAKE, (uint8_t*)FAKE, nullptr, nullptr, ws, need - 1, nullptr);
  CHECK(st == ETA_ERR_WORKSPACE && launches == mid, "short workspace accepted");
  // the library scratch: accepted up to its size, refused past it, nothing launched then
  void* scratch = nullptr;
  eta::scratch_address(nullptr, &scratch);
  g_ws = static_cast<const unsigned char*>(scratch);
  g_ws_bytes = need;
  st = eta_decode_predicted_noalloc(&k, ETA_DT_BF16, FAKE, FAKE, FAKE, (const int32_t*)FAKE, &s,
                                    (const float*)FAKE, (const float*)FAKE, &p, FAKE,
                                    (uint8_t*)FAKE, nullptr, nullptr, nullptr, nullptr);
  if (need <= ETA_DECODE_NOALLOC_SCRATCH_BYTES)
    CHECK(st == ETA_OK, "noalloc refused %zu bytes: %s", need, eta_last_error_string());
  else
    CHECK(st == ETA_ERR_WORKSPACE, "noalloc accepted %zu bytes", need);
  // the dense baseline's own workspace
  size_t dneed = 0;
  st = eta_dense_workspace_size(&k, splits, &dneed);
  CHECK(st == ETA_OK, "dense workspace size");
  void* dws = std::aligned_alloc(256, (dneed + 255) / 256 * 256);
  g_ws = static_cast<const unsigned char*>(dws);
  g_ws_bytes = dneed;
  st = eta_dense_decode(&k, ETA_DT_BF16, FAKE, FAKE, FAKE, (const int32_t*)FAKE, FAKE, splits, dws,
                        dneed, nullptr);
  CHECK(st == ETA_OK, "dense decode: %s", eta_last_error_string());
  std::free(dws);
  std::free(ws);
}

static void invalid_calls() {
  eta_kv_desc_t k = desc(2, 16, 4, 128, 64, 4096);
  eta_decode_params_t p = params();
  eta_summary_t s = summ(k);
  size_t need = 0;
  eta_decode_workspace_size(&k, s.n_blk_cap, &p, &need);
  // a block capacity below capacity_tokens / block_size is refused by the query too
  size_t none = 0;
  CHECK(eta_decode_workspace_size(&k, s.n_blk_cap - 1, &p, &none) == ETA_ERR_INVALID_ARG &&
            none == 0, "workspace query took n_blk_cap < capacity / block_size");
  void* ws = std::aligned_alloc(256, (need + 255) / 256 * 256);
  const int before = launches;
  auto dec = [&](const eta_kv_desc_t& kk, const eta_decode_params_t& pp, const eta_summary_t& ss,
                 const void* q, void* w, size_t wb) {
    return eta_decode(&kk, ETA_DT_BF16, q, FAKE, FAKE, (const int32_t*)FAKE, &ss,
                      (const float*)FAKE, &pp, FAKE, (uint8_t*)FAKE, nullptr, nullptr, w, wb, nullptr);
  };
  struct Case {
    eta_kv_desc_t k;
    eta_decode_params_t p;
    eta_summary_t s;
    const void* q;
    void* w;
    eta_status_t want;
  };
  std::vector<Case> cases;
  auto add = [&](eta_kv_desc_t kk, eta_decode_params_t pp, eta_summary_t ss, const void* q, void* w,
                 eta_status_t want) { cases.push_back({kk, pp, ss, q, w, want}); };
  add(k, p, s, nullptr, ws, ETA_ERR_INVALID_ARG);                     // q NULL
  add(k, p, s, reinterpret_cast<const char*>(FAKE) + 2, ws, ETA_ERR_INVALID_ARG);   // misaligned
  add(k, p, s, FAKE, nullptr, ETA_ERR_WORKSPACE);
  add(k, p, s, FAKE, static_cast<char*>(ws) + 16, ETA_ERR_WORKSPACE);  // not 256-byte aligned
  { auto b = k; b.batch = 0; add(b, p, s, FAKE, ws, ETA_ERR_INVALID_ARG); }
  { auto b = k; b.num_kv_heads = 3; add(b, p, s, FAKE, ws, ETA_ERR_INVALID_ARG); }
  { auto b = k; b.num_kv_heads = 1; add(b, p, s, FAKE, ws, ETA_ERR_UNSUPPORTED); }   // G = 16
  { auto b = k; b.head_dim = 96; b.stride_t = 96; add(b, p, s, FAKE, ws, ETA_ERR_UNSUPPORTED); }
  { auto b = k; b.block_size = 32; add(b, p, s, FAKE, ws, ETA_ERR_UNSUPPORTED); }
  { auto b = k; b.stride_t = 132; add(b, p, s, FAKE, ws, ETA_ERR_INVALID_ARG); }
  { auto b = k; b.kv_dtype = 9; add(b, p, s, FAKE, ws, ETA_ERR_INVALID_ARG); }
  { auto b = p; b.beta = -1.f; add(k, b, s, FAKE, ws, ETA_ERR_INVALID_ARG); }
  { auto b = p; b.rescue_window_blocks = 257; add(k, b, s, FAKE, ws, ETA_ERR_UNSUPPORTED); }
  { auto b = p; b.num_splits = 1025; add(k, b, s, FAKE, ws, ETA_ERR_INVALID_ARG); }
  { auto b = s; b.n_blk_cap = 63; add(k, p, b, FAKE, ws, ETA_ERR_INVALID_ARG); }
  { auto b = s; b.stat_dtype = ETA_DT_BF16; add(k, p, b, FAKE, ws, ETA_ERR_INVALID_ARG); }
  { auto b = s; b.mu = nullptr; add(k, p, b, FAKE, ws, ETA_ERR_INVALID_ARG); }
  { auto b = s; b.n_blk_cap = 131073; add(k, p, b, FAKE, ws, ETA_ERR_UNSUPPORTED); }
  for (size_t i = 0; i < cases.size(); ++i) {
    const Case& c = cases[i];
    const eta_status_t st = dec(c.k, c.p, c.s, c.q, c.w, need);
    CHECK(st == c.want, "invalid case %zu: status %d, want %d (%s)", i, st, c.want,
          eta_last_error_string());
    CHECK(std::strlen(eta_last_error_string()) > 0, "invalid case %zu: no error text", i);
  }
  CHECK(launches == before, "an invalid call launched a kernel");
  std::free(ws);
}

static void other_entry_points() {
  eta_kv_desc_t k = desc(1, 8, 2, 64, 128, 1000);
  eta_summary_t s = summ(k);
  int before = launches;
  CHECK(eta_build_block_summaries(&k, FAKE, (const int32_t*)FAKE, &s, nullptr) == ETA_OK, "summaries");
  CHECK(eta_build_block_summaries_envelope(&k, FAKE, (const int32_t*)FAKE, 8, &s, nullptr) == ETA_OK,
        "envelope");
  CHECK(eta_update_block_summaries(&k, FAKE, (const int32_t*)FAKE, (const int32_t*)FAKE, 1, 0, &s,
                                   nullptr) == ETA_OK, "update");
  CHECK(eta_block_bounds(&k, ETA_DT_BF16, FAKE, (const int32_t*)FAKE, &s, 1.0f, (float*)FAKE,
                         nullptr) == ETA_OK, "bounds");
  CHECK(eta_predict_threshold(3, 8, 64, ETA_DT_BF16, FAKE, (const float*)FAKE, (const float*)FAKE,
                              (float*)FAKE, nullptr) == ETA_OK, "predict");
  CHECK(launches == before + 5, "%d launches for five calls", launches - before);
  eta_calib_desc_t cd{2, 8, 2, 128, 256, ETA_DT_BF16, 4.0f, -4.0f, 4.0f, 512};
  eta_calib_state_t cs{reinterpret_cast<uint64_t*>(FAKE), reinterpret_cast<uint64_t*>(FAKE)};
  CHECK(eta_calib_accumulate(&cd, FAKE, FAKE, (const float*)FAKE, &cs, nullptr) == ETA_OK, "calib");
  CHECK(eta_calib_solve(&cd, &cs, (float*)FAKE, nullptr, nullptr) == ETA_OK, "calib solve");
  eta_prefill_desc_t pd{1, 8, 2, 128, 256, ETA_DT_BF16, 4.0f, 0, 0.0f};
  CHECK(eta_gated_prefill(&pd, FAKE, FAKE, FAKE, (const float*)FAKE, (const int32_t*)FAKE, FAKE,
                          (float*)FAKE, (float*)FAKE, nullptr) == ETA_OK, "prefill");
  // the kernel timer with stub events
  CHECK(eta_profile_begin() == ETA_OK, "profile begin");
  eta_build_block_summaries(&k, FAKE, (const int32_t*)FAKE, &s, nullptr);
  eta_kernel_time_t t[ETA_KERNEL_KINDS];
  CHECK(eta_profile_end(t) == ETA_OK && t[ETA_KERNEL_SUMMARIES].launches == 1, "profile end");
  CHECK(eta_abi_version() == 5, "abi version");
}

int main() {
  // geometries: one sequence and several, T < b, a partial last tile, the largest
  // screening table (2048 tiles), one split and the most
  const int Bs[] = {1, 2, 8, 33};
  const int heads[][2] = {{16, 4}, {32, 8}, {8, 1}, {8, 8}};
  const int64_t caps[] = {1, 63, 64, 4097, 131072};
  const int splits[] = {0, 1, 7, 1024};
  for (int B : Bs)
    for (auto& h : heads)
      for (int d : {64, 128})
        for (int b : {64, 128})
          for (int64_t cap : caps)
            for (int S : splits) decode_geometry(B, h[0], h[1], d, b, cap, S);
  decode_geometry(1, 16, 4, 128, 64, (int64_t)2048 * 64 * 64, 0);   // 2048 screening tiles
  decode_geometry(256, 32, 8, 128, 64, 65536, 0);                   // 2048 groups: uniform plan
  decode_geometry(32, 32, 8, 128, 64, 65536, 0);                    // proportional, 4096 counts
  // summaries larger than the cache: one block past, a tile past, and T < b with a
  // one-block summary (capacity_tokens / block_size = 0)
  for (int B : {1, 8})
    for (int64_t cap : {1, 63, 64, 4097})
      for (int S : {0, 1})
        for (int64_t extra : {1, 65}) decode_geometry(B, 16, 4, 128, 64, cap, S, extra);
  invalid_calls();
  other_entry_points();
  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("api harness: %d launches checked, all checks passed\n", launches);
  return 0;
}
