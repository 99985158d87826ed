// Internal declarations shared by the host API (eta_api.cpp) and the HIP
// kernels (eta_kernels.hip, eta_prefill.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "eta.h"

namespace eta {

// Blocks screened by one workgroup (one lane per block), and the largest top-1
// rescue window (rescue_window_blocks <= kMaxRescueWindow).
constexpr int kScreenTile = 64;
constexpr int kMaxRescueWindow = 256;
constexpr int kRescueTiles = kMaxRescueWindow / kScreenTile;
constexpr int kRescueAny = -2;     // a block of the tile's window part is selected
constexpr int kRescueNone = -1;    // no block of the tile's window part has a bound
constexpr int kMaxSplits = 1024;
// Upper bound on screening tiles per (sequence, kv head): the split-decode
// kernel keeps their prefix sum in LDS.
constexpr int kMaxTiles = 2048;
// Union ids pack the block index below bit 24 and the head bits above it.
constexpr int64_t kMaxBlocks = int64_t(1) << 24;

struct Geom {
  int B, Hq, Hkv, D, BS, G;
  int kv_dtype;
  int64_t cap;               // capacity_tokens
  int64_t sb, sh, st;        // K/V strides in elements
  int64_t ncap;              // summary n_blk_cap
  int n_tiles;               // ceil(ncap / kScreenTile)
  int stat_dtype;            // summary mu / sigma element type (ETA_DT_F32, ETA_DT_F16 or ETA_DT_FP8)
};

// Workspace carve-up of eta_decode.
struct DecodeWs {
  float* resc_best;          // [B][Hq][kRescueTiles] top-1 rescue: window part of each tile
  int32_t* resc_info;        // [B][Hq][kRescueTiles]
  uint8_t* wbits;            // [B][Hkv][kMaxRescueWindow] union head bits of the window blocks
  int32_t* resc_out;         // [B][Hq] rescued block per head, or -1
  int32_t* extra_union;      // [B][Hkv] rescued blocks outside the union
  int2* plan;                // [B][Hkv] (first split workgroup, splits)
  int32_t* ids;              // [B][Hkv][ncap]   union block ids | head bits << 24, compacted
                             //                  per screening tile (tile t's ids start at
                             //                  t * kScreenTile)
  int32_t* tile_cnt;         // [B][Hkv][n_tiles] union blocks per tile
  int32_t* head_cnt;         // [B][Hq][n_tiles]  selected blocks per head per tile
  float2* part_ml;           // [W][G]            (running max, running sum) per split and head
  float* part_acc;           // [W][G][D]         unnormalised output per split and head
  float* tau;                // [B][Hq]           thresholds predicted by the screening kernel
};

// How split decode is laid out: S splits per (sequence, kv head) (uniform), or
// W workgroups dealt to the groups in proportion to their unions (proportional,
// several sequences; every split workgroup then reads all B Hkv n_tiles tile
// counts, which must fit in LDS).
constexpr int kPropMaxGroups = 1024;
constexpr int kPropMaxCounts = 4096;
struct SplitPlan {
  int S;                     // uniform splits per group (0 when proportional)
  int W;                     // split workgroups in all
};
SplitPlan plan_splits(const Geom& g, int num_splits);

size_t decode_ws_bytes(const Geom& g, const SplitPlan& sp, DecodeWs* carve, void* base);
size_t dense_ws_bytes(const Geom& g, int S, DecodeWs* carve, void* base);
int default_splits(const Geom& g);

struct DecodeCfg {
  float beta, z, offset_a;
  int rescue_window, lwb, self_ungated, screen_all;
  SplitPlan plan;
};

// Launchers: validated arguments in, one or more kernels enqueued on `stream`.
// `kind_cb` brackets each launch for the optional kernel timer.
using LaunchHook = void (*)(int kind, hipStream_t stream, bool after);

// prev_lens == nullptr: every full block; else the blocks completed since
// prev_lens (at most max_new_blocks per sequence).  sub_block > 0 (a power of
// two dividing the block size): sigma is the sub-block envelope.
hipError_t launch_summaries(const Geom& g, const void* k, const int32_t* seq_lens,
                            const int32_t* prev_lens, int max_new_blocks, int sub_block,
                            const eta_summary_t& s, hipStream_t stream, LaunchHook hook);

hipError_t launch_predict(int B, int Hq, int D, int q_dtype, const void* q, const float* W,
                          const float* bias, float* tau, hipStream_t stream, LaunchHook hook);

// tau == nullptr: the screening kernel predicts the thresholds from (W, bias)
// and, if tau_out is given, stores them there too.
hipError_t launch_decode(const Geom& g, const DecodeCfg& c, int q_dtype, const void* q,
                         const void* k, const void* v, const int32_t* seq_lens,
                         const eta_summary_t& s, const float* tau, const float* W,
                         const float* bias, float* tau_out, void* out, uint8_t* mask,
                         int32_t* counts, int32_t* union_counts, const DecodeWs& ws,
                         hipStream_t stream, LaunchHook hook);

hipError_t launch_bounds(const Geom& g, int q_dtype, const void* q, const int32_t* seq_lens,
                         const eta_summary_t& s, float z, float* bounds, hipStream_t stream,
                         LaunchHook hook);

hipError_t launch_calib(const eta_calib_desc_t& cd, const void* q, const void* k, const float* tau,
                        const eta_calib_state_t& st, hipStream_t stream, LaunchHook hook);
hipError_t launch_calib_solve(const eta_calib_desc_t& cd, const eta_calib_state_t& st, float* c_out,
                              double* target_out, hipStream_t stream, LaunchHook hook);
constexpr int kCalibBinsMax = 4096;
hipError_t launch_prefill(const eta_prefill_desc_t& pd, const void* q, const void* k, const void* v,
                          const float* tau, const int32_t* seq_lens, void* out, float* R, float* L,
                          hipStream_t stream, LaunchHook hook);

// The library's own device scratch (eta_decode_predicted_noalloc): kScratchBytes
// per GPU; scratch_address gives the address of the copy on the stream's device.
constexpr size_t kScratchBytes = size_t(32) << 20;
hipError_t scratch_address(hipStream_t stream, void** out);

hipError_t launch_dense(const Geom& g, int S, int q_dtype, const void* q, const void* k,
                        const void* v, const int32_t* seq_lens, void* out, const DecodeWs& ws,
                        hipStream_t stream, LaunchHook hook);

}  // namespace eta
