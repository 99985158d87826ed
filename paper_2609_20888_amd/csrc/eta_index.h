// Index arithmetic of the split-decode kernel: the proportional split plan, the
// union list's tile prefix and item lookup, and the splits' shares.  Every
// function is host + device code and touches only the arrays it is given, so
// the CPU bounds harness (tests/cpu_tier) runs the kernels' own arithmetic on
// edge geometries under the address and undefined-behaviour sanitizers.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define ETA_HD __host__ __device__ __forceinline__
#else
#define ETA_HD inline
#endif

namespace eta {

// Work of one (sequence, kv head) group for the proportional plan, in 64-token
// tiles: its union blocks' tiles, plus one when the sequence has a partial tail.
ETA_HD int group_work(int union_blocks, int tiles_per_block, int64_t seq_len, int block) {
  return union_blocks * tiles_per_block + ((seq_len % block) != 0 ? 1 : 0);
}

// Splits of a group under the proportional plan: one each, and the remaining
// W - BG dealt in proportion to the groups' work (rounded down), so the sum over
// the groups never exceeds W.  W >= BG >= 1.
ETA_HD int group_splits(int work, int64_t total_work, int W, int BG) {
  return 1 + (total_work > 0 ? (int)((int64_t)(W - BG) * work / total_work) : 0);
}

// In place: v[0..n) -> exclusive prefix sums; returns the total (callers keep it
// in v[n]).  The split kernel computes the same prefixes with block-wide scans
// (integer sums, so equal whatever the order); this is their definition.
ETA_HD int exclusive_prefix(int* v, int n) {
  int acc = 0;
  for (int x = 0; x < n; ++x) {
    const int k = v[x];
    v[x] = acc;
    acc += k;
  }
  return acc;
}

// Whether split workgroup `me` belongs to the group whose splits are
// [first, first + splits): under the proportional plan each group has at least
// one split and the groups' ranges follow each other, so exactly one group owns
// each workgroup below the number used and none owns the rest.
ETA_HD bool owns_split(int first, int splits, int me) {
  return first <= me && me < first + splits;
}

// Sequence of groups x0, x0 + step, x0 + 2 step, ... where group x is (sequence
// x / hkv, kv head x % hkv): one division, then one step per group.  Holds
// q = x / hkv and rm = x % hkv of the current group.
struct GroupStepper {
  unsigned q, rm, qn, rn, hkv;
  ETA_HD GroupStepper(unsigned x0, unsigned step, unsigned hkv_)
      : q(x0 / hkv_), rm(x0 % hkv_), qn(step / hkv_), rn(step % hkv_), hkv(hkv_) {}
  ETA_HD void next() {
    rm += rn;                      // < 2 hkv
    q += qn + (rm >= hkv ? 1u : 0u);
    rm -= rm >= hkv ? hkv : 0u;
  }
};

// Union list item `it` (pref = exclusive prefix of the per-tile union counts,
// pref[n_tiles] = their total, it < that total) -> the screening tile holding it
// and its slot among that tile's compacted ids: pref[tile] <= it < pref[tile + 1].
ETA_HD void resolve_item(const int* pref, int n_tiles, int64_t it, int* tile, int* slot) {
  int tl = 0, th = n_tiles;
  while (th - tl > 1) {
    const int mid = (tl + th) >> 1;
    if (pref[mid] <= it) tl = mid; else th = mid;
  }
  *tile = tl;
  *slot = (int)(it - pref[tl]);
}

// Number of 64-token tiles of split s of S under the strided share (tiles s,
// s + S, s + 2 S, ... of total_tiles).
ETA_HD int strided_share(int64_t total_tiles, int s, int S) {
  return total_tiles > s ? (int)((total_tiles - s + S - 1) / S) : 0;
}

// Contiguous share [lo, hi) of `items` for split s of S (the fp32 path).
ETA_HD void contiguous_share(int64_t items, int s, int S, int64_t* lo, int64_t* hi) {
  *lo = (items * s) / S;
  *hi = (items * (s + 1)) / S;
}

// Position of a compacted union id: tile t of a group whose ids start at
// group_base, lane l with ballot bal of the tile's union blocks.
ETA_HD int64_t union_slot(int64_t group_base, int tile, uint64_t bal, int lane) {
  const uint64_t below = lane == 0 ? 0ull : (bal & ((~0ull) >> (64 - lane)));
  return group_base + (int64_t)tile * 64 + __builtin_popcountll(below);
}

// Screening's record loads (dimension-major records, rows of n_blk_cap
// entries): element offset of the four consecutive records of row `row` that
// start at block j4 (a multiple of 4), for rows that are four-record aligned
// (ncap a multiple of 4, ncap >= 4), clamped so that all four lie in the row;
// and of one record at block j, clamped into the row (ncap >= 1).
ETA_HD int64_t screen_rec4_offset(int64_t row, int64_t ncap, int64_t j4) {
  return row * ncap + (j4 < ncap ? j4 : ncap - 4);
}
ETA_HD int64_t screen_rec1_offset(int64_t row, int64_t ncap, int64_t j) {
  return row * ncap + (j < ncap ? j : ncap - 1);
}

// The predictor's rows for thread t in pass p: the first of its four rows
// 1024 p + 4 t .. + 3 when they lie in [0, J) (J a multiple of 4), else 0.
ETA_HD int pred_row4(int p, int t, int J) {
  const int j = p * 1024 + 4 * t;
  return j < J ? j : 0;
}

}  // namespace eta
