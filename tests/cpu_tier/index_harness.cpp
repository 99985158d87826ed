// CPU bounds harness of the split-decode kernel's index arithmetic
// (paper_2609_20888_amd/csrc/eta_index.h, the functions the kernels call), built
// with the address and undefined-behaviour sanitizers.  Every array is a heap
// allocation of exactly the size the kernel's buffer has, so an index outside it
// is reported by the sanitizer; the checks add the invariants the kernels rely
// on: each union item / 64-token tile is taken by exactly one split, the
// proportional plan gives every group at least one split and no more than W in
// all, and every workgroup finds its group.  Exit status 0 when all hold.
#include <cstdio>
#include <cstdlib>
#include <cstdint>
#include <random>
#include <vector>

#include "eta_index.h"

using namespace eta;

static int failures = 0;
#define CHECK(c, ...)                                     \
  do {                                                    \
    if (!(c)) {                                           \
      ++failures;                                         \
      if (failures < 20) {                                \
        std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
        std::fprintf(stderr, __VA_ARGS__);                \
        std::fprintf(stderr, "\n");                       \
      }                                                   \
    }                                                     \
  } while (0)

// The proportional plan for BG groups with the given work, W workgroups.
static void check_plan(const std::vector<int>& work, int W) {
  const int BG = (int)work.size();
  int64_t total = 0;
  for (int x : work) total += x;
  int* first = new int[BG + 1];            // the kernel's grp_s
  for (int x = 0; x < BG; ++x) first[x] = group_splits(work[x], total, W, BG);
  for (int x = 0; x < BG; ++x) CHECK(first[x] >= 1, "group %d has %d splits", x, first[x]);
  first[BG] = exclusive_prefix(first, BG);
  CHECK(first[BG] <= W, "plan uses %d of %d workgroups", first[BG], W);
  std::vector<int> seen(BG, 0);
  for (int me = 0; me < W; ++me) {
    const int gi = find_group(first, BG, me);
    if (me >= first[BG]) {
      CHECK(gi == -1, "workgroup %d past the plan got group %d", me, gi);
      continue;
    }
    CHECK(gi >= 0 && gi < BG, "workgroup %d: group %d", me, gi);
    if (gi < 0 || gi >= BG) continue;
    CHECK(first[gi] <= me && me < first[gi + 1], "workgroup %d outside its group's range", me);
    ++seen[gi];
  }
  for (int x = 0; x < BG; ++x)
    CHECK(seen[x] == first[x + 1] - first[x], "group %d: %d workgroups seen", x, seen[x]);
  delete[] first;
}

// A group's union list: per-tile counts -> prefix (as the kernel's pref_s) ->
// every item resolved, every 64-token tile taken by exactly one split.
static void check_list(const std::vector<int>& counts, int S, int tiles_per_block, int ncap) {
  const int n_tiles = (int)counts.size();
  int* pref = new int[n_tiles + 1];
  for (int t = 0; t < n_tiles; ++t) pref[t] = counts[t];
  pref[n_tiles] = exclusive_prefix(pref, n_tiles);
  const int UI = pref[n_tiles];
  int32_t* ids = new int32_t[ncap];        // the group's compacted id slots
  for (int i = 0; i < ncap; ++i) ids[i] = i;
  for (int64_t it = 0; it < UI; ++it) {
    int tl = -1, slot = -1;
    resolve_item(pref, n_tiles, it, &tl, &slot);
    CHECK(tl >= 0 && tl < n_tiles && slot >= 0 && slot < counts[tl],
          "item %lld -> tile %d slot %d", (long long)it, tl, slot);
    const int64_t idx = (int64_t)tl * 64 + slot;
    CHECK(idx < ncap, "id index %lld >= %d", (long long)idx, ncap);
    if (idx < ncap) (void)ids[idx];
  }
  // strided shares of the list's tiles
  const int64_t UT = (int64_t)UI * tiles_per_block;
  std::vector<int> taken(UT, 0);
  int64_t sum = 0;
  for (int s = 0; s < S; ++s) {
    const int nt = strided_share(UT, s, S);
    sum += nt;
    for (int k = 0; k < nt; ++k) {
      const int64_t t = s + (int64_t)S * k;
      CHECK(t < UT, "split %d tile %lld >= %lld", s, (long long)t, (long long)UT);
      if (t < UT) ++taken[t];
    }
  }
  CHECK(sum == UT, "strided shares cover %lld of %lld tiles", (long long)sum, (long long)UT);
  for (int64_t t = 0; t < UT; ++t) CHECK(taken[t] == 1, "tile %lld taken %d times", (long long)t, taken[t]);
  // contiguous shares of the items
  int64_t prev = 0;
  for (int s = 0; s < S; ++s) {
    int64_t lo, hi;
    contiguous_share(UI, s, S, &lo, &hi);
    CHECK(lo == prev && lo <= hi && hi <= UI, "split %d: [%lld, %lld)", s, (long long)lo, (long long)hi);
    prev = hi;
  }
  CHECK(prev == UI, "contiguous shares end at %lld of %d", (long long)prev, UI);
  delete[] ids;
  delete[] pref;
}

// Compacted union id slots of one tile: distinct, inside the tile's 64 slots.
static void check_compaction(uint64_t bal, int tile, int64_t base, int ncap) {
  std::vector<int> used(64, 0);
  for (int lane = 0; lane < 64; ++lane) {
    if (!((bal >> lane) & 1ull)) continue;
    const int64_t at = union_slot(base, tile, bal, lane);
    const int64_t rel = at - base - (int64_t)tile * 64;
    CHECK(rel >= 0 && rel < __builtin_popcountll(bal), "lane %d -> slot %lld", lane, (long long)rel);
    CHECK(at - base < ncap, "slot %lld past the group's %d ids", (long long)(at - base), ncap);
    if (rel >= 0 && rel < 64) ++used[rel];
  }
  for (int r = 0; r < 64; ++r) CHECK(used[r] <= 1, "slot %d used %d times", r, used[r]);
}

int main() {
  std::mt19937_64 rng(12345);
  // plans: one group, the largest table, all work in one group, no work, ragged
  const int Ws[] = {1, 2, 63, 512, 1024, 4096};
  const int BGs[] = {1, 2, 32, 255, 256, 1024};
  for (int BG : BGs) {
    for (int W : Ws) {
      if (W < BG) continue;
      std::vector<int> work(BG);
      for (auto& x : work) x = 0;
      check_plan(work, W);                                          // nothing selected
      for (auto& x : work) x = 1;
      check_plan(work, W);                                          // tails only
      for (auto& x : work) x = (int)(rng() % 262145);               // up to 131072 blocks x 2 tiles + 1
      check_plan(work, W);
      for (auto& x : work) x = 0;
      work[BG - 1] = 262145;
      check_plan(work, W);                                          // one long union
    }
  }
  // union lists: T < b (no tile counted), one tile, ragged, the largest table
  const int tiles[] = {1, 2, 63, 64, 2048};
  const int splits[] = {1, 2, 5, 64, 300, 1024};
  for (int nt : tiles) {
    for (int S : splits) {
      for (int tpb : {1, 2}) {
        std::vector<int> counts(nt);
        for (auto& c : counts) c = 0;
        check_list(counts, S, tpb, nt * 64);
        for (auto& c : counts) c = 64;
        check_list(counts, S, tpb, nt * 64);
        for (auto& c : counts) c = (int)(rng() % 65);
        check_list(counts, S, tpb, nt * 64);
        // a last tile that is only partly inside the capacity (ncap = 64 (nt - 1) + 7)
        for (auto& c : counts) c = 64;
        counts[nt - 1] = 7;
        check_list(counts, S, tpb, 64 * (nt - 1) + 7);
      }
    }
  }
  for (int k = 0; k < 2000; ++k) {
    uint64_t bal = rng();
    if (k % 7 == 0) bal = 0;
    if (k % 11 == 0) bal = ~0ull;
    check_compaction(bal, (int)(rng() % 2048), (int64_t)(rng() % 1000) * 131072, 2048 * 64);
  }
  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("index harness: all checks passed\n");
  return 0;
}
