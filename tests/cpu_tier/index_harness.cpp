// CPU bounds harness of the split-decode kernel's index arithmetic
// (paper_2609_20888_amd/csrc/eta_index.h, the functions the kernels call), built
// with the address and undefined-behaviour sanitizers.  Every array is a heap
// allocation of exactly the size the kernel's buffer has, so an index outside it
// is reported by the sanitizer; the checks add the invariants the kernels rely
// on: each union item / 64-token tile is taken by exactly one split, the
// proportional plan gives every group at least one split and no more than W in
// all, and each workgroup below the number used belongs to exactly one group.  Exit status 0 when all hold.
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
  int* first = new int[BG + 1];            // each group's first split, then the total
  for (int x = 0; x < BG; ++x) first[x] = group_splits(work[x], total, W, BG);
  for (int x = 0; x < BG; ++x) CHECK(first[x] >= 1, "group %d has %d splits", x, first[x]);
  first[BG] = exclusive_prefix(first, BG);
  CHECK(first[BG] <= W, "plan uses %d of %d workgroups", first[BG], W);
  std::vector<int> seen(BG, 0);
  for (int me = 0; me < W; ++me) {
    // the kernel's lookup: every group tests whether it owns the workgroup
    int gi = -1, owners = 0;
    for (int x = 0; x < BG; ++x)
      if (owns_split(first[x], first[x + 1] - first[x], me)) {
        gi = x;
        ++owners;
      }
    if (me >= first[BG]) {
      CHECK(owners == 0, "workgroup %d past the plan got group %d", me, gi);
      continue;
    }
    CHECK(owners == 1, "workgroup %d: %d owning groups", me, owners);
    if (gi < 0) continue;
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

// Screening's record loads over heap arrays of exactly B Hkv d n_blk_cap records:
// every lane (cg = lane / 16, qd = lane % 16) of every wavefront (head-dimension
// quarter w) of every tile, on the four-record path (n_blk_cap a multiple of 4,
// >= 4: the four records in the row, aligned) or the one-record path; and the
// largest-norm load (lane = block).
static void check_screen_loads(int BHkv, int D, int64_t ncap) {
  const int64_t total = (int64_t)BHkv * D * ncap;
  float* rec = new float[total];
  float* mx = new float[(int64_t)BHkv * ncap];
  for (int64_t i = 0; i < total; ++i) rec[i] = 0.f;
  const int n_tiles = ncap < 64 ? 1 : (int)((ncap + 63) / 64);
  const bool vec = ncap >= 4 && ncap % 4 == 0;
  const int DQ = D / 4, NK = DQ / 4;
  float sink = 0.f;
  for (int bg = 0; bg < BHkv; ++bg)
    for (int tile = 0; tile < n_tiles; ++tile)
      for (int w = 0; w < 4; ++w)
        for (int lane = 0; lane < 64; ++lane) {
          const int cg = lane >> 4, qd = lane & 15;
          const int64_t jb = (int64_t)tile * 64;
          for (int k = 0; k < NK; ++k) {
            const int64_t row = (int64_t)bg * D + w * DQ + cg + 4 * k;
            CHECK(row < (int64_t)BHkv * D, "row %lld", (long long)row);
            if (vec) {
              const int64_t o = screen_rec4_offset(row, ncap, jb + 4 * qd);
              CHECK(o >= row * ncap && o + 3 < (row + 1) * ncap && o % 4 == 0,
                    "ncap %lld tile %d lane %d: records [%lld, %lld] outside row %lld",
                    (long long)ncap, tile, lane, (long long)o, (long long)o + 3, (long long)row);
              if (jb + 4 * qd < ncap) CHECK(o == row * ncap + jb + 4 * qd, "in-range quad moved");
              for (int e = 0; e < 4; ++e) sink += rec[o + e];
            } else {
              for (int e = 0; e < 4; ++e) {
                const int64_t o = screen_rec1_offset(row, ncap, jb + 4 * qd + e);
                CHECK(o >= row * ncap && o < (row + 1) * ncap, "record %lld outside row", (long long)o);
                if (jb + 4 * qd + e < ncap) CHECK(o == row * ncap + jb + 4 * qd + e, "in-range record moved");
                sink += rec[o];
              }
            }
          }
          int64_t jm = jb + lane;
          jm = jm < ncap ? jm : ncap - 1;
          sink += mx[bg * ncap + jm] = 0.f;
        }
  (void)sink;
  delete[] mx;
  delete[] rec;
}

// The predictor's passes: every row of [0, J) taken by exactly one (pass,
// thread, e), four consecutive rows per thread and pass (J a multiple of 4).
static void check_pred_rows(int J) {
  std::vector<int> seen(J, 0);
  const int passes = (J + 1023) / 1024;
  for (int p = 0; p < passes + 1; ++p)
    for (int t = 0; t < 256; ++t) {
      const int j = p * 1024 + 4 * t;
      const int jc = pred_row4(p, t, J);
      CHECK(jc >= 0 && jc + 3 < J, "J %d pass %d thread %d -> rows %d..%d", J, p, t, jc, jc + 3);
      if (j < J) {
        CHECK(jc == j, "in-range rows moved");
        for (int e = 0; e < 4; ++e) ++seen[j + e];
      }
    }
  for (int j = 0; j < J; ++j) CHECK(seen[j] == 1, "J %d row %d taken %d times", J, j, seen[j]);
}

// The plan's walk over groups x0, x0 + step, ... (x = sequence * hkv + kv head):
// the stepper's (q, rm) equal x / hkv and x % hkv at every step.
static void check_stepper(unsigned hkv, unsigned step, unsigned steps) {
  for (unsigned x0 = 0; x0 < step; ++x0) {
    GroupStepper gs(x0, step, hkv);
    for (unsigned r = 0; r < steps; ++r) {
      const unsigned x = x0 + r * step;
      CHECK(gs.q == x / hkv && gs.rm == x % hkv, "hkv %u step %u group %u: (%u, %u)", hkv, step,
            x, gs.q, gs.rm);
      gs.next();
    }
  }
}

int main() {
  std::mt19937_64 rng(12345);
  // the split kernel walks groups tid + 256 r, r < 4 (up to 1024 groups)
  for (unsigned hkv = 1; hkv <= 40; ++hkv)
    for (unsigned step : {1u, 7u, 64u, 256u}) check_stepper(hkv, step, 6);
  check_stepper(1024, 256, 4);
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
  // screening record loads: one block, below a tile, a partial last tile, whole
  // tiles, the largest table; both load paths; both head dimensions
  for (int64_t ncap : {1, 3, 4, 5, 63, 64, 65, 68, 130, 2048, 2051})
    for (int D : {64, 128}) check_screen_loads(2, D, ncap);
  check_screen_loads(1, 128, 131072);
  for (int J : {4, 64, 1020, 1024, 1028, 2048, 3072, 8192, 262144}) check_pred_rows(J);
  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("index harness: all checks passed\n");
  return 0;
}
