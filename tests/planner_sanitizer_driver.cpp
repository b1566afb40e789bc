// Host-only driver for tests/test_planner_sanitized.py: builds plans for the
// benchmark sets and for edge-case lists (empty, 1x1, ragged, very large
// or very tall matrices, fp32 and adaptive plans) so that the planner runs
// under AddressSanitizer and UndefinedBehaviorSanitizer. Tensor addresses
// are never dereferenced by the planner; they only need to be distinct.
#include "plan.h"
#include <algorithm>
#include <cstdio>
#include <map>
#include <tuple>
#include <vector>
#include <string>
using namespace lm;

// Invariants of a plan's Newton-Schulz work lists: every XCD split is a
// partition of its list; the Gram and polynomial lists hold each
// lower-triangle tile of each matrix of their precision exactly once; the
// apply's 256-tile (or fp32) list and its small-tile list together cover each
// matrix's padded output exactly once. Returns the number of violations.
static int check_plan(const Plan& p) {
  int bad = 0;
  auto fail = [&](const char* what, int pr, int mat) {
    ++bad;
    printf("plan invariant violated: %s (precision %d, matrix %d)\n", what, pr, mat);
  };
  auto check_split = [&](const std::vector<GemmTask>& t, const XcdSplit& sp, const char* what, int pr) {
    int32_t pos = 0, mx = 0;
    for (int x = 0; x < p.chip.xcds; ++x) {
      if (sp.start[x] != pos || sp.count[x] < 0) return fail(what, pr, -1);
      pos += sp.count[x];
      mx = std::max(mx, sp.count[x]);
    }
    if (pos != int32_t(t.size()) || mx != sp.max_count) fail(what, pr, -1);
  };
  const int nm = int(p.mats.size());
  for (int pr = 0; pr < 2; ++pr) {
    check_split(p.gram[pr], p.gram_split[pr], "gram split", pr);
    check_split(p.poly[pr], p.poly_split[pr], "poly split", pr);
    check_split(p.apply[pr], p.apply_split[pr], "apply split", pr);
    check_split(p.apply_tail[pr], p.apply_tail_split[pr], "small-tile split", pr);
    for (int k = 0; k < 2; ++k) {
      const std::vector<GemmTask>& list = k == 0 ? p.gram[pr] : p.poly[pr];
      const int tile = p.tile[pr][k];
      std::map<std::tuple<int, int, int>, int> seen;
      for (const GemmTask& t : list) {
        if (t.mat < 0 || t.mat >= nm || p.mats[t.mat].fp32 != pr || t.tm < t.tn) {
          fail("symmetric task outside the lower triangle of its precision", pr, t.mat);
          continue;
        }
        seen[std::make_tuple(int(t.mat), int(t.tm), int(t.tn))] += 1;
      }
      size_t expect = 0;
      for (int m = 0; m < nm; ++m) {
        if (p.mats[m].fp32 != pr) continue;
        if (p.mats[m].s_pad % tile) fail("short side not a multiple of the tile", pr, m);
        const int ts = p.mats[m].s_pad / tile;
        for (int tm = 0; tm < ts; ++tm)
          for (int tn = 0; tn <= tm; ++tn) {
            ++expect;
            auto it = seen.find(std::make_tuple(m, tm, tn));
            if (it == seen.end() || it->second != 1) fail(k == 0 ? "Gram tile not once" : "polynomial tile not once", pr, m);
          }
      }
      if (seen.size() != expect) fail("symmetric list holds extra tiles", pr, -1);
    }
    // apply coverage in units of 64 x 64
    const int ta = p.tile[pr][2], tt = p.tail_tile[pr];
    std::vector<std::vector<int>> cover(static_cast<size_t>(nm));
    for (int m = 0; m < nm; ++m)
      if (p.mats[m].fp32 == pr) cover[size_t(m)].assign(size_t(p.mats[m].s_pad / 64) * size_t(p.mats[m].l_pad / 64), 0);
    auto mark = [&](const GemmTask& t, int tile) {
      if (t.mat < 0 || t.mat >= nm || p.mats[t.mat].fp32 != pr) return fail("apply task of another precision", pr, t.mat);
      const MuonMat& mm = p.mats[t.mat];
      const int64_t r0 = int64_t(t.tm) * tile, c0 = int64_t(t.tn) * tile;
      if (r0 < 0 || c0 < 0 || r0 + tile > mm.s_pad || c0 + tile > mm.l_pad) return fail("apply tile outside the matrix", pr, t.mat);
      const int cols = mm.l_pad / 64;
      for (int64_t r = r0 / 64; r < (r0 + tile) / 64; ++r)
        for (int64_t c = c0 / 64; c < (c0 + tile) / 64; ++c) cover[size_t(t.mat)][size_t(r * cols + c)] += 1;
    };
    for (const GemmTask& t : p.apply[pr]) mark(t, ta);
    for (const GemmTask& t : p.apply_tail[pr]) mark(t, tt);
    for (int m = 0; m < nm; ++m)
      for (int v : cover[size_t(m)])
        if (v != 1) {
          fail("apply output not covered exactly once", pr, m);
          break;
        }
  }
  return bad;
}

static int run(const std::vector<std::pair<long, long>>& shapes, StepKind kind, bool fp32,
               int flags = 0, ChipShape chip = ChipShape()) {
  std::vector<TensorIn> x(shapes.size());
  for (size_t i = 0; i < shapes.size(); ++i) {
    x[i] = TensorIn{};
    x[i].w = reinterpret_cast<float*>(0x100000000ull + i * 0x1000000000ull);
    x[i].g = reinterpret_cast<const float*>(0x100000000ull + i * 0x1000000000ull + 0x400000000ull);
    x[i].m = reinterpret_cast<float*>(0x100000000ull + i * 0x1000000000ull + 0x800000000ull);
    x[i].rows = shapes[i].first;
    x[i].cols = shapes[i].second;
    x[i].flags = uint32_t(flags);
  }
  Plan p;
  std::string err;
  NsPrecision prec;
  prec.all_fp32 = fp32;
  Status st = build_plan(x.data(), int(x.size()), kind, prec, false, chip, &p, &err);
  size_t ntask = 0;
  for (int pr = 0; pr < 2; ++pr)
    ntask += p.gram[pr].size() + p.poly[pr].size() + p.apply[pr].size() + p.apply_tail[pr].size();
  printf("status %d tasks %zu ws %zu %s\n", int(st), ntask, size_t(p.ws_bytes), err.c_str());
  if (st != Status::kOk) return 1;
  return check_plan(p) ? 1 : 0;
}

// Random lists of matrices (fixed seed): shapes from 1 x 1 to 3000 x 3000,
// some 1-D or Lion-only, with each step kind, both precisions and three
// device shapes.
static int random_lists() {
  uint64_t state = 0x9E3779B97F4A7C15ull;
  auto next = [&](uint64_t n) {
    state = state * 6364136223846793005ull + 1442695040888963407ull;
    return (state >> 33) % n;
  };
  ChipShape chips[3];
  chips[1].cus = 32;
  chips[1].xcds = 1;
  chips[2].cus = 64;
  chips[2].xcds = 2;
  int bad = 0;
  for (int it = 0; it < 60; ++it) {
    std::vector<std::pair<long, long>> shapes;
    const int n = 1 + int(next(40));
    for (int i = 0; i < n; ++i) {
      const long r = next(5) == 0 ? 1 : 1 + long(next(3000));
      const long c = 1 + long(next(3000));
      shapes.push_back({r, c});
    }
    const StepKind kind = it % 3 == 0 ? StepKind::kAdaptive : StepKind::kMuon;
    bad += run(shapes, kind, it % 4 == 1, it % 7 == 0 ? int(kFlagLionOnly) : 0, chips[it % 3]);
  }
  return bad;
}
int main() {
  int bad = 0;
  std::vector<std::pair<long, long>> s124, s720;
  for (int l = 0; l < 12; ++l) {
    s124.push_back({768, 2304});
    s124.push_back({768, 768});
    s124.push_back({768, 3072});
    s124.push_back({3072, 768});
  }
  for (int l = 0; l < 36; ++l) {
    s720.push_back({1280, 3840});
    s720.push_back({1280, 1280});
    s720.push_back({1280, 5120});
    s720.push_back({5120, 1280});
  }
  const std::vector<std::pair<long, long>> edge = {{1, 1}, {2, 2}, {3, 7}, {0, 5}, {65, 65}, {129, 4097}};
  bad += run(s124, StepKind::kMuon, false);
  bad += run(s124, StepKind::kMuon, true);
  bad += run(s124, StepKind::kAdaptive, false);
  bad += run(s720, StepKind::kMuon, false);
  bad += run(s720, StepKind::kAdaptive, false);
  bad += run({{700, 5000}, {700, 5000}, {700, 5000}, {700, 5000}, {3000, 300}}, StepKind::kMuon, false);
  bad += run(edge, StepKind::kMuon, false);
  bad += run(edge, StepKind::kAdaptive, true);
  bad += run(edge, StepKind::kLion, false);
  bad += run({{8192, 8192}}, StepKind::kMuon, false);
  bad += run({{100000, 64}}, StepKind::kAdaptive, false);
  bad += run({}, StepKind::kMuon, false);
  // partitioned devices: one XCD of 32 CUs, two XCDs of 64
  ChipShape one_xcd;
  one_xcd.cus = 32;
  one_xcd.xcds = 1;
  ChipShape two_xcd;
  two_xcd.cus = 64;
  two_xcd.xcds = 2;
  bad += run(s124, StepKind::kMuon, false, 0, one_xcd);
  bad += run(s720, StepKind::kAdaptive, false, 0, two_xcd);
  bad += run(edge, StepKind::kMuon, true, 0, one_xcd);
  // a last round of 8 and of 48 256-tiles (64-tile and 128-tile small rounds)
  bad += run({{700, 5000}, {700, 5000}, {700, 5000}, {700, 5000}, {300, 3000}}, StepKind::kMuon, false);
  bad += random_lists();
  printf("failures %d\n", bad);
  return bad;
}
