// Host-only driver for tests/test_planner_sanitized.py: builds plans for the
// benchmark sets and for edge-case lists (empty, 1x1, ragged, very large
// or very tall matrices, fp32 and adaptive plans) so that the planner runs
// under AddressSanitizer and UndefinedBehaviorSanitizer. Tensor addresses
// are never dereferenced by the planner; they only need to be distinct.
#include "plan.h"
#include <cstdio>
#include <vector>
#include <string>
using namespace lm;
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
  return st == Status::kOk ? 0 : 1;
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
  printf("failures %d\n", bad);
  return bad;
}
