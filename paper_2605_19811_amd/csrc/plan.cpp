// Host planner of the LionMuon step (see plan.h). No HIP calls.
#include "plan.h"

#include <algorithm>
#include <cstdint>
#include <cmath>
#include <map>
#include <numeric>
#include <utility>

namespace lm {

namespace {

int64_t round_up(int64_t x, int64_t q) { return (x + q - 1) / q * q; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bool finite_nonneg(double v) { return std::isfinite(v) && v >= 0.0; }

// Lower-triangle output tiles of one matrix's s x s product, each with its
// inner dimension as cost.
void sym_tiles(const MuonMat& mm, int32_t mi, int tile, int64_t inner,
               std::vector<GemmTask>* tasks, std::vector<int64_t>* cost) {
  const int ts = int(mm.s_pad / tile);
  for (int tm = 0; tm < ts; ++tm) {
    for (int tn = 0; tn <= tm; ++tn) {
      tasks->push_back({mi, int16_t(tm), int16_t(tn)});
      cost->push_back(inner);
    }
  }
}

// Estimated duration of a one-tile-per-workgroup symmetric product launch,
// in quarters of a 256-tile K stage: each XCD's tiles, longest first, go to
// whichever of its workgroup slots frees first (as the dispatcher hands out
// a full grid), one slot per CU for 256-tiles and two for 128-tiles (LDS).
// Per tile: a K stage of a 256-tile takes 4 units; two 128-tiles sharing a
// CU take 3 units each per stage (a quarter of the work at two thirds of the
// 256-tile rate, measured on the benchmark sets); set-up and epilogue cost
// 7 and 5 units.
int64_t sym_launch_estimate(const std::vector<GemmTask>& tasks, const std::vector<int64_t>& inner,
                            const XcdSplit& split, int tile, ChipShape chip) {
  const bool big = tile == kTileBig;
  const int slots = std::max(1, chip.cus / chip.xcds) * (big ? 1 : 2);
  const int64_t per_stage = big ? 4 : 3, fixed = big ? 7 : 5;
  const int64_t kbk = 64;
  int64_t worst = 0;
  std::vector<int64_t> free_at(size_t(slots), 0);
  for (int x = 0; x < chip.xcds; ++x) {
    std::fill(free_at.begin(), free_at.end(), 0);
    for (int32_t i = split.start[x]; i < split.start[x] + split.count[x]; ++i) {
      auto it = std::min_element(free_at.begin(), free_at.end());
      *it += fixed + per_stage * ((inner[size_t(i)] + kbk - 1) / kbk);
    }
    worst = std::max(worst, *std::max_element(free_at.begin(), free_at.end()));
  }
  return worst;
}

// Tile edge for a bf16 symmetric product (Gram if `gram`, else the
// polynomial): 256 unless 128-tiles are estimated to finish sooner (too few
// 256-tiles to fill the chip, or too uneven a last round).
int32_t pick_sym_tile(const std::vector<MuonMat>& mats, bool gram, ChipShape chip) {
  int64_t est[2] = {0, 0};
  const int32_t sizes[2] = {kTileBig, kTileSmall};
  for (int k = 0; k < 2; ++k) {
    std::vector<GemmTask> tasks;
    std::vector<int64_t> cost;
    for (int32_t mi = 0; mi < int32_t(mats.size()); ++mi) {
      const MuonMat& mm = mats[size_t(mi)];
      if (mm.fp32) continue;
      sym_tiles(mm, mi, sizes[k], gram ? mm.l_pad : mm.s_pad, &tasks, &cost);
    }
    if (tasks.empty()) return kTileBig;
    XcdSplit split;
    split_by_xcd(&tasks, cost, chip.xcds, &split);
    std::vector<int64_t> inner(tasks.size());
    for (size_t i = 0; i < tasks.size(); ++i) {
      const MuonMat& mm = mats[size_t(tasks[i].mat)];
      inner[i] = gram ? mm.l_pad : mm.s_pad;
    }
    est[k] = sym_launch_estimate(tasks, inner, split, sizes[k], chip);
  }
  return est[0] <= est[1] ? kTileBig : kTileSmall;
}

}  // namespace

int sr_tall_bucket(int64_t s) {
  const int64_t n = (s + 255) / 256;
  for (int b : kSrTallBuckets)
    if (n <= b) return b;
  return 0;
}

int sr_wide_bucket(int64_t s) {
  if (s <= 1024) {
    const int64_t n = (s + 127) / 128;
    for (int b : kSrWideBuckets)
      if (n <= b) return b;
  }
  const int64_t n = (s + 255) / 256;
  for (int b : kSrNarrowBuckets)
    if (n <= b) return b;
  return 0;
}

bool is_muon_step(int64_t t, int32_t P) { return P >= 1 && t % P == 0; }

uint32_t align_class(const TensorIn& x) {
  const uintptr_t vbits = (x.flags & kFlagAdamW) ? reinterpret_cast<uintptr_t>(x.v) : 0;
  return ((reinterpret_cast<uintptr_t>(x.w) | reinterpret_cast<uintptr_t>(x.g) |
           reinterpret_cast<uintptr_t>(x.m) | vbits) & 15u) == 0 ? 1u : 0u;
}

bool is_matrix(const TensorIn& x) {
  return x.rows > 1 && x.cols > 1 && !(x.flags & (kFlagLionOnly | kFlagAdamW));
}

Status validate_scalars(int64_t t, int32_t P, double beta1, double beta2, double wd,
                        double lr_muon, double lr_lion, std::string* err) {
  if (t < 0) { *err = "t must be >= 0"; return Status::kInvalid; }
  if (P < 0) { *err = "P must be >= 0 (0 encodes P = infinity)"; return Status::kInvalid; }
  if (!(beta1 >= 0.0 && beta1 < 1.0)) { *err = "beta1 must lie in [0, 1)"; return Status::kInvalid; }
  if (!(beta2 >= 0.0 && beta2 < 1.0)) { *err = "beta2 must lie in [0, 1)"; return Status::kInvalid; }
  if (!finite_nonneg(wd)) { *err = "wd must be finite and >= 0"; return Status::kInvalid; }
  if (!finite_nonneg(lr_muon) || !finite_nonneg(lr_lion)) {
    *err = "learning rates must be finite and >= 0";
    return Status::kInvalid;
  }
  return Status::kOk;
}

Status validate_tensors(const TensorIn* x, int32_t n, std::string* err) {
  if (n < 0) { *err = "n_tensors must be >= 0"; return Status::kInvalid; }
  if (n > 0 && x == nullptr) { *err = "null tensor list"; return Status::kInvalid; }
  // [begin, end) byte ranges: writable (W, M) and read-only (G).
  std::vector<std::pair<uintptr_t, uintptr_t>> wr, rd;
  wr.reserve(2 * size_t(n));
  rd.reserve(size_t(n));
  for (int32_t i = 0; i < n; ++i) {
    const TensorIn& t = x[i];
    if (t.rows < 0 || t.cols < 0) {
      *err = "tensor " + std::to_string(i) + ": negative dimension";
      return Status::kInvalid;
    }
    if (t.reserved != 0 || (t.flags & ~(kFlagLionOnly | kFlagAdamW)) ||
        t.flags == (kFlagLionOnly | kFlagAdamW)) {
      *err = "tensor " + std::to_string(i) + ": unknown or conflicting flag bits, or reserved field set";
      return Status::kInvalid;
    }
    if (t.rows == 0 || t.cols == 0) continue;
    if (t.rows > (int64_t(1) << 40) / t.cols) {
      *err = "tensor " + std::to_string(i) + ": too many elements";
      return Status::kInvalid;
    }
    const bool adamw = (t.flags & kFlagAdamW) != 0;
    if (!t.w || !t.g || !t.m || (adamw && !t.v)) {
      *err = "tensor " + std::to_string(i) +
             ": null params, grads, momentum or (AdamW) second-moment pointer";
      return Status::kInvalid;
    }
    auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; };
    if (!al(t.w) || !al(t.g) || !al(t.m) || (adamw && !al(t.v))) {
      *err = "tensor " + std::to_string(i) + ": pointers must be 4-byte aligned fp32";
      return Status::kInvalid;
    }
    const uintptr_t bytes = uintptr_t(t.rows * t.cols) * 4u;
    wr.push_back({reinterpret_cast<uintptr_t>(t.w), reinterpret_cast<uintptr_t>(t.w) + bytes});
    wr.push_back({reinterpret_cast<uintptr_t>(t.m), reinterpret_cast<uintptr_t>(t.m) + bytes});
    if (adamw)
      wr.push_back({reinterpret_cast<uintptr_t>(t.v), reinterpret_cast<uintptr_t>(t.v) + bytes});
    rd.push_back({reinterpret_cast<uintptr_t>(t.g), reinterpret_cast<uintptr_t>(t.g) + bytes});
  }
  std::sort(wr.begin(), wr.end());
  for (size_t i = 1; i < wr.size(); ++i) {
    if (wr[i].first < wr[i - 1].second) {
      *err = "params / momentum buffers overlap";
      return Status::kInvalid;
    }
  }
  // every read-only range must be disjoint from every writable range
  for (const auto& r : rd) {
    auto it = std::upper_bound(wr.begin(), wr.end(), std::make_pair(r.first, ~uintptr_t(0)));
    if (it != wr.end() && it->first < r.second) {
      *err = "a gradient buffer overlaps params or momentum";
      return Status::kInvalid;
    }
    if (it != wr.begin() && std::prev(it)->second > r.first) {
      *err = "a gradient buffer overlaps params or momentum";
      return Status::kInvalid;
    }
  }
  return Status::kOk;
}

void split_by_xcd(std::vector<GemmTask>* tasks, const std::vector<int64_t>& cost, int xcds,
                  XcdSplit* split) {
  const size_t n = tasks->size();
  const int64_t total = std::accumulate(cost.begin(), cost.end(), int64_t(0));
  *split = XcdSplit{};
  // cut points: segment x ends once the running cost reaches (x+1)/xcds of total
  std::vector<size_t> cut(size_t(xcds) + 1, 0);
  size_t pos = 0;
  int64_t run = 0;
  for (int x = 0; x < xcds; ++x) {
    cut[x] = pos;
    const int64_t goal = (total * (x + 1) + xcds - 1) / xcds;
    while (pos < n && (run < goal || x == xcds - 1)) {
      run += cost[pos];
      ++pos;
    }
  }
  cut[xcds] = n;
  std::vector<GemmTask> out;
  out.reserve(n);
  split->max_count = 0;
  for (int x = 0; x < xcds; ++x) {
    std::vector<size_t> idx(cut[x + 1] - cut[x]);
    std::iota(idx.begin(), idx.end(), cut[x]);
    std::stable_sort(idx.begin(), idx.end(),
                     [&](size_t a, size_t b) { return cost[a] > cost[b]; });
    split->start[x] = int32_t(out.size());
    split->count[x] = int32_t(idx.size());
    split->max_count = std::max(split->max_count, split->count[x]);
    for (size_t i : idx) out.push_back((*tasks)[i]);
  }
  tasks->swap(out);
}

Status build_plan(const TensorIn* x, int32_t n, StepKind kind, NsPrecision prec,
                  bool kappa_rms02, ChipShape chip, Plan* p, std::string* err) {
  *p = Plan();
  if (chip.xcds < 1 || chip.xcds > kMaxXcds || chip.cus < chip.xcds) {
    *err = "unsupported device shape (compute units / XCDs)";
    return Status::kUnsupported;
  }
  p->chip = chip;
  const bool muon_step = kind != StepKind::kLion;
  p->muon_step = muon_step;
  p->adaptive = kind == StepKind::kAdaptive;
  p->lion_block_start.push_back(0);
  p->prep_start.push_back(0);
  p->rd_start.push_back(0);
  p->tensor_mat.assign(size_t(n > 0 ? n : 0), -1);
  std::map<std::pair<int64_t, int64_t>, int> classes;
  int64_t ns_off = 0;   // bytes
  for (int32_t i = 0; i < n; ++i) {
    const TensorIn& t = x[i];
    if (t.rows == 0 || t.cols == 0) continue;
    ++p->n_tensors;
    const bool adamw = (t.flags & kFlagAdamW) != 0;
    const bool vec_ok = align_class(t) != 0;
    const bool candidate = muon_step && is_matrix(t);
    if (!candidate || p->adaptive) {
      LionTensor lt{};
      lt.tensor = i;
      lt.numel = t.rows * t.cols;
      lt.vec_ok = vec_ok ? 1 : 0;
      lt.adamw = adamw ? 1 : 0;
      lt.gate = candidate ? int32_t(p->mats.size()) : -1;
      const int64_t blocks = (lt.numel + kLionBlockElems - 1) / kLionBlockElems;
      if (int64_t(p->lion_block_start.back()) + blocks > INT32_MAX) {
        *err = "too many elements on the Lion branch";
        return Status::kUnsupported;
      }
      p->lion.push_back(lt);
      p->lion_block_start.push_back(p->lion_block_start.back() + int32_t(blocks));
      if (adamw) {
        p->adamw_elements += lt.numel;
        ++p->n_adamw;
      } else if (!candidate) {
        p->lion_elements += lt.numel;
      }
      if (!candidate) continue;
    }
    MuonMat mm{};
    mm.rows = t.rows;
    mm.cols = t.cols;
    mm.transposed = t.rows > t.cols ? 1 : 0;
    const int64_t s = std::min(t.rows, t.cols), l = std::max(t.rows, t.cols);
    if (s > kMaxShortSide || round_up(s, kTileBig) * round_up(l, kTileBig) > kMaxMatrixElems) {
      *err = "tensor " + std::to_string(i) + ": matrix too large for the Newton-Schulz kernels";
      return Status::kUnsupported;
    }
    mm.s = int32_t(s);
    mm.l = int32_t(l);
    mm.fp32 = prec.fp32_for(s) ? 1 : 0;
    const int64_t pad = mm.fp32 ? kTileSmall : kTileBig;
    mm.s_pad = int32_t(round_up(s, pad));
    mm.l_pad = int32_t(round_up(l, pad));
    // vector path on the original rows needs 16-byte aligned rows
    mm.vec_ok = (vec_ok && (t.cols % 4) == 0) ? 1 : 0;
    const int64_t eb = mm.fp32 ? 4 : 2;
    const int64_t sl = int64_t(mm.s_pad) * mm.l_pad * eb, ss = int64_t(mm.s_pad) * mm.s_pad * eb;
    mm.off_x[0] = ns_off;  ns_off += sl;
    mm.off_x[1] = ns_off;  ns_off += sl;
    mm.off_a = ns_off;     ns_off += ss;
    mm.off_b = ns_off;     ns_off += ss;
    const int64_t rows_pad = mm.transposed ? mm.l_pad : mm.s_pad;
    const int64_t cols_pad = mm.transposed ? mm.s_pad : mm.l_pad;
    // preparation tiles: 64 x 128 (64 x 64 for fp32 X) through the LDS
    // transpose for a tall matrix; kPrepElems-element strips of whole 1 KB
    // (or 512 B) row pieces for a wide one
    const int64_t tile_c = mm.transposed ? (mm.fp32 ? kPrepTile : kPrepTallCols)
                                         : (cols_pad % 256 == 0 ? 256 : 128);
    const int64_t tile_r = mm.transposed ? kPrepTile : kPrepElems / tile_c;
    mm.prep_tiles_n = int32_t(cols_pad / tile_c);
    mm.prep_count = int32_t((rows_pad / tile_r) * (cols_pad / tile_c));
    mm.prep_first = p->prep_start.back();
    if (int64_t(mm.prep_first) + mm.prep_count > INT32_MAX) {
      *err = "too many elements on the Muon branch";
      return Status::kUnsupported;
    }
    mm.kappa = kappa_rms02 ? float(0.2 * std::sqrt(double(l))) : 1.0f;
    mm.tensor = i;
    mm.tall = t.rows >= t.cols ? 1 : 0;
    const int bucket = mm.tall ? sr_tall_bucket(s) : sr_wide_bucket(s);
    if (mm.vec_ok && s <= kSrMaxRegSide && bucket > 0) {
      mm.sr_kind = mm.tall ? kSrTall : (s <= 1024 ? kSrWide : kSrWideNarrow);
      mm.sr_bucket = bucket;
      mm.sr_blocks = int32_t((l + (mm.tall ? kSrTallRows : kSrWideCols) - 1) /
                             (mm.tall ? kSrTallRows : kSrWideCols));
    } else {
      mm.sr_kind = kSrGeneric;
      mm.sr_bucket = 0;
      mm.sr_blocks = int32_t((l + kSrBlock - 1) / kSrBlock);
    }
    if (p->adaptive) {
      const int64_t chunks = (s + kSrChunk - 1) / kSrChunk;
      if (int64_t(p->sr_tab.size()) + mm.sr_blocks > INT32_MAX ||
          int64_t(p->rd_start.back()) + chunks > INT32_MAX) {
        *err = "too many elements for the stable-rank passes";
        return Status::kUnsupported;
      }
      for (int32_t b = 0; b < mm.sr_blocks; ++b) p->sr_tab.push_back({int32_t(p->mats.size()), b});
      p->rd_start.push_back(p->rd_start.back() + int32_t(chunks));
      p->candidate_elements += t.rows * t.cols;
    }
    p->tensor_mat[size_t(i)] = int32_t(p->mats.size());
    p->prep_start.push_back(mm.prep_first + mm.prep_count);
    p->mats.push_back(mm);
    p->muon_elements += t.rows * t.cols;
    classes[{s, l}] += 1;
  }
  p->n_shape_classes = int32_t(classes.size());

  // GEMM work lists in canonical order (matrix, then tiles), cost = inner
  // dimension, one list per Newton-Schulz precision.
  // bf16: apply on 256-tiles; Gram and polynomial (s x s outputs, lower
  // triangle) each on whichever of 256- and 128-tiles the launch estimate
  // below favours. fp32: 128-tiles, or 64-tiles for a product whose
  // 128-tiles would not give every CU one.
  if (p->mats.size() > 0) {
    p->tile[0][0] = pick_sym_tile(p->mats, true, chip);
    p->tile[0][1] = pick_sym_tile(p->mats, false, chip);
  }
  p->tile[0][2] = kTileBig;
  {
    int64_t sym = 0, app = 0;
    for (const MuonMat& mm : p->mats) {
      if (!mm.fp32) continue;
      const int64_t ts = mm.s_pad / kTileSmall;
      sym += ts * (ts + 1) / 2;
      app += ts * (mm.l_pad / kTileSmall);
    }
    p->tile[1][0] = p->tile[1][1] = sym < chip.cus ? kTileTiny : kTileSmall;
    p->tile[1][2] = app < chip.cus ? kTileTiny : kTileSmall;
  }
  for (int pr = 0; pr < 2; ++pr) {
    std::vector<int64_t> cg, cp, ca;
    const int t_app = p->tile[pr][2];
    for (int32_t mi = 0; mi < int32_t(p->mats.size()); ++mi) {
      const MuonMat& mm = p->mats[mi];
      if (mm.fp32 != pr) continue;
      sym_tiles(mm, mi, p->tile[pr][0], mm.l_pad, &p->gram[pr], &cg);
      sym_tiles(mm, mi, p->tile[pr][1], mm.s_pad, &p->poly[pr], &cp);
      const int ts_a = mm.s_pad / t_app, tl_a = mm.l_pad / t_app;
      for (int tn = 0; tn < tl_a; ++tn) {
        for (int tm = 0; tm < ts_a; ++tm) {
          p->apply[pr].push_back({mi, int16_t(tm), int16_t(tn)});
          ca.push_back(mm.s_pad);
        }
      }
    }
    // A nearly empty last round of 256-tiles runs as smaller tiles instead:
    // 64-tiles (16 per 256-tile) when they fit one round of the CUs (and
    // their indices fit the task fields), else 128-tiles (4 per 256-tile).
    std::vector<int64_t> ct;
    if (t_app == kTileBig) {
      const size_t cus = size_t(chip.cus);
      const size_t n = p->apply[pr].size(), rem = n % cus;
      if (n > rem && rem > 0 && 2 * rem <= cus) {
        int64_t max_tl = 0;
        for (size_t i = n - rem; i < n; ++i) max_tl = std::max<int64_t>(max_tl, p->apply[pr][i].tn);
        const int split = (16 * rem <= cus && 4 * (max_tl + 1) <= INT16_MAX) ? 4 : 2;
        p->tail_tile[pr] = kTileBig / split;
        for (size_t i = n - rem; i < n; ++i) {
          const GemmTask t = p->apply[pr][i];
          for (int a = 0; a < split; ++a)
            for (int b = 0; b < split; ++b) {
              p->apply_tail[pr].push_back({t.mat, int16_t(split * t.tm + a), int16_t(split * t.tn + b)});
              ct.push_back(ca[i]);
            }
        }
        p->apply[pr].resize(n - rem);
        ca.resize(n - rem);
      }
    }
    split_by_xcd(&p->gram[pr], cg, chip.xcds, &p->gram_split[pr]);
    split_by_xcd(&p->poly[pr], cp, chip.xcds, &p->poly_split[pr]);
    split_by_xcd(&p->apply[pr], ca, chip.xcds, &p->apply_split[pr]);
    split_by_xcd(&p->apply_tail[pr], ct, chip.xcds, &p->apply_tail_split[pr]);
  }

  size_t off = align256(size_t(ns_off));
  p->ws_partials_off = off;
  off = align256(off + size_t(p->prep_start.back()) * sizeof(float));
  p->ws_rscale_off = off;
  off = align256(off + p->mats.size() * sizeof(float));
  if (p->adaptive) {
    // pass workgroups grouped by (kind, bucket), matrices in list order
    std::stable_sort(p->sr_tab.begin(), p->sr_tab.end(), [&](const SrBlock& a, const SrBlock& b) {
      const MuonMat &x = p->mats[size_t(a.mat)], &y = p->mats[size_t(b.mat)];
      return std::make_pair(x.sr_kind, x.sr_bucket) < std::make_pair(y.sr_kind, y.sr_bucket);
    });
    for (size_t i = 0; i < p->sr_tab.size(); ++i) {
      const MuonMat& mm = p->mats[size_t(p->sr_tab[i].mat)];
      if (p->sr_classes.empty() || p->sr_classes.back().kind != mm.sr_kind ||
          p->sr_classes.back().bucket != mm.sr_bucket)
        p->sr_classes.push_back({mm.sr_kind, mm.sr_bucket, int32_t(i), 0});
      ++p->sr_classes.back().count;
    }
    p->ws_decide_off = off;
    off = align256(off + p->mats.size() * sizeof(int32_t));
    for (MuonMat& mm : p->mats) {
      // sized for the generic path's block count (the largest of the three
      // paths), so the workspace a list needs does not depend on which path
      // its alignment selects
      const int64_t nb = std::max<int64_t>(mm.sr_blocks, (mm.l + kSrBlock - 1) / kSrBlock);
      const int64_t s = mm.s;
      mm.off_sr = int64_t(off);
      off = align256(off + size_t(s + nb * s + 2 * nb + (s + kSrChunk - 1) / kSrChunk) *
                               sizeof(double));
    }
  }
  p->ws_bytes = p->mats.empty() ? 0 : off;
  return Status::kOk;
}

double ns_flops_symmetric(const Plan& p, int k) {
  double f = 0.0;
  for (const MuonMat& m : p.mats) {
    const double s = m.s, l = m.l;
    f += s * (s + 1.0) * l + s * s * (s + 1.0) + 2.0 * s * s * l;
  }
  return f * k;
}

double ns_flops_dense(const Plan& p, int k) {
  double f = 0.0;
  for (const MuonMat& m : p.mats) {
    const double s = m.s, l = m.l;
    f += 4.0 * s * s * l + 2.0 * s * s * s;
  }
  return f * k;
}

}  // namespace lm
