// Host planner of the LionMuon step: argument validation, the per-tensor
// Lion / Muon decision of Algorithm 1, Newton-Schulz shape classes and
// transpose flags, workspace layout and the GEMM tile work lists.
// Pure C++: no HIP call, so it runs (and is tested) on a host without a GPU.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "lm_desc.h"

namespace lm {

struct TensorIn {
  float* w;
  const float* g;
  float* m;
  float* v;          // AdamW second moment (flag 2), else unused
  int64_t rows, cols;
  uint32_t flags;
  uint32_t reserved;
};

constexpr uint32_t kFlagLionOnly = 1u, kFlagAdamW = 2u;

enum class Status : int { kOk = 0, kInvalid = 1, kUnsupported = 2, kNoMemory = 3,
                          kWorkspaceTooSmall = 4, kHip = 5 };

// Largest Muon matrix the kernels accept: short side and element count.
constexpr int64_t kMaxShortSide = 16384;
constexpr int64_t kMaxMatrixElems = int64_t(1) << 30;

// Muon branch of Algorithm 1: period P >= 1 and t mod P == 0 (P = 0 is P = inf).
bool is_muon_step(int64_t t, int32_t P);

// A tensor takes the Muon branch on Muon steps iff it is a real matrix
// (rows > 1 and cols > 1) and flagged neither Lion-only nor AdamW.
bool is_matrix(const TensorIn& x);

// Newton-Schulz precision of one matrix: bf16 MFMA unless fp32 is asked for
// or the short side is below bf16_min_side (where bf16 rounding of the s x s
// products no longer meets the bf16 error budget and fp32 costs little).
struct NsPrecision {
  bool all_fp32 = false;
  int32_t bf16_min_side = 64;
  bool fp32_for(int64_t short_side) const { return all_fp32 || short_side < bf16_min_side; }
};

// What a step does with the Muon candidates (matrices per is_matrix):
// the Lion branch, the Muon branch, or the per-matrix stable-rank choice of
// Appendix G made on the device.
enum class StepKind : int { kLion = 0, kMuon = 1, kAdaptive = 2 };

struct Plan {
  bool muon_step = false;
  bool adaptive = false;
  ChipShape chip;

  // Lion branch
  std::vector<LionTensor> lion;
  std::vector<int32_t> lion_block_start;   // lion.size() + 1 prefix
  int64_t lion_elements = 0;               // Lion-branch elements
  int64_t adamw_elements = 0;              // AdamW elements
  int32_t n_adamw = 0;

  // Muon branch
  std::vector<MuonMat> mats;
  std::vector<int32_t> prep_start;         // mats.size() + 1 prefix of prep tiles
  // Newton-Schulz tile lists, [0] bf16 matrices, [1] fp32 matrices, each
  // grouped per XCD segment
  std::vector<GemmTask> gram[2], poly[2], apply[2];
  XcdSplit gram_split[2]{}, poly_split[2]{}, apply_split[2]{};
  // bf16 apply tiles past the last full round of 256-tiles (one per CU),
  // when they fill at most half a round, each split into sixteen 64-tiles
  // (when those fit one round) or four 128-tiles, run by extra workgroups of
  // the same launch as `apply`
  std::vector<GemmTask> apply_tail[2];
  XcdSplit apply_tail_split[2]{};
  int32_t tile[2][3] = {{kTileBig, kTileBig, kTileBig}, {kTileSmall, kTileSmall, kTileSmall}};
  int32_t tail_tile[2] = {kTileSmall, kTileSmall};   // tile edge of apply_tail
  int64_t muon_elements = 0;
  int32_t n_shape_classes = 0;

  // Adaptive step: every candidate sits in `mats` AND in `lion` (gated by its
  // decision); prefix sums of the stable-rank pass blocks and reduction
  // chunks, and the candidate index of each input tensor (-1: none).
  struct SrClass {
    int32_t kind, bucket;    // SrKind and register bucket
    int32_t first, count;    // range of sr_tab
  };
  std::vector<SrBlock> sr_tab;             // pass workgroups, grouped by class
  std::vector<SrClass> sr_classes;
  std::vector<int32_t> rd_start;
  std::vector<int32_t> tensor_mat;
  int64_t candidate_elements = 0;

  // workspace layout, bytes from the (256-byte aligned) base
  size_t ws_partials_off = 0;   // float per preparation tile
  size_t ws_rscale_off = 0;     // float per matrix
  size_t ws_decide_off = 0;     // adaptive: int32 per matrix, 1 = Muon
  size_t ws_bytes = 0;

  int32_t n_tensors = 0;        // non-empty tensors
};

// Validate hyper-parameters of one step. On failure fills *err.
Status validate_scalars(int64_t t, int32_t P, double beta1, double beta2, double wd,
                        double lr_muon, double lr_lion, std::string* err);

// Validate the tensor list: pointers, shapes, flags and buffer overlaps.
Status validate_tensors(const TensorIn* x, int32_t n, std::string* err);

// Build the plan of one step kind for a device of the given shape;
// kappa_rms02 selects Table 3 output scaling. The plan depends on the
// tensors' shapes, flags and 16-byte alignment only, never on their
// addresses (those go into the per-call binding table). Its workspace size
// does not depend on alignment either.
Status build_plan(const TensorIn* x, int32_t n, StepKind kind, NsPrecision prec,
                  bool kappa_rms02, ChipShape chip, Plan* out, std::string* err);

// 16-byte alignment class of one tensor's buffers (the only property of its
// addresses a plan depends on): bit 0 = W, G, M (and V for AdamW) all 16-byte
// aligned.
uint32_t align_class(const TensorIn& x);

// Register buckets of the stable-rank passes: the smallest listed bucket
// holding ceil(s / 256) column chunks (tall, s <= 2048), ceil(s / 128) row
// passes (wide, s <= 1024) or ceil(s / 256) row passes (narrow wide,
// 1024 < s <= 1536); 0 where no bucket fits (generic path).
constexpr int kSrTallBuckets[] = {1, 2, 3, 4, 6, 8};
constexpr int kSrWideBuckets[] = {1, 2, 4, 6, 8};
constexpr int kSrNarrowBuckets[] = {1, 2, 4, 6};
int sr_tall_bucket(int64_t s);
int sr_wide_bucket(int64_t s);

// Split an ordered task list (cost = inner dimension of each tile) into one
// contiguous segment per XCD (xcds of them) with near-equal total cost, then
// order each segment by decreasing cost (stable). Exposed for tests.
void split_by_xcd(std::vector<GemmTask>* tasks, const std::vector<int64_t>& cost, int xcds,
                  XcdSplit* split);

// Algorithmic Newton-Schulz flops of one Muon step over the plan's matrices.
double ns_flops_symmetric(const Plan& p, int ns_steps);
double ns_flops_dense(const Plan& p, int ns_steps);

}  // namespace lm
