// Launchers of the gfx950 kernels of the LionMuon step. Each returns the
// hipError_t of its launch; all work is enqueued on `stream`.
#pragma once

#include <hip/hip_runtime_api.h>

#include "lm_desc.h"

namespace lm {

// fp32 constants of one step, each rounded once from the double
// hyper-parameters (one_minus_beta* formed in double).
struct StepConsts {
  float beta1, one_minus_beta1, beta2, one_minus_beta2;
  float lr_lion, lr_muon, wd, eps;
  // AdamW (LM_TENSOR_ADAMW tensors); c1, c2 = 1 / (1 - beta^step)
  float adam_lr, adam_b1, adam_omb1, adam_b2, adam_omb2, adam_eps, adam_wd, adam_c1, adam_c2;
};

struct LionLaunch {
  const LionTensor* tensors;     // device
  const TensorPtrs* bind;        // device: the call's tensor addresses
  const int32_t* block_start;    // device, n_tensors + 1
  int32_t n_tensors;
  int32_t n_blocks;
  const int32_t* decide;         // adaptive: per-candidate decisions (1 = Muon), else null
  StepConsts k;
};
// Elementwise pass: Lion-branch tensors and AdamW tensors in one launch.
hipError_t launch_lion(const LionLaunch& a, hipStream_t stream);

struct PrepLaunch {
  const MuonMat* mats;           // device
  const TensorPtrs* bind;        // device: the call's tensor addresses
  const int32_t* prep_start;     // device, n_mats + 1
  int32_t n_mats;
  int32_t n_tiles;
  void* ws;                      // workspace base
  float* partials;               // one float per preparation tile
  float* rscale;                 // one float per matrix
  const int32_t* decide;         // adaptive: matrices with decision 0 are skipped
  StepConsts k;
};
// Interpolation, momentum update, X0 / X0^T store and Frobenius partials,
// then the per-matrix 1/(||Ghat||_F + eps).
hipError_t launch_prep(const PrepLaunch& a, hipStream_t stream);
hipError_t launch_norm(const PrepLaunch& a, hipStream_t stream);

enum GemmMode { kGram = 0, kPoly = 1, kApply = 2 };

struct GemmLaunch {
  const MuonMat* mats;           // device
  const TensorPtrs* bind;        // device: the call's tensor addresses (last apply: W)
  ChipShape chip;                // CUs and XCDs: grid of the persistent apply
  const GemmTask* tasks;         // device, grouped by XCD segment
  const XcdSplit* split;         // device: one segment of `tasks` per XCD
  int32_t max_count;             // largest segment (host copy): grid = xcds x max_count
  void* ws;
  const float* rscale;
  int32_t src;                   // ping-pong index of the current X, X^T
  int32_t first;                 // first NS step: apply 1/(||Ghat||_F + eps)
  int32_t last;                  // last NS step: write W (or O)
  int32_t store_o;               // last step stores kappa*X_K instead of a W update
  float a, b, c;                 // odd polynomial coefficients
  float lr, wd;                  // eta_M and lambda of the W update
  int32_t fp32;                  // element type of the matrices in `tasks`
  int32_t tile;                  // output tile edge of `tasks`: 128 or 256
  const int32_t* decide;         // adaptive: tiles of matrices with decision 0 exit
  // apply on bf16 256-tiles only: the last round's smaller tiles (64 or 128),
  // run by extra workgroups of the same launch; none when tail_max_count is 0
  const GemmTask* tail_tasks = nullptr;   // device, grouped by XCD segment
  const XcdSplit* tail_split = nullptr;   // device
  int32_t tail_max_count = 0;             // largest segment (host copy)
  int32_t tail_tile = 0;
};
hipError_t launch_gemm(GemmMode mode, const GemmLaunch& a, hipStream_t stream);

// Adaptive step (Appendix G): stable-rank estimate of each candidate's
// momentum by power iteration on the Gram matrix of its short side, in fp64.
struct SrankLaunch {
  const MuonMat* mats;           // device
  const TensorPtrs* bind;        // device: the call's tensor addresses (M)
  const SrBlock* tab;            // device: pass workgroups, grouped by class
  const int32_t* rd_start;       // device, n_mats + 1: reduction chunks
  const int32_t* tensor_mat;     // device, n_inputs: candidate index or -1
  int32_t n_mats;
  int32_t n_chunks;              // rd_start[n_mats]
  int32_t n_inputs;              // length of the caller's tensor list
  void* ws;
  int32_t* decide;               // workspace: one int32 per candidate
  int32_t* decisions_out;        // optional, per input tensor (device)
  double* srank_out;             // optional, per input tensor (device)
  double alpha;
};
// One pass over M per power step for the workgroups tab[first_block ..
// first_block + n_blocks) of one class (kind, bucket): z' = S^T S (z / ||z||)
// as per-block partials (the first pass starts from the all-ones vector and
// writes the sums of M^2); `last` passes only sum ||S z / ||z|| ||^2.
// `reverse` walks the blocks from the last to the first (same results: each
// block writes its own partials).
hipError_t launch_srank_pass(const SrankLaunch& a, int32_t kind, int32_t bucket,
                             int32_t first_block, int32_t n_blocks, bool first, bool last,
                             bool reverse, hipStream_t stream);
// Fixed-order sum of the partials into z' and the chunk sums of z'^2.
hipError_t launch_srank_reduce(const SrankLaunch& a, hipStream_t stream);
// r_hat = ||M||_F^2 / sigma_hat^2 and the decision r_hat <= alpha * min(m, n).
hipError_t launch_srank_decide(const SrankLaunch& a, hipStream_t stream);

// No-allocation entry point: one file-scope device array per device (its
// size is the most a call of that entry point may use: plan tables, address
// table and workspace together).
constexpr size_t kScratchBytes = size_t(64) << 20;
// Device address of the scratch array on `device`, which must be current
// (looked up on the first call per device, then cached).
hipError_t scratch_address(int device, void** out);
// Copy `bytes` (a multiple of 4; dst 4-byte aligned) from host memory to
// device memory on `stream` through kernel arguments: no staging buffer. The
// source may be reused as soon as this returns.
hipError_t launch_upload(void* dst, const void* src, size_t bytes, hipStream_t stream);

}  // namespace lm
