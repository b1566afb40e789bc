// Plain-old-data descriptors shared by the host planner and the gfx950
// kernels of the LionMuon step. The planner fills them on the host from the
// shapes, flags and alignment of a tensor list (no tensor addresses), uploads
// them once per such signature, and the kernels read them from device memory.
// The caller's tensor addresses reach the kernels separately, as one
// TensorPtrs entry per input tensor (the per-call binding table).
#pragma once

#include <stdint.h>

namespace lm {

// Tile sizes of the Newton-Schulz GEMMs and of the Muon preparation pass.
constexpr int kTileSmall = 128;  // MFMA output tile edges; fp32 buffers are padded
constexpr int kTileBig = 256;    // to 128, bf16 buffers to 256
constexpr int kTileTiny = 64;    // fp32 products with too few 128-tiles to fill the chip
                                   // only with at least this many (two per CU)
constexpr int kPrepTile = 64;    // rows of a tall matrix's preparation / transpose tile
constexpr int kPrepTallCols = 128;  // its columns with bf16 X (64 with fp32 X)
constexpr int kPrepElems = 4096; // elements of every preparation tile (wide: 16 x 256 or 32 x 128)
constexpr int kLionBlockElems = 4096;  // elements per Lion workgroup (256 x float4 x 4)
constexpr int kMaxXcds = 8;      // most accelerator complex dies of one device
                                 // (MI355X: 8 XCDs of 32 CUs; the counts in use
                                 // are read from the device, see ChipShape)
// Stable-rank passes (adaptive step). Matrices with 16-byte rows and a short
// side up to kSrMaxRegSide hold their block in registers (tall: blocks of
// kSrTallRows rows; wide: strips of kSrWideCols columns, taken 32 columns at a
// time, or 16 for short sides above 1024); the others take the generic path
// (blocks of kSrBlock long-side positions, read twice).
constexpr int kSrBlock = 32;
constexpr int kSrTallRows = 128;
constexpr int kSrWideCols = 256;
constexpr int kSrMaxRegSide = 2048;
constexpr int kSrChunk = 64;     // short-side entries per stable-rank reduction workgroup
enum SrKind : int32_t { kSrGeneric = 0, kSrTall = 1, kSrWide = 2, kSrWideNarrow = 3 };

// Compute units and XCDs of the device a plan is built for. Workgroup i of a
// launch runs on XCD i mod xcds; a full round of one-per-CU workgroups is cus.
struct ChipShape {
  int32_t cus = 256;
  int32_t xcds = 8;
};

// Device addresses of one input tensor, uploaded per call (the plan holds
// only tensor indices into this table).
struct TensorPtrs {
  float* w;          // W (the output O for the NS hook)
  const float* g;    // G
  float* m;          // M (null for the NS hook)
  float* v;          // AdamW second moment, or null
};

// One workgroup of a stable-rank pass: matrix index and block index.
struct SrBlock {
  int32_t mat;
  int32_t blk;
};

// One tensor of the elementwise pass: the Lion branch, or AdamW.
struct LionTensor {
  int64_t numel;
  int32_t tensor;   // index into the binding table (w, g, m and, for AdamW, v)
  int32_t vec_ok;   // every buffer of the tensor is 16-byte aligned
  int32_t adamw;    // 1: AdamW, 0: Lion
  int32_t gate;     // adaptive step: Muon-candidate index whose decision gates
                    // this tensor (skipped when the candidate took Muon); -1: always
};

// One matrix on the Muon branch. Workspace offsets are in BYTES from the
// workspace base; the Newton-Schulz buffers of the matrix hold bf16 or fp32
// elements (`fp32`).
struct MuonMat {
  int64_t rows, cols;      // m, n of the original tensor (W, G, M row-major;
                           // their addresses are entry `tensor` of the binding)
  int32_t s, l;            // short and long side
  int32_t s_pad, l_pad;    // padded to 128 (fp32) or 256 (bf16)
  int32_t transposed;      // rows > cols: iterate on G^T
  int32_t vec_ok;          // 16-byte vector access legal on w, g, m rows
  int32_t fp32;            // 1: fp32 Newton-Schulz buffers, 0: bf16
  int32_t tensor;          // index of the tensor in the caller's list
  int64_t off_x[2];        // X (s_pad x l_pad, row-major), ping-pong
  int64_t off_a;           // A = X X^T (s_pad x s_pad)
  int64_t off_b;           // B' = a I + b A + c A A (s_pad x s_pad)
  int32_t prep_first;      // first preparation tile of this matrix
  int32_t prep_tiles_n;    // preparation tiles along the original columns
  int32_t prep_count;      // preparation tiles of this matrix
  float kappa;             // output scale
  // adaptive step (stable-rank estimate of M): pass blocks along the long
  // side, and the byte offset of the matrix's fp64 buffers: the iterate z
  // (s), per-block partial products (sr_blocks x s), per-block sums of u^2
  // and of M^2 (sr_blocks each) and chunk sums of z^2 (ceil(s / kSrChunk)).
  int32_t sr_blocks;
  int32_t tall;            // rows >= cols: blocks of rows, else blocks of columns
  int64_t off_sr;
  int32_t sr_kind;         // SrKind of the matrix's pass
  int32_t sr_bucket;       // register bucket of the tall / wide pass
};

// One output tile of one Newton-Schulz GEMM.
struct GemmTask {
  int32_t mat;
  int16_t tm, tn;          // tile row / column (units of the launch's tile edge)
};

// Per-launch partition of a task list into one contiguous segment per XCD
// (the first ChipShape::xcds entries are used).
struct XcdSplit {
  int32_t start[kMaxXcds];
  int32_t count[kMaxXcds];
  int32_t max_count;
};

}  // namespace lm
