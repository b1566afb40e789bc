// gfx950 kernels of the LionMuon step (Algorithm 1 of arXiv 2605.19811).
//
//  lion_kernel   Lion branch: Ghat = b1*M + (1-b1)*G; W -= lr*(sign(Ghat) + wd*W);
//                M = b2*M + (1-b2)*G. Multi-tensor, 16-byte vectors, HBM bound.
//                Tensors flagged AdamW take the AdamW update in the same launch.
//  prep_kernel   Muon branch, first pass: the same interpolation and momentum
//                update, Ghat stored in the NS element type in the iteration
//                orientation X (rows <= cols; an LDS transpose for tall
//                matrices), and a per-tile partial sum of Ghat^2.
//  norm_kernel   fixed-order reduction of the partials -> 1/(||Ghat||_F + eps).
//  srank_*       adaptive step: fp64 power iteration for the stable rank of
//                each candidate's momentum and the per-matrix Muon / Lion
//                decision, which the kernels above and below then read.
//  ns_*_kernel   the Newton-Schulz products on MFMA with fp32 accumulation:
//                Gram A = X X^T and polynomial B' = a I + b A + c A A on the
//                lower triangle of tiles (mirrored on store), then apply
//                X' = B' X (= a X + (b A + c A A) X), whose X operand is read
//                from row-major X through LDS transpose reads, with the W
//                update fused into the last step's epilogue.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace lm {

namespace {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

// sign with sign(+-0) = 0 and NaN propagated.
__device__ __forceinline__ float sign_f(float x) {
  return x > 0.0f ? 1.0f : (x < 0.0f ? -1.0f : x);
}

// Largest i in [0, n) with start[i] <= b (start is non-decreasing, start[0] = 0).
__device__ __forceinline__ int find_segment(const int32_t* start, int n, int b) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (start[mid] <= b) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// ---------------------------------------------------------------------------
// Lion branch
// ---------------------------------------------------------------------------
struct LionArgs {
  const LionTensor* tensors;
  const TensorPtrs* bind;
  const int32_t* block_start;
  const int32_t* decide;
  int32_t n_tensors;
  float b1, omb1, b2, omb2, lr, wd;
  float ab1, aomb1, ab2, aomb2, alr, aeps, awd, ac1, ac2;   // AdamW
};

__device__ __forceinline__ void lion_elem(float& w, float g, float& m, const LionArgs& a) {
  const float c = fmaf(a.b1, m, a.omb1 * g);
  w = fmaf(-a.lr, fmaf(a.wd, w, sign_f(c)), w);
  m = fmaf(a.b2, m, a.omb2 * g);
}

// AdamW with decoupled weight decay; ac1, ac2 are the bias corrections.
__device__ __forceinline__ void adamw_elem(float& w, float g, float& m, float& v,
                                           const LionArgs& a) {
  m = fmaf(a.ab1, m, a.aomb1 * g);
  v = fmaf(a.ab2, v, a.aomb2 * (g * g));
  const float upd = (m * a.ac1) / (sqrtf(v * a.ac2) + a.aeps);
  w = fmaf(-a.alr, fmaf(a.awd, w, upd), w);
}

constexpr int kLionUnroll = kLionBlockElems / (256 * 4);

__global__ __launch_bounds__(256) void lion_kernel(LionArgs a) {
  const int b = blockIdx.x;
  const int ti = find_segment(a.block_start, a.n_tensors, b);
  const LionTensor t = a.tensors[ti];
  if (t.gate >= 0 && a.decide[t.gate] != 0) return;   // the candidate took Muon
  const TensorPtrs tp = a.bind[t.tensor];
  const int64_t base = int64_t(b - a.block_start[ti]) * kLionBlockElems;
  const int tid = threadIdx.x;
  const bool full = t.vec_ok && base + kLionBlockElems <= t.numel;
  if (full && !t.adamw) {
    f32x4* w4 = reinterpret_cast<f32x4*>(tp.w + base);
    const f32x4* g4 = reinterpret_cast<const f32x4*>(tp.g + base);
    f32x4* m4 = reinterpret_cast<f32x4*>(tp.m + base);
    f32x4 w[kLionUnroll], g[kLionUnroll], m[kLionUnroll];
    // every stream is touched once per step: non-temporal loads and stores
    // (measured: pure-Lion steps 7-8% faster than with cached W, M loads)
#pragma unroll
    for (int u = 0; u < kLionUnroll; ++u) {
      const int i = tid + 256 * u;
      w[u] = __builtin_nontemporal_load(&w4[i]);
      g[u] = __builtin_nontemporal_load(&g4[i]);
      m[u] = __builtin_nontemporal_load(&m4[i]);
    }
#pragma unroll
    for (int u = 0; u < kLionUnroll; ++u) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float we = w[u][e], me = m[u][e];
        lion_elem(we, g[u][e], me, a);
        w[u][e] = we;
        m[u][e] = me;
      }
    }
#pragma unroll
    for (int u = 0; u < kLionUnroll; ++u) {
      const int i = tid + 256 * u;
      __builtin_nontemporal_store(w[u], &w4[i]);
      __builtin_nontemporal_store(m[u], &m4[i]);
    }
  } else if (full) {
    f32x4* w4 = reinterpret_cast<f32x4*>(tp.w + base);
    const f32x4* g4 = reinterpret_cast<const f32x4*>(tp.g + base);
    f32x4* m4 = reinterpret_cast<f32x4*>(tp.m + base);
    f32x4* v4 = reinterpret_cast<f32x4*>(tp.v + base);
#pragma unroll
    for (int u = 0; u < kLionUnroll; ++u) {
      const int i = tid + 256 * u;
      f32x4 w = w4[i], g = g4[i], m = m4[i], v = v4[i];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float we = w[e], me = m[e], ve = v[e];
        adamw_elem(we, g[e], me, ve, a);
        w[e] = we;
        m[e] = me;
        v[e] = ve;
      }
      w4[i] = w;
      m4[i] = m;
      v4[i] = v;
    }
  } else {
    const int64_t end = min(base + int64_t(kLionBlockElems), t.numel);
    for (int64_t i = base + tid; i < end; i += 256) {
      float w = tp.w[i], m = tp.m[i];
      if (t.adamw) {
        float v = tp.v[i];
        adamw_elem(w, tp.g[i], m, v, a);
        tp.v[i] = v;
      } else {
        lion_elem(w, tp.g[i], m, a);
      }
      tp.w[i] = w;
      tp.m[i] = m;
    }
  }
}

// ---------------------------------------------------------------------------
// Muon branch: preparation and norm
// ---------------------------------------------------------------------------
struct PrepArgs {
  const MuonMat* mats;
  const TensorPtrs* bind;
  const int32_t* prep_start;
  int32_t n_mats;
  void* ws;
  float* partials;
  float* rscale;
  const int32_t* decide;
  float b1, omb1, b2, omb2, eps;
};

template <typename T> __device__ __forceinline__ T to_elem(float v);
template <> __device__ __forceinline__ float to_elem<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 to_elem<bf16>(float v) { return bf16(v); }

// Store four consecutive elements (8 bytes for bf16, 16 for fp32; aligned).
__device__ __forceinline__ void store4(bf16* p, const float v[4]) {
  bf16x4 x = {bf16(v[0]), bf16(v[1]), bf16(v[2]), bf16(v[3])};
  *reinterpret_cast<bf16x4*>(p) = x;
}
__device__ __forceinline__ void store4(float* p, const float v[4]) {
  const f32x4 x = {v[0], v[1], v[2], v[3]};
  *reinterpret_cast<f32x4*>(p) = x;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16 a = bf16(lo), b = bf16(hi);
  return uint32_t(__builtin_bit_cast(uint16_t, a)) | (uint32_t(__builtin_bit_cast(uint16_t, b)) << 16);
}
__device__ __forceinline__ void load4(const bf16* p, float v[4]) {
  const bf16x4 x = *reinterpret_cast<const bf16x4*>(p);
  v[0] = float(x[0]); v[1] = float(x[1]); v[2] = float(x[2]); v[3] = float(x[3]);
}
__device__ __forceinline__ void load4(const float* p, float v[4]) {
  const f32x4 x = *reinterpret_cast<const f32x4*>(p);
  v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
}

// LDS block of the transpose tile (bf16 64 x 131 or fp32 64 x 66 elements)
constexpr int kPrepLdsBytes = 64 * 66 * 4;

// Wide matrix (X = Ghat, same layout): a strip of kPrepElems elements, TC
// columns wide, so that each wave reads and writes whole TC-element pieces
// of rows (1 KB of fp32 for TC = 256). G and M are read and M written with
// the non-temporal hint (the step does not touch them again); X is stored
// normally, since the first Gram product reads it next.
template <typename T, int TC>
__device__ __forceinline__ void prep_wide(const PrepArgs& a, const MuonMat& mm, int b) {
  constexpr int kChunks = TC / 4, kRowsPass = 256 / kChunks, kRows = kPrepElems / TC;
  constexpr int kPasses = kRows / kRowsPass;
  static_assert(kPasses * kRowsPass == kRows, "whole passes per strip");
  __shared__ float red[4];
  const float* G = a.bind[mm.tensor].g;
  float* Mp = a.bind[mm.tensor].m;           // null for the NS hook
  const int local = b - mm.prep_first;
  const int ti = local / mm.prep_tiles_n, tj = local - ti * mm.prep_tiles_n;
  T* X = reinterpret_cast<T*>(static_cast<char*>(a.ws) + mm.off_x[0]);
  const int64_t cols_pad = mm.l_pad;
  const int tid = threadIdx.x, r0 = tid / kChunks, c4 = (tid % kChunks) * 4;
  float ss = 0.0f;
#pragma unroll
  for (int u = 0; u < kPasses; ++u) {
    const int64_t p = int64_t(ti) * kRows + r0 + kRowsPass * u;
    const int64_t q = int64_t(tj) * TC + c4;
    float gv[4] = {0.f, 0.f, 0.f, 0.f}, mv[4] = {0.f, 0.f, 0.f, 0.f};
    const bool row_in = p < mm.rows;
    const bool vec = row_in && mm.vec_ok && q + 3 < mm.cols;
    const int64_t idx = p * mm.cols + q;
    if (vec) {
      const f32x4 g = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(G + idx));
      gv[0] = g[0]; gv[1] = g[1]; gv[2] = g[2]; gv[3] = g[3];
      if (Mp) {
        const f32x4 m = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(Mp + idx));
        mv[0] = m[0]; mv[1] = m[1]; mv[2] = m[2]; mv[3] = m[3];
      }
    } else if (row_in) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (q + e < mm.cols) {
          gv[e] = G[idx + e];
          if (Mp) mv[e] = Mp[idx + e];
        }
      }
    }
    float c[4], mn[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      c[e] = fmaf(a.b1, mv[e], a.omb1 * gv[e]);
      mn[e] = fmaf(a.b2, mv[e], a.omb2 * gv[e]);
      ss = fmaf(c[e], c[e], ss);
    }
    if (Mp) {
      if (vec) {
        const f32x4 mv4 = {mn[0], mn[1], mn[2], mn[3]};
        __builtin_nontemporal_store(mv4, reinterpret_cast<f32x4*>(Mp + idx));
      } else if (row_in) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (q + e < mm.cols) Mp[idx + e] = mn[e];
      }
    }
    store4(X + p * cols_pad + q, c);
  }
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  if (tid == 0) a.partials[mm.prep_first + local] = (red[0] + red[1]) + (red[2] + red[3]);
}

// Tall matrix: a kPrepTile x TC tile of Ghat (rows read as 4 TC-byte
// pieces), stored transposed (X = Ghat^T) through LDS as 64-element pieces of
// TC rows of X. TC = kPrepTallCols (bf16 X) or kPrepTile (fp32 X), so both
// tiles fit the same LDS block.
template <typename T, int TC>
__device__ __forceinline__ void prep_tall(const PrepArgs& a, const MuonMat& mm, int b,
                                          char* lds) {
  constexpr int kTR = kPrepTile, kTC = TC;
  constexpr int kPad = 4 / sizeof(T) + 1;        // odd word stride per LDS row
  constexpr int kChunks = kTC / 4, kRowsPass = 256 / kChunks, kPasses = kTR / kRowsPass;
  static_assert(kTR * (kTC + kPad) * sizeof(T) <= kPrepLdsBytes, "tile fits the LDS block");
  T (*tile)[kTC + kPad] = reinterpret_cast<T (*)[kTC + kPad]>(lds);
  __shared__ float red[4];
  const float* G = a.bind[mm.tensor].g;
  float* Mp = a.bind[mm.tensor].m;           // null for the NS hook
  const int local = b - mm.prep_first;
  const int ti = local / mm.prep_tiles_n, tj = local - ti * mm.prep_tiles_n;
  const int64_t rows_pad = mm.l_pad;           // of the original (tall) matrix
  T* X = reinterpret_cast<T*>(static_cast<char*>(a.ws) + mm.off_x[0]);
  const int tid = threadIdx.x, r0 = tid / kChunks, c4 = (tid % kChunks) * 4;
  float ss = 0.0f;
#pragma unroll
  for (int u = 0; u < kPasses; ++u) {
    const int r = r0 + kRowsPass * u;
    const int64_t p = int64_t(ti) * kTR + r;
    const int64_t q = int64_t(tj) * kTC + c4;
    float gv[4] = {0.f, 0.f, 0.f, 0.f}, mv[4] = {0.f, 0.f, 0.f, 0.f};
    const bool row_in = p < mm.rows;
    const bool vec = row_in && mm.vec_ok && q + 3 < mm.cols;
    const int64_t idx = p * mm.cols + q;
    if (vec) {
      const f32x4 g = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(G + idx));
      gv[0] = g[0]; gv[1] = g[1]; gv[2] = g[2]; gv[3] = g[3];
      if (Mp) {
        const f32x4 m = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(Mp + idx));
        mv[0] = m[0]; mv[1] = m[1]; mv[2] = m[2]; mv[3] = m[3];
      }
    } else if (row_in) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (q + e < mm.cols) {
          gv[e] = G[idx + e];
          if (Mp) mv[e] = Mp[idx + e];
        }
      }
    }
    float c[4], mn[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      c[e] = fmaf(a.b1, mv[e], a.omb1 * gv[e]);
      mn[e] = fmaf(a.b2, mv[e], a.omb2 * gv[e]);
      ss = fmaf(c[e], c[e], ss);
    }
    if (Mp) {
      if (vec) {
        const f32x4 mv4 = {mn[0], mn[1], mn[2], mn[3]};
        __builtin_nontemporal_store(mv4, reinterpret_cast<f32x4*>(Mp + idx));
      } else if (row_in) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (q + e < mm.cols) Mp[idx + e] = mn[e];
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) tile[r][c4 + e] = to_elem<T>(c[e]);
  }
  __syncthreads();
  // X^T rows: kTC of them, kTR elements each, 4 per thread
  constexpr int kLpr = kTR / 4, kXRowsPass = 256 / kLpr;
  const int xr0 = tid / kLpr, xc4 = (tid % kLpr) * 4;
#pragma unroll
  for (int u = 0; u < kTC / kXRowsPass; ++u) {
    const int qq = xr0 + kXRowsPass * u;          // column of the source tile
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = float(tile[xc4 + e][qq]);
    store4(X + (int64_t(tj) * kTC + qq) * rows_pad + int64_t(ti) * kTR + xc4, v);
  }
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  if (tid == 0) a.partials[mm.prep_first + local] = (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ __launch_bounds__(256) void prep_kernel(PrepArgs a) {
  __shared__ __attribute__((aligned(16))) char lds[kPrepLdsBytes];
  const int b = blockIdx.x;
  const int mi = find_segment(a.prep_start, a.n_mats, b);
  if (a.decide && a.decide[mi] == 0) return;          // the candidate took Lion
  const MuonMat& mm = a.mats[mi];
  if (mm.transposed) {
    if (mm.fp32) prep_tall<float, kPrepTile>(a, mm, b, lds);
    else prep_tall<bf16, kPrepTallCols>(a, mm, b, lds);
  } else if (mm.l_pad == mm.prep_tiles_n * 256) {
    if (mm.fp32) prep_wide<float, 256>(a, mm, b);
    else prep_wide<bf16, 256>(a, mm, b);
  } else {
    if (mm.fp32) prep_wide<float, 128>(a, mm, b);
    else prep_wide<bf16, 128>(a, mm, b);
  }
}

__global__ __launch_bounds__(256) void norm_kernel(PrepArgs a) {
  __shared__ float red[4];
  if (a.decide && a.decide[blockIdx.x] == 0) return;
  const MuonMat mm = a.mats[blockIdx.x];
  const float* p = a.partials + mm.prep_first;
  float s = 0.0f;
  for (int i = threadIdx.x; i < mm.prep_count; i += 256) s += p[i];
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float total = (red[0] + red[1]) + (red[2] + red[3]);
    a.rscale[blockIdx.x] = 1.0f / (sqrtf(total) + a.eps);
  }
}

// ---------------------------------------------------------------------------
// Adaptive step: stable rank of the momentum (Appendix G)
// ---------------------------------------------------------------------------
// S is the long-side view of M (S = M when rows >= cols, else M^T), so the
// iterate z has s = min(m, n) entries, and S^T S is the sum over blocks of
// long-side positions of S_blk^T S_blk. Per power step one pass reads every
// block of S once: u = S_blk v with v = z / ||z||, then the block's share
// S_blk^T u of the next iterate, written as one fp64 partial vector per block;
// a reduction kernel sums the partials in a fixed order.
// Register paths (16-byte rows, s <= kSrMaxRegSide), v held in LDS:
//   tall M: a block is kSrTallRows rows; each wave streams groups of its rows
//           through registers (lanes along the row, 4 floats each) and keeps
//           its share of S_blk^T u in fp64 registers;
//   wide M: a block is a strip of kSrWideCols columns, taken 32 columns at a
//           time by a 1024-thread workgroup that holds all s rows of those
//           columns in registers (8 lanes per 128-byte row segment).
// Generic path (any alignment or short side): blocks of kSrBlock positions,
// read a second time (from cache) for S_blk^T u.
// All sums are fp64 in a fixed order.
struct SrankArgs {
  const MuonMat* mats;
  const TensorPtrs* bind;
  const SrBlock* tab;
  const int32_t* rd_start;
  const int32_t* tensor_mat;
  int32_t n_mats;
  void* ws;
  int32_t* decide;
  int32_t* decisions_out;
  double* srank_out;
  double alpha;
  int32_t reverse;   // pass blocks in reverse order (alternate passes: the
                     // blocks read last are still in the last-level cache)
};

struct SrBufs {
  double* z;       // s
  double* part;    // sr_blocks x s
  double* usq;     // sr_blocks
  double* fsq;     // sr_blocks
  double* nrm;     // ceil(s / kSrChunk)
  int nchunks;
};

__device__ __forceinline__ SrBufs sr_bufs(void* ws, const MuonMat& mm) {
  SrBufs b;
  b.z = reinterpret_cast<double*>(static_cast<char*>(ws) + mm.off_sr);
  b.part = b.z + mm.s;
  b.usq = b.part + int64_t(mm.sr_blocks) * mm.s;
  b.fsq = b.usq + mm.sr_blocks;
  b.nrm = b.fsq + mm.sr_blocks;
  b.nchunks = (mm.s + kSrChunk - 1) / kSrChunk;
  return b;
}

// Butterfly sum: every lane ends with the same, order-fixed total.
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// 1 / ||z|| from the chunk sums of z^2 (0 for a vanished iterate), or
// 1 / sqrt(s) for the all-ones start vector.
__device__ __forceinline__ double sr_inv_norm(const MuonMat& mm, const SrBufs& B, bool first) {
  if (first) return 1.0 / sqrt(double(mm.s));
  double n2 = 0.0;
  for (int i = 0; i < B.nchunks; ++i) n2 += B.nrm[i];
  return n2 > 0.0 ? 1.0 / sqrt(n2) : 0.0;
}

// v = z / ||z|| into LDS.
template <int NT>
__device__ __forceinline__ void sr_load_v(double* vs, const MuonMat& mm, const SrBufs& B,
                                          bool first) {
  const double inv = sr_inv_norm(mm, B, first);
  for (int c = threadIdx.x; c < mm.s; c += NT) vs[c] = first ? inv : B.z[c] * inv;
  __syncthreads();
}

// Block totals of u^2 (uu_wave: the same value in every lane of a wave) and
// of M^2 (per-lane partials), written by thread 0 in a fixed order.
template <int NW>
__device__ __forceinline__ void sr_block_sums(double* red, double uu_wave, double fs_lane,
                                              bool first, const SrBufs& B, int blk) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const double fs = wave_sum_d(fs_lane);
  __syncthreads();
  if (lane == 0) {
    red[2 * wave] = uu_wave;
    red[2 * wave + 1] = fs;
  }
  __syncthreads();
  if (tid == 0) {
    double u = 0.0, f = 0.0;
    for (int w = 0; w < NW; ++w) {
      u += red[2 * w];
      f += red[2 * w + 1];
    }
    B.usq[blk] = u;
    if (first) B.fsq[blk] = f;
  }
}

template <int NCH>
__global__ __launch_bounds__(256) void srank_tall_kernel(SrankArgs a, int32_t first_block,
                                                         int32_t first, int32_t last) {
  constexpr int kRg = NCH <= 4 ? 4 : 2;           // rows per wave per group
  constexpr int kGroups = kSrTallRows / (4 * kRg);
  __shared__ double vs[kSrMaxRegSide];
  __shared__ double red[4][256];
  const SrBlock sb = a.tab[first_block + (a.reverse ? int(gridDim.x) - 1 - int(blockIdx.x) : int(blockIdx.x))];
  const MuonMat& mm = a.mats[sb.mat];
  const SrBufs B = sr_bufs(a.ws, mm);
  sr_load_v<256>(vs, mm, B, first != 0);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int s = mm.s;
  const int64_t r0 = int64_t(sb.blk) * kSrTallRows;
  const int nr = int(min(int64_t(kSrTallRows), mm.l - r0));
  // per-lane base; row and chunk offsets below are wave-uniform
  const float* Ml = a.bind[mm.tensor].m + (r0 + wave * kRg) * s + lane * 4;
  const int cmax = s - lane * 4;                  // chunk q is in range iff q * 256 < cmax
  double w[NCH][4];
#pragma unroll
  for (int q = 0; q < NCH; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) w[q][e] = 0.0;
  double uu = 0.0, fs[kRg];
#pragma unroll
  for (int j = 0; j < kRg; ++j) fs[j] = 0.0;
#pragma unroll 1
  for (int g = 0; g < kGroups; ++g) {
    const int rb = g * 4 * kRg + wave * kRg;      // this wave's first row of the group
    const float* Mg = Ml + int64_t(g * 4 * kRg) * s;
    f32x4 x[kRg][NCH];
#pragma unroll
    for (int j = 0; j < kRg; ++j)
#pragma unroll
      for (int q = 0; q < NCH; ++q) {
        x[j][q] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (rb + j < nr && q * 256 < cmax)        // s is a multiple of 4
          x[j][q] = *reinterpret_cast<const f32x4*>(Mg + j * s + q * 256);
      }
    double acc[kRg];
#pragma unroll
    for (int j = 0; j < kRg; ++j) acc[j] = 0.0;
#pragma unroll
    for (int q = 0; q < NCH; ++q) {
      double v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = q * 256 < cmax ? vs[q * 256 + lane * 4 + e] : 0.0;
#pragma unroll
      for (int j = 0; j < kRg; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const double xe = double(x[j][q][e]);
          acc[j] = fma(xe, v[e], acc[j]);
          fs[j] = fma(xe, xe, fs[j]);
        }
    }
    double u[kRg];
#pragma unroll
    for (int j = 0; j < kRg; ++j) {
      u[j] = wave_sum_d(acc[j]);
      uu = fma(u[j], u[j], uu);
    }
    if (!last) {
#pragma unroll
      for (int q = 0; q < NCH; ++q)
#pragma unroll
        for (int j = 0; j < kRg; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) w[q][e] = fma(double(x[j][q][e]), u[j], w[q][e]);
    }
  }
  if (!last) {
#pragma unroll
    for (int q = 0; q < NCH; ++q) {
      __syncthreads();                            // previous chunk's reads of red
#pragma unroll
      for (int e = 0; e < 4; ++e) red[wave][lane * 4 + e] = w[q][e];
      __syncthreads();
      const int c = q * 256 + tid;
      if (c < s)
        B.part[int64_t(sb.blk) * s + c] = (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
    }
  }
  double fsl = 0.0;
#pragma unroll
  for (int j = 0; j < kRg; ++j) fsl += fs[j];
  sr_block_sums<4>(&red[0][0], uu, fsl, first != 0, B, sb.blk);
}

// SW: columns per sub-strip (32: 128-byte row pieces, 8 lanes per row; 16:
// 64-byte pieces, 4 lanes per row, twice the rows per pass for larger s).
template <int NP, int SW>
__global__ __launch_bounds__(1024) void srank_wide_kernel(SrankArgs a, int32_t first_block,
                                                          int32_t first, int32_t last) {
  constexpr int kNw = 16;
  constexpr int kLpr = SW / 4;                    // lanes per row piece
  constexpr int kRpw = 64 / kLpr;                 // rows per wave per pass
  constexpr int kRpp = kNw * kRpw;                // rows per pass
  __shared__ double vs[kSrMaxRegSide];
  __shared__ double ured[kNw][SW];
  __shared__ double us[SW];
  __shared__ double red[2 * kNw];
  const SrBlock sb = a.tab[first_block + (a.reverse ? int(gridDim.x) - 1 - int(blockIdx.x) : int(blockIdx.x))];
  const MuonMat& mm = a.mats[sb.mat];
  const SrBufs B = sr_bufs(a.ws, mm);
  sr_load_v<1024>(vs, mm, B, first != 0);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane % kLpr, rsub = lane / kLpr;
  const int s = mm.s;
  const int64_t l = mm.l;
  const int r_lane = wave * kRpw + rsub;          // row of pass 0
  const int rmax = s - r_lane;                    // pass p is in range iff p * kRpp < rmax
  double w[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) w[p] = 0.0;
  double uu = 0.0, fs[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 1
  for (int ss = 0; ss < kSrWideCols / SW; ++ss) {
    const int64_t c = int64_t(sb.blk) * kSrWideCols + ss * SW + sub * 4;
    const bool cok = c < l;                       // l is a multiple of 4
    // per-lane base; pass offsets p * kRpp rows are wave-uniform
    const float* Ml = a.bind[mm.tensor].m + int64_t(r_lane) * l + c;
    f32x4 x[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      x[p] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (cok && p * kRpp < rmax) x[p] = *reinterpret_cast<const f32x4*>(Ml + int64_t(p * kRpp) * l);
    }
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const double vr = p * kRpp < rmax ? vs[r_lane + p * kRpp] : 0.0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double xe = double(x[p][e]);
        acc[e] = fma(xe, vr, acc[e]);
        fs[e] = fma(xe, xe, fs[e]);
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int off = kLpr; off < 64; off <<= 1) acc[e] += __shfl_xor(acc[e], off, 64);
    if (rsub == 0) {
#pragma unroll
      for (int e = 0; e < 4; ++e) ured[wave][sub * 4 + e] = acc[e];
    }
    __syncthreads();
    if (wave == 0) {
      double uc = 0.0;
      if (lane < SW) {
        for (int k = 0; k < kNw; ++k) uc += ured[k][lane];
        us[lane] = uc;
      }
      uu += wave_sum_d(uc * uc);
    }
    __syncthreads();
    if (!last) {
      double uv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) uv[e] = us[sub * 4 + e];
#pragma unroll
      for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int e = 0; e < 4; ++e) w[p] = fma(double(x[p][e]), uv[e], w[p]);
    }
  }
  if (!last) {
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      double wr = w[p];
#pragma unroll
      for (int off = 1; off < kLpr; off <<= 1) wr += __shfl_xor(wr, off, 64);
      if (sub == 0 && p * kRpp < rmax) B.part[int64_t(sb.blk) * s + r_lane + p * kRpp] = wr;
    }
  }
  sr_block_sums<kNw>(red, uu, (fs[0] + fs[1]) + (fs[2] + fs[3]), first != 0, B, sb.blk);
}

template <int VW>
__device__ __forceinline__ void load_vw(const float* p, bool ok, double x[VW]) {
  if (VW == 4) {
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    if (ok) v = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
    for (int e = 0; e < VW; ++e) x[e] = double(v[e]);
  } else {
    x[0] = ok ? double(*p) : 0.0;
  }
}

// Generic path, tall M (rows = l >= cols = s): block = kSrBlock rows; wave w
// owns rows w, w + 4, ... of the block; lanes run along the row, VW floats each.
template <int VW, bool FIRST, bool LAST>
__device__ void srank_generic_tall(double (*red)[256], const MuonMat& mm, const float* Mbase,
                                   const SrBufs& B, int blk, double inv) {
  constexpr int kRows = kSrBlock / 4;
  constexpr int kChunk = 64 * VW;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int s = mm.s;
  const int64_t r0 = int64_t(blk) * kSrBlock;
  const int nr = int(min(int64_t(kSrBlock), mm.l - r0));
  const float* M = Mbase + r0 * s;
  double acc[kRows], fs[kRows];
#pragma unroll
  for (int j = 0; j < kRows; ++j) acc[j] = fs[j] = 0.0;
  for (int c0 = 0; c0 < s; c0 += kChunk) {
    const int c = c0 + lane * VW;
    const bool ok = c < s;                      // VW = 4: s is a multiple of 4
    double zc[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) zc[e] = FIRST ? 1.0 : (ok ? B.z[c + e] : 0.0);
#pragma unroll
    for (int j = 0; j < kRows; ++j) {
      const int r = wave + 4 * j;
      double x[VW];
      load_vw<VW>(M + int64_t(r) * s + c, ok && r < nr, x);
#pragma unroll
      for (int e = 0; e < VW; ++e) {
        acc[j] = fma(x[e], zc[e], acc[j]);
        fs[j] = fma(x[e], x[e], fs[j]);
      }
    }
  }
  double u[kRows], uu = 0.0, fsl = 0.0;
#pragma unroll
  for (int j = 0; j < kRows; ++j) {
    u[j] = wave_sum_d(acc[j]) * inv;
    uu = fma(u[j], u[j], uu);
    fsl += fs[j];
  }
  if (!LAST) {
    for (int c0 = 0; c0 < s; c0 += kChunk) {
      const int c = c0 + lane * VW;
      const bool ok = c < s;
      double wv[VW];
#pragma unroll
      for (int e = 0; e < VW; ++e) wv[e] = 0.0;
#pragma unroll
      for (int j = 0; j < kRows; ++j) {
        const int r = wave + 4 * j;
        double x[VW];
        load_vw<VW>(M + int64_t(r) * s + c, ok && r < nr, x);
#pragma unroll
        for (int e = 0; e < VW; ++e) wv[e] = fma(x[e], u[j], wv[e]);
      }
      __syncthreads();                           // previous chunk's reads of red
#pragma unroll
      for (int e = 0; e < VW; ++e) red[wave][lane * VW + e] = wv[e];
      __syncthreads();
      for (int i = tid; i < kChunk; i += 256) {
        if (c0 + i < s)
          B.part[int64_t(blk) * s + c0 + i] = (red[0][i] + red[1][i]) + (red[2][i] + red[3][i]);
      }
    }
  }
  sr_block_sums<4>(&red[0][0], uu, fsl, FIRST, B, blk);
}

// Generic path, wide M (rows = s < cols = l): block = kSrBlock columns; LPR
// lanes cover one row's kSrBlock columns, VW floats each.
template <int VW, bool FIRST, bool LAST>
__device__ void srank_generic_wide(double (*red)[256], const MuonMat& mm, const float* Mbase,
                                   const SrBufs& B, int blk, double inv) {
  constexpr int kLpr = kSrBlock / VW;
  constexpr int kRpw = 64 / kLpr;
  constexpr int kRpp = 4 * kRpw;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int s = mm.s;
  const int64_t l = mm.l;
  const int sub = lane % kLpr, rsub = lane / kLpr;
  const int64_t c = int64_t(blk) * kSrBlock + sub * VW;
  const bool cok = c < l;                        // VW = 4: l is a multiple of 4
  const int passes = (s + kRpp - 1) / kRpp;
  const float* Mc = Mbase + c;
  double acc[VW], fs[VW];
#pragma unroll
  for (int e = 0; e < VW; ++e) acc[e] = fs[e] = 0.0;
  for (int p = 0; p < passes; ++p) {
    const int r = p * kRpp + wave * kRpw + rsub;
    const bool ok = cok && r < s;
    const double zr = FIRST ? 1.0 : (r < s ? B.z[r] : 0.0);
    double x[VW];
    load_vw<VW>(Mc + int64_t(r) * l, ok, x);
#pragma unroll
    for (int e = 0; e < VW; ++e) {
      acc[e] = fma(x[e], zr, acc[e]);
      fs[e] = fma(x[e], x[e], fs[e]);
    }
  }
  double fsl = 0.0;
#pragma unroll
  for (int e = 0; e < VW; ++e) {
    fsl += fs[e];
#pragma unroll
    for (int off = kLpr; off < 64; off <<= 1) acc[e] += __shfl_xor(acc[e], off, 64);
  }
  double* ured = &red[0][0];                     // [4][kSrBlock]
  double* us = &red[2][0];                       // kSrBlock
  if (rsub == 0) {
#pragma unroll
    for (int e = 0; e < VW; ++e) ured[wave * kSrBlock + sub * VW + e] = acc[e];
  }
  __syncthreads();
  double uu = 0.0;
  if (wave == 0) {
    double uc = 0.0;
    if (lane < kSrBlock) {
      uc = ((ured[lane] + ured[kSrBlock + lane]) +
            (ured[2 * kSrBlock + lane] + ured[3 * kSrBlock + lane])) * inv;
      us[lane] = uc;
    }
    uu = wave_sum_d(uc * uc);
  }
  __syncthreads();
  if (!LAST) {
    double uv[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) uv[e] = us[sub * VW + e];
    for (int p = 0; p < passes; ++p) {
      const int r = p * kRpp + wave * kRpw + rsub;
      double x[VW];
      load_vw<VW>(Mc + int64_t(r) * l, cok && r < s, x);
      double wr = 0.0;
#pragma unroll
      for (int e = 0; e < VW; ++e) wr = fma(x[e], uv[e], wr);
#pragma unroll
      for (int off = 1; off < kLpr; off <<= 1) wr += __shfl_xor(wr, off, 64);
      if (sub == 0 && r < s) B.part[int64_t(blk) * s + r] = wr;
    }
  }
  sr_block_sums<4>(&red[0][0], uu, fsl, FIRST, B, blk);
}

template <bool FIRST, bool LAST>
__global__ __launch_bounds__(256) void srank_generic_kernel(SrankArgs a, int32_t first_block) {
  __shared__ double red[4][256];
  const SrBlock sb = a.tab[first_block + (a.reverse ? int(gridDim.x) - 1 - int(blockIdx.x) : int(blockIdx.x))];
  const MuonMat& mm = a.mats[sb.mat];
  const SrBufs B = sr_bufs(a.ws, mm);
  const double inv = sr_inv_norm(mm, B, FIRST);
  if (mm.tall) {
    if (mm.vec_ok) srank_generic_tall<4, FIRST, LAST>(red, mm, a.bind[mm.tensor].m, B, sb.blk, inv);
    else srank_generic_tall<1, FIRST, LAST>(red, mm, a.bind[mm.tensor].m, B, sb.blk, inv);
  } else {
    if (mm.vec_ok) srank_generic_wide<4, FIRST, LAST>(red, mm, a.bind[mm.tensor].m, B, sb.blk, inv);
    else srank_generic_wide<1, FIRST, LAST>(red, mm, a.bind[mm.tensor].m, B, sb.blk, inv);
  }
}

__global__ __launch_bounds__(256) void srank_reduce_kernel(SrankArgs a) {
  __shared__ double red[4][kSrChunk];
  const int b = blockIdx.x;
  const int mi = find_segment(a.rd_start, a.n_mats, b);
  const MuonMat& mm = a.mats[mi];
  const SrBufs B = sr_bufs(a.ws, mm);
  const int chunk = b - a.rd_start[mi];
  const int tid = threadIdx.x, q = tid >> 6;
  const int j = chunk * kSrChunk + (tid & 63);
  double acc = 0.0;
  if (j < mm.s) {
#pragma unroll 4
    for (int bb = q; bb < mm.sr_blocks; bb += 4) acc += B.part[int64_t(bb) * mm.s + j];
  }
  red[q][tid & 63] = acc;
  __syncthreads();
  if (tid < 64) {
    double zj = (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
    if (j < mm.s) B.z[j] = zj;
    else zj = 0.0;
    const double sq = wave_sum_d(zj * zj);
    if (tid == 0) B.nrm[chunk] = sq;
  }
}

__global__ __launch_bounds__(256) void srank_decide_kernel(SrankArgs a) {
  __shared__ double red[4][2];
  const int i = blockIdx.x, tid = threadIdx.x;
  const int mi = a.tensor_mat[i];
  if (mi < 0) {
    if (tid == 0) {
      if (a.decisions_out) a.decisions_out[i] = 0;
      if (a.srank_out) a.srank_out[i] = -1.0;
    }
    return;
  }
  const MuonMat& mm = a.mats[mi];
  const SrBufs B = sr_bufs(a.ws, mm);
  double f = 0.0, u = 0.0;
  for (int bb = tid; bb < mm.sr_blocks; bb += 256) {
    f += B.fsq[bb];
    u += B.usq[bb];
  }
  f = wave_sum_d(f);
  u = wave_sum_d(u);
  if ((tid & 63) == 0) {
    red[tid >> 6][0] = f;
    red[tid >> 6][1] = u;
  }
  __syncthreads();
  if (tid == 0) {
    const double F = (red[0][0] + red[1][0]) + (red[2][0] + red[3][0]);
    const double U = (red[0][1] + red[1][1]) + (red[2][1] + red[3][1]);
    const double r = U > 0.0 ? F / U : 0.0;
    const int d = r <= a.alpha * double(mm.s) ? 1 : 0;
    a.decide[mi] = d;
    if (a.decisions_out) a.decisions_out[i] = d;
    if (a.srank_out) a.srank_out[i] = r;
  }
}

// ---------------------------------------------------------------------------
// Newton-Schulz GEMMs
// ---------------------------------------------------------------------------
// C[BT x BT] = sum_k Aop[row0 + i][k] * Bop[col0 + j][k]: both operands are
// K-contiguous ("NT"), except the apply's X, which is staged k-major and read
// with transpose reads. K is staged through LDS 128 bytes per row at a time by
// direct global->LDS loads (no register staging), double buffered: the loads
// of stage k+1 are in flight while stage k feeds the MFMAs (the bf16 apply
// on 128- and 64-tiles keeps four stages, three in flight). Rows are
// unpadded; their eight 16-byte chunks are XOR-swizzled by row so that the
// 128-bit fragment reads, served 16 lanes (16 rows) per LDS cycle across 64
// banks, are bank-conflict free.
//   BT = 256: 8 waves (2 x 4), each a 128 x 64 sub-tile of 4 x 2 MFMA 32x32
//             blocks (32 B of operand loads per CU-clock at full MFMA rate);
//   BT = 128: 4 waves (2 x 2), each a 64 x 64 sub-tile of 2 x 2 blocks, for
//             stages with too few 256-tiles to fill the chip;
//   BT = 64:  4 waves (2 x 2), each one 32 x 32 block (fp32 products with
//             too few 128-tiles to fill the chip, and the bf16 apply's last
//             round when sixteen times its leftover 256-tiles fit one round).
// Accumulator element r of block (mi, ni) sits at row
// wm + 32 mi + 8 (r / 4) + 4 (lane / 32) + r % 4, col wn + 32 ni + lane % 32.
// Wait until at most N vector-memory operations of this wave are outstanding
// (they complete in the order they were issued).
// (the builtin, not inline assembly: the compiler then knows which
// operations have completed and adds no waits of its own for them)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // s_waitcnt fields: vmcnt[3:0] in bits 3:0, vmcnt[5:4] in 15:14; expcnt
  // (6:4) and lgkmcnt (11:8) at their maxima, i.e. not waited for
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Descriptor tables are read through the constant address space: they are
// never written while a kernel runs, so the compiler may fetch them with
// scalar loads even after the kernel's own stores.
template <class U>
__device__ __forceinline__ const __attribute__((address_space(4))) U* kconst(const U* p) {
  return (const __attribute__((address_space(4))) U*)(p);
}

// Workgroup barrier that orders LDS accesses only: unlike __syncthreads it
// does not wait for this wave's outstanding global stores, so output tiles
// drain to memory while the workgroup goes on.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Lane exchanges within a quad of lanes through DPP (no LDS traffic).
__device__ __forceinline__ float dpp_quad_xor1(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1,
                                                            0xF, 0xF, true));   // [1,0,3,2]
}
__device__ __forceinline__ float dpp_quad_xor2(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E,
                                                            0xF, 0xF, true));   // [2,3,0,1]
}

// 4 x 4 transpose across the quad: lane b enters with v[e] = C[e][b] and
// leaves with v[j] = C[b][j]. Two exchange rounds (partners b ^ 2, then
// b ^ 1), each lane sending two values and receiving two.
__device__ __forceinline__ void quad_transpose(float v[4], int b) {
  const bool lo = b < 2;
  float s0 = dpp_quad_xor2(lo ? v[2] : v[0]);
  float s1 = dpp_quad_xor2(lo ? v[3] : v[1]);
  if (lo) { v[2] = s0; v[3] = s1; } else { v[0] = s0; v[1] = s1; }
  const bool even = (b & 1) == 0;
  s0 = dpp_quad_xor1(even ? v[1] : v[0]);
  s1 = dpp_quad_xor1(even ? v[3] : v[2]);
  if (even) { v[1] = s0; v[3] = s1; } else { v[0] = s0; v[2] = s1; }
}

// Scheduling directives for the MFMA k-steps of one stage: NM MFMAs with the
// next k-step's NR LDS fragment reads placed one after each of the first NR
// MFMAs, so the matrix core is not left waiting for a whole batch of reads.
template <int I, int NM, int NR>
__device__ __forceinline__ void sched_mfma_reads() {
  if constexpr (I < NM) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if constexpr (I < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    sched_mfma_reads<I + 1, NM, NR>();
  } else if constexpr (NR > NM) {
    __builtin_amdgcn_sched_group_barrier(0x100, NR - NM, 0);
  }
}
template <int S, int NM, int NR>
__device__ __forceinline__ void sched_interleave() {
  if constexpr (S > 0) {
    sched_mfma_reads<0, NM, NR>();
    sched_interleave<S - 1, NM, NR>();
  }
}

template <typename T> struct Mfma;

template <> struct Mfma<bf16> {
  static constexpr int kBK = 64;      // K per stage (128 bytes)
  static constexpr int kKStep = 16;   // K per MFMA
  typedef bf16x8 Frag;
  __device__ static __forceinline__ Frag load(const bf16* row, int lk) {
    return *reinterpret_cast<const bf16x8*>(row + lk * 8);
  }
  __device__ static __forceinline__ f32x16 mma(Frag a, Frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mfma<float> {
  static constexpr int kBK = 32;
  static constexpr int kKStep = 2;
  typedef float Frag;
  __device__ static __forceinline__ Frag load(const float* row, int lk) { return row[lk]; }
  __device__ static __forceinline__ f32x16 mma(Frag a, Frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

template <int BT> struct TileGeom {
  static constexpr int kWM = BT == 256 ? 128 : BT / 2;   // wave sub-tile rows
  static constexpr int kWN = BT == 64 ? 32 : 64;          // wave sub-tile cols
  static constexpr int kWavesN = BT / kWN;
  static constexpr int kThreads = (BT / kWM) * kWavesN * 64;
  static constexpr int kMI = kWM / 32, kNI = kWN / 32;
};

struct GemmArgs {
  const MuonMat* mats;
  const TensorPtrs* bind;
  const GemmTask* tasks;
  const XcdSplit* split;
  void* ws;
  const float* rscale;
  const int32_t* decide;
  int32_t src, first, last, store_o;
  int32_t xcds;                  // workgroup i runs on XCD i mod xcds
  float a, b, c, lr, wd;
};

// LDS of one product tile: kNBuf operand stages during the K loop, then the
// output tile (the kernel declares it; the tile body takes a pointer).
template <typename T, int MODE, int BT>
struct GemmLds {
  static constexpr int kLd = Mfma<T>::kBK;      // LDS row: 128 bytes
  static constexpr int kStR = BT + 16;          // row-major staging row stride
  // Two stages, except for the bf16 apply on 128- or 64-tiles (a nearly
  // empty last round of 256-tiles, one or two such workgroups per CU and too
  // few of them to hide load latency with other workgroups): four, three of
  // them in flight while one feeds the MFMAs.
  static constexpr int kNBuf = (MODE == kApply && BT <= 128 && sizeof(T) == 2) ? 4 : 2;
  static constexpr int kOperand = kNBuf * 2 * BT * kLd, kStage = BT * kStR;
  static constexpr int kElems = kOperand > kStage ? kOperand : kStage;
  static constexpr int kBytes = kElems * int(sizeof(T));
};

// LAST (apply only): the last Newton-Schulz step, whose epilogue updates W
// (its own instantiation: that epilogue's registers would otherwise weigh
// on every other apply step). `smem` is the kernel's LDS block (at least
// GemmLds<T, MODE, BT>::kBytes); the workgroup is number `bid` of the `nblk`
// that run this task list (workgroup i on XCD i mod xcds).
template <typename T, int MODE, int BT, bool LAST = false>
__device__ __forceinline__ void gemm_body(const GemmArgs& g, T* smem, int bid, int nblk) {
  using M = Mfma<T>;
  using Geo = TileGeom<BT>;
  constexpr int kBK = M::kBK;
  constexpr int kEpc = 16 / sizeof(T);           // elements per 16-byte chunk
  constexpr int kLd = kBK;                       // LDS row: 128 bytes, chunks XOR-swizzled
  constexpr int kNT = Geo::kThreads;
  constexpr int kMI = Geo::kMI, kNI = Geo::kNI;
  // Output staging row strides: kStR for row-major staging (16-byte-aligned
  // rows, 8 or 16 dwords apart modulo the 64 banks, so a quad of lanes
  // writing 4 consecutive rows never collides), kStC for transposed staging
  // (4 dwords apart, so 16 lanes writing 16 consecutive rows never collide).
  using L = GemmLds<T, MODE, BT>;
  constexpr int kStR = L::kStR, kStC = BT + kEpc;
  constexpr int kNBuf = L::kNBuf;
  T (*sA)[BT][kLd] = reinterpret_cast<T (*)[BT][kLd]>(smem);
  T (*sB)[BT][kLd] = reinterpret_cast<T (*)[BT][kLd]>(smem + kNBuf * BT * kLd);
  // apply: the B operand (X, K = s along its rows) is staged k-major as
  // kBK rows of BT elements (512 bytes) and read transposed
  constexpr bool kBRows = MODE == kApply;
  T (*sBr)[kBK][BT] = reinterpret_cast<T (*)[kBK][BT]>(smem + kNBuf * BT * kLd);

  // The workgroups of an XCD walk that XCD's tile list with a stride of
  // their number, skipping the tiles of matrices whose adaptive decision
  // went the other way. Only the non-final apply is persistent (a grid of
  // one round, several tiles per workgroup): its epilogue stores from
  // registers, so the next tile's loads overlap them. The other products
  // stage their results through the whole LDS and run one tile per
  // workgroup, so a finished workgroup's successor starts at once.
  constexpr bool kPersistent = MODE == kApply && !LAST;
  const int xcds = g.xcds;
  const int xcd = bid % xcds;
  const int count = kconst(g.split)->count[xcd];
  const auto* tasks = kconst(g.tasks) + kconst(g.split)->start[xcd];
  const int step = nblk / xcds;
  auto live = [&](int s) {
    while (s < count && g.decide && kconst(g.decide)[tasks[s].mat] == 0) s += step;
    return s;
  };
  char* wsb = static_cast<char*>(g.ws);
  auto at = [&](int64_t off) { return reinterpret_cast<T*>(wsb + off); };
  // Non-final apply steps store X' straight from registers; the next tile's
  // first stage is requested during the current tile's last K stage, so it
  // loads while that stage runs and the stores drain. kDirect is the number
  // of those stores per lane.
  constexpr int kDirect = Geo::kMI * Geo::kNI * 4;
  bool prefetched = false;
  int base = 0;                                  // LDS buffer of the tile's first K stage
  for (int slot = live(bid / xcds); slot < count;) {
  // Lane-derived values are recomputed for every tile (the empty asm keeps
  // the compiler from hoisting them out of the tile loop, where they would
  // stay live, in registers, through the epilogue).
  int tid = threadIdx.x;
  if constexpr (kPersistent) asm volatile("" : "+v"(tid));
  __builtin_assume(tid >= 0 && tid < kNT);

  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int wm = (wave / Geo::kWavesN) * Geo::kWM, wn = (wave % Geo::kWavesN) * Geo::kWN;

  // Physical chunk of logical chunk c in row `row` is c ^ swz(row): among
  // any 16 consecutive rows the two rows of each parity class (which share a
  // bank half) get distinct chunks.
  auto swz = [](int row) { return (row & 7) ^ ((row >> 3) & 1); };
  // Each wave instruction fills 8 rows (1 KB): lane L writes row L/8,
  // physical chunk L%8, and fetches the logical chunk that lands there.
  constexpr int kWaves = kNT / 64;
  // Waves that issue the operand copies: on 256-tiles only the first four
  // (one per SIMD), so that the other wave of each SIMD keeps the matrix core
  // busy while the issuing wave stalls on a full memory pipeline (measured:
  // apply 0.5-0.9%, Gram 1-4%, polynomial 0-2.5% faster at 124M-720M); on
  // the 128-tiles of the Gram and polynomial products the first two
  // (polynomial 2.5% faster at 124M).
  constexpr int kDmaWaves = (BT == 256 || (BT == 128 && MODE != kApply)) ? kWaves / 2 : kWaves;
  constexpr int kInst = BT / 8 / kDmaWaves;      // wave instructions per operand per stage
  // k-major B rows (apply): kChunksB 16-byte chunks per row, each wave
  // instruction fills kRpiB rows; chunks are XOR-swizzled by swb(k) so that
  // the 4 rows x 64 bytes a transpose read serves per LDS cycle (32 lanes)
  // fall into disjoint bank ranges.
  constexpr int kChunksB = BT * int(sizeof(T)) / 16;
  constexpr int kRpiB = 64 / kChunksB;
  constexpr int kInstB = kBK / kRpiB / kDmaWaves;
  static_assert(!kBRows || kInstB * kRpiB * kDmaWaves == kBK, "B rows split evenly over the waves");
  // (bf16 rows of 64 elements are only 8 chunks: there the 4 rows of a read
  // take chunk offsets 0, 0, 4, 4, which with the 128-byte row stride puts
  // them in 4 distinct quarters of the banks)
  auto swb = [](int k) { return (sizeof(T) == 2 && BT == 64) ? ((k >> 1) & 1) * 4 : (k & 3) * 4; };
  // Operands of one tile. Copy addresses are a wave-uniform base (operand,
  // K offset, instruction) plus one loop-invariant 32-bit byte offset per
  // lane and operand. Because kWaves (and kWaves * kRpiB) is even (a
  // multiple of 4), the swizzle of a lane's row does not depend on the
  // instruction index.
  static_assert(kDmaWaves % 2 == 0 && (kDmaWaves * kRpiB) % 4 == 0, "swizzle independent of the instruction");
  struct Ops {
    const T* a;
    const T* b;
    int64_t lda, ldb;
    int K;
    uint32_t a_off, b_off;
    bool same;                                   // symmetric product, diagonal tile: B rows = A rows
  };
  auto make_ops = [&](const __attribute__((address_space(4))) GemmTask& t) {
    const auto& m = kconst(g.mats)[t.mat];
    // ping-pong buffers chosen without indexing (keeps descriptors out of scratch)
    const int64_t xcur = g.src ? m.off_x[1] : m.off_x[0];
    Ops o;
    if (MODE == kGram) {
      o.a = o.b = at(xcur);
      o.lda = o.ldb = m.l_pad;
      o.K = int(m.l_pad);
    } else if (MODE == kPoly) {
      o.a = o.b = at(m.off_a);
      o.lda = o.ldb = m.s_pad;
      o.K = int(m.s_pad);
    } else {
      o.a = at(m.off_b);
      o.b = at(xcur);
      o.lda = m.s_pad;
      o.ldb = m.l_pad;
      o.K = int(m.s_pad);
    }
    o.a += int64_t(t.tm) * BT * o.lda;
    o.b += kBRows ? int64_t(t.tn) * BT : int64_t(t.tn) * BT * o.ldb;
    const int dw = wave % kDmaWaves;             // (only issuing waves use the offsets)
    o.a_off = uint32_t(((dw * 8 + (lane >> 3)) * o.lda + ((lane & 7) ^ swz(dw * 8 + (lane >> 3))) * kEpc) * sizeof(T));
    o.b_off = kBRows
        ? uint32_t(((dw * kRpiB + lane / kChunksB) * o.ldb + ((lane % kChunksB) ^ swb(dw * kRpiB + lane / kChunksB)) * kEpc) * sizeof(T))
        : uint32_t(((dw * 8 + (lane >> 3)) * o.ldb + ((lane & 7) ^ swz(dw * 8 + (lane >> 3))) * kEpc) * sizeof(T));
    o.same = MODE != kApply && sizeof(T) == 2 && t.tm == t.tn;
    return o;
  };
  // One 16-byte-per-lane copy in the scalar-base form: wave-uniform base
  // address and LDS destination (M0, one wait state after writing it) in
  // scalar registers, one 32-bit offset per lane. Written as an assembly
  // block: from the builtin, inside the K loop, the compiler formed 64-bit
  // per-lane addresses and moved M0 from vector registers for every copy
  // (apply 2-5%, polynomial 5% slower). The compiler neither counts these
  // copies nor waits for them: every wait for them is explicit (wait_stage).
  // M0 is reserved to the compiler, which does not track the clobber; no
  // other code in these kernels uses M0.
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  auto copy16 = [&](const T* src, uint32_t off, const T* dst) {
    const uint32_t d = uint32_t(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const T*)(dst)));
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(off), "s"(src), "s"(d) : "memory", "m0");
  };
  auto dma = [&](const Ops& o, int buf, int k0) {
    if (wave_u >= kDmaWaves) return;
#pragma unroll
    for (int q = 0; q < kInst; ++q) {
      const int blk = q * kDmaWaves + wave_u;    // 8-row block
      copy16(o.a + int64_t(q * kDmaWaves * 8) * o.lda + k0, o.a_off, &sA[buf][blk * 8][0]);
      if constexpr (!kBRows)
        if (!o.same) copy16(o.b + int64_t(q * kDmaWaves * 8) * o.ldb + k0, o.b_off, &sB[buf][blk * 8][0]);
    }
    if constexpr (kBRows) {
#pragma unroll
      for (int q = 0; q < kInstB; ++q) {
        const int rr = (q * kDmaWaves + wave_u) * kRpiB;  // first of the instruction's rows
        copy16(o.b + int64_t(k0 + q * kDmaWaves * kRpiB) * o.ldb, o.b_off, &sBr[buf][rr][0]);
      }
    }
  };
  constexpr int kOps = kInst + (kBRows ? kInstB : kInst);   // copies per issuing wave per stage
  static_assert(kDirect + (kNBuf - 1) * kOps < 64, "outstanding vector memory operations fit the counter");
  const auto& task = tasks[slot];
  const auto& mm = kconst(g.mats)[task.mat];
  const int64_t off_x_nxt = g.src ? mm.off_x[0] : mm.off_x[1];
  const Ops ops = make_ops(task);
  const int K = ops.K;
  // A bf16 diagonal tile of a symmetric product reads its B fragments from
  // the A operand's buffers (the same rows of X, or of A) and copies only
  // those: Gram 3-4%, polynomial 2-4% faster at 124M-720M (the fp32 small
  // tiles were 1% slower with it and keep both copies).
  T (*sBf)[BT][kLd] = ops.same ? sA : sB;
  const int row0 = task.tm * BT, col0 = task.tn * BT;

  f32x16 acc[kMI][kNI];
#pragma unroll
  for (int i = 0; i < kMI; ++i)
#pragma unroll
    for (int j = 0; j < kNI; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  auto frag = [&](const T* rowp, int row, int kc) {
    const int e = kc + lk * (M::kKStep / 2);
    const int off = (((e / kEpc) ^ swz(row)) * kEpc) + (e % kEpc);
    return M::load(rowp + off, 0);
  };
  // B fragment of block column j from k-major rows: the MFMA wants, in lane
  // (n = lane % 32, half lk), B[kc + lk kKStep/2 + t][n] for t < kKStep/2.
  // fp32 apply: B fragment of block column j from the k-major rows (one
  // element per lane: B[kc + lk][n]); the bf16 apply reads its fragments
  // with transpose reads (preload_b below)
  auto frag_b_rows = [&](int buf, int j, int kc) -> typename M::Frag {
    const int k = kc + lk, n = wn + 32 * j + lr;
    return sBr[buf][k][(((n >> 2) ^ swb(k)) << 2) + (n & 3)];
  };
  constexpr int kSub = kBK / M::kKStep;
  // bf16 apply: the B fragments of a whole stage are read into registers
  // (transpose reads) at the start of the stage, right after the next
  // stage's copies are issued.
  constexpr bool kTrB = kBRows && sizeof(T) == 2;
  typename M::Frag bq[kTrB ? kSub : 1][kNI];
  // The 16 (64-tiles: 8) transpose reads of a stage are one assembly block that ends by
  // waiting for them: the compiler's own form of the read counts as touching
  // memory it cannot see and would first wait for every outstanding global
  // access, including the previous tile's stores still draining. Read
  // (kk, j, t) is at the lane's address for column block j plus
  // (16 kk + 4 t) rows of BT elements. The MFMA wants, in lane (n =
  // lane % 32, half lk), B[kc + 8 lk + t][n] for t < 8: two transpose reads
  // of 4 k each. Within each 16-lane group, lane m points at row
  // kb + (m >> 2), columns n0 + 4 (m & 3) .. +3, and receives column n0 + m
  // of rows kb .. kb + 3.
  auto preload_b = [&](int buf) {
    if constexpr (kTrB) {
      static_assert(kSub == 4 && ((kNI == 2 && (BT == 256 || BT == 128)) || (kNI == 1 && BT == 64)),
                    "transpose-read block layout");
      uint32_t base[kNI];
#pragma unroll
      for (int j = 0; j < kNI; ++j) {
        const int grp = lane >> 4, m = lane & 15;
        const int n = wn + 32 * j + 16 * (grp & 1) + 4 * (m & 3);
        const int k = 8 * (grp >> 1) + (m >> 2);
        const int off = (((n >> 3) ^ swb(k)) << 3) + (n & 7);
        // (a C cast: it converts the generic pointer to the LDS address space)
        base[j] = uint32_t(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) T*)(&sBr[buf][k][off])));
      }
      u32x2 h[8 * kNI];
      if constexpr (BT == 256) {
        asm volatile(
            "ds_read_b64_tr_b16 %0, %16\n"
            "ds_read_b64_tr_b16 %1, %16 offset:2048\n"
            "ds_read_b64_tr_b16 %2, %17\n"
            "ds_read_b64_tr_b16 %3, %17 offset:2048\n"
            "ds_read_b64_tr_b16 %4, %16 offset:8192\n"
            "ds_read_b64_tr_b16 %5, %16 offset:10240\n"
            "ds_read_b64_tr_b16 %6, %17 offset:8192\n"
            "ds_read_b64_tr_b16 %7, %17 offset:10240\n"
            "ds_read_b64_tr_b16 %8, %16 offset:16384\n"
            "ds_read_b64_tr_b16 %9, %16 offset:18432\n"
            "ds_read_b64_tr_b16 %10, %17 offset:16384\n"
            "ds_read_b64_tr_b16 %11, %17 offset:18432\n"
            "ds_read_b64_tr_b16 %12, %16 offset:24576\n"
            "ds_read_b64_tr_b16 %13, %16 offset:26624\n"
            "ds_read_b64_tr_b16 %14, %17 offset:24576\n"
            "ds_read_b64_tr_b16 %15, %17 offset:26624\n"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(h[0]), "=&v"(h[1]), "=&v"(h[2]), "=&v"(h[3]), "=&v"(h[4]), "=&v"(h[5]), "=&v"(h[6]), "=&v"(h[7]),
              "=&v"(h[8]), "=&v"(h[9]), "=&v"(h[10]), "=&v"(h[11]), "=&v"(h[12]), "=&v"(h[13]), "=&v"(h[14]), "=&v"(h[15])
            : "v"(base[0]), "v"(base[1])
            : "memory");
      } else if constexpr (BT == 128) {
        asm volatile(
            "ds_read_b64_tr_b16 %0, %16\n"
            "ds_read_b64_tr_b16 %1, %16 offset:1024\n"
            "ds_read_b64_tr_b16 %2, %17\n"
            "ds_read_b64_tr_b16 %3, %17 offset:1024\n"
            "ds_read_b64_tr_b16 %4, %16 offset:4096\n"
            "ds_read_b64_tr_b16 %5, %16 offset:5120\n"
            "ds_read_b64_tr_b16 %6, %17 offset:4096\n"
            "ds_read_b64_tr_b16 %7, %17 offset:5120\n"
            "ds_read_b64_tr_b16 %8, %16 offset:8192\n"
            "ds_read_b64_tr_b16 %9, %16 offset:9216\n"
            "ds_read_b64_tr_b16 %10, %17 offset:8192\n"
            "ds_read_b64_tr_b16 %11, %17 offset:9216\n"
            "ds_read_b64_tr_b16 %12, %16 offset:12288\n"
            "ds_read_b64_tr_b16 %13, %16 offset:13312\n"
            "ds_read_b64_tr_b16 %14, %17 offset:12288\n"
            "ds_read_b64_tr_b16 %15, %17 offset:13312\n"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(h[0]), "=&v"(h[1]), "=&v"(h[2]), "=&v"(h[3]), "=&v"(h[4]), "=&v"(h[5]), "=&v"(h[6]), "=&v"(h[7]),
              "=&v"(h[8]), "=&v"(h[9]), "=&v"(h[10]), "=&v"(h[11]), "=&v"(h[12]), "=&v"(h[13]), "=&v"(h[14]), "=&v"(h[15])
            : "v"(base[0]), "v"(base[1])
            : "memory");
      } else {
        asm volatile(
            "ds_read_b64_tr_b16 %0, %8\n"
            "ds_read_b64_tr_b16 %1, %8 offset:512\n"
            "ds_read_b64_tr_b16 %2, %8 offset:2048\n"
            "ds_read_b64_tr_b16 %3, %8 offset:2560\n"
            "ds_read_b64_tr_b16 %4, %8 offset:4096\n"
            "ds_read_b64_tr_b16 %5, %8 offset:4608\n"
            "ds_read_b64_tr_b16 %6, %8 offset:6144\n"
            "ds_read_b64_tr_b16 %7, %8 offset:6656\n"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(h[0]), "=&v"(h[1]), "=&v"(h[2]), "=&v"(h[3]), "=&v"(h[4]), "=&v"(h[5]), "=&v"(h[6]), "=&v"(h[7])
            : "v"(base[0])
            : "memory");
      }
#pragma unroll
      for (int kk = 0; kk < kSub; ++kk)
#pragma unroll
        for (int j = 0; j < kNI; ++j) {
          const bf16x4 lo = __builtin_bit_cast(bf16x4, h[(kk * kNI + j) * 2]);
          const bf16x4 hi = __builtin_bit_cast(bf16x4, h[(kk * kNI + j) * 2 + 1]);
          bq[kk][j] = typename M::Frag{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        }
    }
  };
  auto compute = [&](int buf) {
    // fragments double-buffered in registers: the LDS reads of substep kk+1
    // are issued before the MFMAs of substep kk
    typename M::Frag af[2][kMI], bfr[2][kNI];
    auto fetch = [&](int s, int kk) {
      const int kc = kk * M::kKStep;
#pragma unroll
      for (int i = 0; i < kMI; ++i) af[s][i] = frag(&sA[buf][wm + 32 * i + lr][0], wm + 32 * i + lr, kc);
#pragma unroll
      for (int j = 0; j < kNI; ++j) {
        if constexpr (kTrB) bfr[s][j] = bq[kk][j];
        else if constexpr (kBRows) bfr[s][j] = frag_b_rows(buf, j, kc);
        else bfr[s][j] = frag(&sBf[buf][wn + 32 * j + lr][0], wn + 32 * j + lr, kc);
      }
    };
    fetch(0, 0);
#pragma unroll
    for (int kk = 0; kk < kSub; ++kk) {
      if (kk + 1 < kSub) fetch((kk + 1) & 1, kk + 1);
#pragma unroll
      for (int i = 0; i < kMI; ++i)
#pragma unroll
        for (int j = 0; j < kNI; ++j) acc[i][j] = M::mma(af[kk & 1][i], bfr[kk & 1][j], acc[i][j]);
    }
    // region order: the first fragment reads, then per k-step the MFMAs
    // interleaved with the next k-step's reads, then the last k-step's MFMAs
    constexpr int kReads = kMI + (kTrB ? 0 : kNI * (kBRows ? 2 : 1));
    __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
    sched_interleave<kSub - 1, kMI * kNI, kReads>();
    __builtin_amdgcn_sched_group_barrier(0x008, kMI * kNI, 0);
  };

  // The barrier after each stage both publishes the stage just loaded (every
  // wave has waited for its own loads) and frees the buffer just read.
  const int nk = K / kBK;
  // Wait until stage `s` has landed when `later` stages were requested after
  // it (and, for a prefetched first stage, this wave's stores in between).
  auto wait_stage = [&](int later, bool stores) {
    if constexpr (kNBuf == 2) {
      if (stores) wait_vmcnt<kDirect>();
      else wait_vmcnt<0>();
    } else {
      static_assert(kNBuf == 4, "stage waits written out for 2 or 4 buffers");
      // the counts assume kOps copies per stage: a diagonal tile of a
      // symmetric product copies one operand only
      static_assert(MODE == kApply, "four stages only for the apply");
      const int n = later < kNBuf - 2 ? later : kNBuf - 2;
      if (stores) {
        if (n >= 2) wait_vmcnt<kDirect + 2 * kOps>();
        else if (n == 1) wait_vmcnt<kDirect + kOps>();
        else wait_vmcnt<kDirect>();
      } else {
        if (n >= 2) wait_vmcnt<2 * kOps>();
        else if (n == 1) wait_vmcnt<kOps>();
        else wait_vmcnt<0>();
      }
    }
  };
  // stages 0 .. kNBuf - 2 in flight before the first MFMA (stage 0 may have
  // been requested already, during the previous tile's last K stage)
  if (!prefetched) dma(ops, base, 0);
#pragma unroll
  for (int st = 1; st < kNBuf - 1; ++st)
    if (st < nk) dma(ops, (base + st) & (kNBuf - 1), st * kBK);
  wait_stage(nk - 1, prefetched);
  prefetched = false;
  lds_barrier();
  // persistent apply: the next tile's first stage is requested at the start
  // of this tile's last stage, into the buffer no stage of this tile uses
  // then, so that it lands during that stage and the epilogue
  const int nslot = live(slot + step);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = (base + kt) & (kNBuf - 1);
    // the next stage's copies go out first, into the buffer of stage kt - 1,
    // which every wave finished before the barrier that ended the previous
    // step: their issue (which stalls while the memory pipeline is full)
    // then overlaps this stage's transpose reads (an assembly block: the
    // compiler adds no wait for the copies before it)
    const int nxt = kt + kNBuf - 1;
    if (nxt < nk) dma(ops, (base + nxt) & (kNBuf - 1), nxt * kBK);
    if (kPersistent && kt == nk - 1 && nslot < count) {
      dma(make_ops(tasks[nslot]), (base + nk) & (kNBuf - 1), 0);
      prefetched = true;
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (kTrB) {
      preload_b(buf);
      __builtin_amdgcn_sched_barrier(0);
    }
    compute(buf);
    __builtin_amdgcn_sched_barrier(0);
    // stage kt + 1 (after the last stage nothing: the next tile's first
    // stage stays in flight)
    if (kt < nk - 1) wait_stage(nk - 2 - kt, false);
    lds_barrier();
  }
  // (the barrier after the last stage means no wave reads the operand
  // buffers any more)
  if (kPersistent) base = (base + nk) & (kNBuf - 1);

  // ---- epilogues ----------------------------------------------------------
  // The Gram and polynomial results leave through LDS: each lane writes its
  // values into the staging tile (row-major, or transposed with 8-byte
  // writes), then the workgroup stores whole rows with coalesced 16-byte
  // stores. The non-final apply stores from registers; the last one stages
  // its fp32 direction through LDS to update W.
  const int64_t s_pad = mm.s_pad, l_pad = mm.l_pad;
  T (*stage)[kStR] = reinterpret_cast<T (*)[kStR]>(smem);
  T (*stage_t)[kStC] = reinterpret_cast<T (*)[kStC]>(smem);
  constexpr int kRowChunks = BT * int(sizeof(T)) / 16;
  auto flush = [&](T* dst, int64_t ld, const T* stg, int stride) {  // staged tile -> dst rows
    lds_barrier();
#pragma unroll 4
    for (int c = tid; c < BT * kRowChunks; c += kNT) {
      const int r = c / kRowChunks, ch = (c % kRowChunks) * kEpc;
      *reinterpret_cast<u32x4*>(dst + r * ld + ch) = *reinterpret_cast<const u32x4*>(stg + r * stride + ch);
    }
    lds_barrier();
  };
  // v(mi, ni, q, e): value of local row wm + 32 mi + 8 q + 4 lk + e, local
  // column wn + 32 ni + lr. Row-major staging first transposes each 4 x 4
  // block within a quad of lanes (DPP, no LDS traffic), so that every lane
  // writes 4 consecutive columns of one row in a single store.
  auto stage_rows = [&](auto&& val) {
    const int b = lane & 3;
#pragma unroll
    for (int mi = 0; mi < kMI; ++mi)
#pragma unroll
      for (int ni = 0; ni < kNI; ++ni)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = val(mi, ni, q, e);
          quad_transpose(v, b);
          const int r = wm + 32 * mi + 8 * q + 4 * lk + b, c = wn + 32 * ni + (lr & ~3);
          store4(&stage[r][c], v);
        }
  };
  auto stage_cols = [&](auto&& val) {           // transposed: stage_t[col][row..row+3]
#pragma unroll
    for (int mi = 0; mi < kMI; ++mi)
#pragma unroll
      for (int ni = 0; ni < kNI; ++ni)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int r = wm + 32 * mi + 8 * q + 4 * lk, c = wn + 32 * ni + lr;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = val(mi, ni, q, e);
          store4(&stage_t[c][r], v);
        }
  };

  if (MODE == kGram || MODE == kPoly) {
    float alpha = 1.0f;
    if (MODE == kGram && g.first) {
      const float r = kconst(g.rscale)[task.mat];
      alpha = r * r;
    }
    if (MODE == kPoly) {
      // B' = a I + b A + c A A (the a X term of the apply step folded into
      // B'). The old A is read in the accumulator layout: for each of a
      // lane's rows, the 32 lanes of a half-wave read 32 consecutive columns.
      const T* aold = at(mm.off_a);
      const bool diag = task.tm == task.tn;
#pragma unroll
      for (int mi = 0; mi < kMI; ++mi)
#pragma unroll
        for (int ni = 0; ni < kNI; ++ni)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int r = wm + 32 * mi + 8 * q + 4 * lk, c = wn + 32 * ni + lr;
            float old[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) old[e] = float(aold[int64_t(row0 + r + e) * s_pad + col0 + c]);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float v = fmaf(g.b, old[e], g.c * acc[mi][ni][4 * q + e]);
              if (diag && r + e == c) v += g.a;
              acc[mi][ni][4 * q + e] = v;
            }
          }
    }
    T* out = at(MODE == kGram ? mm.off_a : mm.off_b);
    auto val = [&](int mi, int ni, int q, int e) { return alpha * acc[mi][ni][4 * q + e]; };
    stage_rows(val);
    flush(out + row0 * s_pad + col0, s_pad, &stage[0][0], kStR);
    if (task.tm != task.tn) {                    // mirror into the upper triangle
      stage_cols(val);
      flush(out + col0 * s_pad + row0, s_pad, &stage_t[0][0], kStC);
    }
  } else {
    // X' = alpha B' X with B' = a I + b A + c A A from the polynomial step
    // (alpha, the Frobenius scaling, only on the first step)
    if (g.first) {
      const float alpha = kconst(g.rscale)[task.mat];
#pragma unroll
      for (int mi = 0; mi < kMI; ++mi)
#pragma unroll
        for (int ni = 0; ni < kNI; ++ni)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[mi][ni][r] *= alpha;
    }
    if constexpr (!LAST) {
      T* out = at(off_x_nxt) + row0 * l_pad + col0;
      const int b = lane & 3;
      if constexpr (sizeof(T) == 2 && kNI == 2) {
        // Each quad of lanes transposes its 4 x 4 blocks (DPP), so that a
        // lane holds 4 consecutive columns of one row in each of the two
        // column blocks; then the two half-waves trade the second block of
        // the first half's rows for the first block of the second half's
        // (v_permlane32_swap). One store then writes 4 rows x 64 columns,
        // four whole 128-byte lines, where 8 rows x 32 columns (eight half
        // lines) took twice as long per byte. The stores are non-temporal:
        // a round of tiles writes as many bytes of X' as the L2 caches of
        // all XCDs hold, and would otherwise evict the operands the next
        // tiles read (apply 3.7% faster at 124M, 1.5% slower at 355M).
#pragma unroll
        for (int mi = 0; mi < kMI; ++mi)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            uint32_t h0[2], h1[2];               // rows 8 q + 4 lk + b, column block 0 / 1
#pragma unroll
            for (int ni = 0; ni < 2; ++ni) {
              float v[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = acc[mi][ni][4 * q + e];
              quad_transpose(v, b);
              uint32_t* h = ni == 0 ? h0 : h1;
              h[0] = pack_bf16x2(v[0], v[1]);
              h[1] = pack_bf16x2(v[2], v[3]);
            }
            // lanes 32..63 of h0 <-> lanes 0..31 of h1: then h0 holds row
            // 8 q + b and h1 row 8 q + 4 + b, column block lk
#pragma unroll
            for (int k = 0; k < 2; ++k) {
              const auto sw = __builtin_amdgcn_permlane32_swap(h0[k], h1[k], false, false);
              h0[k] = sw[0];
              h1[k] = sw[1];
            }
            const int r = wm + 32 * mi + 8 * q + b, c = wn + 32 * lk + (lr & ~3);
            __builtin_nontemporal_store(u32x2{h0[0], h0[1]}, reinterpret_cast<u32x2*>(out + r * l_pad + c));
            __builtin_nontemporal_store(u32x2{h1[0], h1[1]}, reinterpret_cast<u32x2*>(out + (r + 4) * l_pad + c));
          }
      } else {
        // each quad of lanes transposes its 4 x 4 blocks (DPP) so that every
        // lane stores 4 consecutive columns of one row
#pragma unroll
        for (int mi = 0; mi < kMI; ++mi)
#pragma unroll
          for (int ni = 0; ni < kNI; ++ni)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              float v[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = acc[mi][ni][4 * q + e];
              quad_transpose(v, b);
              const int r = wm + 32 * mi + 8 * q + 4 * lk + b, c = wn + 32 * ni + (lr & ~3);
              store4(out + r * l_pad + c, v);
            }
      }
    } else {
      // last step: W <- W - lr (kappa O + wd W), or O = kappa X_K (NS hook).
      // O is X_K, transposed back for tall matrices. The fp32 O tile goes
      // through LDS in two halves of W rows so that W is read and written in
      // whole 16-byte pieces of its rows. Each thread's W pieces of a half
      // are requested before that half of O is staged, so their latency
      // overlaps the staging instead of being paid once per piece.
      constexpr int kHalf = BT / 2, kFs = BT + 4;
      constexpr int kIter = kHalf * (BT / 4) / kNT;   // 16-byte W pieces per thread per half
      static_assert(kIter * kNT == kHalf * (BT / 4), "W pieces split evenly over the threads");
      float (*fst)[kFs] = reinterpret_cast<float (*)[kFs]>(smem);
      const bool tall = mm.transposed != 0;
      float* Wp = kconst(g.bind)[mm.tensor].w;
      const int64_t wrow0 = tall ? col0 : row0, wcol0 = tall ? row0 : col0;
      const int64_t wrows = mm.rows, wcols = mm.cols;
      const float kappa = mm.kappa;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        f32x4 wv[kIter];
        if (!g.store_o) {
#pragma unroll
          for (int it = 0; it < kIter; ++it) {
            const int idx = tid + it * kNT;
            const int i = idx / (BT / 4), j = (idx % (BT / 4)) * 4;
            const int64_t gr = wrow0 + h * kHalf + i, gc = wcol0 + j;
            wv[it] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (mm.vec_ok && gr < wrows && gc + 3 < wcols)
              wv[it] = *reinterpret_cast<const f32x4*>(Wp + gr * wcols + gc);
          }
        }
#pragma unroll
        for (int mi = 0; mi < kMI; ++mi)
#pragma unroll
          for (int ni = 0; ni < kNI; ++ni)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int r = wm + 32 * mi + 8 * q + 4 * lk, c = wn + 32 * ni + lr;
              if (!tall) {
                if (wm / kHalf == h) {
#pragma unroll
                  for (int e = 0; e < 4; ++e) fst[r - h * kHalf + e][c] = kappa * acc[mi][ni][4 * q + e];
                }
              } else if ((wn + 32 * ni) / kHalf == h) {
                float o[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = kappa * acc[mi][ni][4 * q + e];
                store4(&fst[c - h * kHalf][r], o);
              }
            }
        lds_barrier();
#pragma unroll
        for (int it = 0; it < kIter; ++it) {
          const int idx = tid + it * kNT;
          const int i = idx / (BT / 4), j = (idx % (BT / 4)) * 4;
          const int64_t gr = wrow0 + h * kHalf + i, gc = wcol0 + j;
          if (gr >= wrows || gc >= wcols) continue;
          float* wp = Wp + gr * wcols + gc;
          float o[4];
          load4(&fst[i][j], o);
          if (mm.vec_ok && gc + 3 < wcols) {
            if (g.store_o) {
              store4(wp, o);
            } else {
              float w[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) w[e] = fmaf(-g.lr, fmaf(g.wd, wv[it][e], o[e]), wv[it][e]);
              store4(wp, w);
            }
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              if (gc + e >= wcols) break;
              if (g.store_o) {
                wp[e] = o[e];
              } else {
                const float w = wp[e];
                wp[e] = fmaf(-g.lr, fmaf(g.wd, w, o[e]), w);
              }
            }
          }
        }
        lds_barrier();
      }
    }
  }
  if constexpr (!kPersistent) break;            // one tile per workgroup (full grid)
  slot = nslot;
  }
}

// One entry point per Newton-Schulz product, so profiles name each stage.
template <typename T, int BT>
__global__ __launch_bounds__(TileGeom<BT>::kThreads) void ns_gram_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) char lds[GemmLds<T, kGram, BT>::kBytes];
  gemm_body<T, kGram, BT>(g, reinterpret_cast<T*>(lds), int(blockIdx.x), int(gridDim.x));
}
template <typename T, int BT>
__global__ __launch_bounds__(TileGeom<BT>::kThreads) void ns_poly_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) char lds[GemmLds<T, kPoly, BT>::kBytes];
  gemm_body<T, kPoly, BT>(g, reinterpret_cast<T*>(lds), int(blockIdx.x), int(gridDim.x));
}
template <typename T, int BT>
__global__ __launch_bounds__(TileGeom<BT>::kThreads) void ns_apply_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) char lds[GemmLds<T, kApply, BT>::kBytes];
  gemm_body<T, kApply, BT>(g, reinterpret_cast<T*>(lds), int(blockIdx.x), int(gridDim.x));
}
template <typename T, int BT>
__global__ __launch_bounds__(TileGeom<BT>::kThreads) void ns_apply_last_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) char lds[GemmLds<T, kApply, BT>::kBytes];
  gemm_body<T, kApply, BT, true>(g, reinterpret_cast<T*>(lds), int(blockIdx.x), int(gridDim.x));
}
// An apply step's 256-tiles and the small tiles of its last round in one
// launch: the first `main_grid` workgroups run the 256-tiles, the rest the
// small tiles, so that each small tile starts as soon as a CU frees up
// rather than after the whole 256-tile launch (and one launch gap less).
// The waves a small tile does not use exit at once; a barrier waits only for
// the waves still running. main_grid is a multiple of the XCD count, so a
// small tile's workgroup number keeps its XCD.
template <typename T, int BT, int TT, bool LAST>
__global__ __launch_bounds__(TileGeom<BT>::kThreads) void ns_apply_pair_kernel(GemmArgs g, GemmArgs tail,
                                                                                int32_t main_grid) {
  static_assert(TileGeom<TT>::kThreads <= TileGeom<BT>::kThreads, "small tiles use fewer waves");
  constexpr int kBytes = GemmLds<T, kApply, BT>::kBytes > GemmLds<T, kApply, TT>::kBytes
                             ? GemmLds<T, kApply, BT>::kBytes : GemmLds<T, kApply, TT>::kBytes;
  __shared__ __attribute__((aligned(16))) char lds[kBytes];
  const int b = int(blockIdx.x);
  if (b < main_grid) {
    gemm_body<T, kApply, BT, LAST>(g, reinterpret_cast<T*>(lds), b, main_grid);
  } else if (int(threadIdx.x) < TileGeom<TT>::kThreads) {
    gemm_body<T, kApply, TT, LAST>(tail, reinterpret_cast<T*>(lds), b - main_grid, int(gridDim.x) - main_grid);
  }
}

}  // namespace

hipError_t launch_lion(const LionLaunch& l, hipStream_t stream) {
  if (l.n_blocks == 0) return hipSuccess;
  LionArgs a;
  a.tensors = l.tensors;
  a.bind = l.bind;
  a.block_start = l.block_start;
  a.n_tensors = l.n_tensors;
  a.b1 = l.k.beta1;
  a.omb1 = l.k.one_minus_beta1;
  a.b2 = l.k.beta2;
  a.omb2 = l.k.one_minus_beta2;
  a.lr = l.k.lr_lion;
  a.wd = l.k.wd;
  a.ab1 = l.k.adam_b1;
  a.aomb1 = l.k.adam_omb1;
  a.ab2 = l.k.adam_b2;
  a.aomb2 = l.k.adam_omb2;
  a.alr = l.k.adam_lr;
  a.aeps = l.k.adam_eps;
  a.awd = l.k.adam_wd;
  a.ac1 = l.k.adam_c1;
  a.ac2 = l.k.adam_c2;
  a.decide = l.decide;
  hipLaunchKernelGGL(lion_kernel, dim3(l.n_blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

static PrepArgs prep_args(const PrepLaunch& l) {
  PrepArgs a;
  a.mats = l.mats;
  a.bind = l.bind;
  a.prep_start = l.prep_start;
  a.n_mats = l.n_mats;
  a.ws = l.ws;
  a.partials = l.partials;
  a.rscale = l.rscale;
  a.decide = l.decide;
  a.b1 = l.k.beta1;
  a.omb1 = l.k.one_minus_beta1;
  a.b2 = l.k.beta2;
  a.omb2 = l.k.one_minus_beta2;
  a.eps = l.k.eps;
  return a;
}

hipError_t launch_prep(const PrepLaunch& l, hipStream_t stream) {
  if (l.n_tiles == 0) return hipSuccess;
  hipLaunchKernelGGL(prep_kernel, dim3(l.n_tiles), dim3(256), 0, stream, prep_args(l));
  return hipGetLastError();
}

hipError_t launch_norm(const PrepLaunch& l, hipStream_t stream) {
  if (l.n_mats == 0) return hipSuccess;
  hipLaunchKernelGGL(norm_kernel, dim3(l.n_mats), dim3(256), 0, stream, prep_args(l));
  return hipGetLastError();
}

hipError_t launch_gemm(GemmMode mode, const GemmLaunch& l, hipStream_t stream) {
  if (l.max_count == 0) return hipSuccess;
  if (l.tail_max_count > 0 && (mode != kApply || l.fp32 || l.tile != 256)) return hipErrorInvalidValue;
  GemmArgs a;
  a.mats = l.mats;
  a.bind = l.bind;
  a.xcds = l.chip.xcds;
  a.tasks = l.tasks;
  a.split = l.split;
  a.ws = l.ws;
  a.rscale = l.rscale;
  a.src = l.src;
  a.first = l.first;
  a.last = l.last;
  a.store_o = l.store_o;
  a.a = l.a;
  a.b = l.b;
  a.c = l.c;
  a.lr = l.lr;
  a.wd = l.wd;
  a.decide = l.decide;
  // persistent: at most as many workgroups per XCD as its CUs hold at once,
  // limited by LDS (256-tiles: one per CU; 128-tiles: two, or one for the
  // four-stage bf16 apply; 64-tiles: four, or two for the bf16 apply)
  // (only the non-final apply is persistent; the others keep one workgroup
  // per tile)
  const int per_cu = l.tile == 256 ? 1 : (l.tile == 128 ? (l.fp32 ? 2 : 1) : (l.fp32 ? 4 : 2));
  const int per_xcd = (mode != kApply || l.last) ? l.max_count : (l.chip.cus / l.chip.xcds) * per_cu;
  const dim3 grid(unsigned(l.max_count < per_xcd ? l.max_count : per_xcd) * unsigned(l.chip.xcds));
#define LM_LAUNCH(KERNEL, T, BT) \
  hipLaunchKernelGGL((KERNEL<T, BT>), grid, dim3(TileGeom<BT>::kThreads), 0, stream, a)
#define LM_LAUNCH_MODE(T, BT)                                   \
  do {                                                          \
    if (mode == kGram) LM_LAUNCH(ns_gram_kernel, T, BT);        \
    else if (mode == kPoly) LM_LAUNCH(ns_poly_kernel, T, BT);   \
    else if (!l.last) LM_LAUNCH(ns_apply_kernel, T, BT);        \
    else LM_LAUNCH(ns_apply_last_kernel, T, BT);                \
  } while (0)
  if (l.fp32) {
    if (l.tile == 64) LM_LAUNCH_MODE(float, 64);
    else if (l.tile == 128) LM_LAUNCH_MODE(float, 128);
    else return hipErrorInvalidValue;
  } else if (l.tile == 256) {
    if (mode == kApply && l.tail_max_count > 0) {
      // with the last round's small tiles: one workgroup per CU at a time
      // (the launch's LDS is the 256-tile's), persistent unless last
      GemmArgs at = a;
      at.tasks = l.tail_tasks;
      at.split = l.tail_split;
      const int t_xcd = l.last ? l.tail_max_count
                               : (l.tail_max_count < l.chip.cus / l.chip.xcds ? l.tail_max_count
                                                                              : l.chip.cus / l.chip.xcds);
      const dim3 pair(grid.x + unsigned(t_xcd) * unsigned(l.chip.xcds));
      const int32_t main_grid = int32_t(grid.x);
#define LM_LAUNCH_PAIR(TT, LAST_) \
  hipLaunchKernelGGL((ns_apply_pair_kernel<bf16, 256, TT, LAST_>), pair, dim3(TileGeom<256>::kThreads), 0, stream, a, at, main_grid)
      if (l.tail_tile == 64) {
        if (!l.last) LM_LAUNCH_PAIR(64, false);
        else LM_LAUNCH_PAIR(64, true);
      } else if (l.tail_tile == 128) {
        if (!l.last) LM_LAUNCH_PAIR(128, false);
        else LM_LAUNCH_PAIR(128, true);
      } else {
        return hipErrorInvalidValue;
      }
#undef LM_LAUNCH_PAIR
    } else {
      LM_LAUNCH_MODE(bf16, 256);
    }
  } else if (l.tile == 128) {
    LM_LAUNCH_MODE(bf16, 128);
  } else {
    // bf16 64-tiles exist for the apply only (the last round of 256-tiles)
    if (l.tile != 64 || mode != kApply) return hipErrorInvalidValue;
    if (!l.last) LM_LAUNCH(ns_apply_kernel, bf16, 64);
    else LM_LAUNCH(ns_apply_last_kernel, bf16, 64);
  }
#undef LM_LAUNCH_MODE
#undef LM_LAUNCH
  return hipGetLastError();
}

static SrankArgs srank_args(const SrankLaunch& l) {
  SrankArgs a;
  a.mats = l.mats;
  a.bind = l.bind;
  a.tab = l.tab;
  a.rd_start = l.rd_start;
  a.tensor_mat = l.tensor_mat;
  a.n_mats = l.n_mats;
  a.ws = l.ws;
  a.decide = l.decide;
  a.decisions_out = l.decisions_out;
  a.srank_out = l.srank_out;
  a.alpha = l.alpha;
  a.reverse = 0;
  return a;
}

hipError_t launch_srank_pass(const SrankLaunch& l, int32_t kind, int32_t bucket,
                             int32_t first_block, int32_t n_blocks, bool first, bool last,
                             bool reverse, hipStream_t stream) {
  if (n_blocks == 0) return hipSuccess;
  SrankArgs a = srank_args(l);
  a.reverse = reverse ? 1 : 0;
  const dim3 grid(static_cast<unsigned>(n_blocks));
  const int32_t f = first ? 1 : 0, z = last ? 1 : 0;
  if (kind == kSrTall) {
    switch (bucket) {
#define LM_TALL(N) \
  case N: hipLaunchKernelGGL((srank_tall_kernel<N>), grid, dim3(256), 0, stream, a, first_block, f, z); break;
      LM_TALL(1) LM_TALL(2) LM_TALL(3) LM_TALL(4) LM_TALL(6) LM_TALL(8)
#undef LM_TALL
      default: return hipErrorInvalidValue;
    }
  } else if (kind == kSrWide || kind == kSrWideNarrow) {
#define LM_WIDE(N, SW) \
  case N: hipLaunchKernelGGL((srank_wide_kernel<N, SW>), grid, dim3(1024), 0, stream, a, first_block, f, z); break;
    if (kind == kSrWide) {
      switch (bucket) {
        LM_WIDE(1, 32) LM_WIDE(2, 32) LM_WIDE(4, 32) LM_WIDE(6, 32) LM_WIDE(8, 32)
        default: return hipErrorInvalidValue;
      }
    } else {
      switch (bucket) {
        LM_WIDE(1, 16) LM_WIDE(2, 16) LM_WIDE(4, 16) LM_WIDE(6, 16)
        default: return hipErrorInvalidValue;
      }
    }
#undef LM_WIDE
  } else {
    const dim3 block(256);
    if (first && last) hipLaunchKernelGGL((srank_generic_kernel<true, true>), grid, block, 0, stream, a, first_block);
    else if (first) hipLaunchKernelGGL((srank_generic_kernel<true, false>), grid, block, 0, stream, a, first_block);
    else if (last) hipLaunchKernelGGL((srank_generic_kernel<false, true>), grid, block, 0, stream, a, first_block);
    else hipLaunchKernelGGL((srank_generic_kernel<false, false>), grid, block, 0, stream, a, first_block);
  }
  return hipGetLastError();
}

hipError_t launch_srank_reduce(const SrankLaunch& l, hipStream_t stream) {
  if (l.n_chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(srank_reduce_kernel, dim3(unsigned(l.n_chunks)), dim3(256), 0, stream,
                     srank_args(l));
  return hipGetLastError();
}

hipError_t launch_srank_decide(const SrankLaunch& l, hipStream_t stream) {
  if (l.n_inputs == 0) return hipSuccess;
  hipLaunchKernelGGL(srank_decide_kernel, dim3(unsigned(l.n_inputs)), dim3(256), 0, stream,
                     srank_args(l));
  return hipGetLastError();
}

}  // namespace lm
