/*
 * lionmuon.h -- C ABI of the MI355X (gfx950) LionMuon optimizer step.
 *
 * The operation is Algorithm 1 of "LionMuon: Alternating Spectral and Sign
 * Descent for Efficient Training" (arXiv 2605.19811, Section 3), applied to a
 * list of fp32 parameter tensors that each own one momentum buffer
 * (Section 3, implementation notes):
 *
 *   Ghat = beta1*M + (1-beta1)*G                 Lion interpolation, with the
 *                                                buffer BEFORE this step's update
 *   if t mod P == 0 (Muon step, 2-D tensors that are not Lion-only):
 *       W <- W - lr_muon * (kappa*NS_K(Ghat) + wd*W)
 *   else (Lion step):
 *       W <- W - lr_lion * (sign(Ghat) + wd*W)   sign(0) = 0
 *   M <- beta2*M + (1-beta2)*G                   every step, every tensor
 *
 * NS_K is K steps of the odd quintic Newton-Schulz iteration towards the
 * matrix sign msign(X) = U V^T (Section 2, "Spectral methods" and
 * "Approximating the matrix sign"; K_NS = 5 in Table 3):
 *   X0 = Ghat / (||Ghat||_F + eps), iterated in the orientation with
 *   rows <= cols; each step A = X X^T, B = b*A + c*A A, X <- a*X + B X.
 * kappa is 1 (Algorithm 1) or 0.2*sqrt(max(m, n)) (Table 3 "NS scaling").
 *
 * Adaptive variant (Appendix G; lm_config.adaptive_alpha > 0): instead of the
 * period P, each 2-D tensor that is not Lion-only or AdamW takes the Muon
 * branch on a step iff the stable-rank estimate of its momentum (the buffer
 * before this step's update),
 *   r_hat(M) = ||M||_F^2 / sigma_hat_1(M)^2 <= adaptive_alpha * min(m, n),
 * and the Lion branch otherwise. sigma_hat_1 = ||S v_k|| after k =
 * adaptive_power_steps power-iteration steps v <- S^T S v / ||S^T S v|| from
 * v_0 = ones / sqrt(min(m, n)), where S = M if rows >= cols, else M^T; an
 * iterate that vanishes, or M = 0, gives r_hat = 0. The estimate is computed
 * in fp64 on the device and the decision never leaves it.
 *
 * Conventions shared by every entry point:
 *  - Pointer arrays (params, grads, momentum, shapes) live in HOST memory;
 *    the pointers they hold are DEVICE pointers to fp32, contiguous,
 *    row-major tensors owned by the caller. 1-D tensors use rows = 1.
 *  - params and momentum are updated in place; grads are read only. The
 *    three buffers of one tensor must not overlap (checked).
 *  - Every call is asynchronous on `stream` (0 = the null stream) and returns
 *    once all work is enqueued; no host synchronisation is performed.
 *  - Validation happens before anything is enqueued: an invalid call returns
 *    an error and modifies nothing. A HIP failure after enqueueing started
 *    returns LM_ERR_HIP; tensors may then be partly updated.
 *  - lionmuon_last_error() gives a thread-local message for the last failure.
 *  - Calls that use the library-owned workspace are serialised: on the host
 *    by a mutex, and on the device by an event, so a call on another stream
 *    than the previous user of that workspace first waits (on the device,
 *    without blocking the host) for that user's work. Calls with caller
 *    workspaces may run concurrently on distinct streams.
 *  - The library caches one device plan (tile lists, descriptors) per list
 *    signature: step kind, NS precision and scaling, and each tensor's shape,
 *    flags and 16-byte alignment -- never its address. The tensor addresses
 *    of a call go to the device as a small per-plan table that is rewritten
 *    (one asynchronous copy on the call's stream, staged through a pinned
 *    ring) only when they differ from the previous call's, so callers whose
 *    gradient buffers move between steps pay no plan rebuild or allocation.
 *    Up to 16 signatures stay cached; a 17th evicts the least recently used
 *    (its device memory is freed, which waits for the device).
 *  - Grids are sized from the device's compute-unit and XCD counts.
 */
#ifndef LIONMUON_H
#define LIONMUON_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LIONMUON_ABI_VERSION 3

typedef enum lm_status {
  LM_OK = 0,
  LM_ERR_INVALID_ARGUMENT = 1,   /* null pointer, bad size, beta outside [0,1), ... */
  LM_ERR_UNSUPPORTED = 2,        /* valid request the library does not implement     */
  LM_ERR_OUT_OF_MEMORY = 3,      /* library-owned workspace or plan allocation failed */
  LM_ERR_WORKSPACE_TOO_SMALL = 4,/* caller workspace below lionmuon_workspace_bytes   */
  LM_ERR_HIP = 5                 /* a HIP runtime call or kernel launch failed        */
} lm_status;

/* Per-tensor flags.
 * LM_TENSOR_LION_ONLY: never take the Muon branch (Lion update every step).
 *   A tensor with rows == 1 or cols == 1 is always treated as Lion-only
 *   (1-D parameters do not take the spectral step, Section 3).
 * LM_TENSOR_ADAMW: AdamW with decoupled weight decay on every step instead
 *   of Algorithm 1 -- the fallback Section 3 names for 1-D parameters
 *   (Table 3: betas (0.8, 0.999), lr 1e-3). Its `momentum` buffer is AdamW's
 *   first moment; it also needs a second-moment buffer (lionmuon_step_ex). */
enum { LM_TENSOR_LION_ONLY = 1u, LM_TENSOR_ADAMW = 2u };

/* Precision of the Newton-Schulz matrix products. */
enum { LM_NS_BF16 = 0,   /* bf16 operands on MFMA, fp32 accumulation, for every
                            matrix whose short side is >= ns_bf16_min_side;
                            smaller matrices use the fp32 path              */
       LM_NS_FP32 = 1 }; /* fp32 operands on MFMA, fp32 accumulation        */

/* Output scaling kappa of the Muon direction. */
enum { LM_NS_SCALE_NONE = 0,    /* kappa = 1 (Algorithm 1)                        */
       LM_NS_SCALE_RMS02 = 1 }; /* kappa = 0.2*sqrt(max(rows, cols)) (Table 3)    */

/* Shape of one tensor: rows x cols, row-major; rows = 1 for a vector.
 * rows = 0 or cols = 0 is an empty tensor (skipped). */
typedef struct lm_shape {
  int64_t rows;
  int64_t cols;
  uint32_t flags;      /* LM_TENSOR_* bits */
  uint32_t reserved;   /* must be 0 */
} lm_shape;

/* Step configuration. Initialise with lionmuon_config_default().
 * Hyper-parameters are passed in double; the kernels compute in fp32 with
 * constants rounded once from the double values (1 - beta is formed in
 * double before rounding). */
typedef struct lm_config {
  uint32_t struct_size;     /* sizeof(lm_config)                                 */
  int32_t ns_steps;         /* K_NS in [1, 64], default 5 (Table 3)              */
  double ns_a, ns_b, ns_c;  /* odd polynomial a x + b x^3 + c x^5,
                               default (3.4445, -4.7750, 2.0315)                  */
  double ns_eps;            /* Frobenius guard eps >= 0, default 1e-7            */
  int32_t ns_precision;     /* LM_NS_BF16 (default) or LM_NS_FP32                */
  int32_t ns_scale_mode;    /* LM_NS_SCALE_NONE (default) or LM_NS_SCALE_RMS02   */
  double lr_muon;           /* eta_M >= 0 of the Muon branch (Algorithm 1)       */
  double lr_lion;           /* eta_L >= 0 of the Lion branch (Algorithm 1)       */
  int32_t ns_bf16_min_side; /* LM_NS_BF16 only: matrices with a shorter short
                               side run the fp32 path; default 64, >= 0          */
  int32_t reserved;         /* must be 0                                          */
  /* Per-step odd-polynomial schedule (Section 2: classical, Polar Express and
   * Chebyshev-type schedules share the NS cost structure). 0 (default): step
   * k uses (ns_a, ns_b, ns_c) for every k; otherwise it must equal ns_steps
   * (<= LM_MAX_NS_SCHEDULE) and step k uses ns_schedule[k] = {a_k, b_k, c_k}. */
  int32_t ns_schedule_steps;
  int32_t reserved2;        /* must be 0                                          */
  double ns_schedule[16][3];
  /* AdamW for LM_TENSOR_ADAMW tensors: W <- W - adam_lr (mhat/(sqrt(vhat) +
   * adam_eps) + adam_wd W), bias corrections 1/(1 - beta^k) with the AdamW
   * step count k = adam_step (below). Defaults (1e-3, 0.8, 0.999, 1e-8, 0). */
  double adam_lr, adam_beta1, adam_beta2, adam_eps, adam_wd;
  /* Adaptive Muon / Lion choice (Appendix G): 0 (default) = off, the period
   * P decides; in (0, 1] = threshold alpha of the stable-rank rule, P is then
   * ignored (the Appendix G sweep uses 0.002 ... 0.01). */
  double adaptive_alpha;
  int32_t adaptive_power_steps;  /* power-iteration steps k in [0, 64], default 5 */
  int32_t reserved3;             /* must be 0                                      */
  /* AdamW step count k >= 1 of this call's bias corrections (the first AdamW
   * step is k = 1). 0 (default): k = t + 1, for callers whose t counts from 0
   * as in Algorithm 1; a caller counting steps from 1 passes adam_step = t. */
  int64_t adam_step;
} lm_config;

#define LM_MAX_NS_SCHEDULE 16

/* Fill *cfg with the defaults listed above; lr_muon = lr_lion = 0. */
void lionmuon_config_default(lm_config* cfg);

/*
 * One LionMuon step (Algorithm 1) over n_tensors tensors with
 * eta_M = eta_L = lr, bf16 Newton-Schulz and the other defaults.
 *   params[i], grads[i], momentum[i]: device fp32, shapes[i].rows*cols values.
 *   t >= 0: step index; the Muon branch fires iff P >= 1 and t mod P == 0.
 *   P >= 0: period; P = 0 encodes P = infinity (pure Lion).
 *   beta1, beta2 in [0, 1); lr >= 0; wd >= 0 (decoupled weight decay).
 * Uses a library-owned device workspace, allocated on first Muon step and
 * grown as needed (freed by lionmuon_release).
 */
lm_status lionmuon_step(float* const* params, const float* const* grads,
                        float* const* momentum, const lm_shape* shapes,
                        int32_t n_tensors, int64_t t, int32_t P, double beta1,
                        double beta2, double lr, double wd, hipStream_t stream);

/*
 * lionmuon_step with an explicit configuration (two learning rates, fp32 or
 * bf16 Newton-Schulz, coefficients or a per-step schedule, eps, output
 * scaling, AdamW settings) and an optional caller-owned device workspace.
 * second_moment: host array of n_tensors device pointers, read only for
 *   LM_TENSOR_ADAMW tensors (AdamW's v, same shape, updated in place); may
 *   be NULL when no tensor has that flag.
 * workspace == NULL with workspace_bytes == 0 selects the library-owned
 * workspace; otherwise workspace must hold at least
 * lionmuon_workspace_bytes(...) bytes, be 256-byte aligned, stay valid until
 * the enqueued work finishes, and must not be used by a concurrent call.
 * With cfg->adaptive_alpha > 0 the step is the adaptive variant (P ignored,
 * but still checked >= 0).
 */
lm_status lionmuon_step_ex(float* const* params, const float* const* grads,
                           float* const* momentum, float* const* second_moment,
                           const lm_shape* shapes,
                           int32_t n_tensors, int64_t t, int32_t P, double beta1,
                           double beta2, double wd, const lm_config* cfg,
                           void* workspace, size_t workspace_bytes,
                           hipStream_t stream);

/*
 * lionmuon_step_ex for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments and results as lionmuon_step_ex without a workspace; the
 * call allocates nothing (no hipMalloc / hipHostMalloc / hipFree, no events;
 * phase timing is not recorded). Its plan tables, the call's tensor
 * addresses and the Newton-Schulz workspace live in one static device array
 * of LIONMUON_NOALLOC_SCRATCH_BYTES bytes per device, which each device holds
 * from the library's first use of it until the process ends. Tables reach
 * the array through kernel arguments, on `stream`, only when the list
 * signature (shapes, flags, alignment, step kind, cfg precision and scaling)
 * or the tensor addresses differ from the previous call's.
 * A list whose tables and workspace exceed the array fails with
 * LM_ERR_UNSUPPORTED before anything is enqueued (the message gives the
 * bytes needed): a Muon step over one 768x3072 bf16 matrix needs about
 * 12 MB, one 2048x4096 matrix about 50 MB.
 * All calls on one device share the array, which keeps the last call's
 * contents: calls on one device must not overlap (on different streams they
 * race); consecutive calls on one stream are ordered. No kernel reads scratch
 * it has not written in the same call, so nothing needs clearing.
 */
#define LIONMUON_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
lm_status lionmuon_step_noalloc(float* const* params, const float* const* grads,
                                float* const* momentum, float* const* second_moment,
                                const lm_shape* shapes, int32_t n_tensors, int64_t t, int32_t P,
                                double beta1, double beta2, double wd, const lm_config* cfg,
                                hipStream_t stream);

/*
 * One step of the adaptive variant (Appendix G) with per-tensor diagnostics:
 * lionmuon_step_ex with cfg->adaptive_alpha in (0, 1] (required here), plus
 *   decisions:   optional device int32[n_tensors]: 1 where the tensor took the
 *                Muon branch this step, else 0;
 *   stable_rank: optional device double[n_tensors]: r_hat(M) of each Muon
 *                candidate, -1 for every other tensor (1-D, Lion-only, AdamW,
 *                empty).
 * Both are written on `stream`; either may be NULL. Every matrix that may take
 * the Muon branch keeps Newton-Schulz workspace (lionmuon_workspace_bytes with
 * the same cfg).
 */
lm_status lionmuon_step_adaptive(float* const* params, const float* const* grads,
                                 float* const* momentum, float* const* second_moment,
                                 const lm_shape* shapes, int32_t n_tensors, int64_t t,
                                 double beta1, double beta2, double wd, const lm_config* cfg,
                                 void* workspace, size_t workspace_bytes, int32_t* decisions,
                                 double* stable_rank, hipStream_t stream);

/* Device workspace (bytes) a Muon step -- or, with cfg->adaptive_alpha > 0,
 * an adaptive step -- over these tensors needs with cfg (NULL = defaults).
 * A Lion step needs none. The size depends on shapes, flags and cfg only (not
 * on the tensors' alignment), so it holds for any buffers of these shapes.
 * Host-only: no device work. */
lm_status lionmuon_workspace_bytes(const lm_shape* shapes, int32_t n_tensors,
                                   const lm_config* cfg, size_t* out_bytes);

/*
 * Newton-Schulz hook (Section 2): O[b] = kappa * NS_K(X[b]) for a batch of
 * `batch` same-shape rows x cols fp32 device matrices stored back to back
 * (X and O each hold batch*rows*cols values; they must not overlap).
 * Uses the same kernels as the Muon branch of lionmuon_step_ex.
 * workspace/workspace_bytes as in lionmuon_step_ex, sized by
 * lionmuon_workspace_bytes for `batch` tensors of this shape.
 */
lm_status lionmuon_ns(const float* X, float* O, int64_t rows, int64_t cols,
                      int32_t batch, const lm_config* cfg, void* workspace,
                      size_t workspace_bytes, hipStream_t stream);

/* Host-side description of the work one step would enqueue (no device work;
 * the tile lists are those of the current device's CU and XCD counts, or of
 * a full MI355X -- 256 CUs in 8 XCDs -- when no device is present).
 * With cfg->adaptive_alpha > 0, n_muon / muon_elements count the Muon
 * candidates (each takes Muon or Lion on the device), n_lion / lion_elements
 * the tensors that always take the Lion branch. */
typedef struct lm_plan_info {
  int32_t n_tensors;        /* non-empty tensors                               */
  int32_t n_lion;           /* tensors updated by the Lion branch this step    */
  int32_t n_adamw;          /* tensors updated by AdamW (LM_TENSOR_ADAMW)      */
  int32_t reserved;
  int32_t n_muon;           /* matrices updated by the Muon branch this step   */
  int32_t n_shape_classes;  /* distinct (short side, long side) Muon shapes    */
  int64_t lion_elements;    /* elements on the Lion branch                     */
  int64_t adamw_elements;   /* elements updated by AdamW                       */
  int64_t muon_elements;    /* elements on the Muon branch                     */
  int64_t gram_tiles, poly_tiles, apply_tiles; /* MFMA output tiles per NS step
                               (a nearly empty last round of 256x256 apply tiles
                               is counted as the smaller tiles it runs as)      */
  double ns_flops;          /* algorithmic NS flops, symmetric products counted
                               once: K * sum s(s+1)l + s^2(s+1) + 2 s^2 l       */
  double ns_flops_dense;    /* dense convention K * sum 4 s^2 l + 2 s^3        */
  double lion_bytes;        /* 20 bytes per Lion-branch element, 28 per AdamW   */
  size_t workspace_bytes;   /* device workspace this step needs                */
  double srank_bytes;       /* adaptive: algorithmic bytes of the stable-rank
                               passes, 4 (k+1) per candidate element plus 16 k
                               per fp64 partial product; else 0               */
} lm_plan_info;

lm_status lionmuon_plan_info(const lm_shape* shapes, int32_t n_tensors,
                             int64_t t, int32_t P, const lm_config* cfg,
                             lm_plan_info* out);

/*
 * Phase timing. When enabled, every call records HIP events around each
 * kernel it enqueues, on the call's stream; lionmuon_profiling_read waits for
 * the recorded events and returns per-phase sums (ms) and launch counts since
 * the last reset. Disabled by default; enabling costs one event pair per
 * launch.
 */
enum { LM_PHASE_LION = 0, LM_PHASE_PREP = 1, LM_PHASE_NORM = 2,
       LM_PHASE_GRAM = 3, LM_PHASE_POLY = 4, LM_PHASE_APPLY = 5,
       LM_PHASE_SRANK = 6,   /* adaptive: stable-rank passes and decisions */
       LM_PHASE_COUNT = 7 };
typedef struct lm_phase_times {
  double ms[LM_PHASE_COUNT];
  int64_t launches[LM_PHASE_COUNT];
} lm_phase_times;
lm_status lionmuon_profiling_enable(int32_t enable);
lm_status lionmuon_profiling_read(lm_phase_times* out);
lm_status lionmuon_profiling_reset(void);

/* Free the library-owned workspace and cached plans (device memory). Must not
 * be called while work enqueued by this library is still running. */
void lionmuon_release(void);

const char* lionmuon_status_string(lm_status status);
const char* lionmuon_last_error(void);
int32_t lionmuon_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LIONMUON_H */
