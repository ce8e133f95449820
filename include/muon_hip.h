/*
 * muon_hip.h — C ABI of the MI355X (gfx950) batched Muon step.
 *
 * The operation (HyperParallel-FSDP, arXiv 2609.21594):
 *   Sec. 2.3, Eq. (1): accumulate momentum, normalise X0 = G/(||G||_F + eps),
 *     run K Newton-Schulz steps X <- a_k X + b_k (X X^T) X + c_k (X X^T)^2 X,
 *     rescale by 0.2*sqrt(max(m, n)) (RMS matching);
 *   Sec. 6.6: transpose-first (rows > cols runs on the transpose), shape-fused
 *     batches capped at 2^29 elements, workspace allocated once per batched
 *     invocation, descending-size batch order;
 *   Sec. 6.3: an [E, M, N] expert weight is E independent M x N matrices;
 *   Sec. 6.4 / 6.2 (local programming model): each device sees its own
 *     gradients, momentum and parameters and applies the update with
 *     decoupled weight decay.
 *
 * Readings where the paper prints no formula (the kernels follow these):
 *   momentum   buf' = beta*buf + (1-beta)*g ;
 *              u = (1-beta)*g + beta*buf' (nesterov) or u = buf'
 *   update     W' = (1 - lr*wd) * W - lr * scale * O,
 *              scale = 0.2*sqrt(max(rows, cols)) (scale_mode 0, Sec. 2.3),
 *              1 (mode 1), or sqrt(max(1, rows/cols)) (mode 2, the rule of
 *              the original Muon method that Sec. 2.3 and Sec. 6.2 keep as a
 *              configurable legacy stage)
 *   post       the updated matrix multiplied by the entry's post_scale
 *              (a post-processing stage of Sec. 6.2, e.g. QK-clip factors;
 *              default none)
 *   eps        added to the Frobenius norm, outside the square root
 *   square     matrices (rows == cols) are not transposed
 *   ns_coeffs  NULL selects the constant quintic (3.4445, -4.7750, 2.0315).
 *
 * Conventions for every entry point:
 *   - Device pointers are HIP device addresses on the handle's device; host
 *     pointers (arrays of descriptors, coefficient tables) are read during
 *     the call only and may be freed when it returns.
 *   - Matrices are row-major.  The outputs of ns_orthogonalize_batched and
 *     its inputs are dense; a muon_step entry may be a strided view of a
 *     larger parameter (see muon_param_t).
 *   - All work is enqueued on `stream` (a hipStream_t; NULL is the null
 *     stream) and the call returns without waiting for it.  Every buffer the
 *     caller passes must stay alive until that work has completed.
 *   - Every argument is checked before the first launch: a call that returns
 *     an error other than MUON_ERR_DEVICE changed nothing.  Values inside the
 *     tensors are never checked; NaN and Inf propagate.  The calls that
 *     launch work (muon_step, ns_orthogonalize_batched, muon_adamw_step) also
 *     ask the runtime about every buffer: it must start in device memory of
 *     the handle's device (or managed memory), and if it reaches beyond the
 *     allocation that holds its start, its last byte must be such memory too
 *     (allocations mapped back to back); otherwise MUON_ERR_INVALID_ARGUMENT.  muon_validate_step does not query the
 *     runtime and accepts any address.
 *   - A call that repeats the handle's previous muon_step or
 *     ns_orthogonalize_batched request exactly (the same entries, pointers,
 *     shapes, views, dtypes, coefficient values and options; lr and
 *     weight_decay may differ) reuses that request's checks and plan: its
 *     buffers are not queried from the runtime again.
 *   - A handle is not thread-safe; use one handle per host thread.
 *   - Results are deterministic: the same call on the same data gives the same
 *     bits, and a matrix's result does not depend on which other matrices
 *     share the call.
 *   - No C++ exception crosses this interface.
 */
#ifndef MUON_HIP_H
#define MUON_HIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MUON_HIP_ABI_VERSION 3

typedef struct muon_handle* muon_handle_t;

typedef enum {
  MUON_OK = 0,
  MUON_ERR_INVALID_ARGUMENT = 1,  /* bad pointer, size, dtype, overlap, ... */
  MUON_ERR_UNSUPPORTED = 2,       /* valid request this build does not do */
  MUON_ERR_OUT_OF_MEMORY = 3,     /* workspace would exceed the limit or hipMalloc failed */
  MUON_ERR_DEVICE = 4             /* a HIP runtime call failed */
} muon_status_t;

typedef enum { MUON_F32 = 0, MUON_BF16 = 1 } muon_dtype_t;

/* Arithmetic of the Newton-Schulz products: bf16 operands with fp32
 * accumulation (intermediates X, A = X X^T, B = bA + cA^2 stored as bf16),
 * or fp32 throughout.  Momentum, norm and update are fp32 in both. */
typedef enum { MUON_NS_BF16 = 0, MUON_NS_F32 = 1 } muon_ns_precision_t;

/* One parameter entry: `batch` matrices of rows x cols (Sec. 6.3: a stacked
 * expert weight is E independent matrices).
 *
 * Logical matrices (Sec. 6.6: the matrix as Muon sees it is defined apart
 * from the storage layout): an entry may be a zero-copy strided view of a
 * larger physical parameter, e.g. one of the heads of a fused QKV weight
 * (row blocks), the gate or up half of a packed FC1 weight (a column range,
 * ld > cols), or such a piece of every expert of a stack (plane_stride).
 * Row i of plane e starts at element
 *     e*plane_stride + (i / row_block)*block_stride + (i % row_block)*ld
 * of param and grad (and of momentum unless momentum_dense), and its cols
 * elements are contiguous; the update is written back through the same
 * mapping and nothing outside the view is touched.  Zero selects each
 * field's dense default, so a zeroed tail describes a dense
 * batch x rows x cols array.  The views of all entries must be disjoint
 * (grads may share elements with other grads). */
typedef struct {
  void* param;             /* in/out: param_dtype */
  const void* grad;        /* in:     grad_dtype, same view as param */
  float* momentum;         /* in/out: fp32, same view as param, or dense */
  int64_t rows, cols;      /* the logical matrix, >= 1 */
  int64_t batch;           /* >= 1 */
  int64_t ld;              /* row stride in elements: 0 (= cols) or >= cols */
  muon_dtype_t param_dtype;
  muon_dtype_t grad_dtype;
  int64_t row_block;       /* rows per contiguous-stride block: 0 (= rows) or
                              a divisor of rows */
  int64_t block_stride;    /* elements from one row block to the next:
                              0 (= row_block*ld), else >= (row_block-1)*ld + cols */
  int64_t plane_stride;    /* elements from one plane to the next: 0 (= number
                              of blocks * block_stride), else >= the span of a plane */
  int32_t momentum_dense;  /* 0: momentum has param's view; 1: momentum is a
                              dense batch x rows x cols array */
  float post_scale;        /* post-processing stage (Sec. 6.2 names QK-clip as
                              one): the updated matrix is multiplied by this
                              factor, W' = post_scale * ((1 - lr*wd) W -
                              lr*scale*O), e.g. a per-head query/key factor
                              the caller derives from its attention logits
                              (one entry per head through row-block views).
                              0: none (1); otherwise finite and > 0 */
  /* Per-parameter configuration (Sec. 6.2: step count, coefficients and
   * scaling are per-parameter stages).  Entries whose tables hold the same
   * values are batched together; different tables never share a batch. */
  const float* ns_coeffs;  /* host, ns_steps x 3 {a_k, b_k, c_k}: this entry's
                              table; NULL: the call's (hparams) table */
  int32_t ns_steps;        /* rows of ns_coeffs, 0..64 (ignored when NULL) */
  int32_t scale_mode;      /* 0: the call's scale_mode; 1 + m: scale_mode m */
} muon_param_t;

typedef struct {
  float lr;                /* finite */
  float beta;              /* momentum coefficient, finite */
  float weight_decay;      /* decoupled decay, finite */
  float eps;               /* >= 0, finite; 1e-7 recommended */
  int32_t ns_steps;        /* K, 0 <= K <= 64 */
  int32_t nesterov;        /* 0 or 1 */
  const float* ns_coeffs;  /* host array K x 3 {a_k, b_k, c_k}, or NULL */
  muon_ns_precision_t ns_precision;
  int32_t scale_mode;      /* 0: 0.2*sqrt(max(rows, cols)); 1: none;
                              2: sqrt(max(1, rows/cols)) */
  int64_t max_chunk_elems; /* batch cap in elements of X; 0 = 2^29 (Sec. 6.6) */
} muon_hparams_t;

/* One shape-fused chunk of a plan (what muon_plan reports). */
typedef struct {
  int64_t s, l;            /* short and long side of every matrix in the chunk */
  int64_t s_pad, l_pad;    /* workspace extents (multiples of 128) */
  int64_t first;           /* index of the chunk's first matrix in plan order */
  int64_t count;           /* matrices in the chunk */
  int32_t param_dtype, grad_dtype;
  int32_t ns_steps;        /* K of the chunk's coefficient table */
  int32_t coeff_set;       /* 0: the call's table; k > 0: the k-th distinct
                              per-entry table, in entry order */
  size_t workspace_bytes;  /* workspace this chunk needs */
} muon_chunk_info_t;

/* Handle: owns the workspace and the device descriptor tables of one device.
 * muon_create makes `device` current while it runs and restores the caller's
 * device before it returns.  muon_destroy waits on the host for the work of
 * every call made on the handle (and nothing else on the device), then frees
 * what the handle owns; growing the workspace or a descriptor table waits
 * the same way.  Each call records an event at its end, also when it fails
 * after enqueueing work, and a call on another stream than the previous one
 * waits for that event on the device first. */
muon_status_t muon_create(muon_handle_t* out, int device);
muon_status_t muon_destroy(muon_handle_t h);

/* Chunks of one call that leave compute units idle (their symmetric
 * products fill the last round of tiles less than 90%) run on a second
 * stream owned by the handle, beside the chunks on `stream`; the call forks
 * from and joins back into `stream` through events, so its work is still
 * ordered on `stream` as a whole.  Such a call uses a second workspace slot
 * sized for the chunks it places there, up to twice what muon_plan_step
 * reports (never beyond the workspace limit: then it runs on `stream`
 * alone).  Results are bitwise the same either way.
 * streams: 2 (the default) or 1 (everything on the caller's stream). */
muon_status_t muon_set_streams(muon_handle_t h, int streams);

/* Grouped launches (Sec. 6.6, one batched launch per group of shapes), for
 * calls that run on one stream (muon_set_streams(h, 1)): the chunks of a
 * call that leave compute units idle (as above), run their Newton-Schulz
 * products on the 256 x 256 tile kernels (bf16 NS, padded extents multiples
 * of 256) and share the step count and parameter dtype are run together,
 * up to 8 at a time: per step, one launch per product over the tiles of all
 * of them.  With two streams such chunks overlap on the streams instead.
 * Each member keeps its own workspace region, so the call's workspace can
 * exceed what muon_plan_step reports by the sum of those chunks' sizes
 * (never beyond the workspace limit: then the chunks run one by one).
 * Results are bitwise the same either way.  enable: 1 (the default) or 0. */
muon_status_t muon_set_grouping(muon_handle_t h, int enable);

/* Grows the workspace to at least `bytes` now (hipMalloc synchronises, so do
 * this before timing).  Fails with MUON_ERR_OUT_OF_MEMORY above the limit. */
muon_status_t muon_reserve(muon_handle_t h, size_t bytes);
/* Caps the workspace (0 = no cap).  A call whose plan needs more fails with
 * MUON_ERR_OUT_OF_MEMORY before any launch. */
muon_status_t muon_set_workspace_limit(muon_handle_t h, size_t bytes);
size_t muon_workspace_bytes(muon_handle_t h);

/*
 * One Muon step over n entries (Sec. 2.3, Eq. (1); Sec. 6.6):
 *   momentum <- beta*momentum + (1-beta)*grad                 (in place, fp32)
 *   u        <- (1-beta)*grad + beta*momentum   (or momentum, nesterov = 0)
 *   O        <- NS_K(u / (||u||_F + eps)) per matrix, transpose-first
 *   param    <- (1 - lr*wd)*param - lr*scale*O                 (in place)
 * grad is only read.  param, grad and momentum of all entries must not
 * overlap (two grads may).  Matrices are grouped by (short side, long side,
 * dtypes, coefficient table), chunked at max_chunk_elems, and chunks run
 * largest first.
 */
muon_status_t muon_step(muon_handle_t h, const muon_param_t* params, int64_t n,
                        const muon_hparams_t* hp, void* stream);

/*
 * Standalone batched orthogonalisation (Sec. 6.6): out[i] = NS_K(in[i] /
 * (||in[i]||_F + eps)), rows[i] x cols[i], both in `dtype`, transpose-first
 * inside, result in the input's own layout.  in[i] == out[i] is allowed; any
 * other overlap between an output and another buffer is rejected.
 */
muon_status_t ns_orthogonalize_batched(muon_handle_t h, const void* const* in,
                                       void* const* out, const int64_t* rows,
                                       const int64_t* cols, int64_t n, muon_dtype_t dtype,
                                       int32_t ns_steps, const float* ns_coeffs, float eps,
                                       muon_ns_precision_t prec, void* stream);

/*
 * ns_orthogonalize_batched without any allocation, for callers that cannot
 * allocate: code under HIP stream capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments, checks and results (bit for bit)
 * as ns_orthogonalize_batched.  The workspace and the descriptor table live
 * in a fixed 64 MiB array of device memory that the library holds on each
 * device it runs on until the process ends (its address is resolved by
 * muon_create); the call makes no hipMalloc, hipFree, pinned-host or other
 * allocating call, and queues no host-to-device copy (the descriptors travel
 * as kernel arguments).
 * Limits: at most 64 matrices per call, and each chunk of same-shape
 * matrices must fit the array: a single matrix whose workspace exceeds it
 * (about 2048 x 5632 in bf16) returns MUON_ERR_UNSUPPORTED.  The handle's own
 * workspace, tables, second stream and profiling are not used.
 * Every call on one device shares that device's array and leaves its last
 * contents there: calls that overlap in time on one device race, so issue
 * them one at a time or in order on one stream.
 */
muon_status_t ns_orthogonalize_batched_noalloc(muon_handle_t h, const void* const* in,
                                               void* const* out, const int64_t* rows,
                                               const int64_t* cols, int64_t n, muon_dtype_t dtype,
                                               int32_t ns_steps, const float* ns_coeffs, float eps,
                                               muon_ns_precision_t prec, void* stream);

/*
 * AdamW for the parameters Muon does not take: Sec. 6.4 (Fig. "muon-
 * grouping") sends one-dimensional and scalar parameters to AdamW through a
 * chained optimizer, with decoupled weight decay.  The paper prints no
 * formula; this is AdamW with decoupled decay and bias correction, per
 * element, in fp32:
 *   m' = beta1*m + (1-beta1)*g          v' = beta2*v + (1-beta2)*g^2
 *   p' = (1 - lr*wd)*p - lr/(1 - beta1^t) * m' / (sqrt(v'/(1 - beta2^t)) + eps)
 * for step t (t = 1 on the first call).  Every tensor is taken as `numel`
 * contiguous elements.  param, exp_avg and exp_avg_sq are updated in place;
 * grad is only read.  Buffers of different entries must not overlap (grads
 * may).  Enqueued on `stream` like muon_step, and ordered after the
 * handle's earlier calls.
 */
typedef struct {
  void* param;             /* in/out: numel, param_dtype */
  const void* grad;        /* in:     numel, grad_dtype */
  float* exp_avg;          /* in/out: numel, fp32 (m) */
  float* exp_avg_sq;       /* in/out: numel, fp32 (v) */
  int64_t numel;           /* >= 0 */
  muon_dtype_t param_dtype;
  muon_dtype_t grad_dtype;
} muon_adamw_param_t;

typedef struct {
  float lr;                /* finite */
  float beta1, beta2;      /* in [0, 1) */
  float eps;               /* finite, > 0 */
  float weight_decay;      /* finite */
  int32_t reserved;        /* must be 0 */
  int64_t step;            /* t >= 1 */
} muon_adamw_hparams_t;

muon_status_t muon_adamw_step(muon_handle_t h, const muon_adamw_param_t* params, int64_t n,
                              const muon_adamw_hparams_t* hp, void* stream);

/* Host-only checks and planning (no device needed).  muon_validate_step
 * returns the status muon_step would return for these arguments before
 * launching anything and writes the reason into msg (may be NULL). */
muon_status_t muon_validate_step(const muon_param_t* params, int64_t n,
                                 const muon_hparams_t* hp, char* msg, size_t msg_len);
/* Fills up to `cap` chunk records in execution order; *n_chunks receives the
 * total, *workspace_bytes the workspace the plan needs.  `order` (may be NULL,
 * else room for the total matrix count) receives, per matrix in plan order,
 * its flat index (entry-major, plane-minor). */
muon_status_t muon_plan_step(const muon_param_t* params, int64_t n, const muon_hparams_t* hp,
                             muon_chunk_info_t* chunks, int64_t cap, int64_t* n_chunks,
                             size_t* workspace_bytes, int64_t* order);

/* Per-kernel timing.  When enabled, every kernel the handle launches is
 * bracketed by two HIP events on its launch stream; muon_profile_read waits
 * for them and returns, per kernel family, the launch count, the summed
 * event durations and the algorithmic work of those launches:
 *   flops       dense flop count of the product the kernel computes
 *               (2 s^2 l for X X^T and B X, 2 s^3 for A A; 0 for
 *               elementwise kernels),
 *   exec_flops  flops the kernel issues on the real extents (upper tiles
 *               only for the symmetric products),
 *   bytes       minimal HBM traffic: each operand read once, each output
 *               written once.
 * Families (in this order): momentum_norm (momentum, norm partials and the
 * unscaled X0 in one pass), norm_finalize, rescale (X0 = r*u for matrices
 * whose r is too large or small to be applied in the first products),
 * gram_syrk, poly_syrk, update_gemm, update_apply_gemm,
 * apply_x0, adamw, ns_small (the whole step of a chunk whose short side is
 * at most 128 with fp32 Newton-Schulz, in one fused launch).  `reset` != 0
 * clears the counters after reading. */
typedef struct {
  const char* name;
  int64_t launches;
  double total_ms;
  double flops;
  double exec_flops;
  double bytes;
} muon_kernel_stats_t;
muon_status_t muon_profile_enable(muon_handle_t h, int enable);
muon_status_t muon_profile_read(muon_handle_t h, muon_kernel_stats_t* out, int cap, int* n,
                                int reset);

/* Measurement aid, no part of the Muon step: copies `bytes` from src to dst
 * (device memory of the handle's device, 16-byte aligned, not overlapping)
 * on `stream` with the access pattern that reaches the highest HBM rate
 * (each workgroup a contiguous 256 KiB, 16-byte non-temporal accesses).  Its
 * rate, 2*bytes over its time, is the achievable HBM ceiling the
 * bandwidth-bound kernels (momentum/norm prologue, AdamW) are compared to. */
muon_status_t muon_stream_copy(muon_handle_t h, void* dst, const void* src, size_t bytes,
                               void* stream);

const char* muon_status_string(muon_status_t s);
/* Message of the last failure on h (empty string if none); valid until the
 * next call on h. */
const char* muon_last_error(muon_handle_t h);
int muon_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* MUON_HIP_H */
