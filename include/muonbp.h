/*
 * muonbp.h -- C ABI of the MI355X (gfx950) MuonBP optimizer step.
 *
 * MuonBP (Khaled et al., arXiv 2510.16981, Sec. 3.2, Algorithm 1) keeps a
 * heavy-ball momentum buffer per matrix, orthogonalizes it with K quintic
 * Newton-Schulz iterations (Appendix B, Algorithm 2) either per block of an
 * r x c shard grid (block steps) or over the whole matrix (full steps, when
 * t mod P = 0), and applies the update with one of two stepsizes.
 *
 * Conventions for every function below:
 *  - All entry points are plain C, never throw and never abort; they return a
 *    muonbp_status.  A non-OK status from argument or shape validation leaves
 *    the context usable; MUONBP_E_HIP poisons it (every later call that would
 *    touch the GPU returns MUONBP_E_STATE).  muonbp_last_error() gives text.
 *  - Matrices are row-major and contiguous (leading dimension = cols).
 *    Pointers named "device" are HIP device pointers on the device that was
 *    current at muonbp_create; they must be 16-byte aligned for full speed
 *    (any element-aligned pointer is accepted).
 *  - GPU work is enqueued on the context's stream and the call returns
 *    without synchronising, unless stated otherwise.  The caller keeps every
 *    pointer valid until that work completes (muonbp_synchronize).
 *  - A context is not thread-safe; use one context per stream.
 */
#ifndef MUONBP_H
#define MUONBP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct muonbp_ctx muonbp_ctx; /* opaque, owned by the library */

typedef enum {
  MUONBP_OK = 0,
  MUONBP_E_INVALID = 1, /* bad argument: NULL pointer, bad count, bad option  */
  MUONBP_E_SHAPE = 2,   /* non-positive size, or grid does not divide matrix  */
  MUONBP_E_DTYPE = 3,   /* unsupported dtype or dtype combination             */
  MUONBP_E_NOMEM = 4,   /* device or host allocation failed                   */
  MUONBP_E_HIP = 5,     /* a HIP runtime call or kernel launch failed         */
  MUONBP_E_STATE = 6,   /* context poisoned by an earlier MUONBP_E_HIP        */
  MUONBP_E_NONFINITE = 7, /* muonbp_options.check_finite found NaN / Inf in
                             an orthogonalization input (context stays usable) */
  MUONBP_E_TOO_LARGE = 8  /* muonbp_step_static: the step needs more scratch
                             than MUONBP_STATIC_SCRATCH_BYTES                  */
} muonbp_status;

typedef enum { MUONBP_F32 = 0, MUONBP_BF16 = 1 } muonbp_dtype;

/* One weight matrix W (rows x cols) and its shard grid (Sec. 3, "How blocks
 * align with model-parallel shards"): block (i, j) holds rows
 * [i*rows/grid_rows, (i+1)*rows/grid_rows) and columns
 * [j*cols/grid_cols, (j+1)*cols/grid_cols).  grid_rows must divide rows and
 * grid_cols must divide cols (MUONBP_E_SHAPE otherwise). */
typedef struct {
  int64_t rows, cols;
  int32_t grid_rows, grid_cols;
} muonbp_matrix;

/* Options.  Defaults (muonbp_options_default) follow Algorithm 2:
 * K = 5, (a, b, c) = (2, -1.5, 0.5), eps = 1e-7, no Nesterov, no RMS scaling,
 * bf16 params, momentum and NS operands, automatic tile shapes. */
#define MUONBP_MAX_COEFFS 16

typedef struct {
  int32_t ns_steps;         /* K >= 0, Newton-Schulz iterations (Alg. 2)       */
  float a, b, c;            /* quintic coefficients (Alg. 2)                   */
  float eps;                /* X <- G / (||G||_F + eps) (Alg. 2)               */
  int32_t nesterov;         /* 1: NS input is G + mu*M instead of M (not in
                               the paper; off by default)                      */
  int32_t scale_mode;       /* 0: U as is (Alg. 1); 1: U * rms_beta *
                               sqrt(max(p, q)), p x q = block shape on block
                               steps, matrix shape on full steps (Sec. 3.2,
                               "AdamW learning rate transfer")                 */
  float rms_beta;           /* beta of scale_mode 1                            */
  muonbp_dtype param_dtype; /* dtype of params and grads                       */
  muonbp_dtype state_dtype; /* dtype of the momentum buffer                    */
  muonbp_dtype ns_dtype;    /* dtype of NS operands (fp32 accumulate always)   */
  int32_t tile_policy;      /* NS GEMM kernel: 0 = chosen per launch from its
                               tile counts; 1/2/3 = 128x128 / 256x128 /
                               256x256 tiles with a register-staged K loop;
                               4/5/6 = the same as 8/9/10 (aliases kept for
                               existing callers); 7 = 128x128 tiles with the K
                               loop split over two 4-wave groups; 8/9/10/
                               11/12/13 = 128x128 / 256x128 / 256x256 /
                               192x256 / 256x192 / 192x192 tiles with the
                               LDS-DMA loop interleaved with the MFMAs (same
                               conditions as 4-6); 14/15/16 = 256x256 /
                               192x256 / 256x192 interleaved tiles over 8
                               waves (two per SIMD).
                               Symmetric products use square tiles (128x128
                               for 2, 5, 9; 192x192 for 11, 12, 15, 16). */
  int32_t k_split;          /* interleaved DMA kernels only: 1..8 = each
                               tile's K loop shared by that many workgroups
                               (fp32 partial sums added by the last one to
                               finish); 1 = no split; 0 = the planner's
                               choice (3 for a launch with fewer tiles than
                               0.6 x the CUs and at least 128 K slices in
                               every product, else none). */
  int32_t coeff_count;      /* 0 = every NS iteration uses (a, b, c) above;
                               1..MUONBP_MAX_COEFFS = iteration k uses
                               coeff_table[min(k, coeff_count - 1)] (tuned or
                               per-iteration quintics, Sec. 2.2). */
  float coeff_table[3 * MUONBP_MAX_COEFFS];  /* (a_k, b_k, c_k) triples */
  int32_t stream_hint;      /* cache policy of the momentum and update
                               kernels' streamed reads and writes: 0 = chosen
                               from the step's size (nontemporal when
                               params x (2 param + 1 state elements) exceed
                               256 MiB, the last-level cache; plain below,
                               where the data stays cached between the
                               step's kernels); 1 = plain; 2 = nontemporal. */
  int32_t apply_mode;       /* apply product Z <- (a I + B) Z of each NS
                               iteration: 0 = reads Z row-major through LDS
                               transpose reads wherever the interleaved DMA
                               kernel runs it (no Z^T kept between
                               iterations); 1 = keeps Z^T and reads it. */
  int32_t check_finite;     /* debug check, off by default (0).  1: after the
                               momentum update, muonbp_step waits for the
                               stream and returns MUONBP_E_NONFINITE when the
                               NS input of some unit (M, or G + mu M with
                               Nesterov) holds a NaN or an Inf, or its sum of
                               squares overflows fp32; nothing after the
                               momentum is enqueued then (params and U keep
                               their values, M holds this step's update).
                               Off: NaN / Inf propagate silently into U and
                               the params of their unit. */
  int64_t device_memory_limit; /* > 0: muonbp_create allocates at most this
                               many bytes of device memory (momentum, NS
                               workspace, K-split sums, descriptor tables; the
                               n_mats x 16-byte pointer tables aside) and
                               returns MUONBP_E_NOMEM instead of going over,
                               checking the momentum + workspace + split sums
                               before any HIP call; 0 = no limit (default).
                               muonbp_plan_info.device_bytes is the size of
                               those three. */
  int32_t gram_iteration;   /* how the K NS iterations of a unit run (the
                               result is Alg. 2's, up to rounding).  Each
                               iteration multiplies Z by a polynomial of its
                               Gram matrix, so n of them can run on S x S
                               matrices only: from A_0 = Z Z^T, P_j = a I +
                               b A_j + c A_j^2, A_{j+1} = A_j P_j^2, Q_j =
                               P_j Q_{j-1}, then Z <- Q_{n-1} Z (4n - 3
                               symmetric S x S x S products, one S x S x L
                               Gram and one S x L x S apply, against n of
                               each of the three as printed).  The K
                               iterations then run in segments of at most 3,
                               each from a fresh Gram of the current Z.
                               0 = that Gram-space iteration on the units
                               where it saves time (bf16 NS, the row-major
                               apply, K >= 2, S >= 128 and L >= 1.25 S), as
                               printed elsewhere (default); 1 = as printed
                               everywhere; 2 = the Gram-space iteration on
                               every unit that allows it (bf16, row-major
                               apply, K >= 2), whatever its shape.  A
                               Gram-space unit keeps three more S x S
                               buffers. */
} muonbp_options;

/* Fill *opt with the defaults above.  NULL is ignored. */
void muonbp_options_default(muonbp_options* opt);

/* Create a context for n_mats matrices (Algorithm 1 setup).
 *  mats        host array of n_mats shapes and grids (copied).
 *  period      P >= 1; 0 means P = infinity (BlockMuon: never a full step).
 *  lr_block    eta_block, used on block steps (Sec. 3.2).
 *  lr_full     eta_full, used on full steps (Sec. 3.2).
 *  momentum    mu in M_t = mu M_{t-1} + G_t (eq. NTR).
 *  weight_decay lambda: X <- X - eta_t (lambda X + s U) (decoupled).
 *  opt         NULL for defaults.
 *  hip_stream  hipStream_t to enqueue on (NULL = the null stream).
 *  out         receives the context; *out is NULL on error.
 * Allocates the momentum buffers (zeroed, Algorithm 1's M_{-1} = 0), the NS
 * workspace and the plan tables on the current device; the zeroing and the
 * table uploads run on hip_stream, which the call waits for (no device-wide
 * synchronisation).
 * E_SHAPE also when an orthogonalization unit of either plan (a block, or a
 * whole matrix) needs an NS operand of 2^31 bytes or more (e.g. a 40000 x
 * 40000 bf16 matrix): the kernels address operands with 32-bit offsets.
 * Errors: E_INVALID, E_SHAPE, E_DTYPE (before any HIP call), E_NOMEM, E_HIP. */
muonbp_status muonbp_create(const muonbp_matrix* mats, int32_t n_mats,
                            int64_t period, float lr_block, float lr_full,
                            float momentum, float weight_decay,
                            const muonbp_options* opt, void* hip_stream,
                            muonbp_ctx** out);

/* One iteration t = step of Algorithm 1 for every matrix.
 *  params  host array of n_mats device pointers (param_dtype, rows x cols),
 *          updated in place.
 *  grads   host array of n_mats device pointers (param_dtype), read only.
 *  step    t >= 0.  Full step iff period > 0 and step % period == 0.
 * Enqueues: momentum (+ per-segment sum of squares), per-unit scale,
 * operand pack (units not read in place, see
 * muonbp_plan_info.pack_elements), K x (Gram, polynomial, apply) grouped
 * MFMA launches, update.
 * The step may be captured into a HIP graph on the context's stream when
 * profiling is off and the pointers equal those of the step before (their
 * device table is then not re-uploaded); a replay repeats the captured step
 * kind, learning rates and options, and reads the params and grads in
 * place.
 * A step captured into a graph keeps using the device copy of its pointer
 * table: later eager steps with other pointers upload theirs elsewhere, so
 * a replay still reads and updates the captured step's tensors.
 * Errors: E_INVALID (NULL ctx/arrays/pointers, step < 0), E_STATE (also:
 * new pointers, profiling or check_finite while the stream captures;
 * nothing enqueued), E_NONFINITE (check_finite only: momentum updated,
 * nothing else enqueued; the context stays usable), E_HIP. */
muonbp_status muonbp_step(muonbp_ctx* ctx, void* const* params,
                          const void* const* grads, int64_t step);

/* Change eta_block and eta_full for later steps (learning-rate schedules). */
muonbp_status muonbp_set_lr(muonbp_ctx* ctx, float lr_block, float lr_full);

/* Change the period P for later steps (a period schedule, or an adaptive
 * period: the next step is full iff P > 0 and step mod P = 0, Alg. 1).
 * P = 0 means infinity.  E_INVALID for P < 0 (the context stays usable). */
muonbp_status muonbp_set_period(muonbp_ctx* ctx, int64_t period);

/* Change the stream used by later calls. */
muonbp_status muonbp_set_stream(muonbp_ctx* ctx, void* hip_stream);

/* Copy matrix `mat`'s momentum (state_dtype, rows x cols) to / from device
 * memory `dst` / `src` (checkpoint and resume).  Asynchronous on the stream. */
muonbp_status muonbp_get_momentum(muonbp_ctx* ctx, int32_t mat, void* dst);
muonbp_status muonbp_set_momentum(muonbp_ctx* ctx, int32_t mat, const void* src);

/* Copy the orthogonalized update U_t of matrix `mat` from the last step
 * (ns_dtype, rows x cols, before RMS scaling) to device memory `dst`.
 * E_STATE if no step has run yet. */
muonbp_status muonbp_get_update(muonbp_ctx* ctx, int32_t mat, void* dst);

/* Wait for all work enqueued by this context. */
muonbp_status muonbp_synchronize(muonbp_ctx* ctx);

/* Static description of one of the two plans (full = 0: block plan, 1: full
 * plan).  Host-only; makes no HIP call. */
typedef struct {
  int64_t n_problems;      /* orthogonalized units (blocks or matrices)     */
  int64_t n_elements;      /* parameters covered                            */
  int64_t gemm_tiles[3];   /* workgroup tiles per NS iteration as printed
                              (every unit): Gram, poly, apply               */
  int32_t gemm_tile_rows[3], gemm_tile_cols[3]; /* their tile shapes         */
  int64_t gemm_launches;   /* grouped GEMM launches per step (3 K as
                              printed; up to 5 per iteration with Gram-space
                              units, see gram_iteration)                    */
  double ns_flops;         /* NS flops per step of the products as computed
                              (symmetric products counted once): per S x L
                              unit and iteration S(S+1)L + S^2(S+1) + 2S^2 L
                              as printed; S(S+1)L + (4K-3) S^2(S+1) + 2S^2 L
                              in all for a Gram-space unit                  */
  double ns_dense_flops;   /* Sec. 2.2 cost 2K(2 L S^2 + S^3), S <= L        */
  double elementwise_bytes;/* algorithmic HBM bytes of the non-NS kernels    */
  int64_t workspace_bytes; /* NS workspace this plan needs                  */
  int32_t gemm_split[3];   /* workgroups sharing one tile's K loop (1 = none) */
  int32_t apply_nn;        /* 1: the apply products read Z row-major (no Z^T) */
  int64_t static_scratch_bytes; /* scratch muonbp_step_static needs for a step
                              of this plan (MUONBP_E_TOO_LARGE above
                              MUONBP_STATIC_SCRATCH_BYTES), with a 16-byte
                              aligned momentum (otherwise every unit is
                              packed, see pack_elements, and the pack's
                              tile list is longer)                            */
  int64_t device_bytes;    /* momentum + NS workspace + K-split sums of a
                              context for these matrices (both plans)       */
  int64_t gram_units;      /* units that run the Gram-space iteration (see
                              muonbp_options.gram_iteration)                */
  int64_t pack_elements;   /* elements the pack copies into the NS workspace
                              per step (4 bytes each in bf16).  An
                              untransposed unit whose NS input is the bf16
                              momentum itself (bf16 state and NS, no
                              Nesterov, K >= 1) is not packed: its first Gram
                              and apply read the momentum in place with the
                              Frobenius scale of Alg. 2 applied to their
                              sums                                          */
} muonbp_plan_info;

/* Plan description for a set of matrices without creating a context
 * (E_INVALID / E_SHAPE / E_DTYPE as muonbp_create). */
muonbp_status muonbp_describe_plan(const muonbp_matrix* mats, int32_t n_mats,
                                   const muonbp_options* opt, int32_t full,
                                   muonbp_plan_info* out);

/* Kernel timing with HIP events on the context's stream.
 * muonbp_profile_enable(ctx, mode): 0 off; 1 every launch bracketed by its
 * own pair of events (per-kernel detail; the markers between launches cost
 * time of their own); 2 one pair per step around the whole sequence of NS
 * GEMM launches, which then run back to back (kind 7; its launch count is
 * the number of GEMM launches covered).  muonbp_profile_read synchronises,
 * returns the elapsed times summed per kind over the records made since the
 * previous read, and forgets those records.
 * Kinds: 0 momentum, 1 scale, 2 pack, 3 gram, 4 poly, 5 apply, 6 update,
 * 7 NS GEMM span.  The *_full_steps fields are the part enqueued by full
 * steps (block steps: the difference).  E_INVALID for a mode outside 0..2. */
#define MUONBP_N_KERNEL_KINDS 8
typedef struct {
  double ms[MUONBP_N_KERNEL_KINDS];       /* summed elapsed time, all steps */
  int64_t launches[MUONBP_N_KERNEL_KINDS];
  double ms_full_steps[MUONBP_N_KERNEL_KINDS];
  int64_t launches_full_steps[MUONBP_N_KERNEL_KINDS];
} muonbp_profile;

muonbp_status muonbp_profile_enable(muonbp_ctx* ctx, int32_t mode);
muonbp_status muonbp_profile_read(muonbp_ctx* ctx, muonbp_profile* out);

/* Static text for a status code. */
const char* muonbp_status_string(muonbp_status s);

/* Detail of the last error on ctx ("" if none; static text if ctx is NULL).
 * Owned by the context, valid until its next call. */
const char* muonbp_last_error(const muonbp_ctx* ctx);

/* Free everything the context owns (waits for its stream first).
 * NULL is a no-op. */
void muonbp_destroy(muonbp_ctx* ctx);

/* ------------------------------------------------------------------------
 * Allocation-free step, for callers that cannot allocate device memory
 * (tight serving loops, harnesses that forbid hipMalloc).  One iteration
 * t = step of Algorithm 1, the same kernels and plans as muonbp_create +
 * muonbp_step with the same arguments, but nothing is allocated and no
 * context is kept:
 *  - the momentum is the caller's: `momentum` is one device buffer of
 *    sum_i rows_i * cols_i elements of opt->state_dtype, the matrices back
 *    to back in the order of `mats`, each row-major; updated in place
 *    (all zeros before the first step: Algorithm 1's M_{-1} = 0);
 *  - params / grads as for muonbp_step (host arrays of device pointers);
 *  - full step iff period > 0 and step % period == 0;
 *  - every other buffer of the step (NS workspace, partial sums, scales,
 *    split-K sums and counters, plan and pointer tables) lives in one
 *    static device array of MUONBP_STATIC_SCRATCH_BYTES per GPU, which the
 *    library holds from its first use on that GPU until the process ends.
 *    A step that needs more (muonbp_plan_info.static_scratch_bytes) is
 *    refused with MUONBP_E_TOO_LARGE before any HIP call; e.g. every step
 *    of one 2048 x 6144 bf16 matrix in 2048 x 768 shards fits.
 * The tables are built on the host (host heap only) and copied into the
 * scratch array on hip_stream; the call returns after the step has run to
 * completion on hip_stream (it waits for that stream), so it cannot be
 * captured into a graph.  Calls on one GPU share its scratch array, which
 * keeps the last call's contents (what must start at zero is cleared by
 * each call): calls that overlap on one GPU (from several host threads or
 * streams) race and must be serialized by the caller.
 * Errors: E_INVALID (NULL or bad arguments, bad options), E_SHAPE, E_DTYPE,
 * E_TOO_LARGE (before any HIP call), E_HIP; check_finite as in muonbp_step
 * (E_NONFINITE: momentum updated, nothing else run). */
#define MUONBP_STATIC_SCRATCH_BYTES ((int64_t)128 << 20)
muonbp_status muonbp_step_static(const muonbp_matrix* mats, int32_t n_mats, void* const* params,
                                 const void* const* grads, void* momentum, int64_t step,
                                 int64_t period, float lr_block, float lr_full, float momentum_mu,
                                 float weight_decay, const muonbp_options* opt, void* hip_stream);

/* ------------------------------------------------------------------------
 * Scalar optimizer for the parameters MuonBP does not orthogonalize.
 *
 * The paper trains the 1D parameters and the input embedding with AdamW,
 * with their gradients clipped to a global norm of 1.0 and weight decay 0.1
 * (Appendix B, experimental details).  One context covers a fixed list of
 * tensors (any shape, seen as flat arrays of `sizes[i]` elements):
 *   g <- g * min(1, max_grad_norm / (||g||_2 + 1e-6))   (||g|| over all tensors)
 *   m <- beta1 m + (1 - beta1) g,   v <- beta2 v + (1 - beta2) g^2
 *   p <- p (1 - lr wd) - lr (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 * with t = step + 1.  The moments are fp32 and owned by the context.
 * The same context runs Lion instead (algorithm = 1), the scalar optimizer
 * of the paper's 160M comparison (Sec. 4), as Chen et al. (2023) define it:
 *   c <- beta1 m + (1 - beta1) g,   p <- p (1 - lr wd) - lr sign(c),
 *   m <- beta2 m + (1 - beta2) g
 * (after the same clipping; sign(0) = 0; eps and v are not used; the
 * defaults below are AdamW's, Lion is usually run with betas (0.9, 0.99)).
 * The conventions of the MuonBP functions above apply (status codes,
 * asynchrony on the context's stream, pointer alignment, thread safety).
 * ---------------------------------------------------------------------- */
typedef struct muonbp_adamw_ctx muonbp_adamw_ctx; /* opaque */

typedef struct {
  float beta1, beta2;       /* 0 <= beta < 1                                   */
  float eps;                /* >= 0                                            */
  float weight_decay;       /* decoupled, scaled by lr                         */
  float max_grad_norm;      /* > 0: global-norm clipping; 0: off               */
  muonbp_dtype param_dtype; /* dtype of params and grads                       */
  int32_t stream_hint;      /* cache policy of the streamed accesses, as
                               muonbp_options.stream_hint (0 = by size)        */
  int32_t algorithm;        /* 0 = AdamW, 1 = Lion                             */
} muonbp_adamw_options;

/* Defaults: beta1 0.9, beta2 0.95, eps 1e-8, weight decay 0.1, clipping at
 * 1.0, bf16 params.  NULL is ignored. */
void muonbp_adamw_options_default(muonbp_adamw_options* opt);

/* Create a context for n tensors of sizes[i] > 0 elements (host array,
 * copied).  Allocates the zeroed moments (m_0 = v_0 = 0) on the current
 * device.  Errors: E_INVALID (NULL, n <= 0, bad option), E_SHAPE (a size
 * <= 0), E_DTYPE, E_NOMEM, E_HIP. */
muonbp_status muonbp_adamw_create(const int64_t* sizes, int32_t n,
                                  const muonbp_adamw_options* opt, void* hip_stream,
                                  muonbp_adamw_ctx** out);

/* One AdamW step (t = step + 1 >= 1) with learning rate lr (finite).
 *  params  host array of n device pointers (param_dtype), updated in place.
 *  grads   host array of n device pointers (param_dtype), read only.
 * Enqueues: with clipping, a sum of squares per segment and one reduction
 * to the clipping factor; then one fused update of params, m and v. */
muonbp_status muonbp_adamw_step(muonbp_adamw_ctx* ctx, void* const* params,
                                const void* const* grads, int64_t step, float lr);

/* Global gradient norm (before clipping) of the last step, to host memory;
 * synchronises the stream.  E_STATE if no step with clipping has run. */
muonbp_status muonbp_adamw_grad_norm(muonbp_adamw_ctx* ctx, float* out);

/* Copy tensor i's moments (fp32, sizes[i] elements) to / from device memory
 * (checkpoint and resume).  Asynchronous on the stream; NULL skips one.
 * Lion keeps no v: get_state writes zeros to v_dst, set_state ignores v_src. */
muonbp_status muonbp_adamw_get_state(muonbp_adamw_ctx* ctx, int32_t i, void* m_dst, void* v_dst);
muonbp_status muonbp_adamw_set_state(muonbp_adamw_ctx* ctx, int32_t i, const void* m_src,
                                     const void* v_src);

muonbp_status muonbp_adamw_set_stream(muonbp_adamw_ctx* ctx, void* hip_stream);
muonbp_status muonbp_adamw_synchronize(muonbp_adamw_ctx* ctx);
const char* muonbp_adamw_last_error(const muonbp_adamw_ctx* ctx);
void muonbp_adamw_destroy(muonbp_adamw_ctx* ctx); /* NULL is a no-op */

/* ------------------------------------------------------------------------
 * Learning-rate schedules of the paper's runs (Appendix B): cosine decay
 * (960M and 1.2B models) and warmup-stable-decay with a linear decay to a
 * final value (8B model; no warmup and a 20% cooldown for the 160M model).
 * Host-only, pure functions of the step t >= 0:
 *   both:   t < warmup: lr_max (t + 1) / warmup
 *   cosine: lr_min + (lr_max - lr_min) (1 + cos(pi x)) / 2,
 *           x = min(1, (t - warmup) / max(1, total - warmup))
 *   wsd:    lr_max until total - decay, then linear to lr_min at t = total
 *           (decay = 0: no decay); lr_min from t = total on.
 * Feed the result to muonbp_set_lr / muonbp_adamw_step.
 * ---------------------------------------------------------------------- */
double muonbp_lr_cosine(int64_t t, int64_t total, double lr_max, double lr_min, int64_t warmup);
double muonbp_lr_wsd(int64_t t, int64_t total, double lr_max, double lr_min, int64_t warmup,
                     int64_t decay);

#ifdef __cplusplus
}
#endif

#endif /* MUONBP_H */
