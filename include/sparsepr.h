/*
 * sparsepr.h -- C ABI of the MI355X (gfx950) SparsePR sparse attention library.
 *
 * SparsePR ("Partition the Support, Reconstruct the Residual") replaces dense
 * softmax attention of one head, O = softmax(Q K^T / sqrt(d)) V (Sec. 3,
 * eq. dense_attention), by
 *   1. Response-Coupled Partitioning (Sec. 4.1, App. B): paired K/V groups from
 *      k-means on key-response coordinates phi_K = F_K^T k, then query groups
 *      from k-means on the centroid-induced query coordinates phi_Q;
 *   2. shared block routing of query-group x K/V-group cells under a pair
 *      budget that charges each cell |G_a| |G_b| and reserves the probes' cost
 *      first (Sec. 4.3, eq. pair_density);
 *   3. renormalised hard-drop sparse attention over the routed cells, on
 *      group-major permuted K/V (Sec. 3, eq. hard_drop; Sec. 4.3);
 *   4. Probe-Fitted Residual Reconstruction (Sec. 4.2, App. A): exact rows for
 *      M probe queries, a weighted ridge fit of the residual on the sparse
 *      output restricted to the probes' residual subspace, and the affine
 *      correction applied to every other row (eq. final_reconstructed_output).
 *
 * The work is split in two calls that follow that statement of the problem:
 * sparsepr_plan (steps 1-2 and the probe choice of App. A.2) and
 * sparsepr_attend (steps 3-4 and the restore to the original row order).
 *
 * Conventions (all entry points):
 *  - Q, K, V and the output are DEVICE pointers to [batch, heads, n, d]
 *    tensors addressed with element strides (stride_b, stride_h, stride_n);
 *    the last dimension is contiguous.  dtype is float32 or bfloat16 for all
 *    four; accumulation is always at least float32.
 *  - Every batch x head pair is an independent SparsePR call with the same
 *    parameters; all of them are processed by each launch.
 *  - Grouped-query attention (heads_kv < heads): query heads h*G .. h*G+G-1
 *    (G = heads / heads_kv) attend to K/V head h, and share its partition,
 *    routes and probe rows (Sec. 4.3: K/V partition and routing metadata are
 *    shared across the associated query heads; App. B.1: M_K per K/V head).
 *    The plan of a K/V head pools its G query heads: M_K averages their
 *    strided-sample metrics, the query-response coordinates phi_Q average
 *    their per-head normalised coordinates, and the route scores use the
 *    query-group means averaged over them.  Every query head then runs its
 *    own sparse attention, exact probe rows, fit and correction.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Work is enqueued asynchronously on it; the caller keeps Q, K, V, the
 *    output and the workspace alive until that work has completed.  Only
 *    sparsepr_get_stats and sparsepr_plan_export synchronise the stream.
 *  - The caller owns all memory.  The library never allocates device memory:
 *    everything it needs lives in the caller's workspace (or, for a plan made
 *    by sparsepr_plan_create_static, in the library's static device array).
 *  - Every entry point returns a status; no C++ exception crosses the ABI.
 *    Arguments are validated on the host before anything is enqueued, and a
 *    call that fails validation has no side effects.  sparsepr_last_error()
 *    describes the most recent failure of the calling thread.
 */
#ifndef SPARSEPR_H
#define SPARSEPR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPARSEPR_OK = 0,
  SPARSEPR_ERR_INVALID_ARGUMENT = 1, /* bad pointer, size or parameter range */
  SPARSEPR_ERR_UNSUPPORTED = 2,      /* valid but not implemented (e.g. d = 96) */
  SPARSEPR_ERR_WORKSPACE_TOO_SMALL = 3,
  SPARSEPR_ERR_HIP = 4,              /* a HIP runtime call failed */
  SPARSEPR_ERR_NUMERICAL = 5         /* reported by sparsepr_get_stats only */
} sparsepr_status;

typedef enum { SPARSEPR_F32 = 0, SPARSEPR_BF16 = 1 } sparsepr_dtype;

/* Tensor geometry.  Self-attention only: n_q == n_kv.  d == d_v in {64, 128}. */
typedef struct {
  int32_t batch, heads;                 /* heads = query heads (Q and the output) */
  int32_t n_q, n_kv;
  int32_t d, d_v;
  int64_t stride_b, stride_h, stride_n; /* element strides of Q and O; stride_n also of K, V */
  int32_t dtype;                        /* sparsepr_dtype */
  int32_t heads_kv;                     /* K/V heads, a divisor of heads; 0 = heads */
  int64_t kv_stride_b, kv_stride_h;     /* batch and head strides of K and V; 0 = stride_b,
                                           stride_h (required when heads_kv < heads) */
} sparsepr_shape;

/* Per-call method parameters (paper defaults from App. C.2 where it gives them). */
typedef struct {
  int32_t n_sampled_queries;   /* M_s: strided query sample for M_K (App. B.1); 256 */
  int32_t r_k, r_q;            /* response ranks r_K = 48, r_Q = 64 (clamped to d) */
  int32_t n_kv_groups;         /* C_k, K/V groups over the video rows */
  int32_t n_q_groups;          /* C_q, query groups over the video rows */
  int32_t kmeans_iters;        /* T, Lloyd iterations (cold start); 8 */
  float target_exec_density;   /* rho_exec target incl. probes (Sec. 4.3); 0.22 */
  int32_t n_probes;            /* M exact probe rows per head (App. A.2); 64 */
  int32_t resid_rank;          /* r, probe-residual output rank (Sec. 4.2); 16 */
  float ridge;                 /* lambda (eq. probe_ridge_fit); 0.1 */
  float eps_q;                 /* RMS floor of eq. query_response_feature; 1e-6 */
  float eps_x;                 /* variance floor of eq. app_feature_scale; 1e-6 */
  int32_t n_dense_prefix;      /* leading rows (e.g. text tokens) routed densely,
                                  outside clustering, probes and the budget; 0 */
  int32_t warm_start;          /* 1: both k-means start from the final centroids of
                                  this plan's previous sparsepr_plan call instead of
                                  the strided rows (the warm-started k-means of
                                  App. C.1, for consecutive calls such as denoising
                                  steps); the first call on a plan starts cold; 0 */
  int32_t warm_iters;          /* assignments of a warm-started k-means, in
                                  [1, kmeans_iters]; 0 = kmeans_iters; 0 */
  /* Ablation variants of Sec. 5.2 (Tables partition_repair_ablation and
   * probe_estimator_ablation); the defaults are the method itself. */
  int32_t partition;           /* SPARSEPR_PARTITION_*; RESPONSE */
  int32_t probe_rule;          /* SPARSEPR_PROBES_*; STRATIFIED */
  uint32_t probe_seed;         /* seed of SPARSEPR_PROBES_RANDOM; 0 */
  int32_t ridge_only;          /* 1: ridge estimator without the probe-residual
                                  output subspace (Psi = I, so the correction is
                                  xbar B_lambda); 0 */
  int32_t routing;             /* SPARSEPR_ROUTING_*; PRIORITY */
} sparsepr_params;

/* partition: how the K/V and query groups are formed.
 *   RESPONSE      response-coupled partitioning (Sec. 4.1, App. B);
 *   SEMANTIC      the reference partition of Sec. 3.1: k-means on the raw
 *                 keys (values inherit their key's group) and, separately,
 *                 on the raw queries;
 *   KEY_RESPONSE  K/V groups from the key-response coordinates phi_K, query
 *                 groups from k-means on the raw queries (Sec. 5.2). */
#define SPARSEPR_PARTITION_RESPONSE 0
#define SPARSEPR_PARTITION_SEMANTIC 1
#define SPARSEPR_PARTITION_KEY_RESPONSE 2
/* probe_rule: which rows are evaluated exactly (Table probe_estimator_ablation).
 *   STRATIFIED  query-group-stratified selection (App. A.2, Algorithm
 *               app_probe_selection) with coverage weights |G_a| / m_a;
 *   RANDOM      M distinct video rows uniformly at random: the M rows with the
 *               smallest SplitMix64(probe_seed * 2^32 + row) (the mixing
 *               function of Steele, Lea and Flood 2014), in that order;
 *   UNIFORM     evenly spaced video rows floor((2i + 1) n_v / (2M)), i < M
 *               (tokens are in raster order, so these spread over space and
 *               time).
 * RANDOM and UNIFORM weigh every probe equally, w_p = n_v / M. */
/* routing: which cells the pair budget buys (Sec. 4.3).  Both keep the best
 * cell of every nonempty query group (forced) and walk the other cells in a
 * fixed order, taking the longest prefix whose pair cost fits the budget.
 *   PRIORITY  order of the centroid estimate of the per-pair log probability
 *             pi_ab = s_ab - lse_a, descending (the cost-aware greedy);
 *   TOP_P     per-group top-p with one p for all query groups, the largest
 *             whose cost fits: a group takes its cells in pi order until their
 *             estimated attention mass m_ab = |G_b| exp(pi_ab) (which sums to 1
 *             over b) reaches p.  Cell (a, b) is in the top-p set exactly when
 *             the mass ranked before it in its group, e_ab, is below p, so the
 *             walk is in e_ab ascending order (e_ab in double, the group's
 *             order being pi descending, b ascending).
 * Ties in the walk go to the lower flat index a * C_k + b. */
#define SPARSEPR_ROUTING_PRIORITY 0
#define SPARSEPR_ROUTING_TOP_P 1
#define SPARSEPR_PROBES_STRATIFIED 0
#define SPARSEPR_PROBES_RANDOM 1
#define SPARSEPR_PROBES_UNIFORM 2

/* Realised accounting of one call (Sec. 4.3: rho_exec = rho_route + M/N_q).
 * Pair and probe counts are summed over query heads (every query head of a
 * group evaluates its K/V head's cells); cells, groups and k-means figures
 * over plans (K/V heads). */
typedef struct {
  double rho_route;          /* routed pairs / (n_q n_kv), mean over heads */
  double rho_exec;           /* rho_route + probes / n_q, mean over heads */
  int64_t routed_pairs;      /* sum over heads (includes forced and dense-prefix cells) */
  int64_t exec_pairs;        /* routed_pairs + probes * n_kv, sum over heads */
  int64_t forced_pairs;      /* pairs of cells kept regardless of the budget */
  int32_t routed_cells;      /* sum over heads (video x video cells) */
  int32_t forced_cells;
  int32_t nonempty_q_groups; /* sum over heads */
  int32_t nonempty_kv_groups;
  int32_t n_probes;          /* sum over heads */
  int32_t kmeans_iters_kv;   /* max over heads of assignments performed */
  int32_t kmeans_iters_q;
  int32_t status_flags;      /* OR over heads of SPARSEPR_FLAG_* */
  int64_t kmeans_rescans;    /* points whose assignment needed the exact scan over
                                every centroid, summed over heads, both k-means and
                                all assignments (a cost diagnostic) */
} sparsepr_stats;

#define SPARSEPR_FLAG_NONFINITE_INPUT 1 /* a NaN/Inf reached the partition features */
#define SPARSEPR_FLAG_FIT_NOT_PD 2      /* ridge normal matrix not positive definite; correction
                                           reduced to the mean residual */
#define SPARSEPR_FLAG_BUDGET_BELOW_FORCED 4 /* forced cells alone exceed the pair budget */
#define SPARSEPR_FLAG_EIG_JACOBI 8 /* an eigenproblem (response basis, residual basis) was
                                      solved by cyclic Jacobi instead of the tridiagonal
                                      solver: a numerically repeated retained eigenvalue, or
                                      (double fit) retained eigenvalues below 1e-5 of the
                                      largest.  A cost diagnostic: both give the same basis */

/* Host-side view of one head's plan, for export (diagnostics, oracle replay)
 * and import (running attend on a plan made elsewhere).  All arrays are HOST
 * memory owned by the caller; a NULL pointer skips that array.  Sizes use
 * n = n_q, n_v = n - n_dense_prefix, C_q/C_k = the group counts, and
 * Cq_t = C_q + (n_dense_prefix > 0), Ck_t = C_k + (n_dense_prefix > 0) (the
 * dense prefix forms the extra last group on each side). */
typedef struct {
  /* plan content: exported, and read by import */
  int32_t* labels_q;     /* [n]  query group of each row, in [0, Cq_t) */
  int32_t* labels_kv;    /* [n]  K/V group of each row, in [0, Ck_t) */
  uint8_t* routes;       /* [Cq_t * Ck_t] 1 = cell evaluated */
  int32_t* probes;       /* [n_probes] probe rows in selection order */
  int32_t n_probes;      /* export: written; import: number of entries in probes */
  /* derived data: export only */
  float* probe_weights;  /* [n_probes] coverage weights w_p = |G_a| / m_a */
  int32_t* perm_q;       /* [n]  group-major order of the query rows */
  int32_t* off_q;        /* [Cq_t + 1] */
  int32_t* perm_kv;      /* [n] */
  int32_t* off_kv;       /* [Ck_t + 1] */
  float* m_k;            /* [d*d] key-response metric */
  float* m_q;            /* [d*d] query-response metric */
  float* f_k;            /* [d * r_k] eigen-scaled key basis */
  float* f_q;            /* [d * r_q] */
  float* phi_k;          /* [n_v * r_k] key-response coordinates */
  float* phi_q;          /* [n_v * r_q] query-response coordinates */
  float* cent_k;         /* [C_k * r_k] final K/V k-means centroids */
  float* cent_q;         /* [C_q * r_q] final query k-means centroids (probe means) */
  float* kbar;           /* [C_k * d] key-space group means */
  float* qbar;           /* [C_q * d] query-space group means */
  float* route_prio;     /* [C_q * C_k] route priorities (0 for empty groups) */
  /* after sparsepr_attend: */
  float* o_sparse;       /* [n * d_v] hard-drop output, original row order */
  float* o_dense_probes; /* [n_probes * d_v] exact probe rows */
  float* fit_mu_x;       /* [d_v] */
  float* fit_s_x;        /* [d_v] */
  float* fit_mu_r;       /* [d_v] */
  float* fit_bpsi;       /* [d_v * r] B_lambda Psi_r (the ridge map times the basis) */
  float* fit_psi;        /* [d_v * r] Psi_r (columns beyond fit_rank are 0) */
  int32_t fit_rank;      /* export: retained residual rank */
  float* route_key;      /* [C_q * C_k] key of the routing walk (larger first): route_prio
                            under PRIORITY, -(float)e_ab under TOP_P (0 for empty groups) */
} sparsepr_plan_host;

typedef struct sparsepr_plan_s* sparsepr_plan_t;

/* Fill `p` with the paper's defaults (App. C.2) and C_k = C_q = 0, which
 * sparsepr_plan_create replaces by ceil(n_v / 64). */
void sparsepr_params_default(sparsepr_params* p);

/* Bytes of device workspace one plan needs for this shape and parameters.
 * Errors: INVALID_ARGUMENT / UNSUPPORTED as for sparsepr_plan_create. */
sparsepr_status sparsepr_workspace_size(const sparsepr_shape* shape, const sparsepr_params* params,
                                        size_t* bytes);

/* Validate shape and parameters and bind a device workspace of `bytes`
 * bytes (256-byte aligned) to a new plan handle.  The handle owns only host
 * metadata; the workspace remains the caller's.  Constraints
 * (INVALID_ARGUMENT otherwise): batch, heads >= 1; n_q == n_kv >= 1;
 * 0 <= n_dense_prefix < n_q; 1 <= C_k, C_q <= n_v; 1 <= r_k, r_q;
 * 1 <= M_s; 0 <= M; 1 <= r <= d_v; 0 < rho <= 1; ridge >= 0; eps >= 0;
 * stride_n >= d; heads_kv a divisor of heads, with kv_stride_b and
 * kv_stride_h given when heads_kv < heads.  UNSUPPORTED: d != d_v, d not in {64, 128}, C_k or C_q
 * above 8191, n_q above 2^24, strides not multiples of 8 elements,
 * n_kv * stride_n * element size of 4 GiB or more (one head's K/V rows are
 * addressed with 32-bit byte offsets).
 * Tuning: the bf16 sparse attention runs in key segments of about 6 MiB of
 * one head's group-major K+V each (one launch per segment, sized for one
 * XCD's L2); the environment variable SPARSEPR_SEG_KB, read here, overrides
 * that size in KiB (at least 64).  The result is the same up to the fp32
 * rounding of the regrouped tiles. */
sparsepr_status sparsepr_plan_create(const sparsepr_shape* shape, const sparsepr_params* params,
                                     void* workspace, size_t bytes, sparsepr_plan_t* out);

/* For callers that cannot allocate device memory (code under graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same as
 * sparsepr_plan_create, but the plan is bound to a file-scope device array of
 * the library (64 MiB; each device the library runs on holds one copy until
 * the process ends) instead of a caller workspace.  Nothing is allocated: no
 * hipMalloc, hipFree or allocating library routine.  The array's address on
 * the current device is looked up on the first call on that device.
 * Shapes whose workspace (sparsepr_workspace_size) exceeds 64 MiB are
 * rejected with WORKSPACE_TOO_SMALL.  One device has one array: while a plan
 * made by this entry point is alive (until sparsepr_plan_destroy), another
 * call on the same device fails with INVALID_ARGUMENT; work enqueued for it
 * on several streams at once races like any plan used concurrently.  The
 * array keeps what the last plan left; the plan clears what it must start
 * from.  The returned plan is used with sparsepr_plan, sparsepr_attend and the
 * other calls exactly like one from sparsepr_plan_create. */
sparsepr_status sparsepr_plan_create_static(const sparsepr_shape* shape,
                                            const sparsepr_params* params, sparsepr_plan_t* out);

/* Response-Coupled Partitioning, routing and probe choice for every head
 * (Sec. 4.1, Sec. 4.3, App. A.2, App. B).  Reads Q and K only (values never
 * enter the partition, App. B.1). */
sparsepr_status sparsepr_plan(sparsepr_plan_t plan, const void* q, const void* k, void* stream);

/* Sparse attention over the routed cells, exact probe rows, residual fit and
 * correction (Sec. 4.2-4.3, App. A); writes the output [batch, heads, n, d_v]
 * in the original row order.  Uses the plan made by the last sparsepr_plan or
 * sparsepr_plan_import on this handle; `q`, `k` must be the tensors it was
 * made from. */
sparsepr_status sparsepr_attend(sparsepr_plan_t plan, const void* q, const void* k,
                                const void* v, void* out, void* stream);

/* Dense attention of Sec. 3 (eq. dense_attention) for every head, on the same
 * kernels the probes use; for error reporting.  Needs no plan, allocates
 * nothing; `workspace` must hold sparsepr_dense_workspace_size bytes. */
sparsepr_status sparsepr_dense_workspace_size(const sparsepr_shape* shape, size_t* bytes);
sparsepr_status sparsepr_dense_attend(const sparsepr_shape* shape, const void* q, const void* k,
                                      const void* v, void* out, void* workspace, size_t bytes,
                                      void* stream);

/* Synchronise `stream` and read the realised accounting of the last call. */
sparsepr_status sparsepr_get_stats(sparsepr_plan_t plan, sparsepr_stats* out, void* stream);

/* Copy the plan used by query head `bh` (= b * heads + h), i.e. that of K/V
 * head b * heads_kv + h / G, and, after attend, query head bh's own outputs
 * into caller host buffers.  Synchronises `stream`. */
sparsepr_status sparsepr_plan_export(sparsepr_plan_t plan, int32_t bh, sparsepr_plan_host* out,
                                     void* stream);

/* Replace the plan used by query head `bh` (that of its K/V head, shared by
 * the whole group) by labels_q, labels_kv, routes and probes
 * from host memory (all four required).  Group-major permutations, offsets,
 * route lists and coverage weights are rebuilt on the device.  Errors:
 * INVALID_ARGUMENT for out-of-range labels or probes. */
sparsepr_status sparsepr_plan_import(sparsepr_plan_t plan, int32_t bh, const sparsepr_plan_host* in,
                                     void* stream);

/* Device time per phase, measured with HIP events recorded on the call's
 * stream around each phase (Sec. 4.3 lists what a call's latency covers).
 * Accumulated over the calls made while profiling was enabled. */
typedef struct {
  double plan_ms;         /* partitioning, routing and probe choice */
  double sparse_attn_ms;  /* the block-sparse attention launches alone (one per key
                             segment: a slice of the group-major keys sized to
                             stay resident in L2) */
  double probe_ms;        /* exact probe rows and their merge */
  double fit_ms;          /* residual fit */
  double correct_ms;      /* correction, restore and probe rows */
  int32_t plan_calls;
  int32_t attend_calls;
  int32_t attn_launches;  /* sparse-attention launches per attend call */
} sparsepr_timings;

/* Enable (1) or disable (0) event timing on this handle.  Creating the events
 * is the only thing it does; no device memory is allocated. */
sparsepr_status sparsepr_set_profiling(sparsepr_plan_t plan, int32_t enable);

/* Synchronise `stream`, write the accumulated timings, and reset them when
 * `reset` is nonzero.  INVALID_ARGUMENT when profiling is not enabled. */
sparsepr_status sparsepr_get_timings(sparsepr_plan_t plan, sparsepr_timings* out, int32_t reset,
                                     void* stream);

/* Release the handle (not the workspace).  NULL is ignored. */
void sparsepr_plan_destroy(sparsepr_plan_t plan);

/* Text of the calling thread's most recent failure ("" if none); valid until
 * that thread's next call into the library. */
const char* sparsepr_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SPARSEPR_H */
