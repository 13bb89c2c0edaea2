/*
 * SparsePR CPU oracle: plain, slow, obviously-correct reference for the
 * sparse attention operator of "Partition the Support, Reconstruct the
 * Residual" (Response-Coupled Partitioning, shared block routing, renormalised
 * hard-drop sparse attention, Probe-Fitted Residual Reconstruction).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may call this library.  It shares no code with
 * the GPU library: no headers, kernels, helpers or tables.
 *
 * Every function works on ONE attention head.  Matrices are row-major.
 * Floating point is accumulated in double unless the function says it takes
 * a decision in float on purpose (k-means scores, probe distances), in which
 * case the float expression is spelled out operation by operation.
 */
#ifndef SPARSEPR_ORACLE_H
#define SPARSEPR_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* OpenMP threads the oracle runs on. */
int or_num_threads(void);

/* Dense attention rows (Sec. 3, eq. dense_attention). out: n_rows x dv. */
void or_dense_rows(const float* q, const float* k, const float* v, int n_k, int d, int dv,
                   const int64_t* rows, int n_rows, double* out);

/* Renormalised hard-drop rows (Sec. 3, eq. hard_drop): row i of query group a
 * attends exactly the keys whose K/V group b has z[a*ck + b] = 1. */
void or_sparse_rows(const float* q, const float* k, const float* v, int n_k, int d, int dv,
                    const int32_t* labels_q, const int32_t* labels_kv, int ck, const uint8_t* z,
                    const int64_t* rows, int n_rows, double* out);

/* Key-response metric M_K = Q_s^T Q_s / M_s over the strided sample
 * s_i = floor(i*n/m_s) (Sec. 4.1, App. B.1 eq. app_key_metric). mk: d x d. */
void or_key_metric(const float* q, int n, int d, int m_s, double* mk);

/* Symmetric eigensolver (cyclic Jacobi, double).  evals descending,
 * evecs[i*n + j] = component i of eigenvector j. Returns sweeps used. */
int or_sym_eig(const double* a, int n, double* evals, double* evecs);

/* Eigen-scaled response basis (Sec. 4.1, App. B.1/B.2): leading r eigen-
 * directions of m, each scaled by sqrt(lambda / mean of the retained
 * lambdas); eigenvalues below tau*lambda_1 are clamped to 0 first.
 * f: d x r.  evals_out (optional): d eigenvalues, descending, after clamping. */
void or_response_basis(const double* m, int d, int r, double tau, double* f, double* evals_out);

/* phi = F^T x per row, rounded to float (eq. key_response_feature).  With
 * rms != 0 the row is divided by max(sqrt(|F^T x|^2 / r), eps)
 * (eq. query_response_feature).  phi: n x r. */
void or_project(const float* x, int n, int d, const double* f, int r, int rms, double eps,
                float* phi);

/* Lloyd k-means on float points (Sec. 4.1).  Init: c_b = pts[floor(b*n/c)].
 * Assignment score for point x and centroid c, in float, exactly:
 *   t = 0; for k: t = fmaf(x[k], c[k], t)      (dot product, index order)
 *   u = 0; for k: u = fmaf(c[k], c[k], u)      (squared norm, index order)
 *   score = fmaf(-2, t, u)
 * label = lowest b with the smallest score.  Update: per group, the members'
 * coordinates are summed in double in ascending point index, divided by the
 * count and rounded to float; an empty group keeps its centroid.  Stops after
 * `iters` assignments or when an assignment changes no label.
 * labels: n; cent: c x r (centroids after the update that follows the final
 * assignment); counts: c.  Returns the number of assignments performed. */
int or_kmeans(const float* pts, int n, int r, int c, int iters, int32_t* labels, float* cent,
              int32_t* counts);

/* The same Lloyd iterations started from the centroids `init` (c x r) instead
 * of the strided points: the warm-started k-means of App. C.1, which reuses the
 * previous call's centroids.  Returns the number of assignments performed. */
int or_kmeans_from(const float* pts, int n, int r, int c, int iters, const float* init,
                   int32_t* labels, float* cent, int32_t* counts);

/* One assignment step with the score above (exposed for stage tests).
 * scores (optional): n x c. */
void or_kmeans_assign(const float* pts, int n, int r, const float* cent, int c, int32_t* labels,
                      float* scores);

/* Group means in the input space: per group, double sum in ascending row
 * index / count, rounded to float; empty groups get 0.  mean: c x d. */
void or_group_mean(const float* x, int n, int d, const int32_t* labels, int c, float* mean,
                   int32_t* counts);

/* Query-response metric from key-space group centroids (App. B.2,
 * eq. app_query_metric): only nonempty groups, centred by their uniform mean,
 * M_Q = Kt^T Kt / (C_k^+ d). mq: d x d. */
void or_query_metric(const float* kbar, const int32_t* counts, int c, int d, double* mq);

/* Stable group-major permutation (Sec. 4.3): perm lists row indices ordered
 * by (label, index); off[b] = first slot of group b, off[c] = n. */
void or_stable_perm(const int32_t* labels, int n, int c, int32_t* perm, int32_t* off);

/* Route priorities pi_ab = s_ab - lse_a for nonempty a, b (0 elsewhere):
 *   s_ab = (float dot of qbar_a, kbar_b as an fmaf chain in index order) * scale,
 *          scale = (float)(1/sqrt(d))
 *   lse_a = log sum_b nk_b exp(s_ab) in double, rounded to float
 *   pi_ab = s_ab - lse_a in float.  prio: cq x ck. */
void or_route_priorities(const float* qbar, const int32_t* nq, int cq, const float* kbar,
                         const int32_t* nk, int ck, int d, float* prio);

/* Route selection under a pair budget (Sec. 4.3).  First every nonempty
 * query group takes its best nonempty K/V group (largest priority, lowest b on
 * ties).  The other nonempty cells are walked by (priority descending, a*ck+b
 * ascending) and the longest prefix whose cost nq_a*nk_b, added to the forced
 * cost, stays within `budget` is selected.  z: cq x ck (1 = routed).
 * out[0] = routed pairs, out[1] = forced pairs, out[2] = routed cells,
 * out[3] = forced cells. */
void or_route_select(const float* prio, const int32_t* nq, int cq, const int32_t* nk, int ck,
                     int64_t budget, uint8_t* z, int64_t* out);

/* Keys of the per-group top-p routing walk (reading of Sec. 4.3, one p for
 * every group, the largest that fits the budget): keys[a][b] = -(float)e_ab,
 * e_ab = sum of nk_b' exp((double)prio[a][b']) over the nonempty b' ranked
 * before b in (prio descending, b ascending) order, summed in that order.
 * Routing by top-p is or_route_select on these keys.  0 for empty groups. */
void or_route_topp_keys(const float* prio, const int32_t* nq, int cq, const int32_t* nk, int ck,
                        float* keys);

/* Query-group-stratified probe selection (App. A.2, Algorithm "Query-Group-
 * Stratified Exact Probe Selection") and coverage weights (eq. app_probe_weight).
 * Rows of a group are ordered by their squared distance to the group mean in
 * phi space (float: diff = phi - c; acc = fmaf(diff, diff, acc) in index
 * order), ties by row index.  Group order: ascending id when the number of
 * nonempty groups G <= m, otherwise by (rank mod s, rank) with s = ceil(G/m),
 * rank = position among the nonempty groups in ascending id.  Only rows with
 * labels < c take part.  Returns the number of probes (min(m, rows)). */
int or_probe_select(const float* phi, int n, int r, const int32_t* labels, int c,
                    const float* cent, int m, int32_t* probes, double* w);

/* Probe-fitted residual reconstruction fit (Sec. 4.2, App. A.3).
 * x, od: m x dv (sparse and dense outputs of the probes), w: coverage weights.
 * Outputs mu_x, s_x, mu_r (dv), b (dv x dv, the ridge solution),
 * psi (dv x r, columns beyond *rank are 0), g = b psi psi^T (dv x dv).
 * ridge_only: the estimator without the probe-residual subspace (Table
 * probe_estimator_ablation): Psi = I, g = b, *rank = dv (pass r = dv). 
 * Returns 0, or 1 when the regularised normal matrix is not positive
 * definite (then b = g = 0). */
int or_fit(const double* x, const double* od, const double* w, int m, int dv, int r,
           int ridge_only, double lambda, double eps, double* mu_x, double* s_x, double* mu_r,
           double* b, double* psi, double* g, int* rank);

/* Probe rules of the ablation (Sec. 5.2, Table probe_estimator_ablation),
 * over rows [0, n), equal weights n / m (as float):
 *   or_probe_uniform: rows floor((2i + 1) n / (2m)), i < m (evenly spaced in
 *     the raster token order);
 *   or_probe_random: the m rows with the smallest or_splitmix64(seed * 2^32 +
 *     row) (the SplitMix64 mixing function of Steele, Lea and Flood 2014), in
 *     increasing key order.
 * Return the number of probes, min(m, n). */
uint64_t or_splitmix64(uint64_t x);
int or_probe_uniform(int n, int m, int32_t* probes, double* w);
int or_probe_random(int n, int m, uint32_t seed, int32_t* probes, double* w);

/* Corrected rows (eq. probe_residual_estimate): out = x + mu_r + ((x-mu_x)/s_x) g. */
void or_correct_rows(const double* x, int n_rows, int dv, const double* mu_x, const double* s_x,
                     const double* mu_r, const double* g, double* out);

/* Whole plan for one head (Response-Coupled Partitioning, routing, probes).
 * Video rows are [n_text, n); the n_text leading text rows form one extra
 * query group (id cq) and one extra K/V group (id ck) that are routed
 * densely and excluded from clustering and probes.  Arrays sized with
 * cq_t = cq + (n_text > 0), ck_t = ck + (n_text > 0):
 *   labels_q, labels_kv: n;  z: cq_t x ck_t;  probes, w: m;
 *   fk: d x r_k;  fq: d x r_q;  phik: n_v x r_k;  phiq: n_v x r_q;
 *   kbar: ck x d;  qbar: cq x d;  cqphi: cq x r_q;  prio: cq x ck;
 *   stats[0] routed pairs, [1] forced pairs (incl. text), [2] routed cells,
 *   [3] forced cells, [4] probes, [5] k-means assignments (K/V),
 *   [6] k-means assignments (Q).
 * Any diagnostic pointer may be NULL.
 *
 * Grouped-query attention (Sec. 4.3: the K/V partition and routing metadata
 * are shared by the query heads of a K/V head; App. B.1: M_K per K/V head):
 * q holds the nqh query heads of one K/V head, one n x d block each, and the
 * plan pools them -- M_K is the mean of their metrics (or_key_metric_pooled),
 * phi_Q the mean of their normalised coordinates (or_project_pooled), and
 * the query-group means feeding the route scores the mean over heads and
 * members (or_group_mean_pooled).  nqh = 1 is the single-head plan.
 *
 * Ablation variants (Sec. 5.2): partition 0 = response-coupled, 1 = semantic
 * (k-means on the raw keys and on the raw queries, Sec. 3.1; r_k = r_q = d),
 * 2 = key-response K/V groups with semantic query groups (r_q = d);
 * probe_rule 0 = or_probe_select, 1 = or_probe_random(probe_seed),
 * 2 = or_probe_uniform. */
int or_plan(const float* q, int nqh, const float* k, int n, int d, int n_text, int m_s, int r_k,
            int r_q, int ck, int cq, int iters, double density, int m, int partition,
            int probe_rule, uint32_t probe_seed, int routing, int32_t* labels_q,
            int32_t* labels_kv, uint8_t* z, int32_t* probes, double* w, double* fk, double* fq,
            float* phik, float* phiq, float* kbar, float* qbar, float* cqphi, float* prio,
            int64_t* stats);

/* Pooled forms for grouped-query attention, over nqh query heads stored as
 * consecutive n x d blocks of x (nqh = 1 gives the single-head functions):
 *   M_K = (1/nqh) sum_h Q_s,h^T Q_s,h / M_s;
 *   phi_i = (1/nqh) sum_h F^T x_h,i / max(sqrt(|F^T x_h,i|^2 / r), eps)
 *     (eq. query_response_feature per head, then averaged; float output;
 *     rms = 0 leaves out the division);
 *   mean_b = sum_h sum_{j in b} x_h,j / (nqh |b|), 0 for an empty group. */
void or_key_metric_pooled(const float* q, int nqh, int n, int d, int m_s, double* mk);
void or_project_pooled(const float* x, int nqh, int n, int d, const double* f, int r, int rms,
                       double eps, float* phi);
void or_group_mean_pooled(const float* x, int nqh, int n, int d, const int32_t* labels, int c,
                          float* mean);

/* Whole attend for one head given a plan: sparse rows, exact probes, fit,
 * correction, output in original row order (Eq. final_reconstructed_output).
 * Text rows (the n_text leading rows) keep their (dense) sparse output.
 * out: n x dv (double).  fit_out (optional): 3*dv + dv*dv = mu_x, s_x, mu_r, g.
 * Returns the or_fit status. */
int or_attend(const float* q, const float* k, const float* v, int n, int d, int dv, int n_text,
              const int32_t* labels_q, const int32_t* labels_kv, int cq_t, int ck_t,
              const uint8_t* z, const int32_t* probes, const double* w, int m, int r,
              int ridge_only, double lambda, double eps, double* out, double* fit_out);

/* Diagnostics of Sec. 3.1 (observations O1 and O3); they need the dense
 * attention, so they exist on the oracle side only.
 *
 * or_support_sets: for each query row rows[t], the dense attention
 * probabilities over the n_k keys (double, scale 1/sqrt(d)) and D_i(alpha),
 * the smallest set of highest-weight keys (ties to the lower key index) whose
 * cumulative mass reaches alpha.  counts[t] = |D_i(alpha)| (tau_i = counts /
 * n_k); member (nrows x n_k bytes, zeroed by the caller, optional) marks the
 * keys of D_i, so the pooled support of a set of rows is the size of the
 * union of their marks. */
void or_support_sets(const float* q, const float* k, int n_k, int d, const int32_t* rows,
                     int nrows, double alpha, int32_t* counts, uint8_t* member);

/* or_affine_fraction (eq. projection_decomposition): X = [1, O_sp] (n x (dv+1)),
 * R the residual (n x dv).  out[0] = ||P_X R||_F^2 / ||R||_F^2, out[1] =
 * ||(I - P_X) R||_F^2, out[2] = ||R||_F^2.  Returns the rank used for X. */
int or_affine_fraction(const double* osp, const double* r, int n, int dv, double* out);

#ifdef __cplusplus
}
#endif
#endif
