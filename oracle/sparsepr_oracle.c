/*
 * SparsePR CPU oracle (test infrastructure only; see sparsepr_oracle.h).
 *
 * Plain loops, double accumulation, one head per call.  Written from the
 * paper's definitions: Sec. 3 (dense attention, pair density, hard drop),
 * Sec. 4.1 and App. B (Response-Coupled Partitioning), Sec. 4.2 and App. A
 * (Probe-Fitted Residual Reconstruction), Sec. 4.3 (sparse execution and
 * exact-pair accounting).  Readings of points the paper leaves open are
 * stated next to the code that takes them.
 */
#include "sparsepr_oracle.h"

#include <math.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

int or_num_threads(void) { return omp_get_max_threads(); }

/* ------------------------------------------------------------------------ */
/* Attention rows                                                            */
/* ------------------------------------------------------------------------ */

/* softmax(q k^T / sqrt(d)) V over the keys flagged in `use` (all when NULL).
 * Max-subtracted, double throughout. */
static void attend_row(const float* qi, const float* k, const float* v, int n_k, int d, int dv,
                       const unsigned char* use, double* logit, double* out) {
  const double scale = 1.0 / sqrt((double)d);
  double mx = -INFINITY;
  for (int j = 0; j < n_k; ++j) {
    if (use && !use[j]) continue;
    double s = 0.0;
    const float* kj = k + (size_t)j * d;
    for (int c = 0; c < d; ++c) s += (double)qi[c] * (double)kj[c];
    logit[j] = s * scale;
    if (logit[j] > mx) mx = logit[j];
  }
  for (int c = 0; c < dv; ++c) out[c] = 0.0;
  double z = 0.0;
  for (int j = 0; j < n_k; ++j) {
    if (use && !use[j]) continue;
    double p = exp(logit[j] - mx);
    z += p;
    const float* vj = v + (size_t)j * dv;
    for (int c = 0; c < dv; ++c) out[c] += p * (double)vj[c];
  }
  for (int c = 0; c < dv; ++c) out[c] /= z;
}

void or_dense_rows(const float* q, const float* k, const float* v, int n_k, int d, int dv,
                   const int64_t* rows, int n_rows, double* out) {
#pragma omp parallel
  {
    double* logit = (double*)malloc(sizeof(double) * (size_t)n_k);
#pragma omp for schedule(dynamic, 4)
    for (int r = 0; r < n_rows; ++r)
      attend_row(q + (size_t)rows[r] * d, k, v, n_k, d, dv, NULL, logit, out + (size_t)r * dv);
    free(logit);
  }
}

void or_sparse_rows(const float* q, const float* k, const float* v, int n_k, int d, int dv,
                    const int32_t* labels_q, const int32_t* labels_kv, int ck, const uint8_t* z,
                    const int64_t* rows, int n_rows, double* out) {
#pragma omp parallel
  {
    double* logit = (double*)malloc(sizeof(double) * (size_t)n_k);
    unsigned char* use = (unsigned char*)malloc((size_t)n_k);
#pragma omp for schedule(dynamic, 4)
    for (int r = 0; r < n_rows; ++r) {
      const int64_t i = rows[r];
      const int a = labels_q[i];
      /* Eq. hard_drop: every row of group a keeps exactly the keys of the
       * K/V groups routed to a, and renormalises over them. */
      for (int j = 0; j < n_k; ++j) use[j] = z[(size_t)a * ck + labels_kv[j]];
      attend_row(q + (size_t)i * d, k, v, n_k, d, dv, use, logit, out + (size_t)r * dv);
    }
    free(use);
    free(logit);
  }
}

/* ------------------------------------------------------------------------ */
/* Response coordinates (Sec. 4.1, App. B)                                   */
/* ------------------------------------------------------------------------ */

void or_key_metric(const float* q, int n, int d, int m_s, double* mk) {
  /* Reading: the "deterministic sample" of query rows is the strided one,
   * s_i = floor(i*n/m_s). */
  if (m_s > n) m_s = n;
  for (int a = 0; a < d * d; ++a) mk[a] = 0.0;
  for (int i = 0; i < m_s; ++i) {
    const float* qs = q + (size_t)(((int64_t)i * n) / m_s) * d;
    for (int a = 0; a < d; ++a)
      for (int b = 0; b < d; ++b) mk[a * d + b] += (double)qs[a] * (double)qs[b];
  }
  for (int a = 0; a < d * d; ++a) mk[a] /= (double)m_s;
}

int or_sym_eig(const double* a_in, int n, double* evals, double* evecs) {
  double* a = (double*)malloc(sizeof(double) * (size_t)n * n);
  memcpy(a, a_in, sizeof(double) * (size_t)n * n);
  for (int i = 0; i < n; ++i)
    for (int j = 0; j < n; ++j) evecs[i * n + j] = (i == j) ? 1.0 : 0.0;
  int sweep = 0;
  for (; sweep < 100; ++sweep) {
    double off = 0.0, tot = 0.0;
    for (int i = 0; i < n; ++i)
      for (int j = 0; j < n; ++j) {
        tot += a[i * n + j] * a[i * n + j];
        if (i != j) off += a[i * n + j] * a[i * n + j];
      }
    if (off <= 1e-30 * tot || off == 0.0) break;
    for (int p = 0; p < n - 1; ++p)
      for (int qq = p + 1; qq < n; ++qq) {
        const double apq = a[p * n + qq];
        if (apq == 0.0) continue;
        /* Rotation in the (p, q) plane that zeroes a_pq:
         * theta = (a_qq - a_pp) / (2 a_pq), t = sgn(theta)/(|theta| + sqrt(theta^2+1)). */
        const double theta = (a[qq * n + qq] - a[p * n + p]) / (2.0 * apq);
        const double t = (theta >= 0 ? 1.0 : -1.0) / (fabs(theta) + sqrt(theta * theta + 1.0));
        const double c = 1.0 / sqrt(t * t + 1.0), s = t * c;
        for (int i = 0; i < n; ++i) { /* columns p, q */
          const double aip = a[i * n + p], aiq = a[i * n + qq];
          a[i * n + p] = c * aip - s * aiq;
          a[i * n + qq] = s * aip + c * aiq;
        }
        for (int j = 0; j < n; ++j) { /* rows p, q */
          const double apj = a[p * n + j], aqj = a[qq * n + j];
          a[p * n + j] = c * apj - s * aqj;
          a[qq * n + j] = s * apj + c * aqj;
        }
        for (int i = 0; i < n; ++i) {
          const double vip = evecs[i * n + p], viq = evecs[i * n + qq];
          evecs[i * n + p] = c * vip - s * viq;
          evecs[i * n + qq] = s * vip + c * viq;
        }
      }
  }
  /* sort descending (selection sort, columns move with their values) */
  for (int i = 0; i < n; ++i) evals[i] = a[i * n + i];
  for (int i = 0; i < n; ++i) {
    int best = i;
    for (int j = i + 1; j < n; ++j)
      if (evals[j] > evals[best]) best = j;
    if (best != i) {
      double tmp = evals[i];
      evals[i] = evals[best];
      evals[best] = tmp;
      for (int r = 0; r < n; ++r) {
        tmp = evecs[r * n + i];
        evecs[r * n + i] = evecs[r * n + best];
        evecs[r * n + best] = tmp;
      }
    }
  }
  free(a);
  return sweep;
}

void or_response_basis(const double* m, int d, int r, double tau, double* f, double* evals_out) {
  double* ev = (double*)malloc(sizeof(double) * d);
  double* u = (double*)malloc(sizeof(double) * (size_t)d * d);
  or_sym_eig(m, d, ev, u);
  /* Reading: eigenvalues below tau * lambda_1 (including negative round-off)
   * are clamped to zero before the unit-mean normalisation, so null
   * directions get zero weight. */
  const double l1 = ev[0];
  for (int i = 0; i < d; ++i)
    if (!(ev[i] >= tau * l1) || l1 <= 0.0) ev[i] = 0.0;
  if (r > d) r = d;
  /* App. B.1 eq. app_key_response_coordinate (Sec. 3.2): divide the r kept
   * eigenvalues by their mean, then weight each kept eigenvector by the
   * square root of its normalised eigenvalue. */
  double mean = 0.0;
  for (int i = 0; i < r; ++i) mean += ev[i];
  mean /= (double)r;
  for (int row = 0; row < d; ++row)
    for (int i = 0; i < r; ++i)
      f[row * r + i] = (mean > 0.0) ? u[row * d + i] * sqrt(ev[i] / mean) : 0.0;
  if (evals_out)
    for (int i = 0; i < d; ++i) evals_out[i] = ev[i];
  free(ev);
  free(u);
}

void or_project(const float* x, int n, int d, const double* f, int r, int rms, double eps,
                float* phi) {
#pragma omp parallel for schedule(static)
  for (int i = 0; i < n; ++i) {
    double y[256];
    double ss = 0.0;
    for (int c = 0; c < r; ++c) {
      double s = 0.0;
      for (int a = 0; a < d; ++a) s += f[a * r + c] * (double)x[(size_t)i * d + a];
      y[c] = s;
      ss += s * s;
    }
    double den = 1.0;
    if (rms) { /* eq. query_response_feature: divide by max(RMS, eps) */
      den = sqrt(ss / (double)r);
      if (den < eps) den = eps;
    }
    for (int c = 0; c < r; ++c) phi[(size_t)i * r + c] = (float)(y[c] / den);
  }
}

/* ------------------------------------------------------------------------ */
/* k-means (Sec. 4.1: k-means on phi_K gives the paired K/V groups, on      */
/* phi_Q the query groups)                                                   */
/* ------------------------------------------------------------------------ */

void or_kmeans_assign(const float* pts, int n, int r, const float* cent, int c, int32_t* labels,
                      float* scores) {
  /* squared norms u_b, float fma chain in index order */
  float* u = (float*)malloc(sizeof(float) * c);
  float* ct = (float*)malloc(sizeof(float) * (size_t)c * r); /* ct[k*c + b] */
  for (int b = 0; b < c; ++b) {
    float acc = 0.0f;
    for (int k = 0; k < r; ++k) acc = fmaf(cent[(size_t)b * r + k], cent[(size_t)b * r + k], acc);
    u[b] = acc;
    for (int k = 0; k < r; ++k) ct[(size_t)k * c + b] = cent[(size_t)b * r + k];
  }
#pragma omp parallel
  {
    float* t = (float*)malloc(sizeof(float) * c);
#pragma omp for schedule(static)
    for (int j = 0; j < n; ++j) {
      const float* x = pts + (size_t)j * r;
      /* t_b = fmaf chain over k in index order; the loop over b only
       * interleaves independent chains, every single chain is unchanged. */
      for (int b = 0; b < c; ++b) t[b] = 0.0f;
      for (int k = 0; k < r; ++k) {
        const float xk = x[k];
        const float* row = ct + (size_t)k * c;
        for (int b = 0; b < c; ++b) t[b] = fmaf(xk, row[b], t[b]);
      }
      int best = 0;
      float bs = fmaf(-2.0f, t[0], u[0]);
      if (scores) scores[(size_t)j * c] = bs;
      for (int b = 1; b < c; ++b) {
        const float s = fmaf(-2.0f, t[b], u[b]);
        if (scores) scores[(size_t)j * c + b] = s;
        if (s < bs) { /* strict: ties keep the lowest index */
          bs = s;
          best = b;
        }
      }
      labels[j] = best;
    }
    free(t);
  }
  free(ct);
  free(u);
}

/* Lloyd iterations from the centroids already in `cent`. */
static int kmeans_iterate(const float* pts, int n, int r, int c, int iters, int32_t* labels,
                          float* cent, int32_t* counts) {
  int32_t* prev = (int32_t*)malloc(sizeof(int32_t) * n);
  double* sum = (double*)malloc(sizeof(double) * (size_t)c * r);
  int done = 0;
  for (int it = 0; it < iters; ++it) {
    or_kmeans_assign(pts, n, r, cent, c, labels, NULL);
    ++done;
    int changed = (it == 0);
    if (it > 0)
      for (int j = 0; j < n && !changed; ++j) changed = (labels[j] != prev[j]);
    memcpy(prev, labels, sizeof(int32_t) * n);
    /* update: double sums in ascending point index */
    memset(sum, 0, sizeof(double) * (size_t)c * r);
    for (int b = 0; b < c; ++b) counts[b] = 0;
    for (int j = 0; j < n; ++j) {
      const int b = labels[j];
      counts[b] += 1;
      for (int k = 0; k < r; ++k) sum[(size_t)b * r + k] += (double)pts[(size_t)j * r + k];
    }
    for (int b = 0; b < c; ++b)
      if (counts[b] > 0)
        for (int k = 0; k < r; ++k)
          cent[(size_t)b * r + k] = (float)(sum[(size_t)b * r + k] / (double)counts[b]);
    if (!changed) break; /* the next assignment would repeat this one */
  }
  free(sum);
  free(prev);
  return done;
}

int or_kmeans(const float* pts, int n, int r, int c, int iters, int32_t* labels, float* cent,
              int32_t* counts) {
  /* Reading: cold start from the strided points floor(b*n/c); a fixed number
   * of Lloyd iterations; empty groups keep their centroid. */
  for (int b = 0; b < c; ++b)
    memcpy(cent + (size_t)b * r, pts + (size_t)(((int64_t)b * n) / c) * r, sizeof(float) * r);
  return kmeans_iterate(pts, n, r, c, iters, labels, cent, counts);
}

int or_kmeans_from(const float* pts, int n, int r, int c, int iters, const float* init,
                   int32_t* labels, float* cent, int32_t* counts) {
  /* Warm start (App. C.1): the same iterations from given centroids. */
  memcpy(cent, init, sizeof(float) * (size_t)c * r);
  return kmeans_iterate(pts, n, r, c, iters, labels, cent, counts);
}

void or_group_mean(const float* x, int n, int d, const int32_t* labels, int c, float* mean,
                   int32_t* counts) {
  double* sum = (double*)calloc((size_t)c * d, sizeof(double));
  for (int b = 0; b < c; ++b) counts[b] = 0;
  for (int j = 0; j < n; ++j) {
    const int b = labels[j];
    counts[b] += 1;
    for (int a = 0; a < d; ++a) sum[(size_t)b * d + a] += (double)x[(size_t)j * d + a];
  }
  for (int b = 0; b < c; ++b)
    for (int a = 0; a < d; ++a)
      mean[(size_t)b * d + a] =
          counts[b] ? (float)(sum[(size_t)b * d + a] / (double)counts[b]) : 0.0f;
  free(sum);
}

void or_query_metric(const float* kbar, const int32_t* counts, int c, int d, double* mq) {
  /* App. B.2: nonempty groups only, equal weights, centred by their uniform
   * mean, normalised by C_k^+ d (the appendix's normaliser; it cancels in the
   * unit-mean eigenvalue scaling anyway). */
  int cp = 0;
  double* mu = (double*)calloc(d, sizeof(double));
  for (int b = 0; b < c; ++b)
    if (counts[b] > 0) {
      ++cp;
      for (int a = 0; a < d; ++a) mu[a] += (double)kbar[(size_t)b * d + a];
    }
  for (int a = 0; a < d * d; ++a) mq[a] = 0.0;
  if (cp == 0) {
    free(mu);
    return;
  }
  for (int a = 0; a < d; ++a) mu[a] /= (double)cp;
  for (int b = 0; b < c; ++b) {
    if (counts[b] == 0) continue;
    for (int a1 = 0; a1 < d; ++a1) {
      const double x1 = (double)kbar[(size_t)b * d + a1] - mu[a1];
      for (int a2 = 0; a2 < d; ++a2)
        mq[a1 * d + a2] += x1 * ((double)kbar[(size_t)b * d + a2] - mu[a2]);
    }
  }
  for (int a = 0; a < d * d; ++a) mq[a] /= (double)cp * (double)d;
  free(mu);
}

void or_stable_perm(const int32_t* labels, int n, int c, int32_t* perm, int32_t* off) {
  for (int b = 0; b <= c; ++b) off[b] = 0;
  for (int j = 0; j < n; ++j) off[labels[j] + 1] += 1;
  for (int b = 0; b < c; ++b) off[b + 1] += off[b];
  int32_t* fill = (int32_t*)malloc(sizeof(int32_t) * (c + 1));
  memcpy(fill, off, sizeof(int32_t) * (c + 1));
  for (int j = 0; j < n; ++j) perm[fill[labels[j]]++] = j;
  free(fill);
}

/* ------------------------------------------------------------------------ */
/* Routing under a pair budget (Sec. 4.3)                                    */
/* ------------------------------------------------------------------------ */

void or_route_priorities(const float* qbar, const int32_t* nq, int cq, const float* kbar,
                         const int32_t* nk, int ck, int d, float* prio) {
  /* Reading: the paper fixes the budget and the true cell cost but not the
   * score.  A cell is ranked by the centroid estimate of the attention
   * probability of one of its pairs: s_ab = qbar_a . kbar_b / sqrt(d) minus
   * the log of the size-weighted partition sum of row a. */
  const float scale = (float)(1.0 / sqrt((double)d));
  float* s = (float*)malloc(sizeof(float) * ck);
  for (int a = 0; a < cq; ++a) {
    for (int b = 0; b < ck; ++b) prio[(size_t)a * ck + b] = 0.0f;
    if (nq[a] == 0) continue;
    double mx = -INFINITY;
    for (int b = 0; b < ck; ++b) {
      if (nk[b] == 0) continue;
      float t = 0.0f;
      for (int c = 0; c < d; ++c) t = fmaf(qbar[(size_t)a * d + c], kbar[(size_t)b * d + c], t);
      s[b] = t * scale;
      if (s[b] > mx) mx = s[b];
    }
    double z = 0.0;
    for (int b = 0; b < ck; ++b)
      if (nk[b] > 0) z += (double)nk[b] * exp((double)s[b] - mx);
    const float lse = (float)(mx + log(z));
    for (int b = 0; b < ck; ++b)
      if (nk[b] > 0) prio[(size_t)a * ck + b] = s[b] - lse;
  }
  free(s);
}

typedef struct {
  float p;
  int64_t idx;
} cell_t;

static int cell_cmp(const void* x, const void* y) {
  const cell_t* a = (const cell_t*)x;
  const cell_t* b = (const cell_t*)y;
  if (a->p > b->p) return -1; /* priority descending */
  if (a->p < b->p) return 1;
  return (a->idx < b->idx) ? -1 : (a->idx > b->idx); /* flat index ascending */
}

void or_route_select(const float* prio, const int32_t* nq, int cq, const int32_t* nk, int ck,
                     int64_t budget, uint8_t* z, int64_t* out) {
  memset(z, 0, (size_t)cq * ck);
  int64_t forced_pairs = 0, forced_cells = 0;
  /* Reading: every nonempty query group keeps its best K/V group even when
   * that exceeds the budget, so every row has a nonempty support. */
  for (int a = 0; a < cq; ++a) {
    if (nq[a] == 0) continue;
    int best = -1;
    for (int b = 0; b < ck; ++b) {
      if (nk[b] == 0) continue;
      if (best < 0 || prio[(size_t)a * ck + b] > prio[(size_t)a * ck + best]) best = b;
    }
    if (best >= 0) {
      z[(size_t)a * ck + best] = 1;
      forced_pairs += (int64_t)nq[a] * nk[best];
      forced_cells += 1;
    }
  }
  cell_t* cells = (cell_t*)malloc(sizeof(cell_t) * (size_t)cq * ck);
  int64_t nc = 0;
  for (int a = 0; a < cq; ++a)
    for (int b = 0; b < ck; ++b)
      if (nq[a] > 0 && nk[b] > 0 && !z[(size_t)a * ck + b]) {
        cells[nc].p = prio[(size_t)a * ck + b];
        cells[nc].idx = (int64_t)a * ck + b;
        ++nc;
      }
  qsort(cells, (size_t)nc, sizeof(cell_t), cell_cmp);
  /* the longest prefix of that order that fits next to the forced cells */
  int64_t used = forced_pairs, taken = 0;
  for (int64_t t = 0; t < nc; ++t) {
    const int a = (int)(cells[t].idx / ck), b = (int)(cells[t].idx % ck);
    const int64_t cost = (int64_t)nq[a] * nk[b];
    if (used + cost > budget) break;
    used += cost;
    z[cells[t].idx] = 1;
    ++taken;
  }
  free(cells);
  out[0] = used;
  out[1] = forced_pairs;
  out[2] = taken + forced_cells;
  out[3] = forced_cells;
}

/* Per-group top-p routing with one p for every query group (the alternative
 * reading of the routing rule, Sec. 4.3).  Row a's estimated attention mass on
 * cell b is m_ab = nk_b exp(pi_ab); a group takes its cells in (pi descending,
 * b ascending) order until their mass reaches p.  So cell (a, b) is taken
 * exactly when the mass ranked before it, e_ab, is below p, and the largest p
 * that fits the budget takes the longest prefix of the cells ordered by e_ab
 * ascending: the walk of or_route_select on keys -e_ab (the best cell of each
 * group has e = 0 and stays the forced one). */
static const float* topp_prio_row;
static int topp_cmp(const void* x, const void* y) {
  const int a = *(const int*)x, b = *(const int*)y;
  const float pa = topp_prio_row[a], pb = topp_prio_row[b];
  if (pa > pb) return -1;
  if (pa < pb) return 1;
  return (a > b) - (a < b);
}

void or_route_topp_keys(const float* prio, const int32_t* nq, int cq, const int32_t* nk, int ck,
                        float* keys) {
  int* order = (int*)malloc(sizeof(int) * (ck > 0 ? ck : 1));
  for (int a = 0; a < cq; ++a) {
    float* out = keys + (size_t)a * ck;
    for (int b = 0; b < ck; ++b) out[b] = 0.0f;
    if (nq[a] == 0) continue;
    int cnt = 0;
    for (int b = 0; b < ck; ++b)
      if (nk[b] > 0) order[cnt++] = b;
    topp_prio_row = prio + (size_t)a * ck;
    qsort(order, (size_t)cnt, sizeof(int), topp_cmp);
    double e = 0.0;
    for (int t = 0; t < cnt; ++t) {
      const int b = order[t];
      out[b] = -(float)e;
      e += (double)nk[b] * exp((double)topp_prio_row[b]);
    }
  }
  free(order);
}

/* ------------------------------------------------------------------------ */
/* Probe selection (App. A.2)                                                */
/* ------------------------------------------------------------------------ */

typedef struct {
  float d2;
  int32_t row;
} rowkey_t;

static int rowkey_cmp(const void* x, const void* y) {
  const rowkey_t* a = (const rowkey_t*)x;
  const rowkey_t* b = (const rowkey_t*)y;
  if (a->d2 < b->d2) return -1;
  if (a->d2 > b->d2) return 1;
  return (a->row > b->row) - (a->row < b->row);
}

int or_probe_select(const float* phi, int n, int r, const int32_t* labels, int c,
                    const float* cent, int m, int32_t* probes, double* w) {
  int32_t* cnt = (int32_t*)calloc(c, sizeof(int32_t));
  int total = 0;
  for (int i = 0; i < n; ++i)
    if (labels[i] >= 0 && labels[i] < c) {
      cnt[labels[i]]++;
      ++total;
    }
  if (m > total) m = total;
  /* per-group orderings by (squared distance to the group mean, row);
   * ordering by the squared distance is ordering by the distance */
  int32_t* start = (int32_t*)calloc(c + 1, sizeof(int32_t));
  for (int b = 0; b < c; ++b) start[b + 1] = start[b] + cnt[b];
  rowkey_t* keys = (rowkey_t*)malloc(sizeof(rowkey_t) * (size_t)(total > 0 ? total : 1));
  int32_t* fill = (int32_t*)malloc(sizeof(int32_t) * (c + 1));
  memcpy(fill, start, sizeof(int32_t) * (c + 1));
  for (int i = 0; i < n; ++i) {
    const int b = labels[i];
    if (b < 0 || b >= c) continue;
    float acc = 0.0f;
    for (int k = 0; k < r; ++k) {
      const float diff = phi[(size_t)i * r + k] - cent[(size_t)b * r + k];
      acc = fmaf(diff, diff, acc);
    }
    keys[fill[b]].d2 = acc;
    keys[fill[b]].row = i;
    fill[b]++;
  }
  for (int b = 0; b < c; ++b)
    if (cnt[b] > 1) qsort(keys + start[b], (size_t)cnt[b], sizeof(rowkey_t), rowkey_cmp);
  /* deterministic group order over the nonempty groups */
  int g = 0;
  int32_t* ne = (int32_t*)malloc(sizeof(int32_t) * (c > 0 ? c : 1));
  for (int b = 0; b < c; ++b)
    if (cnt[b] > 0) ne[g++] = b;
  int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (g > 0 ? g : 1));
  if (g <= m || m == 0) {
    for (int t = 0; t < g; ++t) order[t] = ne[t];
  } else {
    /* Reading: with fewer probes than groups, a literal ascending order would
     * probe only the first groups; a stride-s interleave (s = ceil(G/m))
     * spreads one probe per group over the whole sequence instead. */
    const int s = (g + m - 1) / m;
    int t = 0;
    for (int res = 0; res < s; ++res)
      for (int rank = res; rank < g; rank += s) order[t++] = ne[rank];
  }
  /* round robin over the radial orderings */
  int taken = 0;
  int32_t* mcount = (int32_t*)calloc(c, sizeof(int32_t));
  int32_t* plabel = (int32_t*)malloc(sizeof(int32_t) * (m > 0 ? m : 1));
  for (int t = 0; taken < m; ++t) {
    for (int o = 0; o < g && taken < m; ++o) {
      const int b = order[o];
      if (t < cnt[b]) {
        probes[taken] = keys[start[b] + t].row;
        plabel[taken] = b;
        mcount[b]++;
        ++taken;
      }
    }
  }
  /* eq. app_probe_weight: w_p = |G_a| / m_a */
  for (int p = 0; p < taken; ++p) w[p] = (double)cnt[plabel[p]] / (double)mcount[plabel[p]];
  free(plabel);
  free(mcount);
  free(order);
  free(ne);
  free(fill);
  free(keys);
  free(start);
  free(cnt);
  return taken;
}

/* ------------------------------------------------------------------------ */
/* Probe-fitted residual reconstruction (Sec. 4.2, App. A.3)                 */
/* ------------------------------------------------------------------------ */

/* Cholesky a = L L^T in place (lower triangle); returns 0 or 1 if not PD. */
static int cholesky(double* a, int n) {
  for (int j = 0; j < n; ++j) {
    double s = a[j * n + j];
    for (int k = 0; k < j; ++k) s -= a[j * n + k] * a[j * n + k];
    if (!(s > 0.0)) return 1;
    const double l = sqrt(s);
    a[j * n + j] = l;
    for (int i = j + 1; i < n; ++i) {
      double t = a[i * n + j];
      for (int k = 0; k < j; ++k) t -= a[i * n + k] * a[j * n + k];
      a[i * n + j] = t / l;
    }
  }
  return 0;
}

/* Probe rules of the ablation (Table probe_estimator_ablation), equal
 * weights n_v / M.  Readings: "uniform spatiotemporal" = evenly spaced rows of
 * the raster token order, floor((2i + 1) n / (2m)); "random" = the m rows with
 * the smallest SplitMix64 keys (Steele, Lea and Flood 2014) of seed * 2^32 +
 * row, a uniformly random subset, in key order. */
uint64_t or_splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

int or_probe_uniform(int n, int m, int32_t* probes, double* w) {
  if (m > n) m = n;
  for (int i = 0; i < m; ++i) {
    probes[i] = (int32_t)(((int64_t)(2 * i + 1) * n) / (2 * (int64_t)m));
    w[i] = (double)(float)((float)n / (float)m);
  }
  return m;
}

typedef struct {
  uint64_t key;
  int32_t row;
} KeyRow;

static int keyrow_cmp(const void* a, const void* b) {
  const KeyRow* x = (const KeyRow*)a;
  const KeyRow* y = (const KeyRow*)b;
  if (x->key != y->key) return x->key < y->key ? -1 : 1;
  return x->row < y->row ? -1 : (x->row > y->row);
}

int or_probe_random(int n, int m, uint32_t seed, int32_t* probes, double* w) {
  if (m > n) m = n;
  KeyRow* kr = (KeyRow*)malloc(sizeof(KeyRow) * (size_t)(n > 0 ? n : 1));
  for (int i = 0; i < n; ++i) {
    kr[i].key = or_splitmix64(((uint64_t)seed << 32) | (uint32_t)i);
    kr[i].row = i;
  }
  qsort(kr, (size_t)n, sizeof(KeyRow), keyrow_cmp);
  for (int i = 0; i < m; ++i) {
    probes[i] = kr[i].row;
    w[i] = (double)(float)((float)n / (float)m);
  }
  free(kr);
  return m;
}

int or_fit(const double* x, const double* od, const double* w, int m, int dv, int r,
           int ridge_only, double lambda, double eps, double* mu_x, double* s_x, double* mu_r,
           double* b, double* psi, double* g, int* rank) {
  int status = 0;
  for (int c = 0; c < dv; ++c) mu_x[c] = s_x[c] = mu_r[c] = 0.0;
  memset(b, 0, sizeof(double) * (size_t)dv * dv);
  memset(g, 0, sizeof(double) * (size_t)dv * dv);
  memset(psi, 0, sizeof(double) * (size_t)dv * r);
  *rank = 0;
  if (m <= 0) {
    for (int c = 0; c < dv; ++c) s_x[c] = 1.0;
    return 0;
  }
  double sw = 0.0;
  for (int p = 0; p < m; ++p) sw += w[p];
  double* res = (double*)malloc(sizeof(double) * (size_t)m * dv); /* R_p = O_dense - O_sp */
  for (int p = 0; p < m; ++p)
    for (int c = 0; c < dv; ++c) res[p * dv + c] = od[p * dv + c] - x[p * dv + c];
  /* eq. app_normalized_weights and app_weighted_means */
  for (int p = 0; p < m; ++p) {
    const double al = w[p] / sw;
    for (int c = 0; c < dv; ++c) {
      mu_x[c] += al * x[p * dv + c];
      mu_r[c] += al * res[p * dv + c];
    }
  }
  /* eq. app_feature_scale */
  for (int p = 0; p < m; ++p) {
    const double al = w[p] / sw;
    for (int c = 0; c < dv; ++c) {
      const double t = x[p * dv + c] - mu_x[c];
      s_x[c] += al * t * t;
    }
  }
  for (int c = 0; c < dv; ++c) s_x[c] = sqrt(s_x[c] + eps);
  /* eq. app_standardized_probe_data and app_regression_weights */
  double* xb = (double*)malloc(sizeof(double) * (size_t)m * dv);
  double* rb = (double*)malloc(sizeof(double) * (size_t)m * dv);
  double* wt = (double*)malloc(sizeof(double) * m);
  for (int p = 0; p < m; ++p) {
    wt[p] = (double)m * w[p] / sw;
    for (int c = 0; c < dv; ++c) {
      xb[p * dv + c] = (x[p * dv + c] - mu_x[c]) / s_x[c];
      rb[p * dv + c] = res[p * dv + c] - mu_r[c];
    }
  }
  /* eq. app_ridge_closed_form, solved as a linear system (Cholesky) */
  double* s = (double*)calloc((size_t)dv * dv, sizeof(double));
  double* rhs = (double*)calloc((size_t)dv * dv, sizeof(double));
  for (int p = 0; p < m; ++p)
    for (int i = 0; i < dv; ++i) {
      const double a = wt[p] * xb[p * dv + i];
      for (int j = 0; j < dv; ++j) {
        s[i * dv + j] += a * xb[p * dv + j];
        rhs[i * dv + j] += a * rb[p * dv + j];
      }
    }
  for (int i = 0; i < dv; ++i) s[i * dv + i] += lambda;
  if (cholesky(s, dv) != 0) {
    status = 1;
  } else {
    for (int col = 0; col < dv; ++col) {
      double* y = (double*)malloc(sizeof(double) * dv);
      for (int i = 0; i < dv; ++i) { /* L y = rhs */
        double t = rhs[i * dv + col];
        for (int k = 0; k < i; ++k) t -= s[i * dv + k] * y[k];
        y[i] = t / s[i * dv + i];
      }
      for (int i = dv - 1; i >= 0; --i) { /* L^T b = y */
        double t = y[i];
        for (int k = i + 1; k < dv; ++k) t -= s[k * dv + i] * b[k * dv + col];
        b[i * dv + col] = t / s[i * dv + i];
      }
      free(y);
    }
  }
  if (ridge_only) {
    /* the ridge estimator alone (Table probe_estimator_ablation): Psi = I,
     * so the correction map is B_lambda itself (psi holds the first r
     * columns of I) */
    for (int i = 0; i < dv && i < r; ++i) psi[i * r + i] = 1.0;
    *rank = dv;
    if (status == 0) memcpy(g, b, sizeof(double) * (size_t)dv * dv);
    free(rhs);
    free(s);
    free(wt);
    free(rb);
    free(xb);
    free(res);
    return status;
  }
  /* eq. app_probe_residual_basis: right singular vectors of W^1/2 Rbar are
   * the eigenvectors of (W^1/2 Rbar)^T (W^1/2 Rbar); sigma = sqrt(eigenvalue).
   * Reading: directions with sigma <= 1e-6 sigma_1 are dropped. */
  double* h = (double*)calloc((size_t)dv * dv, sizeof(double));
  for (int p = 0; p < m; ++p)
    for (int i = 0; i < dv; ++i)
      for (int j = 0; j < dv; ++j) h[i * dv + j] += wt[p] * rb[p * dv + i] * rb[p * dv + j];
  double* ev = (double*)malloc(sizeof(double) * dv);
  double* u = (double*)malloc(sizeof(double) * (size_t)dv * dv);
  or_sym_eig(h, dv, ev, u);
  const double sig1 = ev[0] > 0.0 ? sqrt(ev[0]) : 0.0;
  int rk = 0;
  for (int i = 0; i < r && i < dv; ++i) {
    const double si = ev[i] > 0.0 ? sqrt(ev[i]) : 0.0;
    if (sig1 > 0.0 && si > 1e-6 * sig1) ++rk;
    else break;
  }
  for (int i = 0; i < dv; ++i)
    for (int t = 0; t < rk; ++t) psi[i * r + t] = u[i * dv + t];
  *rank = rk;
  /* g = b psi psi^T */
  if (status == 0) {
    double* bp = (double*)calloc((size_t)dv * (r > 0 ? r : 1), sizeof(double));
    for (int i = 0; i < dv; ++i)
      for (int t = 0; t < rk; ++t) {
        double acc = 0.0;
        for (int k = 0; k < dv; ++k) acc += b[i * dv + k] * psi[k * r + t];
        bp[i * r + t] = acc;
      }
    for (int i = 0; i < dv; ++i)
      for (int j = 0; j < dv; ++j) {
        double acc = 0.0;
        for (int t = 0; t < rk; ++t) acc += bp[i * r + t] * psi[j * r + t];
        g[i * dv + j] = acc;
      }
    free(bp);
  }
  free(u);
  free(ev);
  free(h);
  free(rhs);
  free(s);
  free(wt);
  free(rb);
  free(xb);
  free(res);
  return status;
}

void or_correct_rows(const double* x, int n_rows, int dv, const double* mu_x, const double* s_x,
                     const double* mu_r, const double* g, double* out) {
  /* eq. probe_residual_estimate: R_hat = mu_R + xbar G, added to the sparse
   * output; no norm cap. */
#pragma omp parallel for schedule(static)
  for (int i = 0; i < n_rows; ++i) {
    double xb[256];
    for (int c = 0; c < dv; ++c) xb[c] = (x[(size_t)i * dv + c] - mu_x[c]) / s_x[c];
    for (int c = 0; c < dv; ++c) {
      double acc = 0.0;
      for (int k = 0; k < dv; ++k) acc += xb[k] * g[k * dv + c];
      out[(size_t)i * dv + c] = x[(size_t)i * dv + c] + mu_r[c] + acc;
    }
  }
}

/* ------------------------------------------------------------------------ */
/* Whole call                                                                */
/* ------------------------------------------------------------------------ */

/* Grouped-query pooling (Sec. 4.3 shares the K/V partition and routes
 * across a K/V head's query heads; App. B.1 builds M_K per K/V head).  The
 * readings: the metric, the query coordinates and the query-group means are
 * the plain means over the nqh query heads. */
void or_key_metric_pooled(const float* q, int nqh, int n, int d, int m_s, double* mk) {
  double* one = (double*)malloc(sizeof(double) * (size_t)d * d);
  for (int a = 0; a < d * d; ++a) mk[a] = 0.0;
  for (int h = 0; h < nqh; ++h) {
    or_key_metric(q + (size_t)h * n * d, n, d, m_s, one);
    for (int a = 0; a < d * d; ++a) mk[a] += one[a];
  }
  for (int a = 0; a < d * d; ++a) mk[a] /= (double)nqh;
  free(one);
}

void or_project_pooled(const float* x, int nqh, int n, int d, const double* f, int r, int rms,
                       double eps, float* phi) {
#pragma omp parallel for schedule(static)
  for (int i = 0; i < n; ++i) {
    double acc[256];
    for (int c = 0; c < r; ++c) acc[c] = 0.0;
    for (int h = 0; h < nqh; ++h) {
      const float* xi = x + ((size_t)h * n + i) * d;
      double y[256];
      double ss = 0.0;
      for (int c = 0; c < r; ++c) {
        double s = 0.0;
        for (int a = 0; a < d; ++a) s += f[a * r + c] * (double)xi[a];
        y[c] = s;
        ss += s * s;
      }
      double den = 1.0;
      if (rms) { /* eq. query_response_feature */
        den = sqrt(ss / (double)r);
        if (den < eps) den = eps;
      }
      for (int c = 0; c < r; ++c) acc[c] += y[c] / den;
    }
    for (int c = 0; c < r; ++c) phi[(size_t)i * r + c] = (float)(acc[c] / (double)nqh);
  }
}

void or_group_mean_pooled(const float* x, int nqh, int n, int d, const int32_t* labels, int c,
                          float* mean) {
  double* sum = (double*)calloc((size_t)c * d, sizeof(double));
  int64_t* cnt = (int64_t*)calloc((size_t)c, sizeof(int64_t));
  for (int h = 0; h < nqh; ++h)
    for (int j = 0; j < n; ++j) {
      const int b = labels[j];
      cnt[b] += 1;
      for (int a = 0; a < d; ++a) sum[(size_t)b * d + a] += (double)x[((size_t)h * n + j) * d + a];
    }
  for (int b = 0; b < c; ++b)
    for (int a = 0; a < d; ++a)
      mean[(size_t)b * d + a] = cnt[b] ? (float)(sum[(size_t)b * d + a] / (double)cnt[b]) : 0.0f;
  free(cnt);
  free(sum);
}

int or_plan(const float* q, int nqh, const float* k, int n, int d, int n_text, int m_s, int r_k,
            int r_q, int ck, int cq, int iters, double density, int m, int partition,
            int probe_rule, uint32_t probe_seed, int routing, int32_t* labels_q,
            int32_t* labels_kv, uint8_t* z, int32_t* probes, double* w, double* fk_out,
            double* fq_out, float* phik_out, float* phiq_out, float* kbar_out, float* qbar_out,
            float* cqphi_out, float* prio_out, int64_t* stats) {
  const int nv = n - n_text;
  const float* kv = k + (size_t)n_text * d;
  /* the video rows of every query head, one nv x d block each */
  float* qv = (float*)malloc(sizeof(float) * (size_t)nqh * nv * d);
  for (int h = 0; h < nqh; ++h)
    memcpy(qv + (size_t)h * nv * d, q + ((size_t)h * n + n_text) * d, sizeof(float) * (size_t)nv * d);
  if (r_k > d) r_k = d;
  if (r_q > d) r_q = d;
  /* the semantic partitions cluster the raw rows (Sec. 3.1, Sec. 5.2) */
  if (partition == 1) r_k = d;
  if (partition != 0) r_q = d;
  const int cq_t = cq + (n_text > 0), ck_t = ck + (n_text > 0);
  const double tau = 1e-6;

  /* Key-response coordinates and paired K/V groups (Sec. 4.1, App. B.1) */
  double* mk = (double*)malloc(sizeof(double) * (size_t)d * d);
  double* fk = (double*)malloc(sizeof(double) * (size_t)d * r_k);
  float* phik = (float*)malloc(sizeof(float) * (size_t)nv * r_k);
  float* centk = (float*)malloc(sizeof(float) * (size_t)ck * r_k);
  int32_t* labk = (int32_t*)malloc(sizeof(int32_t) * nv);
  int32_t* cntk = (int32_t*)malloc(sizeof(int32_t) * ck);
  if (partition == 1) { /* semantic K/V groups: phi_K = k */
    memset(mk, 0, sizeof(double) * (size_t)d * d);
    for (int a = 0; a < d * d; ++a) fk[a] = (a / d == a % d) ? 1.0 : 0.0;
  } else {
    or_key_metric_pooled(qv, nqh, nv, d, m_s, mk);
    or_response_basis(mk, d, r_k, tau, fk, NULL);
  }
  or_project(kv, nv, d, fk, r_k, 0, 0.0, phik);
  const int itk = or_kmeans(phik, nv, r_k, ck, iters, labk, centk, cntk);

  /* Query-response coordinates from the K/V groups (App. B.2) */
  float* kbar = (float*)malloc(sizeof(float) * (size_t)ck * d);
  double* mq = (double*)malloc(sizeof(double) * (size_t)d * d);
  double* fq = (double*)malloc(sizeof(double) * (size_t)d * r_q);
  float* phiq = (float*)malloc(sizeof(float) * (size_t)nv * r_q);
  float* centq = (float*)malloc(sizeof(float) * (size_t)cq * r_q);
  int32_t* labq = (int32_t*)malloc(sizeof(int32_t) * nv);
  int32_t* cntq = (int32_t*)malloc(sizeof(int32_t) * cq);
  int32_t* cnt_dummy = (int32_t*)malloc(sizeof(int32_t) * ck);
  or_group_mean(kv, nv, d, labk, ck, kbar, cnt_dummy);
  if (partition == 0) {
    or_query_metric(kbar, cntk, ck, d, mq);
    or_response_basis(mq, d, r_q, tau, fq, NULL);
    or_project_pooled(qv, nqh, nv, d, fq, r_q, 1, 1e-6, phiq);
  } else { /* semantic query groups: phi_Q = q (pooled over the query heads) */
    memset(mq, 0, sizeof(double) * (size_t)d * d);
    for (int a = 0; a < d * d; ++a) fq[a] = (a / d == a % d) ? 1.0 : 0.0;
    or_project_pooled(qv, nqh, nv, d, fq, r_q, 0, 0.0, phiq);
  }
  const int itq = or_kmeans(phiq, nv, r_q, cq, iters, labq, centq, cntq);

  /* Routing (Sec. 4.3) */
  float* qbar = (float*)malloc(sizeof(float) * (size_t)cq * d);
  int32_t* cntq2 = (int32_t*)malloc(sizeof(int32_t) * cq);
  float* prio = (float*)malloc(sizeof(float) * (size_t)cq * ck);
  uint8_t* zv = (uint8_t*)malloc((size_t)cq * ck);
  or_group_mean_pooled(qv, nqh, nv, d, labq, cq, qbar);
  (void)cntq2;
  or_route_priorities(qbar, cntq, cq, kbar, cntk, ck, d, prio);
  const int meff = m < nv ? m : nv;
  /* the probe rows' cost against all keys is reserved first */
  const int64_t budget = (int64_t)floor(density * (double)nv * (double)nv) - (int64_t)meff * n;
  int64_t rs[4];
  if (routing == 1) {
    float* keys = (float*)malloc(sizeof(float) * (size_t)cq * ck);
    or_route_topp_keys(prio, cntq, cq, cntk, ck, keys);
    or_route_select(keys, cntq, cq, cntk, ck, budget, zv, rs);
    free(keys);
  } else {
    or_route_select(prio, cntq, cq, cntk, ck, budget, zv, rs);
  }

  /* Probes (App. A.2) */
  int np;
  if (probe_rule == 1)
    np = or_probe_random(nv, m, probe_seed, probes, w);
  else if (probe_rule == 2)
    np = or_probe_uniform(nv, m, probes, w);
  else
    np = or_probe_select(phiq, nv, r_q, labq, cq, centq, m, probes, w);
  for (int p = 0; p < np; ++p) probes[p] += n_text;

  /* Assemble labels and the full route matrix.  Reading for text tokens:
   * they form one extra query group and one extra K/V group, routed densely
   * and outside the budget. */
  for (int i = 0; i < n_text; ++i) {
    labels_q[i] = cq;
    labels_kv[i] = ck;
  }
  for (int i = 0; i < nv; ++i) {
    labels_q[n_text + i] = labq[i];
    labels_kv[n_text + i] = labk[i];
  }
  memset(z, 0, (size_t)cq_t * ck_t);
  for (int a = 0; a < cq; ++a)
    for (int b = 0; b < ck; ++b) z[(size_t)a * ck_t + b] = zv[(size_t)a * ck + b];
  int64_t text_pairs = 0;
  if (n_text > 0) {
    for (int a = 0; a < cq_t; ++a) z[(size_t)a * ck_t + ck] = 1;
    for (int b = 0; b < ck_t; ++b) z[(size_t)cq * ck_t + b] = 1;
    text_pairs = (int64_t)n_text * n + (int64_t)nv * n_text;
  }
  if (stats) {
    stats[0] = rs[0] + text_pairs;
    stats[1] = rs[1] + text_pairs;
    stats[2] = rs[2];
    stats[3] = rs[3];
    stats[4] = np;
    stats[5] = itk;
    stats[6] = itq;
  }
  if (fk_out) memcpy(fk_out, fk, sizeof(double) * (size_t)d * r_k);
  if (fq_out) memcpy(fq_out, fq, sizeof(double) * (size_t)d * r_q);
  if (phik_out) memcpy(phik_out, phik, sizeof(float) * (size_t)nv * r_k);
  if (phiq_out) memcpy(phiq_out, phiq, sizeof(float) * (size_t)nv * r_q);
  if (kbar_out) memcpy(kbar_out, kbar, sizeof(float) * (size_t)ck * d);
  if (qbar_out) memcpy(qbar_out, qbar, sizeof(float) * (size_t)cq * d);
  if (cqphi_out) memcpy(cqphi_out, centq, sizeof(float) * (size_t)cq * r_q);
  if (prio_out) memcpy(prio_out, prio, sizeof(float) * (size_t)cq * ck);
  free(zv);
  free(prio);
  free(cntq2);
  free(qbar);
  free(cnt_dummy);
  free(cntq);
  free(labq);
  free(centq);
  free(phiq);
  free(fq);
  free(mq);
  free(kbar);
  free(cntk);
  free(labk);
  free(centk);
  free(phik);
  free(fk);
  free(mk);
  free(qv);
  return 0;
}

int or_attend(const float* q, const float* k, const float* v, int n, int d, int dv, int n_text,
              const int32_t* labels_q, const int32_t* labels_kv, int cq_t, int ck_t,
              const uint8_t* z, const int32_t* probes, const double* w, int m, int r,
              int ridge_only, double lambda, double eps, double* out, double* fit_out) {
  (void)cq_t;
  int64_t* rows = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
  for (int i = 0; i < n; ++i) rows[i] = i;
  double* osp = (double*)malloc(sizeof(double) * (size_t)n * dv);
  or_sparse_rows(q, k, v, n, d, dv, labels_q, labels_kv, ck_t, z, rows, n, osp);
  /* exact probe rows against all keys */
  double* x = (double*)malloc(sizeof(double) * (size_t)(m > 0 ? m : 1) * dv);
  double* od = (double*)malloc(sizeof(double) * (size_t)(m > 0 ? m : 1) * dv);
  int64_t* prow = (int64_t*)malloc(sizeof(int64_t) * (m > 0 ? m : 1));
  for (int p = 0; p < m; ++p) {
    prow[p] = probes[p];
    memcpy(x + (size_t)p * dv, osp + (size_t)probes[p] * dv, sizeof(double) * dv);
  }
  or_dense_rows(q, k, v, n, d, dv, prow, m, od);
  double* mu_x = (double*)malloc(sizeof(double) * dv);
  double* s_x = (double*)malloc(sizeof(double) * dv);
  double* mu_r = (double*)malloc(sizeof(double) * dv);
  double* b = (double*)malloc(sizeof(double) * (size_t)dv * dv);
  double* g = (double*)malloc(sizeof(double) * (size_t)dv * dv);
  double* psi = (double*)malloc(sizeof(double) * (size_t)dv * (r > 0 ? r : 1));
  int rank = 0;
  const int st =
      or_fit(x, od, w, m, dv, r, ridge_only, lambda, eps, mu_x, s_x, mu_r, b, psi, g, &rank);
  /* eq. final_reconstructed_output; text rows are exact already */
  const int nv = n - n_text;
  if (m > 0) {
    or_correct_rows(osp + (size_t)n_text * dv, nv, dv, mu_x, s_x, mu_r, g,
                    out + (size_t)n_text * dv);
  } else {
    memcpy(out + (size_t)n_text * dv, osp + (size_t)n_text * dv, sizeof(double) * (size_t)nv * dv);
  }
  memcpy(out, osp, sizeof(double) * (size_t)n_text * dv);
  for (int p = 0; p < m; ++p)
    memcpy(out + (size_t)probes[p] * dv, od + (size_t)p * dv, sizeof(double) * dv);
  if (fit_out) {
    memcpy(fit_out, mu_x, sizeof(double) * dv);
    memcpy(fit_out + dv, s_x, sizeof(double) * dv);
    memcpy(fit_out + 2 * dv, mu_r, sizeof(double) * dv);
    memcpy(fit_out + 3 * dv, g, sizeof(double) * (size_t)dv * dv);
  }
  free(psi);
  free(g);
  free(b);
  free(mu_r);
  free(s_x);
  free(mu_x);
  free(prow);
  free(od);
  free(x);
  free(osp);
  free(rows);
  return st;
}

/* ------------------------------------------------------------------------ */
/* Diagnostics of Sec. 3.1 (oracle side only: they need the dense attention) */
/* ------------------------------------------------------------------------ */

typedef struct {
  double p;
  int32_t j;
} pk_t;

static int pk_cmp(const void* x, const void* y) {
  const pk_t* a = (const pk_t*)x;
  const pk_t* b = (const pk_t*)y;
  if (a->p > b->p) return -1; /* weight descending */
  if (a->p < b->p) return 1;
  return (a->j > b->j) - (a->j < b->j); /* then key index ascending */
}

void or_support_sets(const float* q, const float* k, int n_k, int d, const int32_t* rows,
                     int nrows, double alpha, int32_t* counts, uint8_t* member) {
  /* Observation O1: D_i(alpha) is the smallest set of highest-weight keys
   * whose dense attention mass for query i reaches alpha. */
  const double scale = 1.0 / sqrt((double)d);
#pragma omp parallel for schedule(dynamic, 1)
  for (int t = 0; t < nrows; ++t) {
    const float* qi = q + (size_t)rows[t] * d;
    pk_t* a = (pk_t*)malloc(sizeof(pk_t) * (size_t)n_k);
    double mx = -INFINITY;
    for (int j = 0; j < n_k; ++j) {
      double s = 0.0;
      for (int c = 0; c < d; ++c) s += (double)qi[c] * (double)k[(size_t)j * d + c];
      a[j].p = s * scale;
      a[j].j = j;
      if (a[j].p > mx) mx = a[j].p;
    }
    double z = 0.0;
    for (int j = 0; j < n_k; ++j) {
      a[j].p = exp(a[j].p - mx);
      z += a[j].p;
    }
    for (int j = 0; j < n_k; ++j) a[j].p /= z;
    qsort(a, (size_t)n_k, sizeof(pk_t), pk_cmp);
    double cum = 0.0;
    int cnt = 0;
    while (cnt < n_k && cum < alpha) {
      cum += a[cnt].p;
      if (member) member[(size_t)t * n_k + a[cnt].j] = 1;
      ++cnt;
    }
    counts[t] = cnt;
    free(a);
  }
}

int or_affine_fraction(const double* osp, const double* r, int n, int dv, double* out) {
  /* Observation O3: with X = [1, O_sp], the residual splits into P_X R (the
   * best least-squares affine function of the sparse output) and
   * (I - P_X) R.  ||P_X R||_F^2 = tr(C^T G^+ C) with G = X^T X and
   * C = X^T R, through the eigenvectors of G (eigenvalues below 1e-12 of the
   * largest count as zero, so a rank-deficient X is handled). */
  const int p = dv + 1;
  double* g = (double*)calloc((size_t)p * p, sizeof(double));
  double* c = (double*)calloc((size_t)p * dv, sizeof(double));
  double* x = (double*)malloc(sizeof(double) * p);
  double rr = 0.0;
  for (int i = 0; i < n; ++i) {
    x[0] = 1.0;
    for (int a = 0; a < dv; ++a) x[a + 1] = osp[(size_t)i * dv + a];
    const double* ri = r + (size_t)i * dv;
    for (int a = 0; a < p; ++a) {
      for (int b = 0; b < p; ++b) g[(size_t)a * p + b] += x[a] * x[b];
      for (int b = 0; b < dv; ++b) c[(size_t)a * dv + b] += x[a] * ri[b];
    }
    for (int b = 0; b < dv; ++b) rr += ri[b] * ri[b];
  }
  double* ev = (double*)malloc(sizeof(double) * p);
  double* u = (double*)malloc(sizeof(double) * (size_t)p * p);
  or_sym_eig(g, p, ev, u);
  double e = 0.0;
  int rank = 0;
  for (int kk = 0; kk < p; ++kk) {
    if (!(ev[kk] > 1e-12 * ev[0])) continue;
    ++rank;
    for (int b = 0; b < dv; ++b) {
      double t = 0.0;
      for (int a = 0; a < p; ++a) t += u[(size_t)a * p + kk] * c[(size_t)a * dv + b];
      e += t * t / ev[kk];
    }
  }
  out[0] = rr > 0.0 ? e / rr : 0.0; /* affine-explainable fraction */
  out[1] = rr - e;                  /* affine-orthogonal energy */
  out[2] = rr;                      /* residual energy */
  free(u);
  free(ev);
  free(x);
  free(c);
  free(g);
  return rank;
}
