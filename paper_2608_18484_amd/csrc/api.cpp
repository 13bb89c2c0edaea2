// C ABI of the SparsePR library (declared in include/sparsepr.h): argument
// validation, device-workspace layout, the plan handle and host<->device
// transfers for export/import.  All device work is enqueued on the caller's
// stream; nothing here allocates device memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/sparsepr.h"
#include "sparsepr_internal.hpp"

using namespace sparsepr;

namespace {

thread_local std::string g_last_error;

sparsepr_status fail(sparsepr_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

sparsepr_status ok() {
  g_last_error.clear();
  return SPARSEPR_OK;
}

sparsepr_status hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return SPARSEPR_OK;
  (void)hipGetLastError();  // do not leave the error behind for the caller's next HIP call
  return fail(SPARSEPR_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

std::string ptrs(const void* dst, const void* src, size_t n) {
  char buf[128];
  snprintf(buf, sizeof buf, " (dst %p, src %p, %zu bytes)", dst, src, n);
  return buf;
}

// Per-head byte sizes of every workspace array, in layout order.  Plan
// arrays are [BH][...] (one per K/V head); the attend outputs are
// [G][BH][...] (one per query head, query head j < G of every K/V head
// forming slab j, so that the view of slab j is again [BH][...]).
struct Layout {
  struct Item {
    size_t field;     // byte offset of the pointer member inside Work
    size_t per_head;  // bytes per head
    bool per_query;   // one per query head instead of per K/V head
  };
  std::vector<Item> items;
  size_t total = 0;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

void describe(const Geom& g, Work* w, Layout& L) {
  const size_t d = g.d, dv = g.dv, N = g.N, NV = g.NV, M = std::max(g.M, 1), r = g.r;
  auto add = [&](void* field, size_t bytes) {
    L.items.push_back({(size_t)((char*)field - (char*)w), bytes, false});
  };
  auto addq = [&](void* field, size_t bytes) {
    L.items.push_back({(size_t)((char*)field - (char*)w), bytes, true});
  };
  add(&w->gram_k, d * d * 8);
  add(&w->gram_q, d * d * 8);
  add(&w->evals_k, d * 4);
  add(&w->evals_q, d * 4);
  add(&w->fk, d * g.rk * 4);
  add(&w->fq, d * g.rq * 4);
  add(&w->phik, NV * g.rk * 4);
  add(&w->phiq, NV * g.rq * 4);
  add(&w->centk, (size_t)g.CK * g.rk * 4);
  add(&w->centq, (size_t)g.CQ * g.rq * 4);
  add(&w->labk, N * 4);
  add(&w->labq, N * 4);
  add(&w->permk, N * 4);
  add(&w->permq, N * 4);
  add(&w->offk, (size_t)(g.CKt + 1) * 4);
  add(&w->offq, (size_t)(g.CQt + 1) * 4);
  add(&w->blkhist, (size_t)g.nsort_blk_full * g.cmax * 4);
  add(&w->kmstate, (size_t)2 * (g.T + 1) * 4);
  add(&w->km_xhi, NV * g.rpad * 2);
  add(&w->km_xlo, NV * g.rpad * 2);
  add(&w->km_xn, NV * 4);
  add(&w->km_chi, (size_t)g.cpad * g.rpad * 2);
  add(&w->km_clo, (size_t)g.cpad * g.rpad * 2);
  add(&w->km_cu, (size_t)g.cpad * 4);
  add(&w->km_cn3, (size_t)g.cpad * 2 * 4);
  add(&w->km_fbcnt, (size_t)2 * g.T * 4);
  add(&w->kbar, (size_t)g.CK * d * 4);
  add(&w->qbar, (size_t)g.CQ * d * 4);
  add(&w->prio, (size_t)g.CQ * g.CK * 4);
  add(&w->skey, g.routing == SPARSEPR_ROUTING_TOP_P ? (size_t)g.CQ * g.CK * 4 : 0);
  add(&w->forced, (size_t)g.CQ * 4);
  add(&w->selhist, (size_t)kSelPasses * kSelBins * 8);
  add(&w->selstate, 8 * 8);
  add(&w->z, (size_t)g.CQt * g.CKt);
  add(&w->rng_cnt, (size_t)g.CQt * 4);
  add(&w->rng, (size_t)g.CQt * g.CKt * 8);
  add(&w->keytot, (size_t)g.CQt * 4);
  add(&w->chunks, (size_t)g.nchunk_max * 16);
  add(&w->nchunks, 4);
  add(&w->d2, NV * 4);
  add(&w->probes, M * 4);
  add(&w->pw, M * 4);
  add(&w->nprobes, 4);
  add(&w->picks, M * 4);
  add(&w->kperm, g.bf16 ? N * d * 2 : 0);
  add(&w->vperm, g.bf16 ? N * dv * 2 : 0);
  addq(&w->osp, N * dv * 4);
  addq(&w->odp, M * dv * 4);
  addq(&w->part, M * g.nsplit * (dv + 2) * 4);
  addq(&w->mlst, N * 4 * 4);
  addq(&w->fitv, 3 * dv * 4);
  addq(&w->fity, dv * r * 4);
  addq(&w->fitpsi, dv * r * 4);
  addq(&w->fitscr, (2 * M * dv + M * r + dv * r + M) * 8);
  addq(&w->fitgram, 2 * dv * dv * 8);
  addq(&w->fitvec, (!g.bf16 && dv > 64) ? dv * (dv + 4) * 8 : 0);
  addq(&w->eigscr, 4 * std::max(d, dv) * std::max(d, dv) * 8);
  add(&w->stats, 16 * 8);
  size_t off = 0;
  for (auto& it : L.items) off += align256((size_t)g.BH * it.per_head * (it.per_query ? g.G : 1));
  L.total = off;
}

// Bind the layout to a base address: whole-batch view, or the view of a
// single K/V head (bh >= 0) in which that head appears as head 0; the attend
// outputs are those of query head j of each K/V head's group.
void bind(const Geom& g, Work* w, const Layout& L, char* base, int bh, int j = 0) {
  size_t off = 0;
  for (auto& it : L.items) {
    const size_t head = bh >= 0 ? (size_t)bh : 0;
    const size_t idx = it.per_query ? (size_t)j * g.BH + head : (bh >= 0 ? head : 0);
    char* ptr = base + off + idx * it.per_head;
    std::memcpy((char*)w + it.field, &ptr, sizeof ptr);  // every Work member is a pointer
    off += align256((size_t)g.BH * it.per_head * (it.per_query ? g.G : 1));
  }
}

sparsepr_status validate(const sparsepr_shape* s, const sparsepr_params* p, Geom& g) {
  if (!s || !p) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "shape and params must not be NULL");
  if (s->batch < 1 || s->heads < 1) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "batch and heads must be >= 1");
  if (s->n_q < 1 || s->n_kv < 1) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "n_q and n_kv must be >= 1");
  if (s->n_q != s->n_kv) return fail(SPARSEPR_ERR_UNSUPPORTED, "only self-attention (n_q == n_kv) is supported");
  if (s->n_q > (1 << 24)) return fail(SPARSEPR_ERR_UNSUPPORTED, "n_q above 2^24 is not supported");
  if (s->d != s->d_v) return fail(SPARSEPR_ERR_UNSUPPORTED, "d must equal d_v");
  if (s->d != 64 && s->d != 128) return fail(SPARSEPR_ERR_UNSUPPORTED, "d must be 64 or 128");
  if (s->dtype != SPARSEPR_F32 && s->dtype != SPARSEPR_BF16)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "dtype must be SPARSEPR_F32 or SPARSEPR_BF16");
  if (s->stride_n < s->d || s->stride_h < 0 || s->stride_b < 0)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "strides must be non-negative and stride_n >= d");
  if (s->stride_n % 8 != 0 || s->stride_h % 8 != 0 || s->stride_b % 8 != 0)
    return fail(SPARSEPR_ERR_UNSUPPORTED, "strides must be multiples of 8 elements");
  // grouped-query attention: heads_kv K/V heads, each shared by heads / heads_kv
  // consecutive query heads
  const int hkv = s->heads_kv > 0 ? s->heads_kv : s->heads;
  if (s->heads_kv < 0 || s->heads % hkv != 0)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "heads_kv must be 0 or a divisor of heads");
  int64_t kvsb = s->kv_stride_b, kvsh = s->kv_stride_h;
  if (hkv == s->heads) {
    if (kvsb == 0) kvsb = s->stride_b;
    if (kvsh == 0) kvsh = s->stride_h;
  } else if (kvsb <= 0 || kvsh <= 0) {
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "kv_stride_b and kv_stride_h are required when heads_kv < heads");
  }
  if (kvsb < 0 || kvsh < 0)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "kv strides must be non-negative");
  if (kvsb % 8 != 0 || kvsh % 8 != 0)
    return fail(SPARSEPR_ERR_UNSUPPORTED, "strides must be multiples of 8 elements");
  // the attention kernels address one head's K/V rows with 32-bit byte offsets
  if ((int64_t)s->n_kv * s->stride_n * (s->dtype == SPARSEPR_BF16 ? 2 : 4) >= (int64_t(1) << 32))
    return fail(SPARSEPR_ERR_UNSUPPORTED, "n_kv * stride_n must stay below 4 GiB per head");
  const int N = s->n_q;
  if (p->n_dense_prefix < 0 || p->n_dense_prefix >= N)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "n_dense_prefix must be in [0, n_q)");
  const int NV = N - p->n_dense_prefix;
  const int CK = p->n_kv_groups > 0 ? p->n_kv_groups : (NV + 63) / 64;
  const int CQ = p->n_q_groups > 0 ? p->n_q_groups : (NV + 63) / 64;
  if (p->n_kv_groups < 0 || p->n_q_groups < 0 || CK > NV || CQ > NV)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "group counts must be in [1, n_q - n_dense_prefix]");
  if (CK > 8191 || CQ > 8191) return fail(SPARSEPR_ERR_UNSUPPORTED, "more than 8191 groups");
  if (p->r_k < 1 || p->r_q < 1) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "r_k and r_q must be >= 1");
  if (p->n_sampled_queries < 1) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "n_sampled_queries must be >= 1");
  if (p->kmeans_iters < 1 || p->kmeans_iters > 1000)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "kmeans_iters must be in [1, 1000]");
  if (p->n_probes < 0) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "n_probes must be >= 0");
  if (p->warm_start != 0 && p->warm_start != 1)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "warm_start must be 0 or 1");
  if (p->warm_iters < 0 || p->warm_iters > p->kmeans_iters)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "warm_iters must be in [0, kmeans_iters]");
  if (p->partition < SPARSEPR_PARTITION_RESPONSE || p->partition > SPARSEPR_PARTITION_KEY_RESPONSE)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "partition must be one of SPARSEPR_PARTITION_*");
  if (p->probe_rule < SPARSEPR_PROBES_STRATIFIED || p->probe_rule > SPARSEPR_PROBES_UNIFORM)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "probe_rule must be one of SPARSEPR_PROBES_*");
  if (p->ridge_only != 0 && p->ridge_only != 1)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "ridge_only must be 0 or 1");
  if (p->routing != SPARSEPR_ROUTING_PRIORITY && p->routing != SPARSEPR_ROUTING_TOP_P)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "routing must be one of SPARSEPR_ROUTING_*");
  if (p->routing == SPARSEPR_ROUTING_TOP_P && CK > 4096)
    return fail(SPARSEPR_ERR_UNSUPPORTED, "top-p routing takes at most 4096 K/V groups");
  if (p->probe_rule == SPARSEPR_PROBES_RANDOM && p->n_probes > 1024 &&
      s->n_q - p->n_dense_prefix > 1024)
    return fail(SPARSEPR_ERR_UNSUPPORTED, "the random probe rule takes at most 1024 probes");
  if (p->resid_rank < 1 || p->resid_rank > s->d_v)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "resid_rank must be in [1, d_v]");
  if (!(p->target_exec_density > 0.f) || !(p->target_exec_density <= 1.f))
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "target_exec_density must be in (0, 1]");
  if (!(p->ridge >= 0.f) || !(p->eps_q >= 0.f) || !(p->eps_x >= 0.f) || !std::isfinite(p->ridge))
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "ridge, eps_q and eps_x must be finite and >= 0");
  g = Geom{};
  g.B = s->batch;
  g.H = s->heads;
  g.Hkv = hkv;
  g.G = s->heads / hkv;
  g.gq = 0;
  g.BH = s->batch * hkv;
  g.N = N;
  g.ntext = p->n_dense_prefix;
  g.NV = NV;
  g.d = s->d;
  g.dv = s->d_v;
  g.partition = p->partition;
  g.probe_rule = p->probe_rule;
  g.probe_seed = p->probe_seed;
  g.ridge_only = p->ridge_only;
  g.routing = p->routing;
  // the semantic partitions cluster the raw d-dimensional rows
  g.rk = p->partition == SPARSEPR_PARTITION_SEMANTIC ? s->d : std::min(p->r_k, s->d);
  g.rq = p->partition != SPARSEPR_PARTITION_RESPONSE ? s->d : std::min(p->r_q, s->d);
  g.CK = CK;
  g.CQ = CQ;
  g.CKt = CK + (g.ntext > 0);
  g.CQt = CQ + (g.ntext > 0);
  g.Ms = std::min(p->n_sampled_queries, NV);
  g.T = p->kmeans_iters;
  g.warm = p->warm_start;
  g.T_warm = p->warm_iters > 0 ? p->warm_iters : p->kmeans_iters;
  g.M = std::min(p->n_probes, NV);
  g.r = p->ridge_only ? s->d_v : p->resid_rank;  // ridge only: Psi = I, all d_v directions
  g.bf16 = s->dtype == SPARSEPR_BF16;
  g.sb = s->stride_b;
  g.sh = s->stride_h;
  g.sn = s->stride_n;
  g.kvsb = kvsb;
  g.kvsh = kvsh;
  g.rho = p->target_exec_density;
  g.ridge = p->ridge;
  g.eps_q = p->eps_q;
  g.eps_x = p->eps_x;
  // the probe rows' cost against all keys is reserved before the cells
  g.budget = (int64_t)std::floor((double)p->target_exec_density * (double)NV * (double)NV) -
             (int64_t)g.M * (int64_t)N;
  g.nchunk_max = (N + kQTile - 1) / kQTile + g.CQt;
  g.nchunk_per_xcd = (g.nchunk_max + 7) / 8;
  g.nsplit = (N + kProbeSplit - 1) / kProbeSplit;
  {
    // Key segments of the sparse attention: each launch reads one slice of
    // the group-major K/V, sized to stay resident in one XCD's 4 MB L2 while
    // every XCD works through that slice for all query groups (6 MiB measured
    // best on the long-video workload among 2-12 MiB and a single pass).
    const double head_kv = (double)N * (double)(g.d + g.dv) * (g.bf16 ? 2.0 : 4.0);
    double seg_bytes = 6.0 * 1024 * 1024;
    if (const char* e = getenv("SPARSEPR_SEG_KB")) seg_bytes = std::max(64.0, atof(e)) * 1024.0;
    g.nseg = (int)std::min(64.0, std::max(1.0, std::ceil(head_kv / seg_bytes)));
  }
  g.nsort_blk = (NV + kSortBlock - 1) / kSortBlock;
  g.nsort_blk_full = (N + kSortBlock - 1) / kSortBlock;
  {
    // The route-selection histograms add a bucket's pair cost (at most NV^2)
    // and, above it, its cell count (at most CQ * CK) in one 64-bit word when
    // both fit; the count lets the selection stop at a one-cell bucket.
    auto bits = [](unsigned long long x) { int b = 0; while (x) { ++b; x >>= 1; } return b; };
    const int wb = bits((unsigned long long)NV * (unsigned long long)NV);
    const int cb = bits((unsigned long long)g.CQ * (unsigned long long)g.CK);
    g.sel_cshift = (wb + cb <= 64 && wb < 64) ? wb : 0;
  }
  g.cmax = std::max(g.CKt, g.CQt);
  g.rpad = (std::max(g.rk, g.rq) + 15) / 16 * 16;
  g.cpad = (std::max(g.CK, g.CQ) + 31) / 32 * 32;
  return SPARSEPR_OK;
}

}  // namespace

struct sparsepr_plan_s {
  Geom g;
  Work w;                // whole-batch view (attend outputs of query head 0 of each group)
  std::vector<Work> wq;  // the same with the attend outputs of query head j, j < G
  Layout L;
  char* base;
  size_t bytes;
  bool planned;
  bool have_centroids = false;  // a previous sparsepr_plan call left its centroids
  // event timing (sparsepr_set_profiling): a ring of event sets, so timed
  // loops of up to kRing calls need no host synchronisation
  static constexpr int kRing = 64;
  bool profiling = false;
  hipEvent_t ev_plan[kRing][2] = {};
  hipEvent_t ev_att[kRing][5] = {};
  int n_plan = 0, n_att = 0;  // pending (recorded, not yet harvested) calls
  sparsepr_timings acc{};
  int static_dev = -1;  // device whose static scratch array this plan holds (-1: none)
};

namespace sparsepr {
sparsepr_status set_error(sparsepr_status st, const std::string& msg) { return fail(st, msg); }
void mark_static_plan(sparsepr_plan_t plan, int dev) { plan->static_dev = dev; }
}  // namespace sparsepr

namespace {

void destroy_events(sparsepr_plan_s* p) {
  for (auto& set : p->ev_plan)
    for (auto& e : set)
      if (e) (void)hipEventDestroy(e), e = nullptr;
  for (auto& set : p->ev_att)
    for (auto& e : set)
      if (e) (void)hipEventDestroy(e), e = nullptr;
  p->profiling = false;
}

// Fold the pending events into the totals (the stream has been synchronised).
void harvest(sparsepr_plan_s* p) {
  float ms = 0.f;
  for (int i = 0; i < p->n_plan; ++i)
    if (hipEventElapsedTime(&ms, p->ev_plan[i][0], p->ev_plan[i][1]) == hipSuccess) {
      p->acc.plan_ms += ms;
      p->acc.plan_calls += 1;
    }
  double* dst[4] = {&p->acc.sparse_attn_ms, &p->acc.probe_ms, &p->acc.fit_ms, &p->acc.correct_ms};
  for (int i = 0; i < p->n_att; ++i) {
    for (int k = 0; k < 4; ++k)
      if (hipEventElapsedTime(&ms, p->ev_att[i][k], p->ev_att[i][k + 1]) == hipSuccess) *dst[k] += ms;
    p->acc.attend_calls += 1;
  }
  p->n_plan = p->n_att = 0;
}

}  // namespace

extern "C" {

void sparsepr_params_default(sparsepr_params* p) {
  if (!p) return;
  p->n_sampled_queries = 256;
  p->r_k = 48;
  p->r_q = 64;
  p->n_kv_groups = 0;
  p->n_q_groups = 0;
  p->kmeans_iters = 8;
  p->target_exec_density = 0.22f;
  p->n_probes = 64;
  p->resid_rank = 16;
  p->ridge = 0.1f;
  p->eps_q = 1e-6f;
  p->eps_x = 1e-6f;
  p->n_dense_prefix = 0;
  p->warm_start = 0;
  p->warm_iters = 0;
  p->partition = SPARSEPR_PARTITION_RESPONSE;
  p->probe_rule = SPARSEPR_PROBES_STRATIFIED;
  p->probe_seed = 0;
  p->ridge_only = 0;
  p->routing = SPARSEPR_ROUTING_PRIORITY;
}

sparsepr_status sparsepr_workspace_size(const sparsepr_shape* shape, const sparsepr_params* params,
                                        size_t* bytes) {
  if (!bytes) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "bytes must not be NULL");
  Geom g;
  const sparsepr_status st = validate(shape, params, g);
  if (st != SPARSEPR_OK) return st;
  Work w{};
  Layout L;
  describe(g, &w, L);
  *bytes = L.total;
  return ok();
}

sparsepr_status sparsepr_plan_create(const sparsepr_shape* shape, const sparsepr_params* params,
                                     void* workspace, size_t bytes, sparsepr_plan_t* out) {
  if (!out) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "out must not be NULL");
  Geom g;
  sparsepr_status st = validate(shape, params, g);
  if (st != SPARSEPR_OK) return st;
  if (!workspace) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "workspace must not be NULL");
  if (((uintptr_t)workspace & 255) != 0)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  sparsepr_plan_s* p = new (std::nothrow) sparsepr_plan_s();
  if (!p) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "out of host memory");
  p->g = g;
  describe(g, &p->w, p->L);
  if (bytes < p->L.total) {
    const size_t need = p->L.total;
    delete p;
    return fail(SPARSEPR_ERR_WORKSPACE_TOO_SMALL,
                "workspace holds " + std::to_string(bytes) + " bytes, needs " + std::to_string(need));
  }
  p->base = (char*)workspace;
  p->bytes = bytes;
  bind(g, &p->w, p->L, p->base, -1);
  p->wq.resize(g.G);
  for (int j = 0; j < g.G; ++j) bind(g, &p->wq[j], p->L, p->base, -1, j);
  // no work item and no probe until a plan exists
  st = hip_check(hipMemset(p->w.nchunks, 0, sizeof(int32_t) * g.BH), "hipMemset");
  if (st == SPARSEPR_OK) st = hip_check(hipMemset(p->w.nprobes, 0, sizeof(int32_t) * g.BH), "hipMemset");
  if (st == SPARSEPR_OK) st = hip_check(hipMemset(p->w.stats, 0, sizeof(int64_t) * 16 * g.BH), "hipMemset");
  if (st != SPARSEPR_OK) {
    delete p;
    return st;
  }
  p->planned = false;
  *out = p;
  return ok();
}

sparsepr_status sparsepr_plan(sparsepr_plan_t plan, const void* q, const void* k, void* stream) {
  if (!plan || !q || !k) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "plan, q and k must not be NULL");
  (void)hipGetLastError();  // report only this call's launch errors
  hipEvent_t* ev = nullptr;
  if (plan->profiling) {
    if (plan->n_plan == sparsepr_plan_s::kRing) {
      (void)hipStreamSynchronize((hipStream_t)stream);
      harvest(plan);
    }
    ev = plan->ev_plan[plan->n_plan++];
    (void)hipEventRecord(ev[0], (hipStream_t)stream);
  }
  launch_plan(plan->g, plan->w, q, k, (hipStream_t)stream, plan->g.warm && plan->have_centroids);
  if (ev) (void)hipEventRecord(ev[1], (hipStream_t)stream);
  const sparsepr_status st = hip_check(hipGetLastError(), "sparsepr_plan launch");
  if (st != SPARSEPR_OK) return st;
  plan->planned = true;
  plan->have_centroids = true;
  return ok();
}

sparsepr_status sparsepr_attend(sparsepr_plan_t plan, const void* q, const void* k, const void* v,
                                void* out, void* stream) {
  if (!plan || !q || !k || !v || !out)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "plan, q, k, v and out must not be NULL");
  if (!plan->planned) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "no plan: call sparsepr_plan or sparsepr_plan_import first");
  (void)hipGetLastError();
  hipEvent_t* ev = nullptr;
  if (plan->profiling) {
    if (plan->n_att == sparsepr_plan_s::kRing) {
      (void)hipStreamSynchronize((hipStream_t)stream);
      harvest(plan);
    }
    ev = plan->ev_att[plan->n_att++];
  }
  launch_attend(plan->g, plan->wq.data(), q, k, v, out, (hipStream_t)stream, ev);
  const sparsepr_status st = hip_check(hipGetLastError(), "sparsepr_attend launch");
  if (st != SPARSEPR_OK) return st;
  return ok();
}

sparsepr_status sparsepr_dense_workspace_size(const sparsepr_shape* shape, size_t* bytes) {
  if (!bytes) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "bytes must not be NULL");
  sparsepr_params p;
  sparsepr_params_default(&p);
  Geom g;
  const sparsepr_status st = validate(shape, &p, g);
  if (st != SPARSEPR_OK) return st;
  *bytes = 0;
  return ok();
}

sparsepr_status sparsepr_dense_attend(const sparsepr_shape* shape, const void* q, const void* k,
                                      const void* v, void* out, void* workspace, size_t bytes,
                                      void* stream) {
  (void)workspace;
  (void)bytes;
  if (!q || !k || !v || !out) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "q, k, v and out must not be NULL");
  sparsepr_params p;
  sparsepr_params_default(&p);
  Geom g;
  const sparsepr_status st = validate(shape, &p, g);
  if (st != SPARSEPR_OK) return st;
  (void)hipGetLastError();
  launch_dense(g, q, k, v, out, nullptr, (hipStream_t)stream);
  return hip_check(hipGetLastError(), "sparsepr_dense_attend launch") == SPARSEPR_OK ? ok()
                                                                                     : SPARSEPR_ERR_HIP;
}

sparsepr_status sparsepr_get_stats(sparsepr_plan_t plan, sparsepr_stats* out, void* stream) {
  if (!plan || !out) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "plan and out must not be NULL");
  sparsepr_status st = hip_check(hipStreamSynchronize((hipStream_t)stream), "hipStreamSynchronize");
  if (st != SPARSEPR_OK) return st;
  const Geom& g = plan->g;
  std::vector<int64_t> s((size_t)g.BH * 16);
  st = hip_check(hipMemcpy(s.data(), plan->w.stats, s.size() * 8, hipMemcpyDeviceToHost), "hipMemcpy");
  if (st != SPARSEPR_OK) return st;
  std::memset(out, 0, sizeof(*out));
  double rr = 0.0, re = 0.0;
  const double nn = (double)g.N * (double)g.N;
  for (int bh = 0; bh < g.BH; ++bh) {
    const int64_t* h = &s[(size_t)bh * 16];
    // every query head sharing the K/V head evaluates the plan's pairs
    out->routed_pairs += h[ST_ROUTED_PAIRS] * g.G;
    out->exec_pairs += (h[ST_ROUTED_PAIRS] + h[ST_NPROBES] * (int64_t)g.N) * g.G;
    out->forced_pairs += h[ST_FORCED_PAIRS] * g.G;
    out->routed_cells += (int32_t)h[ST_ROUTED_CELLS];
    out->forced_cells += (int32_t)h[ST_FORCED_CELLS];
    out->nonempty_q_groups += (int32_t)h[ST_NE_Q];
    out->nonempty_kv_groups += (int32_t)h[ST_NE_K];
    out->n_probes += (int32_t)h[ST_NPROBES] * g.G;
    out->kmeans_iters_kv = std::max(out->kmeans_iters_kv, (int32_t)h[ST_ITK]);
    out->kmeans_iters_q = std::max(out->kmeans_iters_q, (int32_t)h[ST_ITQ]);
    out->status_flags |= (int32_t)h[ST_FLAGS];
    out->kmeans_rescans += h[ST_RESCAN];
    rr += (double)h[ST_ROUTED_PAIRS] / nn;
    re += (double)h[ST_ROUTED_PAIRS] / nn + (double)h[ST_NPROBES] / (double)g.N;
  }
  out->rho_route = rr / g.BH;
  out->rho_exec = re / g.BH;
  return ok();
}

sparsepr_status sparsepr_plan_export(sparsepr_plan_t plan, int32_t bh, sparsepr_plan_host* out,
                                     void* stream) {
  if (!plan || !out) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "plan and out must not be NULL");
  const Geom& g = plan->g;
  if (bh < 0 || bh >= g.B * g.H) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "bh out of range");
  sparsepr_status st = hip_check(hipStreamSynchronize((hipStream_t)stream), "hipStreamSynchronize");
  if (st != SPARSEPR_OK) return st;
  // query head bh = b*H + h uses the plan of K/V head b*Hkv + h/G
  const int hq = bh % g.H;
  Work h;
  bind(g, &h, plan->L, plan->base, (bh / g.H) * g.Hkv + hq / g.G, hq % g.G);
  int32_t np = 0;
  st = hip_check(hipMemcpy(&np, h.nprobes, 4, hipMemcpyDeviceToHost),
                 ("export n_probes" + ptrs(&np, h.nprobes, 4)).c_str());
  if (st != SPARSEPR_OK) return st;
  out->n_probes = np;
  int64_t rank = 0;
  st = hip_check(hipMemcpy(&rank, h.stats + ST_FIT_RANK, 8, hipMemcpyDeviceToHost),
                 ("export fit_rank" + ptrs(&rank, h.stats, 8)).c_str());
  if (st != SPARSEPR_OK) return st;
  out->fit_rank = (int32_t)rank;
  struct Cp {
    void* dst;
    const void* src;
    size_t bytes;
    const char* name;
  };
  const size_t N = g.N, NV = g.NV, d = g.d, dv = g.dv, r = g.r;
  std::vector<float> mk, mq;
  const Cp cps[] = {
      {out->labels_q, h.labq, N * 4, "labels_q"},
      {out->labels_kv, h.labk, N * 4, "labels_kv"},
      {out->routes, h.z, (size_t)g.CQt * g.CKt, "routes"},
      {out->probes, h.probes, (size_t)np * 4, "probes"},
      {out->probe_weights, h.pw, (size_t)np * 4, "probe_weights"},
      {out->perm_q, h.permq, N * 4, "perm_q"},
      {out->off_q, h.offq, (size_t)(g.CQt + 1) * 4, "off_q"},
      {out->perm_kv, h.permk, N * 4, "perm_kv"},
      {out->off_kv, h.offk, (size_t)(g.CKt + 1) * 4, "off_kv"},
      {out->f_k, h.fk, d * g.rk * 4, "f_k"},
      {out->f_q, h.fq, d * g.rq * 4, "f_q"},
      {out->phi_k, h.phik, NV * g.rk * 4, "phi_k"},
      {out->phi_q, h.phiq, NV * g.rq * 4, "phi_q"},
      {out->cent_k, h.centk, (size_t)g.CK * g.rk * 4, "cent_k"},
      {out->cent_q, h.centq, (size_t)g.CQ * g.rq * 4, "cent_q"},
      {out->kbar, h.kbar, (size_t)g.CK * d * 4, "kbar"},
      {out->qbar, h.qbar, (size_t)g.CQ * d * 4, "qbar"},
      {out->route_prio, h.prio, (size_t)g.CQ * g.CK * 4, "route_prio"},
      {out->route_key, g.routing == SPARSEPR_ROUTING_TOP_P ? h.skey : h.prio,
       (size_t)g.CQ * g.CK * 4, "route_key"},
      {out->o_sparse, h.osp, N * dv * 4, "o_sparse"},
      {out->o_dense_probes, h.odp, (size_t)np * dv * 4, "o_dense_probes"},
      {out->fit_mu_x, h.fitv, dv * 4, "fit_mu_x"},
      {out->fit_s_x, h.fitv + dv, dv * 4, "fit_s_x"},
      {out->fit_mu_r, h.fitv + 2 * dv, dv * 4, "fit_mu_r"},
      {out->fit_bpsi, h.fity, dv * r * 4, "fit_bpsi"},
      {out->fit_psi, h.fitpsi, dv * r * 4, "fit_psi"},
  };
  for (const Cp& c : cps) {
    if (!c.dst || c.bytes == 0) continue;
    st = hip_check(hipMemcpy(c.dst, c.src, c.bytes, hipMemcpyDeviceToHost),
                   (std::string("export ") + c.name + ptrs(c.dst, c.src, c.bytes)).c_str());
    if (st != SPARSEPR_OK) return st;
  }
  // the metrics are kept in double on the device
  for (int which = 0; which < 2; ++which) {
    float* dst = which == 0 ? out->m_k : out->m_q;
    if (!dst) continue;
    std::vector<double> tmp(d * d);
    st = hip_check(hipMemcpy(tmp.data(), which == 0 ? h.gram_k : h.gram_q, d * d * 8,
                             hipMemcpyDeviceToHost),
                   ("export metric" + ptrs(tmp.data(), h.gram_k, d * d * 8)).c_str());
    if (st != SPARSEPR_OK) return st;
    for (size_t i = 0; i < d * d; ++i) dst[i] = (float)tmp[i];
  }
  return ok();
}

sparsepr_status sparsepr_plan_import(sparsepr_plan_t plan, int32_t bh, const sparsepr_plan_host* in,
                                     void* stream) {
  if (!plan || !in) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "plan and in must not be NULL");
  const Geom& g = plan->g;
  if (bh < 0 || bh >= g.B * g.H) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "bh out of range");
  if (!in->labels_q || !in->labels_kv || !in->routes || (in->n_probes > 0 && !in->probes))
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "labels_q, labels_kv, routes and probes are required");
  if (in->n_probes < 0 || in->n_probes > g.M)
    return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "n_probes must be in [0, min(M, n_v)]");
  const int N = g.N;
  std::vector<int> nq(g.CQt, 0), nk(g.CKt, 0);
  for (int i = 0; i < N; ++i) {
    const int a = in->labels_q[i], b = in->labels_kv[i];
    if (a < 0 || a >= g.CQt || b < 0 || b >= g.CKt)
      return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "label out of range at row " + std::to_string(i));
    nq[a]++;
    nk[b]++;
  }
  for (int a = 0; a < g.CQt; ++a) {
    if (nq[a] == 0) continue;
    bool any = false;
    for (int b = 0; b < g.CKt && !any; ++b) any = in->routes[(size_t)a * g.CKt + b] && nk[b] > 0;
    if (!any)
      return fail(SPARSEPR_ERR_INVALID_ARGUMENT,
                  "query group " + std::to_string(a) + " routes no nonempty K/V group");
  }
  std::vector<char> seen(N, 0);
  for (int p = 0; p < in->n_probes; ++p) {
    const int row = in->probes[p];
    if (row < g.ntext || row >= N || seen[row])
      return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "probe rows must be distinct rows in [n_dense_prefix, n)");
    seen[row] = 1;
  }
  hipStream_t s = (hipStream_t)stream;
  sparsepr_status st = hip_check(hipStreamSynchronize(s), "hipStreamSynchronize");
  if (st != SPARSEPR_OK) return st;
  Work h;
  bind(g, &h, plan->L, plan->base, (bh / g.H) * g.Hkv + (bh % g.H) / g.G);
  const int32_t np = in->n_probes;
  struct Cp {
    void* dst;
    const void* src;
    size_t bytes;
  };
  const Cp cps[] = {
      {h.labq, in->labels_q, (size_t)N * 4},
      {h.labk, in->labels_kv, (size_t)N * 4},
      {h.z, in->routes, (size_t)g.CQt * g.CKt},
      {h.probes, in->probes, (size_t)np * 4},
      {h.nprobes, &np, 4},
  };
  for (const Cp& c : cps) {
    if (c.bytes == 0) continue;
    st = hip_check(hipMemcpy(c.dst, c.src, c.bytes, hipMemcpyHostToDevice), "hipMemcpy");
    if (st != SPARSEPR_OK) return st;
  }
  Geom g1 = g;
  g1.B = 1;
  g1.H = g.G;
  g1.Hkv = 1;
  g1.BH = 1;
  (void)hipGetLastError();
  launch_rebuild(g1, h, 0, s);
  st = hip_check(hipGetLastError(), "sparsepr_plan_import launch");
  if (st != SPARSEPR_OK) return st;
  st = hip_check(hipStreamSynchronize(s), "hipStreamSynchronize");
  if (st != SPARSEPR_OK) return st;
  plan->planned = true;
  return ok();
}

sparsepr_status sparsepr_set_profiling(sparsepr_plan_t plan, int32_t enable) {
  if (!plan) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "plan must not be NULL");
  if (!enable) {
    destroy_events(plan);
    return ok();
  }
  if (plan->profiling) return ok();
  for (auto& set : plan->ev_plan)
    for (auto& e : set) {
      const sparsepr_status st = hip_check(hipEventCreate(&e), "hipEventCreate");
      if (st != SPARSEPR_OK) {
        destroy_events(plan);
        return st;
      }
    }
  for (auto& set : plan->ev_att)
    for (auto& e : set) {
      const sparsepr_status st = hip_check(hipEventCreate(&e), "hipEventCreate");
      if (st != SPARSEPR_OK) {
        destroy_events(plan);
        return st;
      }
    }
  plan->acc = sparsepr_timings{};
  plan->n_plan = plan->n_att = 0;
  plan->profiling = true;
  return ok();
}

sparsepr_status sparsepr_get_timings(sparsepr_plan_t plan, sparsepr_timings* out, int32_t reset,
                                     void* stream) {
  if (!plan || !out) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "plan and out must not be NULL");
  if (!plan->profiling) return fail(SPARSEPR_ERR_INVALID_ARGUMENT, "profiling is not enabled");
  const sparsepr_status st = hip_check(hipStreamSynchronize((hipStream_t)stream), "hipStreamSynchronize");
  if (st != SPARSEPR_OK) return st;
  harvest(plan);
  *out = plan->acc;
  out->attn_launches = plan->g.bf16 ? plan->g.nseg : 1;
  if (reset) plan->acc = sparsepr_timings{};
  return ok();
}

void sparsepr_plan_destroy(sparsepr_plan_t plan) {
  if (!plan) return;
  destroy_events(plan);
  if (plan->static_dev >= 0) release_static_scratch(plan->static_dev);
  delete plan;
}

const char* sparsepr_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
