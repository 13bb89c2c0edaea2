// Internal declarations shared by the HIP translation units of the SparsePR
// library: problem geometry, the device workspace layout and the host-side
// launchers of every kernel.  Nothing here is part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>

#include "../../include/sparsepr.h"

namespace sparsepr {

// Attention-kernel query tile: rows of one query group handled by a block.
constexpr int kQTile = 64;
// Key tile of the attention kernels.
constexpr int kKTile = 64;
// Probe-row dense attention: keys per split.
constexpr int kProbeSplit = 2048;
// Tokens per block of the counting sort.
constexpr int kSortBlock = 1024;
// Bins of one radix-select pass (8-bit digits over 64-bit keys).
constexpr int kSelBins = 256;
constexpr int kSelPasses = 8;

struct Geom {
  int B, H, BH;           // batch, query heads, batch * K/V heads (one plan each)
  int Hkv, G;             // K/V heads; query heads per K/V head (H = Hkv * G)
  int gq;                 // attend: which query head of each K/V head's group
  int N, NV, ntext;       // rows, video rows, dense-prefix rows
  int d, dv;              // head dims (equal)
  int rk, rq;             // response ranks, clamped to d
  int CK, CQ;             // video groups
  int CKt, CQt;           // + the dense-prefix group when ntext > 0
  int Ms;                 // sampled queries (clamped to NV)
  int T;                  // k-means iterations (cold start; sizes the per-iteration state)
  int T_warm;             // k-means iterations when warm-started (<= T)
  int warm;               // warm start requested
  int partition;          // SPARSEPR_PARTITION_*
  int probe_rule;         // SPARSEPR_PROBES_*
  uint32_t probe_seed;    // seed of the random probe rule
  int ridge_only;         // fit without the probe-residual subspace (Psi = I)
  int routing;            // SPARSEPR_ROUTING_*
  int sel_cshift;         // bit where the selection histograms count cells (0: not counted)
  int M;                  // probes per head, min(n_probes, NV)
  int r;                  // residual rank
  int bf16;               // 1: bf16 tensors, 0: fp32
  int64_t sb, sh, sn;     // element strides of Q and O (sn also of K and V)
  int64_t kvsb, kvsh;     // batch and head strides of K and V
  float rho, ridge, eps_q, eps_x;
  int64_t budget;         // video x video pair budget after the probe reservation
  int nchunk_max;         // attention work items per head (upper bound)
  int nchunk_per_xcd;     // ceil(nchunk_max / 8): chunks of one head per XCD
  int nsplit;             // probe attention key splits
  int nseg;               // key segments of the sparse attention (one launch each)
  int nsort_blk;          // counting-sort blocks over NV rows
  int nsort_blk_full;     // counting-sort blocks over N rows
  int cmax;               // max(CKt, CQt)
  int rpad;               // max(rk, rq) rounded up to 16 (MFMA k-steps)
  int cpad;               // max(CK, CQ) rounded up to 32 (MFMA tiles)
};

// Device workspace: every array is [BH][...] contiguous.
struct Work {
  double* gram_k;   // [BH][d][d]
  double* gram_q;   // [BH][d][d]
  float* evals_k;   // [BH][d]
  float* evals_q;   // [BH][d]
  float* fk;        // [BH][d][rk]
  float* fq;        // [BH][d][rq]
  float* phik;      // [BH][NV][rk]
  float* phiq;      // [BH][NV][rq]
  float* centk;     // [BH][CK][rk]
  float* centq;     // [BH][CQ][rq]
  int32_t* labk;    // [BH][N]  (row order; dense prefix -> CK)
  int32_t* labq;    // [BH][N]
  int32_t* permk;   // [BH][N]
  int32_t* permq;   // [BH][N]
  int32_t* offk;    // [BH][CKt+1]
  int32_t* offq;    // [BH][CQt+1]
  int32_t* blkhist; // [BH][nsort_blk_full][cmax]
  int32_t* kmstate; // [BH][2][T+1]: labels changed per assignment (kv, q)
  uint16_t* km_xhi; // [BH][NV][rpad] bf16 high part of the k-means points
  uint16_t* km_xlo; // [BH][NV][rpad] bf16 low part (x - hi)
  float* km_xn;     // [BH][NV] point norms
  uint16_t* km_chi; // [BH][cpad][rpad] bf16 high part of the centroids
  uint16_t* km_clo; // [BH][cpad][rpad]
  float* km_cu;     // [BH][cpad] exact squared centroid norms (+inf for padding)
  uint32_t* km_cn3; // [BH][cpad][2] the norms as three bf16 parts (operand of the MFMA norm step)
  int32_t* km_fbcnt;// [BH][2][T] number of such points per assignment
  float* kbar;      // [BH][CK][d]
  float* qbar;      // [BH][CQ][d]
  float* prio;      // [BH][CQ][CK]
  float* skey;      // [BH][CQ][CK] key of the routing walk (prio itself, or the top-p keys)
  int32_t* forced;  // [BH][CQ]
  uint64_t* selhist;  // [BH][kSelPasses][kSelBins]
  int64_t* selstate;  // [BH][8]
  uint8_t* z;         // [BH][CQt][CKt]
  int32_t* rng_cnt;   // [BH][CQt]
  int2* rng;          // [BH][CQt][CKt]: (start position in perm_kv, length)
  int32_t* keytot;    // [BH][CQt]
  int4* chunks;       // [BH][nchunk_max]: (a, row start in group, rows, keys)
  int32_t* nchunks;   // [BH]
  float* d2;          // [BH][NV] probe radial distances
  int32_t* probes;    // [BH][M]
  float* pw;          // [BH][M]
  int32_t* nprobes;   // [BH]
  int32_t* picks;     // [BH][M] probe-selection scratch
  uint16_t* kperm;    // [BH][N][d]  bf16 K in group-major order
  uint16_t* vperm;    // [BH][N][dv] bf16 V in group-major order
  float* osp;         // [BH][N][dv]
  float* odp;         // [BH][M][dv]
  float* part;        // [BH][M][nsplit][dv+2] split partials (o, m, l)
  float* mlst;        // [BH][N][4] running (m, l_lo, l_hi) of the sparse attention between key segments
  float* fitv;        // [BH][3*dv] mu_x, s_x, mu_r
  float* fity;        // [BH][dv][r] B Psi
  float* fitpsi;      // [BH][dv][r]
  double* fitscr;     // [BH][2*M*dv + M*r + dv*r + M] fit scratch
  double* fitgram;    // [BH][2][dv][dv] Rbar^T W Rbar and xbar^T W xbar + lambda I
  double* fitvec;     // [BH][dv][dv+4] eigenvectors (transposed) of a double fit solve kept out of LDS
  double* eigscr;     // [G][BH][4][D][D] pivots and ratios of the tridiagonal eigensolver's twisted factorisations (D = max(d, dv))
  int64_t* stats;     // [BH][16]
};

// stats slots
enum {
  ST_ROUTED_PAIRS = 0,
  ST_FORCED_PAIRS = 1,
  ST_ROUTED_CELLS = 2,
  ST_FORCED_CELLS = 3,
  ST_NPROBES = 4,
  ST_ITK = 5,
  ST_ITQ = 6,
  ST_FLAGS = 7,
  ST_NE_Q = 8,
  ST_NE_K = 9,
  ST_RESCAN = 10,
  ST_FIT_RANK = 11,
};

// ---- plan kernels -------------------------------------------------------
void launch_plan(const Geom& g, const Work& w, const void* q, const void* k, hipStream_t s,
                 bool warm);
// Rebuild permutations, route lists, chunks and probe weights from labels,
// z and probes already placed in the workspace for head bh (import path).
void launch_rebuild(const Geom& g, const Work& w, int bh, hipStream_t s);
// ---- attend kernels -----------------------------------------------------
// Optional events recorded between the phases of attend (null = none):
// ev[0] before the sparse attention, ev[1] after it, ev[2] after the probe
// rows, ev[3] after the fit, ev[4] after the correction.  wq[j] (j < G) is the
// workspace view holding the attend outputs of query head j of every K/V
// head; each phase runs for the G query heads in turn.
void launch_attend(const Geom& g, const Work* wq, const void* q, const void* k, const void* v,
                   void* out, hipStream_t s, hipEvent_t* ev = nullptr);
// Fit, correction and restore after the sparse and probe attention
// (records ev[3] after the solve and ev[4] at the end when ev is set).
void launch_fit_correct(const Geom& g, const Work& w0, void* out, hipStream_t s, hipEvent_t* ev);
void launch_dense(const Geom& g, const void* q, const void* k, const void* v, void* out,
                  float* part, hipStream_t s);

// ---- plans on the static scratch array (noalloc.hip) ---------------------
// Size of the file-scope device array behind sparsepr_plan_create_static.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
// Record the calling thread's error message and return `st` (api.cpp).
sparsepr_status set_error(sparsepr_status st, const std::string& msg);
// Mark a plan as holding device `dev`'s static array; destroying it releases
// the array (api.cpp / noalloc.hip).
void mark_static_plan(sparsepr_plan_t plan, int dev);
void release_static_scratch(int dev);

}  // namespace sparsepr
