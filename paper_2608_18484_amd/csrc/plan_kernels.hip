// Planner kernels of the SparsePR operator for gfx950: Response-Coupled
// Partitioning (Sec. 4.1, App. B), budgeted shared block routing (Sec. 4.3)
// and query-group-stratified probe selection (App. A.2).
//
// Decisions that must be reproducible bit for bit (k-means labels, group
// order, route set, probe set) are taken on float values computed in a fixed
// operation order, with the lowest index winning ties:
//  * k-means score of point x and centroid c: t = fmaf chain of x_k c_k over
//    k in index order, u = fmaf chain of c_k c_k, score = fmaf(-2, t, u);
//  * centroids: double sums over members in ascending row order / count;
//  * probe radial key: fmaf chain of (phi_k - c_k)^2 in index order.
#include <hip/hip_runtime.h>
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "device_utils.hpp"
#include "sparsepr_internal.hpp"
#include "jacobi_lds.hpp"
#include "tridiag_eig.hpp"

namespace sparsepr {

// ---------------------------------------------------------------------------
// Per-call initialisation
// ---------------------------------------------------------------------------

__global__ void k_plan_init(Geom g, Work w) {
  const int bh = blockIdx.x;
  for (int i = threadIdx.x; i < 16; i += blockDim.x) w.stats[bh * 16 + i] = 0;
  for (int i = threadIdx.x; i < 2 * (g.T + 1); i += blockDim.x)
    w.kmstate[bh * 2 * (g.T + 1) + i] = (i % (g.T + 1) == 0) ? 1 : 0;
  for (int i = threadIdx.x; i < 2 * g.T; i += blockDim.x) w.km_fbcnt[bh * 2 * g.T + i] = 0;
}

// ---------------------------------------------------------------------------
// Key-response metric M_K = Q_s^T Q_s / M_s over the strided query sample
// s_i = floor(i * n_v / M_s) (Sec. 4.1; App. B.1 eq. app_key_metric).  With
// grouped-query attention the sample is pooled over the G query heads that
// share the K/V head (App. B.1 builds M_K per K/V head): the G per-head
// metrics are averaged.
// ---------------------------------------------------------------------------

template <int D>
__global__ __launch_bounds__(256) void k_key_metric(const void* q, Geom g, double* gram) {
  // block (x, bh) forms output rows [RB x, RB x + RB)
  constexpr int RB = 16;
  constexpr int ENT = RB * D / 256;
  constexpr int SB = 32;
  __shared__ float qs[SB][D];
  const int bh = blockIdx.y, tid = threadIdx.x;
  const int e0 = tid * ENT, ra = blockIdx.x * RB + e0 / D, cb = e0 % D;
  double acc[ENT];
#pragma unroll
  for (int e = 0; e < ENT; ++e) acc[e] = 0.0;
  for (int j = 0; j < g.G; ++j) {
    const int64_t base = q_base(g, bh, j);
    for (int s0 = 0; s0 < g.Ms; s0 += SB) {
      // eight consecutive elements per load (16 bytes of bf16, two float4)
#pragma unroll
      for (int t8 = tid; t8 < SB * D / 8; t8 += 256) {
        const int i = s0 + t8 / (D / 8), c = (t8 % (D / 8)) * 8;
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;
        if (i < g.Ms) {
          const int64_t row = g.ntext + ((int64_t)i * g.NV) / g.Ms;
          const int64_t off = base + row * g.sn + c;
          if (g.bf16) {
            const uint4 u = *(const uint4*)((const uint16_t*)q + off);
            const uint32_t wds[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              v[2 * e] = __uint_as_float(wds[e] << 16);
              v[2 * e + 1] = __uint_as_float(wds[e] & 0xffff0000u);
            }
          } else {
            const float4 u0 = *(const float4*)((const float*)q + off);
            const float4 u1 = *(const float4*)((const float*)q + off + 4);
            v[0] = u0.x; v[1] = u0.y; v[2] = u0.z; v[3] = u0.w;
            v[4] = u1.x; v[5] = u1.y; v[6] = u1.z; v[7] = u1.w;
          }
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) qs[t8 / (D / 8)][c + e] = v[e];
      }
      __syncthreads();
      const int cnt = min(SB, g.Ms - s0);
#pragma unroll 4
      for (int i = 0; i < cnt; ++i) {
        const double a = qs[i][ra];
#pragma unroll
        for (int e = 0; e < ENT; ++e) acc[e] += a * (double)qs[i][cb + e];
      }
      __syncthreads();
    }
  }
  double* out = gram + (size_t)bh * D * D + (size_t)ra * D + cb;
#pragma unroll
  for (int e = 0; e < ENT; ++e) out[e] = acc[e] / ((double)g.Ms * (double)g.G);
}

// Sort the eigenvalues on A's diagonal in descending order (ties by index):
// order[t] = index of the t-th largest.  Needs D threads.
template <int D, typename T>
__device__ void eig_order(const T* A, int* order) {
  constexpr int LD = D + 1;
  const int i = threadIdx.x;
  if (i < D) {
    // a NaN diagonal (non-finite input) ranks as -inf, so the ranks stay a
    // permutation and every order[] entry is written
    const T li = eig_rank_key(A[i * LD + i]);
    int rank = 0;
    for (int j = 0; j < D; ++j) {
      const T lj = eig_rank_key(A[j * LD + j]);
      rank += (lj > li) || (lj == li && j < i);
    }
    order[rank] = i;
  }
  __syncthreads();
}

// Eigen-scaled response basis (Sec. 4.1; App. B.1, B.2): the leading r
// eigendirections, each scaled by sqrt(lambda / mean of the r retained
// lambdas); eigenvalues below tau * lambda_1 are clamped to 0 first.  The
// tridiagonal solver gives the eigenvalues and the vectors of the retained
// ones; when its check fails (a numerically repeated retained eigenvalue)
// the block reloads the matrix and solves it by cyclic Jacobi instead.
template <int D>
__global__ __launch_bounds__(1024) void k_eig_basis(const double* gram, int r, float tau, float* F,
                                                    float* evals, double* scr, int64_t* stats) {
  using T = typename std::conditional<D <= 64, double, float>::type;
  constexpr int LD = D + 1;
  constexpr int LV = jacobi_vt_ld<D>();
  __shared__ T A[D * LD];
  __shared__ __attribute__((aligned(16))) T VT[D * LV];
  __shared__ JacobiRot<T> rot[D / 2];
  __shared__ TriWork<D, T, 1024> tw;
  __shared__ int order[D];
  __shared__ double lam[D];
  __shared__ int flag, nvec;
  __shared__ double meanv;
  const int bh = blockIdx.x, tid = threadIdx.x;
  const double* G = gram + (size_t)bh * D * D;
  for (int i = tid; i < D * D; i += blockDim.x) A[(i / D) * LD + (i % D)] = (T)G[i];
  __syncthreads();
  tri_reduce<D, T, 1024>(A, tw);
  tri_eigvals<D, T, 1024>(tw);
  if (tid == 0) {
    const float l1 = tw.lamf[0];
    int n = 0;
    while (n < r && n < D && l1 > 0.f && tw.lamf[n] >= tau * l1) ++n;
    nvec = n;
  }
  __syncthreads();
  tri_vectors<D, T, 1024>(tw, VT, LV, nvec, scr + (size_t)bh * 4 * D * D);
  if (tw.ok) {
    tri_back<D, T, 1024>(A, tw, VT, LV, nvec);
    if (tid < D) {
      order[tid] = tid;
      lam[tid] = tid < nvec ? tw.lamv[tid]
                            : ((tw.lamf[0] > 0.f && tw.lamf[tid] >= tau * tw.lamf[0]) ? (double)tw.lamf[tid] : 0.0);
    }
  } else {
    if (tid == 0)
      atomicOr((unsigned long long*)&stats[(size_t)bh * 16 + ST_FLAGS], (unsigned long long)SPARSEPR_FLAG_EIG_JACOBI);
    for (int i = tid; i < D * D; i += blockDim.x) A[(i / D) * LD + (i % D)] = (T)G[i];
    __syncthreads();
    // In float the basis reaches its rounding floor at a relative off-diagonal
    // norm of about 1e-4 (measured on the long-video key metric: the weighted
    // projector then differs from a double solve by 2.7e-5).
    jacobi_eig_lds<D, T, 1024>(A, VT, rot, &flag, sizeof(T) == 8 ? T(1e-12) : T(1e-4));
    eig_order<D, T>(A, order);
    const double l1 = A[order[0] * LD + order[0]];
    if (tid < D) {
      const double l = A[order[tid] * LD + order[tid]];
      lam[tid] = (l1 > 0.0 && l >= (double)tau * l1) ? l : 0.0;
    }
  }
  __syncthreads();
  if (tid == 0) {
    double s = 0.0;
    for (int t = 0; t < r; ++t) s += lam[t];
    meanv = s / r;
  }
  __syncthreads();
  float* Fo = F + (size_t)bh * D * r;
  for (int i = tid; i < D * r; i += blockDim.x) {
    const int row = i / r, t = i % r;
    const double wgt = (meanv > 0.0 && lam[t] > 0.0) ? sqrt(lam[t] / meanv) : 0.0;
    Fo[i] = wgt > 0.0 ? (float)((double)VT[order[t] * LV + row] * wgt) : 0.f;
  }
  if (tid < D) evals[(size_t)bh * D + tid] = (float)lam[tid];
}

// ---------------------------------------------------------------------------
// Response coordinates phi = F^T x (eq. key_response_feature), optionally
// divided by max(RMS, eps) (eq. query_response_feature).  64 rows per block;
// thread (ty, tx) computes rows ty + 16u (u < 4) x columns [tx*CPT, tx*CPT +
// CPT), so each LDS read of F feeds four rows.  Keys come from the K/V head;
// queries (`query`) from its G query heads, whose (normalised) coordinates
// are averaged (grouped-query attention shares one query partition per K/V
// head; G = 1 is the single-head case).
// ---------------------------------------------------------------------------

constexpr int PROJ_CHUNKS = 8;

template <int D, int MAXR, bool MF>
__global__ __launch_bounds__(256) void k_project(const void* x, Geom g, const float* F, int R,
                                                 int query, int rms, float eps, float* phi,
                                                 int64_t* stats, uint16_t* xhi, uint16_t* xlo,
                                                 float* xn, int RP) {
  // MF (bf16 inputs): the products run on MFMA.  F is split into three bf16
  // parts (hi + mid + lo reproduce its float value), each bf16 input times a
  // part is exact in float, so the accumulation is the only rounding, as in
  // the float loop.  Each wave takes 32 x 32 output tiles (A = 32 input
  // rows read straight from memory, B = 32 columns of the split F in LDS);
  // the tiles go through LDS to the same thread mapping as the float loop.
  constexpr int ROWS = 64, CPT = MAXR / 16;
  constexpr int FLD = D + 8;  // bf16 pitch of the split F rows
  constexpr int NCT = MAXR / 32, KS = D / 16;
  constexpr size_t XS_BYTES = MF ? 4 : (size_t)ROWS * (D + 1) * 4;
  constexpr size_t FS_BYTES = MF ? (size_t)3 * MAXR * FLD * 2 : (size_t)D * MAXR * 4;
  constexpr size_t OT_BYTES = MF ? (size_t)ROWS * (MAXR + 1) * 4 : 4;
  __shared__ __attribute__((aligned(16))) unsigned char xs_raw[XS_BYTES];
  __shared__ __attribute__((aligned(16))) unsigned char fs_raw[FS_BYTES];
  __shared__ __attribute__((aligned(16))) unsigned char ot_raw[OT_BYTES];
  float(*xs)[D + 1] = (float(*)[D + 1])xs_raw;
  float* fs = (float*)fs_raw;
  uint16_t* fsp = (uint16_t*)fs_raw;  // [3][MAXR][FLD]
  float(*ot)[MAXR + 1] = (float(*)[MAXR + 1])ot_raw;
  const int bh = blockIdx.y, tid = threadIdx.x;
  const float* Fh = F + (size_t)bh * D * R;
  if constexpr (MF) {
    // eight loads in flight per thread, then their splits
    constexpr int PER = D * MAXR / 256, BATCH = 8;
    static_assert(PER % BATCH == 0, "F split batches");
    for (int i0 = 0; i0 < PER; i0 += BATCH) {
      float f[BATCH];
#pragma unroll
      for (int e = 0; e < BATCH; ++e) {
        const int i = (i0 + e) * 256 + tid;
        const int k = i / MAXR, c = i % MAXR;
        f[e] = c < R ? Fh[k * R + c] : 0.f;
      }
#pragma unroll
      for (int e = 0; e < BATCH; ++e) {
        const int i = (i0 + e) * 256 + tid;
        const int k = i / MAXR, c = i % MAXR;
        const uint16_t hi = __builtin_bit_cast(uint16_t, (__bf16)f[e]);
        const float r1 = f[e] - bf16_bits_to_f32(hi);
        const uint16_t mid = __builtin_bit_cast(uint16_t, (__bf16)r1);
        const uint16_t lo = __builtin_bit_cast(uint16_t, (__bf16)(r1 - bf16_bits_to_f32(mid)));
        fsp[(0 * MAXR + c) * FLD + k] = hi;
        fsp[(1 * MAXR + c) * FLD + k] = mid;
        fsp[(2 * MAXR + c) * FLD + k] = lo;
      }
    }
  } else if (R == MAXR) {
    for (int i = tid; i < D * MAXR / 4; i += 256) ((float4*)fs)[i] = ((const float4*)Fh)[i];
  } else {
    for (int i = tid; i < D * MAXR; i += 256) {
      const int k = i / MAXR, c = i % MAXR;
      fs[i] = c < R ? Fh[k * R + c] : 0.f;
    }
  }
  const int ty = tid >> 4, tx = tid & 15;
  const int nsrc = query ? g.G : 1;
  bool bad = false;
  // PROJ_CHUNKS chunks of 64 rows per block share the staged F
  for (int chunk = 0; chunk < PROJ_CHUNKS; ++chunk) {
    const int r0 = (blockIdx.x * PROJ_CHUNKS + chunk) * ROWS;
    if (r0 >= g.NV) break;
    if (chunk > 0) __syncthreads();
    float pooled[4][CPT];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int c = 0; c < CPT; ++c) pooled[u][c] = 0.f;
    for (int j = 0; j < nsrc; ++j) {
      const int64_t base = query ? q_base(g, bh, j) : kv_base(g, bh);
      float acc[4][CPT];
      if constexpr (MF) {
        __syncthreads();  // split F ready; the previous head's tile consumed
        const int wv = tid >> 6, lane = tid & 63, n = lane & 31, h = lane >> 5;
        for (int tile = wv; tile < 2 * NCT; tile += 4) {
          const int rt = tile & 1, ct = tile >> 1;
          const int row = r0 + rt * 32 + n;
          bf16x8 av[KS];
          if (row < g.NV) {
            const uint16_t* xr = (const uint16_t*)x + base + (int64_t)(g.ntext + row) * g.sn;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) av[ks] = __builtin_bit_cast(bf16x8, *(const uint4*)(xr + ks * 16 + h * 8));
          } else {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) av[ks] = __builtin_bit_cast(bf16x8, make_uint4(0u, 0u, 0u, 0u));
          }
          f32x16 S;
#pragma unroll
          for (int i = 0; i < 16; ++i) S[i] = 0.f;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
            for (int part = 0; part < 3; ++part) {
              const bf16x8 bv = __builtin_bit_cast(
                  bf16x8, *(const uint4*)(fsp + (size_t)(part * MAXR + ct * 32 + n) * FLD + ks * 16 + h * 8));
              S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[ks], bv, S, 0, 0, 0);
            }
          }
          // register i holds input row rt*32 + (i/4)*8 + h*4 + i%4, column ct*32 + n
#pragma unroll
          for (int i = 0; i < 16; ++i) ot[rt * 32 + (i / 4) * 8 + h * 4 + (i % 4)][ct * 32 + n] = S[i];
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int c = 0; c < CPT; ++c) acc[u][c] = ot[ty + 16 * u][tx * CPT + c];
      } else {
        if (j > 0) __syncthreads();
        for (int i = tid; i < ROWS * D / 8; i += 256) {
          const int rr = i / (D / 8), c8 = i % (D / 8);
          const int row = r0 + rr;
          float v[8];
          if (row < g.NV) {
            const int64_t off = base + (int64_t)(g.ntext + row) * g.sn + c8 * 8;
            if (g.bf16) {
              const uint4 u = *(const uint4*)((const uint16_t*)x + off);
              const uint32_t wds[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                v[2 * e] = __uint_as_float(wds[e] << 16);
                v[2 * e + 1] = __uint_as_float(wds[e] & 0xffff0000u);
              }
            } else {
              const float4 u0 = *(const float4*)((const float*)x + off);
              const float4 u1 = *(const float4*)((const float*)x + off + 4);
              v[0] = u0.x; v[1] = u0.y; v[2] = u0.z; v[3] = u0.w;
              v[4] = u1.x; v[5] = u1.y; v[6] = u1.z; v[7] = u1.w;
            }
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = 0.f;
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) xs[rr][c8 * 8 + e] = v[e];
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int c = 0; c < CPT; ++c) acc[u][c] = 0.f;
        for (int k = 0; k < D; ++k) {
          float xv[4], fv[CPT];
#pragma unroll
          for (int u = 0; u < 4; ++u) xv[u] = xs[ty + 16 * u][k];
#pragma unroll
          for (int c = 0; c < CPT; ++c) fv[c] = fs[k * MAXR + tx * CPT + c];
#pragma unroll
          for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int c = 0; c < CPT; ++c) acc[u][c] = fmaf(xv[u], fv[c], acc[u][c]);
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        float den = 1.f;
        if (rms) {
          float ss = 0.f;
#pragma unroll
          for (int c = 0; c < CPT; ++c) ss = fmaf(acc[u][c], acc[u][c], ss);
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) ss += __shfl_xor(ss, o);
          den = fmaxf(sqrtf(ss / (float)R), eps);
        }
        const float inv = 1.f / den;  // one division per row, not per element
#pragma unroll
        for (int c = 0; c < CPT; ++c) pooled[u][c] = fmaf(acc[u][c], inv, pooled[u][c]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int row = r0 + ty + 16 * u;
      // the k-means operands of the same coordinates: bf16 hi + lo halves
      // (zero-padded to RP) and the row norm (its error-bound input)
      float ssq = 0.f;
      float vv[CPT];
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        const int col = tx * CPT + c;
        vv[c] = col < R ? (nsrc == 1 ? pooled[u][c] : pooled[u][c] / (float)nsrc) : 0.f;
        ssq = fmaf(vv[c], vv[c], ssq);
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) ssq += __shfl_xor(ssq, o);
      if (row >= g.NV) continue;
      float* out = phi + ((size_t)bh * g.NV + row) * R;
      uint16_t* oh = xhi + ((size_t)bh * g.NV + row) * RP;
      uint16_t* ol = xlo + ((size_t)bh * g.NV + row) * RP;
      uint16_t hbs[CPT], lbs[CPT];
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        hbs[c] = __builtin_bit_cast(uint16_t, (__bf16)vv[c]);
        lbs[c] = __builtin_bit_cast(uint16_t, (__bf16)(vv[c] - bf16_bits_to_f32(hbs[c])));
        if (tx * CPT + c < R) bad |= !isfinite(vv[c]);
      }
      if (CPT == 4 && R % 4 == 0 && RP % 4 == 0) {
        // a thread's four columns as one 16-byte and two 8-byte stores (row
        // pitches of R floats and RP halves keep them aligned)
        const int col = tx * 4;
        if (col < R) *(float4*)(out + col) = make_float4(vv[0], vv[1], vv[2], vv[3]);
        if (col < RP) {
          *(uint2*)(oh + col) = make_uint2(hbs[0] | ((uint32_t)hbs[1] << 16), hbs[2] | ((uint32_t)hbs[3] << 16));
          *(uint2*)(ol + col) = make_uint2(lbs[0] | ((uint32_t)lbs[1] << 16), lbs[2] | ((uint32_t)lbs[3] << 16));
        }
      } else {
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
          const int col = tx * CPT + c;
          if (col < R) out[col] = vv[c];
          if (col < RP) {
            oh[col] = hbs[c];
            ol[col] = lbs[c];
          }
        }
      }
      if (tx == 0) xn[(size_t)bh * g.NV + row] = sqrtf(ssq) * 1.000001f;
    }
  }
  if (bad)
    atomicOr((unsigned long long*)&stats[(size_t)bh * 16 + ST_FLAGS],
             (unsigned long long)SPARSEPR_FLAG_NONFINITE_INPUT);
}

// ---------------------------------------------------------------------------
// k-means (Sec. 4.1: paired K/V groups from phi_K, query groups from phi_Q)
// and the stable group-major counting sort (Sec. 4.3) it maintains.
// ---------------------------------------------------------------------------

struct KmArgs {
  const float* pts;   // [BH][n][R] (k-means only)
  float* cent;        // [BH][C][R] (k-means only)
  int32_t* labels;    // [BH][N] in row order; the sorted rows start at row0
  int32_t* perm;      // [BH][N]
  int32_t* off;       // [BH][offstride]
  int32_t* blkhist;   // [BH][nblk][cmax]
  int32_t* changed;   // [BH][2][T+1]
  int n;              // rows taking part (sorted rows are row0 .. row0+n-1)
  int row0, N;
  int R, C;           // coordinate rank (at most the head dimension, 128), groups
  int offstride, nblk, cmax, sel, T;
  // MFMA screening of the assignment
  uint16_t* xhi;      // [BH][n][RP]
  uint16_t* xlo;
  float* xn;          // [BH][n]
  uint16_t* chi;      // [BH][CP][RP]
  uint16_t* clo;
  float* cu;          // [BH][CP]
  uint32_t* cn3;      // [BH][CP][2]: the norm's three bf16 parts (p0 | p1 << 16, p2)
  int32_t* fbcnt;     // [BH][2][T]: points left to the exact scan per assignment
  int RP, CP;         // rank padded to 16, groups padded to 32 (strides of the above)
  int warm;           // the first assignment starts from an earlier call's centroids
};

__device__ __forceinline__ int32_t* km_changed(const KmArgs& a, int bh) {
  return a.changed + (size_t)bh * 2 * (a.T + 1) + a.sel * (a.T + 1);
}

__device__ __forceinline__ bool km_skip(const KmArgs& a, int bh, int it) {
  return it >= 0 && km_changed(a, bh)[it] == 0;
}

// An assignment is skipped once the previous one changed no label: the
// centroids, and hence every later assignment, are then final.
__device__ __forceinline__ bool km_skip_assign(const KmArgs& a, int bh, int it) {
  return it > 0 && km_changed(a, bh)[it - 1] == 0;
}

__global__ void k_km_init(KmArgs a) {
  const int bh = blockIdx.y;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.C * a.R) return;
  const int b = i / a.R, c = i % a.R;
  // cold start from the strided points floor(b * n / C)
  const int src = (int)(((int64_t)b * a.n) / a.C);
  a.cent[(size_t)bh * a.C * a.R + i] = a.pts[((size_t)bh * a.n + src) * a.R + c];
}

// ---- MFMA-screened exact assignment -------------------------------------
// The assignment is defined by the exact float scores above.  To avoid
// scanning every centroid on the VALU, the scores are first estimated with
// bf16 MFMA on a three-term split (x = x_hi + x_lo, c = c_hi + c_lo;
// t~ = x_hi c_hi + x_hi c_lo + x_lo c_hi) and bounded.  The centroid operands
// hold -2c (a power-of-two scaling, exact in bf16) and one more K block adds
// the centroid norm in three bf16 parts against ones and, against a one,
// the point's shift s = bf16(|x|^2), last, so the accumulator ends with the
// whole score u - 2 x.c plus s and no VALU pass forms it.  The shift is the
// same for every centroid of a point, so it cancels in every comparison; it
// makes the smallest scores about |x - c|^2 instead of about -|x|^2, ten
// times smaller here, and with them the index packing's perturbation below.
// Bounds: the neglected lo*lo terms are below 3.1 * 2^-16 sum|x_k c_k|, the
// fp32 accumulation of the 3R exact bf16 products and the exact float chain
// each below gamma_{3R} and gamma_R times sum|x_k c_k| (both doubled by the
// factor 2), the norm block below five roundings of at most 2^-23 of
// u_max + 2|x| c_max + s plus the 2^-24 u left out of the split, and the
// exact score's own fma below 2^-24 (u_max + 2|x| c_max); with
// |sum| <= |x||c| every estimated score is within
// Delta = 1.62e-4 |x| c_max + 8.0e-7 (u_max + |x|^2) of the exact one plus s
// (Delta below carries another factor 2).  When the best estimate beats the
// runner-up by more than 2 Delta, its centroid is the exact argmin; when only
// the third is farther, the two candidates are rescored exactly; every other
// point is rescored against all centroids by its block at the end of the
// kernel.

__device__ __forceinline__ uint16_t bf16_rne_bits(float x) {
  return __builtin_bit_cast(uint16_t, (__bf16)x);
}

// u = p0 + p1 + p2 + e with |e| <= 2^-24 |u|: three round-to-nearest bf16
// parts, each subtraction exact; packed as (p0 | p1 << 16, p2), the operand
// of the assignment's norm step.
__device__ __forceinline__ uint2 norm_parts(float u) {
  const uint16_t p0 = bf16_rne_bits(u);
  const float r1 = u - bf16_bits_to_f32(p0);
  const uint16_t p1 = bf16_rne_bits(r1);
  const uint16_t p2 = bf16_rne_bits(r1 - bf16_bits_to_f32(p1));
  return make_uint2((uint32_t)p0 | ((uint32_t)p1 << 16), (uint32_t)p2);
}

// Points: the bf16 hi/lo split (padded to RP with zeros) and the norms are
// written by k_project together with the coordinates.

// Centroids: hi/lo split of -2c and exact squared norms (+inf for the padding rows).
__global__ __launch_bounds__(256) void k_km_prep_cent(KmArgs a, int it) {
  // 64 centroids per block, staged in LDS by coalesced loads; thread t < 64
  // forms the squared norm of centroid b0 + t as one fmaf chain in index
  // order, and the hi/lo operand rows go out as one contiguous block.
  __shared__ float cs[64][129];
  const int bh = blockIdx.y, tid = threadIdx.x;
  if (km_skip_assign(a, bh, it)) return;
  const int b0 = blockIdx.x * 64;
  if (b0 >= a.CP) return;
  const int R = a.R, RP = a.RP;
  const float* cb = a.cent + (size_t)bh * a.C * R;
  for (int e = tid; e < 64 * R; e += 256) {
    const int r = e / R, k = e - r * R;
    cs[r][k] = b0 + r < a.C ? cb[(size_t)(b0 + r) * R + k] : 0.f;
  }
  __syncthreads();
  if (tid < 64 && b0 + tid < a.CP) {
    float u = INFINITY;
    if (b0 + tid < a.C) {
      u = 0.f;
      for (int k = 0; k < R; ++k) u = fmaf(cs[tid][k], cs[tid][k], u);
    }
    a.cu[(size_t)bh * a.CP + b0 + tid] = u;
    // padding centroids get a huge finite norm in the MFMA step: their
    // scores stay finite (an index packed into +inf would make a NaN)
    ((uint2*)a.cn3)[(size_t)bh * a.CP + b0 + tid] = norm_parts(b0 + tid < a.C ? u : 3.0e38f);
  }
  uint16_t* hi = a.chi + ((size_t)bh * a.CP + b0) * RP;
  uint16_t* lo = a.clo + ((size_t)bh * a.CP + b0) * RP;
  const int rows = min(64, a.CP - b0);
  for (int e = tid; e < rows * RP; e += 256) {
    const int r = e / RP, k = e - r * RP;
    const float v = (b0 + r < a.C && k < R) ? -2.f * cs[r][k] : 0.f;
    const uint16_t h = bf16_rne_bits(v);
    hi[e] = h;
    lo[e] = bf16_rne_bits(v - bf16_bits_to_f32(h));
  }
}

// The sorted-triple update on packed (score, index) values.  The packed
// values come from integer bit operations, so the compiler would quiet each
// one with an extra v_max before a float min or med3 (IEEE mode); the packed
// scores are finite, so the plain instructions are issued directly.
__device__ __forceinline__ float med3_packed(float x, float y, float z) {
  float d;
  asm("v_med3_f32 %0, %1, %2, %3" : "=v"(d) : "v"(x), "v"(y), "v"(z));
  return d;
}
__device__ __forceinline__ float min_packed(float x, float y) {
  float d;
  asm("v_min_f32 %0, %1, %2" : "=v"(d) : "v"(x), "v"(y));
  return d;
}

// s_waitcnt vmcnt(n) for a wave-uniform n below 7 (gfx9 encoding: vmcnt in
// bits 3:0, expcnt and lgkmcnt left at their maxima); larger n waits for all
__device__ __forceinline__ void km_wait_vm(int n) {
  switch (n) {
    case 0: __builtin_amdgcn_s_waitcnt(0x3f70); break;
    case 1: __builtin_amdgcn_s_waitcnt(0x3f71); break;
    case 2: __builtin_amdgcn_s_waitcnt(0x3f72); break;
    case 3: __builtin_amdgcn_s_waitcnt(0x3f73); break;
    case 4: __builtin_amdgcn_s_waitcnt(0x3f74); break;
    case 5: __builtin_amdgcn_s_waitcnt(0x3f75); break;
    case 6: __builtin_amdgcn_s_waitcnt(0x3f76); break;
    default: __builtin_amdgcn_s_waitcnt(0x3f70); break;
  }
}
// Direct global -> LDS copies for the centroid tiles: lane l's 16 (or 4)
// bytes land at lds + 16 l (4 l), with lds the same for the whole wave; the
// compiler does not see these loads, so the kernel orders them with explicit
// vmcnt waits.  No other code in this file uses M0.
__device__ __forceinline__ void km_g2lds16(const void* src, uint32_t lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(m0)
               : "memory");
}
__device__ __forceinline__ void km_g2lds4(const void* src, uint32_t lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :
               : "v"(src), "s"(m0)
               : "memory");
}

// Screening: a block of 4 waves takes 256 points, 64 per wave as two sets
// of 32 (the N side of v_mfma_f32_32x32x16_bf16), against 32-centroid tiles
// in LDS (the M side); every centroid fragment read from LDS feeds both
// sets.  The tiles (hi and lo rows, padded, and the norms' bf16 parts) are
// in a ring of three LDS buffers filled by direct global -> LDS copies
// issued two tiles ahead, one barrier per tile.  Lane (n, h) ends with the
// three best estimates of point n of each set over half of the centroids; the halves
// are merged with one exchange, and lane h then decides set h's point.  The
// second launch bound (three blocks per CU up to rank 64, two above) caps
// the registers at 168 / 256, so the accumulators stay in VGPRs that the
// VALU reads directly.
template <int RP>
__global__ __launch_bounds__(256, RP <= 64 ? 3 : 2) void k_km_assign_mfma(KmArgs a, int it) {
  constexpr int KS = RP / 16;
  constexpr int LD = RP + 8;            // padded LDS row (bf16)
  constexpr int ARR = 32 * LD * 2;      // bytes of one array (hi or lo) of a tile
  constexpr int PPR = LD / 8;           // 16-byte pieces per padded row
  constexpr int NPIECE = 2 * ARR / 16;  // pieces of hi + lo
  constexpr int NINST = (NPIECE + 63) / 64;
  constexpr int TILE = 2 * ARR + 256;   // + the 32 norms' parts
  constexpr int NPS = 2;                // sets of 32 points per wave
  __shared__ __attribute__((aligned(1024))) unsigned char tiles[3][TILE];
  __shared__ int sfb[256];  // the block's points left to the exact scan
  __shared__ int nfb;
  __shared__ __attribute__((aligned(16))) float xs[RP];
  __shared__ float rsb[4];
  __shared__ int rsi[4];
  const int bh = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (km_skip_assign(a, bh, it)) return;
  if (tid == 0) nfb = 0;  // ordered by the tile loop's barriers
  const int n = lane & 31, h = lane >> 5;
  const int jbase = blockIdx.x * (128 * NPS) + wv * (32 * NPS);
  // Points are taken in the order of the previous assignment's counting
  // sort (group-major, so a wave's points mostly share a centroid); the
  // first assignment takes them in row order.  Slot s holds row
  // perm[s] - row0 of this k-means.
  const int32_t* prm = it > 0 ? a.perm + (size_t)bh * a.N : nullptr;
  auto row_of = [&](int s) { return prm ? prm[s] - a.row0 : s; };
  bf16x8 bhi[NPS][KS], blo[NPS][KS];
#pragma unroll
  for (int ps = 0; ps < NPS; ++ps) {
    const int jc = row_of(min(jbase + ps * 32 + n, a.n - 1));
    const uint16_t* xh = a.xhi + ((size_t)bh * a.n + jc) * RP;
    const uint16_t* xl = a.xlo + ((size_t)bh * a.n + jc) * RP;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      bhi[ps][ks] = __builtin_bit_cast(bf16x8, *(const uint4*)(xh + ks * 16 + h * 8));
      blo[ps][ks] = __builtin_bit_cast(bf16x8, *(const uint4*)(xl + ks * 16 + h * 8));
    }
  }
  // Largest centroid squared norm of the head (for the error bound), the
  // same value in every wave.
  float umax = 0.f;
  const float* cu = a.cu + (size_t)bh * a.CP;
  for (int b0 = 0; b0 < a.C; b0 += 64 * 8) {  // eight loads in flight per lane
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = b0 + e * 64 + lane < a.C ? cu[b0 + e * 64 + lane] : 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) umax = fmaxf(umax, v[e]);
  }
  umax = wave_max(umax);
  // Three smallest estimates per point, ascending, each with its centroid
  // index in the low IB mantissa bits (C <= 2^IB).  Replacing those bits
  // moves a value by at most 2^(IB-23) of its magnitude, which the decision
  // below adds to the error bound.  Keeping (value, index) in one float lets
  // min / med3 maintain the sorted triple in three instructions per score.
  // The start value is finite and above every score.
  const int ib = 32 - __clz(a.CP - 1);
  const uint32_t keep = ~((1u << ib) - 1u);
  const float ek = ldexpf(1.f, ib - 22);
  float t1[NPS], t2[NPS], t3[NPS];
#pragma unroll
  for (int ps = 0; ps < NPS; ++ps) t1[ps] = t2[ps] = t3[ps] = 3.4e38f;
  // Skipping tiles.  Let e be a point's smallest packed estimate and M twice
  // the error bound of its scores (mrg below).  The decision only looks at
  // estimates p with p - e <= M + ek (|e| + |p|); a larger one can stay out
  // of the triple without changing it (p - ek |p| grows with p, and an entry
  // left at the start value passes the same test).  For any U >= e every such
  // p has a raw score at most
  //   L(U) = U + M + 2 ek |U| + ek |U|          when U + M + 2 ek |U| <= 0
  //   L(U) = U + M + 5 ek (|U| + M) + 2^-20 ... otherwise,
  // both growing with U (the packing moves a raw score by at most ek/2 of
  // it, and the small absolute terms cover the rounding of L).  U is the
  // smallest estimate folded so far over both halves of the centroids, so a
  // wave folds a tile into set ps's triples only when some lane has a raw
  // score at or below L(U) (or a NaN); until the first fold U is infinite.
  float mrg[NPS], thr[NPS];
  // the norm block's point operand: ones at k = 0, 1, 2 and the shift at
  // k = 3 (held by the h = 0 lanes), zeros elsewhere, so the centroid lanes'
  // k >= 4 entries drop out
  bf16x8 bnorm[NPS];
#pragma unroll
  for (int ps = 0; ps < NPS; ++ps) {
    const float xn = a.xn[(size_t)bh * a.n + row_of(min(jbase + ps * 32 + n, a.n - 1))];
    mrg[ps] = 2.f * (3.24e-4f * xn * sqrtf(umax) * 1.000001f + 8.0e-7f * (umax + xn * xn));
    thr[ps] = INFINITY;
    const uint32_t sh = bf16_rne_bits(xn * xn);
    bnorm[ps] = __builtin_bit_cast(
        bf16x8, h ? make_uint4(0u, 0u, 0u, 0u) : make_uint4(0x3F803F80u, 0x3F80u | (sh << 16), 0u, 0u));
  }
  auto bound = [&](int ps) {
    const float u = fminf(t1[ps], __shfl_xor(t1[ps], 32));
    const float au = fabsf(u), m = mrg[ps];
    const float lp = u + fmaf(2.f * ek, au, m);
    const float slack = 0x1p-20f * (au + m);
    return lp <= 0.f ? lp + fmaf(ek, au, slack) : u + m + fmaf(5.f * ek, au + m, slack);
  };
  const uint16_t* chi = a.chi + (size_t)bh * a.CP * RP;
  const uint16_t* clo = a.clo + (size_t)bh * a.CP * RP;
  const uint32_t* cn3 = a.cn3 + (size_t)bh * a.CP * 2;
  const uint32_t lds0 = (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)&tiles[0][0];
  // the copies of tile c0 into buffer b: piece p = inst * 64 + lane lands at
  // byte 16 p of the buffer (row p / PPR of hi, then of lo; the padding
  // pieces of a row fetch its first piece), then the norms' parts
  auto issue = [&](int c0, int b) {
    const uint32_t base = lds0 + (uint32_t)(b * TILE);
#pragma unroll
    for (int i0 = 0; i0 < NINST; i0 += 4) {
      const int inst = i0 + wv;
      const int p = inst * 64 + lane;
      if (inst < NINST && p < NPIECE) {
        const int arr = p >= NPIECE / 2;
        const int q = p - arr * (NPIECE / 2);
        const int r = q / PPR, c8 = q - (q / PPR) * PPR;
        const uint16_t* src = (arr ? clo : chi) + (size_t)(c0 + r) * RP + (c8 < RP / 8 ? c8 : 0) * 8;
        km_g2lds16(src, base + (uint32_t)(inst * 1024));
      }
    }
    if (wv == 0) km_g2lds4(cn3 + (size_t)c0 * 2 + lane, base + (uint32_t)(2 * ARR));
  };
  // s_waitcnt immediate (gfx9 encoding) waiting for vmcnt(0) only
  constexpr int kWaitVm0 = 0x3f70;
  // the point operands and the norms above are ordinary loads: wait for
  // them once here, so no later wait of the compiler's covers the copies
  // The block sweeps the tiles from the one holding its first point's
  // previous label (that of the earlier call in a warm first assignment; in
  // a cold one, the start centroid of a nearby row), wrapping around: the
  // running minima are tight early.  Any start gives the same result.
  int32_t* lab = a.labels + (size_t)bh * a.N + a.row0;
  const int jb0 = blockIdx.x * (128 * NPS);
  int cst = (it > 0 || a.warm) ? lab[row_of(jb0)] : (int)(((int64_t)jb0 * a.C) / a.n);
  cst = __builtin_amdgcn_readfirstlane(min(max(cst, 0), a.C - 1) & ~31);
  // copy instructions this wave issues per tile (vmcnt counts them in order)
  const int ncopy = (NINST - wv + 3) / 4 + (wv == 0);
  // three buffers: the copies run two tiles ahead of the MFMAs
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  issue(cst, 0);
  const int cnx0 = cst + 32 < a.CP ? cst + 32 : 0;
  if (32 < a.CP) issue(cnx0, 1);
  int buf = 0, c0 = cst;
  for (int t = 0; t < a.CP; t += 32, buf = buf == 2 ? 0 : buf + 1) {
    // this wave's copies of the tile have landed (only the next tile's may
    // still be in flight); after the barrier every wave's have, and every
    // wave is done with the previous tile's buffer, which takes tile t + 2
    if (t + 32 < a.CP)
      km_wait_vm(ncopy);
    else
      __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();
    const int cnext = c0 + 32 < a.CP ? c0 + 32 : 0;
    const int cn2 = cnext + 32 < a.CP ? cnext + 32 : 0;
    if (t + 64 < a.CP) issue(cn2, buf == 0 ? 2 : buf - 1);
    const unsigned char* tb = &tiles[buf][0];
    const uint16_t* shi = (const uint16_t*)tb;
    const uint16_t* slo = (const uint16_t*)(tb + ARR);
    const uint32_t* su3 = (const uint32_t*)(tb + 2 * ARR);
    bf16x8 ah[KS], al[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      ah[ks] = __builtin_bit_cast(bf16x8, *(const uint4*)(shi + n * LD + ks * 16 + h * 8));
      al[ks] = __builtin_bit_cast(bf16x8, *(const uint4*)(slo + n * LD + ks * 16 + h * 8));
    }
    const uint2 w = *(const uint2*)&su3[2 * n];
    const bf16x8 an = __builtin_bit_cast(bf16x8, make_uint4(w.x, w.y | 0x3F800000u, 0u, 0u));
    // scores S = u - 2 x.c, the norm block last
    f32x16 S[NPS];
#pragma unroll
    for (int ps = 0; ps < NPS; ++ps)
#pragma unroll
      for (int i = 0; i < 16; ++i) S[ps][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int ps = 0; ps < NPS; ++ps) {
        S[ps] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[ks], bhi[ps][ks], S[ps], 0, 0, 0);
        S[ps] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[ks], blo[ps][ks], S[ps], 0, 0, 0);
        S[ps] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[ks], bhi[ps][ks], S[ps], 0, 0, 0);
      }
#pragma unroll
    for (int ps = 0; ps < NPS; ++ps)
      S[ps] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(an, bnorm[ps], S[ps], 0, 0, 0);
#pragma unroll
    for (int ps = 0; ps < NPS; ++ps) {
      // the lane's smallest raw score of the tile (NaN only if all are);
      // plain code, so the compiler keeps the wait states an MFMA result
      // needs before a VALU instruction reads it
      float m = fminf(fminf(S[ps][0], S[ps][1]), S[ps][2]);
#pragma unroll
      for (int i = 3; i < 15; i += 2) m = fminf(fminf(m, S[ps][i]), S[ps][i + 1]);
      m = fminf(m, S[ps][15]);
      if (__builtin_amdgcn_ballot_w64(!(m > thr[ps])) == 0) continue;
      // fold the tile into set ps's sorted triples
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        // centroid index of accumulator register i: c0 + (i/4)*8 + h*4 + i%4
        const uint32_t idx = (uint32_t)(c0 + h * 4) + (uint32_t)((i >> 2) * 8 + (i & 3));
        const float pk = __uint_as_float((__float_as_uint(S[ps][i]) & keep) | idx);
        const float n3 = med3_packed(t2[ps], t3[ps], pk);
        const float n2 = med3_packed(t1[ps], t2[ps], pk);
        t1[ps] = min_packed(t1[ps], pk);
        t2[ps] = n2;
        t3[ps] = n3;
      }
      thr[ps] = bound(ps);
    }
    c0 = cnext;
  }
  // merge with the other half of the centroids (lane l ^ 32, same points)
#pragma unroll
  for (int ps = 0; ps < NPS; ++ps) {
    const float ov[3] = {__shfl_xor(t1[ps], 32), __shfl_xor(t2[ps], 32), __shfl_xor(t3[ps], 32)};
#pragma unroll
    for (int e = 0; e < 3; ++e) {
      const float n3 = med3_packed(t2[ps], t3[ps], ov[e]);
      const float n2 = med3_packed(t1[ps], t2[ps], ov[e]);
      t1[ps] = min_packed(t1[ps], ov[e]);
      t2[ps] = n2;
      t3[ps] = n3;
    }
  }
  // lane (n, h) decides point n of set h (slot j, row jr)
  const int j = jbase + h * 32 + n;
  if (j < a.n) {
    const int jr = row_of(j);
    const float T1 = h ? t1[1] : t1[0], T2 = h ? t2[1] : t2[0], T3 = h ? t3[1] : t3[0];
    // the packed indices are below C whenever a real centroid has a finite
    // score; non-finite coordinates (flagged by k_project) could leave a
    // padding index or NaN bits, so the indices are clamped into range
    const int i1 = min((int)(__float_as_uint(T1) & ~keep), a.C - 1);
    const int i2 = min((int)(__float_as_uint(T2) & ~keep), a.C - 1);
    const float delta = 0.5f * (h ? mrg[1] : mrg[0]);
    int label = -1;
    if (T2 - T1 > 2.f * delta + ek * (fabsf(T1) + fabsf(T2))) {
      label = i1;  // unique candidate: the exact argmin
    } else if (T3 - T1 > 2.f * delta + ek * (fabsf(T1) + fabsf(T3))) {
      // exactly two candidates: rescore both with the defining float score
      const float* xp = a.pts + ((size_t)bh * a.n + jr) * a.R;
      const float* c1 = a.cent + ((size_t)bh * a.C + i1) * a.R;
      const float* c2 = a.cent + ((size_t)bh * a.C + i2) * a.R;
      float d1 = 0.f, d2 = 0.f;
      if ((a.R & 3) == 0) {
        for (int k = 0; k < a.R; k += 4) {
          const float4 x4 = *(const float4*)(xp + k);
          const float4 p4 = *(const float4*)(c1 + k), q4 = *(const float4*)(c2 + k);
          d1 = fmaf(x4.x, p4.x, d1);
          d2 = fmaf(x4.x, q4.x, d2);
          d1 = fmaf(x4.y, p4.y, d1);
          d2 = fmaf(x4.y, q4.y, d2);
          d1 = fmaf(x4.z, p4.z, d1);
          d2 = fmaf(x4.z, q4.z, d2);
          d1 = fmaf(x4.w, p4.w, d1);
          d2 = fmaf(x4.w, q4.w, d2);
        }
      } else {
        for (int k = 0; k < a.R; ++k) {
          const float xk = xp[k];
          d1 = fmaf(xk, c1[k], d1);
          d2 = fmaf(xk, c2[k], d2);
        }
      }
      const float s1 = fmaf(-2.f, d1, cu[i1]), s2 = fmaf(-2.f, d2, cu[i2]);
      label = (s2 < s1 || (s2 == s1 && i2 < i1)) ? i2 : i1;
    } else {
      // more than two candidates: the block's exact scan below
      sfb[atomicAdd(&nfb, 1)] = jr;
      atomicAdd(a.fbcnt + (size_t)bh * 2 * a.T + a.sel * a.T + it, 1);
    }
    if (label >= 0) {
      const int old = lab[jr];
      lab[jr] = label;
      if (it > 0 && old != label) atomicAdd(&km_changed(a, bh)[it], 1);
    }
  }
  __syncthreads();
  // Exact scan (the defining float score) of the block's undecided points:
  // the point sits in LDS, every thread scores a strided subset of the
  // centroids with the float chain, and the block keeps the smallest score,
  // lowest index among equal scores.
  const int nundecided = nfb;
  const int R = a.R;
  for (int e = 0; e < nundecided; ++e) {
    const int jj = sfb[e];
    if (tid < RP) xs[tid] = tid < R ? a.pts[((size_t)bh * a.n + jj) * R + tid] : 0.f;
    __syncthreads();
    float best = INFINITY;
    int bi = 0x7fffffff;
    for (int b = tid; b < a.C; b += 256) {  // ascending within the thread
      const float* cb = a.cent + ((size_t)bh * a.C + b) * R;
      float t = 0.f;
      if ((R & 3) == 0) {
        // sixteen of the centroid's 16-byte loads in flight ahead of the chain
#pragma unroll 16
        for (int k = 0; k < R; k += 4) {
          const float4 c4 = *(const float4*)(cb + k);
          t = fmaf(xs[k], c4.x, t);
          t = fmaf(xs[k + 1], c4.y, t);
          t = fmaf(xs[k + 2], c4.z, t);
          t = fmaf(xs[k + 3], c4.w, t);
        }
      } else {
        for (int k = 0; k < R; ++k) t = fmaf(xs[k], cb[k], t);
      }
      const float sc = fmaf(-2.f, t, cu[b]);
      if (sc < best) {
        best = sc;
        bi = b;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ob = __shfl_xor(best, o);
      const int oi = __shfl_xor(bi, o);
      if (ob < best || (ob == best && oi < bi)) {
        best = ob;
        bi = oi;
      }
    }
    if (lane == 0) {
      rsb[wv] = best;
      rsi[wv] = bi;
    }
    __syncthreads();
    if (tid == 0) {
      for (int w2 = 1; w2 < 4; ++w2)
        if (rsb[w2] < best || (rsb[w2] == best && rsi[w2] < bi)) {
          best = rsb[w2];
          bi = rsi[w2];
        }
      if (bi >= a.C) bi = 0;  // no finite score (non-finite input, flagged): keep labels in range
      const int old = lab[jj];
      lab[jj] = bi;
      if (it > 0 && old != bi) atomicAdd(&km_changed(a, bh)[it], 1);
    }
    __syncthreads();  // xs and the reduction slots are reused by the next point
  }
}

// Counting sort, pass 1: per-block label histograms.
__global__ __launch_bounds__(256) void k_sort_hist(KmArgs a, int it) {
  extern __shared__ int hs[];
  const int bh = blockIdx.y, blk = blockIdx.x, tid = threadIdx.x;
  if (km_skip(a, bh, it)) return;
  for (int b = tid; b < a.C; b += 256) hs[b] = 0;
  __syncthreads();
  const int32_t* lab = a.labels + (size_t)bh * a.N + a.row0;
  const int j0 = blk * kSortBlock, j1 = min(a.n, j0 + kSortBlock);
  for (int j = j0 + tid; j < j1; j += 256) atomicAdd(&hs[lab[j]], 1);
  __syncthreads();
  int32_t* out = a.blkhist + ((size_t)bh * a.nblk + blk) * a.cmax;
  for (int b = tid; b < a.C; b += 256) out[b] = hs[b];
}

// Counting sort, pass 2: per-label running offsets over the blocks, then the
// exclusive scan over labels gives the group offsets.
__global__ __launch_bounds__(1024) void k_sort_scan(KmArgs a, int it) {
  extern __shared__ int cnt[];  // C + 1 ints, then 17 ints of scan scratch
  const int bh = blockIdx.x, tid = threadIdx.x;
  if (km_skip(a, bh, it)) return;
  int32_t* hist = a.blkhist + (size_t)bh * a.nblk * a.cmax;
  for (int b = tid; b < a.C; b += 1024) {
    // the block counts are read 16 at a time ahead of their running sums
    int run = 0;
    for (int k0 = 0; k0 < a.nblk; k0 += 16) {
      int v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = k0 + u < a.nblk ? hist[(size_t)(k0 + u) * a.cmax + b] : 0;
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        if (k0 + u < a.nblk) {
          hist[(size_t)(k0 + u) * a.cmax + b] = run;
          run += v[u];
        }
      }
    }
    cnt[b] = run;
  }
  __syncthreads();
  const int total = block_exclusive_scan(cnt, a.C, cnt + a.C + 1);
  int32_t* off = a.off + (size_t)bh * a.offstride;
  for (int b = tid; b < a.C; b += 1024) off[b] = cnt[b];
  if (tid == 0) off[a.C] = total;
}

// Counting sort, pass 3: stable scatter.  A block of 4 waves takes the
// block's rows; wave w owns rows [j0 + 256 w, j0 + 256 (w + 1)).  Each wave
// counts its labels, the per-label slots of the waves follow by a prefix over
// the waves, and every wave then walks its rows in order, 64 at a time: each
// lane reads its label's next slot; the slice's labels go through LDS, every
// lane marks the lanes holding its label, its stable rank is the number of
// them before it, and the lane with the last rank advances the slot.
constexpr int kScatterWaves = 4;
constexpr int kScatterRows = kSortBlock / kScatterWaves;  // rows per wave

__host__ __device__ __forceinline__ int sort_scatter_cstride(int C) { return (C + 3) & ~3; }

__global__ __launch_bounds__(256) void k_sort_scatter(KmArgs a, int it) {
  // [kScatterWaves][cs] per-wave counts, then slots; [kScatterWaves][64] slice labels
  extern __shared__ __attribute__((aligned(16))) int sm[];
  const int cs = sort_scatter_cstride(a.C);
  const int bh = blockIdx.y, blk = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (km_skip(a, bh, it)) return;
  int* pos = sm + wv * cs;
  int* sl = sm + kScatterWaves * cs + wv * 64;
  const int32_t* lab = a.labels + (size_t)bh * a.N + a.row0;
  const int j0 = blk * kSortBlock + wv * kScatterRows;
  const int j1 = min(a.n, j0 + kScatterRows);
  for (int b = lane; b < a.C; b += 64) pos[b] = 0;
  // the wave's own counts (its LDS accesses complete in program order)
  for (int j = j0 + lane; j < j1; j += 64) atomicAdd(&pos[lab[j]], 1);
  __syncthreads();
  // slots: the block's start of each label plus the counts of earlier waves
  const int32_t* hist = a.blkhist + ((size_t)bh * a.nblk + blk) * a.cmax;
  const int32_t* off = a.off + (size_t)bh * a.offstride;
  for (int b = tid; b < a.C; b += 256) {
    int run = off[b] + hist[b];
#pragma unroll
    for (int w = 0; w < kScatterWaves; ++w) {
      const int c = sm[w * cs + b];
      sm[w * cs + b] = run;
      run += c;
    }
  }
  __syncthreads();
  int32_t* perm = a.perm + (size_t)bh * a.N;
  const uint32_t below_lo = lane >= 32 ? 0xffffffffu : (1u << lane) - 1u;
  const uint32_t below_hi = lane <= 32 ? 0u : (1u << (lane - 32)) - 1u;
  for (int s = j0; s < j1; s += 64) {
    const int j = s + lane;
    const bool valid = j < j1;
    const int L = valid ? lab[j] : -1 - lane;  // invalid lanes match nothing
    const int base = valid ? pos[L] : 0;
    sl[lane] = L;
    uint32_t mlo = 0u, mhi = 0u;  // lanes holding this lane's label
#pragma unroll
    for (int k4 = 0; k4 < 16; ++k4) {
      const int4 q = *(const int4*)&sl[4 * k4];
      const int qv[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = 4 * k4 + e;
        if (k < 32)
          mlo |= (qv[e] == L ? 1u : 0u) << k;
        else
          mhi |= (qv[e] == L ? 1u : 0u) << (k - 32);
      }
    }
    const int rank = __popc(mlo & below_lo) + __popc(mhi & below_hi);
    const int cnt = __popc(mlo) + __popc(mhi);
    if (valid) {
      perm[base + rank] = a.row0 + j;
      if (rank == cnt - 1) pos[L] = base + cnt;
    }
  }
}

// Centroid update: per group, double sums of the members' coordinates in
// ascending row order (the stable permutation order) / count, rounded to
// float; an empty group keeps its centroid (and its assignment operands).
// One wave per group: the members' rows are fetched 64 at a time (lane i
// holds member m0 + i) and exchanged by readlane; lane l owns coordinates l
// and l + 64, whose values are loaded sixteen members at a time and added in
// ascending member order.
__global__ __launch_bounds__(256) void k_km_update(KmArgs a, int it) {
  const int bh = blockIdx.y, wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (km_changed(a, bh)[it] == 0) return;
  const int b = blockIdx.x * 4 + wv;
  if (b >= a.C) return;
  const int32_t* off = a.off + (size_t)bh * a.offstride;
  const int32_t* perm = a.perm + (size_t)bh * a.N;
  const int s0 = __builtin_amdgcn_readfirstlane(off[b]), s1 = __builtin_amdgcn_readfirstlane(off[b + 1]);
  if (s1 == s0) return;
  const float* pts = a.pts + (size_t)bh * a.n * a.R;
  const int R = a.R;
  // loads are unconditional (columns clamped into the row); lanes past R
  // drop their sums
  const int k0 = min(lane, R - 1), k1 = min(lane + 64, R - 1);
  double sum0 = 0.0, sum1 = 0.0;
  auto members = [&](auto two) {
    constexpr bool TWO = decltype(two)::value;
    for (int m0 = s0; m0 < s1; m0 += 64) {
      const int cnt = min(64, s1 - m0);
      const int myrow = lane < cnt ? perm[m0 + lane] - a.row0 : 0;
      // 16 members' loads in flight; past the last member the loads read a
      // member row again and their values are not added
      for (int u = 0; u < cnt; u += 16) {
        float v0[16], v1[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float* pr = pts + (size_t)__builtin_amdgcn_readlane(myrow, (u + e) & 63) * R;
          v0[e] = pr[k0];
          if constexpr (TWO) v1[e] = pr[k1];
        }
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (u + e < cnt) {
            sum0 += (double)v0[e];
            if constexpr (TWO) sum1 += (double)v1[e];
          }
      }
    }
  };
  if (R > 64)
    members(std::true_type{});
  else
    members(std::false_type{});
  const double inv = (double)(s1 - s0);
  float* c = a.cent + ((size_t)bh * a.C + b) * R;
  const float v0 = (float)(sum0 / inv), v1 = (float)(sum1 / inv);
  if (lane < R) c[lane] = v0;
  if (lane + 64 < R) c[lane + 64] = v1;
  // The next assignment's operands of this centroid (as k_km_prep_cent
  // forms them): the hi/lo split of -2c and the squared norm, one fmaf chain
  // in coordinate order through LDS, with its three bf16 parts.
  __shared__ float cw[4][128];
  const int RP = a.RP;
  uint16_t* hi = a.chi + ((size_t)bh * a.CP + b) * RP;
  uint16_t* lo = a.clo + ((size_t)bh * a.CP + b) * RP;
  if (lane < R) {
    cw[wv][lane] = v0;
    const uint16_t h = bf16_rne_bits(-2.f * v0);
    hi[lane] = h;
    lo[lane] = bf16_rne_bits(-2.f * v0 - bf16_bits_to_f32(h));
  }
  if (lane + 64 < R) {
    cw[wv][lane + 64] = v1;
    const uint16_t h = bf16_rne_bits(-2.f * v1);
    hi[lane + 64] = h;
    lo[lane + 64] = bf16_rne_bits(-2.f * v1 - bf16_bits_to_f32(h));
  }
  // one wave: its LDS writes land before its reads below
  if (lane == 0) {
    float u = 0.f;
    for (int k = 0; k < R; ++k) u = fmaf(cw[wv][k], cw[wv][k], u);
    a.cu[(size_t)bh * a.CP + b] = u;
    ((uint2*)a.cn3)[(size_t)bh * a.CP + b] = norm_parts(u);
  }
}

// The dense-prefix rows (before row0) form the extra last group: label C and
// the last permutation slots, in row order.
__global__ void k_prefix_group(KmArgs a) {
  const int bh = blockIdx.y;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < a.row0) {
    a.labels[(size_t)bh * a.N + i] = a.C;
    a.perm[(size_t)bh * a.N + a.n + i] = i;
  }
  if (i == 0 && a.row0 > 0) a.off[(size_t)bh * a.offstride + a.C + 1] = a.N;
}

// ---------------------------------------------------------------------------
// Group means in the input space (kbar, qbar): double sums in ascending row
// order / count, rounded to float; empty groups get 0.  One wave per group.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void k_group_mean(const void* x, Geom g, const int32_t* perm,
                                                    const int32_t* off, int C, int offstride,
                                                    float* mean, int query) {
  // One wave per group; lane l owns channels 2l and 2l + 1.  The members'
  // rows are fetched 64 at a time (lane i holds member m0 + i), their values
  // loaded eight at a time and added in ascending member order.  Key means
  // come from the K/V head; query means (`query`) are pooled over its G query
  // heads, head by head.
  const int bh = blockIdx.y, wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + wv;
  if (b >= C) return;
  const int nsrc = query ? g.G : 1;
  const int32_t* o = off + (size_t)bh * offstride;
  const int32_t* p = perm + (size_t)bh * g.N;
  const int s0 = __builtin_amdgcn_readfirstlane(o[b]), s1 = __builtin_amdgcn_readfirstlane(o[b + 1]);
  // d <= 128: every channel pair has a lane; all lanes run the member loop
  // (the row indices are exchanged with readlane), idle lanes only skip the adds
  const int c = 2 * lane;
  const bool cin = c < g.d;
  double s0d = 0.0, s1d = 0.0;
  // loads are unconditional (lanes past d read channel 0 and drop their
  // sums) and the dtype is decided outside the member loop
  const int cl = cin ? c : 0;
  auto members = [&](auto bfv) {
    constexpr bool BF = decltype(bfv)::value;
    auto ld2 = [&](int64_t base, int row) -> float2 {
      const int64_t idx = base + (int64_t)row * g.sn + cl;
      if constexpr (BF) {
        const uint32_t u = *(const uint32_t*)((const uint16_t*)x + idx);
        return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
      } else {
        return *(const float2*)((const float*)x + idx);
      }
    };
    for (int j = 0; j < nsrc; ++j) {
      const int64_t base = query ? q_base(g, bh, j) : kv_base(g, bh);
      for (int m0 = s0; m0 < s1; m0 += 64) {
        const int cm = min(64, s1 - m0);
        const int pv = lane < cm ? p[m0 + lane] : 0;
        int i = 0;
        for (; i + 8 <= cm; i += 8) {
          float2 v[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) v[u] = ld2(base, __builtin_amdgcn_readlane(pv, i + u));
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            s0d += (double)v[u].x;
            s1d += (double)v[u].y;
          }
        }
        for (; i < cm; ++i) {
          const float2 v = ld2(base, __builtin_amdgcn_readlane(pv, i));
          s0d += (double)v.x;
          s1d += (double)v.y;
        }
      }
    }
  };
  if (g.bf16)
    members(std::true_type{});
  else
    members(std::false_type{});
  if (!cin) return;
  const double n = (double)(s1 - s0) * (double)nsrc;
  float* dst = mean + ((size_t)bh * C + b) * g.d + c;
  dst[0] = (s1 > s0) ? (float)(s0d / n) : 0.f;
  dst[1] = (s1 > s0) ? (float)(s1d / n) : 0.f;
}

// Query-response metric M_Q = Kt^T Kt / (C_k^+ d) from the nonempty key-space
// group means centred by their uniform mean, equal weights
// (App. B.2 eq. app_query_metric).  One sweep over the groups: with d_b the
// nonempty means shifted by the first nonempty one (s) and S = sum_b d_b,
//   sum_b (x_b - mu)(x_b - mu)^T = sum_b d_b d_b^T - S S^T / C_k^+,
// since mu - s = S / C_k^+; the shift keeps both terms of the size of the
// spread, so the fp64 difference loses no digits to a large common mean.
template <int D>
__global__ __launch_bounds__(256) void k_query_metric(const float* kbar, const int32_t* offk,
                                                      Geom g, double* gram) {
  // Block (x, bh) computes output rows [RB x, RB x + RB).  Thread (tr, tc)
  // holds rows RB x + 2 tr, +1 and columns 4 tc .. 4 tc + 3; every entry is
  // one fp64 chain over the groups in ascending order.  Shifted means are
  // staged in LDS GB groups at a time; the next chunk's loads are issued
  // into registers before the current chunk is used.
  constexpr int CQD = D / 4;               // column quads
  constexpr int TRN = 256 / CQD;           // row pairs per block
  constexpr int RB = 2 * TRN;              // rows per block
  constexpr int GB = 32;
  constexpr int LPT = GB * D / 4 / 256;    // float4 loads per thread per chunk
  static_assert(LPT >= 1 && 256 % CQD == 0 && D % RB == 0, "thread mapping");
  __shared__ __attribute__((aligned(32))) double ks[GB][D];
  __shared__ double sh[D];
  __shared__ __attribute__((aligned(32))) double ssum[256 / CQD][D];
  __shared__ int fl[GB];
  __shared__ int first_s, cnt_s;
  const int bh = blockIdx.y, tid = threadIdx.x;
  const int C = g.CK;
  const int32_t* o = offk + (size_t)bh * (g.CKt + 1);
  const float* kb = kbar + (size_t)bh * C * D;
  if (tid == 0) {
    first_s = C;
    cnt_s = 0;
  }
  __syncthreads();
  // the first nonempty group (its mean is the shift) and the nonempty count
  {
    int first = C, cnt = 0;
    for (int b = tid; b < C; b += 256) {
      const bool ne = o[b + 1] > o[b];
      cnt += ne;
      if (ne && first == C) first = b;
    }
    if (first < C) atomicMin(&first_s, first);
    atomicAdd(&cnt_s, cnt);
  }
  __syncthreads();
  const int first = first_s, cplus = cnt_s;
  if (tid < D) sh[tid] = first < C ? (double)kb[(size_t)first * D + tid] : 0.0;
  const int tc = tid % CQD, tr = tid / CQD;
  const int r0 = blockIdx.x * RB + 2 * tr, c0 = 4 * tc;
  // acc: the thread's entries of sum_b d_b d_b^T; sp: its staging columns'
  // sums over the groups it stages (b = tid / CQD + k * 256 / CQD)
  double acc[2][4], sp[4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[a][e] = 0.0;
#pragma unroll
  for (int e = 0; e < 4; ++e) sp[e] = 0.0;
  float4 pre[LPT];
  int pfl = 0;
  auto load_chunk = [&](int b0) {
#pragma unroll
    for (int l = 0; l < LPT; ++l) {
      const int e4 = tid + 256 * l, bb = b0 + e4 / CQD;
      pre[l] = bb < C ? ((const float4*)(kb + (size_t)bb * D))[e4 % CQD] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (tid < GB) pfl = (b0 + tid < C) && (o[b0 + tid + 1] > o[b0 + tid]);
  };
  load_chunk(0);
  for (int b0 = 0; b0 < C; b0 += GB) {
    if (tid < GB) fl[tid] = pfl;
    __syncthreads();  // flags and the shift visible; the previous chunk is consumed
#pragma unroll
    for (int l = 0; l < LPT; ++l) {
      const int e4 = tid + 256 * l, i = e4 / CQD, c = (e4 % CQD) * 4;
      const bool ne = fl[i] != 0;
      double4 v;
      v.x = ne ? (double)pre[l].x - sh[c + 0] : 0.0;
      v.y = ne ? (double)pre[l].y - sh[c + 1] : 0.0;
      v.z = ne ? (double)pre[l].z - sh[c + 2] : 0.0;
      v.w = ne ? (double)pre[l].w - sh[c + 3] : 0.0;
      *(double4*)&ks[i][c] = v;
      sp[0] += v.x;
      sp[1] += v.y;
      sp[2] += v.z;
      sp[3] += v.w;
    }
    if (b0 + GB < C) load_chunk(b0 + GB);
    __syncthreads();
    // groups past the end were staged as zeros, so whole chunks are summed
    // (four groups' operands loaded together)
#pragma unroll 4
    for (int i = 0; i < GB; ++i) {
      const double2 rv = *(const double2*)&ks[i][r0];
      const double4 cv = *(const double4*)&ks[i][c0];
      const double r[2] = {rv.x, rv.y};
      const double c[4] = {cv.x, cv.y, cv.z, cv.w};
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[a][e] = fma(r[a], c[e], acc[a][e]);
    }
  }
  // S = sum_b d_b from the staging threads' partial sums
  *(double4*)&ssum[tr][4 * tc] = make_double4(sp[0], sp[1], sp[2], sp[3]);
  __syncthreads();
  double rs[2], cs[4];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    rs[a] = 0.0;
    for (int q = 0; q < 256 / CQD; ++q) rs[a] += ssum[q][r0 + a];
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    cs[e] = 0.0;
    for (int q = 0; q < 256 / CQD; ++q) cs[e] += ssum[q][c0 + e];
  }
  const double np = (double)max(cplus, 1);
  const double den = np * (double)D;
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    double* out = gram + (size_t)bh * D * D + (size_t)(r0 + a) * D + c0;
    double4 v;
    v.x = (acc[a][0] - rs[a] * cs[0] / np) / den;
    v.y = (acc[a][1] - rs[a] * cs[1] / np) / den;
    v.z = (acc[a][2] - rs[a] * cs[2] / np) / den;
    v.w = (acc[a][3] - rs[a] * cs[3] / np) / den;
    *(double4*)out = v;
  }
}

// ---------------------------------------------------------------------------
// Routing under a pair budget (Sec. 4.3).  Priority of cell (a, b): the
// centroid estimate of the log attention probability of one of its pairs,
//   s_ab = (float fmaf chain of qbar_a . kbar_b) * (float)(1/sqrt(d)),
//   pi_ab = s_ab - (float)log(sum_b |G_b| exp(s_ab)).
// Every nonempty query group keeps its best cell (forced); the other cells are
// taken in (pi desc, a*C_k + b asc) order while the cumulative pair cost
// |G_a||G_b| fits in the budget, which already excludes the probes' cost.
// ---------------------------------------------------------------------------

template <int D>
__global__ __launch_bounds__(256) void k_route_prio(const float* qbar, const float* kbar, Geom g,
                                                    const int32_t* offq, const int32_t* offk,
                                                    float* prio, int32_t* forced) {
  // Block (x, bh) owns query groups [64x, 64x + 64).  Phase 1: s_ab for every
  // K/V group on MFMA.  Both group means are split into three bf16 parts
  // (hi + mid + lo reproduce the float value) and the six products whose
  // terms reach 2^-16 of the leading one (hh; hm, mh; hl, lh, mm) are
  // accumulated, the five small ones apart from hh, so s_ab keeps float
  // accuracy.  Wave w holds the parts of query rows 32*(w&1) .. +32 in
  // registers and takes key columns 32*(w>>1) .. +32 of each 64-group chunk,
  // staged in LDS.  Phase 2: one wave per query group computes lse_a (double
  // sum), pi_ab and the forced (best) cell.
  constexpr int TR = 64, KS = D / 16, FLD = D + 8;
  __shared__ __attribute__((aligned(16))) uint16_t ks3[3][TR][FLD];
  const int bh = blockIdx.y, tid = threadIdx.x;
  const int a0 = blockIdx.x * TR;
  const int CK = g.CK, CQ = g.CQ;
  const int32_t* oq = offq + (size_t)bh * (g.CQt + 1);
  const int32_t* ok = offk + (size_t)bh * (g.CKt + 1);
  const float scale = (float)(1.0 / sqrt((double)D));
  const float* qb = qbar + (size_t)bh * CQ * D;
  const float* kb = kbar + (size_t)bh * CK * D;
  float* prh = prio + (size_t)bh * CQ * CK;
  {
    const int wv = tid >> 6, lane = tid & 63, n = lane & 31, h = lane >> 5;
    const int rt = wv & 1, ct = wv >> 1;
    const int qa = a0 + rt * 32 + n;  // this lane's A row
    bf16x8 qp[3][KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      float v[8];
      if (qa < CQ) {
        const float4 u0 = *(const float4*)(qb + (size_t)qa * D + ks * 16 + h * 8);
        const float4 u1 = *(const float4*)(qb + (size_t)qa * D + ks * 16 + h * 8 + 4);
        v[0] = u0.x; v[1] = u0.y; v[2] = u0.z; v[3] = u0.w;
        v[4] = u1.x; v[5] = u1.y; v[6] = u1.z; v[7] = u1.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const __bf16 hi = (__bf16)v[e];
        const float r1 = v[e] - (float)hi;
        const __bf16 mid = (__bf16)r1;
        qp[0][ks][e] = hi;
        qp[1][ks][e] = mid;
        qp[2][ks][e] = (__bf16)(r1 - (float)mid);
      }
    }
    // a chunk's key means: every 16-byte load issued before the splits
    constexpr int LPT4 = TR * D / 4 / 256;
    for (int b0 = 0; b0 < CK; b0 += TR) {
      __syncthreads();  // the previous chunk is consumed
      float4 pre[LPT4];
#pragma unroll
      for (int j = 0; j < LPT4; ++j) {
        const int i4 = tid + 256 * j, r = i4 * 4 / D, c = i4 * 4 % D;
        pre[j] = b0 + r < CK ? *(const float4*)(kb + (size_t)(b0 + r) * D + c) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int j = 0; j < LPT4; ++j) {
        const int i4 = tid + 256 * j, r = i4 * 4 / D, c = i4 * 4 % D;
        const float fv[4] = {pre[j].x, pre[j].y, pre[j].z, pre[j].w};
        uint32_t pw[3][2];  // the four values' parts, two per word (8-byte stores)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float f = fv[e];
          const uint16_t hi = __builtin_bit_cast(uint16_t, (__bf16)f);
          const float r1 = f - bf16_bits_to_f32(hi);
          const uint16_t mid = __builtin_bit_cast(uint16_t, (__bf16)r1);
          const uint16_t lo = __builtin_bit_cast(uint16_t, (__bf16)(r1 - bf16_bits_to_f32(mid)));
          const int sh = 16 * (e & 1);
          if ((e & 1) == 0) pw[0][e >> 1] = pw[1][e >> 1] = pw[2][e >> 1] = 0u;
          pw[0][e >> 1] |= (uint32_t)hi << sh;
          pw[1][e >> 1] |= (uint32_t)mid << sh;
          pw[2][e >> 1] |= (uint32_t)lo << sh;
        }
#pragma unroll
        for (int part = 0; part < 3; ++part) *(uint2*)&ks3[part][r][c] = make_uint2(pw[part][0], pw[part][1]);
      }
      __syncthreads();
      f32x16 Sb, Ss;
#pragma unroll
      for (int i = 0; i < 16; ++i) Sb[i] = Ss[i] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int col = ct * 32 + n;
        const bf16x8 kh = __builtin_bit_cast(bf16x8, *(const uint4*)&ks3[0][col][ks * 16 + h * 8]);
        const bf16x8 km = __builtin_bit_cast(bf16x8, *(const uint4*)&ks3[1][col][ks * 16 + h * 8]);
        const bf16x8 kl = __builtin_bit_cast(bf16x8, *(const uint4*)&ks3[2][col][ks * 16 + h * 8]);
        Sb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qp[0][ks], kh, Sb, 0, 0, 0);
        Ss = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qp[0][ks], km, Ss, 0, 0, 0);
        Ss = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qp[1][ks], kh, Ss, 0, 0, 0);
        Ss = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qp[0][ks], kl, Ss, 0, 0, 0);
        Ss = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qp[2][ks], kh, Ss, 0, 0, 0);
        Ss = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qp[1][ks], km, Ss, 0, 0, 0);
      }
      // register i holds query row rt*32 + (i/4)*8 + h*4 + i%4, key column ct*32 + n
      const int b = b0 + ct * 32 + n;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int a = a0 + rt * 32 + (i / 4) * 8 + h * 4 + (i % 4);
        if (a < CQ && b < CK) prh[(size_t)a * CK + b] = (Sb[i] + Ss[i]) * scale;
      }
    }
  }
  __syncthreads();
  // Phase 2, one wave per query group.  When a row fits in NR cells per lane
  // (cells b = lane + 64u) its scores stay in registers for the max, the
  // normaliser and the output, and the K/V group sizes are read once per
  // wave; longer rows go through global memory 8 cells per lane at a time.
  constexpr int NR = 24, NB = 8;
  const int wv = tid >> 6, lane = tid & 63;
  const bool inreg = CK <= 64 * NR;
  int nbr[NR];
  if (inreg) {
#pragma unroll
    for (int u = 0; u < NR; ++u) {
      const int b = lane + 64 * u;
      nbr[u] = b < CK ? ok[b + 1] - ok[b] : 0;
    }
  }
  for (int rr = wv; rr < TR; rr += 4) {
    const int a = a0 + rr;
    if (a >= CQ) break;
    float* pr = prh + (size_t)a * CK;
    if (oq[a + 1] == oq[a]) {
      for (int b = lane; b < CK; b += 64) pr[b] = 0.f;
      if (lane == 0) forced[(size_t)bh * CQ + a] = -1;
      continue;
    }
    float bestv = -INFINITY;
    int besti = 0x7fffffff;
    if (inreg) {
      float sv[NR];
#pragma unroll
      for (int u = 0; u < NR; ++u) {
        const int b = lane + 64 * u;
        sv[u] = b < CK ? pr[b] : 0.f;
      }
      float mx = -INFINITY;
#pragma unroll
      for (int u = 0; u < NR; ++u)
        if (nbr[u] > 0) mx = fmaxf(mx, sv[u]);
      mx = wave_max(mx);
      // terms exp(s - max) <= 1 in float (about 1 ulp each), summed in double
      double z = 0.0;
#pragma unroll
      for (int u = 0; u < NR; ++u)
        if (nbr[u] > 0) z += (double)nbr[u] * (double)expf(sv[u] - mx);
      z = wave_sum_d(z);
      const float lse = (float)((double)mx + log(z));
#pragma unroll
      for (int u = 0; u < NR; ++u) {
        const int b = lane + 64 * u;
        if (b < CK) {
          float pv = 0.f;
          if (nbr[u] > 0) {
            pv = sv[u] - lse;
            if (besti == 0x7fffffff || pv > bestv) {  // b ascending within the lane
              bestv = pv;
              besti = b;
            }
          }
          pr[b] = pv;
        }
      }
    } else {
      float mx = -INFINITY;
      for (int b0 = 0; b0 < CK; b0 += 64 * NB) {
        float sv[NB];
        int nb[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
          const int b = b0 + lane + 64 * u;
          sv[u] = b < CK ? pr[b] : 0.f;
          nb[u] = b < CK ? ok[b + 1] - ok[b] : 0;
        }
#pragma unroll
        for (int u = 0; u < NB; ++u)
          if (nb[u] > 0) mx = fmaxf(mx, sv[u]);
      }
      mx = wave_max(mx);
      double z = 0.0;
      for (int b0 = 0; b0 < CK; b0 += 64 * NB) {
        float sv[NB];
        int nb[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
          const int b = b0 + lane + 64 * u;
          sv[u] = b < CK ? pr[b] : 0.f;
          nb[u] = b < CK ? ok[b + 1] - ok[b] : 0;
        }
#pragma unroll
        for (int u = 0; u < NB; ++u)
          if (nb[u] > 0) z += (double)nb[u] * (double)expf(sv[u] - mx);
      }
      z = wave_sum_d(z);
      const float lse = (float)((double)mx + log(z));
      for (int b0 = 0; b0 < CK; b0 += 64 * NB) {
        float sv[NB];
        int nb[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
          const int b = b0 + lane + 64 * u;
          sv[u] = b < CK ? pr[b] : 0.f;
          nb[u] = b < CK ? ok[b + 1] - ok[b] : 0;
        }
#pragma unroll
        for (int u = 0; u < NB; ++u) {
          const int b = b0 + lane + 64 * u;
          if (b < CK) {
            float pv = 0.f;
            if (nb[u] > 0) {
              pv = sv[u] - lse;
              if (besti == 0x7fffffff || pv > bestv) {  // b ascending within the lane
                bestv = pv;
                besti = b;
              }
            }
            pr[b] = pv;
          }
        }
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bestv, o);
      const int oi = __shfl_xor(besti, o);
      if (oi != 0x7fffffff && (besti == 0x7fffffff || ov > bestv || (ov == bestv && oi < besti))) {
        bestv = ov;
        besti = oi;
      }
    }
    if (lane == 0) forced[(size_t)bh * CQ + a] = (besti == 0x7fffffff) ? -1 : besti;
  }
}

// Top-p routing keys (SPARSEPR_ROUTING_TOP_P): for query group a, the cells
// in (pi desc, b asc) order over nonempty K/V groups, and key(a, b) =
// -(float)e_ab with e_ab the estimated attention mass ranked before b, the
// sum of |G_b'| exp(pi_ab') in double.  One block per (a, head): the 64-bit
// order keys are bitonic-sorted in LDS; each thread sums a contiguous run of
// the sorted masses and a block scan of the run totals gives every prefix.
// np2 = C_k rounded up to a power of two (dynamic LDS: np2 * 8 bytes).
__global__ __launch_bounds__(256) void k_route_topp(Geom g, Work w, int np2) {
  extern __shared__ __attribute__((aligned(16))) unsigned char topp_lds[];
  uint64_t* key = (uint64_t*)topp_lds;
  __shared__ double run_tot[256];
  const int a = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int32_t* oq = w.offq + (size_t)bh * (g.CQt + 1);
  const int32_t* ok = w.offk + (size_t)bh * (g.CKt + 1);
  const float* pr = w.prio + ((size_t)bh * g.CQ + a) * g.CK;
  float* out = w.skey + ((size_t)bh * g.CQ + a) * g.CK;
  if (oq[a + 1] == oq[a]) {
    for (int b = tid; b < g.CK; b += 256) out[b] = 0.f;
    return;
  }
  // larger key first: priority descending, then b ascending; 0 = no cell
  for (int i = tid; i < np2; i += 256) {
    uint64_t k = 0;
    if (i < g.CK && ok[i + 1] > ok[i])
      k = ((uint64_t)float_order_bits(pr[i]) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)i);
    key[i] = k;
  }
  for (int b = tid; b < g.CK; b += 256)
    if (ok[b + 1] == ok[b]) out[b] = 0.f;
  __syncthreads();
  for (int size = 2; size <= np2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < np2; i += 256) {
        const int j = i ^ stride;
        if (j > i) {
          const bool desc = (i & size) == 0;
          const uint64_t ki = key[i], kj = key[j];
          if (desc ? (ki < kj) : (ki > kj)) {
            key[i] = kj;
            key[j] = ki;
          }
        }
      }
      __syncthreads();
    }
  }
  // thread t owns sorted positions [t * per, (t + 1) * per)
  const int per = (np2 + 255) / 256;
  const int i0 = min(tid * per, np2), i1 = min(i0 + per, np2);
  auto mass_at = [&](int i, int& b) -> double {
    const uint64_t k = key[i];
    if (k == 0) {
      b = -1;
      return 0.0;
    }
    b = (int)(0xFFFFFFFFu - (uint32_t)(k & 0xFFFFFFFFu));
    return (double)(ok[b + 1] - ok[b]) * exp((double)pr[b]);
  };
  double tot = 0.0;
  for (int i = i0; i < i1; ++i) {
    int b;
    tot += mass_at(i, b);
  }
  run_tot[tid] = tot;
  __syncthreads();
  if (tid < 64) {  // exclusive scan of the 256 run totals by one wave
    double v[4], t4 = 0.0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      v[u] = run_tot[tid * 4 + u];
      t4 += v[u];
    }
    double incl = t4;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const double y = __shfl_up(incl, o);
      if (tid >= o) incl += y;
    }
    const double before = __shfl_up(incl, 1);
    double e = tid > 0 ? before : 0.0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const double next = e + v[u];
      run_tot[tid * 4 + u] = e;
      e = next;
    }
  }
  __syncthreads();
  double e = run_tot[tid];
  for (int i = i0; i < i1; ++i) {
    int b;
    const double m = mass_at(i, b);
    if (b < 0) break;
    out[b] = -(float)e;
    e += m;
  }
}

// The selection histograms hold, per bucket, the pair cost of its cells and,
// from bit g.sel_cshift up (when it is nonzero), their count.
__device__ __forceinline__ unsigned long long sel_count_unit(const Geom& g) {
  return g.sel_cshift ? (1ull << g.sel_cshift) : 0ull;
}

// selstate slots.  SS_DONE: 0 searching, 1 every eligible cell fits,
// 2 boundary key found (cells with larger keys are taken), 3 nothing beyond
// the forced cells fits.
enum { SS_REM = 0, SS_PREFIX = 1, SS_ABOVE = 2, SS_DONE = 3, SS_BOUND = 4 };

// Total order of the walk: larger key first = priority descending, then flat
// index ascending.
__device__ __forceinline__ uint64_t cell_key(float p, int64_t idx) {
  return ((uint64_t)float_order_bits(p) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)idx);
}

__global__ __launch_bounds__(256) void k_sel_init(Geom g, Work w) {
  __shared__ long long red[4];
  __shared__ int redc[4];
  const int bh = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int32_t* oq = w.offq + (size_t)bh * (g.CQt + 1);
  const int32_t* ok = w.offk + (size_t)bh * (g.CKt + 1);
  const int32_t* fo = w.forced + (size_t)bh * g.CQ;
  long long fc = 0;
  int ncell = 0;
  for (int a = tid; a < g.CQ; a += 256) {
    const int b = fo[a];
    if (b >= 0) {
      fc += (long long)(oq[a + 1] - oq[a]) * (ok[b + 1] - ok[b]);
      ++ncell;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    fc += __shfl_xor(fc, o);
    ncell += __shfl_xor(ncell, o);
  }
  if (lane == 0) {
    red[wv] = fc;
    redc[wv] = ncell;
  }
  uint64_t* hist = w.selhist + (size_t)bh * kSelPasses * kSelBins;
  for (int i = tid; i < kSelPasses * kSelBins; i += 256) hist[i] = 0;
  __syncthreads();
  if (tid == 0) {
    const long long forced = red[0] + red[1] + red[2] + red[3];
    const int fcells = redc[0] + redc[1] + redc[2] + redc[3];
    int64_t* st = w.selstate + (size_t)bh * 8;
    const long long rem = (long long)g.budget - forced;
    const long long all = (long long)g.NV * (long long)g.NV - forced;
    st[SS_REM] = rem;
    st[SS_PREFIX] = 0;
    st[SS_ABOVE] = 0;
    st[SS_BOUND] = 0;
    st[SS_DONE] = (rem < 0) ? 3 : (all <= rem ? 1 : 0);
    int64_t* stats = w.stats + (size_t)bh * 16;
    stats[ST_FORCED_PAIRS] = forced;
    stats[ST_FORCED_CELLS] = fcells;
    if (rem < 0) stats[ST_FLAGS] |= SPARSEPR_FLAG_BUDGET_BELOW_FORCED;
  }
}

// Weighted radix select, one 8-bit digit of the 64-bit cell key per pass:
// histogram of pair cost per digit over the cells still in the bucket.
// Blocks take rows of the route matrix (two at a time), threads up to KB
// columns each; the columns' sizes stay in registers across the rows.  The
// leading digits are shared by most cells (the priorities span a few
// binades), so each thread sums the cost of the first two digits it meets in
// registers and adds only its other cells to LDS one by one.
__global__ __launch_bounds__(256) void k_sel_hist(Geom g, Work w, int p) {
  constexpr int KB = 8, RR = 2;
  __shared__ unsigned long long hs[kSelBins];
  const int bh = blockIdx.y, tid = threadIdx.x;
  const int64_t* st = w.selstate + (size_t)bh * 8;
  if (st[SS_DONE] != 0) return;
  for (int i = tid; i < kSelBins; i += 256) hs[i] = 0;
  __syncthreads();
  const int shift = 56 - 8 * p;
  const uint64_t prefix = (uint64_t)st[SS_PREFIX];
  const int32_t* oq = w.offq + (size_t)bh * (g.CQt + 1);
  const int32_t* ok = w.offk + (size_t)bh * (g.CKt + 1);
  const int32_t* fo = w.forced + (size_t)bh * g.CQ;
  const float* pr = (g.routing == SPARSEPR_ROUTING_TOP_P ? w.skey : w.prio) + (size_t)bh * g.CQ * g.CK;
  const unsigned long long cunit = sel_count_unit(g);
  // two digits per thread are summed in registers, the others added to LDS
  int dA = -1, dB = -1;
  unsigned long long sA = 0ull, sB = 0ull;
  auto hist_add = [&](bool act, int dig, unsigned long long wgt) {
    if (!act) return;
    if (dig == dA) {
      sA += wgt;
    } else if (dig == dB) {
      sB += wgt;
    } else if (dA < 0) {
      dA = dig;
      sA = wgt;
    } else if (dB < 0) {
      dB = dig;
      sB = wgt;
    } else {
      atomicAdd(&hs[dig], wgt);
    }
  };
  for (int cb = 0; cb < g.CK; cb += 256 * KB) {
    int nb[KB];
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      const int b = cb + tid + 256 * k;
      nb[k] = b < g.CK ? ok[b + 1] - ok[b] : 0;
    }
    for (int a0 = blockIdx.x; a0 < g.CQ; a0 += RR * gridDim.x) {
      int na[RR], fa[RR];
      float pv[RR][KB];
#pragma unroll
      for (int r = 0; r < RR; ++r) {
        const int a = a0 + r * gridDim.x;
        na[r] = a < g.CQ ? oq[a + 1] - oq[a] : 0;
        fa[r] = na[r] ? fo[a] : -1;
#pragma unroll
        for (int k = 0; k < KB; ++k) {
          const int b = cb + tid + 256 * k;
          pv[r][k] = (na[r] && b < g.CK && nb[k]) ? pr[(int64_t)a * g.CK + b] : 0.f;
        }
      }
#pragma unroll
      for (int r = 0; r < RR; ++r) {
        if (na[r] == 0) continue;  // uniform
        const int64_t row = (int64_t)(a0 + r * gridDim.x) * g.CK;
#pragma unroll
        for (int k = 0; k < KB; ++k) {
          if (cb + 256 * k >= g.CK) break;  // uniform
          const int b = cb + tid + 256 * k;
          const uint64_t key = cell_key(pv[r][k], row + b);
          bool act = b < g.CK && nb[k] != 0 && b != fa[r];
          if (p > 0) act = act && (key >> (shift + 8)) == (prefix >> (shift + 8));
          hist_add(act, (int)((key >> shift) & 255),
                   (unsigned long long)na[r] * (unsigned long long)nb[k] + cunit);
        }
      }
    }
  }
  if (dA >= 0) atomicAdd(&hs[dA], sA);
  if (dB >= 0) atomicAdd(&hs[dB], sB);
  __syncthreads();
  uint64_t* gh = w.selhist + ((size_t)bh * kSelPasses + p) * kSelBins;
  for (int i = tid; i < kSelBins; i += 256)
    if (hs[i]) atomicAdd((unsigned long long*)&gh[i], hs[i]);
}

// Pick the digit bucket where the cumulative cost (from the largest keys
// down) first exceeds the remaining budget.
__global__ __launch_bounds__(256) void k_sel_choose(Geom g, Work w, int p) {
  // Thread t takes digit 255 - t: an inclusive scan of the pair costs from
  // the largest digit down gives, per digit, the cost of it and every digit
  // above, and the first digit where that exceeds the budget is the bucket.
  static_assert(kSelBins == 256, "one digit per thread");
  __shared__ long long wsum[4];
  __shared__ int hit;
  const int bh = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int64_t* st = w.selstate + (size_t)bh * 8;
  if (st[SS_DONE] != 0) return;  // uniform over the block
  const uint64_t* ghg = w.selhist + ((size_t)bh * kSelPasses + p) * kSelBins;
  const int dg = kSelBins - 1 - tid;
  const uint64_t raw = ghg[dg];
  const unsigned long long cunit = sel_count_unit(g);
  const long long h = (long long)(cunit ? (raw & (cunit - 1ull)) : raw);
  long long x = h;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const long long y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wv] = x;
  if (tid == 0) hit = kSelBins;
  __syncthreads();
  long long cum = st[SS_ABOVE] + x;
  for (int k = 0; k < wv; ++k) cum += wsum[k];
  if (cum > (long long)st[SS_REM]) atomicMin(&hit, tid);
  __syncthreads();  // every thread has read the state before it changes
  if (hit == kSelBins) {
    if (tid == 0) st[SS_DONE] = 1;
    return;
  }
  if (tid != hit) return;
  const int shift = 56 - 8 * p;
  const uint64_t prefix = (uint64_t)st[SS_PREFIX] | ((uint64_t)dg << shift);
  st[SS_PREFIX] = (int64_t)prefix;
  st[SS_ABOVE] = cum - h;
  if (shift == 0) {
    st[SS_BOUND] = (int64_t)prefix;
    st[SS_DONE] = 2;
  } else if (cunit && (raw >> g.sel_cshift) == 1) {
    // the boundary cell is the only one with this prefix: every cell of
    // a higher bucket is taken and it is not, which is what comparing
    // keys with the largest key of the prefix selects
    st[SS_BOUND] = (int64_t)(prefix | ((1ull << shift) - 1ull));
    st[SS_DONE] = 2;
  }
}

// Route matrix over all cells (dense-prefix group included): forced cells,
// cells above the boundary key, and every cell of the dense-prefix group.
__global__ __launch_bounds__(256) void k_sel_mark(Geom g, Work w) {
  __shared__ int red[4];
  const int bh = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t* st = w.selstate + (size_t)bh * 8;
  const int done = (int)st[SS_DONE];
  const uint64_t bound = (uint64_t)st[SS_BOUND];
  const int32_t* oq = w.offq + (size_t)bh * (g.CQt + 1);
  const int32_t* ok = w.offk + (size_t)bh * (g.CKt + 1);
  const int32_t* fo = w.forced + (size_t)bh * g.CQ;
  const float* pr = (g.routing == SPARSEPR_ROUTING_TOP_P ? w.skey : w.prio) + (size_t)bh * g.CQ * g.CK;
  uint8_t* z = w.z + (size_t)bh * g.CQt * g.CKt;
  int cnt = 0;
  // rows of the route matrix per block, up to KB columns per thread (their
  // group sizes held in registers across the rows)
  constexpr int KB = 8;
  for (int cb = 0; cb < g.CKt; cb += 256 * KB) {
    int nb[KB];
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      const int b = cb + tid + 256 * k;
      nb[k] = b < g.CK ? ok[b + 1] - ok[b] : 0;
    }
    for (int a = blockIdx.x; a < g.CQt; a += gridDim.x) {
      uint8_t* zr = z + (size_t)a * g.CKt;
      const bool arow = a < g.CQ;
      const int na = arow ? oq[a + 1] - oq[a] : 0;
      const int fa = na > 0 ? fo[a] : -1;
      const int64_t row = (int64_t)a * g.CK;
      float pv[KB];
#pragma unroll
      for (int k = 0; k < KB; ++k) {
        const int b = cb + tid + 256 * k;
        pv[k] = (done == 2 && na > 0 && b < g.CK && nb[k] > 0) ? pr[row + b] : 0.f;
      }
#pragma unroll
      for (int k = 0; k < KB; ++k) {
        const int b = cb + tid + 256 * k;
        if (b >= g.CKt) break;
        uint8_t sel = 0;
        if (arow && b < g.CK) {
          if (na > 0 && nb[k] > 0) {
            if (fa == b) {
              sel = 1;
            } else if (done == 1) {
              sel = 1;
            } else if (done == 2) {
              sel = cell_key(pv[k], row + b) > bound;
            }
            cnt += sel;
          }
        } else {
          sel = 1;  // dense-prefix query group or K/V group
        }
        zr[b] = sel;
      }
    }
  }
  cnt = wave_sum_i(cnt);
  if (lane == 0) red[wv] = cnt;
  __syncthreads();
  if (tid == 0) {
    const int c = red[0] + red[1] + red[2] + red[3];
    if (c) atomicAdd((unsigned long long*)&w.stats[(size_t)bh * 16 + ST_ROUTED_CELLS],
                     (unsigned long long)c);
  }
}

// Per query group, the routed K/V groups as maximal contiguous ranges of the
// group-major K/V order, and their total length.  One wave per query group
// walks the K/V groups 64 at a time.  Among the nonempty groups, a range
// starts where routing switches on and ends where it switches off (empty
// groups hold no keys, so they neither break nor extend a range): each lane
// at a switch-off emits the range from the previous switch's key (a ballot
// finds that lane, or the carry from earlier chunks) to its own start key,
// at the index given by the switch-offs before it.
__global__ __launch_bounds__(256) void k_ranges(Geom g, Work w) {
  const int bh = blockIdx.y, wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int a = blockIdx.x * 4 + wv;
  if (a >= g.CQt) return;
  const int32_t* oq = w.offq + (size_t)bh * (g.CQt + 1);
  const int32_t* ok = w.offk + (size_t)bh * (g.CKt + 1);
  const uint8_t* z = w.z + ((size_t)bh * g.CQt + a) * g.CKt;
  int2* rg = w.rng + ((size_t)bh * g.CQt + a) * g.CKt;
  const int na = oq[a + 1] - oq[a];
  const uint64_t below = (1ull << lane) - 1ull;
  int cnt = 0, tot = 0;
  if (na > 0) {
    int prev_rt = 0;    // routing of the last nonempty group so far
    int start_key = 0;  // key of the last switch so far (a range start when prev_rt)
    // the next 64 groups' offsets and routes are loaded before this slice
    // is processed
    int nks = lane < g.CKt ? ok[lane] : 0, nke = lane < g.CKt ? ok[lane + 1] : 0;
    uint8_t nz = lane < g.CKt ? z[lane] : 0;
    for (int b0 = 0; b0 < g.CKt; b0 += 64) {
      const int b = b0 + lane;
      const bool in = b < g.CKt;
      const int ks = nks, ke = nke;
      const uint8_t zb = nz;
      if (b0 + 64 < g.CKt) {
        const int bn = b + 64;
        const bool inn = bn < g.CKt;
        nks = inn ? ok[bn] : 0;
        nke = inn ? ok[bn + 1] : 0;
        nz = inn ? z[bn] : 0;
      }
      const bool ne = in && ke > ks;
      const bool rt = ne && zb != 0;
      const uint64_t NE = __ballot(ne), RT = __ballot(rt);
      const uint64_t nb = NE & below;
      const int pr = nb ? (int)((RT >> (63 - __clzll((long long)nb))) & 1ull) : prev_rt;
      const bool sw = ne && ((int)rt != pr);
      const uint64_t SW = __ballot(sw);
      const uint64_t sb = SW & below;
      const int pkey = __shfl(ks, sb ? 63 - __clzll((long long)sb) : lane);
      const bool off = sw && !rt;
      const uint64_t OFF = __ballot(off);
      if (off) {
        const int sk = sb ? pkey : start_key;
        rg[cnt + __popcll(OFF & below)] = make_int2(sk, ks - sk);
        tot += ks - sk;
      }
      cnt += __popcll(OFF);
      if (SW) start_key = __shfl(ks, 63 - __clzll((long long)SW));
      if (NE) prev_rt = (int)((RT >> (63 - __clzll((long long)NE))) & 1ull);
    }
    tot = wave_sum_i(tot);
    if (prev_rt) {
      // the last nonempty group is routed: its range runs to the end
      const int endk = ok[g.CKt];
      if (lane == 0) rg[cnt] = make_int2(start_key, endk - start_key);
      tot += endk - start_key;
      ++cnt;
    }
  }
  if (lane == 0) {
    w.rng_cnt[(size_t)bh * g.CQt + a] = cnt;
    w.keytot[(size_t)bh * g.CQt + a] = tot;
    if (na > 0)
      atomicAdd((unsigned long long*)&w.stats[(size_t)bh * 16 + ST_ROUTED_PAIRS],
                (unsigned long long)((long long)na * tot));
  }
}

// Attention work items: each query group split into tiles of kQTile rows.
__global__ __launch_bounds__(1024) void k_chunks(Geom g, Work w) {
  // A head's chunks in decreasing order of their group's routed key count
  // (64 buckets of similar counts, heaviest first; any order inside a
  // bucket): the attention launches dispatch chunks in list order, so the
  // blocks left at the end of each launch are the short ones.  Every chunk's
  // rows and arithmetic are the same in any order.
  constexpr int NB = 64;
  __shared__ int bcnt[NB];
  __shared__ int wmax_s, total_s;
  extern __shared__ int nch[];  // CQt
  const int bh = blockIdx.x, tid = threadIdx.x;
  const int32_t* oq = w.offq + (size_t)bh * (g.CQt + 1);
  const int32_t* kt = w.keytot + (size_t)bh * g.CQt;
  if (tid < NB) bcnt[tid] = 0;
  if (tid == 0) wmax_s = 0;
  __syncthreads();
  for (int a = tid; a < g.CQt; a += 1024) {
    nch[a] = (oq[a + 1] - oq[a] + kQTile - 1) / kQTile;
    if (nch[a] > 0) atomicMax(&wmax_s, kt[a]);
  }
  __syncthreads();
  const int64_t wmax = wmax_s;
  auto bucket = [&](int a) { return (int)(((wmax - kt[a]) * NB) / (wmax + 1)); };
  for (int a = tid; a < g.CQt; a += 1024)
    if (nch[a] > 0) atomicAdd(&bcnt[bucket(a)], nch[a]);
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int b = 0; b < NB; ++b) {
      const int c = bcnt[b];
      bcnt[b] = run;
      run += c;
    }
    total_s = run;
  }
  __syncthreads();
  int4* ch = w.chunks + (size_t)bh * g.nchunk_max;
  for (int a = tid; a < g.CQt; a += 1024) {
    if (nch[a] == 0) continue;
    const int na = oq[a + 1] - oq[a];
    int c = atomicAdd(&bcnt[bucket(a)], nch[a]);
    for (int r0 = 0; r0 < na; r0 += kQTile) ch[c++] = make_int4(a, r0, min(kQTile, na - r0), kt[a]);
  }
  if (tid == 0) w.nchunks[bh] = total_s;
}

// ---------------------------------------------------------------------------
// Probe selection (App. A.2, Algorithm "Query-Group-Stratified Exact Probe
// Selection") and coverage weights w_p = |G_a| / m_a (eq. app_probe_weight).
// ---------------------------------------------------------------------------

// Radial key of every video row: squared distance to its group mean in phi_Q
// space (ordering by it is ordering by the distance), one fmaf chain in
// coordinate order per row.  When the rank is a multiple of 4, a block stages
// the coordinates of its 128 rows in LDS (16-byte pitch) with coalesced loads
// and reads them and the gathered centroid four at a time.
__global__ __launch_bounds__(128) void k_probe_d2(Geom g, Work w) {
  extern __shared__ __attribute__((aligned(16))) float ps[];  // 128 * (rq + 4) floats when rq % 4 == 0
  const int bh = blockIdx.y, tid = threadIdx.x;
  const int i0 = blockIdx.x * 128;
  const int R = g.rq;
  const int rows = min(128, g.NV - i0);
  const float* phb = w.phiq + ((size_t)bh * g.NV + i0) * R;
  const bool vec = (R & 3) == 0;
  const int LDP = R + 4;
  if (vec) {
#pragma unroll 8
    for (int e = tid; e < rows * (R / 4); e += 128) {
      const int r = e / (R / 4), k4 = e - r * (R / 4);
      *(float4*)&ps[r * LDP + 4 * k4] = ((const float4*)phb)[e];
    }
  }
  __syncthreads();
  if (tid >= rows) return;
  const int i = i0 + tid;
  const int a = w.labq[(size_t)bh * g.N + g.ntext + i];
  const float* c = w.centq + ((size_t)bh * g.CQ + a) * R;
  float acc = 0.f;
  if (vec) {
    const float* ph = ps + tid * LDP;
    for (int k = 0; k < R; k += 4) {
      const float4 p4 = *(const float4*)(ph + k), c4 = *(const float4*)(c + k);
      float diff = p4.x - c4.x;
      acc = fmaf(diff, diff, acc);
      diff = p4.y - c4.y;
      acc = fmaf(diff, diff, acc);
      diff = p4.z - c4.z;
      acc = fmaf(diff, diff, acc);
      diff = p4.w - c4.w;
      acc = fmaf(diff, diff, acc);
    }
  } else {
    const float* ph = phb + (size_t)tid * R;
    for (int k = 0; k < R; ++k) {
      const float diff = ph[k] - c[k];
      acc = fmaf(diff, diff, acc);
    }
  }
  w.d2[(size_t)bh * g.NV + i] = acc;
}

__device__ __forceinline__ uint64_t probe_key(float d2, int row) {
  return ((uint64_t)float_order_bits(d2) << 32) | (uint32_t)row;
}

// One block per head.  Groups are visited in a deterministic order (ascending
// id when there are at most M nonempty groups, otherwise the stride-s
// interleave (rank mod s, rank), s = ceil(G / M)); each visit takes the
// group's next row by (distance, row index).
__global__ __launch_bounds__(1024) void k_probe_select(Geom g, Work w) {
  extern __shared__ int sh[];  // cnt[CQ] | ne[CQ] | mcount[CQ] | base[CQ + 1 + 17]
  int* cnt = sh;
  int* ne = cnt + g.CQ;
  int* mcount = ne + g.CQ;
  int* base = mcount + g.CQ;
  __shared__ int G;
  const int bh = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int M = g.M;
  const int32_t* oq = w.offq + (size_t)bh * (g.CQt + 1);
  const int32_t* perm = w.permq + (size_t)bh * g.N;
  int32_t* probes = w.probes + (size_t)bh * M;
  int32_t* picks = w.picks + (size_t)bh * M;
  float* pw = w.pw + (size_t)bh * M;
  const float* d2 = w.d2 + (size_t)bh * g.NV;
  for (int a = tid; a < g.CQ; a += 1024) {
    cnt[a] = oq[a + 1] - oq[a];
    mcount[a] = 0;
    base[a] = (cnt[a] > 0);
  }
  __syncthreads();
  const int ng = block_exclusive_scan(base, g.CQ, base + g.CQ + 1);
  for (int a = tid; a < g.CQ; a += 1024)
    if (cnt[a] > 0) ne[base[a]] = a;
  if (tid == 0) G = ng;
  __syncthreads();
  // probes per group
  if (G > M) {
    const int s = (G + M - 1) / M, qs = G / s, rem = G % s;
    for (int k = tid; k < G; k += 1024) {
      const int res = k % s;
      const int pos = res * qs + min(res, rem) + k / s;
      if (pos < M) mcount[ne[k]] = 1;
    }
  } else if (tid == 0) {
    int taken = 0;
    for (int t = 0; taken < M; ++t)
      for (int o = 0; o < G && taken < M; ++o)
        if (cnt[ne[o]] > t) {
          mcount[ne[o]]++;
          ++taken;
        }
  }
  __syncthreads();
  for (int a = tid; a < g.CQ; a += 1024) base[a] = mcount[a];
  __syncthreads();
  block_exclusive_scan(base, g.CQ, base + g.CQ + 1);
  // each wave selects the mcount smallest (d2, row) rows of its groups
  for (int a = wv; a < g.CQ; a += 16) {
    const int m = mcount[a];
    if (m == 0) continue;
    const int s0 = oq[a], s1 = oq[a + 1];
    uint64_t last = 0;
    for (int t = 0; t < m; ++t) {
      uint64_t best = ~0ull;
      for (int i = s0 + lane; i < s1; i += 64) {
        const int row = perm[i];
        const uint64_t key = probe_key(d2[row - g.ntext], row);
        if ((t == 0 || key > last) && key < best) best = key;
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const uint64_t ob = __shfl_xor(best, o);
        best = ob < best ? ob : best;
      }
      if (lane == 0) picks[base[a] + t] = (int)(best & 0xffffffffu);
      last = best;
    }
  }
  __syncthreads();
  // emit in visit order
  if (tid == 0) {
    int taken = 0;
    if (G > M) {
      const int s = (G + M - 1) / M;
      for (int res = 0; res < s && taken < M; ++res)
        for (int k = res; k < G && taken < M; k += s) {
          const int a = ne[k];
          probes[taken] = picks[base[a]];
          pw[taken] = (float)cnt[a];
          ++taken;
        }
    } else {
      for (int t = 0; taken < M; ++t)
        for (int o = 0; o < G && taken < M; ++o) {
          const int a = ne[o];
          if (cnt[a] > t) {
            probes[taken] = picks[base[a] + t];
            pw[taken] = (float)cnt[a] / (float)mcount[a];
            ++taken;
          }
        }
    }
    w.nprobes[bh] = taken;
    w.stats[(size_t)bh * 16 + ST_NPROBES] = taken;
  }
}

// Probe rules other than the stratified one (Table probe_estimator_ablation),
// both with equal weights w_p = n_v / M.
// UNIFORM: evenly spaced video rows floor((2i + 1) n_v / (2M)).
__global__ __launch_bounds__(256) void k_probe_uniform(Geom g, Work w) {
  const int bh = blockIdx.x, tid = threadIdx.x;
  const int M = g.M;  // <= n_v, so the rows are distinct
  for (int i = tid; i < M; i += 256) {
    w.probes[(size_t)bh * M + i] = g.ntext + (int)(((int64_t)(2 * i + 1) * g.NV) / (2 * (int64_t)M));
    w.pw[(size_t)bh * M + i] = (float)g.NV / (float)M;
  }
  if (tid == 0) {
    w.nprobes[bh] = M;
    w.stats[(size_t)bh * 16 + ST_NPROBES] = M;
  }
}

// The mixing function of SplitMix64 (Steele, Lea and Flood 2014), a
// bijection of 64-bit words.
__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// RANDOM: the M video rows with the smallest keys SplitMix64(seed * 2^32 +
// row), in key order -- a uniformly random M-subset in random order.  The
// M-th smallest key is found by an 8-bit radix select (the keys of distinct
// rows are distinct), then the M rows at or below it are ranked by key.
__global__ __launch_bounds__(1024) void k_probe_random(Geom g, Work w) {
  __shared__ int hist[256];
  __shared__ uint64_t sel_key[1024];
  __shared__ int sel_row[1024];
  __shared__ int nsel;
  __shared__ unsigned long long prefix_s;
  __shared__ int need_s;
  const int bh = blockIdx.x, tid = threadIdx.x;
  const int M = min(g.M, 1024);  // validated: M <= 1024 for this rule
  const uint64_t seed = (uint64_t)g.probe_seed << 32;
  if (tid == 0) {
    prefix_s = 0;
    need_s = M;
    nsel = 0;
  }
  __syncthreads();
  for (int pass = 0; pass < 8; ++pass) {
    const int shift = 56 - 8 * pass;
    for (int b = tid; b < 256; b += 1024) hist[b] = 0;
    __syncthreads();
    const uint64_t prefix = prefix_s;
    for (int i = tid; i < g.NV; i += 1024) {
      const uint64_t k = splitmix64(seed | (uint32_t)i);
      if (pass == 0 || (k >> (shift + 8)) == (prefix >> (shift + 8)))
        atomicAdd(&hist[(int)((k >> shift) & 255)], 1);
    }
    __syncthreads();
    if (tid == 0) {
      int need = need_s, cum = 0, digit = 255;
      for (int b = 0; b < 256; ++b) {
        if (cum + hist[b] >= need) {
          digit = b;
          break;
        }
        cum += hist[b];
      }
      need_s = need - cum;
      prefix_s = prefix | ((uint64_t)digit << shift);
    }
    __syncthreads();
  }
  const uint64_t kth = prefix_s;  // the M-th smallest key
  for (int i = tid; i < g.NV; i += 1024) {
    const uint64_t k = splitmix64(seed | (uint32_t)i);
    if (k <= kth) {
      const int slot = atomicAdd(&nsel, 1);
      if (slot < M) {
        sel_key[slot] = k;
        sel_row[slot] = i;
      }
    }
  }
  __syncthreads();
  if (tid < M) {
    const uint64_t k = sel_key[tid];
    int rank = 0;
    for (int o = 0; o < M; ++o) rank += sel_key[o] < k;
    w.probes[(size_t)bh * g.M + rank] = g.ntext + sel_row[tid];
    w.pw[(size_t)bh * g.M + rank] = (float)g.NV / (float)M;
  }
  if (tid == 0) {
    w.nprobes[bh] = M;
    w.stats[(size_t)bh * 16 + ST_NPROBES] = M;
  }
}

// Weights of imported probes: coverage weights w_p = |G_a| / m_a for the
// stratified rule, n_v / (number of probes) for the others.
__global__ __launch_bounds__(256) void k_probe_weights(Geom g, Work w) {
  const int bh = blockIdx.x, tid = threadIdx.x;
  const int np = w.nprobes[bh];
  if (g.probe_rule != SPARSEPR_PROBES_STRATIFIED) {
    for (int p = tid; p < np; p += 256) w.pw[(size_t)bh * g.M + p] = (float)g.NV / (float)np;
    if (tid == 0) w.stats[(size_t)bh * 16 + ST_NPROBES] = np;
    return;
  }
  const int32_t* lab = w.labq + (size_t)bh * g.N;
  const int32_t* oq = w.offq + (size_t)bh * (g.CQt + 1);
  for (int p = tid; p < np; p += 256) {
    const int a = lab[w.probes[(size_t)bh * g.M + p]];
    int m = 0;
    for (int t = 0; t < np; ++t) m += (lab[w.probes[(size_t)bh * g.M + t]] == a);
    w.pw[(size_t)bh * g.M + p] = (float)(oq[a + 1] - oq[a]) / (float)m;
  }
  if (tid == 0) w.stats[(size_t)bh * 16 + ST_NPROBES] = np;
}

// Final per-head counters: k-means assignments performed, nonempty groups.
__global__ __launch_bounds__(256) void k_plan_stats(Geom g, Work w, int with_kmeans, int iters) {
  __shared__ int red[2][4];
  const int bh = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int32_t* oq = w.offq + (size_t)bh * (g.CQt + 1);
  const int32_t* ok = w.offk + (size_t)bh * (g.CKt + 1);
  int nq = 0, nk = 0;
  for (int a = tid; a < g.CQt; a += 256) nq += oq[a + 1] > oq[a];
  for (int b = tid; b < g.CKt; b += 256) nk += ok[b + 1] > ok[b];
  nq = wave_sum_i(nq);
  nk = wave_sum_i(nk);
  if (lane == 0) {
    red[0][wv] = nq;
    red[1][wv] = nk;
  }
  __syncthreads();
  if (tid == 0) {
    int64_t* st = w.stats + (size_t)bh * 16;
    st[ST_NE_Q] = red[0][0] + red[0][1] + red[0][2] + red[0][3];
    st[ST_NE_K] = red[1][0] + red[1][1] + red[1][2] + red[1][3];
    if (with_kmeans) {
      for (int sel = 0; sel < 2; ++sel) {
        const int32_t* chg = w.kmstate + (size_t)bh * 2 * (g.T + 1) + sel * (g.T + 1);
        int n = 1;
        for (int it = 1; it < iters && chg[it - 1] != 0; ++it) ++n;
        st[sel == 0 ? ST_ITK : ST_ITQ] = n;
      }
      int64_t rescans = 0;
      for (int e = 0; e < 2 * g.T; ++e) rescans += w.km_fbcnt[(size_t)bh * 2 * g.T + e];
      st[ST_RESCAN] = rescans;
    }
  }
}

__global__ void k_zero_routed(Geom g, Work w) {
  const int bh = blockIdx.x;
  if (threadIdx.x == 0) {
    w.stats[(size_t)bh * 16 + ST_ROUTED_PAIRS] = 0;
  }
}

// ---------------------------------------------------------------------------
// Host launchers
// ---------------------------------------------------------------------------

static void run_sort(const KmArgs& a, int BH, int it, hipStream_t s) {
  const int shm = (a.C + 1 + 17) * (int)sizeof(int);
  k_sort_hist<<<dim3(a.nblk, BH), 256, a.C * sizeof(int), s>>>(a, it);
  k_sort_scan<<<BH, 1024, shm, s>>>(a, it);
  k_sort_scatter<<<dim3(a.nblk, BH), 256,
                   (size_t)kScatterWaves * (sort_scatter_cstride(a.C) + 64) * sizeof(int), s>>>(a, it);
}

static void assign_step(const Geom& g, const KmArgs& a, int it, hipStream_t s) {
  const int BH = g.BH;
  // the first assignment's operands; later ones come from k_km_update
  if (it == 0) k_km_prep_cent<<<dim3((a.CP + 63) / 64, BH), 256, 0, s>>>(a, it);
  const dim3 grid((a.n + 255) / 256, BH);
  if (a.RP == 16)
    k_km_assign_mfma<16><<<grid, 256, 0, s>>>(a, it);
  else if (a.RP == 32)
    k_km_assign_mfma<32><<<grid, 256, 0, s>>>(a, it);
  else if (a.RP == 48)
    k_km_assign_mfma<48><<<grid, 256, 0, s>>>(a, it);
  else if (a.RP == 64)
    k_km_assign_mfma<64><<<grid, 256, 0, s>>>(a, it);
  else if (a.RP == 80)
    k_km_assign_mfma<80><<<grid, 256, 0, s>>>(a, it);
  else if (a.RP == 96)
    k_km_assign_mfma<96><<<grid, 256, 0, s>>>(a, it);
  else if (a.RP == 112)
    k_km_assign_mfma<112><<<grid, 256, 0, s>>>(a, it);
  else
    k_km_assign_mfma<128><<<grid, 256, 0, s>>>(a, it);
}

static void run_kmeans(const Geom& g, const KmArgs& a0, hipStream_t s, bool warm) {
  const int BH = g.BH;
  KmArgs a = a0;
  a.RP = (a.R + 15) / 16 * 16;
  a.CP = (a.C + 31) / 32 * 32;
  // warm start: the centroids left by the previous call are the initial ones
  if (!warm) k_km_init<<<dim3((a.C * a.R + 255) / 256, BH), 256, 0, s>>>(a);
  a.warm = warm;
  const int iters = warm ? g.T_warm : g.T;
  for (int it = 0; it < iters; ++it) {
    assign_step(g, a, it, s);
    run_sort(a, BH, it, s);
    k_km_update<<<dim3((a.C + 3) / 4, BH), 256, 0, s>>>(a, it);
  }
  if (a.row0 > 0) k_prefix_group<<<dim3((a.row0 + 255) / 256, BH), 256, 0, s>>>(a);
}

template <int D>
static void project(const Geom& g, const Work& w, const void* x, const float* F, int R, int query,
                    int rms, float eps, float* phi, hipStream_t s) {
  const dim3 grid((g.NV + 64 * PROJ_CHUNKS - 1) / (64 * PROJ_CHUNKS), g.BH);
  const int RP = (R + 15) / 16 * 16;
  auto run = [&](auto maxr, auto mf) {
    k_project<D, decltype(maxr)::value, decltype(mf)::value><<<grid, 256, 0, s>>>(
        x, g, F, R, query, rms, eps, phi, w.stats, w.km_xhi, w.km_xlo, w.km_xn, RP);
  };
  auto by_rank = [&](auto mf) {
    if (R <= 32)
      run(std::integral_constant<int, 32>{}, mf);
    else if (R <= 64)
      run(std::integral_constant<int, 64>{}, mf);
    else
      run(std::integral_constant<int, 128>{}, mf);
  };
  if (g.bf16)
    by_rank(std::true_type{});
  else
    by_rank(std::false_type{});
}

// The semantic partitions cluster the raw rows: coordinates phi = I^T x.
__global__ __launch_bounds__(256) void k_identity_basis(float* F, double* gram, float* evals, int D) {
  const int bh = blockIdx.x;
  for (int i = threadIdx.x; i < D * D; i += 256) {
    F[(size_t)bh * D * D + i] = (i / D == i % D) ? 1.f : 0.f;
    gram[(size_t)bh * D * D + i] = 0.0;
  }
  for (int i = threadIdx.x; i < D; i += 256) evals[(size_t)bh * D + i] = 0.f;
}

template <int D>
static void plan_d(const Geom& g, const Work& w, const void* q, const void* k, hipStream_t s,
                   bool warm) {
  const int BH = g.BH;
  k_plan_init<<<BH, 64, 0, s>>>(g, w);
  // Key-response coordinates and the paired K/V partition (Sec. 4.1, App. B.1);
  // the semantic partition clusters the raw keys instead (Sec. 3.1)
  if (g.partition == SPARSEPR_PARTITION_SEMANTIC) {
    k_identity_basis<<<BH, 256, 0, s>>>(w.fk, w.gram_k, w.evals_k, D);
  } else {
    k_key_metric<D><<<dim3(D / 16, BH), 256, 0, s>>>(q, g, w.gram_k);
    k_eig_basis<D><<<BH, 1024, 0, s>>>(w.gram_k, g.rk, 1e-6f, w.fk, w.evals_k, w.eigscr, w.stats);
  }
  project<D>(g, w, k, w.fk, g.rk, 0, 0, 0.f, w.phik, s);
  KmArgs ak{w.phik, w.centk, w.labk, w.permk, w.offk, w.blkhist, w.kmstate, g.NV, g.ntext, g.N,
            g.rk, g.CK, g.CKt + 1, g.nsort_blk, g.cmax, 0, g.T,
            w.km_xhi, w.km_xlo, w.km_xn, w.km_chi, w.km_clo, w.km_cu, w.km_cn3, w.km_fbcnt, 0, 0};
  run_kmeans(g, ak, s, warm);
  // Query-response coordinates from the K/V groups (App. B.2)
  k_group_mean<<<dim3((g.CK + 3) / 4, BH), 256, 0, s>>>(k, g, w.permk, w.offk, g.CK, g.CKt + 1,
                                                         w.kbar, 0);
  if (g.partition == SPARSEPR_PARTITION_RESPONSE) {
    k_query_metric<D><<<dim3(D * D / 2048, BH), 256, 0, s>>>(w.kbar, w.offk, g, w.gram_q);
    k_eig_basis<D><<<BH, 1024, 0, s>>>(w.gram_q, g.rq, 1e-6f, w.fq, w.evals_q, w.eigscr, w.stats);
    project<D>(g, w, q, w.fq, g.rq, 1, 1, g.eps_q, w.phiq, s);
  } else {
    // semantic query groups: k-means on the raw queries
    k_identity_basis<<<BH, 256, 0, s>>>(w.fq, w.gram_q, w.evals_q, D);
    project<D>(g, w, q, w.fq, g.rq, 1, 0, 0.f, w.phiq, s);
  }
  KmArgs aq{w.phiq, w.centq, w.labq, w.permq, w.offq, w.blkhist, w.kmstate, g.NV, g.ntext, g.N,
            g.rq, g.CQ, g.CQt + 1, g.nsort_blk, g.cmax, 1, g.T,
            w.km_xhi, w.km_xlo, w.km_xn, w.km_chi, w.km_clo, w.km_cu, w.km_cn3, w.km_fbcnt, 0, 0};
  run_kmeans(g, aq, s, warm);
  k_group_mean<<<dim3((g.CQ + 3) / 4, BH), 256, 0, s>>>(q, g, w.permq, w.offq, g.CQ, g.CQt + 1,
                                                         w.qbar, 1);
  // Routing (Sec. 4.3)
  k_route_prio<D><<<dim3((g.CQ + 63) / 64, BH), 256, 0, s>>>(w.qbar, w.kbar, g, w.offq, w.offk,
                                                             w.prio, w.forced);
  if (g.routing == SPARSEPR_ROUTING_TOP_P) {
    int np2 = 1;
    while (np2 < g.CK) np2 <<= 1;
    k_route_topp<<<dim3(g.CQ, BH), 256, (size_t)np2 * 8, s>>>(g, w, np2);
  }
  k_sel_init<<<BH, 256, 0, s>>>(g, w);
  // about 2048 blocks over all heads, each taking rows of one head
  const int gsel = std::max(1, std::min(g.CQ, (2048 + BH - 1) / BH));
  for (int p = 0; p < kSelPasses; ++p) {
    k_sel_hist<<<dim3(gsel, BH), 256, 0, s>>>(g, w, p);
    k_sel_choose<<<BH, 256, 0, s>>>(g, w, p);
  }
  const int64_t ncell_t = (int64_t)g.CQt * g.CKt;
  const int gmark = (int)std::min<int64_t>(std::max<int64_t>((ncell_t + 4095) / 4096, 1), 512);
  k_sel_mark<<<dim3(gmark, BH), 256, 0, s>>>(g, w);
  k_ranges<<<dim3((g.CQt + 3) / 4, BH), 256, 0, s>>>(g, w);
  k_chunks<<<BH, 1024, (g.CQt + 1 + 17) * sizeof(int), s>>>(g, w);
  // Probes (App. A.2)
  if (g.M > 0) {
    if (g.probe_rule == SPARSEPR_PROBES_STRATIFIED) {
      k_probe_d2<<<dim3((g.NV + 127) / 128, BH), 128, (g.rq % 4 == 0) ? (size_t)128 * (g.rq + 4) * 4 : 0, s>>>(g, w);
      k_probe_select<<<BH, 1024, (4 * g.CQ + 1 + 17) * sizeof(int), s>>>(g, w);
    } else if (g.probe_rule == SPARSEPR_PROBES_UNIFORM) {
      k_probe_uniform<<<BH, 256, 0, s>>>(g, w);
    } else {
      k_probe_random<<<BH, 1024, 0, s>>>(g, w);
    }
  }
  k_plan_stats<<<BH, 256, 0, s>>>(g, w, 1, warm ? g.T_warm : g.T);
}

void launch_plan(const Geom& g, const Work& w, const void* q, const void* k, hipStream_t s,
                 bool warm) {
  if (g.d == 64)
    plan_d<64>(g, w, q, k, s, warm);
  else
    plan_d<128>(g, w, q, k, s, warm);
}

void launch_rebuild(const Geom& g, const Work& w, int bh, hipStream_t s) {
  (void)bh;  // every head is rebuilt; heads not imported reproduce their own data
  const int BH = g.BH;
  KmArgs ak{nullptr, nullptr, w.labk, w.permk, w.offk, w.blkhist, w.kmstate, g.N, 0, g.N,
            0, g.CKt, g.CKt + 1, g.nsort_blk_full, g.cmax, 0, g.T,
            nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, 0};
  run_sort(ak, BH, -1, s);
  KmArgs aq{nullptr, nullptr, w.labq, w.permq, w.offq, w.blkhist, w.kmstate, g.N, 0, g.N,
            0, g.CQt, g.CQt + 1, g.nsort_blk_full, g.cmax, 1, g.T,
            nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, 0};
  run_sort(aq, BH, -1, s);
  k_zero_routed<<<BH, 64, 0, s>>>(g, w);
  k_ranges<<<dim3((g.CQt + 3) / 4, BH), 256, 0, s>>>(g, w);
  k_chunks<<<BH, 1024, (g.CQt + 1 + 17) * sizeof(int), s>>>(g, w);
  if (g.M > 0) k_probe_weights<<<BH, 256, 0, s>>>(g, w);
  k_plan_stats<<<BH, 256, 0, s>>>(g, w, 0, g.T);
}

}  // namespace sparsepr
