// Probe-fitted residual reconstruction of the SparsePR operator for gfx950
// (Sec. 4.2; App. A.3): the weighted probe statistics, the residual basis and
// ridge solve, and the correction + restore of every row to the original order
// (eq. final_reconstructed_output), with the probe rows taking their exact
// dense rows.
#include <hip/hip_runtime.h>
#include <math.h>

#include <type_traits>

#include "device_utils.hpp"
#include "sparsepr_internal.hpp"
#include "jacobi_lds.hpp"
#include "tridiag_eig.hpp"

namespace sparsepr {

// ---------------------------------------------------------------------------
// Probe-fitted residual fit (Sec. 4.2; App. A.3), one block of 1024 threads
// per head:
//   alpha_p = w_p / sum w;  mu_x, mu_R weighted means;
//   s_x = sqrt(sum alpha (x - mu_x)^2 + eps);  xbar = (x - mu_x)/s_x;
//   Rbar = R - mu_R;  w~_p = M w_p / sum w;
//   Psi = leading r eigenvectors of Rbar^T W Rbar (right singular vectors of
//         W^1/2 Rbar), keeping sigma > 1e-6 sigma_1;
//   (xbar^T W xbar + lambda I) Y = xbar^T W (Rbar Psi)   (Cholesky),
// so Y = B_lambda Psi and the correction of row i is xbar_i Y Psi^T + mu_R.
// ---------------------------------------------------------------------------

// Per-head scratch of the fit: xbar [M][D], rbar [M][D], rbar*Psi [M][r],
// rhs [D][r], w~ [M] (all double).
struct FitScratch {
  double *xb, *rb, *rp, *rhs, *wt;
};

__device__ __forceinline__ FitScratch fit_scratch(const Geom& g, const Work& w, int bh) {
  const size_t D = g.dv, M = g.M, r = g.r;
  double* base = w.fitscr + (size_t)bh * (2 * M * D + M * r + D * r + M);
  FitScratch f;
  f.xb = base;
  f.rb = f.xb + M * D;
  f.rp = f.rb + M * D;
  f.rhs = f.rp + M * r;
  f.wt = f.rhs + D * r;
  return f;
}

// Weighted statistics of the probes (eqs. app_normalized_weights ...
// app_regression_weights): mu_x, mu_R, s_x, xbar, Rbar and w~.
template <int D>
__global__ __launch_bounds__(256) void k_fit_prep(Geom g, Work w) {
  __shared__ double swsh;
  const int bq = blockIdx.x, bh = bq % g.BH, tid = threadIdx.x;
  const int np = w.nprobes[bh];
  const int r = g.r;
  float* fv = w.fitv + (size_t)bq * 3 * D;
  float* Y = w.fity + (size_t)bq * D * r;
  float* Psi = w.fitpsi + (size_t)bq * D * r;
  for (int i = tid; i < D * r; i += 256) {
    Y[i] = 0.f;
    Psi[i] = 0.f;
  }
  if (np == 0) {
    for (int c = tid; c < D; c += 256) {
      fv[c] = 0.f;
      fv[D + c] = 1.f;
      fv[2 * D + c] = 0.f;
    }
    if (tid == 0) w.stats[(size_t)bh * 16 + ST_FIT_RANK] = 0;
    return;
  }
  const FitScratch f = fit_scratch(g, w, bq);
  const int32_t* pr = w.probes + (size_t)bh * g.M;
  const float* pwt = w.pw + (size_t)bh * g.M;
  const float* osp = w.osp + (size_t)bq * g.N * D;
  const float* odp = w.odp + (size_t)bq * g.M * D;
  if (tid < 64) {
    // fixed order: lane-strided partial sums, then the wave sum
    double s = 0.0;
    for (int p = tid; p < np; p += 64) s += (double)pwt[p];
    s = wave_sum_d(s);
    if (tid == 0) swsh = s;
  }
  __syncthreads();
  const double sw = swsh;
  for (int p = tid; p < np; p += 256) f.wt[p] = (double)np * (double)pwt[p] / sw;
  for (int c = tid; c < D; c += 256) {
    double mx = 0.0, mr = 0.0;
#pragma unroll 8
    for (int p = 0; p < np; ++p) {
      const double al = (double)pwt[p] / sw;
      const double x = osp[(size_t)pr[p] * D + c];
      mx += al * x;
      mr += al * ((double)odp[(size_t)p * D + c] - x);
    }
    double vx = 0.0;
#pragma unroll 8
    for (int p = 0; p < np; ++p) {
      const double al = (double)pwt[p] / sw;
      const double t = (double)osp[(size_t)pr[p] * D + c] - mx;
      vx += al * t * t;
    }
    const double sx = sqrt(vx + (double)g.eps_x);
#pragma unroll 8
    for (int p = 0; p < np; ++p) {
      const double x = osp[(size_t)pr[p] * D + c];
      f.xb[(size_t)p * D + c] = (x - mx) / sx;
      f.rb[(size_t)p * D + c] = ((double)odp[(size_t)p * D + c] - x) - mr;
    }
    fv[c] = (float)mx;
    fv[D + c] = (float)sx;
    fv[2 * D + c] = (float)mr;
  }
}

// The two weighted Gram matrices of the fit, one 32 x 32 tile per block:
// which = 0: H = Rbar^T W Rbar (its eigenvectors are the right singular
// vectors of W^1/2 Rbar, eq. app_probe_residual_basis); which = 1:
// S = xbar^T W xbar + lambda I (eq. app_ridge_closed_form).
template <int D>
__global__ __launch_bounds__(256) void k_fit_gram(Geom g, Work w) {
  constexpr int PB = 64;
  __shared__ double sa[PB][33], sb[PB][33];
  __shared__ double swt[PB];
  const int bq = blockIdx.z, bh = bq % g.BH, which = blockIdx.y, tid = threadIdx.x;
  const int np = w.nprobes[bh];
  if (np == 0) return;
  const int ti = blockIdx.x / (D / 32), tj = blockIdx.x % (D / 32);
  const FitScratch f = fit_scratch(g, w, bq);
  const double* src = which == 0 ? f.rb : f.xb;
  const int li = tid / 8, lj = (tid % 8) * 4;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int p0 = 0; p0 < np; p0 += PB) {
    const int pn = min(PB, np - p0);
    __syncthreads();
    for (int i = tid; i < pn * 32; i += 256) {
      const int p = i / 32, c = i % 32;
      sa[p][c] = src[(size_t)(p0 + p) * D + ti * 32 + c];
      sb[p][c] = src[(size_t)(p0 + p) * D + tj * 32 + c];
    }
    for (int p = tid; p < pn; p += 256) swt[p] = f.wt[p0 + p];
    __syncthreads();
    for (int p = 0; p < pn; ++p) {
      const double a = swt[p] * sa[p][li];
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] += a * sb[p][lj + e];
    }
  }
  double* G = w.fitgram + ((size_t)bq * 2 + which) * D * D;
  const int i = ti * 32 + li;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int j = tj * 32 + lj + e;
    G[(size_t)i * D + j] = acc[e] + ((which == 1 && i == j) ? (double)g.ridge : 0.0);
  }
}

// Residual subspace and ridge solve, one block of 1024 threads per head:
// Psi = leading r eigenvectors of H with sigma > 1e-6 sigma_1 (tridiagonal
// solver in LDS, or cyclic Jacobi when its check fails); then
// (xbar^T W xbar + lambda I) Y = xbar^T W (Rbar Psi) by Cholesky, so
// Y = B_lambda Psi and the correction of row i is xbar_i Y Psi^T + mu_R.
// T is the eigensolver's precision.  Double A and V of a 128 x 128 problem do not
// both fit in LDS; V (VG) then lives in the head's global scratch.
template <int D, typename T>
__global__ __launch_bounds__(1024) void k_fit_solve(Geom g, Work w) {
  constexpr int LD = D + 1, LV = jacobi_vt_ld<D>();
  constexpr bool VG = (size_t)D * (LD + LV) * sizeof(T) > 140 * 1024;
  constexpr size_t JAC = (size_t)D * (LD + (VG ? 0 : LV)) * sizeof(T),
                   CHOL = (size_t)D * D * sizeof(double);
  __shared__ __attribute__((aligned(16))) unsigned char smem[JAC > CHOL ? JAC : CHOL];
  __shared__ JacobiRot<T> rot[D / 2];
  __shared__ TriWork<D, T, 1024> tw;
  __shared__ int order[D];
  __shared__ int flag, rank_s, fail;
  const int bq = blockIdx.x, bh = bq % g.BH, tid = threadIdx.x;
  const int np = w.nprobes[bh];
  if (np == 0) return;
  const int r = g.r;
  float* Y = w.fity + (size_t)bq * D * r;
  float* Psi = w.fitpsi + (size_t)bq * D * r;
  const FitScratch f = fit_scratch(g, w, bq);
  const double* H = w.fitgram + ((size_t)bq * 2 + 0) * D * D;
  const double* Sg = w.fitgram + ((size_t)bq * 2 + 1) * D * D;
  T* Am = (T*)smem;
  T* Vm = VG ? (T*)(w.fitvec + (size_t)bq * D * LV) : Am + D * LD;  // transposed (jacobi_eig_lds)
  if (g.ridge_only) {
    // ridge estimator alone (Table probe_estimator_ablation): Psi = I
    for (int e = tid; e < D * D; e += 1024) Vm[(e / D) * LV + (e % D)] = (e / D == e % D) ? T(1) : T(0);
    if (tid < D) order[tid] = tid;
    if (tid == 0) {
      rank_s = D;
      fail = 0;
    }
    __syncthreads();
  } else {
    for (int e = tid; e < D * D; e += 1024) Am[(e / D) * LD + (e % D)] = (T)H[e];
    __syncthreads();
    tri_reduce<D, T, 1024>(Am, tw);
    tri_eigvals<D, T, 1024>(tw);
    if (tid == 0) {
      // rank: the leading t < r with sigma_t > 1e-6 sigma_1.  In double the
      // float eigenvalues of the multisection cannot place an eigenvalue
      // near 1e-12 lambda_1, so a retained range reaching below 1e-5
      // lambda_1 is left to the Jacobi solve.
      const double l1 = tw.lamf[0];
      const double s1 = l1 > 0.0 ? sqrt(l1) : 0.0;
      int rk = 0;
      bool amb = false;
      for (int t = 0; t < r && t < D; ++t) {
        const double lt = tw.lamf[t];
        if (sizeof(T) == 8 && !(lt >= 1e-5 * l1)) amb = true;
        const double st = lt > 0.0 ? sqrt(lt) : 0.0;
        if (s1 > 0.0 && st > 1e-6 * s1)
          ++rk;
        else
          break;
      }
      rank_s = amb ? -1 : rk;
      fail = 0;
    }
    __syncthreads();
    if (rank_s >= 0) tri_vectors<D, T, 1024>(tw, Vm, LV, rank_s, w.eigscr + (size_t)bq * 4 * D * D);
    if (rank_s >= 0 && tw.ok) {
      tri_back<D, T, 1024>(Am, tw, Vm, LV, rank_s);
      if (tid < D) order[tid] = tid;
    } else {
      if (tid == 0)
        atomicOr((unsigned long long*)&w.stats[(size_t)bh * 16 + ST_FLAGS], (unsigned long long)SPARSEPR_FLAG_EIG_JACOBI);
      for (int e = tid; e < D * D; e += 1024) Am[(e / D) * LD + (e % D)] = (T)H[e];
      __syncthreads();
      jacobi_eig_lds<D, T, 1024>(Am, Vm, rot, &flag, sizeof(T) == 8 ? T(1e-12) : T(1e-4));
      if (tid < D) {
        // a NaN diagonal (non-finite input) ranks as -inf, so the ranks stay
        // a permutation and every order[] entry is written
        const T li = eig_rank_key(Am[tid * LD + tid]);
        int rank = 0;
        for (int j = 0; j < D; ++j) {
          const T lj = eig_rank_key(Am[j * LD + j]);
          rank += (lj > li) || (lj == li && j < tid);
        }
        order[rank] = tid;
      }
      __syncthreads();
      if (tid == 0) {
        const double l1 = Am[order[0] * LD + order[0]];
        const double s1 = l1 > 0.0 ? sqrt(l1) : 0.0;
        int rk = 0;
        for (int t = 0; t < r && t < D; ++t) {
          const double lt = Am[order[t] * LD + order[t]];
          const double st = lt > 0.0 ? sqrt(lt) : 0.0;
          if (s1 > 0.0 && st > 1e-6 * s1)
            ++rk;
          else
            break;
        }
        rank_s = rk;
      }
    }
    __syncthreads();
  }
  const int rk = rank_s;
  for (int i = tid; i < D * rk; i += 1024) {
    const int row = i / rk, t = i % rk;
    Psi[row * r + t] = (float)Vm[order[t] * LV + row];
  }
  for (int i = tid; i < np * rk; i += 1024) {
    const int p = i / rk, t = i % rk;
    double acc = 0.0;
    for (int c = 0; c < D; ++c) acc += f.rb[(size_t)p * D + c] * (double)Vm[order[t] * LV + c];
    f.rp[(size_t)p * r + t] = acc;
  }
  __syncthreads();
  // rhs = xbar^T W (Rbar Psi): the probe weights and Rbar Psi are staged in
  // the LDS (free again here) when they fit; each sum runs over the probes in
  // order either way
  double* rps = (double*)smem;  // [np][rk], then [np] weights
  const bool staged = (size_t)np * (rk + 1) * sizeof(double) <= sizeof(smem);
  if (staged) {
    for (int i = tid; i < np * rk; i += 1024) rps[i] = f.rp[(size_t)(i / rk) * r + i % rk];
    for (int p = tid; p < np; p += 1024) rps[np * rk + p] = f.wt[p];
  }
  __syncthreads();
  for (int i = tid; i < D * rk; i += 1024) {
    const int c = i / rk, t = i % rk;
    double acc = 0.0;
    if (staged) {
#pragma unroll 8
      for (int p = 0; p < np; ++p) acc += rps[np * rk + p] * f.xb[(size_t)p * D + c] * rps[p * rk + t];
    } else {
      for (int p = 0; p < np; ++p) acc += f.wt[p] * f.xb[(size_t)p * D + c] * f.rp[(size_t)p * r + t];
    }
    f.rhs[(size_t)c * r + t] = acc;
  }
  // Cholesky S = L L^T in LDS (double), right-looking: at step j every
  // thread takes sqrt(S_jj) itself, scales its part of column j, and after
  // one barrier updates the lower triangle of the trailing block by column
  // (k = tid % D) and rows (i = j + 1 + tid / D + NT/D * u, i >= k).
  double* S = (double*)smem;
  __syncthreads();
  for (int e = tid; e < D * D; e += 1024) S[e] = Sg[e];
  __syncthreads();
  {
    constexpr int RS = 1024 / D;  // row strips
    const int kc = tid % D, i0 = tid / D;
    for (int j = 0; j < D; ++j) {
      const double dj = S[j * D + j];
      const double ljj = dj > 0.0 ? sqrt(dj) : 1.0;
      for (int i = j + 1 + tid; i < D; i += 1024) S[i * D + j] /= ljj;
      __syncthreads();
      if (tid == 0) {
        if (!(dj > 0.0)) fail = 1;
        S[j * D + j] = ljj;
      }
      if (kc > j) {
        const double lk = S[kc * D + j];
        for (int i = j + 1 + i0; i < D; i += RS)
          if (i >= kc) S[i * D + kc] -= S[i * D + j] * lk;
      }
      __syncthreads();
    }
  }
  // L^T into the strict upper triangle (S[i][k] = L[k][i], k > i), so that
  // both triangular solves below read rows
  for (int e = tid; e < D * D; e += 1024) {
    const int i = e / D, k = e % D;
    if (k > i) S[i * D + k] = S[k * D + i];
  }
  __syncthreads();
  // L L^T Y = rhs: wave t solves right-hand side t, lane l holding rows
  // l, l + 64, ... in registers.  Both solves subtract each solved unknown
  // from the rows still open: L y = b from the first row down (row i of the
  // upper copy holds column i of L), then L^T x = y from the last row up
  // (row i of L).
  {
    constexpr int U = (D + 63) / 64;
    static_assert(U <= 2, "rows per lane");
    const int lane = tid & 63;
    for (int wv = tid >> 6; wv < rk && !fail; wv += 1024 / 64) {
      double y[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = lane + 64 * u;
        y[u] = i < D ? f.rhs[(size_t)i * r + wv] : 0.0;
      }
      for (int i = 0; i < D; ++i) {
        const double yi = tri_readlane(U > 1 && i >= 64 ? y[U - 1] : y[0], i & 63) / S[i * D + i];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int k = lane + 64 * u;
          if (k > i && k < D) y[u] -= S[i * D + k] * yi;
          if (k == i) y[u] = yi;
        }
      }
      for (int i = D - 1; i >= 0; --i) {
        const double xi = tri_readlane(U > 1 && i >= 64 ? y[U - 1] : y[0], i & 63) / S[i * D + i];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int k = lane + 64 * u;
          if (k < i) y[u] -= S[i * D + k] * xi;
          if (k == i) y[u] = xi;
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = lane + 64 * u;
        if (i < D) Y[i * r + wv] = (float)y[u];
      }
    }
  }
  if (tid == 0) {
    int64_t* st = w.stats + (size_t)bh * 16;
    st[ST_FIT_RANK] = rk;
    if (fail) atomicOr((unsigned long long*)&st[ST_FLAGS], (unsigned long long)SPARSEPR_FLAG_FIT_NOT_PD);
  }
}

// Correction and restore (eq. probe_residual_estimate and
// final_reconstructed_output): out_i = x_i + mu_R + ((x_i - mu_x)/s_x) Y Psi^T
// for the video rows; dense-prefix rows keep their (exact) sparse output.
// Probe rows are overwritten afterwards by k_probe_scatter.
constexpr int CORR_CHUNKS = 8;

template <int D>
__global__ __launch_bounds__(256) void k_correct(Geom g, Work w, void* out) {
  // CORR_CHUNKS chunks of 64 rows per block.  Thread (row = tid / 4,
  // quarter = tid % 4) owns the columns [quarter * D/4, quarter * D/4 + D/4)
  // of its row, held in registers; its partial of t = xbar Y
  // (Y = B_lambda Psi) over those columns is summed with the other quarters'
  // by lane exchange within the quad, and it forms its columns of
  // x + mu_R + t Psi^T.  The rank is processed in slices of 16 directions,
  // staged in LDS once per block when the rank fits one slice.
  constexpr int CW = D / 4, RS = 16;
  __shared__ __attribute__((aligned(16))) float fy[D][RS];
  __shared__ __attribute__((aligned(16))) float fp[D][RS];
  __shared__ __attribute__((aligned(16))) float fvs[3][D];  // mu_x, 1 / s_x, mu_R
  const int bq = blockIdx.y, bh = bq % g.BH, tid = threadIdx.x;
  const int r = g.r;
  const int rw = tid >> 2, qtr = tid & 3;
  const float* fv = w.fitv + (size_t)bq * 3 * D;
  const float* Y = w.fity + (size_t)bq * D * r;
  const float* Psi = w.fitpsi + (size_t)bq * D * r;
  const bool one_slice = r <= RS;
  auto stage = [&](int t0) {
    const int tn = min(RS, r - t0);
    for (int i = tid; i < D * RS; i += 256) {
      const int c = i / RS, t = i % RS;
      // 16-byte slot t/4 is XOR-swizzled by the column's quarter, so the
      // four quarters of a quad read different banks
      const int sl = (((t >> 2) ^ (c / CW)) & 3) * 4 + (t & 3);
      fy[c][sl] = t < tn ? Y[c * r + t0 + t] : 0.f;
      fp[c][sl] = t < tn ? Psi[c * r + t0 + t] : 0.f;
    }
  };
  // mu_x, 1 / s_x (one division per column and block, not per row), mu_R
  for (int i = tid; i < 3 * D; i += 256) fvs[i / D][i % D] = i / D == 1 ? 1.f / fv[i] : fv[i];
  if (one_slice) stage(0);
  __syncthreads();
  for (int chunk = 0; chunk < CORR_CHUNKS; ++chunk) {
    const int row = (blockIdx.x * CORR_CHUNKS + chunk) * 64 + rw;
    if ((blockIdx.x * CORR_CHUNKS + chunk) * 64 >= g.N) break;  // uniform over the block
    const bool valid = row < g.N;
    const bool text = row < g.ntext;
    const float* src = w.osp + ((size_t)bq * g.N + (valid ? row : 0)) * D + qtr * CW;
    float x[CW], acc[CW];
#pragma unroll
    for (int c4 = 0; c4 < CW / 4; ++c4) {
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (valid) v = *(const float4*)(src + 4 * c4);
      x[4 * c4] = v.x;
      x[4 * c4 + 1] = v.y;
      x[4 * c4 + 2] = v.z;
      x[4 * c4 + 3] = v.w;
    }
#pragma unroll
    for (int c = 0; c < CW; ++c) acc[c] = 0.f;
    for (int t0 = 0; t0 < r; t0 += RS) {
      if (!one_slice) {
        __syncthreads();
        stage(t0);
        __syncthreads();
      }
      float tp[RS];
#pragma unroll
      for (int t = 0; t < RS; ++t) tp[t] = 0.f;
#pragma unroll
      for (int c = 0; c < CW; ++c) {
        const int col = qtr * CW + c;
        const float xb = (x[c] - fvs[0][col]) * fvs[1][col];
#pragma unroll
        for (int t4 = 0; t4 < RS / 4; ++t4) {
          const float4 y4 = *(const float4*)&fy[col][(t4 ^ qtr) * 4];
          tp[4 * t4] = fmaf(xb, y4.x, tp[4 * t4]);
          tp[4 * t4 + 1] = fmaf(xb, y4.y, tp[4 * t4 + 1]);
          tp[4 * t4 + 2] = fmaf(xb, y4.z, tp[4 * t4 + 2]);
          tp[4 * t4 + 3] = fmaf(xb, y4.w, tp[4 * t4 + 3]);
        }
      }
#pragma unroll
      for (int t = 0; t < RS; ++t) {
        tp[t] += tri_dpp<kDppXor1>(tp[t]);
        tp[t] += tri_dpp<kDppXor2>(tp[t]);
      }
#pragma unroll
      for (int c = 0; c < CW; ++c) {
        const int col = qtr * CW + c;
        float a = acc[c];
#pragma unroll
        for (int t4 = 0; t4 < RS / 4; ++t4) {
          const float4 p4 = *(const float4*)&fp[col][(t4 ^ qtr) * 4];
          a = fmaf(tp[4 * t4], p4.x, a);
          a = fmaf(tp[4 * t4 + 1], p4.y, a);
          a = fmaf(tp[4 * t4 + 2], p4.z, a);
          a = fmaf(tp[4 * t4 + 3], p4.w, a);
        }
        acc[c] = a;
      }
    }
    if (!valid) continue;
    const int64_t dst = q_base(g, bh, bq / g.BH) + (int64_t)row * g.sn + qtr * CW;
    float o[CW];
#pragma unroll
    for (int c = 0; c < CW; ++c) o[c] = text ? x[c] : x[c] + fvs[2][qtr * CW + c] + acc[c];
    if (g.bf16) {
      uint16_t* op = (uint16_t*)out + dst;
#pragma unroll
      for (int c8 = 0; c8 < CW / 8; ++c8) {
        uint32_t wd[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint16_t lo = __builtin_bit_cast(uint16_t, (__bf16)o[c8 * 8 + 2 * e]);
          const uint16_t hi = __builtin_bit_cast(uint16_t, (__bf16)o[c8 * 8 + 2 * e + 1]);
          wd[e] = (uint32_t)lo | ((uint32_t)hi << 16);
        }
        *(uint4*)(op + c8 * 8) = make_uint4(wd[0], wd[1], wd[2], wd[3]);
      }
    } else {
      float* op = (float*)out + dst;
#pragma unroll
      for (int c4 = 0; c4 < CW / 4; ++c4)
        *(float4*)(op + 4 * c4) = make_float4(o[4 * c4], o[4 * c4 + 1], o[4 * c4 + 2], o[4 * c4 + 3]);
    }
  }
}

// Probe rows take their exact dense rows (eq. final_reconstructed_output).
__global__ __launch_bounds__(128) void k_probe_scatter(Geom g, Work w, void* out) {
  const int p = blockIdx.x, bq = blockIdx.y, bh = bq % g.BH, c = threadIdx.x;
  if (p >= w.nprobes[bh] || c >= g.dv) return;
  const int row = w.probes[(size_t)bh * g.M + p];
  const float v = w.odp[((size_t)bq * g.M + p) * g.dv + c];
  const int64_t idx = q_base(g, bh, bq / g.BH) + (int64_t)row * g.sn + c;
  if (g.bf16) {
    const __bf16 b = (__bf16)v;
    ((uint16_t*)out)[idx] = __builtin_bit_cast(uint16_t, b);
  } else {
    ((float*)out)[idx] = v;
  }
}

template <int D>
static void fit_d(const Geom& g, const Work& w0, void* out, hipStream_t s, hipEvent_t* ev) {
  // all G * BH query heads in one launch (view of query head 0, whose [G][BH]
  // arrays continue with the other query heads)
  const int BQ = g.BH * g.G;
  k_fit_prep<D><<<BQ, 256, 0, s>>>(g, w0);
  k_fit_gram<D><<<dim3((D / 32) * (D / 32), 2, BQ), 256, 0, s>>>(g, w0);
  // float inputs (whose outputs are held to float rounding) get the double
  // solve; bf16 inputs the float one
  if (D <= 64 || !g.bf16)
    k_fit_solve<D, double><<<BQ, 1024, 0, s>>>(g, w0);
  else
    k_fit_solve<D, float><<<BQ, 1024, 0, s>>>(g, w0);
  if (ev) (void)hipEventRecord(ev[3], s);
  k_correct<D><<<dim3((g.N + 64 * CORR_CHUNKS - 1) / (64 * CORR_CHUNKS), BQ), 256, 0, s>>>(g, w0, out);
  if (g.M > 0) k_probe_scatter<<<dim3(g.M, BQ), 128, 0, s>>>(g, w0, out);
  if (ev) (void)hipEventRecord(ev[4], s);
}

void launch_fit_correct(const Geom& g, const Work& w0, void* out, hipStream_t s, hipEvent_t* ev) {
  if (g.d == 64)
    fit_d<64>(g, w0, out, s, ev);
  else
    fit_d<128>(g, w0, out, s, ev);
}

}  // namespace sparsepr
