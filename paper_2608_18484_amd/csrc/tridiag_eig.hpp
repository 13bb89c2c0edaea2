// Symmetric eigensolver for the response bases (App. B.1, B.2) and the
// probe-residual basis (App. A.3 eq. app_probe_residual_basis), one block of
// NT threads per D x D matrix, in four stages:
//
//  1. tri_reduce: Householder reduction to tridiagonal form in LDS,
//     A = Q T Q^T with Q = H_0 H_1 ... H_{D-3}; reflector k is stored in
//     column k below the subdiagonal, its scale in beta[k].
//  2. tri_eigvals: every eigenvalue of T by multisection of its Sturm counts
//     in float (NT / D threads per eigenvalue, each counting at one point of
//     the current bracket), sorted descending.
//  3. tri_vectors: for the leading nvec eigenvalues, the twisted
//     factorisation of T - lambda I in double (stationary and progressive
//     pivot chains, each vector's two chains in different waves; twist index
//     at the smallest |gamma|, found by a group of 8 lanes per vector), one
//     Rayleigh-quotient correction lambda += gamma / |z|^2, a second
//     factorisation and the twisted vector (its two sides swept by two lanes
//     of the group).  The vectors' tridiagonal residuals and mutual
//     orthogonality are then checked; ok = 0 reports a numerically repeated
//     eigenvalue (whose twisted vectors coincide) so that the caller can use
//     its Jacobi solver instead.
//  4. tri_back: the vectors are multiplied by Q (reflectors applied last to
//     first), each by a group of NT / D lanes of one wave with no barriers.
//
// The reduction moves O(D^3) words through LDS once, against the O(D^3) per
// sweep of cyclic Jacobi; the tridiagonal stages are O(D^2).
#pragma once
#include <hip/hip_runtime.h>
#include <float.h>
#include <math.h>

namespace sparsepr {

template <int D, typename T, int NT = 1024>
struct TriWork {
  double d[D], e[D], e2[D];  // diagonal, subdiagonal e[i] = T[i+1][i], e^2; e[D-1] = 0
  float2 de[D];              // float (d[i], e2[i-1]) for the Sturm counts
  float lamf[D];             // eigenvalues from multisection, descending
  double lamv[D];            // Rayleigh-corrected eigenvalues of the vectors
  T beta[D];                 // reflector scales
  T hv[D], hw[D];            // reflector v and w = p - K v of the current step
  T part[NT / D][D];         // partial sums of p = A v
  float glo, ghi, fnorm;
  double pivd;
  int ok;
};

// Lane exchanges by DPP (no LDS round trip): quad_perm [1,0,3,2] and
// [2,3,0,1] swap neighbours and pairs within each group of four lanes,
// row_half_mirror reverses each group of eight, row_mirror each row of 16.
enum : int { kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140 };

template <int CTRL>
__device__ __forceinline__ float tri_dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

template <int CTRL>
__device__ __forceinline__ double tri_dpp(double v) {
  const long long u = __builtin_bit_cast(long long, v);
  const int lo = __builtin_amdgcn_mov_dpp((int)(u & 0xffffffff), CTRL, 0xF, 0xF, true);
  const int hi = __builtin_amdgcn_mov_dpp((int)(u >> 32), CTRL, 0xF, 0xF, true);
  return __builtin_bit_cast(double, ((long long)hi << 32) | (unsigned int)lo);
}

// Sum over each aligned group of W lanes (W = 8 or 16), in every lane.
template <int W, typename T>
__device__ __forceinline__ T tri_group_sum(T v) {
  static_assert(W == 8 || W == 16, "group width");
  v += tri_dpp<kDppXor1>(v);
  v += tri_dpp<kDppXor2>(v);
  v += tri_dpp<kDppHalfMirror>(v);
  if constexpr (W == 16) v += tri_dpp<kDppMirror>(v);
  return v;
}

template <typename T>
__device__ __forceinline__ T tri_readlane(T v, int l) {
  if constexpr (sizeof(T) == 4) {
    return __builtin_bit_cast(T, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
  } else {
    const long long u = __builtin_bit_cast(long long, v);
    const int lo = __builtin_amdgcn_readlane((int)(u & 0xffffffff), l);
    const int hi = __builtin_amdgcn_readlane((int)(u >> 32), l);
    return __builtin_bit_cast(T, ((long long)hi << 32) | (unsigned int)lo);
  }
}

// Sum over the whole wave, in every lane.
template <typename T>
__device__ __forceinline__ T tri_wave_sum(T v) {
  v = tri_group_sum<16>(v);
  return (tri_readlane(v, 0) + tri_readlane(v, 16)) + (tri_readlane(v, 32) + tri_readlane(v, 48));
}

// Stage 1.  A: D x D symmetric in LDS, row stride D + 1 (overwritten: the
// updated trailing blocks and, below the subdiagonal, the reflectors).
template <int D, typename T, int NT>
__device__ void tri_reduce(T* A, TriWork<D, T, NT>& tw) {
  constexpr int LD = D + 1, S = NT / D, U = (D + 63) / 64;
  static_assert(S >= 1 && NT % D == 0, "thread mapping");
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int c = tid % D, s = tid / D;
  for (int k = 0; k < D - 1; ++k) {
    if (wid == 0) {
      // reflector H = I - beta v v^T taking x = A[k+1.., k] to alpha e_1
      T x[U];
      T st = 0;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = k + 1 + lane + 64 * u;
        x[u] = i < D ? A[i * LD + k] : T(0);
        if (i > k + 1) st += x[u] * x[u];
      }
      st = tri_wave_sum(st);
      const T x0 = A[(k + 1) * LD + k];
      T alpha = x0, b = 0, v0 = x0;
      if (st > T(0)) {
        const T nrm = sqrt(x0 * x0 + st);
        alpha = x0 >= T(0) ? -nrm : nrm;
        v0 = x0 - alpha;
        b = T(-1) / (alpha * v0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = k + 1 + lane + 64 * u;
        if (i < D) {
          const T vi = i == k + 1 ? v0 : x[u];
          tw.hv[i] = vi;
          A[i * LD + k] = vi;
        }
      }
      if (lane == 0) {
        tw.beta[k] = b;
        tw.e[k] = (double)alpha;
        tw.d[k] = (double)A[k * LD + k];
      }
    }
    __syncthreads();
    const T b = tw.beta[k];
    if (b == T(0)) continue;  // uniform: the trailing block is already reduced
    // p = beta A22 v, column c summed over rows j = k+1+s, k+1+s+S, ...
    if (c > k) {
      T acc = 0;
      for (int j = k + 1 + s; j < D; j += S) acc += A[j * LD + c] * tw.hv[j];
      tw.part[s][c] = acc;
    }
    __syncthreads();
    if (wid == 0) {
      T p[U], pv = 0;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = k + 1 + lane + 64 * u;
        p[u] = 0;
        if (i < D) {
          T acc = 0;
#pragma unroll
          for (int q = 0; q < S; ++q) acc += tw.part[q][i];
          p[u] = b * acc;
          pv += p[u] * tw.hv[i];
        }
      }
      const T K = T(0.5) * b * tri_wave_sum(pv);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = k + 1 + lane + 64 * u;
        if (i < D) tw.hw[i] = p[u] - K * tw.hv[i];
      }
    }
    __syncthreads();
    // A22 -= v w^T + w v^T
    if (c > k) {
      const T vc = tw.hv[c], wc = tw.hw[c];
      for (int i = k + 1 + s; i < D; i += S) A[i * LD + c] -= tw.hv[i] * wc + tw.hw[i] * vc;
    }
    __syncthreads();
  }
  if (tid == 0) {
    tw.d[D - 1] = (double)A[(D - 1) * LD + D - 1];
    tw.e[D - 1] = 0.0;
  }
  __syncthreads();
}

// Number of eigenvalues of T below x (float Sturm sequence).  Every e^2 is
// at least FLT_MIN, so a zero pivot gives an infinite next pivot (never a
// NaN) and the sequence continues from the one after, as with a pivot of
// -0 or an infinitesimal one.
template <int D>
__device__ __forceinline__ int tri_sturm_f(const float2* de, float x) {
  float q = 1.f;
  int cnt = 0;
#pragma unroll 16
  for (int i = 0; i < D; ++i) {
    const float2 v = de[i];
    q = fmaf(-v.y, __builtin_amdgcn_rcpf(q), v.x - x);
    cnt += q < 0.f;
  }
  return cnt;
}

// Stage 2: tw.lamf = eigenvalues of T, descending.
template <int D, typename T, int NT>
__device__ void tri_eigvals(TriWork<D, T, NT>& tw) {
  constexpr int G = NT / D;
  static_assert(G >= 2 && G <= 64 && (G & (G - 1)) == 0, "group of lanes per eigenvalue");
  constexpr int ROUNDS = G >= 16 ? 7 : (G >= 8 ? 9 : 16);
  const int tid = threadIdx.x;
  if (tid < D) {
    tw.e2[tid] = tw.e[tid] * tw.e[tid];
    tw.de[tid] = make_float2((float)tw.d[tid], tid > 0 ? fmaxf((float)(tw.e[tid - 1] * tw.e[tid - 1]), FLT_MIN) : 0.f);
  }
  __syncthreads();
  if (tid < 64) {
    // Gershgorin interval and the double pivot floor
    float lo = FLT_MAX, hi = -FLT_MAX;
    double md2 = 0.0;
    for (int i = tid; i < D; i += 64) {
      const float r = (float)(fabs(tw.e[i]) + (i > 0 ? fabs(tw.e[i - 1]) : 0.0));
      lo = fminf(lo, (float)tw.d[i] - r);
      hi = fmaxf(hi, (float)tw.d[i] + r);
      md2 = fmax(md2, tw.e2[i]);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      lo = fminf(lo, __shfl_xor(lo, o));
      hi = fmaxf(hi, __shfl_xor(hi, o));
      md2 = fmax(md2, __shfl_xor(md2, o));
    }
    if (tid == 0) {
      const float w = fmaxf(fabsf(lo), fabsf(hi));
      tw.glo = lo - 1e-6f * w - FLT_MIN;
      tw.ghi = hi + 1e-6f * w + FLT_MIN;
      tw.fnorm = w;
      tw.pivd = DBL_MIN * fmax(1.0, md2);
    }
  }
  __syncthreads();
  const int j = tid / G, sl = tid % G;  // ascending index j, lane sl of its group
  float a = tw.glo, b = tw.ghi;
  for (int rnd = 0; rnd < ROUNDS; ++rnd) {
    const float h = (b - a) / (float)(G + 1);
    const float x = fmaf((float)(sl + 1), h, a);
    const int below = tri_sturm_f<D>(tw.de, x) <= j;  // lambda_j >= x
    // the points whose count is <= j form a prefix of the group
    int u = 0;
#pragma unroll
    for (int o = 0; o < G; ++o) u += __shfl(below, (tid & ~(G - 1)) + o);
    const float na = u == 0 ? a : fmaf((float)u, h, a);
    const float nb = u == G ? b : fmaf((float)(u + 1), h, a);
    a = na;
    b = fmaxf(nb, na);
  }
  if (sl == 0) tw.lamf[D - 1 - j] = 0.5f * (a + b);
  __syncthreads();
}

template <int D>
__device__ __forceinline__ double tri_guard(double x, double piv) {
  return fabs(x) < piv ? -piv : x;
}

// One chain of the twisted factorisation of T - lam I for vector t: the
// stationary pivots dp (top down, `fwd`) or the progressive pivots dm
// (bottom up), each with the ratios that build the vector,
// rho_i = e_i / dp_i and sig_i = e_i / dm_{i+1}.  scr holds [4][D][D]
// doubles (dp, dm, rho, sig), entry (i, t) at i * D + t, so that each
// wave's accesses are contiguous.
template <int D, typename T, int NT>
__device__ void tri_chain(const TriWork<D, T, NT>& tw, double lam, double* __restrict__ scr, int t,
                          bool fwd) {
  const double piv = tw.pivd;
  if (fwd) {
    double* __restrict__ sdp = scr;
    double* __restrict__ srho = scr + 2 * D * D;
    double dp = tri_guard<D>(tw.d[0] - lam, piv);
    sdp[t] = dp;
    for (int i = 0; i < D - 1; ++i) {
      const double rho = tw.e[i] / dp;
      srho[i * D + t] = rho;
      dp = tri_guard<D>((tw.d[i + 1] - lam) - tw.e[i] * rho, piv);
      sdp[(i + 1) * D + t] = dp;
    }
  } else {
    double* __restrict__ sdm = scr + D * D;
    double* __restrict__ ssig = scr + 3 * D * D;
    double dm = tri_guard<D>(tw.d[D - 1] - lam, piv);
    sdm[(D - 1) * D + t] = dm;
    for (int i = D - 2; i >= 0; --i) {
      const double sig = tw.e[i] / dm;
      ssig[i * D + t] = sig;
      dm = tri_guard<D>((tw.d[i] - lam) - tw.e[i] * sig, piv);
      sdm[i * D + t] = dm;
    }
  }
}

// Product sweep of one side of the twisted vector (z_r = 1): above r,
// z_i = -rho_i z_{i+1}; below it, z_{i+1} = -sig_i z_i.  Both sides take
// the same instruction stream (the side is per lane), so two lanes of one
// wave sweep them together.  Multiplies each entry by `scale` and stores it
// to row when `store`; returns the sum of the squares of the unscaled
// entries.  Ratios are loaded 16 at a time ahead of the dependent products.
template <int D, typename T>
__device__ double tri_sweep(const double* __restrict__ scr, int t, int r, bool up, double scale, bool store,
                            T* __restrict__ row) {
  // step j uses ratio index up ? r-1-j : r+j and stores entry r -/+ (1+j)
  const double* __restrict__ base = up ? scr + 2 * D * D : scr + 3 * D * D;
  const int len = up ? r : D - 1 - r;
  const int dir = up ? -1 : 1;
  const int i0 = up ? r - 1 : r;
  double nrm = 0.0, z = 1.0;
  for (int j0 = 0; j0 < len; j0 += 16) {
    double f[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) f[u] = j0 + u < len ? base[(i0 + dir * (j0 + u)) * D + t] : 0.0;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      if (j0 + u < len) {
        z = -f[u] * z;
        nrm += z * z;
        if (store) row[r + dir * (1 + j0 + u)] = (T)(z * scale);
      }
    }
  }
  return nrm;
}

// Stage 3.  VT: row t (stride LV) receives the eigenvector of lamf[t] for
// t < nvec (tridiagonal coordinates); tw.lamv[t] its corrected eigenvalue.
// scr: this block's [4][D][D] doubles of global scratch.  The two pivot
// chains of a factorisation run in different waves; the twist search, the
// product sweeps and the checks use a group of 8 lanes per vector.
template <int D, typename T, int NT>
__device__ void tri_vectors(TriWork<D, T, NT>& tw, T* VT, int LV, int nvec, double* scr) {
  static_assert(NT >= 8 * D && D % 8 == 0, "8 lanes per vector");
  const int tid = threadIdx.x;
  const int t8 = tid >> 3, s8 = tid & 7;  // vector and lane of its group
  if (tid < D) tw.lamv[tid] = (double)tw.lamf[tid];
  if (tid == 0) tw.ok = 1;
  __syncthreads();
  for (int pass = 0; pass < 2; ++pass) {
    // pivot chains: threads [0, D) bottom up, [D, 2D) top down
    if (tid < 2 * D && (tid % D) < nvec) tri_chain<D, T, NT>(tw, tw.lamv[tid % D], scr, tid % D, tid >= D);
    __syncthreads();
    if (t8 < nvec) {
      const int t = t8;
      const double lam = tw.lamv[t];
      // twist index: smallest |gamma_k|, k = s8 + 8j; ties to the smaller k
      double bg = 0.0, ba = -1.0;
      int bk = D;
      for (int k = s8; k < D; k += 8) {
        const double gk = scr[k * D + t] + scr[D * D + k * D + t] - (tw.d[k] - lam);
        const double ak = fabs(gk);
        if (ba < 0.0 || ak < ba) {
          ba = ak;
          bg = gk;
          bk = k;
        }
      }
      auto take = [&](double oa, double og, int ok) {
        if (oa < ba || (oa == ba && ok < bk)) {
          ba = oa;
          bg = og;
          bk = ok;
        }
      };
      take(tri_dpp<kDppXor1>(ba), tri_dpp<kDppXor1>(bg), __builtin_amdgcn_mov_dpp(bk, kDppXor1, 0xF, 0xF, true));
      take(tri_dpp<kDppXor2>(ba), tri_dpp<kDppXor2>(bg), __builtin_amdgcn_mov_dpp(bk, kDppXor2, 0xF, 0xF, true));
      take(tri_dpp<kDppHalfMirror>(ba), tri_dpp<kDppHalfMirror>(bg),
           __builtin_amdgcn_mov_dpp(bk, kDppHalfMirror, 0xF, 0xF, true));
      const int r = bk;
      // |z|^2 from the two sides (lanes 0 and 1 of the group)
      T* row = VT + (size_t)t * LV;
      double side = s8 < 2 ? tri_sweep<D, T>(scr, t, r, s8 == 0, 1.0, false, row) : 0.0;
      side += tri_dpp<kDppXor1>(side);
      const double nrm = 1.0 + side;
      if (pass == 0) {
        if (s8 == 0) tw.lamv[t] = lam + bg / nrm;
      } else if (s8 < 2) {
        const double sc = 1.0 / sqrt(nrm);
        if (s8 == 0) row[r] = (T)sc;
        tri_sweep<D, T>(scr, t, r, s8 == 0, sc, true, row);
      }
    }
    __syncthreads();
  }
  // residual |T z - lam z| per vector (8 lanes), then pairwise orthogonality
  const double tol = sizeof(T) == 4 ? 1e-4 : 1e-9;
  const double tn = fmax((double)tw.fnorm, DBL_MIN);
  bool bad = false;
  if (t8 < nvec) {
    const T* z = VT + (size_t)t8 * LV;
    const double lam = tw.lamv[t8];
    double res = 0.0;
    for (int i = s8; i < D; i += 8) {
      double y = (tw.d[i] - lam) * (double)z[i];
      if (i > 0) y += tw.e[i - 1] * (double)z[i - 1];
      if (i < D - 1) y += tw.e[i] * (double)z[i + 1];
      res = fmax(res, fabs(y));
    }
    bad = !(res <= tol * tn);
  }
  const int npair = nvec * (nvec - 1) / 2;
  for (int pi = tid; pi < npair; pi += NT) {
    // pair index -> (a, b), a < b
    int a = (int)((sqrt(8.0 * pi + 1.0) - 1.0) * 0.5);
    while ((a + 1) * (a + 2) / 2 <= pi) ++a;
    while (a * (a + 1) / 2 > pi) --a;
    const int bb = a + 1, aa = pi - a * (a + 1) / 2;  // bb > aa
    const T* za = VT + (size_t)aa * LV;
    const T* zb = VT + (size_t)bb * LV;
    double dot = 0.0;
    for (int i = 0; i < D; ++i) dot += (double)za[i] * (double)zb[i];
    if (!(fabs(dot) <= tol)) bad = true;
  }
  if (bad) tw.ok = 0;
  __syncthreads();
}

// Stage 4.  VT rows t < nvec <- Q applied to them.  A holds the reflectors
// of tri_reduce below its subdiagonal.  Vector t belongs to the GV = NT / D
// lanes of one group, lane s holding its entries s, s + GV, ... in
// registers for all D - 2 reflectors; group sums go by DPP, so the stage
// needs no barrier and each reflector costs one read of its column.
template <int D, typename T, int NT>
__device__ void tri_back(const T* A, const TriWork<D, T, NT>& tw, T* VT, int LV, int nvec) {
  constexpr int LD = D + 1, GV = NT / D, NZ = D / GV;
  static_assert(GV == 8 || GV == 16, "lanes per vector");
  const int tid = threadIdx.x, t = tid / GV, s = tid % GV;
  if (t < nvec) {  // whole groups of lanes
    T* row = VT + (size_t)t * LV;
    T z[NZ];
#pragma unroll
    for (int u = 0; u < NZ; ++u) z[u] = row[s + GV * u];
    for (int k = D - 3; k >= 0; --k) {
      const T b = tw.beta[k];
      if (b == T(0)) continue;
      T v[NZ];
      T dot = 0;
#pragma unroll
      for (int u = 0; u < NZ; ++u) {
        const int i = s + GV * u;
        const T a = A[i * LD + k];
        v[u] = i > k ? a : T(0);
        dot += v[u] * z[u];
      }
      const T f = b * tri_group_sum<GV>(dot);
#pragma unroll
      for (int u = 0; u < NZ; ++u) z[u] -= f * v[u];
    }
#pragma unroll
    for (int u = 0; u < NZ; ++u) row[s + GV * u] = z[u];
  }
  __syncthreads();
}

}  // namespace sparsepr
