// Symmetric eigensolver used by the response bases (App. B.1, B.2) and the
// probe-residual basis (App. A.3 eq. app_probe_residual_basis): parallel
// cyclic Jacobi in LDS, one block of NT threads per matrix.
//
// Each step applies the D/2 disjoint rotations of the round-robin (circle)
// ordering.  One thread per pair computes the rotation; then A <- J^T A J is
// applied as independent 2x2 blocks (pair i rows x pair j columns) and the
// eigenvector matrix as independent row pairs of its transpose, in one pass
// with one barrier.  With NT a multiple of D/2 every thread keeps the same
// column pair j for the whole step, so its rotation is read from LDS once.
// On return A's diagonal (row stride D + 1) holds the eigenvalues and row k
// of VT (row stride D + 4, 16-byte aligned) the eigenvector of A[k][k]: the
// transposed layout turns each rotation of two eigenvector columns into two
// contiguous rows, updated four elements per access.  A is in LDS; VT is in
// LDS or, when both do not fit, in the block's own global scratch (the block
// barriers order those accesses as well).
#pragma once
#include <hip/hip_runtime.h>
#include <math.h>

namespace sparsepr {

template <typename T>
struct alignas(16) JacobiRot {
  T c, s;
  int p, q;
};

// Eigenvalue sort key: NaN (from non-finite inputs) as -inf, so that ranks
// by (key descending, index ascending) are a permutation.
template <typename T>
__device__ __forceinline__ T eig_rank_key(T v) {
  return v == v ? v : -(T)INFINITY;
}

template <int D>
constexpr int jacobi_vt_ld() {
  return D + 4;
}

template <int D, typename T, int NT>
__device__ void jacobi_eig_lds(T* A, T* VT, JacobiRot<T>* rot, int* flag, T stop) {
  constexpr int LD = D + 1, LV = jacobi_vt_ld<D>(), P = D / 2;
  static_assert(NT % P == 0 && (P * P) % NT == 0, "thread mapping");
  typedef T T4 __attribute__((ext_vector_type(4)));
  const int tid = threadIdx.x;
  for (int i = tid; i < D * D; i += NT) {
    const int r = i / D, c = i % D;
    VT[r * LV + c] = (r == c) ? T(1) : T(0);
  }
  __syncthreads();
  for (int sweep = 0; sweep < 20; ++sweep) {
    if (tid == 0) *flag = 0;
    __syncthreads();
    for (int step = 0; step < D - 1; ++step) {
      if (tid < P) {
        int p, q;
        if (tid == 0) {
          p = step;
          q = D - 1;
        } else {
          p = (step + tid) % (D - 1);
          q = (step - tid + D - 1) % (D - 1);
        }
        const T app = A[p * LD + p], aqq = A[q * LD + q], apq = A[p * LD + q];
        T c = 1, s = 0;
        const T tol = sizeof(T) == 8 ? T(1e-15) : T(3e-7);
        // rotate unless |apq| <= tol * sqrt(|app aqq|) (compared squared)
        if (apq != T(0) && apq * apq > tol * tol * fabs(app * aqq)) {
          // tan of the rotation angle: the smaller root of t^2 + 2 theta t - 1
          const T theta = (aqq - app) / (T(2) * apq);
          const T at = fabs(theta);
          T t;
          if constexpr (sizeof(T) == 4) {
            // hardware reciprocal, square root and reciprocal square root
            // (each about 1 ulp): the chain of this one wave is what every
            // other wave waits for, and c = rsq(1 + t^2), s = t c keeps
            // c^2 + s^2 = 1 to the same rounding as exact operations would
            t = (at > T(1e10)) ? T(0.5) * __builtin_amdgcn_rcpf(theta)
                               : copysign(__builtin_amdgcn_rcpf(at + __builtin_amdgcn_sqrtf(fmaf(theta, theta, 1.f))), theta);
            c = __builtin_amdgcn_rsqf(fmaf(t, t, 1.f));
          } else {
            t = (at > T(1e10)) ? T(0.5) / theta
                               : copysign(T(1), theta) / (at + sqrt(theta * theta + T(1)));
            c = T(1) / sqrt(t * t + T(1));
          }
          s = t * c;
          *flag = 1;
        }
        rot[tid] = JacobiRot<T>{c, s, p, q};
      }
      __syncthreads();
      // All of a thread's loads are issued before any of its stores: its
      // 2x2 blocks and eigenvector row pairs are disjoint from every other
      // thread's, so one LDS round trip serves the whole update.
      constexpr int NB = P * P / NT, NVI = (P * (D / 4) + NT - 1) / NT;
      const int j = tid % P;
      const JacobiRot<T> rj = rot[j];
      JacobiRot<T> ri[NB];
      T x[NB][4];
#pragma unroll
      for (int k = 0; k < NB; ++k) ri[k] = rot[tid / P + k * (NT / P)];
#pragma unroll
      for (int k = 0; k < NB; ++k) {
        const int p = ri[k].p, q = ri[k].q;
        x[k][0] = A[p * LD + rj.p];
        x[k][1] = A[p * LD + rj.q];
        x[k][2] = A[q * LD + rj.p];
        x[k][3] = A[q * LD + rj.q];
      }
      // eigenvector rows: item e = (pair e / (D/4), four elements e % (D/4))
      T4 vp[NVI], vq[NVI];
      JacobiRot<T> rv[NVI];
#pragma unroll
      for (int k = 0; k < NVI; ++k) {
        const int e = tid + k * NT;
        if (e < P * (D / 4)) {
          rv[k] = rot[e / (D / 4)];
          const int c4 = (e % (D / 4)) * 4;
          vp[k] = *(const T4*)(VT + rv[k].p * LV + c4);
          vq[k] = *(const T4*)(VT + rv[k].q * LV + c4);
        }
      }
#pragma unroll
      for (int k = 0; k < NB; ++k) {
        const int i = tid / P + k * (NT / P);
        if (ri[k].s == T(0) && rj.s == T(0)) continue;
        const int p = ri[k].p, q = ri[k].q;
        const T y00 = x[k][0] * rj.c - x[k][1] * rj.s, y01 = x[k][0] * rj.s + x[k][1] * rj.c;
        const T y10 = x[k][2] * rj.c - x[k][3] * rj.s, y11 = x[k][2] * rj.s + x[k][3] * rj.c;
        T z00 = ri[k].c * y00 - ri[k].s * y10, z01 = ri[k].c * y01 - ri[k].s * y11;
        T z10 = ri[k].s * y00 + ri[k].c * y10, z11 = ri[k].s * y01 + ri[k].c * y11;
        if (i == j) z01 = z10 = T(0);
        A[p * LD + rj.p] = z00;
        A[p * LD + rj.q] = z01;
        A[q * LD + rj.p] = z10;
        A[q * LD + rj.q] = z11;
      }
#pragma unroll
      for (int k = 0; k < NVI; ++k) {
        const int e = tid + k * NT;
        if (e < P * (D / 4) && rv[k].s != T(0)) {
          const int c4 = (e % (D / 4)) * 4;
          *(T4*)(VT + rv[k].p * LV + c4) = rv[k].c * vp[k] - rv[k].s * vq[k];
          *(T4*)(VT + rv[k].q * LV + c4) = rv[k].s * vp[k] + rv[k].c * vq[k];
        }
      }
      __syncthreads();
    }
    // Stop once the off-diagonal norm falls below `stop` times the matrix
    // norm (convergence is quadratic, so one more sweep takes a relative
    // off-diagonal norm of 1e-4 to the float rounding floor).
    {
      __shared__ T red[2][NT / 64];
      T off = 0, tot = 0;
      for (int i = tid; i < D * D; i += NT) {
        const int r = i / D, c = i % D;
        const T x = A[r * LD + c];
        tot += x * x;
        if (r != c) off += x * x;
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        off += __shfl_xor(off, o);
        tot += __shfl_xor(tot, o);
      }
      if ((tid & 63) == 0) {
        red[0][tid >> 6] = off;
        red[1][tid >> 6] = tot;
      }
      __syncthreads();
      if (tid == 0) {
        T o2 = 0, t2 = 0;
        for (int w = 0; w < NT / 64; ++w) {
          o2 += red[0][w];
          t2 += red[1][w];
        }
        if (o2 <= stop * stop * t2) *flag = 0;
      }
    }
    __syncthreads();
    const int more = *flag;
    __syncthreads();
    if (!more) break;
  }
}

}  // namespace sparsepr
