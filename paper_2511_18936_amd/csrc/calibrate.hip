// Offline calibration (Sec. 4.1.2): the projection P is the right singular
// matrix of the joint matrix S, i.e. the eigenvector matrix of S^T S.
//
//   gram_kernel     G = S^T S in float64 (products of float32 are exact in
//                   float64), 16x16 output tile per workgroup
//   jacobi_kernel   one workgroup, G held in LDS: parallel cyclic Jacobi in float64 with
//                   round-robin pairing (64 disjoint rotations per round, 127
//                   rounds per sweep) until the off-diagonal mass is negligible;
//                   then columns sorted by eigenvalue (descending, stable),
//                   signs canonicalised (largest-magnitude entry positive,
//                   lowest row on ties), sigma = sqrt(lambda), P written in
//                   float32
#include "swan_device.h"
#include "swan_internal.h"

namespace swan {

__global__ __launch_bounds__(256) void gram_kernel(const float* __restrict__ S, int64_t n,
                                                   double* __restrict__ G) {
  __shared__ float si[64][16];
  __shared__ float sj[64][16];
  const int ti = threadIdx.x / 16, tj = threadIdx.x % 16;
  const int i0 = (blockIdx.x / (kD / 16)) * 16, j0 = (blockIdx.x % (kD / 16)) * 16;
  double acc = 0.0;
  for (int64_t r0 = 0; r0 < n; r0 += 64) {
    for (int e = threadIdx.x; e < 64 * 16; e += 256) {
      const int rr = e / 16, cc = e % 16;
      const int64_t r = r0 + rr;
      si[rr][cc] = r < n ? S[r * kD + i0 + cc] : 0.f;
      sj[rr][cc] = r < n ? S[r * kD + j0 + cc] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int rr = 0; rr < 64; ++rr) acc = fma((double)si[rr][ti], (double)sj[rr][tj], acc);
    __syncthreads();
  }
  G[(i0 + ti) * kD + j0 + tj] = acc;
}

// round r (0..126) of the circle method: pair i joins players arr[i], arr[127-i]
// with arr[0] = 0 and arr[k] = 1 + (k - 1 + r) mod 127
__device__ __forceinline__ void rr_pair(int r, int i, int& p, int& q) {
  const int a = (i == 0) ? 0 : 1 + (i - 1 + r) % (kD - 1);
  const int b = 1 + (kD - 2 - i + r) % (kD - 1);
  p = a < b ? a : b;
  q = a < b ? b : a;
}

constexpr int kLdA = kD + 1;  // LDS row stride of A, in doubles

__global__ __launch_bounds__(1024) void jacobi_kernel(double* __restrict__ Ag,
                                                      double* __restrict__ V,
                                                      float* __restrict__ P_out,
                                                      float* __restrict__ sigma_out,
                                                      int32_t* __restrict__ status) {
  // A lives in LDS for the whole solve, rows padded to kLdA doubles so that a
  // column walk (one row per lane) spreads over the banks.  The eigenvectors
  // are kept transposed in the workspace, W = V^T: the column updates V J are
  // row updates of W, contiguous across lanes.
  extern __shared__ __attribute__((aligned(16))) double A[];  // [kD][kLdA]
  double* __restrict__ W = V;
  __shared__ double cs_c[kD / 2], cs_s[kD / 2];
  __shared__ int pp[kD / 2], qq[kD / 2];
  __shared__ double red[1024 / 64];
  __shared__ double red2[1024 / 64];
  __shared__ int done;
  const int tid = threadIdx.x;
  for (int e = tid; e < kD * kD; e += 1024) {
    A[(e / kD) * kLdA + e % kD] = Ag[e];
    W[e] = (e / kD == e % kD) ? 1.0 : 0.0;
  }
  if (tid == 0) done = 0;
  __syncthreads();
  constexpr int kPerThread = (kD / 2) * kD / 1024;  // (pair, row) updates per thread
  int sweep = 0;
  for (; sweep < kJacobiMaxSweeps; ++sweep) {
    // convergence test: off-diagonal Frobenius mass vs the diagonal's
    double off = 0.0, dia = 0.0;
    for (int e = tid; e < kD * kD; e += 1024) {
      const double v = A[(e / kD) * kLdA + e % kD];
      if (e / kD == e % kD) dia += v * v; else off += v * v;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      off += __shfl_xor(off, o, 64);
      dia += __shfl_xor(dia, o, 64);
    }
    if ((tid & 63) == 0) {
      red[tid / 64] = off;
      red2[tid / 64] = dia;
    }
    __syncthreads();
    if (tid == 0) {
      double o = 0.0, d = 0.0;
      for (int w = 0; w < 1024 / 64; ++w) {
        o += red[w];
        d += red2[w];
      }
      done = (o <= 1e-30 * d) ? 1 : 0;
    }
    __syncthreads();
    if (done) break;
    for (int r = 0; r < kD - 1; ++r) {
      if (tid < kD / 2) {
        int p, q;
        rr_pair(r, tid, p, q);
        pp[tid] = p;
        qq[tid] = q;
        const double apq = A[p * kLdA + q];
        const double app = A[p * kLdA + p], aqq = A[q * kLdA + q];
        double c = 1.0, s = 0.0;
        if (fabs(apq) > 1e-300 && fabs(apq) > 1e-18 * sqrt(fabs(app) * fabs(aqq))) {
          const double tau = (aqq - app) / (2.0 * apq);
          const double t = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
          c = 1.0 / sqrt(1.0 + t * t);
          s = t * c;
        }
        cs_c[tid] = c;
        cs_s[tid] = s;
      }
      __syncthreads();
      // V <- V J, i.e. rows p, q of W: all of this thread's loads first
      {
        double wp[kPerThread], wq[kPerThread];
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
          const int e = tid + 1024 * u, i = e / kD, col = e % kD;
          wp[u] = W[pp[i] * kD + col];
          wq[u] = W[qq[i] * kD + col];
        }
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
          const int e = tid + 1024 * u, i = e / kD, col = e % kD;
          const double c = cs_c[i], s = cs_s[i];
          W[pp[i] * kD + col] = c * wp[u] - s * wq[u];
          W[qq[i] * kD + col] = s * wp[u] + c * wq[u];
        }
      }
      // A <- A J (column pairs)
      for (int e = tid; e < (kD / 2) * kD; e += 1024) {
        const int i = e / kD, row = e % kD;
        const double c = cs_c[i], s = cs_s[i];
        if (s == 0.0) continue;
        const int p = pp[i], q = qq[i];
        const double ap = A[row * kLdA + p], aq = A[row * kLdA + q];
        A[row * kLdA + p] = c * ap - s * aq;
        A[row * kLdA + q] = s * ap + c * aq;
      }
      __syncthreads();
      // A <- J^T A (row pairs)
      for (int e = tid; e < (kD / 2) * kD; e += 1024) {
        const int i = e / kD, col = e % kD;
        const double c = cs_c[i], s = cs_s[i];
        if (s == 0.0) continue;
        const int p = pp[i], q = qq[i];
        const double ap = A[p * kLdA + col], aq = A[q * kLdA + col];
        A[p * kLdA + col] = c * ap - s * aq;
        A[q * kLdA + col] = s * ap + c * aq;
      }
      __syncthreads();
    }
  }
  // sort by eigenvalue (descending; equal values keep ascending solver index),
  // canonical sign, write float32 P and sigma
  if (tid < kD) {
    const int j = tid;
    const double lj = A[j * kLdA + j];
    int rank = 0;
    for (int i = 0; i < kD; ++i) {
      const double li = A[i * kLdA + i];
      rank += (li > lj || (li == lj && i < j)) ? 1 : 0;
    }
    int arg = 0;
    double best = -1.0;
    for (int i = 0; i < kD; ++i) {
      const double v = fabs(W[j * kD + i]);
      if (v > best) {
        best = v;
        arg = i;
      }
    }
    const double sgn = W[j * kD + arg] < 0.0 ? -1.0 : 1.0;
    for (int i = 0; i < kD; ++i) P_out[i * kD + rank] = (float)(sgn * W[j * kD + i]);
    if (sigma_out) sigma_out[rank] = (float)sqrt(lj > 0.0 ? lj : 0.0);
  }
  if (tid == 0) {
    status[0] = done;
    status[1] = sweep;
  }
}

hipError_t launch_calibrate(const CalibLaunch& a) {
  hipLaunchKernelGGL(gram_kernel, dim3((kD / 16) * (kD / 16)), dim3(256), 0, a.stream, a.rows,
                     a.n_rows, a.gram);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  constexpr size_t kLds = sizeof(double) * kD * kLdA;  // A in LDS
  e = hipFuncSetAttribute((const void*)jacobi_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)kLds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(jacobi_kernel, dim3(1), dim3(1024), kLds, a.stream, a.gram, a.vecs, a.P_out,
                     a.sigma_out, a.status);
  return hipGetLastError();
}

}  // namespace swan
