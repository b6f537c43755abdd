// Data-informed starting factor (Appendix D, "Initialization") for gfx950.
//
// The randomized range finder on the Gram matrix of the normalised data,
//     V = Xhat Xhat^T Z,   V = Q R,   U_0 = Pi_Omega(Q),
// with the QR taken as the appendix's Cholesky QR in feature space:
//     M = Xhat^T Z (d x r),  C = Xhat^T Xhat (d x d, reused from the spectral
//     normalisation),  V^T V = M^T C M = R^T R,  Q = Xhat (M R^{-1}).
// M comes from one pass A over (Xhat, Z) (the Theta product with U = Z); the
// small algebra (C M, M^T C M, the Cholesky factor and the triangular solve) runs
// in FP64 in one workgroup; Q = Xhat T is one more pass over Xhat, written over
// Z, after which the usual projection onto Omega follows.  A pivot that is not
// above 1e-14 of its diagonal entry (V numerically rank deficient) marks the
// control block degenerate.
#include "k_common.hpp"

namespace nlr {

__global__ void k_start_prep(Bufs B, int r32) {
  for (int c = threadIdx.x; c < r32; c += blockDim.x) B.p[c] = 0.f;  // pass A reads p for its row work
}

// C / a^2 = Xhat^T Xhat from the centred Gram matrix of the normalisation.
__global__ __launch_bounds__(kThreads) void k_start_copy_c(Geometry g, Bufs B) {
  const double a = B.ctl->spectral_a;
  const double s = 1.0 / (a * a);
  const int64_t dd = (int64_t)g.d * g.d;
  for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < dd; e += (int64_t)gridDim.x * kThreads)
    B.s_C[e] = B.i_C[e] * s;
}

__global__ void k_start_zero_xbar(Geometry g, Bufs B) {
  for (int f = threadIdx.x; f < g.d; f += blockDim.x) B.i_xbar[f] = 0.0;
}

// M[f][c] = sum of the pass-A segment sums (fixed order), FP64.
__global__ __launch_bounds__(kThreads) void k_start_m(Geometry g, Bufs B) {
  const int64_t tot = (int64_t)g.d32 * g.r32;
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= tot) return;
  double sum = 0.0;
  for (int s = 0; s < g.SA; ++s) sum += B.seg_theta[(int64_t)s * g.theta_cols + e];
  const int f = (int)(e / g.r32), c = (int)(e % g.r32);
  if (f < g.d && c < g.r) B.s_M[(int64_t)f * g.r + c] = sum;
}

// One workgroup: CM = C M, G = M^T CM, G = L L^T (L lower, R = L^T), T = M L^{-T}.
__global__ __launch_bounds__(kThreads) void k_start_chol(Geometry g, Bufs B) {
  const int d = g.d, r = g.r;
  const int tid = threadIdx.x;
  double* CM = B.s_CM;
  double* G = B.s_G;
  for (int e = tid; e < d * r; e += kThreads) {
    const int f = e / r, c = e - (e / r) * r;
    double acc = 0.0;
    for (int k = 0; k < d; ++k) acc += B.s_C[(int64_t)f * d + k] * B.s_M[(int64_t)k * r + c];
    CM[e] = acc;
  }
  __syncthreads();
  for (int e = tid; e < r * r; e += kThreads) {
    const int i = e / r, j = e - (e / r) * r;
    double acc = 0.0;
    for (int f = 0; f < d; ++f) acc += B.s_M[(int64_t)f * r + i] * CM[(int64_t)f * r + j];
    G[e] = acc;
  }
  __syncthreads();
  __shared__ int bad;
  if (tid == 0) bad = 0;
  __syncthreads();
  // Cholesky, column by column: L[j][j] = sqrt(G[j][j] - sum_k L[j][k]^2), then the column below
  for (int j = 0; j < r; ++j) {
    if (tid == 0) {
      const double g0 = G[j * r + j];
      double s = g0;
      for (int k = 0; k < j; ++k) s -= G[j * r + k] * G[j * r + k];
      // a pivot at rounding level of the diagonal means V has (numerically) dependent columns
      if (!(s > 1e-14 * g0) || !isfinite(s)) bad = 1;
      G[j * r + j] = (s > 0.0) ? sqrt(s) : 1.0;
    }
    __syncthreads();
    const double ljj = G[j * r + j];
    for (int i = j + 1 + tid; i < r; i += kThreads) {
      double s = G[i * r + j];
      for (int k = 0; k < j; ++k) s -= G[i * r + k] * G[j * r + k];
      G[i * r + j] = s / ljj;
    }
    __syncthreads();
  }
  // T row f: T[f][j] = (M[f][j] - sum_{k<j} T[f][k] L[j][k]) / L[j][j]
  for (int f = tid; f < d; f += kThreads) {
    for (int j = 0; j < r; ++j) {
      double s = B.s_M[(int64_t)f * r + j];
      for (int k = 0; k < j; ++k) s -= B.s_T[(int64_t)f * r + k] * G[j * r + k];
      B.s_T[(int64_t)f * r + j] = s / G[j * r + j];
    }
  }
  if (tid == 0 && bad) B.ctl->degenerate = 1;
}

// U = Xhat T (FP64 accumulation), 64-row tiles, grid-stride.  Thread (g, c):
// column c of the current 64-column block, rows g, g + 4, ..., g + 60.
__global__ __launch_bounds__(kThreads) void k_start_apply(Geometry g, Bufs B) {
  if (B.ctl->degenerate) return;
  __shared__ float xt[64][65];
  const int tid = threadIdx.x;
  const int rg = tid >> 6, cl = tid & 63;
  const int d = g.d, r = g.r;
  const int64_t n = g.n;
  const int64_t tiles = (n + 63) / 64;
  for (int64_t t = blockIdx.x; t < tiles; t += gridDim.x) {
    const int64_t row0 = t * 64;
    for (int cb = 0; cb < r; cb += 64) {
      const int c = cb + cl;
      double acc[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[i] = 0.0;
      for (int f0 = 0; f0 < d; f0 += 64) {
        __syncthreads();
        for (int e = tid; e < 64 * 64; e += kThreads) {
          const int rr = e >> 6, ff = e & 63;
          const int64_t row = row0 + rr;
          xt[rr][ff] = (row < n && f0 + ff < d) ? B.X[row * d + f0 + ff] : 0.f;
        }
        __syncthreads();
        const int fe = (d - f0) < 64 ? (d - f0) : 64;
        for (int ff = 0; ff < fe; ++ff) {
          const double tv = (c < r) ? B.s_T[(int64_t)(f0 + ff) * r + c] : 0.0;
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[i] += (double)xt[4 * i + rg][ff] * tv;
        }
      }
      if (c < r) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int64_t row = row0 + 4 * i + rg;
          if (row < n) B.U[row * r + c] = (float)acc[i];
        }
      }
    }
  }
}

hipError_t launch_data_start(const Geometry& g, const Bufs& b, const StepArgs& a0, bool x_normalised,
                             hipStream_t st) {
  hipError_t e;
  if (x_normalised) {
    // C = Xhat^T Xhat from the given Xhat (no re-centring)
    hipLaunchKernelGGL(k_start_zero_xbar, dim3(1), dim3(kThreads), 0, st, g, b);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_gram(g, b, st)) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_start_copy_c, dim3(64), dim3(kThreads), 0, st, g, b);
  hipLaunchKernelGGL(k_start_prep, dim3(1), dim3(kThreads), 0, st, b, g.r32);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // M = Xhat^T Z: the pass-A product with U = Z (c_f = 1)
  if ((e = launch_pass_a(g, b, a0, false, st)) != hipSuccess) return e;
  const int C = g.d32 * g.r32;
  if ((e = launch_seg_theta(g, b, g.GA, g.SA, st)) != hipSuccess) return e;
  hipLaunchKernelGGL(k_start_m, dim3((C + kThreads - 1) / kThreads), dim3(kThreads), 0, st, g, b);
  hipLaunchKernelGGL(k_start_chol, dim3(1), dim3(kThreads), 0, st, g, b);
  const int64_t tiles = (g.n + 63) / 64;
  hipLaunchKernelGGL(k_start_apply, dim3((unsigned)(tiles < 4096 ? tiles : 4096)), dim3(kThreads), 0, st, g, b);
  return hipGetLastError();
}

}  // namespace nlr
