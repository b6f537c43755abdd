// Cluster labels from the factor by spectral embedding and K-means (Appendix D,
// "Recover cluster labels from U") for gfx950.
//
//   G = U^T U (FP64, r x r, fixed-order partial sums);
//   G = V Lambda V^T by cyclic Jacobi rotations in one workgroup (round-robin
//   pairing, r/2 disjoint rotations per step);
//   P = V_K Lambda_K^{-1/2}: the embedding E = U P holds the leading K left
//   singular vectors of U (up to a rotation inside their span, which leaves all
//   distances, and so the labels, unchanged);
//   Lloyd's iteration on the rows of E from the embedded seed rows: every pass
//   recomputes E_i = U_i P, assigns row i to its nearest centroid (squared
//   distance in FP64, lowest index on ties), counts changed labels and forms
//   per-workgroup cluster sums in a fixed row order; a single workgroup turns
//   them into the new centroids (a centroid without rows stays in place).
// The host stops after the first pass that changes no label.
#include "k_common.hpp"

namespace nlr {

constexpr int kLabTile = 64;  // rows per tile of the assignment pass

// Partial G over a row chunk: block (bi, bj) of 32 x 32 entries, 64-row LDS tiles.
__global__ __launch_bounds__(kThreads) void k_lab_gram(Geometry g, Bufs B, LabScratch L) {
  __shared__ double ua[64][33];
  __shared__ double ub[64][33];
  const int tid = threadIdx.x;
  const int r = g.r;
  const int rb = (r + 31) / 32;
  const int bi = blockIdx.y / rb, bj = blockIdx.y - (blockIdx.y / rb) * rb;
  const int64_t n = g.n;
  const int64_t r0 = (int64_t)blockIdx.x * n / L.GU;
  const int64_t r1 = (int64_t)(blockIdx.x + 1) * n / L.GU;
  const int ta = tid >> 3, tb = tid & 7;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int64_t t0 = r0; t0 < r1; t0 += 64) {
    __syncthreads();
    for (int v = tid; v < 64 * 32; v += kThreads) {
      const int rr = v >> 5, cc = v & 31;
      const int64_t i = t0 + rr;
      const int ca = bi * 32 + cc, cb = bj * 32 + cc;
      ua[rr][cc] = (i < r1 && ca < r) ? (double)B.U[i * r + ca] : 0.0;
      ub[rr][cc] = (i < r1 && cb < r) ? (double)B.U[i * r + cb] : 0.0;
    }
    __syncthreads();
    for (int rr = 0; rr < 64; ++rr) {
      const double a = ua[rr][ta];
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] += a * ub[rr][4 * tb + e];
    }
  }
  double* out = L.gpart + (int64_t)blockIdx.x * r * r;
  const int ia = bi * 32 + ta;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int jb = bj * 32 + 4 * tb + e;
    if (ia < r && jb < r) out[(int64_t)ia * r + jb] = acc[e];
  }
}

__global__ __launch_bounds__(kThreads) void k_lab_gram_reduce(Geometry g, LabScratch L) {
  const int rr = g.r * g.r;
  const int e = blockIdx.x * kThreads + threadIdx.x;
  if (e == 0) L.flag[0] = L.flag[1] = 0;
  if (e >= rr) return;
  double s = 0.0;
  for (int k = 0; k < L.GU; ++k) s += L.gpart[(int64_t)k * rr + e];
  L.A[e] = s;
}

// Cyclic Jacobi on A (r x r, symmetric) in one workgroup; V accumulates the
// rotations.  Then P = V_K Lambda_K^{-1/2} for the K largest eigenvalues
// (descending, lowest index on ties).  A non-positive K-th eigenvalue marks the
// control block degenerate.
__global__ __launch_bounds__(kThreads) void k_lab_eig(Geometry g, LabScratch L, int K) {
  const int r = g.r;
  const int m = (r + 1) & ~1;  // even number of players; index r (odd r) is a bye
  const int tid = threadIdx.x;
  double* A = L.A;
  double* V = L.V;
  __shared__ int top[kMaxR / 2 + 1], bot[kMaxR / 2 + 1];
  __shared__ double cs[kMaxR / 2 + 1], sn[kMaxR / 2 + 1];
  __shared__ double red[4];
  __shared__ int order[kMaxR];
  __shared__ int stop;
  for (int e = tid; e < r * r; e += kThreads) V[e] = ((e / r) == (e % r)) ? 1.0 : 0.0;
  for (int k = tid; k < m / 2; k += kThreads) {
    top[k] = 2 * k;
    bot[k] = 2 * k + 1;
  }
  if (tid == 0) stop = 0;
  __syncthreads();
  double total = 0.0;
  for (int e = tid; e < r * r; e += kThreads) total += A[e] * A[e];
  total = block_sum_d(total, red);
  __shared__ double tot_s;
  if (tid == 0) tot_s = total;
  __syncthreads();
  for (int sweep = 0; sweep < 60; ++sweep) {
    // off-diagonal mass
    double off = 0.0;
    for (int e = tid; e < r * r; e += kThreads)
      if ((e / r) != (e % r)) off += A[e] * A[e];
    off = block_sum_d(off, red);
    if (tid == 0) stop = !(off > 1e-30 * tot_s);
    __syncthreads();
    if (stop) break;
    for (int step = 0; step < m - 1; ++step) {
      // rotations of this step (disjoint pairs)
      for (int k = tid; k < m / 2; k += kThreads) {
        const int p = top[k] < bot[k] ? top[k] : bot[k];
        const int q = top[k] < bot[k] ? bot[k] : top[k];
        double c = 1.0, s = 0.0;
        if (q < r) {
          const double apq = A[p * r + q];
          if (apq != 0.0) {
            const double th = (A[q * r + q] - A[p * r + p]) / (2.0 * apq);
            const double t = (th >= 0.0 ? 1.0 : -1.0) / (fabs(th) + sqrt(th * th + 1.0));
            c = 1.0 / sqrt(t * t + 1.0);
            s = t * c;
          }
        }
        cs[k] = c;
        sn[k] = s;
      }
      __syncthreads();
      // rows: A <- J^T A
      for (int e = tid; e < (m / 2) * r; e += kThreads) {
        const int k = e / r, j = e - (e / r) * r;
        const int p = top[k] < bot[k] ? top[k] : bot[k];
        const int q = top[k] < bot[k] ? bot[k] : top[k];
        if (q < r && sn[k] != 0.0) {
          const double ap = A[p * r + j], aq = A[q * r + j];
          A[p * r + j] = cs[k] * ap - sn[k] * aq;
          A[q * r + j] = sn[k] * ap + cs[k] * aq;
        }
      }
      __syncthreads();
      // columns: A <- A J, V <- V J
      for (int e = tid; e < (m / 2) * r; e += kThreads) {
        const int k = e / r, i = e - (e / r) * r;
        const int p = top[k] < bot[k] ? top[k] : bot[k];
        const int q = top[k] < bot[k] ? bot[k] : top[k];
        if (q < r && sn[k] != 0.0) {
          const double ap = A[i * r + p], aq = A[i * r + q];
          A[i * r + p] = cs[k] * ap - sn[k] * aq;
          A[i * r + q] = sn[k] * ap + cs[k] * aq;
          const double vp = V[i * r + p], vq = V[i * r + q];
          V[i * r + p] = cs[k] * vp - sn[k] * vq;
          V[i * r + q] = sn[k] * vp + cs[k] * vq;
        }
      }
      __syncthreads();
      // next round-robin pairing: player top[0] stays, the others rotate
      if (tid == 0 && m > 2) {
        const int h = m / 2;
        const int last_top = top[h - 1];
        for (int k = h - 1; k > 1; --k) top[k] = top[k - 1];
        if (h > 1) top[1] = bot[0];
        for (int k = 0; k < h - 1; ++k) bot[k] = bot[k + 1];
        bot[h - 1] = last_top;
      }
      __syncthreads();
    }
  }
  // order of eigenvalues, descending, lowest index first among equals
  if (tid == 0) {
    for (int i = 0; i < r; ++i) order[i] = i;
    for (int i = 0; i < K; ++i) {
      int best = i;
      for (int j = i + 1; j < r; ++j)
        if (A[order[j] * r + order[j]] > A[order[best] * r + order[best]]) best = j;
      const int t = order[i];
      order[i] = order[best];
      order[best] = t;
    }
    const double lk = A[order[K - 1] * r + order[K - 1]];
    if (!(lk > 1e-14 * A[order[0] * r + order[0]])) L.flag[0] = 1;
  }
  __syncthreads();
  for (int e = tid; e < r * K; e += kThreads) {
    const int c = e / K, k = e - (e / K) * K;
    const double lam = A[order[k] * r + order[k]];
    L.P[e] = (lam > 0.0) ? V[c * r + order[k]] / sqrt(lam) : 0.0;  // P[c][k]
  }
}

// Initial centroids: E rows at the seed rows.
__global__ __launch_bounds__(kThreads) void k_lab_seed(Geometry g, Bufs B, LabScratch L, int K) {
  const int r = g.r;
  for (int e = threadIdx.x; e < K * K; e += kThreads) {
    const int k = e / K, j = e - (e / K) * K;
    const int64_t row = L.seeds[k];
    double s = 0.0;
    for (int c = 0; c < r; ++c) s += (double)B.U[row * r + c] * L.P[c * K + j];
    L.cent[e] = s;
  }
}

// One assignment pass over a row chunk.  Rows are handled in 64-row tiles: 4
// threads per row compute E_i = U_i P and the distances, the row's label is
// the argmin; then thread (k, j) pairs add the tile's rows of cluster k in row
// order.  Partials: [sums K x K][counts K][changes].
template <int KP>
__global__ __launch_bounds__(kThreads) void k_lab_assign(Geometry g, Bufs B, LabScratch L, int K,
                                                         int32_t* labels, int first) {
  __shared__ double et[kLabTile][KP + 1];
  __shared__ int lt[kLabTile];
  __shared__ int chg[kThreads];
  const int tid = threadIdx.x;
  const int r = g.r;
  const int64_t n = g.n;
  const int64_t r0 = (int64_t)blockIdx.x * n / L.GA2;
  const int64_t r1 = (int64_t)(blockIdx.x + 1) * n / L.GA2;
  const int row_in = tid >> 2, part = tid & 3;
  constexpr int PPT = (KP * KP + kThreads - 1) / kThreads;  // (k, j) pairs per thread
  double acc[PPT];
#pragma unroll
  for (int i = 0; i < PPT; ++i) acc[i] = 0.0;
  int cnt_local = 0, changes = 0;
  for (int64_t t0 = r0; t0 < r1; t0 += kLabTile) {
    const int64_t row = t0 + row_in;
    const bool valid = row < r1;
    // embedding values j = part, part + 4, ...
    for (int j = part; j < K; j += 4) {
      double s = 0.0;
      if (valid)
        for (int c = 0; c < r; ++c) s += (double)B.U[row * r + c] * L.P[c * K + j];
      et[row_in][j] = s;
    }
    __syncthreads();
    // distances for clusters k = part, part + 4, ...; argmin over the 4 threads of the row
    double best = 1e300;
    int bk = 0x7fffffff;
    for (int k = part; k < K; k += 4) {
      double dsum = 0.0;
      for (int j = 0; j < K; ++j) {
        const double t = et[row_in][j] - L.cent[k * K + j];
        dsum += t * t;
      }
      if (dsum < best) {
        best = dsum;
        bk = k;
      }
    }
#pragma unroll
    for (int msk = 1; msk <= 2; msk <<= 1) {
      const double ob = __shfl_xor(best, msk, 64);
      const int ok = __shfl_xor(bk, msk, 64);
      if (ob < best || (ob == best && ok < bk)) {
        best = ob;
        bk = ok;
      }
    }
    if (part == 0) {
      lt[row_in] = valid ? bk : -1;
      if (valid) {
        if (first || labels[row] != bk) ++changes;
        labels[row] = bk;
      }
    }
    __syncthreads();
    // cluster sums, rows in order
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int pr = tid + i * kThreads;
      if (pr < K * K) {
        const int k = pr / K, j = pr - (pr / K) * K;
        double a = acc[i];
        for (int rr = 0; rr < kLabTile; ++rr)
          if (lt[rr] == k) a += et[rr][j];
        acc[i] = a;
      }
    }
    if (tid < K)
      for (int rr = 0; rr < kLabTile; ++rr) cnt_local += (lt[rr] == tid) ? 1 : 0;
    __syncthreads();
  }
  double* out = L.apart + (int64_t)blockIdx.x * (K * K + K + 1);
#pragma unroll
  for (int i = 0; i < PPT; ++i) {
    const int pr = tid + i * kThreads;
    if (pr < K * K) out[pr] = acc[i];
  }
  if (tid < K) out[K * K + tid] = (double)cnt_local;
  chg[tid] = changes;
  __syncthreads();
  if (tid == 0) {
    int c = 0;
    for (int i = 0; i < kThreads; ++i) c += chg[i];
    out[K * K + K] = (double)c;
  }
}

// New centroids from the partials (fixed order); total changed labels to flag[1].
__global__ __launch_bounds__(kThreads) void k_lab_update(LabScratch L, int K) {
  const int stride = K * K + K + 1;
  for (int e = threadIdx.x; e < K * K; e += kThreads) {
    const int k = e / K;
    double s = 0.0, c = 0.0;
    for (int w = 0; w < L.GA2; ++w) {
      s += L.apart[(int64_t)w * stride + e];
      c += L.apart[(int64_t)w * stride + K * K + k];
    }
    if (c > 0.0) L.cent[e] = s / c;
  }
  if (threadIdx.x == 0) {
    double ch = 0.0;
    for (int w = 0; w < L.GA2; ++w) ch += L.apart[(int64_t)w * stride + K * K + K];
    L.flag[1] = (int32_t)ch;
  }
}

hipError_t launch_lab_embed(const Geometry& g, const Bufs& b, const LabScratch& L, int K, hipStream_t st) {
  const int rb = (g.r + 31) / 32;
  hipLaunchKernelGGL(k_lab_gram, dim3(L.GU, rb * rb), dim3(kThreads), 0, st, g, b, L);
  hipLaunchKernelGGL(k_lab_gram_reduce, dim3((g.r * g.r + kThreads - 1) / kThreads), dim3(kThreads), 0, st, g, L);
  hipLaunchKernelGGL(k_lab_eig, dim3(1), dim3(kThreads), 0, st, g, L, K);
  hipLaunchKernelGGL(k_lab_seed, dim3(1), dim3(kThreads), 0, st, g, b, L, K);
  return hipGetLastError();
}

hipError_t launch_lab_pass(const Geometry& g, const Bufs& b, const LabScratch& L, int K, int32_t* labels,
                           int first, hipStream_t st) {
  if (K <= 16)
    hipLaunchKernelGGL((k_lab_assign<16>), dim3(L.GA2), dim3(kThreads), 0, st, g, b, L, K, labels, first);
  else if (K <= 32)
    hipLaunchKernelGGL((k_lab_assign<32>), dim3(L.GA2), dim3(kThreads), 0, st, g, b, L, K, labels, first);
  else if (K <= 64)
    hipLaunchKernelGGL((k_lab_assign<64>), dim3(L.GA2), dim3(kThreads), 0, st, g, b, L, K, labels, first);
  else if (K <= 128)
    hipLaunchKernelGGL((k_lab_assign<128>), dim3(L.GA2), dim3(kThreads), 0, st, g, b, L, K, labels, first);
  else
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_lab_update, dim3(1), dim3(kThreads), 0, st, L, K);
  return hipGetLastError();
}

}  // namespace nlr
