// Initialisation kernels for gfx950: centring and spectral normalisation
// (Section 3: X_c = X - 1 xbar^T, a = ||X_c||_2, Xhat = X_c / a), projection of
// the starting factor onto Omega (eq. projected-primal-step) and p = U^T 1.
//
// a is found as sqrt(lambda_max(C)) with C = X_c^T X_c (FP64), by the power
// method: C is first squared kSquarings times with trace normalisation
// (B_{k+1} = (B_k / tr B_k)^2, i.e. the power C^(2^k) up to scale), the column
// of the last B with the largest diagonal entry starts kPowerIters ordinary
// power iterations on C, and the Rayleigh quotient of the final unit vector is
// lambda_max.  Appendix D notes C is reused from this normalisation by the
// data-informed initialisation.
#include "nlr_internal.hpp"

namespace nlr {

__global__ void k_ctl_init(Bufs B, float gamma_f) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    DevCtl* c = B.ctl;
    c->stop = 0;
    c->breakdown = 0;
    c->gate = 0;
    c->degenerate = 0;
    c->t_done = 0;
    c->c_f = 1.0f;
    c->x_scale = 1.0f;
    c->th_scale = 1.0f;
    c->rows_first = 0;
    c->rows_run = 0;
    c->a = c->b = c->h = 0.0;
    c->Delta = c->delta = 0.0;
    c->rho = c->objective = c->theta_fro2 = 0.0;
    c->spectral_a = 1.0;
    c->c_gram = 1.0;
  }
}

__global__ void k_clear_stop(Bufs B) {
  if (threadIdx.x == 0 && blockIdx.x == 0) B.ctl->stop = 0;
}

// Column sums of X over row chunks (FP64).  Threads map to (column, row offset).
__global__ __launch_bounds__(kThreads) void k_colsum(Geometry g, Bufs B) {
  __shared__ double red[kThreads];
  const int tid = threadIdx.x;
  const int64_t n = g.n;
  const int d = g.d;
  const int64_t r0 = (int64_t)blockIdx.x * n / g.GI;
  const int64_t r1 = (int64_t)(blockIdx.x + 1) * n / g.GI;
  double* out = B.i_colsum + (int64_t)blockIdx.x * d;
  if (d <= kThreads) {
    const int rstep = kThreads / d;
    const int col = tid % d;
    const int rsub = tid / d;
    double acc = 0.0;
    if (rsub < rstep) {
      // sixteen rows' loads in flight, added in row order
      int64_t i = r0 + rsub;
      for (; i + 15 * rstep < r1; i += 16 * rstep) {
        float v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) v[u] = B.X[(i + u * rstep) * d + col];
#pragma unroll
        for (int u = 0; u < 16; ++u) acc += (double)v[u];
      }
      for (; i < r1; i += rstep) acc += (double)B.X[i * d + col];
    }
    red[tid] = acc;
    __syncthreads();
    if (tid < d) {
      double t = 0.0;
      for (int k = 0; k < rstep; ++k) t += red[tid + k * d];
      out[tid] = t;
    }
  } else {
    for (int col = tid; col < d; col += kThreads) {
      double acc = 0.0;
      int64_t i = r0;
      for (; i + 7 < r1; i += 8) {  // eight rows' loads in flight, added in row order
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = B.X[(i + u) * d + col];
#pragma unroll
        for (int u = 0; u < 8; ++u) acc += (double)v[u];
      }
      for (; i < r1; ++i) acc += (double)B.X[i * d + col];
      out[col] = acc;
    }
  }
}

__global__ __launch_bounds__(kThreads) void k_colmean(Geometry g, Bufs B) {
  const int j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= g.d) return;
  double t = 0.0;
  for (int gx = 0; gx < g.GI; ++gx) t += B.i_colsum[(int64_t)gx * g.d + j];
  B.i_xbar[j] = t / (double)g.n;
}

// Partial centred Gram blocks on the fp64 matrix cores (v_mfma_f64_16x16x4f64):
// workgroup (chunk gx, block pair bp) adds the 64 x 64 block (bi, bj), bi <= bj, of
// the sum over the chunk's rows of (x - xbar)(x - xbar)^T.  Wave w owns the block
// rows 16 w .. 16 w + 15 and all 64 columns (four 16 x 16 tiles).  A product step
// takes 4 data rows: lane l reads row l / 16 of the step and feature l % 16 of its
// tile from LDS (the A operand from the block's rows, the B operands from its columns), and
// holds result element (4 v + l / 16, l % 16) of a tile in entry v.  The blocks
// below the diagonal are not formed (the sum is symmetric; k_gram_reduce reads
// their mirror).
typedef double f64x4_t __attribute__((ext_vector_type(4)));
static_assert(kThreads == 256, "k_gram stages a 32 x 64 operand as 8 elements per thread of 4 waves");
__global__ __launch_bounds__(kThreads) void k_gram(Geometry g, Bufs B) {
  const int tid = threadIdx.x;
  const int d = g.d;
  const int nb = (d + 63) / 64;
  int bp = blockIdx.y, bi = 0;
  while (bp >= nb - bi) {
    bp -= nb - bi;
    ++bi;
  }
  const int bj = bi + bp;
  const int64_t n = g.n;
  const int64_t r0 = (int64_t)blockIdx.x * n / g.GG;
  const int64_t r1 = (int64_t)(blockIdx.x + 1) * n / g.GG;
  const int lane = tid & 63, w = tid >> 6;
  const int kq = lane >> 4, cl = lane & 15;
  f64x4_t acc[4];
#pragma unroll
  for (int J = 0; J < 4; ++J) acc[J] = (f64x4_t){0.0, 0.0, 0.0, 0.0};
  // Rounds of 32 rows.  The round's centred values of the block's 64 row features
  // and 64 column features are formed once in FP64 by the workgroup and staged in
  // LDS (rows padded to 80 doubles, so that the 32 lanes of a read pass meet all 64
  // banks); the next round's raw values are loaded while the matrix cores take this
  // round's.
  __shared__ double xs[2][32][80];
  const bool same = bi == bj;
  // element k = tid + 256 q (q = 0..7) of a 32 x 64 operand: row k / 64, feature k % 64
  const int sf = tid & 63, sr = tid >> 6;  // feature, first row (rows sr + 4 q)
  const int fsa = 64 * bi + sf, fsb = 64 * bj + sf;
  const bool oksa = fsa < d, oksb = fsb < d;
  const double msa = oksa ? B.i_xbar[fsa] : 0.0, msb = oksb ? B.i_xbar[fsb] : 0.0;
  float ra[8], rb[8];
  auto load_round = [&](int64_t t0) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int64_t row = t0 + sr + 4 * q;
      const int64_t rb0 = (row < r1 ? row : r0) * (int64_t)d;
      ra[q] = B.X[rb0 + (oksa ? fsa : 0)];
      rb[q] = same ? 0.f : B.X[rb0 + (oksb ? fsb : 0)];
    }
  };
  if (r0 < r1) load_round(r0);
  for (int64_t t0 = r0; t0 < r1; t0 += 32) {
    __syncthreads();  // the previous round's operands are consumed
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const bool okr = t0 + sr + 4 * q < r1;
      xs[0][sr + 4 * q][sf] = (okr && oksa) ? (double)ra[q] - msa : 0.0;
      if (!same) xs[1][sr + 4 * q][sf] = (okr && oksb) ? (double)rb[q] - msb : 0.0;
    }
    __syncthreads();
    if (t0 + 32 < r1) load_round(t0 + 32);
    const int ob = same ? 0 : 1;
#pragma unroll
    for (int st = 0; st < 8; ++st) {
      const int row = 4 * st + kq;
      const double a = xs[0][row][16 * w + cl];
#pragma unroll
      for (int J = 0; J < 4; ++J) {
        const double b = xs[ob][row][16 * J + cl];
        acc[J] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc[J], 0, 0, 0);
      }
    }
  }
  double* out = B.i_gram + (int64_t)blockIdx.x * d * d;
#pragma unroll
  for (int J = 0; J < 4; ++J)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int ia = 64 * bi + 16 * w + 4 * v + kq;
      const int jb = 64 * bj + 16 * J + cl;
      if (ia < d && jb < d) out[(int64_t)ia * d + jb] = acc[J][v];
    }
}

// C = the sum of the chunks' partials in chunk order; entries below the block
// diagonal from the mirrored entry.
__global__ __launch_bounds__(kThreads) void k_gram_reduce(Geometry g, Bufs B) {
  const int64_t dd = (int64_t)g.d * g.d;
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= dd) return;
  const int i = (int)(e / g.d), j = (int)(e - (int64_t)i * g.d);
  const int64_t src = (i / 64 > j / 64) ? (int64_t)j * g.d + i : e;
  double t = 0.0;
  for (int gx = 0; gx < g.GG; ++gx) t += B.i_gram[(int64_t)gx * dd + src];
  B.i_C[e] = t;
}

// scal[slot] = 1 / trace(M) (0 when the trace is not positive).
__global__ __launch_bounds__(kThreads) void k_trace(Geometry g, const double* __restrict__ M, double* scal, int slot) {
  __shared__ double red[8];
  double t = 0.0;
  for (int i = threadIdx.x; i < g.d; i += kThreads) t += M[(int64_t)i * g.d + i];
  t = block_sum_d(t, red);
  if (threadIdx.x == 0) scal[slot] = (t > 0.0 && isfinite(t)) ? 1.0 / t : 0.0;
}

// out = (in * scal[slot])^2 for a symmetric d x d matrix (32 x 32 tiles).
__global__ __launch_bounds__(kThreads) void k_square(Geometry g, const double* __restrict__ in, double* __restrict__ out,
                                                     const double* scal, int slot) {
  __shared__ double As[32][33];
  __shared__ double Bs[32][33];
  const int d = g.d;
  const int tid = threadIdx.x;
  const int ty = tid >> 3, tx = tid & 7;
  const int bi = blockIdx.y, bj = blockIdx.x;
  const double s = scal[slot];
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int k0 = 0; k0 < d; k0 += 32) {
    __syncthreads();
    for (int v = tid; v < 32 * 32; v += kThreads) {
      const int rr = v >> 5, cc = v & 31;
      const int ia = bi * 32 + rr, ka = k0 + cc;
      const int kb = k0 + rr, jb = bj * 32 + cc;
      As[rr][cc] = (ia < d && ka < d) ? in[(int64_t)ia * d + ka] * s : 0.0;
      Bs[rr][cc] = (kb < d && jb < d) ? in[(int64_t)kb * d + jb] * s : 0.0;
    }
    __syncthreads();
#pragma unroll 8
    for (int k = 0; k < 32; ++k) {
      const double a = As[ty][k];
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] += a * Bs[k][4 * tx + e];
    }
  }
  const int ia = bi * 32 + ty;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int jb = bj * 32 + 4 * tx + e;
    if (ia < d && jb < d) out[(int64_t)ia * d + jb] = acc[e];
  }
}

// Power iterations on C from the dominant column of Bf; a = sqrt(Rayleigh quotient).
__global__ __launch_bounds__(kThreads) void k_power(Geometry g, Bufs B, const double* __restrict__ Bf) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  double* v = reinterpret_cast<double*>(smem_raw);  // d
  double* w = v + g.d;                               // d
  __shared__ double red[8];
  __shared__ double sh[2];
  __shared__ int shi[1];
  const int d = g.d;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const double* C = B.i_C;
  // start column: largest diagonal of Bf, lowest index on ties
  if (tid == 0) {
    double best = -1.0;
    int arg = 0;
    for (int j = 0; j < d; ++j) {
      const double x = Bf[(int64_t)j * d + j];
      if (x > best) {
        best = x;
        arg = j;
      }
    }
    shi[0] = arg;
  }
  __syncthreads();
  const int j0 = shi[0];
  double nn = 0.0;
  for (int i = tid; i < d; i += kThreads) {
    v[i] = Bf[(int64_t)i * d + j0];
    nn += v[i] * v[i];
  }
  nn = block_sum_d(nn, red);
  if (tid == 0) sh[0] = nn;
  __syncthreads();
  double inv = (sh[0] > 0.0) ? 1.0 / sqrt(sh[0]) : 0.0;
  for (int i = tid; i < d; i += kThreads) v[i] *= inv;
  __syncthreads();
  double lam = 0.0;
  for (int it = 0; it <= kPowerIters; ++it) {
    // w = C v, one wave per row (four rows of a wave at a time, their loads in
    // flight together), lanes stride the columns
    for (int i0 = 4 * wave; i0 < d; i0 += 16) {
      double t[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
      for (int j = lane; j < d; j += 64) {
        const double vj = v[j];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (i0 + q < d) t[q] += C[(int64_t)(i0 + q) * d + j] * vj;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        double tq = t[q];
        for (int m = 32; m >= 1; m >>= 1) tq += shfl_xor_d(tq, m);
        if (lane == 0 && i0 + q < d) w[i0 + q] = tq;
      }
    }
    __syncthreads();
    double vw = 0.0, ww = 0.0;
    for (int i = tid; i < d; i += kThreads) {
      vw += v[i] * w[i];
      ww += w[i] * w[i];
    }
    vw = block_sum_d(vw, red);
    ww = block_sum_d(ww, red);
    if (tid == 0) {
      sh[0] = vw;
      sh[1] = ww;
    }
    __syncthreads();
    lam = sh[0];  // Rayleigh quotient of the unit vector v
    if (it == kPowerIters) break;
    inv = (sh[1] > 0.0) ? 1.0 / sqrt(sh[1]) : 0.0;
    for (int i = tid; i < d; i += kThreads) v[i] = w[i] * inv;
    __syncthreads();
  }
  if (tid == 0) {
    const double a = (lam > 0.0) ? sqrt(lam) : 0.0;
    B.ctl->spectral_a = a;
    if (!(a > 0.0) || !isfinite(a)) B.ctl->degenerate = 1;
  }
}

// X <- (X - 1 xbar^T) / a in place; 256 rows per workgroup.
// Threads map to (column, row offset) as in k_colsum, eight rows' loads in flight.
__global__ __launch_bounds__(kThreads) void k_normalise(Geometry g, Bufs B) {
  if (B.ctl->degenerate) return;
  const double a = B.ctl->spectral_a;
  const int d = g.d;
  const int tid = threadIdx.x;
  const int64_t row0 = (int64_t)blockIdx.x * 256;
  const int64_t row1 = (g.n - row0) < 256 ? g.n : row0 + 256;
  auto one = [&](int64_t i, int col, double xb) {
    float* p = B.X + i * d + col;
    *p = (float)(((double)*p - xb) / a);
  };
  if (d <= kThreads) {
    const int rstep = kThreads / d;
    const int col = tid % d;
    const int rsub = tid / d;
    if (rsub >= rstep) return;
    const double xb = B.i_xbar[col];
    int64_t i = row0 + rsub;
    for (; i + 7 * rstep < row1; i += 8 * rstep) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = B.X[(i + u * rstep) * d + col];
#pragma unroll
      for (int u = 0; u < 8; ++u) B.X[(i + u * rstep) * d + col] = (float)(((double)v[u] - xb) / a);
    }
    for (; i < row1; i += rstep) one(i, col, xb);
  } else {
    for (int col = tid; col < d; col += kThreads) {
      const double xb = B.i_xbar[col];
      int64_t i = row0;
      for (; i + 7 < row1; i += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = B.X[(i + u) * d + col];
#pragma unroll
        for (int u = 0; u < 8; ++u) B.X[(i + u) * d + col] = (float)(((double)v[u] - xb) / a);
      }
      for (; i < row1; ++i) one(i, col, xb);
    }
  }
}

// Projection statistics over row chunks: sum of (u_+)^2 and column sums of u_+.
__global__ __launch_bounds__(kThreads) void k_proj_partial(Geometry g, Bufs B) {
  __shared__ double red[kThreads];
  __shared__ double red8[8];
  const int tid = threadIdx.x;
  const int64_t n = g.n;
  const int r = g.r;
  const int64_t r0 = (int64_t)blockIdx.x * n / g.GI;
  const int64_t r1 = (int64_t)(blockIdx.x + 1) * n / g.GI;
  double* out = B.i_proj + (int64_t)blockIdx.x * (4 + g.r32);
  // r <= 256: column tid % r, every (256 / r)-th row; else columns tid, tid + 256, every row
  const int rstep = r <= kThreads ? kThreads / r : 1;
  const int col = tid % r;
  const int rsub = r <= kThreads ? tid / r : 0;
  double cs = 0.0, sq = 0.0;
  if (r > kThreads) {
    for (int c = tid; c < r; c += kThreads) {
      double csc = 0.0;
      for (int64_t i = r0; i < r1; ++i) {
        const float u = fmaxf(B.U[i * r + c], 0.f);
        csc += (double)u;
        sq += (double)u * (double)u;
      }
      out[4 + c] = csc;
    }
  } else if (rsub < rstep) {
    // sixteen rows' loads in flight, added in row order
    int64_t i = r0 + rsub;
    for (; i + 15 * rstep < r1; i += 16 * rstep) {
      float v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = B.U[(i + u * rstep) * r + col];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const float uu = fmaxf(v[u], 0.f);
        cs += (double)uu;
        sq += (double)uu * (double)uu;
      }
    }
    for (; i < r1; i += rstep) {
      const float u = fmaxf(B.U[i * r + col], 0.f);
      cs += (double)u;
      sq += (double)u * (double)u;
    }
  }
  red[tid] = cs;
  __syncthreads();
  if (tid < r && r <= kThreads) {
    double t = 0.0;
    for (int k = 0; k < rstep; ++k) t += red[tid + k * r];
    out[4 + tid] = t;
  }
  const double tsq = block_sum_d(sq, red8);
  if (tid == 0) {
    out[0] = tsq;
    out[1] = out[2] = out[3] = 0.0;
  }
}

// c_f = FP32(sqrt(K) / ||U_+||_F) (1 when U is already in Omega); p = FP32(c colsum).
__global__ __launch_bounds__(kThreads) void k_proj_ctl(Geometry g, Bufs B, double K, int in_omega) {
  __shared__ double red[8];
  __shared__ double cbuf[1];
  const int tid = threadIdx.x;
  const int stride = 4 + g.r32;
  double S = 0.0;
  for (int gx = tid; gx < g.GI; gx += kThreads) S += B.i_proj[(int64_t)gx * stride];
  S = block_sum_d(S, red);
  if (tid == 0) {
    double c = 1.0;
    if (!in_omega) {
      const double nu = sqrt(S);
      if (!(nu > 1e-20) || !isfinite(S)) {
        B.ctl->breakdown = 1;
        c = 0.0;
      } else {
        c = (double)(float)(sqrt(K) / nu);
      }
    }
    cbuf[0] = c;
    B.i_scal[0] = c;
  }
  __syncthreads();
  const double c = cbuf[0];
  for (int col = tid; col < g.r32; col += kThreads) {
    double t = 0.0;
    if (col < g.r)
      for (int gx = 0; gx < g.GI; ++gx) t += B.i_proj[(int64_t)gx * stride + 4 + col];
    B.p[col] = (col < g.r) ? (float)(c * t) : 0.f;
  }
}

__global__ __launch_bounds__(kThreads) void k_proj_apply(Geometry g, Bufs B) {
  if (B.ctl->breakdown) return;
  const float cf = (float)B.i_scal[0];
  const int64_t tot = g.n * (int64_t)g.r;
  for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < tot; e += (int64_t)gridDim.x * kThreads)
    B.U[e] = cf * fmaxf(B.U[e], 0.f);
}

__global__ __launch_bounds__(kThreads) void k_zero_y(Geometry g, Bufs B) {
  for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < g.n; e += (int64_t)gridDim.x * kThreads)
    B.y[e] = 0.f;
}

// ---------------------------------------------------------------------------
// The same power method for wide inputs (d > 256), the matrix-vector products
// spread over workgroups: C does not stay in one compute unit's cache there, and
// one workgroup streaming it each iteration dominates the initialisation.
// v and w live in the squaring buffer the last squaring did not write (vw[0..d),
// vw[d..2d)); state[0] the Rayleigh quotient.
// ---------------------------------------------------------------------------
// v = the column of Bf with the largest diagonal entry (lowest index on ties), normalised.
__global__ __launch_bounds__(kThreads) void k_power_start(Geometry g, const double* __restrict__ Bf,
                                                          double* __restrict__ vw) {
  __shared__ double red[8];
  __shared__ int shi[1];
  __shared__ double sh[1];
  const int d = g.d, tid = threadIdx.x;
  if (tid == 0) {
    double best = -1.0;
    int arg = 0;
    for (int j = 0; j < d; ++j) {
      const double x = Bf[(int64_t)j * d + j];
      if (x > best) {
        best = x;
        arg = j;
      }
    }
    shi[0] = arg;
  }
  __syncthreads();
  const int j0 = shi[0];
  double nn = 0.0;
  for (int i = tid; i < d; i += kThreads) {
    const double x = Bf[(int64_t)i * d + j0];
    nn += x * x;
  }
  nn = block_sum_d(nn, red);
  if (tid == 0) sh[0] = nn;
  __syncthreads();
  const double inv = (sh[0] > 0.0) ? 1.0 / sqrt(sh[0]) : 0.0;
  for (int i = tid; i < d; i += kThreads) vw[i] = Bf[(int64_t)i * d + j0] * inv;
}

// w = C v: workgroup b forms rows 64 b .. 64 b + 63; lane l row 64 b + l (column l of the
// symmetric C, read row by row: coalesced), wave k the terms j = k, k + 4, ...; the four
// partial sums are added in order.
__global__ __launch_bounds__(kThreads) void k_power_mv(Geometry g, const double* __restrict__ C,
                                                       double* __restrict__ vw) {
  __shared__ double part[kThreads];
  const int d = g.d, tid = threadIdx.x;
  const int i = blockIdx.x * 64 + (tid & 63), sub = tid >> 6;
  const double* v = vw;
  double t = 0.0;
  if (i < d)
#pragma unroll 4
    for (int j = sub; j < d; j += 4) t += C[(int64_t)j * d + i] * v[j];
  part[tid] = t;
  __syncthreads();
  if (sub == 0 && i < d) vw[d + i] = ((part[tid] + part[64 + tid]) + part[128 + tid]) + part[192 + tid];
}

// Rayleigh quotient of v, then v = w / |w| (not after the last product); with last set,
// a = sqrt(Rayleigh quotient) to the control block.
__global__ __launch_bounds__(kThreads) void k_power_norm(Geometry g, Bufs B, double* __restrict__ vw, int last) {
  __shared__ double red[8];
  __shared__ double sh[2];
  const int d = g.d, tid = threadIdx.x;
  double s1 = 0.0, s2 = 0.0;
  for (int i = tid; i < d; i += kThreads) {
    s1 += vw[i] * vw[d + i];
    s2 += vw[d + i] * vw[d + i];
  }
  s1 = block_sum_d(s1, red);
  s2 = block_sum_d(s2, red);
  if (tid == 0) {
    sh[0] = s1;
    sh[1] = s2;
  }
  __syncthreads();
  if (last) {
    if (tid == 0) {
      const double lam = sh[0];
      const double a = (lam > 0.0) ? sqrt(lam) : 0.0;
      B.ctl->spectral_a = a;
      if (!(a > 0.0) || !isfinite(a)) B.ctl->degenerate = 1;
    }
    return;
  }
  const double inv = (sh[1] > 0.0) ? 1.0 / sqrt(sh[1]) : 0.0;
  for (int i = tid; i < d; i += kThreads) vw[i] = vw[d + i] * inv;
}

// ---------------------------------------------------------------------------
hipError_t launch_ctl_init(const Bufs& b, float gamma_f, hipStream_t st) {
  hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(64), 0, st, b, gamma_f);
  return hipGetLastError();
}

hipError_t launch_clear_stop(const Bufs& b, hipStream_t st) {
  hipLaunchKernelGGL(k_clear_stop, dim3(1), dim3(64), 0, st, b);
  return hipGetLastError();
}

hipError_t launch_colsum(const Geometry& g, const Bufs& b, hipStream_t st) {
  hipLaunchKernelGGL(k_colsum, dim3(g.GI), dim3(kThreads), 0, st, g, b);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_colmean, dim3((g.d + kThreads - 1) / kThreads), dim3(kThreads), 0, st, g, b);
  return hipGetLastError();
}

hipError_t launch_gram(const Geometry& g, const Bufs& b, hipStream_t st) {
  const int nb = (g.d + 63) / 64;
  hipLaunchKernelGGL(k_gram, dim3(g.GG, nb * (nb + 1) / 2), dim3(kThreads), 0, st, g, b);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t dd = (int64_t)g.d * g.d;
  hipLaunchKernelGGL(k_gram_reduce, dim3((unsigned)((dd + kThreads - 1) / kThreads)), dim3(kThreads), 0, st, g, b);
  return hipGetLastError();
}

hipError_t launch_spectral(const Geometry& g, const Bufs& b, hipStream_t st) {
  // B_0 = C; scal[k] = 1/tr(B_k); B_{k+1} = (B_k scal[k])^2, ping-ponging B0/B1.
  hipLaunchKernelGGL(k_trace, dim3(1), dim3(kThreads), 0, st, g, (const double*)b.i_C, b.i_scal, 1);
  const double* in = b.i_C;
  double* bufs[2] = {b.i_B0, b.i_B1};
  const dim3 grid(g.gblk, g.gblk);
  for (int k = 0; k < kSquarings; ++k) {
    double* out = bufs[k & 1];
    hipLaunchKernelGGL(k_square, grid, dim3(kThreads), 0, st, g, in, out, (const double*)b.i_scal, 1 + k);
    hipLaunchKernelGGL(k_trace, dim3(1), dim3(kThreads), 0, st, g, (const double*)out, b.i_scal, 2 + k);
    in = out;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (g.d > kThreads) {
    // wide inputs: the products over workgroups; v and w in the buffer the last
    // squaring did not write
    double* vw = (in == b.i_B0) ? b.i_B1 : b.i_B0;
    hipLaunchKernelGGL(k_power_start, dim3(1), dim3(kThreads), 0, st, g, in, vw);
    for (int it = 0; it <= kPowerIters; ++it) {
      hipLaunchKernelGGL(k_power_mv, dim3((g.d + 63) / 64), dim3(kThreads), 0, st, g, (const double*)b.i_C, vw);
      hipLaunchKernelGGL(k_power_norm, dim3(1), dim3(kThreads), 0, st, g, b, vw, it == kPowerIters ? 1 : 0);
    }
    return hipGetLastError();
  }
  const size_t lds = 2 * (size_t)g.d * sizeof(double);
  if (lds > (64u << 10)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_power), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_power, dim3(1), dim3(kThreads), lds, st, g, b, in);
  return hipGetLastError();
}

hipError_t launch_normalise(const Geometry& g, const Bufs& b, hipStream_t st) {
  const int64_t blocks = (g.n + 255) / 256;
  hipLaunchKernelGGL(k_normalise, dim3((unsigned)blocks), dim3(kThreads), 0, st, g, b);
  return hipGetLastError();
}

hipError_t launch_project(const Geometry& g, const Bufs& b, double K, int in_omega, hipStream_t st) {
  hipLaunchKernelGGL(k_proj_partial, dim3(g.GI), dim3(kThreads), 0, st, g, b);
  hipLaunchKernelGGL(k_proj_ctl, dim3(1), dim3(kThreads), 0, st, g, b, K, in_omega);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || in_omega) return e;
  hipLaunchKernelGGL(k_proj_apply, dim3(2048), dim3(kThreads), 0, st, g, b);
  return hipGetLastError();
}

hipError_t launch_zero_y(const Geometry& g, const Bufs& b, hipStream_t st) {
  hipLaunchKernelGGL(k_zero_y, dim3(1024), dim3(kThreads), 0, st, g, b);
  return hipGetLastError();
}

}  // namespace nlr
