// Per-iteration kernels of the NLR iteration (Algorithm 1, Section 4) for gfx950.
//
// One iteration is
//   pass A        Theta partials = Xhat^T U over row chunks (fp32 matrix cores),
//                 fused with the row work that ends the previous iteration and
//                 prepares this one: u = fl(c_f w) (lazy normalisation), q = u.p - 1,
//                 gated dual step ytilde += (beta/n) q, ybar = ytilde + (beta/n) q,
//                 s partials = U^T ybar, ||q||^2 and ytilde^T q partials
//                 (eq. gpu-vectors; Appendix C call sites 2, 3, 7-11);
//   reduce_theta  fixed-order FP64 sum of the Theta partials, ||Theta||_F^2;
//   ctl_a         s, rho, objective fhat (eq. normalized), stopping rule (Section 4.3);
//   pass B        G = Xhat Theta on fp32 matrix cores with the epilogue of
//                 eq. (entrywise-fusion): w = max(u + 2 alpha G - alpha ybar p - alpha s, 0),
//                 FP64 statistics a = ||W||^2, b = ||U||^2, h = <W, U> (eq. fused-statistics)
//                 and column sums of W, W stored over U in place;
//   ctl_b         a, b, h, column sums -> c_f = FP32(sqrt(K)/sqrt(a)), breakdown test,
//                 Delta = max(c^2 a + b - 2 c h, 0), delta, dual gate Delta < eps_d^2 K,
//                 p = FP32(c * colsum) (eq. movement-estimate, Appendix B Alg. 2 (d)-(f)).
// The rescale U <- c W is never a separate pass: every consumer reads fl(c_f w).
// "finish" is pass A without the matrix product: it materialises U = fl(c_f w)
// and applies the pending end-of-iteration work, so a host call always returns
// a materialised factor.
#include "k_common.hpp"

namespace nlr {

// ---------------------------------------------------------------------------
// Tile staging: rows [row0, row0+kTPA) x cols [c0, c0+cw) of a row-major matrix
// with leading dimension ld, multiplied by `scale`, into LDS with row stride ls.
// Rows >= n and cols >= cmax are zero-filled.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void stage_tile(float* __restrict__ dst, int ls, const float* __restrict__ src,
                                           int64_t ld, int64_t n, int64_t row0, int c0, int cw,
                                           int cmax, float scale, bool vec) {
  if (vec) {
    const int cw4 = cw >> 2;
    const int total = kTPA * cw4;
    for (int v = threadIdx.x; v < total; v += kThreads) {
      const int row = v / cw4;
      const int c = (v - row * cw4) * 4;
      const int64_t gr = row0 + row;
      f32x4 x = {0.f, 0.f, 0.f, 0.f};
      if (gr < n && c0 + c < cmax) {
        x = *reinterpret_cast<const f32x4*>(src + gr * ld + c0 + c);
        x.x = x.x * scale;
        x.y = x.y * scale;
        x.z = x.z * scale;
        x.w = x.w * scale;
      }
      *reinterpret_cast<f32x4*>(dst + row * ls + c) = x;
    }
  } else {
    const int total = kTPA * cw;
    for (int v = threadIdx.x; v < total; v += kThreads) {
      const int row = v / cw;
      const int c = v - row * cw;
      const int64_t gr = row0 + row;
      float x = 0.f;
      if (gr < n && c0 + c < cmax) x = src[gr * ld + c0 + c] * scale;
      dst[row * ls + c] = x;
    }
  }
}

// ---------------------------------------------------------------------------
// Pass A.  Grid (GA, mgroups*ngroups).  Workgroup (gx, gy) owns a contiguous
// range of kTPA-row tiles and the Theta blocks of group gy (MBG x NBG blocks of
// 32 x 32).  Wave w owns m-block w % MBG and all NBG n-blocks, over the k-slice
// w / MBG of each tile (KS = 4 / MBG slices).  Group 0 also does the row work.
// MODE kAFinish: no matrix product; materialise U and do the row work only.
// Above 128 columns the iteration's pass A runs as two launches: the row work
// (k_rows_wide, below) and kATheta: the product alone, every group staging only its
// own columns of U, so that a workgroup's LDS is about a third of the combined form's.
// ---------------------------------------------------------------------------
constexpr int kAIter = 0, kAFinish = 1, kATheta = 2;
template <int MBG, int NBG, int MODE>
__global__ __launch_bounds__(kThreads) void k_pass_a(Geometry g, Bufs B, StepArgs S) {
  constexpr bool FINISH = MODE == kAFinish;
  constexpr bool THETA = MODE == kAIter || MODE == kATheta;  // the matrix product
  constexpr bool ROWS = MODE != kATheta;                     // the row work (group 0)
  // The finish pass runs after a stop (it still materialises U) but not after a breakdown.
  if (FINISH ? (B.ctl->breakdown != 0) : halted(B.ctl)) return;
  const bool stopped = FINISH && (B.ctl->stop != 0);
  constexpr int KS = 4 / MBG;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  float* smem = reinterpret_cast<float*>(smem_raw);
  const int xs_stride = g.xs_stride;  // MBG*32
  const int us_stride = MODE == kATheta ? NBG * 32 + 4 : g.us_stride;  // staged columns + 4
  float* Xs = smem;                                  // kTPA x xs_stride
  float* Us = Xs + (THETA ? kTPA * xs_stride : 0);   // kTPA x us_stride
  float* ybar_s = Us + kTPA * us_stride;             // kTPA
  float* p_s = ybar_s + kTPA;                        // r32
  double* dred = reinterpret_cast<double*>(p_s + g.r32);  // 256 + 8 doubles (8-byte aligned: r32 even)

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int gx = blockIdx.x;
  const int gy = blockIdx.y;
  const int mg = gy / g.ngroups;
  const int ng = gy - mg * g.ngroups;
  const bool do_rows = ROWS && (gy == 0);
  const int64_t n = g.n;
  const int d = g.d, r = g.r, r32 = g.r32;
  const int f0 = mg * MBG * 32;       // first feature of the group
  const int c0 = ng * NBG * 32;       // first column of the group
  const float cf = B.ctl->c_f;
  // after a stop the end-of-iteration work was already done by pass A
  const bool gate = (S.end_work != 0) && (B.ctl->gate != 0) && !stopped;
  const float gam = S.gamma_f;

  // the grid is GA (Theta product) or GAF (finish pass, row-work launch)
  const int64_t tb = (int64_t)gx * g.tilesA / gridDim.x;
  const int64_t te = (int64_t)(gx + 1) * g.tilesA / gridDim.x;

  if (do_rows)
    for (int c = tid; c < r32; c += kThreads) p_s[c] = (c < r) ? B.p[c] : 0.f;

  // row-work accumulators
  double acc_qq = 0.0, acc_yq = 0.0, acc_s = 0.0, acc_s2 = 0.0;
  // s ownership: column sc, points ps0, ps0 + pstep, ...; above 256 columns every
  // point, columns tid and tid + 256 (acc_s2)
  const int pstep = kThreads / r32 > 0 ? kThreads / r32 : 1;
  const int sc = tid % r32;
  const int ps0 = tid / r32;
  const int sc2 = tid + kThreads;

  // matrix-core accumulators
  const int mb = wave % MBG;
  const int ks = wave / MBG;
  f32x16 acc[NBG];
#pragma unroll
  for (int j = 0; j < NBG; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;

  const int ucols = do_rows ? r32 : NBG * 32;      // staged U columns
  const int ucol0 = do_rows ? 0 : c0;              // first staged U column
  const int ub = do_rows ? c0 : 0;                 // offset of the group's columns in Us

  for (int64_t tile = tb; tile < te; ++tile) {
    const int64_t row0 = tile * kTPA;
    __syncthreads();
    if (THETA)
      stage_tile(Xs, xs_stride, B.X, d, n, row0, f0, MBG * 32, d, 1.0f, g.vec_x != 0);
    stage_tile(Us, us_stride, B.U, r, n, row0, ucol0, ucols, r, cf, g.vec_u != 0);
    __syncthreads();

    if (do_rows) {
      // R1: four threads per row: q = u.p - 1 (FP64 dot), dual step, ybar.
      const int tp = tid >> 2;
      const int j4 = tid & 3;
      double dot = 0.0;
      for (int c = j4; c < r; c += 4) dot += (double)Us[tp * us_stride + c] * (double)p_s[c];
      dot += shfl_xor_d(dot, 1);
      dot += shfl_xor_d(dot, 2);
      const int64_t gr = row0 + tp;
      float ybar = 0.f;
      if (gr < n) {
        const float q = (float)(dot - 1.0);
        float yt = B.y[gr];
        if (gate) {
          yt = fmaf(gam, q, yt);
          if (j4 == 0) B.y[gr] = yt;
        }
        ybar = fmaf(gam, q, yt);
        if (j4 == 0) {
          acc_qq += (double)q * (double)q;
          acc_yq += (double)yt * (double)q;
        }
      }
      if (j4 == 0) ybar_s[tp] = ybar;
      if (FINISH) {
        // materialise U = fl(c_f w) from the staged tile
        const int64_t rows_here = (n - row0) < kTPA ? (n - row0) : kTPA;
        const int64_t total = rows_here * r;
        for (int64_t v = tid; v < total; v += kThreads) {
          const int rr = (int)(v / r);
          const int cc = (int)(v - (int64_t)rr * r);
          B.U[(row0 + rr) * r + cc] = Us[rr * us_stride + cc];
        }
      }
      __syncthreads();
      if (!FINISH && sc < r) {
        // R2: s_c += ybar_p u_pc
        for (int pt = ps0; pt < kTPA; pt += pstep)
          acc_s += (double)ybar_s[pt] * (double)Us[pt * us_stride + sc];
      }
      if (!FINISH && sc2 < r)
        for (int pt = 0; pt < kTPA; ++pt) acc_s2 += (double)ybar_s[pt] * (double)Us[pt * us_stride + sc2];
    }

    if (THETA) {
      // Theta_blk += Xs^T Us over this wave's k-slice (2 rows per instruction).
      const int kbeg = ks * (kTPA / KS);
      const int kend = kbeg + kTPA / KS;
      const int lr = lane >> 5;   // row within the pair
      const int lc = lane & 31;
#pragma unroll 4
      for (int k = kbeg; k < kend; k += 2) {
        const float a = Xs[(k + lr) * xs_stride + mb * 32 + lc];
#pragma unroll
        for (int j = 0; j < NBG; ++j) {
          const float bv = Us[(k + lr) * us_stride + ub + j * 32 + lc];
          acc[j] = mfma32x32x2(a, bv, acc[j]);
        }
      }
    }
  }

  // ---- write partials ----
  if (THETA) {
    // combine k-slices (waves with the same m-block) in a fixed order
    __syncthreads();
    float* comb = smem;  // MBG * NBG * 16 * 64 floats
    for (int slice = 1; slice < KS; ++slice) {
      if (ks == slice) {
#pragma unroll
        for (int j = 0; j < NBG; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) comb[((mb * NBG + j) * 16 + v) * 64 + lane] = acc[j][v];
      }
      __syncthreads();
      if (ks == 0) {
#pragma unroll
        for (int j = 0; j < NBG; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) acc[j][v] += comb[((mb * NBG + j) * 16 + v) * 64 + lane];
      }
      __syncthreads();
    }
    if (ks == 0) {
      float* part = B.theta_part + (int64_t)gx * g.theta_cols;
      const int lr = lane >> 5, lc = lane & 31;
#pragma unroll
      for (int j = 0; j < NBG; ++j) {
        const int col = c0 + j * 32 + lc;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int f = f0 + mb * 32 + 8 * (v >> 2) + 4 * lr + (v & 3);
          if (f < g.d32 && col < r32) part[(int64_t)f * r32 + col] = acc[j][v];
        }
      }
    }
  }
  if (do_rows) {
    double* ap = B.a_part + (int64_t)gx * (4 + r32);
    const double qq = block_sum_d(acc_qq, dred + 256);
    const double yq = block_sum_d(acc_yq, dred + 256);
    if (tid == 0) {
      ap[0] = qq;
      ap[1] = yq;
      ap[2] = ap[3] = 0.0;
    }
    // s: threads sharing a column reduce in a fixed order
    __syncthreads();
    dred[tid] = acc_s;
    __syncthreads();
    if (tid < r32) {
      double t = 0.0;
      for (int k = 0; k < pstep; ++k) t += dred[tid + k * r32];
      ap[4 + tid] = FINISH ? 0.0 : t;
    }
    if (sc2 < r32) ap[4 + sc2] = FINISH ? 0.0 : acc_s2;
  }
}

// ---------------------------------------------------------------------------
// Theta = Xhat^T U of the generic pass A above 128 columns for 16-byte aligned rows
// (d % 4 == 0, r % 4 == 0): the product of k_pass_a's Theta mode (same groups, waves,
// k-slices and summation order, so the same bits) with the next tile's rows loaded
// into registers while the matrix cores work on the current one.  Per tile a thread
// holds XV + UV 16-byte pieces; loads past the last row or column read a valid
// address and are zeroed, so none waits behind a branch.  The waves whose m-block
// lies past the last feature skip the product (their partial rows are not written).
// ---------------------------------------------------------------------------
template <int MBG, int NBG>
__global__ __launch_bounds__(kThreads) void k_theta_wide(Geometry g, Bufs B) {
  if (halted(B.ctl)) return;
  constexpr int KS = 4 / MBG;
  constexpr int XS = MBG * 32 + 4;                // LDS row strides (floats)
  constexpr int US = NBG * 32 + 4;
  constexpr int XR4 = MBG * 8, UR4 = NBG * 8;     // 16-byte pieces per tile row
  constexpr int XV = kTPA * XR4 / kThreads;       // pieces per thread and tile
  constexpr int UV = kTPA * UR4 / kThreads;
  static_assert(XV * kThreads == kTPA * XR4 && UV * kThreads == kTPA * UR4, "whole pieces per thread");
  extern __shared__ __align__(16) unsigned char smem_raw[];
  float* Xs = reinterpret_cast<float*>(smem_raw);  // kTPA x XS
  float* Us = Xs + kTPA * XS;                      // kTPA x US

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int gx = blockIdx.x;
  const int gy = blockIdx.y;
  const int mg = gy / g.ngroups;
  const int ng = gy - mg * g.ngroups;
  const int64_t n = g.n;
  const int d = g.d, r = g.r, r32 = g.r32;
  const int f0 = mg * MBG * 32;
  const int c0 = ng * NBG * 32;
  const float cf = B.ctl->c_f;
  const int64_t tb = (int64_t)gx * g.tilesA / gridDim.x;
  const int64_t te = (int64_t)(gx + 1) * g.tilesA / gridDim.x;
  const int mb = wave % MBG;
  const int ks = wave / MBG;
  const bool active = f0 + mb * 32 < g.d32;

  // this thread's pieces: tile row and column offset (fixed), validity of the column
  int xo[XV], uo[UV];
  bool xk[XV], uk[UV];
#pragma unroll
  for (int i = 0; i < XV; ++i) {
    const int v = tid + i * kThreads, row = v / XR4, c = 4 * (v - row * XR4);
    xk[i] = f0 + c < d;
    xo[i] = row * d + (xk[i] ? f0 + c : 0);
  }
#pragma unroll
  for (int i = 0; i < UV; ++i) {
    const int v = tid + i * kThreads, row = v / UR4, c = 4 * (v - row * UR4);
    uk[i] = c0 + c < r;
    uo[i] = row * r + (uk[i] ? c0 + c : 0);
  }
  f32x4 xr[XV], ur[UV];
  // rows of tile t: a row past the last is read as row 0 of the tile and zeroed
  auto load = [&](int64_t tile) {
    const int64_t row0 = tile * kTPA;
    const int valid = (int)((n - row0) < kTPA ? (n - row0) : kTPA);
    const float* xb = B.X + row0 * d;
    const float* ub = B.U + row0 * r;
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int row = (tid + i * kThreads) / XR4;
      xr[i] = *reinterpret_cast<const f32x4*>(xb + (row < valid ? xo[i] : xo[i] - row * d));
    }
#pragma unroll
    for (int i = 0; i < UV; ++i) {
      const int row = (tid + i * kThreads) / UR4;
      ur[i] = *reinterpret_cast<const f32x4*>(ub + (row < valid ? uo[i] : uo[i] - row * r));
    }
  };

  f32x16 acc[NBG];
#pragma unroll
  for (int j = 0; j < NBG; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;

  if (tb < te) load(tb);
  for (int64_t tile = tb; tile < te; ++tile) {
    const int64_t row0 = tile * kTPA;
    const int valid = (int)((n - row0) < kTPA ? (n - row0) : kTPA);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int v = tid + i * kThreads, row = v / XR4, c = 4 * (v - row * XR4);
      const bool ok = xk[i] && row < valid;
      const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
      *reinterpret_cast<f32x4*>(Xs + row * XS + c) = ok ? xr[i] : zero;
    }
#pragma unroll
    for (int i = 0; i < UV; ++i) {
      const int v = tid + i * kThreads, row = v / UR4, c = 4 * (v - row * UR4);
      const bool ok = uk[i] && row < valid;
      f32x4 t = ur[i];
      t.x = ok ? t.x * cf : 0.f;
      t.y = ok ? t.y * cf : 0.f;
      t.z = ok ? t.z * cf : 0.f;
      t.w = ok ? t.w * cf : 0.f;
      *reinterpret_cast<f32x4*>(Us + row * US + c) = t;
    }
    __syncthreads();
    if (tile + 1 < te) load(tile + 1);
    if (active) {
      const int kbeg = ks * (kTPA / KS);
      const int kend = kbeg + kTPA / KS;
      const int lr = lane >> 5;
      const int lc = lane & 31;
#pragma unroll 4
      for (int k = kbeg; k < kend; k += 2) {
        const float a = Xs[(k + lr) * XS + mb * 32 + lc];
#pragma unroll
        for (int j = 0; j < NBG; ++j) {
          const float bv = Us[(k + lr) * US + j * 32 + lc];
          acc[j] = mfma32x32x2(a, bv, acc[j]);
        }
      }
    }
  }

  // combine k-slices (waves with the same m-block) in a fixed order, then write
  __syncthreads();
  float* comb = Xs;  // MBG * NBG * 16 * 64 floats
  for (int slice = 1; slice < KS; ++slice) {
    if (ks == slice) {
#pragma unroll
      for (int j = 0; j < NBG; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) comb[((mb * NBG + j) * 16 + v) * 64 + lane] = acc[j][v];
    }
    __syncthreads();
    if (ks == 0) {
#pragma unroll
      for (int j = 0; j < NBG; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[j][v] += comb[((mb * NBG + j) * 16 + v) * 64 + lane];
    }
    __syncthreads();
  }
  if (ks == 0 && active) {
    float* part = B.theta_part + (int64_t)gx * g.theta_cols;
    const int lr = lane >> 5, lc = lane & 31;
#pragma unroll
    for (int j = 0; j < NBG; ++j) {
      const int col = c0 + j * 32 + lc;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int f = f0 + mb * 32 + 8 * (v >> 2) + 4 * lr + (v & 3);
        if (f < g.d32 && col < r32) part[(int64_t)f * r32 + col] = acc[j][v];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Row work of the generic pass A above 128 columns (its first launch): no LDS
// staging; each wave streams whole rows of U, lane l holding the columns
// l + 64 j (CPL = ceil(r / 64) of them), RPI rows at a time.  Per row: u = fl(c_f w),
// q = u.p - 1 (FP64, summed over the wave by an xor butterfly, so every lane has
// the same bits), the gated dual step (eq. of the stored dual), ybar (stored for
// pass B); then s += ybar u, ||q||^2 and ytilde^T q in FP64.  Grid GAF; workgroup gx takes a
// contiguous range of rows, its waves every fourth row of it, and writes partial row
// gx in the layout of pass A (qq, yq, 0, 0, s).
// ---------------------------------------------------------------------------
template <int CPL>
__global__ __launch_bounds__(kThreads) void k_rows_wide(Geometry g, Bufs B, StepArgs S) {
  if (halted(B.ctl)) return;
  constexpr int RPI = 8;  // rows per wave and step
  __shared__ double sred[4 * 64 * CPL];
  __shared__ double dred[kThreads + 8];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t n = g.n;
  const int r = g.r;
  const float cf = B.ctl->c_f;
  const bool gate = (S.end_work != 0) && (B.ctl->gate != 0);
  const float gam = S.gamma_f;

  float pl[CPL];
  bool okc[CPL];
  int colo[CPL];  // column read (0 for the lanes past the last column)
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    const int col = lane + 64 * j;
    okc[j] = col < r;
    colo[j] = okc[j] ? col : 0;
    pl[j] = okc[j] ? B.p[col] : 0.f;
  }
  double sacc[CPL];
#pragma unroll
  for (int j = 0; j < CPL; ++j) sacc[j] = 0.0;
  double acc_qq = 0.0, acc_yq = 0.0;

  const int64_t rb = (int64_t)blockIdx.x * n / gridDim.x;
  const int64_t re = (int64_t)(blockIdx.x + 1) * n / gridDim.x;
  for (int64_t base = rb + (int64_t)wave * RPI; base < re; base += 4 * RPI) {
    float u[RPI][CPL];
    float yt[RPI];
    // every load reads a valid address (row rb, column 0 in place of those out of range)
    // and the value is dropped afterwards, so that no load sits behind a branch; all
    // loads of the step are issued before any of their values is used
#pragma unroll
    for (int i = 0; i < RPI; ++i) {
      const int64_t row = base + i;
      const float* src = B.U + (row < re ? row : rb) * r;
#pragma unroll
      for (int j = 0; j < CPL; ++j) u[i][j] = src[colo[j]];
      yt[i] = B.y[row < re ? row : rb];
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < RPI; ++i) {
      const bool okr = base + i < re;
#pragma unroll
      for (int j = 0; j < CPL; ++j) u[i][j] = (okr && okc[j]) ? u[i][j] * cf : 0.f;
      yt[i] = okr ? yt[i] : 0.f;
    }
    double dot[RPI];
#pragma unroll
    for (int i = 0; i < RPI; ++i) {
      dot[i] = 0.0;
#pragma unroll
      for (int j = 0; j < CPL; ++j) dot[i] += (double)u[i][j] * (double)pl[j];
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1)
#pragma unroll
      for (int i = 0; i < RPI; ++i) dot[i] += shfl_xor_d(dot[i], m);
#pragma unroll
    for (int i = 0; i < RPI; ++i) {
      const int64_t row = base + i;
      if (row < re) {
        const float q = (float)(dot[i] - 1.0);
        float y = yt[i];
        if (gate) {
          y = fmaf(gam, q, y);
          if (lane == 0) B.y[row] = y;
        }
        const float ybar = fmaf(gam, q, y);
        if (lane == 0) {
          B.ybar[row] = ybar;
          acc_qq += (double)q * (double)q;
          acc_yq += (double)y * (double)q;
        }
#pragma unroll
        for (int j = 0; j < CPL; ++j) sacc[j] += (double)ybar * (double)u[i][j];
      }
    }
  }

  double* ap = B.a_part + (int64_t)blockIdx.x * (4 + g.r32);
  const double qq = block_sum_d(acc_qq, dred);
  const double yq = block_sum_d(acc_yq, dred);
  if (tid == 0) {
    ap[0] = qq;
    ap[1] = yq;
    ap[2] = ap[3] = 0.0;
  }
  // s: the four waves' sums of a column, added in wave order
#pragma unroll
  for (int j = 0; j < CPL; ++j) sred[(wave * CPL + j) * 64 + lane] = sacc[j];
  __syncthreads();
  for (int c = tid; c < g.r32; c += kThreads) {
    double t = 0.0;
    if (c < 64 * CPL) {
      const int j = c >> 6, l = c & 63;
      t = ((sred[(0 * CPL + j) * 64 + l] + sred[(1 * CPL + j) * 64 + l]) + sred[(2 * CPL + j) * 64 + l]) +
          sred[(3 * CPL + j) * 64 + l];
    }
    ap[4 + c] = t;
  }
}

// ---------------------------------------------------------------------------
// Pass A, register-resident form on the 16x16x4 fp32 matrix core (all of Theta
// fits one wave: FV*NGF*CV <= 32 blocks of 16x16).  Grid GA; each wave owns a
// contiguous range of 4-row steps.  Per k-step lane l works on row 4k + l/16:
// it loads FV consecutive features for each of NGF groups (feature
// 16*FV*g + FV*(l%16) + e) and CV consecutive columns of U (column CV*(l%16) + c);
// MFMA (g, e, c) accumulates Theta[16*FV*g + FV*i + e][CV*j + c] at D[i][j].
// A row's columns live in one 16-lane DPP row, so the row work (q = u.p - 1,
// dual step, ybar, s, ||q||^2, ytilde^T q) uses a 4-step DPP butterfly whose
// result is bitwise identical in all 16 lanes.
// MODE kPassFinish: no matrix product; writes u = fl(c_f w) back (materialises U).
// MODE kPassRows: no matrix product and no write of U: the row work of the fused
// iteration, whose Theta comes from the previous pass B.
// ---------------------------------------------------------------------------
template <int FV, int NGF, int CV, int MODE>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8))) void k_pass_a_rows(
    Geometry g, Bufs B, StepArgs S) {
  constexpr bool FINISH = MODE == kPassFinish;
  constexpr bool THETA = MODE == kPassIter;
  // on breakdown the unnormalised update W already holds the factor's place
  const float* Usrc = B.U;
  if (FINISH && B.ctl->breakdown != 0) return;
  if (!FINISH && halted(B.ctl)) return;
  // the one-pass iteration launches the row pass every iteration; it runs only when
  // the previous iteration's stopping rule may fire (the pass then does no row work)
  if (MODE == kPassRows && g.fused8 && !B.ctl->rows_first) return;
  const bool stopped = FINISH && (B.ctl->stop != 0);
  constexpr int NBLK = FV * NGF * CV;  // 16x16 blocks of Theta
  // k-steps in flight: fewer when Theta takes 128 registers, more when only U and y stream
  constexpr int PF = THETA ? (NBLK >= 32 ? 2 : 4) : 8;
  __shared__ double dred[kThreads + 8];
  __shared__ float comb[THETA ? 2 * NBLK * 4 * 64 : 4];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int grp = lane >> 4;   // row within the k-step
  const int li = lane & 15;    // lane within the DPP row
  const int64_t n = g.n;
  const int d = g.d, r = g.r;
  const float cf = B.ctl->c_f;
  const bool gate = (S.end_work != 0) && (B.ctl->gate != 0) && !stopped;
  const float gam = S.gamma_f;

  float pl[CV];
#pragma unroll
  for (int c = 0; c < CV; ++c) {
    const int col = CV * li + c;
    pl[c] = (col < r) ? B.p[col] : 0.f;
  }

  // 4-row steps of this wave
  const int64_t steps = (n + 3) >> 2;
  const int64_t wid = (int64_t)blockIdx.x * 4 + wave;
  const int64_t nw = (int64_t)g.GA * 4;
  const int64_t k0 = wid * steps / nw;
  const int64_t k1 = (wid + 1) * steps / nw;

  f32x4v acc[NBLK];
  if (THETA) {
#pragma unroll
    for (int b = 0; b < NBLK; ++b) acc[b] = (f32x4v){0.f, 0.f, 0.f, 0.f};
  }
  double s_acc[CV];
#pragma unroll
  for (int c = 0; c < CV; ++c) s_acc[c] = 0.0;
  double qq = 0.0, yq = 0.0;

  float xr[PF][NGF][FV];
  float ur[PF][CV];
  float yr[PF];
  // The ring holds raw loads; masks and the lazy scale are applied where the
  // values are used, so that no instruction waits on a load right after issuing it.
  bool fx[NGF];
#pragma unroll
  for (int gg = 0; gg < NGF; ++gg) fx[gg] = (16 * FV * gg + FV * li) < d;
  const int cu = CV * li;
  const bool cx = cu < r;
  auto issue = [&](int slot, int64_t k) {
    const int64_t row = 4 * k + grp;
    const bool ok = (k < k1) && (row < n);
    const int64_t rr = ok ? row : 0;
    if (THETA) {
#pragma unroll
      for (int gg = 0; gg < NGF; ++gg) {
        const int f = 16 * FV * gg + FV * li;
        load_vec<FV>(xr[slot][gg], B.X + rr * d + (f < d ? f : 0), true);
      }
    }
    load_vec<CV>(ur[slot], Usrc + rr * r + (cx ? cu : 0), true);
    yr[slot] = B.y[rr];
  };
#pragma unroll
  for (int i = 0; i < PF; ++i) {
    __builtin_amdgcn_sched_barrier(0);
    issue(i, k0 + i);
  }
  __builtin_amdgcn_sched_barrier(0);

  for (int64_t kb = k0; kb < k1; kb += PF) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      // keep consumption of slot i and the refill of slot i in program order, so
      // that the loads of the other slots stay in flight
      __builtin_amdgcn_sched_barrier(0);
      const int64_t k = kb + i;
      const int64_t row = 4 * k + grp;
      const bool valid = (k < k1) && (row < n);
      float u[CV];
#pragma unroll
      for (int c = 0; c < CV; ++c) u[c] = (valid && cx) ? ur[i][c] * cf : 0.f;
      if (THETA) {
#pragma unroll
        for (int gg = 0; gg < NGF; ++gg)
#pragma unroll
          for (int e = 0; e < FV; ++e) {
            const float x = fx[gg] ? xr[i][gg][e] : 0.f;
#pragma unroll
            for (int c = 0; c < CV; ++c)
              acc[(gg * FV + e) * CV + c] = mfma16x16x4(x, u[c], acc[(gg * FV + e) * CV + c]);
          }
      }
      // q = u.p - 1 over the 16 lanes of this row (FP64)
      double dot = 0.0;
#pragma unroll
      for (int c = 0; c < CV; ++c) dot += (double)u[c] * (double)pl[c];
      dot = row16_sum_d(dot);
      const float q = (float)(dot - 1.0);
      float yt = valid ? yr[i] : 0.f;
      if (gate) yt = fmaf(gam, q, yt);
      const float ybar = fmaf(gam, q, yt);
      // branch-free: invalid rows have u = 0; stores of invalid lanes go to the dump slot
      if (gate) *(valid ? (B.y + row) : B.dump) = yt;  // the 16 lanes of a row store the same value
#pragma unroll
      for (int c = 0; c < CV; ++c) s_acc[c] += (double)ybar * (double)u[c];
      const bool lead = valid && li == 0;
      qq += lead ? (double)q * (double)q : 0.0;
      yq += lead ? (double)yt * (double)q : 0.0;
      if (FINISH) {
        float* dst = (valid && cx) ? (B.U + row * r + cu) : B.dump;
        if constexpr (CV == 4) {
          f32x4 o = {u[0], u[1], u[2], u[3]};
          *reinterpret_cast<f32x4*>(dst) = o;
        } else if constexpr (CV == 2) {
          typedef float f32x2 __attribute__((ext_vector_type(2)));
          f32x2 o = {u[0], u[1]};
          *reinterpret_cast<f32x2*>(dst) = o;
        } else {
          dst[0] = u[0];
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      issue(i, k + PF);
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- partials ----
  if (THETA) {
    // Theta: ((wave0 + wave2) + (wave1 + wave3)) through two LDS regions
    constexpr int REG = NBLK * 4 * 64;
    if (wave < 2) {
      float* dst = comb + wave * REG;
#pragma unroll
      for (int b = 0; b < NBLK; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) dst[(b * 4 + v) * 64 + lane] = acc[b][v];
    }
    __syncthreads();
    if (wave >= 2) {
      float* dst = comb + (wave - 2) * REG;
#pragma unroll
      for (int b = 0; b < NBLK; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int idx = (b * 4 + v) * 64 + lane;
          dst[idx] = dst[idx] + acc[b][v];
        }
    }
    __syncthreads();
    float* part = B.theta_part + (int64_t)blockIdx.x * g.theta_cols;
    const int tot = g.d32 * g.r32;
    for (int e = tid; e < tot; e += kThreads) {
      const int f = e / g.r32, col = e - (e / g.r32) * g.r32;
      const int gg = f / (16 * FV), rem = f - gg * 16 * FV;
      const int i = rem / FV, ef = rem - i * FV;
      const int c = col % CV, j = col / CV;
      float val = 0.f;
      if (gg < NGF && j < 16) {
        const int idx = (((gg * FV + ef) * CV + c) * 4 + (i & 3)) * 64 + 16 * (i >> 2) + j;
        val = comb[idx] + comb[REG + idx];
      }
      part[e] = val;
    }
  }
  // s: rows 0..3 of a k-step hold the same columns; waves hold disjoint rows
  __syncthreads();
#pragma unroll
  for (int c = 0; c < CV; ++c) {
    double v = s_acc[c] + shfl_xor_d(s_acc[c], 16);
    v = v + shfl_xor_d(v, 32);
    if (grp == 0) dred[wave * 16 * CV + CV * li + c] = v;  // 4 * 16 * CV <= 256
  }
  __syncthreads();
  double* ap = B.a_part + (int64_t)blockIdx.x * (4 + g.r32);
  for (int c = tid; c < g.r32; c += kThreads) {
    double t = 0.0;
    if (c < 16 * CV)
      t = ((dred[c] + dred[16 * CV + c]) + dred[32 * CV + c]) + dred[48 * CV + c];
    ap[4 + c] = FINISH ? 0.0 : t;
  }
  const double tq = block_sum_d(qq, dred + kThreads);
  const double ty = block_sum_d(yq, dred + kThreads);
  if (tid == 0) {
    ap[0] = tq;
    ap[1] = ty;
    ap[2] = ap[3] = 0.0;
  }
}

// ---------------------------------------------------------------------------
// Row pass and finish pass of the single-Xhat-pass form for narrow factors (r <= 16,
// r even): eight lanes per row (two columns each, 8-byte loads) and eight rows per
// wave and step, so that the per-row work (the FP64 dot and its butterfly, q, the
// dual step, ybar and the FP64 statistics) is not repeated over 16 lanes for a few
// columns.  The row dot sums over the 8 lanes of a DPP half row (row8_sum_d); both
// modes use it, so q, ytilde and ybar agree bitwise whichever of them does the row
// work (nlr_run(T) equals T nlr_step).  Outputs as k_pass_a_rows.
// ---------------------------------------------------------------------------
template <int MODE>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8))) void k_rows_narrow(
    Geometry g, Bufs B, StepArgs S) {
  constexpr bool FINISH = MODE == kPassFinish;
  static_assert(MODE == kPassFinish || MODE == kPassRows, "row work only");
  const float* Usrc = B.U;
  if (FINISH && B.ctl->breakdown != 0) return;
  if (!FINISH && halted(B.ctl)) return;
  // the one-pass iteration launches the row pass every iteration; it runs only when
  // the previous iteration's stopping rule may fire (the pass then does no row work)
  if (MODE == kPassRows && g.fused8 && !B.ctl->rows_first) return;
  const bool stopped = FINISH && (B.ctl->stop != 0);
  constexpr int PF = 8;  // steps in flight (16 halves the waves per SIMD: no more bytes in flight)
  __shared__ double dred[kThreads + 8];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int grp = lane >> 3;  // row within the step
  const int li = lane & 7;    // lane within the row
  const int64_t n = g.n;
  const int r = g.r;
  const float cf = B.ctl->c_f;
  const bool gate = (S.end_work != 0) && (B.ctl->gate != 0) && !stopped;
  const float gam = S.gamma_f;
  const int cu = 2 * li;
  const bool cx = cu < r;  // r even: both columns of the lane are valid, or neither
  const float pl[2] = {cx ? B.p[cu] : 0.f, cx ? B.p[cu + 1] : 0.f};

  const int64_t steps = (n + 7) >> 3;
  const int64_t wid = (int64_t)blockIdx.x * 4 + wave;
  const int64_t nw = (int64_t)g.GA * 4;
  const int64_t k0 = wid * steps / nw;
  const int64_t k1 = (wid + 1) * steps / nw;

  double s_acc[2] = {0.0, 0.0};
  double qq = 0.0, yq = 0.0;
  float ur[PF][2];
  float yr[PF];
  auto issue = [&](int slot, int64_t k) {
    const int64_t row = 8 * k + grp;
    const bool ok = (k < k1) && (row < n);
    const int64_t rr = ok ? row : 0;
    load_vec<2>(ur[slot], Usrc + rr * r + (cx ? cu : 0), true);
    yr[slot] = B.y[rr];
  };
#pragma unroll
  for (int i = 0; i < PF; ++i) {
    __builtin_amdgcn_sched_barrier(0);
    issue(i, k0 + i);
  }
  __builtin_amdgcn_sched_barrier(0);

  for (int64_t kb = k0; kb < k1; kb += PF) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      __builtin_amdgcn_sched_barrier(0);
      const int64_t k = kb + i;
      const int64_t row = 8 * k + grp;
      const bool valid = (k < k1) && (row < n);
      float u[2];
#pragma unroll
      for (int c = 0; c < 2; ++c) u[c] = (valid && cx) ? ur[i][c] * cf : 0.f;
      double dot = 0.0;
#pragma unroll
      for (int c = 0; c < 2; ++c) dot += (double)u[c] * (double)pl[c];
      dot = row8_sum_d(dot);
      const float q = (float)(dot - 1.0);
      float yt = valid ? yr[i] : 0.f;
      if (gate) yt = fmaf(gam, q, yt);
      const float ybar = fmaf(gam, q, yt);
      if (gate) *(valid ? (B.y + row) : B.dump) = yt;  // the 8 lanes of a row store the same value
#pragma unroll
      for (int c = 0; c < 2; ++c) s_acc[c] += (double)ybar * (double)u[c];
      const bool lead = valid && li == 0;
      qq += lead ? (double)q * (double)q : 0.0;
      yq += lead ? (double)yt * (double)q : 0.0;
      if (FINISH) {
        typedef float f32x2 __attribute__((ext_vector_type(2)));
        float* dst = (valid && cx) ? (B.U + row * r + cu) : B.dump;
        *reinterpret_cast<f32x2*>(dst) = (f32x2){u[0], u[1]};
      }
      __builtin_amdgcn_sched_barrier(0);
      issue(i, k + PF);
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // s: the eight rows of a step hold the same columns; waves hold disjoint rows
  __syncthreads();
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    double v = s_acc[c] + shfl_xor_d(s_acc[c], 8);
    v = v + shfl_xor_d(v, 16);
    v = v + shfl_xor_d(v, 32);
    if (grp == 0) dred[wave * 16 + cu + c] = v;
  }
  __syncthreads();
  double* ap = B.a_part + (int64_t)blockIdx.x * (4 + g.r32);
  for (int c = tid; c < g.r32; c += kThreads) {
    double t = 0.0;
    if (c < 16) t = ((dred[c] + dred[16 + c]) + dred[32 + c]) + dred[48 + c];
    ap[4 + c] = FINISH ? 0.0 : t;
  }
  const double tq = block_sum_d(qq, dred + kThreads);
  const double ty = block_sum_d(yq, dred + kThreads);
  if (tid == 0) {
    ap[0] = tq;
    ap[1] = ty;
    ap[2] = ap[3] = 0.0;
  }
}

// ---------------------------------------------------------------------------
// Segmented column sums, fixed order: out[s][c] = sum over rows of segment s of
// P[row][c] (rows [s R/S, (s+1) R/S)).  Grid (ceil(C/64), S); thread (col, sub)
// sums rows sub, sub+4, ... of the segment, then the four subs are added in order.
// ---------------------------------------------------------------------------
// sum over s < S of p[s * stride] in the order s = 0, 1, ...: the loads of eight terms
// are issued before their additions (a clamped index, so that no load waits behind a
// branch), which keeps the small reduction kernels from waiting on one load at a time
template <typename T>
__device__ __forceinline__ double seq_sum(const T* __restrict__ p, int64_t stride, int64_t S) {
  double acc = 0.0;
  for (int64_t s0 = 0; s0 < S; s0 += 8) {
    double v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (double)p[(s0 + i < S ? s0 + i : S - 1) * stride];
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (s0 + i < S) acc += v[i];
  }
  return acc;
}

template <typename T>
__device__ __forceinline__ void seg_sum_block(const T* __restrict__ P, int64_t R, int C, double* __restrict__ out,
                                              int S, int bx, int by, double* red) {
  const int tid = threadIdx.x;
  const int col = bx * 64 + (tid & 63);
  const int sub = tid >> 6;
  const int64_t lo = (int64_t)by * R / S;
  const int64_t hi = (int64_t)(by + 1) * R / S;
  double acc = 0.0;
  if (col < C && lo + sub < hi) acc = seq_sum<T>(P + (lo + sub) * C + col, 4 * (int64_t)C, (hi - lo - sub + 3) / 4);
  red[tid] = acc;
  __syncthreads();
  if (tid < 64 && col < C)
    out[(int64_t)by * C + col] = ((red[tid] + red[64 + tid]) + red[128 + tid]) + red[192 + tid];
}

// mode 0: run unless broken down (after the finish pass); 1: unless halted; 2: unless
// halted or the one-pass iteration's row pass did not run (rows_first unset)
template <typename T>
__global__ __launch_bounds__(kThreads) void k_seg_sum(const T* __restrict__ P, int64_t R, int C,
                                                      double* __restrict__ out, int S, const DevCtl* ctl,
                                                      int mode) {
  if (mode == 0 ? (ctl->breakdown != 0) : halted(ctl)) return;
  if (mode == 2 && !ctl->rows_first) return;
  __shared__ double red[kThreads];
  seg_sum_block<T>(P, R, C, out, S, blockIdx.x, blockIdx.y, red);
}

// ---------------------------------------------------------------------------
// Theta = sum of the segment sums (fixed order, FP64), written in the pass-B
// operand layout, plus per-workgroup ||Theta||_F^2 partials.
// Layout: chunk ch of 32 features, quarter j (4 features), m-block mb, lane l,
// element e  <->  Theta[32 ch + 16 (l/32) + 4 j + e][32 mb + l%32].
// ---------------------------------------------------------------------------
__device__ __forceinline__ float s_from_gram(const Bufs& B, int r32, int k, double gp, float gamma_f);

// gamma_f >= 0 (one-pass iteration): the extra blocks also form s for the next pass.
__global__ __launch_bounds__(kThreads) void k_reduce_theta(Geometry g, Bufs B, int nseg, int scaled, float gamma_f) {
  if (halted(B.ctl)) return;
  __shared__ double red[kThreads];
  __shared__ float mred[4];
  if (blockIdx.x >= g.RT) {
    // one-pass iteration: the W^T W columns of the partial rows, times P (the column
    // sums of W, already reduced): (W^T W P)_k, each row's products added in a tree
    const int r32 = g.r32;
    const int e = (blockIdx.x - g.RT) * kThreads + threadIdx.x;  // entry k r32 + l
    const int k = e / r32, l = e - k * r32;
    const double G = seq_sum<double>(B.seg_theta + (int64_t)g.d32 * r32 + e, g.theta_cols, nseg);
    red[threadIdx.x] = G * B.gram_vec[l];
    __syncthreads();
    for (int w = r32 >> 1; w >= 1; w >>= 1) {
      if (l < w) red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + w];
      __syncthreads();
    }
    if (l == 0) {
      const double gp = red[threadIdx.x];
      B.gram_vec[2 * r32 + k] = gp;
      if (gamma_f >= 0.f) {
        const float sk = s_from_gram(B, r32, k, gp, gamma_f);
        B.s[k] = (k < g.r) ? sk : 0.f;
      }
    }
    return;
  }
  const int64_t tot = (int64_t)g.d32 * g.r32;
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  double sum = 0.0;
  if (e < tot) {
    sum = seq_sum<double>(B.seg_theta + e, g.theta_cols, nseg);
    const int f = (int)(e / g.r32);
    // partials of Xhat^T W (fused pass B) carry the scale c of U = c W
    if (scaled) sum *= (double)B.ctl->c_f;
    if (f >= g.d) sum = 0.0;  // padded features: zero rows of Theta
    const int c = (int)(e - (int64_t)f * g.r32);
    const int ch = f >> 5, fin = f & 31;
    const int hh = fin >> 4, j = (fin & 15) >> 2, ee = fin & 3;
    const int mbk = c >> 5, l = hh * 32 + (c & 31);
    const int64_t idx = ((((int64_t)ch * 4 + j) * g.NB + mbk) * 64 + l) * 4 + ee;
    B.theta[idx] = (float)sum;
  }
  const double t2 = block_sum_d(sum * sum, red);
  if (threadIdx.x == 0) B.th2_part[blockIdx.x] = t2;
  // max |Theta| of the block (the panel form scales its split Theta operand by it)
  float m = fabsf((float)sum);
  for (int k = 32; k >= 1; k >>= 1) m = fmaxf(m, shfl_xor_f(m, k));
  if ((threadIdx.x & 63) == 0) mred[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) B.thmax_part[blockIdx.x] = fmaxf(fmaxf(mred[0], mred[1]), fmaxf(mred[2], mred[3]));
}

// ---------------------------------------------------------------------------
// Control after pass A (one workgroup): s, rho, objective, stopping rule of the
// previous iteration.  finish = the call after the finish pass.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_ctl_a(Geometry g, Bufs B, StepArgs S, int finish) {
  DevCtl* ctl = B.ctl;
  if (ctl->breakdown) return;
  if (ctl->stop) {
    // stopped earlier in this call: the finish pass only materialised U
    if (finish && threadIdx.x == 0) ctl->c_f = 1.0f;
    return;
  }
  // one-pass iteration: after its row pass only (which runs when the stop may fire)
  if (g.fused8 && !finish && !ctl->rows_first) return;
  __shared__ double red[8];
  const int tid = threadIdx.x;
  const int C = 4 + g.r32;
  // (one-pass iteration with valid Gram terms, rows_first == 1: s is the Gram-derived
  // one already in place, as when the pass does the row work itself)
  if (!finish && !(g.fused8 && ctl->rows_first == 1)) {
    for (int c = tid; c < g.r32; c += kThreads) {
      const double t = seq_sum<double>(B.seg_a + 4 + c, C, g.SA);
      B.s[c] = (c < g.r) ? (float)t : 0.f;
    }
  }
  // ||q||^2 and ytilde^T q summed by two threads at the same time (past those of s)
  __shared__ double qy[2];
  const int tq = g.r32 + 2 <= kThreads ? g.r32 : 0;
  if (tid == tq || tid == tq + 1) qy[tid - tq] = seq_sum<double>(B.seg_a + (tid - tq), C, g.SA);
  double th2 = 0.0;
  if (!finish)
    for (int k = tid; k < g.RT; k += kThreads) th2 += B.th2_part[k];
  th2 = block_sum_d(th2, red);  // (its barriers also publish qy)
  if (tid == 0) {
    const double qq = qy[0], yq = qy[1];
    const double rho = sqrt(qq * S.inv_n);
    ctl->rho = rho;
    const int64_t t = ctl->t_done;
    if (S.end_work && t > 0) {
      nlr_iter_stats* prev = &B.hist[(t - 1) % kHistCap];
      const int stop = (ctl->Delta < S.eps_d * S.eps_d * S.K) && (ctl->delta < S.eps_c) &&
                       (rho < S.eps_c) && (t >= S.T_min);
      prev->rho = rho;
      prev->stop = stop;
      if (stop) ctl->stop = 1;
    }
    if (!finish && !ctl->stop) {
      const double obj = -th2 + yq + 0.5 * S.beta * S.inv_n * qq;
      ctl->objective = obj;
      ctl->theta_fro2 = th2;
      nlr_iter_stats* cur = &B.hist[t % kHistCap];
      cur->t = t;
      cur->objective = obj;
      cur->theta_fro2 = th2;
      cur->a = cur->b = cur->h = cur->delta = 0.0;
      cur->rho = 0.0;
      cur->c = 0.f;
      cur->dual_step = 0;
      cur->stop = 0;
      cur->breakdown = 0;
    }
    if (finish) ctl->c_f = 1.0f;
    if (g.fused8 && !finish) ctl->rows_run += 1;
  }
}

// ---------------------------------------------------------------------------
// Pass B.  Grid GB, persistent over 128-row super-tiles; wave w computes rows
// [32w, 32w+32) of each super-tile for all r32 columns:
//   acc (D layout) = Theta^T (A operand, from LDS or global) x Xhat^T (B operand,
//   lane l loads row l%32, features 32ch + 16 (l/32) + [0, 16)).
// Epilogue per element: w = max(u + 2 alpha acc - alpha ybar p - alpha s, 0).
// ---------------------------------------------------------------------------
template <int NB, bool THETA_LDS, bool VEC>
__global__ __launch_bounds__(kThreads) void k_pass_b(Geometry g, Bufs B, StepArgs S) {
  if (halted(B.ctl)) return;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  float* th_s = reinterpret_cast<float*>(smem_raw);                 // d32*r32 if THETA_LDS
  float* ps = th_s + (THETA_LDS ? g.d32 * g.r32 : 0);               // r32
  float* ss = ps + g.r32;                                           // r32
  double* colred = reinterpret_cast<double*>(ss + g.r32);          // 4 x r32
  double* dred = colred + 4 * g.r32;                                // 8

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5;
  const int li = lane & 31;
  const int64_t n = g.n;
  const int d = g.d, r = g.r, r32 = g.r32;
  const int nch = g.nch;
  const float cf = B.ctl->c_f;
  const float gam = S.gamma_f;
  const float two_alpha = S.two_alpha_f;
  const float neg_alpha = -S.alpha_f;

  if (THETA_LDS) {
    const int tot4 = (g.d32 * r32) >> 2;
    const f32x4* src = reinterpret_cast<const f32x4*>(B.theta);
    f32x4* dst = reinterpret_cast<f32x4*>(th_s);
    for (int v = tid; v < tot4; v += kThreads) dst[v] = src[v];
  }
  for (int c = tid; c < r32; c += kThreads) {
    ps[c] = B.p[c];
    ss[c] = B.s[c];
  }
  __syncthreads();
  const float* theta = THETA_LDS ? th_s : B.theta;

  double sa = 0.0, sb = 0.0, sh = 0.0;
  // column sums: per 32-column block, a 16-value reduce-scatter over lane bits
  // 16, 8, 4, 2 leaves one value per lane; lanes l and l^1 then share a column
  double colacc[NB];
#pragma unroll
  for (int m = 0; m < NB; ++m) colacc[m] = 0.0;
  int base = 0;  // local index (8 qd + e ordering) of the value this lane keeps
  {
    if (li & 16) base += 8;
    if (li & 8) base += 4;
    if (li & 4) base += 2;
    if (li & 2) base += 1;
  }

  const int64_t sb0 = (int64_t)blockIdx.x * g.tilesB / g.GB;
  const int64_t sb1 = (int64_t)(blockIdx.x + 1) * g.tilesB / g.GB;
  for (int64_t st = sb0; st < sb1; ++st) {
    const int64_t pt = st * kTPB + wave * 32 + li;
    const bool vpt = pt < n;
    f32x16 acc[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;

    const float* xrow = B.X + (vpt ? pt : 0) * (int64_t)d;
    for (int ch = 0; ch < nch; ++ch) {
      const int fb = ch * 32 + h * 16;
      float xv[16];
      if (VEC) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          f32x4 t = {0.f, 0.f, 0.f, 0.f};
          if (vpt && fb + 4 * q < d) t = *reinterpret_cast<const f32x4*>(xrow + fb + 4 * q);
          xv[4 * q + 0] = t.x;
          xv[4 * q + 1] = t.y;
          xv[4 * q + 2] = t.z;
          xv[4 * q + 3] = t.w;
        }
      } else {
#pragma unroll
        for (int q = 0; q < 16; ++q) xv[q] = (vpt && fb + q < d) ? xrow[fb + q] : 0.f;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int m = 0; m < NB; ++m) {
          const f32x4 a = *reinterpret_cast<const f32x4*>(theta + ((((int64_t)ch * 4 + j) * NB + m) * 64 + lane) * 4);
          acc[m] = mfma32x32x2(a.x, xv[4 * j + 0], acc[m]);
          acc[m] = mfma32x32x2(a.y, xv[4 * j + 1], acc[m]);
          acc[m] = mfma32x32x2(a.z, xv[4 * j + 2], acc[m]);
          acc[m] = mfma32x32x2(a.w, xv[4 * j + 3], acc[m]);
        }
      }
    }

    // ---- epilogue ----
    // lane holds row pt and columns 32 m + 8 qd + 4 h + e (m < NB, qd < 4, e < 4)
    // (the opaque copy keeps the p/s reads inside the tile loop instead of
    // hoisting 2*16*NB loop-invariant registers out of it)
    int lds_off = 0;  // opaque zero offset: keeps the reads in LDS address space
    asm volatile("" : "+v"(lds_off));
    const float* psl = ps + lds_off;
    const float* ssl = ss + lds_off;
    float* urow = B.U + (vpt ? pt : 0) * (int64_t)r;
    auto load_u4 = [&](int c, float out[4]) {
      if (VEC) {
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
        if (vpt && c < r) t = *reinterpret_cast<const f32x4*>(urow + c);
        out[0] = t.x * cf;
        out[1] = t.y * cf;
        out[2] = t.z * cf;
        out[3] = t.w * cf;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = (vpt && c + e < r) ? urow[c + e] * cf : 0.f;
      }
    };
    // q = u.p - 1 (fp32 dot over the lane's half of the row, then the other half)
    float dotf = 0.f;
#pragma unroll
    for (int m = 0; m < NB; ++m)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int c = 32 * m + 8 * qd + 4 * h;
        float u4[4];
        load_u4(c, u4);
        const f32x4 pv = *reinterpret_cast<const f32x4*>(psl + c);
        dotf = fmaf(u4[0], pv.x, dotf);
        dotf = fmaf(u4[1], pv.y, dotf);
        dotf = fmaf(u4[2], pv.z, dotf);
        dotf = fmaf(u4[3], pv.w, dotf);
      }
    dotf += shfl_xor_f(dotf, 32);
    float ybar = 0.f;
    if (vpt) ybar = fmaf(gam, dotf - 1.0f, B.y[pt]);
#pragma unroll
    for (int m = 0; m < NB; ++m) {
      float wv[16];
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int c = 32 * m + 8 * qd + 4 * h;
        float u4[4];
        load_u4(c, u4);
        const f32x4 pv = *reinterpret_cast<const f32x4*>(psl + c);
        const f32x4 sv = *reinterpret_cast<const f32x4*>(ssl + c);
        const float pe[4] = {pv.x, pv.y, pv.z, pv.w};
        const float se[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float uu = u4[e];
          float t = fmaf(two_alpha, acc[m][4 * qd + e], uu);
          t = fmaf(neg_alpha, ybar * pe[e], t);
          t = fmaf(neg_alpha, se[e], t);
          float w = fmaxf(t, 0.f);
          if (!vpt || c + e >= r) w = 0.f;
          wv[4 * qd + e] = w;
          const double wd = (double)w, ud = (double)uu;
          sa = fma(wd, wd, sa);
          sb = fma(ud, ud, sb);
          sh = fma(wd, ud, sh);
        }
        if (vpt) {
          if (VEC) {
            if (c < r) {
              f32x4 o = {wv[4 * qd + 0], wv[4 * qd + 1], wv[4 * qd + 2], wv[4 * qd + 3]};
              *reinterpret_cast<f32x4*>(urow + c) = o;
            }
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (c + e < r) urow[c + e] = wv[4 * qd + e];
          }
        }
      }
      reduce_scatter<16, 16>(wv, li);
      colacc[m] += (double)wv[0];
    }
  }

  // ---- workgroup partials ----
  for (int c = tid; c < 4 * r32; c += kThreads) colred[c] = 0.0;
  __syncthreads();
#pragma unroll
  for (int m = 0; m < NB; ++m) {
    const double v = colacc[m] + shfl_xor_d(colacc[m], 1);
    if ((li & 1) == 0) {
      const int col = 32 * m + 8 * (base >> 2) + 4 * h + (base & 3);
      colred[wave * r32 + col] = v;
    }
  }
  __syncthreads();
  double* out = B.b_part + (int64_t)blockIdx.x * (4 + r32);
  for (int c = tid; c < r32; c += kThreads)
    out[4 + c] = ((colred[c] + colred[r32 + c]) + colred[2 * r32 + c]) + colred[3 * r32 + c];
  const double ta = block_sum_d(sa, dred);
  const double tb2 = block_sum_d(sb, dred);
  const double th = block_sum_d(sh, dred);
  if (tid == 0) {
    out[0] = ta;
    out[1] = tb2;
    out[2] = th;
    out[3] = 0.0;
  }
}

// ---------------------------------------------------------------------------
// Pass B with Theta streamed through LDS, for a Theta that does not fit pass B's 64 KiB
// of LDS beside p, s and the reductions, and 16-byte rows.  As k_pass_b (waves, rows, the operand
// layout of Theta and the k-order of the products), with the columns in groups of
// CG blocks (the last group may be short): per 128-row super-tile, for each group
// and each 32-feature chunk, the workgroup stages the chunk's Theta operands (4 KiB
// per block) in one of two LDS buffers and every wave multiplies its rows by them.
// The next chunk's Theta operands and Xhat features are loaded into registers while
// the matrix cores work on the current one (one barrier per chunk); during a group's
// last chunk the rows of U its epilogue needs are loaded instead, and the next
// group's first chunk during the epilogue.  Loads past the last row, feature, block
// or column read a valid address and are zeroed or unused, so that no load waits
// behind a branch.  Above 128 columns ybar comes from the row launch of pass A
// (which stores it), else from q = u.p - 1 formed here.  Column sums: lanes l and
// l ^ 1 combined, then added to the wave's row of an LDS table per super-tile.
// ---------------------------------------------------------------------------
template <int CG>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8))) void k_pass_b_stream(
    Geometry g, Bufs B, StepArgs S) {
  if (halted(B.ctl)) return;
  constexpr int TCF = 4 * CG * 256;  // floats of a chunk's Theta operands
  extern __shared__ __align__(16) unsigned char smem_raw[];
  float* tbuf = reinterpret_cast<float*>(smem_raw);           // 2 x TCF
  double* colred = reinterpret_cast<double*>(tbuf + 2 * TCF);  // 4 x r32
  float* ps = reinterpret_cast<float*>(colred + 4 * g.r32);    // r32
  float* ss = ps + g.r32;                                      // r32
  double* dred = reinterpret_cast<double*>(ss + g.r32);       // 4

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5;
  const int li = lane & 31;
  const int64_t n = g.n;
  const int d = g.d, r = g.r, r32 = g.r32, NB = g.NB;
  const int nch = g.nch;
  const int ngr = (NB + CG - 1) / CG;  // column groups
  const bool ystored = pass_a_split(g);  // the row launch of pass A stored ybar
  const float cf = B.ctl->c_f;
  const float gam = S.gamma_f;
  const float two_alpha = S.two_alpha_f;
  const float neg_alpha = -S.alpha_f;

  for (int c = tid; c < r32; c += kThreads) {
    ps[c] = B.p[c];
    ss[c] = B.s[c];
  }
  for (int c = tid; c < 4 * r32; c += kThreads) colred[c] = 0.0;
  __syncthreads();  // p and s are read before the first chunk's barrier (q below 129 columns)

  double sa = 0.0, sb = 0.0, sh = 0.0;
  int base = 0;  // local index (8 qd + e ordering) of the column sum this lane keeps
  if (li & 16) base += 8;
  if (li & 8) base += 4;
  if (li & 4) base += 2;
  if (li & 2) base += 1;

  const int64_t sb0 = (int64_t)blockIdx.x * g.tilesB / g.GB;
  const int64_t sb1 = (int64_t)(blockIdx.x + 1) * g.tilesB / g.GB;

  // Theta operands of chunk (group cgi, chunk ch): piece v = tid + 256 i of the chunk is
  // j = v / (64 CG), block m = v / 64 % CG (clamped to the last block), lane v % 64
  int tj[CG], tm[CG];
#pragma unroll
  for (int i = 0; i < CG; ++i) {
    const int v = tid + kThreads * i;
    tj[i] = v / (64 * CG);
    tm[i] = (v / 64) % CG;
  }
  f32x4 tr[CG];
  f32x4 xr[4];
  auto load_chunk = [&](int64_t st, int cgi, int ch) {
    // (an opaque zero keeps the address arithmetic here, not hoisted out of the loops
    // into registers that would stay live across them)
    int z = 0;
    asm volatile("" : "+v"(z));
#pragma unroll
    for (int i = 0; i < CG; ++i) {
      const int mb = cgi * CG + tm[i] < NB ? cgi * CG + tm[i] : NB - 1;
      const int64_t piece = (((int64_t)ch * 4 + tj[i]) * NB + mb) * 64 + ((tid + z) & 63);
      tr[i] = *reinterpret_cast<const f32x4*>(B.theta + piece * 4);
    }
    const int64_t pt = st * kTPB + wave * 32 + li + z;
    const float* xrow = B.X + (pt < n ? pt : 0) * (int64_t)d;
    const int fb = ch * 32 + h * 16;
#pragma unroll
    for (int q = 0; q < 4; ++q) xr[q] = *reinterpret_cast<const f32x4*>(xrow + (fb + 4 * q < d ? fb + 4 * q : 0));
  };

  if (sb0 < sb1) load_chunk(sb0, 0, 0);
  int kbuf = 0;
  for (int64_t st = sb0; st < sb1; ++st) {
    const int64_t pt = st * kTPB + wave * 32 + li;
    const bool vpt = pt < n;
    float* urow = B.U + (vpt ? pt : 0) * (int64_t)r;
    // (the opaque copy keeps the p/s reads inside the tile loop instead of hoisting
    // loop-invariant registers out of it)
    int lds_off = 0;
    asm volatile("" : "+v"(lds_off));
    const float* psl = ps + lds_off;
    const float* ssl = ss + lds_off;
    float ybar;
    if (ystored) {
      // ybar of the row pass of this iteration (q from an FP64 dot)
      const float yb = B.ybar[vpt ? pt : 0];
      ybar = vpt ? yb : 0.f;
    } else {
      // q = u.p - 1 over the whole row (fp32 dot over the lane's half, then the other half)
      float dotf = 0.f;
      for (int m = 0; m < NB; ++m)
#pragma unroll
        for (int qd = 0; qd < 4; ++qd) {
          const int c = 32 * m + 8 * qd + 4 * h;
          const f32x4 t = *reinterpret_cast<const f32x4*>(urow + (c < r ? c : 0));
          const bool ok = vpt && c < r;
          const f32x4 pv = *reinterpret_cast<const f32x4*>(psl + c);
          dotf = fmaf(ok ? t.x * cf : 0.f, pv.x, dotf);
          dotf = fmaf(ok ? t.y * cf : 0.f, pv.y, dotf);
          dotf = fmaf(ok ? t.z * cf : 0.f, pv.z, dotf);
          dotf = fmaf(ok ? t.w * cf : 0.f, pv.w, dotf);
        }
      dotf += shfl_xor_f(dotf, 32);
      const float yv = B.y[vpt ? pt : 0];
      ybar = vpt ? fmaf(gam, dotf - 1.0f, yv) : 0.f;
    }

    for (int cgi = 0; cgi < ngr; ++cgi) {
      const int nbg = NB - cgi * CG < CG ? NB - cgi * CG : CG;  // blocks of this group
      f32x16 acc[CG];
#pragma unroll
      for (int m = 0; m < CG; ++m)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[m][v] = 0.f;
      // one chunk: stage its Theta operands (the barrier also ends every wave's reads of
      // the buffer two chunks back), then `next` issues the loads that overlap the
      // products, then the products
      auto chunk = [&](int ch, auto&& next) {
        float* tb = tbuf + kbuf * TCF;
#pragma unroll
        for (int i = 0; i < CG; ++i) *reinterpret_cast<f32x4*>(tb + (tid + kThreads * i) * 4) = tr[i];
        float xv[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const bool ok = vpt && (ch * 32 + h * 16 + 4 * q < d);
          xv[4 * q + 0] = ok ? xr[q].x : 0.f;
          xv[4 * q + 1] = ok ? xr[q].y : 0.f;
          xv[4 * q + 2] = ok ? xr[q].z : 0.f;
          xv[4 * q + 3] = ok ? xr[q].w : 0.f;
        }
        __syncthreads();
        next();
        // the loads are issued before the products (not sunk below them to reuse the
        // registers of this chunk's X operands)
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          f32x4 a[CG];
#pragma unroll
          for (int m = 0; m < CG; ++m) a[m] = *reinterpret_cast<const f32x4*>(tb + ((j * CG + m) * 64 + lane) * 4);
          // every block of the group, also past the last of a short group (its operands
          // are the last block's, its products unused): a conditional product would make
          // the compiler copy the accumulators
#pragma unroll
          for (int m = 0; m < CG; ++m) {
            acc[m] = mfma32x32x2(a[m].x, xv[4 * j + 0], acc[m]);
            acc[m] = mfma32x32x2(a[m].y, xv[4 * j + 1], acc[m]);
            acc[m] = mfma32x32x2(a[m].z, xv[4 * j + 2], acc[m]);
            acc[m] = mfma32x32x2(a[m].w, xv[4 * j + 3], acc[m]);
          }
        }
        kbuf ^= 1;
      };
      for (int ch = 0; ch + 1 < nch; ++ch) chunk(ch, [&]() { load_chunk(st, cgi, ch + 1); });
      // the last chunk: the rows of U the epilogue needs are loaded meanwhile
      f32x4 ua[CG][4];
      chunk(nch - 1, [&]() {
#pragma unroll
        for (int m = 0; m < CG; ++m)
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            const int c = 32 * (cgi * CG + m) + 8 * qd + 4 * h;
            ua[m][qd] = *reinterpret_cast<const f32x4*>(urow + (c < r ? c : 0));
          }
      });
      // ---- epilogue of the group: lane holds row pt, columns 32 (CG cgi + m) + 8 qd + 4 h + e ----
#pragma unroll
      for (int m = 0; m < CG; ++m) {
        if (m == CG / 2) {
          // the next group's (or super-tile's) first chunk, behind the rest of the epilogue
          // (in the registers of the blocks done)
          const bool ng = cgi + 1 < ngr;
          const int64_t st2 = ng ? st : st + 1;
          if (st2 < sb1) load_chunk(st2, ng ? cgi + 1 : 0, 0);
        }
        if (m < nbg) {
          const int mb = cgi * CG + m;
          float wv[16];
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            const int c = 32 * mb + 8 * qd + 4 * h;
            const bool ok = vpt && c < r;
            const float u4[4] = {ok ? ua[m][qd].x * cf : 0.f, ok ? ua[m][qd].y * cf : 0.f,
                                 ok ? ua[m][qd].z * cf : 0.f, ok ? ua[m][qd].w * cf : 0.f};
            const f32x4 pv = *reinterpret_cast<const f32x4*>(psl + c);
            const f32x4 sv = *reinterpret_cast<const f32x4*>(ssl + c);
            const float pe[4] = {pv.x, pv.y, pv.z, pv.w};
            const float se[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float uu = u4[e];
              float t = fmaf(two_alpha, acc[m][4 * qd + e], uu);
              t = fmaf(neg_alpha, ybar * pe[e], t);
              t = fmaf(neg_alpha, se[e], t);
              float w = fmaxf(t, 0.f);
              if (!vpt || c + e >= r) w = 0.f;
              wv[4 * qd + e] = w;
              const double wd = (double)w, ud = (double)uu;
              sa = fma(wd, wd, sa);
              sb = fma(ud, ud, sb);
              sh = fma(wd, ud, sh);
            }
            if (ok) {
              const f32x4 o = {wv[4 * qd + 0], wv[4 * qd + 1], wv[4 * qd + 2], wv[4 * qd + 3]};
              *reinterpret_cast<f32x4*>(urow + c) = o;
            }
          }
          reduce_scatter<16, 16>(wv, li);
          const double v = (double)wv[0] + shfl_xor_d((double)wv[0], 1);
          if ((li & 1) == 0) colred[wave * r32 + 32 * mb + 8 * (base >> 2) + 4 * h + (base & 3)] += v;
        }
        // one block at a time (its LDS reads are not hoisted above the previous block)
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }

  // ---- workgroup partials ----
  __syncthreads();
  double* out = B.b_part + (int64_t)blockIdx.x * (4 + r32);
  for (int c = tid; c < r32; c += kThreads)
    out[4 + c] = ((colred[c] + colred[r32 + c]) + colred[2 * r32 + c]) + colred[3 * r32 + c];
  const double ta = block_sum_d(sa, dred);
  const double tb2 = block_sum_d(sb, dred);
  const double th = block_sum_d(sh, dred);
  if (tid == 0) {
    out[0] = ta;
    out[1] = tb2;
    out[2] = th;
    out[3] = 0.0;
  }
}

// ---------------------------------------------------------------------------
// Pass B above 256 columns (NB = 10, 12 or 14 blocks of 32).  As k_pass_b, with
// the columns taken two blocks at a time: per 128-row super-tile each wave forms
// q = u.p - 1 over the whole row first, then for each pair of column blocks the
// product (the Xhat row chunks re-read from cache), the epilogue and W; column
// sums go to the wave's row of LDS per tile (lanes l and l^1 combined first).
// ---------------------------------------------------------------------------
template <bool THETA_LDS, bool VEC>
__global__ __launch_bounds__(kThreads) void k_pass_b_wide(Geometry g, Bufs B, StepArgs S) {
  if (halted(B.ctl)) return;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  float* th_s = reinterpret_cast<float*>(smem_raw);                 // d32*r32 if THETA_LDS
  float* ps = th_s + (THETA_LDS ? g.d32 * g.r32 : 0);               // r32
  float* ss = ps + g.r32;                                           // r32
  double* colred = reinterpret_cast<double*>(ss + g.r32);          // 4 x r32
  double* dred = colred + 4 * g.r32;                                // 8

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5;
  const int li = lane & 31;
  const int64_t n = g.n;
  const int d = g.d, r = g.r, r32 = g.r32, NBt = g.NB;
  const int nch = g.nch;
  const float cf = B.ctl->c_f;
  const float gam = S.gamma_f;
  const float two_alpha = S.two_alpha_f;
  const float neg_alpha = -S.alpha_f;

  if (THETA_LDS) {
    const int tot4 = (g.d32 * r32) >> 2;
    const f32x4* src = reinterpret_cast<const f32x4*>(B.theta);
    f32x4* dst = reinterpret_cast<f32x4*>(th_s);
    for (int v = tid; v < tot4; v += kThreads) dst[v] = src[v];
  }
  for (int c = tid; c < r32; c += kThreads) {
    ps[c] = B.p[c];
    ss[c] = B.s[c];
  }
  for (int c = tid; c < 4 * r32; c += kThreads) colred[c] = 0.0;
  __syncthreads();
  const float* theta = THETA_LDS ? th_s : B.theta;

  double sa = 0.0, sb = 0.0, sh = 0.0;
  int base = 0;  // local index (8 qd + e ordering) of the column sum this lane keeps
  if (li & 16) base += 8;
  if (li & 8) base += 4;
  if (li & 4) base += 2;
  if (li & 2) base += 1;

  const int64_t sb0 = (int64_t)blockIdx.x * g.tilesB / g.GB;
  const int64_t sb1 = (int64_t)(blockIdx.x + 1) * g.tilesB / g.GB;
  for (int64_t st = sb0; st < sb1; ++st) {
    const int64_t pt = st * kTPB + wave * 32 + li;
    const bool vpt = pt < n;
    const float* xrow = B.X + (vpt ? pt : 0) * (int64_t)d;
    float* urow = B.U + (vpt ? pt : 0) * (int64_t)r;
    auto load_u4 = [&](int c, float out[4]) {
      if (VEC) {
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
        if (vpt && c < r) t = *reinterpret_cast<const f32x4*>(urow + c);
        out[0] = t.x * cf;
        out[1] = t.y * cf;
        out[2] = t.z * cf;
        out[3] = t.w * cf;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = (vpt && c + e < r) ? urow[c + e] * cf : 0.f;
      }
    };
    // q = u.p - 1 over the whole row (fp32 dot over the lane's half, then the other half)
    float dotf = 0.f;
    for (int m = 0; m < NBt; ++m)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int c = 32 * m + 8 * qd + 4 * h;
        float u4[4];
        load_u4(c, u4);
        const f32x4 pv = *reinterpret_cast<const f32x4*>(ps + c);
        dotf = fmaf(u4[0], pv.x, dotf);
        dotf = fmaf(u4[1], pv.y, dotf);
        dotf = fmaf(u4[2], pv.z, dotf);
        dotf = fmaf(u4[3], pv.w, dotf);
      }
    dotf += shfl_xor_f(dotf, 32);
    float ybar = 0.f;
    if (vpt) ybar = fmaf(gam, dotf - 1.0f, B.y[pt]);

    for (int cg = 0; cg < NBt; cg += 2) {
      f32x16 acc[2];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;
      for (int ch = 0; ch < nch; ++ch) {
        const int fb = ch * 32 + h * 16;
        float xv[16];
        if (VEC) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            f32x4 t = {0.f, 0.f, 0.f, 0.f};
            if (vpt && fb + 4 * q < d) t = *reinterpret_cast<const f32x4*>(xrow + fb + 4 * q);
            xv[4 * q + 0] = t.x;
            xv[4 * q + 1] = t.y;
            xv[4 * q + 2] = t.z;
            xv[4 * q + 3] = t.w;
          }
        } else {
#pragma unroll
          for (int q = 0; q < 16; ++q) xv[q] = (vpt && fb + q < d) ? xrow[fb + q] : 0.f;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
          for (int m = 0; m < 2; ++m) {
            const f32x4 a =
                *reinterpret_cast<const f32x4*>(theta + ((((int64_t)ch * 4 + j) * NBt + cg + m) * 64 + lane) * 4);
            acc[m] = mfma32x32x2(a.x, xv[4 * j + 0], acc[m]);
            acc[m] = mfma32x32x2(a.y, xv[4 * j + 1], acc[m]);
            acc[m] = mfma32x32x2(a.z, xv[4 * j + 2], acc[m]);
            acc[m] = mfma32x32x2(a.w, xv[4 * j + 3], acc[m]);
          }
        }
      }
      // ---- epilogue of the pair: lane holds row pt, columns 32 (cg + m) + 8 qd + 4 h + e ----
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        float wv[16];
#pragma unroll
        for (int qd = 0; qd < 4; ++qd) {
          const int c = 32 * (cg + m) + 8 * qd + 4 * h;
          float u4[4];
          load_u4(c, u4);
          const f32x4 pv = *reinterpret_cast<const f32x4*>(ps + c);
          const f32x4 sv = *reinterpret_cast<const f32x4*>(ss + c);
          const float pe[4] = {pv.x, pv.y, pv.z, pv.w};
          const float se[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float uu = u4[e];
            float t = fmaf(two_alpha, acc[m][4 * qd + e], uu);
            t = fmaf(neg_alpha, ybar * pe[e], t);
            t = fmaf(neg_alpha, se[e], t);
            float w = fmaxf(t, 0.f);
            if (!vpt || c + e >= r) w = 0.f;
            wv[4 * qd + e] = w;
            const double wd = (double)w, ud = (double)uu;
            sa = fma(wd, wd, sa);
            sb = fma(ud, ud, sb);
            sh = fma(wd, ud, sh);
          }
          if (vpt) {
            if (VEC) {
              if (c < r) {
                f32x4 o = {wv[4 * qd + 0], wv[4 * qd + 1], wv[4 * qd + 2], wv[4 * qd + 3]};
                *reinterpret_cast<f32x4*>(urow + c) = o;
              }
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (c + e < r) urow[c + e] = wv[4 * qd + e];
            }
          }
        }
        reduce_scatter<16, 16>(wv, li);
        double v = (double)wv[0];
        v += shfl_xor_d(v, 1);
        if ((li & 1) == 0) colred[wave * r32 + 32 * (cg + m) + 8 * (base >> 2) + 4 * h + (base & 3)] += v;
      }
    }
  }

  // ---- workgroup partials ----
  __syncthreads();
  double* out = B.b_part + (int64_t)blockIdx.x * (4 + r32);
  for (int c = tid; c < r32; c += kThreads)
    out[4 + c] = ((colred[c] + colred[r32 + c]) + colred[2 * r32 + c]) + colred[3 * r32 + c];
  const double ta = block_sum_d(sa, dred);
  const double tb2 = block_sum_d(sb, dred);
  const double th = block_sum_d(sh, dred);
  if (tid == 0) {
    out[0] = ta;
    out[1] = tb2;
    out[2] = th;
    out[3] = 0.0;
  }
}

// ---------------------------------------------------------------------------
// Pass B, resident-tile form (d <= 128, r <= 128, 16-byte rows).  Same
// arithmetic and partial layout as k_pass_b; each wave holds its tile's whole
// Xhat slab (NCH chunks) and U slab in registers: the U loads of a tile are
// issued before its matrix product and the next tile's Xhat before its epilogue.
// ---------------------------------------------------------------------------
template <int NB, int NCH>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8))) void k_pass_b_res(
    Geometry g, Bufs B, StepArgs S) {
  if (halted(B.ctl)) return;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  float* th_s = reinterpret_cast<float*>(smem_raw);  // d32*r32
  float* ps = th_s + g.d32 * g.r32;                   // r32
  float* ss = ps + g.r32;                             // r32
  double* colred = reinterpret_cast<double*>(ss + g.r32);
  double* dred = colred + 4 * g.r32;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5;
  const int li = lane & 31;
  const int64_t n = g.n;
  const int d = g.d, r = g.r, r32 = g.r32;
  const float cf = B.ctl->c_f;
  const float gam = S.gamma_f;
  const float two_alpha = S.two_alpha_f;
  const float neg_alpha = -S.alpha_f;

  {
    const int tot4 = (g.d32 * r32) >> 2;
    const f32x4* src = reinterpret_cast<const f32x4*>(B.theta);
    f32x4* dst = reinterpret_cast<f32x4*>(th_s);
    for (int v = tid; v < tot4; v += kThreads) dst[v] = src[v];
  }
  for (int c = tid; c < r32; c += kThreads) {
    ps[c] = B.p[c];
    ss[c] = B.s[c];
  }
  __syncthreads();

  double sa = 0.0, sb = 0.0, sh = 0.0;
  double colacc[NB];
#pragma unroll
  for (int m = 0; m < NB; ++m) colacc[m] = 0.0;
  int base = 0;
  if (li & 16) base += 8;
  if (li & 8) base += 4;
  if (li & 4) base += 2;
  if (li & 2) base += 1;

  const int64_t sb0 = (int64_t)blockIdx.x * g.tilesB / g.GB;
  const int64_t sb1 = (int64_t)(blockIdx.x + 1) * g.tilesB / g.GB;

  float xv[NCH][16];
  auto load_x = [&](int64_t st, int ch) {
    const int64_t pt = st * kTPB + wave * 32 + li;
    const bool ok = (st < sb1) && (pt < n);
    const float* xrow = B.X + (ok ? pt : 0) * (int64_t)d;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int f = ch * 32 + h * 16 + 4 * q;
      // raw values: features >= d meet zero rows of Theta, rows >= n are masked in the epilogue
      const f32x4 t = *reinterpret_cast<const f32x4*>(xrow + (f < d ? f : 0));
      xv[ch][4 * q + 0] = t.x;
      xv[ch][4 * q + 1] = t.y;
      xv[ch][4 * q + 2] = t.z;
      xv[ch][4 * q + 3] = t.w;
    }
  };
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    __builtin_amdgcn_sched_barrier(0);
    load_x(sb0, ch);
  }
  __builtin_amdgcn_sched_barrier(0);

  for (int64_t st = sb0; st < sb1; ++st) {
    __builtin_amdgcn_sched_barrier(0);
    const int64_t pt = st * kTPB + wave * 32 + li;
    const bool vpt = pt < n;
    float* urow = B.U + (vpt ? pt : 0) * (int64_t)r;
    // epilogue operands, issued before the matrix product (raw; scaled and masked at use)
    f32x4 uraw[NB][4];
#pragma unroll
    for (int m = 0; m < NB; ++m)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int c = 32 * m + 8 * qd + 4 * h;
        uraw[m][qd] = *reinterpret_cast<const f32x4*>(urow + (c < r ? c : 0));
      }
    const float yraw = B.y[vpt ? pt : 0];
    __builtin_amdgcn_sched_barrier(0);

    f32x16 acc[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int m = 0; m < NB; ++m) {
          const f32x4 a = *reinterpret_cast<const f32x4*>(th_s + (((ch * 4 + j) * NB + m) * 64 + lane) * 4);
          acc[m] = mfma32x32x2(a.x, xv[ch][4 * j + 0], acc[m]);
          acc[m] = mfma32x32x2(a.y, xv[ch][4 * j + 1], acc[m]);
          acc[m] = mfma32x32x2(a.z, xv[ch][4 * j + 2], acc[m]);
          acc[m] = mfma32x32x2(a.w, xv[ch][4 * j + 3], acc[m]);
        }
      __builtin_amdgcn_sched_barrier(0);
      load_x(st + 1, ch);  // this chunk of the next tile: a whole tile of lead time
      __builtin_amdgcn_sched_barrier(0);
    }

    int lds_off = 0;  // opaque zero offset: keeps the reads in LDS address space
    asm volatile("" : "+v"(lds_off));
    const float* psl = ps + lds_off;
    const float* ssl = ss + lds_off;
    float u[NB][16];
#pragma unroll
    for (int m = 0; m < NB; ++m)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const bool ok = vpt && (32 * m + 8 * qd + 4 * h) < r;
        u[m][4 * qd + 0] = ok ? uraw[m][qd].x * cf : 0.f;
        u[m][4 * qd + 1] = ok ? uraw[m][qd].y * cf : 0.f;
        u[m][4 * qd + 2] = ok ? uraw[m][qd].z * cf : 0.f;
        u[m][4 * qd + 3] = ok ? uraw[m][qd].w * cf : 0.f;
      }
    float dotf = 0.f;
#pragma unroll
    for (int m = 0; m < NB; ++m)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const f32x4 pv = *reinterpret_cast<const f32x4*>(psl + 32 * m + 8 * qd + 4 * h);
        dotf = fmaf(u[m][4 * qd + 0], pv.x, dotf);
        dotf = fmaf(u[m][4 * qd + 1], pv.y, dotf);
        dotf = fmaf(u[m][4 * qd + 2], pv.z, dotf);
        dotf = fmaf(u[m][4 * qd + 3], pv.w, dotf);
      }
    dotf += shfl_xor_f(dotf, 32);
    const float ybar = vpt ? fmaf(gam, dotf - 1.0f, yraw) : 0.f;
#pragma unroll
    for (int m = 0; m < NB; ++m) {
      float wv[16];
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int c = 32 * m + 8 * qd + 4 * h;
        const f32x4 pv = *reinterpret_cast<const f32x4*>(psl + c);
        const f32x4 sv = *reinterpret_cast<const f32x4*>(ssl + c);
        const float pe[4] = {pv.x, pv.y, pv.z, pv.w};
        const float se[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float uu = u[m][4 * qd + e];
          float t = fmaf(two_alpha, acc[m][4 * qd + e], uu);
          t = fmaf(neg_alpha, ybar * pe[e], t);
          t = fmaf(neg_alpha, se[e], t);
          float w = fmaxf(t, 0.f);
          if (!vpt || c + e >= r) w = 0.f;
          wv[4 * qd + e] = w;
          const double wd = (double)w, ud = (double)uu;
          sa = fma(wd, wd, sa);
          sb = fma(ud, ud, sb);
          sh = fma(wd, ud, sh);
        }
        // unconditional store (invalid lanes write the dump slot): no branch around it
        float* dst = (vpt && c < r) ? (urow + c) : B.dump;
        f32x4 o = {wv[4 * qd + 0], wv[4 * qd + 1], wv[4 * qd + 2], wv[4 * qd + 3]};
        *reinterpret_cast<f32x4*>(dst) = o;
      }
      reduce_scatter<16, 16>(wv, li);
      colacc[m] += (double)wv[0];
    }
  }

  for (int c = tid; c < 4 * r32; c += kThreads) colred[c] = 0.0;
  __syncthreads();
#pragma unroll
  for (int m = 0; m < NB; ++m) {
    const double v = colacc[m] + shfl_xor_d(colacc[m], 1);
    if ((li & 1) == 0) {
      const int col = 32 * m + 8 * (base >> 2) + 4 * h + (base & 3);
      colred[wave * r32 + col] = v;
    }
  }
  __syncthreads();
  double* out = B.b_part + (int64_t)blockIdx.x * (4 + r32);
  for (int c = tid; c < r32; c += kThreads)
    out[4 + c] = ((colred[c] + colred[r32 + c]) + colred[2 * r32 + c]) + colred[3 * r32 + c];
  const double ta = block_sum_d(sa, dred);
  const double tb2 = block_sum_d(sb, dred);
  const double th = block_sum_d(sh, dred);
  if (tid == 0) {
    out[0] = ta;
    out[1] = tb2;
    out[2] = th;
    out[3] = 0.0;
  }
}

// ---------------------------------------------------------------------------
// Control after pass B (one workgroup): Algorithm 2 steps (d)-(f).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_ctl_b(Geometry g, Bufs B, StepArgs S) {
  DevCtl* ctl = B.ctl;
  if (halted(ctl)) return;
  __shared__ double cbuf[1];
  __shared__ double abh[4];
  const int tid = threadIdx.x;
  const int C = 4 + g.r32;
  // a, b, h and the range flag summed by threads 0..3 at the same time
  if (tid < 4) abh[tid] = seq_sum<double>(B.seg_b + tid, C, g.SB);
  __syncthreads();
  if (tid == 0) {
    const double a = abh[0], b = abh[1], h = abh[2], over = abh[3];
    const double nu = sqrt(a);
    const int64_t t = ctl->t_done;
    nlr_iter_stats* rec = &B.hist[t % kHistCap];
    rec->a = a;
    rec->b = b;
    rec->h = h;
    if (over > 0.0) {
      // a split-fp16 operand of W left fp16's range (the fused pass's flag)
      ctl->breakdown = kRangeError;
      rec->breakdown = kRangeError;
      cbuf[0] = 0.0;
    } else if (!(nu > 1e-20) || !isfinite(a)) {
      ctl->breakdown = 1;
      rec->breakdown = 1;
      cbuf[0] = 0.0;
    } else {
      const float cf = (float)(sqrt(S.K) / nu);
      const double c = (double)cf;
      double D = c * c * a + b - 2.0 * c * h;
      if (D < 0.0) D = 0.0;
      const double delta = sqrt(D) / sqrt(S.K);
      const int gate = D < S.eps_d * S.eps_d * S.K;
      ctl->a = a;
      ctl->b = b;
      ctl->h = h;
      ctl->Delta = D;
      ctl->delta = delta;
      ctl->gate = gate;
      ctl->c_f = cf;
      ctl->t_done = t + 1;
      rec->c = cf;
      rec->delta = delta;
      rec->dual_step = gate;
      cbuf[0] = c;
    }
  }
  __syncthreads();
  const double c = cbuf[0];
  if (c > 0.0) {
    for (int col = tid; col < g.r32; col += kThreads) {
      const double t = seq_sum<double>(B.seg_b + 4 + col, C, g.SB);
      B.p[col] = (col < g.r) ? (float)(c * t) : 0.f;
    }
  }
}

// ---------------------------------------------------------------------------
// One-pass iteration (the eight-wave fused pass B does the row work too), control
// after the pass (one workgroup).  Unless the row pass ran first (rows_first: the
// previous iteration's stopping rule could fire, and k_ctl_a has decided it and
// written the record), the pass did the row work of this iteration -- the end of
// the previous one: its gated dual step, q and the objective terms -- before the
// primal step; the stopping rule could not fire then, and rho and the objective
// are recorded here.  Then as k_ctl_b, the column sums P of W and W^T ytilde for
// the next iteration's s, and whether the next iteration's row pass runs first.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_ctl_one(Geometry g, Bufs B, StepArgs S) {
  DevCtl* ctl = B.ctl;
  if (halted(ctl)) return;
  __shared__ double red[8];
  __shared__ double cbuf[1];
  const int tid = threadIdx.x;
  double th2 = 0.0;
  for (int k = tid; k < g.RT; k += kThreads) th2 += B.th2_part[k];
  th2 = block_sum_d(th2, red);
  if (tid == 0) {
    const int64_t t = ctl->t_done;
    if (!ctl->rows_first) {
      const double qq = B.seg_a[0], yq = B.seg_a[1];
      const double rho = sqrt(qq * S.inv_n);
      ctl->rho = rho;
      if (S.end_work && t > 0) {
        nlr_iter_stats* prev = &B.hist[(t - 1) % kHistCap];
        prev->rho = rho;
        prev->stop = 0;
      }
      const double obj = -th2 + yq + 0.5 * S.beta * S.inv_n * qq;
      ctl->objective = obj;
      ctl->theta_fro2 = th2;
      nlr_iter_stats* cur = &B.hist[t % kHistCap];
      cur->t = t;
      cur->objective = obj;
      cur->theta_fro2 = th2;
      cur->rho = 0.0;
      cur->stop = 0;
    }
    cbuf[0] = 0.0;
    const double a = B.seg_b[0], b = B.seg_b[1], h = B.seg_b[2];
    const double nu = sqrt(a);
    nlr_iter_stats* rec = &B.hist[t % kHistCap];
    rec->a = a;
    rec->b = b;
    rec->h = h;
    rec->dual_step = 0;
    rec->breakdown = 0;
    if (B.seg_b[3] > 0.0) {
      // the split W operand left fp16's range: stop before Theta and s use it
      ctl->breakdown = kRangeError;
      rec->breakdown = kRangeError;
      rec->c = 0.f;
      rec->delta = 0.0;
    } else if (!(nu > 1e-20) || !isfinite(a)) {
      // W_{t+1} has overwritten the factor (Algorithm 2 order)
      ctl->breakdown = 1;
      rec->breakdown = 1;
      rec->c = 0.f;
      rec->delta = 0.0;
    } else {
      const float cf = (float)(sqrt(S.K) / nu);
      const double c = (double)cf;
      double D = c * c * a + b - 2.0 * c * h;
      if (D < 0.0) D = 0.0;
      const double delta = sqrt(D) / sqrt(S.K);
      const int gate = D < S.eps_d * S.eps_d * S.K;
      ctl->a = a;
      ctl->b = b;
      ctl->h = h;
      ctl->Delta = D;
      ctl->delta = delta;
      ctl->gate = gate;
      ctl->c_f = cf;
      ctl->c_gram = c;
      ctl->t_done = t + 1;
      rec->c = cf;
      rec->delta = delta;
      rec->dual_step = gate;
      cbuf[0] = c;
      // the next iteration of this call has this one's end-of-iteration work pending
      StepArgs nx = S;
      nx.end_work = 1;
      ctl->rows_first = stop_possible(ctl, nx) ? 1 : 0;
    }
  }
  __syncthreads();
  const double c = cbuf[0];
  if (c > 0.0) {
    for (int col = tid; col < g.r32; col += kThreads) {
      const double P = B.seg_b[4 + col], wy = B.seg_a[4 + col];
      B.p[col] = (col < g.r) ? (float)(c * P) : 0.f;
      B.gram_vec[col] = P;
      B.gram_vec[g.r32 + col] = wy;
    }
  }
}

// ---------------------------------------------------------------------------
// Fixed-order sums over the GB rows of the one-pass iteration's per-workgroup
// statistics, one segment each: by 0 a_part -> seg_a, 1 b_part -> seg_b.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void seg_ab_block(const Geometry& g, const Bufs& B, int bx, int by, double* red) {
  const double* P = by ? B.b_part : B.a_part;
  double* out = by ? B.seg_b : B.seg_a;
  const int C = 4 + g.r32;
  const int tid = threadIdx.x;
  // 8 columns x 32 row phases per block; the phases are added in a fixed tree
  const int col = bx * 8 + (tid & 7);
  const int sub = tid >> 3;
  double acc = 0.0;
  if (col < C && sub < g.GB) acc = seq_sum<double>(P + (int64_t)sub * C + col, 32 * (int64_t)C, (g.GB - sub + 31) / 32);
  red[tid] = acc;
  __syncthreads();
  for (int w = 16; w >= 1; w >>= 1) {
    if (sub < w) red[tid] = red[tid] + red[tid + 8 * w];
    __syncthreads();
  }
  if (tid < 8 && col < C) out[col] = red[tid];
}

// The segment sums after the fused pass B of the single-Xhat-pass form in one launch:
// blockIdx.y < SAF the segments of the Theta partial rows, SAF .. SAF + SB - 1 those of
// the statistics rows (b_part; the first (4 + r32 + 63) / 64 blocks of those rows).
__global__ __launch_bounds__(kThreads) void k_seg_fused(Geometry g, Bufs B) {
  if (halted(B.ctl)) return;
  __shared__ double red[kThreads];
  const int by = blockIdx.y;
  if (by < g.SAF) {
    seg_sum_block<float>(B.theta_part, g.GB, g.theta_cols, B.seg_theta, g.SAF, blockIdx.x, by, red);
  } else if ((int)blockIdx.x < (4 + g.r32 + 63) / 64) {
    seg_sum_block<double>(B.b_part, g.GB, 4 + g.r32, B.seg_b, g.SB, blockIdx.x, by - g.SAF, red);
  }
}

// The segment sums after a one-pass kernel in one launch: blockIdx.y < nseg the
// segments of the Theta and W^T W partial rows, nseg and nseg + 1 the statistics
// (a_part, b_part; the first (4 + r32 + 7) / 8 blocks of those rows).
__global__ __launch_bounds__(kThreads) void k_seg_onepass(Geometry g, Bufs B, int nseg) {
  if (halted(B.ctl)) return;
  __shared__ double red[kThreads];
  const int by = blockIdx.y;
  if (by < nseg) {
    seg_sum_block<float>(B.theta_part, g.GB, g.theta_cols, B.seg_theta, nseg, blockIdx.x, by, red);
  } else if ((int)blockIdx.x < (4 + g.r32 + 7) / 8) {
    seg_ab_block(g, B, blockIdx.x, by - nseg, red);
  }
}

// ---------------------------------------------------------------------------
// s = U^T ybar of the one-pass iteration from the Gram terms of the pass that
// produced U = c W.  Per row q = u.p - 1 = c^2 w.P - 1 and ybar = ytilde_prev +
// (1 + gate) gamma q (the pending gated dual step, then the penalty term; gamma =
// beta / n), so
//   s = c W^T ytilde_prev + (1 + gate) gamma c (c^2 (W^T W) P - P)
// with W^T W (the columns after Theta in the Theta partial rows, reduced with them
// and multiplied by P in k_reduce_theta), P and W^T ytilde_prev summed in a fixed
// order (FP64).  The last term is U^T q: small near feasibility and weighted by
// gamma, so the fp32-accumulated Gram partials carry it well below the iteration's
// rounding.  k_reduce_theta forms s right after the pass with the step arguments of
// the call; k_s_gram (one workgroup) forms it again at the start of a host call,
// whose step arguments (beta) may differ.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float s_from_gram(const Bufs& B, int r32, int k, double gp, float gamma_f) {
  const double c = B.ctl->c_gram;
  const double gmul = (1.0 + (B.ctl->gate ? 1.0 : 0.0)) * (double)gamma_f;
  const double P = B.gram_vec[k], wy = B.gram_vec[r32 + k];
  return (float)(c * wy + gmul * c * (c * c * gp - P));
}

// At the start of a host call (one workgroup): s from the stored Gram terms with the
// beta of this call when they are valid, and whether the first iteration's row pass
// runs before its pass: 2 when there are no Gram terms (after nlr_init; s then comes
// from the row pass), 1 when the stopping rule of the previous iteration may fire
// under this call's arguments (eps, T_min; the row pass settles the rule, s stays
// the Gram-derived one), else 0.
__global__ __launch_bounds__(64) void k_onepass_begin(Geometry g, Bufs B, StepArgs S, int gram_valid) {
  if (halted(B.ctl)) return;
  const int r32 = g.r32;
  const int k = threadIdx.x;
  if (k == 0) B.ctl->rows_first = !gram_valid ? 2 : (stop_possible(B.ctl, S) ? 1 : 0);
  if (!gram_valid || k >= r32) return;
  const float sk = s_from_gram(B, r32, k, B.gram_vec[2 * r32 + k], S.gamma_f);
  B.s[k] = (k < g.r) ? sk : 0.f;
}

// ---------------------------------------------------------------------------
// Row-argmax labels, lowest index on ties.  A row is read by the 16 lanes of a DPP
// row, four rows per wave and step: with 16-byte rows (VEC) lane j reads columns
// 4j .. 4j + 3, 64 + 4j .. (NCK = ceil(r / 64) pieces), so one load instruction covers
// 256 contiguous bytes of each of its four rows, and a workgroup takes 16 RPS
// consecutive rows per step, all their loads issued before any is compared (pieces
// past the last column or row read a valid address and are skipped); otherwise lane j
// reads columns
// j, j + 16, ...  Each lane keeps its first maximum (columns in increasing order,
// strict >), then the 16 candidates are reduced pairwise: the larger value, the lower
// column on equal values.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void label_reduce16(float& best, int& arg) {
  constexpr int kNone = 0x7fffffff;
#pragma unroll
  for (int m = 1; m < 16; m <<= 1) {
    const float ob = shfl_xor_f(best, m);
    const int oa = __shfl_xor(arg, m, 64);
    if (oa != kNone && (arg == kNone || ob > best || (ob == best && oa < arg))) {
      best = ob;
      arg = oa;
    }
  }
}

template <bool VEC, int NCK, int RPS>
__global__ __launch_bounds__(kThreads) void k_labels(Geometry g, const float* __restrict__ U,
                                                     int32_t* __restrict__ labels) {
  constexpr int kNone = 0x7fffffff;  // no column seen yet
  const int lane = threadIdx.x & 63;
  const int j = lane & 15;
  const int64_t n = g.n;
  const int r = g.r;
  if (VEC) {
    // a workgroup takes 16 RPS consecutive rows per step; group g its rows 16 k + g
    const int64_t bstep = (int64_t)gridDim.x * 16 * RPS;
    for (int64_t b0 = (int64_t)blockIdx.x * 16 * RPS; b0 < n; b0 += bstep) {
      const int64_t i0 = b0 + (threadIdx.x >> 4);
      f32x4 v[RPS][NCK];
#pragma unroll
      for (int k = 0; k < RPS; ++k) {
        const int64_t i = i0 + 16 * k;
        const float* row = U + (i < n ? i : 0) * (int64_t)r;
#pragma unroll
        for (int q = 0; q < NCK; ++q) {
          const int c0 = 4 * j + 64 * q;
          v[k][q] = *reinterpret_cast<const f32x4*>(row + (c0 < r ? c0 : 0));
        }
      }
#pragma unroll
      for (int k = 0; k < RPS; ++k) {
        float best = 0.f;
        int arg = kNone;
#pragma unroll
        for (int q = 0; q < NCK; ++q) {
          const int c0 = 4 * j + 64 * q;  // r % 4 == 0: c0 + 3 < r when c0 < r
          if (c0 < r) {
            const float e[4] = {v[k][q].x, v[k][q].y, v[k][q].z, v[k][q].w};
#pragma unroll
            for (int e4 = 0; e4 < 4; ++e4)
              if (arg == kNone || e[e4] > best) {
                best = e[e4];
                arg = c0 + e4;
              }
          }
        }
        label_reduce16(best, arg);
        const int64_t i = i0 + 16 * k;
        if (i < n && j == 0) labels[i] = arg;
      }
    }
  } else {
    const int64_t rows_per_step = (int64_t)gridDim.x * (kThreads / 16);
    const int64_t first = (int64_t)blockIdx.x * (kThreads / 16) + (threadIdx.x >> 4);
    for (int64_t i = first; i - (threadIdx.x >> 4) < n; i += rows_per_step) {
      const bool vrow = i < n;
      const float* row = U + (vrow ? i : 0) * (int64_t)r;
      float best = 0.f;
      int arg = kNone;
      for (int c = j; c < r; c += 16) {
        const float v = row[c];
        if (arg == kNone || v > best) {
          best = v;
          arg = c;
        }
      }
      label_reduce16(best, arg);
      if (vrow && j == 0) labels[i] = arg;
    }
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
// Kernels whose dynamic LDS exceeds 64 KiB need the per-function limit raised
// (gfx950 has 160 KiB of LDS per workgroup).
template <typename F>
static hipError_t allow_lds(F* kern, size_t lds) {
  if (lds <= (64u << 10)) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)lds);
}

// Dynamic LDS of k_pass_a in a mode: the staged tiles, ybar and p, the reductions; the
// combine of the k-slices (MBG < 4) overlaps the tiles
template <int MBG, int NBG, int MODE>
static size_t pass_a_lds(const Geometry& g) {
  const bool theta = MODE == kAIter || MODE == kATheta;
  const int64_t us = MODE == kATheta ? NBG * 32 + 4 : g.us_stride;
  const int64_t floats = (theta ? (int64_t)kTPA * g.xs_stride : 0) + (int64_t)kTPA * us + kTPA + g.r32;
  int64_t bytes = floats * 4 + (256 + 8) * 8;
  const int64_t comb = (int64_t)MBG * NBG * 16 * 64 * 4;
  if (theta && MBG < 4 && comb > floats * 4) bytes = comb + (256 + 8) * 8 + 64;
  return (size_t)((bytes + 15) & ~15);
}

template <int MBG, int NBG, int MODE>
static hipError_t pass_a_launch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  // the finish pass writes no Theta partials: its grid is sized for the rows alone
  const dim3 grid(MODE == kAFinish ? g.GAF : g.GA, MODE == kAFinish ? 1 : g.mgroups * g.ngroups);
  const size_t lds = pass_a_lds<MBG, NBG, MODE>(g);
  if (lds > (160u << 10)) return hipErrorInvalidValue;
  hipError_t e = allow_lds(k_pass_a<MBG, NBG, MODE>, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_pass_a<MBG, NBG, MODE>), grid, dim3(kThreads), lds, st, g, b, a);
  return hipGetLastError();
}

template <int MBG, int MODE>
static hipError_t pass_a_nbg(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  switch (g.NBG) {
    case 1: return pass_a_launch<MBG, 1, MODE>(g, b, a, st);
    case 2: return pass_a_launch<MBG, 2, MODE>(g, b, a, st);
    case 4: return pass_a_launch<MBG, 4, MODE>(g, b, a, st);
    case 5: return pass_a_launch<MBG, 5, MODE>(g, b, a, st);
    case 7: return pass_a_launch<MBG, 7, MODE>(g, b, a, st);
    default: return hipErrorInvalidValue;
  }
}

template <int MBG, int NBG>
static hipError_t theta_wide_launch(const Geometry& g, const Bufs& b, hipStream_t st) {
  const size_t tiles = (size_t)kTPA * ((MBG * 32 + 4) + (NBG * 32 + 4)) * 4;
  const size_t comb = MBG < 4 ? (size_t)MBG * NBG * 16 * 64 * 4 : 0;
  const size_t lds = tiles > comb ? tiles : comb;
  hipError_t e = allow_lds(k_theta_wide<MBG, NBG>, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_theta_wide<MBG, NBG>), dim3(g.GA, g.mgroups * g.ngroups), dim3(kThreads), lds, st, g, b);
  return hipGetLastError();
}

template <int MBG>
static hipError_t theta_wide_nbg(const Geometry& g, const Bufs& b, hipStream_t st) {
  switch (g.NBG) {
    case 4: return theta_wide_launch<MBG, 4>(g, b, st);
    case 5: return theta_wide_launch<MBG, 5>(g, b, st);
    case 7: return theta_wide_launch<MBG, 7>(g, b, st);
    default: return hipErrorInvalidValue;
  }
}

static hipError_t launch_theta_wide(const Geometry& g, const Bufs& b, hipStream_t st) {
  switch (g.MBG) {
    case 1: return theta_wide_nbg<1>(g, b, st);
    case 2: return theta_wide_nbg<2>(g, b, st);
    case 4: return theta_wide_nbg<4>(g, b, st);
    default: return hipErrorInvalidValue;
  }
}

static hipError_t launch_rows_wide(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  const dim3 grid(g.GAF), blk(kThreads);
  switch ((g.r + 63) / 64) {
    case 3: hipLaunchKernelGGL(k_rows_wide<3>, grid, blk, 0, st, g, b, a); break;
    case 4: hipLaunchKernelGGL(k_rows_wide<4>, grid, blk, 0, st, g, b, a); break;
    case 5: hipLaunchKernelGGL(k_rows_wide<5>, grid, blk, 0, st, g, b, a); break;
    case 6: hipLaunchKernelGGL(k_rows_wide<6>, grid, blk, 0, st, g, b, a); break;
    case 7: hipLaunchKernelGGL(k_rows_wide<7>, grid, blk, 0, st, g, b, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int MODE>
static hipError_t pass_a_mbg(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  switch (g.MBG) {
    case 1: return pass_a_nbg<1, MODE>(g, b, a, st);
    case 2: return pass_a_nbg<2, MODE>(g, b, a, st);
    case 4: return pass_a_nbg<4, MODE>(g, b, a, st);
    default: return hipErrorInvalidValue;
  }
}

template <int FV, int NGF, int CV>
static hipError_t pass_a_rows_launch(const Geometry& g, const Bufs& b, const StepArgs& a, int mode,
                                     hipStream_t st) {
  if (mode == kPassFinish)
    hipLaunchKernelGGL((k_pass_a_rows<FV, NGF, CV, kPassFinish>), dim3(g.GA), dim3(kThreads), 0, st, g, b, a);
  else if (mode == kPassRows)
    hipLaunchKernelGGL((k_pass_a_rows<FV, NGF, CV, kPassRows>), dim3(g.GA), dim3(kThreads), 0, st, g, b, a);
  else
    hipLaunchKernelGGL((k_pass_a_rows<FV, NGF, CV, kPassIter>), dim3(g.GA), dim3(kThreads), 0, st, g, b, a);
  return hipGetLastError();
}

static hipError_t pass_a_rows_dispatch(const Geometry& g, const Bufs& b, const StepArgs& a, int finish,
                                       hipStream_t st) {
  // narrow factors in the single-Xhat-pass form: the row and finish passes (both, so
  // that their row dots agree) pack eight lanes per row; pass A with its product keeps
  // the 16-lane layout
  if (g.fused && g.r <= 16 && g.r % 2 == 0 && (finish == kPassRows || finish == kPassFinish)) {
    if (finish == kPassFinish)
      hipLaunchKernelGGL((k_rows_narrow<kPassFinish>), dim3(g.GA), dim3(kThreads), 0, st, g, b, a);
    else
      hipLaunchKernelGGL((k_rows_narrow<kPassRows>), dim3(g.GA), dim3(kThreads), 0, st, g, b, a);
    return hipGetLastError();
  }
  const int key = g.a_fv * 100 + g.a_ngf * 10 + g.a_cv;
  switch (key) {
    case 111: return pass_a_rows_launch<1, 1, 1>(g, b, a, finish, st);
    case 112: return pass_a_rows_launch<1, 1, 2>(g, b, a, finish, st);
    case 114: return pass_a_rows_launch<1, 1, 4>(g, b, a, finish, st);
    case 211: return pass_a_rows_launch<2, 1, 1>(g, b, a, finish, st);
    case 212: return pass_a_rows_launch<2, 1, 2>(g, b, a, finish, st);
    case 214: return pass_a_rows_launch<2, 1, 4>(g, b, a, finish, st);
    case 221: return pass_a_rows_launch<2, 2, 1>(g, b, a, finish, st);
    case 222: return pass_a_rows_launch<2, 2, 2>(g, b, a, finish, st);
    case 224: return pass_a_rows_launch<2, 2, 4>(g, b, a, finish, st);
    case 241: return pass_a_rows_launch<2, 4, 1>(g, b, a, finish, st);
    case 242: return pass_a_rows_launch<2, 4, 2>(g, b, a, finish, st);
    case 244: return pass_a_rows_launch<2, 4, 4>(g, b, a, finish, st);
    case 411: return pass_a_rows_launch<4, 1, 1>(g, b, a, finish, st);
    case 412: return pass_a_rows_launch<4, 1, 2>(g, b, a, finish, st);
    case 414: return pass_a_rows_launch<4, 1, 4>(g, b, a, finish, st);
    case 421: return pass_a_rows_launch<4, 2, 1>(g, b, a, finish, st);
    case 422: return pass_a_rows_launch<4, 2, 2>(g, b, a, finish, st);
    case 424: return pass_a_rows_launch<4, 2, 4>(g, b, a, finish, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_pass_u(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  if (!g.a_rows) return hipErrorInvalidValue;
  return pass_a_rows_dispatch(g, b, a, kPassRows, st);
}

hipError_t launch_pass_a(const Geometry& g, const Bufs& b, const StepArgs& a, bool finish, hipStream_t st) {
  if (g.a_rows) return pass_a_rows_dispatch(g, b, a, finish ? kPassFinish : kPassIter, st);
  if (finish) return pass_a_nbg<4, kAFinish>(g, b, a, st);
  if (pass_a_split(g)) {
    // wide factors: the row work (all columns staged) and the product (own columns only)
    const hipError_t e = launch_rows_wide(g, b, a, st);
    if (e != hipSuccess) return e;
    // 16-byte rows: the product with the next tile prefetched into registers
    if (g.vec_x && g.vec_u && (g.NBG == 4 || g.NBG == 5 || g.NBG == 7)) return launch_theta_wide(g, b, st);
    return pass_a_mbg<kATheta>(g, b, a, st);
  }
  return pass_a_mbg<kAIter>(g, b, a, st);
}

hipError_t launch_seg_theta(const Geometry& g, const Bufs& b, int64_t rows, int nseg, hipStream_t st) {
  const int C = g.theta_cols;
  hipLaunchKernelGGL((k_seg_sum<float>), dim3((C + 63) / 64, nseg), dim3(kThreads), 0, st,
                     (const float*)b.theta_part, rows, C, b.seg_theta, nseg, (const DevCtl*)b.ctl, 1);
  return hipGetLastError();
}

hipError_t launch_reduce_theta_rows(const Geometry& g, const Bufs& b, int64_t rows, int nseg, bool scaled,
                                    hipStream_t st) {
  const int C = g.theta_cols;
  hipLaunchKernelGGL((k_seg_sum<float>), dim3((C + 63) / 64, nseg), dim3(kThreads), 0, st,
                     (const float*)b.theta_part, rows, C, b.seg_theta, nseg, (const DevCtl*)b.ctl, 1);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // one-pass iteration (partials of its pass): blocks after the RT Theta blocks form
  // (W^T W) P from the r32 r32 Gram entries
  const int gb = (g.fused8 && scaled) ? (g.r32 * g.r32) / kThreads : 0;
  hipLaunchKernelGGL(k_reduce_theta, dim3(g.RT + gb), dim3(kThreads), 0, st, g, b, nseg, scaled ? 1 : 0, -1.0f);
  return hipGetLastError();
}

hipError_t launch_reduce_theta(const Geometry& g, const Bufs& b, bool fused_partials, hipStream_t st) {
  return fused_partials ? launch_reduce_theta_rows(g, b, g.GB, g.SAF, true, st)
                        : launch_reduce_theta_rows(g, b, g.GA, g.SA, false, st);
}

// a_part rows -> g.SA segment sums (the segment count k_ctl_a reads); in the one-pass
// iteration they follow its row pass, and run when that did
hipError_t launch_seg_a_rows(const Geometry& g, const Bufs& b, int64_t rows, bool finish, hipStream_t st) {
  const int C = 4 + g.r32;
  const int mode = finish ? 0 : (g.fused8 ? 2 : 1);
  hipLaunchKernelGGL((k_seg_sum<double>), dim3((C + 63) / 64, g.SA), dim3(kThreads), 0, st,
                     (const double*)b.a_part, rows, C, b.seg_a, g.SA, (const DevCtl*)b.ctl, mode);
  return hipGetLastError();
}

hipError_t launch_seg_a(const Geometry& g, const Bufs& b, bool finish, hipStream_t st) {
  // the register-resident finish runs on the pass-A grid; the generic one, and the
  // row-work launch of the split generic pass A, on GAF
  const int64_t rows = ((finish && !g.a_rows) || (!finish && pass_a_split(g))) ? g.GAF : g.GA;
  return launch_seg_a_rows(g, b, rows, finish, st);
}

hipError_t launch_seg_b(const Geometry& g, const Bufs& b, hipStream_t st) {
  const int C = 4 + g.r32;
  hipLaunchKernelGGL((k_seg_sum<double>), dim3((C + 63) / 64, g.SB), dim3(kThreads), 0, st,
                     (const double*)b.b_part, (int64_t)g.GB, C, b.seg_b, g.SB, (const DevCtl*)b.ctl, 1);
  return hipGetLastError();
}


hipError_t launch_ctl_a(const Geometry& g, const Bufs& b, const StepArgs& a, bool finish, hipStream_t st) {
  hipLaunchKernelGGL(k_ctl_a, dim3(1), dim3(kThreads), 0, st, g, b, a, finish ? 1 : 0);
  return hipGetLastError();
}

template <int CG>
static hipError_t pass_b_stream_launch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  // Theta buffers, the column-sum table, p, s, the reduction
  const size_t lds = (size_t)2 * 4 * CG * 256 * 4 + (size_t)4 * g.r32 * 8 + (size_t)2 * g.r32 * 4 + 4 * 8;
  if (lds > (160u << 10)) return hipErrorInvalidValue;
  hipError_t e = allow_lds(k_pass_b_stream<CG>, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_pass_b_stream<CG>), dim3(g.GB), dim3(kThreads), lds, st, g, b, a);
  return hipGetLastError();
}

template <int NB>
static hipError_t pass_b_nb(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  const size_t lds = g.ldsB_bytes;
  const dim3 grid(g.GB), blk(kThreads);
  const bool vec = g.vec_x && g.vec_u;
  if (lds > (64u << 10)) return hipErrorInvalidValue;  // the layout keeps pass B under 64 KiB
  if (g.theta_lds) {
    if (vec) hipLaunchKernelGGL((k_pass_b<NB, true, true>), grid, blk, lds, st, g, b, a);
    else hipLaunchKernelGGL((k_pass_b<NB, true, false>), grid, blk, lds, st, g, b, a);
  } else {
    if (vec) hipLaunchKernelGGL((k_pass_b<NB, false, true>), grid, blk, lds, st, g, b, a);
    else hipLaunchKernelGGL((k_pass_b<NB, false, false>), grid, blk, lds, st, g, b, a);
  }
  return hipGetLastError();
}

template <int NB, int NCH>
static hipError_t pass_b_res_launch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((k_pass_b_res<NB, NCH>), dim3(g.GB), dim3(kThreads), g.ldsB_bytes, st, g, b, a);
  return hipGetLastError();
}

hipError_t launch_pass_b(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  if (g.split_b) return launch_pass_b_split(g, b, a, st);
  if (g.b_res) {
    switch (g.NB * 10 + g.nch) {
      case 11: return pass_b_res_launch<1, 1>(g, b, a, st);
      case 12: return pass_b_res_launch<1, 2>(g, b, a, st);
      case 13: return pass_b_res_launch<1, 3>(g, b, a, st);
      case 14: return pass_b_res_launch<1, 4>(g, b, a, st);
      case 21: return pass_b_res_launch<2, 1>(g, b, a, st);
      case 22: return pass_b_res_launch<2, 2>(g, b, a, st);
      case 23: return pass_b_res_launch<2, 3>(g, b, a, st);
      case 24: return pass_b_res_launch<2, 4>(g, b, a, st);
      case 41: return pass_b_res_launch<4, 1>(g, b, a, st);
      case 42: return pass_b_res_launch<4, 2>(g, b, a, st);
      case 43: return pass_b_res_launch<4, 3>(g, b, a, st);
      case 44: return pass_b_res_launch<4, 4>(g, b, a, st);
      default: return hipErrorInvalidValue;
    }
  }
  if (!g.theta_lds && g.vec_x && g.vec_u) {
    // Theta streamed through LDS in chunks, columns in groups of up to four blocks
    switch (g.NB) {
      case 1: return pass_b_stream_launch<1>(g, b, a, st);
      case 2: return pass_b_stream_launch<2>(g, b, a, st);
      case 10: return pass_b_stream_launch<2>(g, b, a, st);  // five exact groups of two
      default: return pass_b_stream_launch<4>(g, b, a, st);  // groups of four blocks
    }
  }
  if (g.NB > 8) {
    // more than 256 columns, in pairs of column blocks
    if (g.NB % 2 != 0 || g.NB > kMaxR / 32) return hipErrorInvalidValue;
    const size_t lds = g.ldsB_bytes;
    if (lds > (64u << 10)) return hipErrorInvalidValue;
    const dim3 grid(g.GB), blk(kThreads);
    const bool vec = g.vec_x && g.vec_u;
    if (g.theta_lds) {
      if (vec) hipLaunchKernelGGL((k_pass_b_wide<true, true>), grid, blk, lds, st, g, b, a);
      else hipLaunchKernelGGL((k_pass_b_wide<true, false>), grid, blk, lds, st, g, b, a);
    } else {
      if (vec) hipLaunchKernelGGL((k_pass_b_wide<false, true>), grid, blk, lds, st, g, b, a);
      else hipLaunchKernelGGL((k_pass_b_wide<false, false>), grid, blk, lds, st, g, b, a);
    }
    return hipGetLastError();
  }
  switch (g.NB) {
    case 1: return pass_b_nb<1>(g, b, a, st);
    case 2: return pass_b_nb<2>(g, b, a, st);
    case 4: return pass_b_nb<4>(g, b, a, st);
    case 8: return pass_b_nb<8>(g, b, a, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_ctl_b(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_ctl_b, dim3(1), dim3(kThreads), 0, st, g, b, a);
  return hipGetLastError();
}

hipError_t launch_ctl_one(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_ctl_one, dim3(1), dim3(kThreads), 0, st, g, b, a);
  return hipGetLastError();
}

hipError_t launch_seg_onepass(const Geometry& g, const Bufs& b, hipStream_t st) {
  const int cx = (g.theta_cols + 63) / 64, ax = (4 + g.r32 + 7) / 8;
  hipLaunchKernelGGL(k_seg_onepass, dim3(cx > ax ? cx : ax, g.SAF + 2), dim3(kThreads), 0, st, g, b, g.SAF);
  return hipGetLastError();
}

hipError_t launch_seg_fused(const Geometry& g, const Bufs& b, hipStream_t st) {
  const int cx = (g.theta_cols + 63) / 64, bx = (4 + g.r32 + 63) / 64;
  hipLaunchKernelGGL(k_seg_fused, dim3(cx > bx ? cx : bx, g.SAF + g.SB), dim3(kThreads), 0, st, g, b);
  return hipGetLastError();
}

hipError_t launch_reduce_theta_fused(const Geometry& g, const Bufs& b, hipStream_t st) {
  // the Theta segments come from k_seg_fused
  hipLaunchKernelGGL(k_reduce_theta, dim3(g.RT), dim3(kThreads), 0, st, g, b, g.SAF, 1, -1.0f);
  return hipGetLastError();
}

hipError_t launch_reduce_theta_onepass(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  // blocks after the RT Theta blocks form (W^T W) P from the r32 r32 Gram entries, and s
  hipLaunchKernelGGL(k_reduce_theta, dim3(g.RT + (g.r32 * g.r32) / kThreads), dim3(kThreads), 0, st, g, b, g.SAF, 1,
                     a.gamma_f);
  return hipGetLastError();
}

hipError_t launch_onepass_begin(const Geometry& g, const Bufs& b, const StepArgs& a, bool gram_valid,
                                hipStream_t st) {
  hipLaunchKernelGGL(k_onepass_begin, dim3(1), dim3(64), 0, st, g, b, a, gram_valid ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_labels(const Geometry& g, const Bufs& b, int32_t* labels, hipStream_t st) {
  // 16 rows per workgroup and step; enough workgroups for eight per CU
  int64_t blocks = (g.n + 15) / 16;
  if (blocks > 2048) blocks = 2048;
  const dim3 grid((unsigned)blocks), blk(kThreads);
  const float* U = b.U;
  if (!g.vec_u) {
    hipLaunchKernelGGL((k_labels<false, 1, 1>), grid, blk, 0, st, g, U, labels);
  } else {
    // rows per step so that a lane has four to eight pieces in flight
    switch ((g.r + 63) / 64) {
      case 1: hipLaunchKernelGGL((k_labels<true, 1, 4>), grid, blk, 0, st, g, U, labels); break;
      case 2: hipLaunchKernelGGL((k_labels<true, 2, 4>), grid, blk, 0, st, g, U, labels); break;
      case 3: hipLaunchKernelGGL((k_labels<true, 3, 2>), grid, blk, 0, st, g, U, labels); break;
      case 4: hipLaunchKernelGGL((k_labels<true, 4, 2>), grid, blk, 0, st, g, U, labels); break;
      case 5: hipLaunchKernelGGL((k_labels<true, 5, 1>), grid, blk, 0, st, g, U, labels); break;
      case 6: hipLaunchKernelGGL((k_labels<true, 6, 1>), grid, blk, 0, st, g, U, labels); break;
      case 7: hipLaunchKernelGGL((k_labels<true, 7, 1>), grid, blk, 0, st, g, U, labels); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

}  // namespace nlr
