// Split-fp16 forms of the two products of the NLR iteration for gfx950.
//
// Every fp32 operand v of a product is written as v = (hi + lo) / s with
// hi = fp16(v s), lo = fp16(v s - hi) and s a power of two that keeps |v s| below
// 2^15; the product v w is taken as (hi_v hi_w + hi_v lo_w + lo_v hi_w) / (s_v s_w)
// on the fp16 matrix cores with fp32 accumulation.  The dropped lo_v lo_w term and
// the rounding of lo leave about 2^-22 relative error per operand (fp32: 2^-24;
// the TF32 products of the paper's GEMM, Appendix C: 2^-11).  The gfx950 fp16
// matrix core does 16x the fp32 rate, so the three products cost about a fifth
// of the fp32 matrix work.  Scales: Xhat from max |Xhat| measured at
// initialisation (|Xhat| <= ||Xhat||_2 = 1 after the spectral normalisation of
// Section 3), Theta from max |Theta| of the current iteration.
// Everything outside the products (epilogue, statistics, reductions) is the
// fp32/FP64 arithmetic of the fp32 kernels.
#include "k_common.hpp"

namespace nlr {

// ---------------------------------------------------------------------------
// Scale of Xhat: max |X| over row chunks, then one workgroup picks the power of two.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_xmax_partial(Geometry g, Bufs B) {
  __shared__ float red[4];
  const int64_t e0 = (int64_t)blockIdx.x * g.n / g.GI * g.d;
  const int64_t e1 = (int64_t)(blockIdx.x + 1) * g.n / g.GI * g.d;
  float m = 0.f;
  int64_t e = e0 + threadIdx.x;
  for (; e + 15 * kThreads < e1; e += 16 * kThreads) {  // sixteen loads in flight
    float v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = B.X[e + u * kThreads];
#pragma unroll
    for (int u = 0; u < 16; ++u) m = fmaxf(m, fabsf(v[u]));
  }
  for (; e < e1; e += kThreads) m = fmaxf(m, fabsf(B.X[e]));
  for (int k = 32; k >= 1; k >>= 1) m = fmaxf(m, shfl_xor_f(m, k));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) B.i_colsum[blockIdx.x] = (double)fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

__global__ __launch_bounds__(kThreads) void k_xmax_final(Geometry g, Bufs B) {
  __shared__ float red[4];
  float m = 0.f;
  for (int k = threadIdx.x; k < g.GI; k += kThreads) m = fmaxf(m, (float)B.i_colsum[k]);
  for (int k = 32; k >= 1; k >>= 1) m = fmaxf(m, shfl_xor_f(m, k));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) B.ctl->x_scale = f16_range_scale(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])));
}

// ---------------------------------------------------------------------------
// Pass B, split-fp16 form of the resident-tile kernel: Theta (hi/lo) resident in
// LDS as 32x32x16 A operands, Xhat rows split in registers as B operands; same
// tiles, prefetch, epilogue and statistics as the fp32 kernel.
// ---------------------------------------------------------------------------
template <int NB, int NCH>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8))) void k_pass_b_h(
    Geometry g, Bufs B, StepArgs S) {
  if (halted(B.ctl)) return;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  constexpr int KS = 2 * NCH;  // 16-feature k-steps
  f16x8* th_h = reinterpret_cast<f16x8*>(smem_raw);  // KS * NB * 64 operand vectors
  f16x8* th_l = th_h + KS * NB * 64;
  float* ps = reinterpret_cast<float*>(th_l + KS * NB * 64);  // r32
  float* ss = ps + g.r32;                                     // r32
  double* colred = reinterpret_cast<double*>(ss + g.r32);     // 4 x r32
  double* dred = colred + 4 * g.r32;                          // 8
  float* fred = reinterpret_cast<float*>(dred + 8);           // 4

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
  const float sx = B.ctl->x_scale;
  const float neg_alpha = -S.alpha_f;

  // Scale of Theta: every workgroup reduces the same values, so all agree.
  float tmax = 0.f;
  for (int e = tid; e < g.d32 * r32; e += kThreads) tmax = fmaxf(tmax, fabsf(B.theta[e]));
  for (int m = 32; m >= 1; m >>= 1) tmax = fmaxf(tmax, shfl_xor_f(tmax, m));
  if (lane == 0) fred[wave] = tmax;
  __syncthreads();
  tmax = fmaxf(fmaxf(fred[0], fred[1]), fmaxf(fred[2], fred[3]));
  const float sth = f16_range_scale(tmax);
  // acc holds sx * sth * (Xhat Theta); powers of two, so the rescale is exact
  const float two_alpha_s = two_alpha * (1.0f / sx) * (1.0f / sth);
  // A operand of k-step 2 ch + s, m-block m, lane l: Theta[32 ch + 16 (l/32) + 8 s + e][32 m + l%32],
  // split into fp16 hi/lo.  Source layout: quarter j = 2 s + e/4 of the fp32 operand layout.
  for (int idx = tid; idx < KS * NB * 64; idx += kThreads) {
    const int l = idx & 63;
    const int m = (idx >> 6) % NB;
    const int ks = (idx >> 6) / NB;
    const int ch = ks >> 1, s2 = ks & 1;
    const f32x4 v0 = *reinterpret_cast<const f32x4*>(B.theta + ((((ch * 4 + 2 * s2) * NB + m) * 64 + l) * 4));
    const f32x4 v1 = *reinterpret_cast<const f32x4*>(B.theta + ((((ch * 4 + 2 * s2 + 1) * NB + m) * 64 + l) * 4));
    const float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
    f16x8 hi, lo;
    split_f16(v, sth, hi, lo);
    th_h[idx] = hi;
    th_l[idx] = lo;
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
      // lane l's features 32 ch + 16 (l/32) + 8 s + e fill k-slots 8 (l/32) + e of k-step 2 ch + s
      f16x8 xh[2], xl[2];
      split_f16(&xv[ch][0], sx, xh[0], xl[0]);
      split_f16(&xv[ch][8], sx, xh[1], xl[1]);
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int m = 0; m < NB; ++m) {
          const f16x8 ah = th_h[((ch * 2 + s2) * NB + m) * 64 + lane];
          const f16x8 al = th_l[((ch * 2 + s2) * NB + m) * 64 + lane];
          acc[m] = mfma32x32x16h(ah, xl[s2], acc[m]);
          acc[m] = mfma32x32x16h(al, xh[s2], acc[m]);
          acc[m] = mfma32x32x16h(ah, xh[s2], acc[m]);
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
          float t = fmaf(two_alpha_s, acc[m][4 * qd + e], uu);
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


template <int NB, int NCH>
static hipError_t pass_b_h_launch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  const int lds = 2 * NCH * NB * 64 * 16 * 2 + 2 * g.r32 * 4 + (4 * g.r32 + 8) * 8 + 16;
  if (lds > (64 << 10)) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pass_b_h<NB, NCH>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((k_pass_b_h<NB, NCH>), dim3(g.GB), dim3(kThreads), lds, st, g, b, a);
  return hipGetLastError();
}

hipError_t launch_pass_b_split(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  switch (g.NB * 10 + g.nch) {
    case 11: return pass_b_h_launch<1, 1>(g, b, a, st);
    case 12: return pass_b_h_launch<1, 2>(g, b, a, st);
    case 13: return pass_b_h_launch<1, 3>(g, b, a, st);
    case 14: return pass_b_h_launch<1, 4>(g, b, a, st);
    case 21: return pass_b_h_launch<2, 1>(g, b, a, st);
    case 22: return pass_b_h_launch<2, 2>(g, b, a, st);
    case 23: return pass_b_h_launch<2, 3>(g, b, a, st);
    case 24: return pass_b_h_launch<2, 4>(g, b, a, st);
    default: return hipErrorInvalidValue;
  }
}

// Xhat in place into split form (the single-pass iteration's only reader of X):
// each 16-byte unit of 4 features becomes their 4 hi halves then their 4 lo halves
// of x * x_scale, the same split the products would otherwise form every iteration.
__global__ __launch_bounds__(kThreads) void k_split_x(Bufs B, int64_t units) {
  const float s = B.ctl->x_scale;
  for (int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x; u < units; u += (int64_t)gridDim.x * kThreads) {
    f32x4* p = reinterpret_cast<f32x4*>(B.X) + u;
    const f32x4 v = *p;
    const float x[4] = {v.x, v.y, v.z, v.w};
    typedef _Float16 f16x4s __attribute__((ext_vector_type(4)));
    f16x4s hi, lo;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float t = x[e] * s;
      const _Float16 h = (_Float16)t;
      hi[e] = h;
      lo[e] = (_Float16)(t - (float)h);
    }
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    const f32x2 hb = __builtin_bit_cast(f32x2, hi);
    const f32x2 lb = __builtin_bit_cast(f32x2, lo);
    const f32x4 o = {hb.x, hb.y, lb.x, lb.y};
    *p = o;
  }
}

hipError_t launch_split_x(const Geometry& g, const Bufs& b, hipStream_t st) {
  const int64_t units = g.n * (int64_t)g.d / 4;  // d % 4 == 0
  hipLaunchKernelGGL(k_split_x, dim3(4096), dim3(kThreads), 0, st, b, units);
  return hipGetLastError();
}

hipError_t launch_xscale(const Geometry& g, const Bufs& b, hipStream_t st) {
  hipLaunchKernelGGL(k_xmax_partial, dim3(g.GI), dim3(kThreads), 0, st, g, b);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_xmax_final, dim3(1), dim3(kThreads), 0, st, g, b);
  return hipGetLastError();
}

}  // namespace nlr
