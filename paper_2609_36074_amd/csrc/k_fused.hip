// Fused pass B of the single-Xhat-pass iteration (gfx950).
//
// The two-pass iteration reads Xhat twice: pass A for Theta_t = Xhat^T U_t and
// pass B for Xhat Theta_t.  Because U_{t+1} = c_{t+1} W_{t+1} (Algorithm 1, the
// normalising rescale) and c_{t+1} is a scalar,
//     Theta_{t+1} = Xhat^T U_{t+1} = c_{t+1} (Xhat^T W_{t+1}),
// so the partial sums of Xhat^T W_{t+1} can be formed inside pass B while the
// Xhat rows and the freshly computed W rows are still on chip, and scaled by
// c_{t+1} once it is known.  The statistics of the movement identity are formed
// before W overwrites U for the same reason (eq. fused-statistics).  What pass A
// did besides Theta -- the per-row q = u.p - 1, the gated dual step, ybar, s =
// U^T ybar, ||q||^2, ytilde^T q -- needs only U and ytilde, and is left to a
// light row pass (k_pass_a_rows in kPassRows mode).  Xhat is read once per
// iteration: 4(nd + 3nr + 2n) bytes instead of 4(2nd + 3nr + 2n).
//
// Per workgroup (4 waves, one workgroup per compute unit, persistent over
// 128-row tiles in grid-stride order), per wave and 32-row slab:
//   phase 1  G = Xhat Theta_t on the matrix cores (Theta_t resident in LDS), the
//            epilogue of eq. (entrywise-fusion), FP64 a, b, h and column sums of
//            W, W stored over U (as the resident pass B);
//   phase 2  the slab of Xhat (written to LDS during phase 1) and of W (written
//            in the epilogue) are multiplied as Xhat_slab^T W_slab into per-wave
//            accumulators holding all of the d x r partial.
// At the end the four waves' partials are added in a fixed order and written as
// this workgroup's partial; a fixed-order reduction and the scale c_{t+1} give
// Theta_{t+1}.
// SPLIT: both products use the two-term fp16 split of k_split.hip; otherwise
// fp32 matrix cores (32x32x2 for phase 1, 16x16x4 for phase 2).
#include <type_traits>

#include "k_common.hpp"

namespace nlr {

// Power-of-two scale of W in the split phase 2: |w| < 32 (= 4 sqrt(K) at the
// largest split-supported K = 64; a normalised factor has |u| <= sqrt(K)).
constexpr float kWScale = 1024.0f;

typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef __fp16 h16x4 __attribute__((__vector_size__(4 * sizeof(__fp16))));

// Transposing LDS read (gfx950 ds_read_b64_tr_b16).  Within each 16-lane group,
// source lane s points at 4 consecutive halves; lane i receives element i%4 of
// the chunks of source lanes i/4, 4 + i/4, 8 + i/4, 12 + i/4 (in that order).
__device__ __forceinline__ f16x4 lds_read_tr16(const _Float16* p) {
  h16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4f16(
      (__attribute__((address_space(3))) h16x4*)(p));
  f16x4 o;
  o[0] = (_Float16)v[0];
  o[1] = (_Float16)v[1];
  o[2] = (_Float16)v[2];
  o[3] = (_Float16)v[3];
  return o;
}

// Two stored 4-feature units of split Xhat (8 dwords: hi, hi, lo, lo, hi, hi, lo, lo)
// as the hi and lo operands of 8 features.
__device__ __forceinline__ void unpack_split(const float* v, f16x8& hi, f16x8& lo) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 h = {__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[4]), __float_as_uint(v[5])};
  const u32x4 l = {__float_as_uint(v[2]), __float_as_uint(v[3]), __float_as_uint(v[6]), __float_as_uint(v[7])};
  hi = __builtin_bit_cast(f16x8, h);
  lo = __builtin_bit_cast(f16x8, l);
}

// 32x32x16 operand with k = row from a row-major fp16 tile T (row stride ts):
// lane l gets T[r0 + 8 (l/32) + e][c0 + l%32], e = 0..7.
__device__ __forceinline__ f16x8 tile_operand_rows(const _Float16* T, int ts, int r0, int c0, int lane) {
  const int g = lane >> 4, s = lane & 15;
  const _Float16* p = T + (r0 + 8 * (g >> 1) + (s >> 2)) * ts + c0 + 16 * (g & 1) + 4 * (s & 3);
  const f16x4 a = lds_read_tr16(p);
  const f16x4 b = lds_read_tr16(p + 4 * ts);
  f16x8 o;
  o[0] = a[0]; o[1] = a[1]; o[2] = a[2]; o[3] = a[3];
  o[4] = b[0]; o[5] = b[1]; o[6] = b[2]; o[7] = b[3];
  return o;
}

// Bytes of dynamic LDS the fused pass B needs.
constexpr int fused_lds_bytes(int NB, int NCH, bool split, bool uflat) {
  const int d32 = 32 * NCH, r32 = 32 * NB;
  const int xs = split ? d32 + 8 : d32 + 4, ws = split ? r32 + 8 : r32 + 4, esz = split ? 2 : 4;
  const int tile = (split ? 2 : 1) * 32 * (xs + ws) * esz + (uflat ? (32 * r32 + 4) * 4 : 0);
  const int head = d32 * r32 * 4 + 2 * r32 * 4 + (4 * r32 + 8) * 8 + 16;
  const int tiles = 4 * tile > 2 * d32 * r32 * 4 ? 4 * tile : 2 * d32 * r32 * 4;
  return head + tiles;
}

// UFLAT (rows of U not 16-byte aligned, r % 4 != 0): each wave moves its 32-row
// slab of U (32 r contiguous floats, 16-byte aligned because the slab starts at a
// multiple of 32 rows) with whole-slab vector loads and stores through LDS.
// Waves per SIMD: two for the small shapes (registers allow it, and a second
// wave is what hides a tile's memory latency), one when the d x r partial takes
// 128 accumulator registers.
template <int NB, int NCH>
constexpr int fused_waves_per_simd() { return (NB == 1 && NCH <= 2) ? 2 : 1; }

template <int NB, int NCH, bool SPLIT, bool UFLAT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(fused_waves_per_simd<NB, NCH>(),
                                                                            fused_waves_per_simd<NB, NCH>()))) void k_pass_bf(
    Geometry g, Bufs B, StepArgs S) {
  if (halted(B.ctl)) return;
  constexpr int KS = 2 * NCH;                      // 16-feature k-steps (split phase 1)
  constexpr int D32 = 32 * NCH, R32 = 32 * NB;
  constexpr int XS = SPLIT ? D32 + 8 : D32 + 4;    // tile row strides (halves / floats)
  constexpr int WS = SPLIT ? R32 + 8 : R32 + 4;
  constexpr int ESZ = SPLIT ? 2 : 4;
  constexpr int SLAB_BYTES = (SPLIT ? 2 : 1) * 32 * (XS + WS) * ESZ;
  constexpr int TILE_BYTES = SLAB_BYTES + (UFLAT ? (32 * R32 + 4) * 4 : 0);  // per wave
  constexpr int NCU = UFLAT ? R32 / 8 : 1;  // 16-byte chunks of a U slab per lane (8 r <= 64 NCU)
  extern __shared__ __align__(16) unsigned char smem_raw[];
  unsigned char* th_raw = smem_raw;                                    // D32 * R32 * 4 bytes
  float* ps = reinterpret_cast<float*>(smem_raw + D32 * R32 * 4);     // R32
  float* ss = ps + R32;                                                // R32
  double* colred = reinterpret_cast<double*>(ss + R32);                // 4 x R32
  double* dred = colred + 4 * R32;                                     // 8
  float* fred = reinterpret_cast<float*>(dred + 8);                    // 4
  unsigned char* tiles = reinterpret_cast<unsigned char*>(fred + 4);   // 4 x TILE_BYTES

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5;
  const int li = lane & 31;
  const int64_t n = g.n;
  const int d = g.d, r = g.r;
  const float cf = B.ctl->c_f;
  const float gam = S.gamma_f;
  const float two_alpha = S.two_alpha_f;
  const float neg_alpha = -S.alpha_f;
  const float sx = SPLIT ? B.ctl->x_scale : 1.0f;

  unsigned char* mytile = tiles + wave * TILE_BYTES;
  // SPLIT: Xh, Xl (32 x XS halves), Wh, Wl (32 x WS halves); else Xs (32 x XS), Ws (32 x WS) floats
  _Float16* xh_t = reinterpret_cast<_Float16*>(mytile);
  _Float16* xl_t = xh_t + 32 * XS;
  _Float16* wh_t = xl_t + 32 * XS;
  _Float16* wl_t = wh_t + 32 * WS;
  float* xs_t = reinterpret_cast<float*>(mytile);
  float* ws_t = xs_t + 32 * XS;
  float* uslab = reinterpret_cast<float*>(mytile + SLAB_BYTES);  // UFLAT: 32 r floats + 4 dump
  float* udump = uslab + 32 * R32;

  // ---- Theta_t operand ----
  float two_alpha_s = two_alpha;
  if constexpr (SPLIT) {
    f16x8* th_h = reinterpret_cast<f16x8*>(th_raw);
    f16x8* th_l = th_h + KS * NB * 64;
    float tmax = 0.f;
    for (int e = tid; e < D32 * R32; e += kThreads) tmax = fmaxf(tmax, fabsf(B.theta[e]));
    for (int m = 32; m >= 1; m >>= 1) tmax = fmaxf(tmax, shfl_xor_f(tmax, m));
    if (lane == 0) fred[wave] = tmax;
    __syncthreads();
    tmax = fmaxf(fmaxf(fred[0], fred[1]), fmaxf(fred[2], fred[3]));
    const float sth = f16_range_scale(tmax);
    two_alpha_s = two_alpha * (1.0f / sx) * (1.0f / sth);
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
  } else {
    const f32x4* src = reinterpret_cast<const f32x4*>(B.theta);
    f32x4* dst = reinterpret_cast<f32x4*>(th_raw);
    for (int v = tid; v < (D32 * R32) / 4; v += kThreads) dst[v] = src[v];
  }
  for (int c = tid; c < R32; c += kThreads) {
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

  // phase-2 accumulators: all of the d x r partial of this wave
  constexpr int P2F = SPLIT ? NCH : 2 * NCH;   // feature blocks (32 or 16 wide)
  constexpr int P2C = SPLIT ? NB : 2 * NB;     // column blocks
  typedef typename std::conditional<SPLIT, f32x16, f32x4v>::type acc2_t;
  constexpr int AV = SPLIT ? 16 : 4;
  acc2_t acc2[P2F][P2C];
#pragma unroll
  for (int a = 0; a < P2F; ++a)
#pragma unroll
    for (int b = 0; b < P2C; ++b)
#pragma unroll
      for (int v = 0; v < AV; ++v) acc2[a][b][v] = 0.f;

  const int64_t T = g.tilesB;
  const int64_t step = g.GB;

  float xv[NCH][16];
  auto load_x = [&](int64_t st, int ch) {
    const int64_t pt = st * kTPB + wave * 32 + li;
    const bool ok = (st < T) && (pt < n);
    const float* xrow = B.X + (ok ? pt : 0) * (int64_t)d;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int f = ch * 32 + h * 16 + 4 * q;
      // raw values: features >= d meet zero rows of Theta_t (and their rows of the
      // new partial are discarded by the reduction); rows >= n have w = 0
      const f32x4 t = *reinterpret_cast<const f32x4*>(xrow + (f < d ? f : 0));
      xv[ch][4 * q + 0] = t.x;
      xv[ch][4 * q + 1] = t.y;
      xv[ch][4 * q + 2] = t.z;
      xv[ch][4 * q + 3] = t.w;
    }
  };
  f32x4 unext[NB][4];
  f32x4 ufl[NCU];
  float ynext;
  // valid floats of the U slab of tile st (32 r for every slab but the last)
  auto slab_valid = [&](int64_t st) -> int {
    const int64_t row0 = st * kTPB + wave * 32;
    if (st >= T || row0 >= n) return 0;
    const int64_t rows = n - row0 < 32 ? n - row0 : 32;
    return (int)rows * r;
  };
  auto load_u = [&](int64_t st) {
    const int64_t pt = st * kTPB + wave * 32 + li;
    const bool ok = (st < T) && (pt < n);
    if constexpr (UFLAT) {
      const int nval = slab_valid(st);
      const float* base = B.U + (nval > 0 ? (st * kTPB + wave * 32) * (int64_t)r : 0);
      if (nval == 32 * r) {
#pragma unroll
        for (int i = 0; i < NCU; ++i) {
          const int j = lane + 64 * i;
          ufl[i] = *reinterpret_cast<const f32x4*>(base + 4 * (j < 8 * r ? j : 0));
        }
      } else {
#pragma unroll
        for (int i = 0; i < NCU; ++i) {
          const int j = lane + 64 * i;
          f32x4 t = {0.f, 0.f, 0.f, 0.f};
          if (4 * j + 0 < nval) t.x = base[4 * j + 0];
          if (4 * j + 1 < nval) t.y = base[4 * j + 1];
          if (4 * j + 2 < nval) t.z = base[4 * j + 2];
          if (4 * j + 3 < nval) t.w = base[4 * j + 3];
          ufl[i] = t;
        }
      }
    } else {
      const float* ur = B.U + (ok ? pt : 0) * (int64_t)r;
#pragma unroll
      for (int m = 0; m < NB; ++m)
#pragma unroll
        for (int qd = 0; qd < 4; ++qd) {
          const int c = 32 * m + 8 * qd + 4 * h;
          unext[m][qd] = *reinterpret_cast<const f32x4*>(ur + (c < r ? c : 0));
        }
    }
    ynext = B.y[ok ? pt : 0];
  };
  const int64_t st0 = blockIdx.x;
  __builtin_amdgcn_sched_barrier(0);
  load_u(st0);
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    __builtin_amdgcn_sched_barrier(0);
    load_x(st0, ch);
  }
  __builtin_amdgcn_sched_barrier(0);

  for (int64_t st = st0; st < T; st += step) {
    __builtin_amdgcn_sched_barrier(0);
    const int64_t pt = st * kTPB + wave * 32 + li;
    const bool vpt = pt < n;
    float* urow = B.U + (vpt ? pt : 0) * (int64_t)r;
    f32x4 uraw[NB][4];
    f32x4 ucur[NCU];
    if constexpr (UFLAT) {
#pragma unroll
      for (int i = 0; i < NCU; ++i) ucur[i] = ufl[i];
    } else {
#pragma unroll
      for (int m = 0; m < NB; ++m)
#pragma unroll
        for (int qd = 0; qd < 4; ++qd) uraw[m][qd] = unext[m][qd];
    }
    const float yraw = ynext;
    __builtin_amdgcn_sched_barrier(0);
    load_u(st + step);  // the next tile's factor rows: a whole tile of lead time
    __builtin_amdgcn_sched_barrier(0);

    // ---- phase 1: G = Xhat_slab Theta_t ----
    f32x16 acc[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      if constexpr (SPLIT) {
        const f16x8* th_h = reinterpret_cast<const f16x8*>(th_raw);
        const f16x8* th_l = th_h + KS * NB * 64;
        // Xhat is stored split since initialisation: the 16 bytes of features 4q..4q+3 hold
        // their four hi halves, then their four lo halves
        f16x8 xh[2], xl[2];
        unpack_split(&xv[ch][0], xh[0], xl[0]);
        unpack_split(&xv[ch][8], xh[1], xl[1]);
        // the slab for phase 2: row li, features 32 ch + 16 h + [0, 16)
        _Float16* xrh = xh_t + li * XS + 32 * ch + 16 * h;
        _Float16* xrl = xl_t + li * XS + 32 * ch + 16 * h;
        *reinterpret_cast<f16x8*>(xrh) = xh[0];
        *reinterpret_cast<f16x8*>(xrh + 8) = xh[1];
        *reinterpret_cast<f16x8*>(xrl) = xl[0];
        *reinterpret_cast<f16x8*>(xrl + 8) = xl[1];
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
      } else {
        const float* th_s = reinterpret_cast<const float*>(th_raw);
        float* xr = xs_t + li * XS + 32 * ch + 16 * h;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x4 o = {xv[ch][4 * q + 0], xv[ch][4 * q + 1], xv[ch][4 * q + 2], xv[ch][4 * q + 3]};
          *reinterpret_cast<f32x4*>(xr + 4 * q) = o;
        }
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
      }
      __builtin_amdgcn_sched_barrier(0);
      load_x(st + step, ch);  // this chunk of the next tile
      __builtin_amdgcn_sched_barrier(0);
    }

    // ---- epilogue (eq. entrywise-fusion) ----
    int lds_off = 0;  // opaque zero offset: keeps the reads in LDS address space
    asm volatile("" : "+v"(lds_off));
    const float* psl = ps + lds_off;
    const float* ssl = ss + lds_off;
    float u[NB][16];
    if constexpr (UFLAT) {
      // the slab into LDS as loaded, then each lane picks its row's columns
#pragma unroll
      for (int i = 0; i < NCU; ++i) *reinterpret_cast<f32x4*>(uslab + 4 * (lane + 64 * i)) = ucur[i];
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int m = 0; m < NB; ++m)
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const int c = 32 * m + 8 * (k >> 2) + 4 * h + (k & 3);
          const float v = uslab[li * r + (c < r ? c : 0)];
          u[m][k] = (vpt && c < r) ? v * cf : 0.f;
        }
      __builtin_amdgcn_wave_barrier();
    } else {
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
        f32x4 o = {wv[4 * qd + 0], wv[4 * qd + 1], wv[4 * qd + 2], wv[4 * qd + 3]};
        if constexpr (UFLAT) {
          // W over the slab's U (every lane has read its u values above); columns >= r to a dump word
#pragma unroll
          for (int e = 0; e < 4; ++e) *((c + e < r) ? (uslab + li * r + c + e) : udump) = wv[4 * qd + e];
        } else {
          // unconditional store (invalid lanes write the dump slot): no branch around it
          float* dst = (vpt && c < r) ? (urow + c) : B.dump;
          *reinterpret_cast<f32x4*>(dst) = o;
        }
        // the slab of W for phase 2: row li, columns c .. c+3
        if constexpr (SPLIT) {
          f16x4 hi, lo;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float t = wv[4 * qd + e] * kWScale;
            const _Float16 hh = (_Float16)t;
            hi[e] = hh;
            lo[e] = (_Float16)(t - (float)hh);
          }
          *reinterpret_cast<f16x4*>(wh_t + li * WS + c) = hi;
          *reinterpret_cast<f16x4*>(wl_t + li * WS + c) = lo;
        } else {
          *reinterpret_cast<f32x4*>(ws_t + li * WS + c) = o;
        }
      }
      reduce_scatter<16, 16>(wv, li);
      colacc[m] += (double)wv[0];
    }
    if constexpr (UFLAT) {
      // the slab of W back to HBM as whole 16-byte chunks
      __builtin_amdgcn_wave_barrier();
      const int nval = slab_valid(st);
      float* base = B.U + (nval > 0 ? (st * kTPB + wave * 32) * (int64_t)r : 0);
      if (nval == 32 * r) {
#pragma unroll
        for (int i = 0; i < NCU; ++i) {
          const int j = lane + 64 * i;
          const f32x4 v = *reinterpret_cast<const f32x4*>(uslab + 4 * j);
          float* dst = (j < 8 * r) ? (base + 4 * j) : B.dump;
          *reinterpret_cast<f32x4*>(dst) = v;
        }
      } else {
#pragma unroll
        for (int i = 0; i < NCU; ++i) {
          const int j = lane + 64 * i;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (4 * j + e < nval) base[4 * j + e] = uslab[4 * j + e];
        }
      }
      __builtin_amdgcn_wave_barrier();
    }

    // ---- phase 2: partial += Xhat_slab^T W_slab (this wave's 32 rows) ----
    if constexpr (SPLIT) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        f16x8 wbh[NB], wbl[NB];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          wbh[cb] = tile_operand_rows(wh_t, WS, 16 * kk, 32 * cb, lane);
          wbl[cb] = tile_operand_rows(wl_t, WS, 16 * kk, 32 * cb, lane);
        }
#pragma unroll
        for (int fb = 0; fb < NCH; ++fb) {
          const f16x8 xah = tile_operand_rows(xh_t, XS, 16 * kk, 32 * fb, lane);
          const f16x8 xal = tile_operand_rows(xl_t, XS, 16 * kk, 32 * fb, lane);
#pragma unroll
          for (int cb = 0; cb < NB; ++cb) {
            acc2[fb][cb] = mfma32x32x16h(xah, wbl[cb], acc2[fb][cb]);
            acc2[fb][cb] = mfma32x32x16h(xal, wbh[cb], acc2[fb][cb]);
            acc2[fb][cb] = mfma32x32x16h(xah, wbh[cb], acc2[fb][cb]);
          }
        }
      }
    } else {
      const int rg = lane >> 4, ci = lane & 15;
#pragma unroll 2
      for (int kk = 0; kk < 8; ++kk) {
        const int row = 4 * kk + rg;
        float wb[2 * NB];
#pragma unroll
        for (int cb = 0; cb < 2 * NB; ++cb) wb[cb] = ws_t[row * WS + 16 * cb + ci];
#pragma unroll
        for (int fb = 0; fb < 2 * NCH; ++fb) {
          const float xa = xs_t[row * XS + 16 * fb + ci];
#pragma unroll
          for (int cb = 0; cb < 2 * NB; ++cb) acc2[fb][cb] = mfma16x16x4(xa, wb[cb], acc2[fb][cb]);
        }
      }
    }
  }

  // ---- statistics of this workgroup ----
  for (int c = tid; c < 4 * R32; c += kThreads) colred[c] = 0.0;
  __syncthreads();
#pragma unroll
  for (int m = 0; m < NB; ++m) {
    const double v = colacc[m] + shfl_xor_d(colacc[m], 1);
    if ((li & 1) == 0) {
      const int col = 32 * m + 8 * (base >> 2) + 4 * h + (base & 3);
      colred[wave * R32 + col] = v;
    }
  }
  __syncthreads();
  double* out = B.b_part + (int64_t)blockIdx.x * (4 + R32);
  for (int c = tid; c < R32; c += kThreads)
    out[4 + c] = ((colred[c] + colred[R32 + c]) + colred[2 * R32 + c]) + colred[3 * R32 + c];
  const double ta = block_sum_d(sa, dred);
  const double tb2 = block_sum_d(sb, dred);
  const double th = block_sum_d(sh, dred);
  if (tid == 0) {
    out[0] = ta;
    out[1] = tb2;
    out[2] = th;
    out[3] = 0.0;
  }

  // ---- partial of Xhat^T W_{t+1}: ((wave0 + wave2) + (wave1 + wave3)) in [f][c] order ----
  float* comb = reinterpret_cast<float*>(tiles);  // 2 x D32 x R32 (the slabs are no longer needed)
  const float unscale = SPLIT ? (1.0f / sx) * (1.0f / kWScale) : 1.0f;
  __syncthreads();
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    if ((wave >> 1) == pass) {
      float* dst = comb + (wave & 1) * (D32 * R32);
#pragma unroll
      for (int a = 0; a < P2F; ++a)
#pragma unroll
        for (int b = 0; b < P2C; ++b)
#pragma unroll
          for (int v = 0; v < AV; ++v) {
            int f, c;
            if constexpr (SPLIT) {
              f = 32 * a + 8 * (v >> 2) + 4 * h + (v & 3);
              c = 32 * b + li;
            } else {
              f = 16 * a + 4 * (lane >> 4) + v;
              c = 16 * b + (lane & 15);
            }
            const float val = acc2[a][b][v] * unscale;
            if (pass == 0) dst[f * R32 + c] = val;
            else dst[f * R32 + c] = dst[f * R32 + c] + val;
          }
    }
    __syncthreads();
  }
  float* part = B.theta_part + (int64_t)blockIdx.x * D32 * R32;
  for (int e = tid; e < D32 * R32; e += kThreads) part[e] = comb[e] + comb[D32 * R32 + e];
}

template <int NB, int NCH, bool SPLIT, bool UFLAT>
static hipError_t pass_bf_launch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  constexpr int lds = fused_lds_bytes(NB, NCH, SPLIT, UFLAT);
  if (lds > kMaxFusedLds) return hipErrorInvalidValue;
  if (lds > (64 << 10)) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pass_bf<NB, NCH, SPLIT, UFLAT>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((k_pass_bf<NB, NCH, SPLIT, UFLAT>), dim3(g.GB), dim3(kThreads), lds, st, g, b, a);
  return hipGetLastError();
}

template <bool SPLIT, bool UFLAT>
static hipError_t pass_bf_dispatch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  switch (g.NB * 10 + g.nch) {
    case 11: return pass_bf_launch<1, 1, SPLIT, UFLAT>(g, b, a, st);
    case 12: return pass_bf_launch<1, 2, SPLIT, UFLAT>(g, b, a, st);
    case 13: return pass_bf_launch<1, 3, SPLIT, UFLAT>(g, b, a, st);
    case 14: return pass_bf_launch<1, 4, SPLIT, UFLAT>(g, b, a, st);
    case 21: return pass_bf_launch<2, 1, SPLIT, UFLAT>(g, b, a, st);
    case 22: return pass_bf_launch<2, 2, SPLIT, UFLAT>(g, b, a, st);
    case 23: return pass_bf_launch<2, 3, SPLIT, UFLAT>(g, b, a, st);
    case 24: return pass_bf_launch<2, 4, SPLIT, UFLAT>(g, b, a, st);
    default: return hipErrorInvalidValue;
  }
}

int fused_lds_need(int NB, int nch, bool split, bool uflat) { return fused_lds_bytes(NB, nch, split, uflat); }

hipError_t launch_pass_bf(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  if (g.uflat) return g.split_b ? pass_bf_dispatch<true, true>(g, b, a, st) : pass_bf_dispatch<false, true>(g, b, a, st);
  return g.split_b ? pass_bf_dispatch<true, false>(g, b, a, st) : pass_bf_dispatch<false, false>(g, b, a, st);
}

}  // namespace nlr
