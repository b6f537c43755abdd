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
// Theta_{t+1}.  Split shapes with 97..128 features and 33..64 columns run the
// one-pass iteration kernel k_pass_bf8 further below instead.
// SPLIT: both products use the two-term fp16 split of k_split.hip; otherwise
// fp32 matrix cores (32x32x2 for phase 1, 16x16x4 for phase 2).
#include <type_traits>

#include "k_common.hpp"

namespace nlr {

// Power-of-two scale of W in the split second product (and the one-pass kernel's
// W^T W): w 2^10 stays a finite fp16 for w <= 65504 / 2^10 ~ 64.  A normalised factor
// has |u| <= sqrt(K) <= 8 at the largest split-supported K = 64, and a step within
// the Prop. 1 bound moves an entry by less than that; a larger step size or dual can
// exceed it.  Each workgroup reports whether its W did (column 3 of its statistics
// row: 1.0 if so), and the control kernel then stops the iteration with a range
// error before the inf/NaN operands reach Theta or s.
constexpr float kWScale = 1024.0f;
constexpr float kWMax = 65504.0f / kWScale;

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

// X2 (fp32 products, d % 4 == 2): rows of Xhat are 8-byte aligned only and load as 8-byte pieces.
template <int NB, int NCH, bool SPLIT, bool UFLAT, bool X2>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(fused_waves_per_simd<NB, NCH>(),
                                                                            fused_waves_per_simd<NB, NCH>()))) void k_pass_bf(
    Geometry g, Bufs B, StepArgs S) {
  static_assert(!(SPLIT && X2), "the split Xhat needs 16-byte units of 4 features");
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
  float wmx = 0.f;  // SPLIT: largest w of this lane (the fp16 range of the W operand)
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
      if constexpr (X2) {
        typedef float f32x2 __attribute__((ext_vector_type(2)));
        const f32x2 t0 = *reinterpret_cast<const f32x2*>(xrow + (f < d ? f : 0));
        const f32x2 t1 = *reinterpret_cast<const f32x2*>(xrow + (f + 2 < d ? f + 2 : 0));
        xv[ch][4 * q + 0] = t0.x;
        xv[ch][4 * q + 1] = t0.y;
        xv[ch][4 * q + 2] = t1.x;
        xv[ch][4 * q + 3] = t1.y;
      } else {
        const f32x4 t = *reinterpret_cast<const f32x4*>(xrow + (f < d ? f : 0));
        xv[ch][4 * q + 0] = t.x;
        xv[ch][4 * q + 1] = t.y;
        xv[ch][4 * q + 2] = t.z;
        xv[ch][4 * q + 3] = t.w;
      }
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
          if constexpr (SPLIT) wmx = fmaxf(wmx, w);
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
  // 1.0 when some w of this workgroup left the range of the split W operand (w != w: NaN)
  const double over = block_sum_d((wmx > kWMax || wmx != wmx) ? 1.0 : 0.0, dred);
  if (tid == 0) {
    out[0] = ta;
    out[1] = tb2;
    out[2] = th;
    out[3] = over > 0.0 ? 1.0 : 0.0;
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
  float* part = B.theta_part + (int64_t)blockIdx.x * g.theta_cols;
  for (int e = tid; e < D32 * R32; e += kThreads) part[e] = comb[e] + comb[D32 * R32 + e];
}

// ===========================================================================
// One-pass iteration kernel: the eight-wave form of the split fused pass B, which
// also does the iteration's row work (97..128 features, 33..64 columns, 16-byte
// aligned rows, r % 4 == 0).
//
// The form above keeps the whole d x r partial of Xhat^T W in every wave, which
// leaves room for one wave per SIMD only.  Here one 512-thread workgroup per
// compute unit walks 128-row tiles; wave w owns the 16-row slab 16w .. 16w + 15
// of a tile for the first product (16x16x32 fp16 matrix cores: lane l holds row
// l % 16 and, of each 16-column block, the columns 4 (l / 16) .. + 3), the row
// work and the epilogue, and the second product is shared out by 32 x 32 blocks
// of the result: wave w owns the features 32 (w % 4) .. + 31 and the columns
// 32 (w / 4) .. + 31 of the partial over all 128 rows of the tile, reading the
// split Xhat and W tiles that the slab owners wrote to LDS (one workgroup
// barrier before, one after).  The rows of the next tile are requested as soon
// as a tile has consumed its own.
//
// Row work (the end of the previous iteration): q = u.p - 1 in FP64, the pending
// gated dual step (ytilde stored), ybar, ||q||^2 and ytilde^T q -- as the row
// pass does, so that the row pass is not needed.  Its s = U^T ybar is instead
// formed (by k_reduce_theta after the pass, or by k_onepass_begin at the start of
// a host call) from terms this kernel accumulates while W is on chip: the
// column sums of W and of W ytilde (FP64 across tiles) and the Gram W^T W (a
// third product on the matrix cores, from the W tile; wave w adds the block
// (rows 32 (w % 2) .., columns 32 (w / 4) ..) of the tile's row half w / 2 % 2).
// W is written over the factor in place.  The stopping rule of the previous
// iteration needs the residual rho of the current factor, which the row work
// computes; when that rule can fire at all (movement below min(eps_d, eps_c),
// t >= T_min: known before the pass), the row pass runs first and decides it, and
// this kernel then skips the dual step (rows_first).  W leaves through LDS: each
// wave stages its slab's rows, packed as in U, in its own rows of the W tile and
// stores them as whole contiguous 1 KiB pieces before the same rows take the
// split of W.
// ===========================================================================
namespace bf8 {

constexpr int kThreads8 = 512;
constexpr int kRows = 128;  // rows per tile: 8 waves x 16
static_assert(kRows == kTPB, "the fused pass B tiles are kTPB rows");

// Tiles in LDS: row R of a tile is a run of 16-byte units (four features or four
// columns: their fp16 hi halves, then their lo halves, as Xhat is stored).  Unit u
// of row R sits in slot u ^ swz(R), and on odd rows its two 8-byte halves are
// exchanged.  A transposing read (32 lanes: rows R0 .. R0 + 3, eight consecutive
// units, one half) then touches 64 distinct 4-byte banks.  The unit writes (two
// 8-byte writes; gfx950 serves those with conflicts whenever lanes whose indices
// differ modulo 16 share a bank) are not conflict-free, but are off the critical
// path: one 16-byte write per unit with the halves exchanged in registers is not
// faster.
__device__ __forceinline__ int swz(int R) { return (R ^ ((R & 2) << 2)) & 15; }

template <int NB, int NCH>
struct Shape {
  static constexpr int CB16 = 2 * NB;                     // 16-column blocks
  static constexpr int R32 = 32 * NB, D32 = 32 * NCH;
  static constexpr int XU = 8 * NCH > 16 ? 8 * NCH : 16;  // units per Xhat tile row
  static constexpr int WU = 8 * NB > 16 ? 8 * NB : 16;    // units per W tile row
  static constexpr int XRS = 16 * XU, WRS = 16 * WU;      // tile row bytes
  static constexpr int RS2 = 8 / (NCH * NB);              // row splits of the second product
  static constexpr int KPW = 8 / RS2;                     // its 16-row steps per wave
  static constexpr int TH = NCH * CB16 * 64 * 16;         // bytes of one plane of the Theta operand
  static constexpr int OFF_X = 2 * TH;
  static constexpr int OFF_W = OFF_X + kRows * XRS;
  static constexpr int OFF_P = OFF_W + kRows * WRS;      // R32 doubles: p (the row work's FP64 dot)
  static constexpr int OFF_S = OFF_P + R32 * 8;           // 2 x R32 floats: -alpha p, -alpha s
  static constexpr int OFF_COL = OFF_S + 2 * R32 * 4;     // 8 x R32 doubles: column sums of W
  static constexpr int OFF_COLY = OFF_COL + 8 * R32 * 8;  // 8 x R32 doubles: W^T ytilde
  static constexpr int OFF_D = OFF_COLY + 8 * R32 * 8;    // 8 x 8 doubles
  static constexpr int OFF_F = OFF_D + 8 * 8 * 8;         // 8 floats
  static constexpr int LDS = OFF_F + 8 * 4;
  static_assert(RS2 * NCH * NB == 8, "eight waves share the second product");
  static_assert(RS2 * D32 * R32 * 4 <= kRows * XRS, "the partial combine fits the Xhat tile");
  static constexpr int GS = NB == 1 ? 8 : 2;              // Gram partials per workgroup
  static_assert(GS * R32 * R32 * 4 <= kRows * WRS, "the Gram combine fits the W tile");
};

// Byte offset within a tile (rows of RS bytes) of this lane's transposing read
// for k-rows 8 (l / 32) + 4 half + (l % 16) / 4 and the units u0 + 4 ((l / 16) % 2)
// + l % 4 (u0 a multiple of 8), half hl (0 hi, 1 lo): the two reads (half 0, 1)
// of a 16-row step give lane l the 8 k-rows 8 (l / 32) + e of column 4 u0 + l % 32.
__device__ __forceinline__ uint32_t tr_off(int RS, int u0, int hl, int half, int lane) {
  const int gq = lane >> 4, s = lane & 15;
  const int R = 8 * (gq >> 1) + 4 * half + (s >> 2);
  const int u = u0 + 4 * (gq & 1) + (s & 3);
  return (uint32_t)(R * RS + 16 * (u ^ swz(R)) + 8 * (hl ^ (R & 1)));
}

// Index of Theta[f][c] in the pass-B operand layout written by the Theta reduction.
template <int NB>
__device__ __forceinline__ int theta_index(int f, int c) {
  const int ch = f >> 5, fin = f & 31;
  const int hh = fin >> 4, jq = (fin & 15) >> 2, ee = fin & 3;
  const int mb = c >> 5, l = hh * 32 + (c & 31);
  return ((((ch * 4 + jq) * NB + mb) * 64 + l) * 4) + ee;
}

__device__ __forceinline__ f16x8 join4(f16x4 a, f16x4 b) {
  return (f16x8){a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// The transposing reads of one 16-row step of the second product, as assembly:
// the compiler orders the ds_read_b64_tr_b16 builtin after every global store in
// flight (it waits for the vector memory counter first), which would drain the
// prefetched rows each tile.  One statement issues the reads and waits for their
// data, so its outputs are defined only when they hold it.  xa[half][hl],
// wa[half][hl]: LDS byte addresses; OX / OW: the step's byte offset.
#define BF8_TR(o, a, f) "ds_read_b64_tr_b16 %" #o ", %" #a " offset:%" #f "\n\t"
template <int OX, int OW>
__device__ __forceinline__ void step_reads(const uint32_t (&xa)[2][2], const uint32_t (&wa)[2][2], f16x8& xh,
                                           f16x8& xl, f16x8& wh, f16x8& wl) {
  f16x4 x0, x1, x2, x3, w0, w1, w2, w3;
  asm volatile(BF8_TR(0, 8, 16) BF8_TR(1, 9, 16) BF8_TR(2, 10, 16) BF8_TR(3, 11, 16)
               BF8_TR(4, 12, 17) BF8_TR(5, 13, 17) BF8_TR(6, 14, 17) BF8_TR(7, 15, 17)
               "s_waitcnt lgkmcnt(0)"
               : "=&v"(x0), "=&v"(x1), "=&v"(x2), "=&v"(x3), "=&v"(w0), "=&v"(w1), "=&v"(w2), "=&v"(w3)
               : "v"(xa[0][0]), "v"(xa[1][0]), "v"(xa[0][1]), "v"(xa[1][1]),
                 "v"(wa[0][0]), "v"(wa[1][0]), "v"(wa[0][1]), "v"(wa[1][1]), "n"(OX), "n"(OW)
               : "memory");
  xh = join4(x0, x1);
  xl = join4(x2, x3);
  wh = join4(w0, w1);
  wl = join4(w2, w3);
}
// The W operand of a column block for the Gram product (4 reads).
template <int OW>
__device__ __forceinline__ void gram_reads(const uint32_t (&ga)[2][2], f16x8& gh, f16x8& gl) {
  f16x4 w0, w1, w2, w3;
  asm volatile(BF8_TR(0, 4, 8) BF8_TR(1, 5, 8) BF8_TR(2, 6, 8) BF8_TR(3, 7, 8)
               "s_waitcnt lgkmcnt(0)"
               : "=&v"(w0), "=&v"(w1), "=&v"(w2), "=&v"(w3)
               : "v"(ga[0][0]), "v"(ga[1][0]), "v"(ga[0][1]), "v"(ga[1][1]), "n"(OW)
               : "memory");
  gh = join4(w0, w1);
  gl = join4(w2, w3);
}
#undef BF8_TR

// Slot of unit q of a wave's staged fp32 slab: the low four bits exchanged with the
// 16-unit block index, so a store of 16 rows' unit u and a read of 16 consecutive
// units each meet 64 distinct banks (rows of 16 units).
__device__ __forceinline__ int stage_slot(int q) { return q ^ ((q >> 4) & 15); }

__device__ __forceinline__ f32x4 mfma16x16x32h(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// Reduce-scatter of 16 values over the 16 lanes of a DPP row: afterwards lane li
// holds the sum over the row of element li.  The four exchanges pair lane li with
// 15 - li, then 7 - li within each half row, then li ^ 2 and li ^ 1 (DPP, no LDS);
// the lane whose index has the exchange's bit set keeps the upper half.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int LEN, int BIT, int CTRL>
__device__ __forceinline__ void rs_step(float* v, int li) {
  const bool up = (li & BIT) != 0;
#pragma unroll
  for (int k = 0; k < LEN / 2; ++k) {
    const float send = up ? v[k] : v[k + LEN / 2];
    const float keep = up ? v[k + LEN / 2] : v[k];
    v[k] = keep + dpp_f<CTRL>(send);
  }
}
__device__ __forceinline__ void reduce_scatter16_row(float* v, int li) {
  rs_step<16, 8, 0x140>(v, li);  // row_mirror
  rs_step<8, 4, 0x141>(v, li);   // row_half_mirror
  rs_step<4, 2, 0x4E>(v, li);    // quad_perm [2, 3, 0, 1]
  rs_step<2, 1, 0xB1>(v, li);    // quad_perm [1, 0, 3, 2]
}
// The same for 8 values: lanes li and 15 - li first add all 8 (each half row then
// covers the 16 rows), then the half-row steps; lane li keeps element li % 8.
__device__ __forceinline__ void reduce_scatter8_row(float* v, int li) {
#pragma unroll
  for (int k = 0; k < 8; ++k) v[k] = v[k] + dpp_f<0x140>(v[k]);  // row_mirror
  rs_step<8, 4, 0x141>(v, li);
  rs_step<4, 2, 0x4E>(v, li);
  rs_step<2, 1, 0xB1>(v, li);
}

// A 16-byte unit (hi halves, lo halves) into its LDS slot, its two 8-byte halves
// exchanged when `odd` (by address: two 8-byte writes, no data movement).
__device__ __forceinline__ void put_unit(unsigned char* slot, f32x4 v, bool odd) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  const int o = odd ? 8 : 0;
  *reinterpret_cast<f32x2*>(slot + o) = (f32x2){v.x, v.y};
  *reinterpret_cast<f32x2*>(slot + (o ^ 8)) = (f32x2){v.z, v.w};
}

}  // namespace bf8

// PAIRS (one column block, r % 4 == 2): the rows of U are 8-byte aligned only; the
// factor moves in column pairs (8-byte loads, and 8-byte pieces of the packed slab).
template <int NB, int NCH, bool PAIRS>
__global__ __launch_bounds__(bf8::kThreads8) __attribute__((amdgpu_waves_per_eu(NB * NCH == 1 ? 4 : 2, NB * NCH == 1 ? 4 : 2))) void k_pass_bf8(
    Geometry g, Bufs B, StepArgs S) {
  using P = bf8::Shape<NB, NCH>;
  static_assert(!PAIRS || NB == 1, "column pairs: one column block");
  constexpr int CB16 = P::CB16, R32 = P::R32, D32 = P::D32;
  constexpr int KPW = P::KPW;
  // the row work's dot and the Gram blocks are laid out for 33..64 columns and 97..128
  // features, or for at most 16 columns (one 32-column block) and at most 64 features
  static_assert((NB == 2 && NCH == 4) || (NB == 1 && NCH <= 2), "one-pass shapes");
  if (halted(B.ctl)) return;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  f16x8* th_h = reinterpret_cast<f16x8*>(smem_raw);
  f16x8* th_l = reinterpret_cast<f16x8*>(smem_raw + P::TH);
  unsigned char* xt = smem_raw + P::OFF_X;
  unsigned char* wt = smem_raw + P::OFF_W;
  double* pds = reinterpret_cast<double*>(smem_raw + P::OFF_P);
  float* naps = reinterpret_cast<float*>(smem_raw + P::OFF_S);  // -alpha p
  float* nass = naps + R32;                                      // -alpha s
  double* colred = reinterpret_cast<double*>(smem_raw + P::OFF_COL);
  double* colyred = reinterpret_cast<double*>(smem_raw + P::OFF_COLY);
  double* dred = reinterpret_cast<double*>(smem_raw + P::OFF_D);
  float* fred = reinterpret_cast<float*>(smem_raw + P::OFF_F);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j = lane & 15, gq = lane >> 4;
  const int64_t n = g.n;
  const int d = g.d, r = g.r;
  const float cf = B.ctl->c_f;
  const float gam = S.gamma_f;
  const float neg_alpha = -S.alpha_f;
  const float sx = B.ctl->x_scale;
  // W_{t+1} is written over the factor rows this workgroup has read (each tile's rows
  // are read and written by the same workgroup, the reads first): the pass runs only
  // once the previous iteration's stopping rule can no longer discard it
  const float* Usrc = B.U;
  float* Udst = B.U;
  // the pending gated dual step (the end of the previous iteration), unless the row
  // pass has applied it
  const bool gate = (S.end_work != 0) && (B.ctl->gate != 0) && (B.ctl->rows_first == 0);

  // ---- Theta_t as the A operand of the first product: lane l of block (ks, cb)
  // holds column 16 cb + l % 16 and, for q = l / 16, features 32 ks + 4 q + e and
  // 32 ks + 16 + 4 q + e (e = 0..3), the features of the two Xhat units that lane
  // q of a row loads ----
  float tmax = 0.f;
  for (int e = tid; e < D32 * R32; e += bf8::kThreads8) tmax = fmaxf(tmax, fabsf(B.theta[e]));
  for (int m = 32; m >= 1; m >>= 1) tmax = fmaxf(tmax, shfl_xor_f(tmax, m));
  if (lane == 0) fred[wave] = tmax;
  __syncthreads();
  tmax = fred[0];
#pragma unroll
  for (int w = 1; w < 8; ++w) tmax = fmaxf(tmax, fred[w]);
  const float sth = f16_range_scale(tmax);
  const float two_alpha_s = S.two_alpha_f * (1.0f / sx) * (1.0f / sth);
  for (int idx = tid; idx < NCH * CB16 * 64; idx += bf8::kThreads8) {
    const int l = idx & 63;
    const int cb = (idx >> 6) % CB16;
    const int ks = (idx >> 6) / CB16;
    const int c = 16 * cb + (l & 15), q = l >> 4;
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int f = 32 * ks + 4 * q + (e < 4 ? e : 12 + e);
      v[e] = B.theta[bf8::theta_index<NB>(f, c)];
    }
    f16x8 hi, lo;
    split_f16(v, sth, hi, lo);
    th_h[idx] = hi;
    th_l[idx] = lo;
  }
  for (int c = tid; c < R32; c += bf8::kThreads8) {
    pds[c] = (double)B.p[c];
    naps[c] = neg_alpha * B.p[c];
    nass[c] = neg_alpha * B.s[c];
  }
  __syncthreads();

  // ---- per-lane constants ----
  // second product: wave w owns the 32 x 32 block (fb, cb2) of the partial over the
  // 16-row steps KPW rsp .. KPW (rsp + 1) - 1 of each tile; and the block (ga, cb2)
  // of the Gram partial W^T W over the steps 4 gh .. 4 gh + 3
  const int fb = wave % NCH, cb2 = (wave / NCH) % NB, rsp = wave / (NCH * NB);
  const int ga = fb & 1, gh = fb >> 1;
  const uint32_t lds0 =
      (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) unsigned char*)smem_raw);
  uint32_t xa[2][2], wa[2][2], wg[2][2];
#pragma unroll
  for (int half = 0; half < 2; ++half)
#pragma unroll
    for (int hl = 0; hl < 2; ++hl) {
      xa[half][hl] = lds0 + P::OFF_X + (uint32_t)(16 * KPW * rsp * P::XRS) + (uint32_t)(256 * (fb >> 1)) +
                     bf8::tr_off(P::XRS, 8 * (fb & 1), hl, half, lane);
      wa[half][hl] = lds0 + P::OFF_W + (uint32_t)(16 * KPW * rsp * P::WRS) + bf8::tr_off(P::WRS, 8 * cb2, hl, half, lane);
      wg[half][hl] = lds0 + P::OFF_W + (uint32_t)(64 * gh * P::WRS) + bf8::tr_off(P::WRS, 8 * ga, hl, half, lane);
    }

  double sa = 0.0, sb = 0.0, sh = 0.0, colacc = 0.0, colyacc = 0.0, qq = 0.0, yq = 0.0;
  float wmx = 0.f;  // largest w of this lane (the fp16 range of the split W operand)
  f32x16 acc2, accg;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc2[v] = accg[v] = 0.f;

  const int64_t T = g.tilesB;
  const int64_t step = gridDim.x;

  // the next tile's rows are requested as soon as this tile has consumed its own
  struct Buf {
    f32x4 x[NCH][2];
  };
  struct UBuf {
    f32x4 u[CB16];
    float y;
  };
  // lane-derived offsets are recomputed where used (from an opaque copy of the lane
  // id), not kept live across the tile loop
  auto opaque_lane = [&]() -> int {
    int lo = lane;
    asm volatile("" : "+v"(lo));
    return lo;
  };
  // row of this lane within tile st (row 0 of the tile for rows >= n; a tile >= T
  // reads tile 0, whose values are never used)
  auto lane_row = [&](int64_t st, int jj, int64_t& tile_base) -> uint32_t {
    const int64_t stc = st < T ? st : 0;
    tile_base = stc * bf8::kRows;
    const int rr = 16 * wave + jj;
    return (tile_base + rr < n) ? (uint32_t)rr : 0u;
  };
  // uniform tile base + 32-bit lane byte offset (the scalar-base form of the loads)
  // the two units of 32-feature step ks (all of them for ks < 0)
  auto load_x = [&](Buf& b, int64_t st, int kso) {
    const int lo = opaque_lane(), gq = lo >> 4;
    int64_t tb;
    const uint32_t rr = lane_row(st, lo & 15, tb);
    const char* base = reinterpret_cast<const char*>(B.X + tb * (int64_t)d);
#pragma unroll
    for (int ks = 0; ks < NCH; ++ks)
      if (kso < 0 || ks == kso) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int f = 32 * ks + 16 * hh + 4 * gq;  // features >= d meet zero rows of Theta_t
          const uint32_t off = 4u * (rr * (uint32_t)d + (uint32_t)(f < d ? f : 0));
          b.x[ks][hh] = *reinterpret_cast<const f32x4*>(base + off);
        }
      }
  };
  auto load_u = [&](UBuf& b, int64_t st) {
    const int lo = opaque_lane(), gq = lo >> 4;
    int64_t tb;
    const uint32_t rr = lane_row(st, lo & 15, tb);
    const char* base = reinterpret_cast<const char*>(Usrc + tb * (int64_t)r);
    // (one column block: at most 16 columns, all in the first 16-column block)
    if constexpr (PAIRS) {
      // columns c, c + 1 and c + 2, c + 3 as two 8-byte loads; a pair at or beyond r reads
      // column 0 of the row instead (its values are masked)
      typedef float f32x2 __attribute__((ext_vector_type(2)));
      const int c = 4 * gq;
      const uint32_t o0 = 4u * (rr * (uint32_t)r + (uint32_t)(c < r ? c : 0));
      const uint32_t o1 = 4u * (rr * (uint32_t)r + (uint32_t)(c + 2 < r ? c + 2 : 0));
      const f32x2 v0 = *reinterpret_cast<const f32x2*>(base + o0);
      const f32x2 v1 = *reinterpret_cast<const f32x2*>(base + o1);
      b.u[0] = (f32x4){v0.x, v0.y, v1.x, v1.y};
    } else {
#pragma unroll
      for (int cb = 0; cb < (NB == 1 ? 1 : CB16); ++cb) {
        const int c = 16 * cb + 4 * gq;
        const uint32_t off = 4u * (rr * (uint32_t)r + (uint32_t)(c < r ? c : 0));
        b.u[cb] = *reinterpret_cast<const f32x4*>(base + off);
      }
    }
    b.y = *reinterpret_cast<const float*>(reinterpret_cast<const char*>(B.y + tb) + 4u * rr);
  };

  // nst: the tile whose rows replace this tile's in bx and ub once they are consumed
  auto tile = [&](Buf& bx, UBuf& ub, int64_t st, int64_t nst) {
    __builtin_amdgcn_sched_barrier(0);
    const int lane = opaque_lane();
    const int j = lane & 15, gq = lane >> 4;
    const int sj = bf8::swz(j);
    const bool oddj = (j & 1) != 0;
    const int gs = gq ^ sj;
    const uint32_t xrow = (uint32_t)((16 * wave + j) * P::XRS);
    const uint32_t wrow = (uint32_t)((16 * wave + j) * P::WRS);
    const int64_t pt = st * bf8::kRows + 16 * wave + j;
    const bool vpt = pt < n;
    // ---- first product: G = Xhat_slab Theta_t ----
    f32x4 acc1[CB16];
#pragma unroll
    for (int cb = 0; cb < CB16; ++cb) acc1[cb] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < NCH; ++ks) {
      typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
      const f32x4 xa0 = bx.x[ks][0], xa1 = bx.x[ks][1];
      const u32x4 hb = {__float_as_uint(xa0.x), __float_as_uint(xa0.y), __float_as_uint(xa1.x), __float_as_uint(xa1.y)};
      const u32x4 lb = {__float_as_uint(xa0.z), __float_as_uint(xa0.w), __float_as_uint(xa1.z), __float_as_uint(xa1.w)};
      const f16x8 xh = __builtin_bit_cast(f16x8, hb);
      const f16x8 xl = __builtin_bit_cast(f16x8, lb);
      // the slab's units into the Xhat tile of the second product
      bf8::put_unit(xt + xrow + 16 * ((8 * ks) ^ gs), xa0, oddj);
      bf8::put_unit(xt + xrow + 16 * ((8 * ks + 4) ^ gs), xa1, oddj);
#pragma unroll
      for (int cb = 0; cb < CB16; ++cb) {
        const f16x8 ah = th_h[(ks * CB16 + cb) * 64 + lane];
        const f16x8 al = th_l[(ks * CB16 + cb) * 64 + lane];
        acc1[cb] = bf8::mfma16x16x32h(ah, xl, acc1[cb]);
        acc1[cb] = bf8::mfma16x16x32h(al, xh, acc1[cb]);
        acc1[cb] = bf8::mfma16x16x32h(ah, xh, acc1[cb]);
      }
      __builtin_amdgcn_sched_barrier(0);
      load_x(bx, nst, ks);  // this step's Xhat units of the next tile
      __builtin_amdgcn_sched_barrier(0);
    }

    // ---- row work on row pt, columns 16 cb + 4 gq + v ----
    int lds_off = 0;  // opaque zero offset: p and s are read from LDS here, not kept in registers
    asm volatile("" : "+v"(lds_off));
    const double* pdl = pds + lds_off;
    const float* napl = naps + lds_off;
    const float* nasl = nass + lds_off;
    // okf: 1 for a valid row and column, else 0 (masked lanes compute on finite
    // values and their results are multiplied away: no branches)
    // (okf2: the same for the group's second column pair, which PAIRS can lose alone)
    float okf[CB16], okf2[CB16];
    float u[CB16][4];
#pragma unroll
    for (int cb = 0; cb < CB16; ++cb) {
      okf[cb] = (vpt && (16 * cb + 4 * gq) < r) ? 1.0f : 0.0f;
      okf2[cb] = PAIRS ? ((vpt && (16 * cb + 4 * gq + 2) < r) ? 1.0f : 0.0f) : okf[cb];
      const float sc = cf * okf[cb], sc2 = cf * okf2[cb];
      const f32x4 uv = (NB == 1 && cb > 0) ? (f32x4){0.f, 0.f, 0.f, 0.f} : ub.u[cb];
      u[cb][0] = uv.x * sc;
      u[cb][1] = uv.y * sc;
      u[cb][2] = uv.z * sc2;
      u[cb][3] = uv.w * sc2;
    }
    // q = u.p - 1 (FP64): the partial of each group of four columns, then the pairs
    // (columns 4k.. with 4(k^1).., then 4(k^2)..), then the groups of 16 and 32 --
    // the order of the row pass and the finish pass, so that q, the stored dual and
    // ybar are bitwise the same whichever kernel does the row work
    double dot;
    typedef double f64x2 __attribute__((ext_vector_type(2)));
    if constexpr (NB == 1) {
      // at most 16 columns, all in block 0: the order of the narrow row pass -- pairs of
      // columns, then groups of 4, 8 and 16 (the products are exact in FP64)
      const f64x2 p01 = *reinterpret_cast<const f64x2*>(pdl + 4 * gq);
      const f64x2 p23 = *reinterpret_cast<const f64x2*>(pdl + 4 * gq + 2);
      const double a01 = (double)u[0][0] * p01.x + (double)u[0][1] * p01.y;
      const double a23 = (double)u[0][2] * p23.x + (double)u[0][3] * p23.y;
      double v = a01 + a23;
      v += shfl_xor_d(v, 16);
      v += shfl_xor_d(v, 32);
      dot = v;
    } else {
      double pd[CB16];
#pragma unroll
      for (int cb = 0; cb < CB16; ++cb) {
        const f64x2 p01 = *reinterpret_cast<const f64x2*>(pdl + 16 * cb + 4 * gq);
        const f64x2 p23 = *reinterpret_cast<const f64x2*>(pdl + 16 * cb + 4 * gq + 2);
        const double pe[4] = {p01.x, p01.y, p23.x, p23.y};
        double dd = 0.0;
#pragma unroll
        for (int e = 0; e < 4; ++e) dd += (double)u[cb][e] * pe[e];
        pd[cb] = dd;
      }
#pragma unroll
      for (int cb = 0; cb < CB16; ++cb) pd[cb] += shfl_xor_d(pd[cb], 16);
#pragma unroll
      for (int cb = 0; cb < CB16; ++cb) pd[cb] += shfl_xor_d(pd[cb], 32);
      dot = (pd[0] + pd[1]) + (pd[2] + pd[3]);
    }
    const float q = (float)(dot - 1.0);
    float yt = vpt ? ub.y : 0.f;
    if (gate) yt = fmaf(gam, q, yt);
    const float ybar = fmaf(gam, q, yt);
    // the factor rows and ytilde of this tile are consumed: request the next tile's
    __builtin_amdgcn_sched_barrier(0);
    load_u(ub, nst);
    __builtin_amdgcn_sched_barrier(0);
    if (gate) *(vpt ? (B.y + pt) : B.dump) = yt;  // the four lanes of a row store the same value
    {
      const bool lead = vpt && gq == 0;
      qq += lead ? (double)q * (double)q : 0.0;
      yq += lead ? (double)yt * (double)q : 0.0;
    }

    // ---- epilogue (eq. entrywise-fusion).  W of the slab: kept in registers, staged
    // fp32 in this wave's rows of the W tile (private to the wave until the barrier
    // below) as the packed rows of U, so that it goes to HBM in whole, contiguous
    // 1 KiB stores; then the same rows take its split for the second product ----
    unsigned char* wst = wt + 16 * wave * P::WRS;
    const int ru = r >> 2;  // 16-byte units per row of U
    float wv[4 * CB16];
#pragma unroll
    for (int cb = 0; cb < CB16; ++cb) {
      const int c = 16 * cb + 4 * gq;
      const f32x4 pv = *reinterpret_cast<const f32x4*>(napl + c);
      const f32x4 sv = *reinterpret_cast<const f32x4*>(nasl + c);
      const float pe[4] = {pv.x, pv.y, pv.z, pv.w};  // -alpha p
      const float se[4] = {sv.x, sv.y, sv.z, sv.w};  // -alpha s
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float uu = u[cb][e];
        float t = fmaf(two_alpha_s, acc1[cb][e], uu);
        t = fmaf(ybar, pe[e], t);
        t = t + se[e];
        const float w = fmaxf(t, 0.f) * (e < 2 ? okf[cb] : okf2[cb]);
        wv[4 * cb + e] = w;
        wmx = fmaxf(wmx, w);
        const double wd = (double)w, ud = (double)uu;
        sa = fma(wd, wd, sa);
        sb = fma(ud, ud, sb);
        sh = fma(wd, ud, sh);
      }
      const f32x4 o = {wv[4 * cb + 0], wv[4 * cb + 1], wv[4 * cb + 2], wv[4 * cb + 3]};
      if constexpr (PAIRS) {
        // floats j r + c .. of the packed slab as two 8-byte pieces (unit (j r + c) / 4,
        // half ((j r + c) / 2) % 2); pairs at or beyond r to the last unit, never stored
        typedef float f32x2 __attribute__((ext_vector_type(2)));
        const int f0 = j * r + c;
        const int q0 = (c < r) ? (f0 >> 2) : (16 * P::WU - 1), h0 = (c < r) ? ((f0 >> 1) & 1) : 0;
        const int q1 = (c + 2 < r) ? ((f0 + 2) >> 2) : (16 * P::WU - 1), h1 = (c + 2 < r) ? (((f0 + 2) >> 1) & 1) : 1;
        *reinterpret_cast<f32x2*>(wst + 16 * bf8::stage_slot(q0) + 8 * h0) = (f32x2){o.x, o.y};
        *reinterpret_cast<f32x2*>(wst + 16 * bf8::stage_slot(q1) + 8 * h1) = (f32x2){o.z, o.w};
      } else {
        // unit j ru + c / 4 of the packed slab (columns >= r to the last unit, never stored)
        const int uq = (c < r) ? (j * ru + 4 * cb + gq) : (16 * P::WU - 1);
        *reinterpret_cast<f32x4*>(wst + 16 * bf8::stage_slot(uq)) = o;
      }
    }
    __builtin_amdgcn_wave_barrier();
    {
      const int64_t row0 = st * bf8::kRows + 16 * wave;
      const int64_t rows = n - row0 < 16 ? n - row0 : 16;
      // 16-byte units of the slab in U (PAIRS: rows r floats, a last half unit when rows r % 4 == 2)
      const int nfl = rows > 0 ? (int)rows * r : 0;
      const int nvalid = nfl >> 2;
      char* sbase = reinterpret_cast<char*>(Udst + (rows > 0 ? row0 : 0) * (int64_t)r);
#pragma unroll
      for (int i = 0; i < 2 * NB; ++i) {  // 16 rows x R32 floats = 128 NB units
        const int q = lane + 64 * i;
        const f32x4 v = *reinterpret_cast<const f32x4*>(wst + 16 * bf8::stage_slot(q));
        if (q < nvalid) *reinterpret_cast<f32x4*>(sbase + 16u * (uint32_t)q) = v;
        if (PAIRS && q == nvalid && (nfl & 3) != 0) {
          typedef float f32x2 __attribute__((ext_vector_type(2)));
          *reinterpret_cast<f32x2*>(sbase + 16u * (uint32_t)q) = (f32x2){v.x, v.y};
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int cb = 0; cb < CB16; ++cb) {
      f16x4 hi, lo;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float ts = wv[4 * cb + e] * kWScale;
        const _Float16 hh = (_Float16)ts;
        hi[e] = hh;
        lo[e] = (_Float16)(ts - (float)hh);
      }
      typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
      const u32x2 hu = __builtin_bit_cast(u32x2, hi);
      const u32x2 lu = __builtin_bit_cast(u32x2, lo);
      const f32x4 unit = {__uint_as_float(hu.x), __uint_as_float(hu.y), __uint_as_float(lu.x), __uint_as_float(lu.y)};
      bf8::put_unit(wt + wrow + 16 * ((4 * cb + gq) ^ sj), unit, oddj);
    }
    // column sums of the slab, of W and of W ytilde_t (ytilde after this pass's dual
    // step: the Gram terms of the next iteration's s): lane (j, gq) keeps the
    // column of element j of its 16 values
    {
      float wy[4 * CB16];
#pragma unroll
      for (int k = 0; k < 4 * CB16; ++k) wy[k] = wv[k] * yt;
      if constexpr (NB == 1) {
        // 8 values: lane j keeps element j % 8
        bf8::reduce_scatter8_row(wv, j);
        bf8::reduce_scatter8_row(wy, j);
      } else {
        bf8::reduce_scatter16_row(wv, j);
        bf8::reduce_scatter16_row(wy, j);
      }
      colacc += (double)wv[0];
      colyacc += (double)wy[0];
    }
    __syncthreads();

    // ---- second product: partial += Xhat_tile^T W_tile (this wave's block and
    // steps), and the Gram block W_ga^T W_cb2 over this wave's four steps ----
    // the wave's four Gram steps first: steps k = 0..3 are the tile's 16-row steps
    // 4 gh + k, where the Gram block W_ga^T W_cb2 takes the W operand just read as
    // its B operand; steps k = 4..7 are the tile's steps k - 4 gh
    uint32_t xr[2][2], wr[2][2];
    auto rebase = [&](int sign) {
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int hl = 0; hl < 2; ++hl) {
          xr[half][hl] = xa[half][hl] + (uint32_t)(sign * 64 * gh * P::XRS);
          wr[half][hl] = wa[half][hl] + (uint32_t)(sign * 64 * gh * P::WRS);
        }
    };
    auto p2 = [&](auto kc) {
      constexpr int K = decltype(kc)::value;
      f16x8 xh, xl, wh, wl;
      bf8::step_reads<16 * K * P::XRS, 16 * K * P::WRS>(xr, wr, xh, xl, wh, wl);
      acc2 = mfma32x32x16h(xh, wl, acc2);
      acc2 = mfma32x32x16h(xl, wh, acc2);
      acc2 = mfma32x32x16h(xh, wh, acc2);
      if constexpr (K < 4) {
        f16x8 gah, gal;
        bf8::gram_reads<16 * K * P::WRS>(wg, gah, gal);
        accg = mfma32x32x16h(gah, wl, accg);
        accg = mfma32x32x16h(gal, wh, accg);
        accg = mfma32x32x16h(gah, wh, accg);
      }
    };
    if constexpr (NB == 1) {
      // one column block: wave w does its KPW steps of block (fb, 0) and the Gram block
      // W^T W over the tile's 16-row step w, one of its own steps (k = w - KPW rsp), from
      // the W operand just read (as A it is W^T)
      const int gk = wave - KPW * rsp;
      auto p2n = [&](auto kc) {
        constexpr int K = decltype(kc)::value;
        f16x8 xh, xl, wh, wl;
        bf8::step_reads<16 * K * P::XRS, 16 * K * P::WRS>(xa, wa, xh, xl, wh, wl);
        acc2 = mfma32x32x16h(xh, wl, acc2);
        acc2 = mfma32x32x16h(xl, wh, acc2);
        acc2 = mfma32x32x16h(xh, wh, acc2);
        if (gk == K) {
          accg = mfma32x32x16h(wh, wl, accg);
          accg = mfma32x32x16h(wl, wh, accg);
          accg = mfma32x32x16h(wh, wh, accg);
        }
      };
      p2n(std::integral_constant<int, 0>{});
      if constexpr (KPW > 1) p2n(std::integral_constant<int, 1>{});
    } else {
      rebase(1);
      p2(std::integral_constant<int, 0>{});
      p2(std::integral_constant<int, 1>{});
      p2(std::integral_constant<int, 2>{});
      p2(std::integral_constant<int, 3>{});
      rebase(-1);
      p2(std::integral_constant<int, 4>{});
      p2(std::integral_constant<int, 5>{});
      p2(std::integral_constant<int, 6>{});
      p2(std::integral_constant<int, 7>{});
    }
    __syncthreads();
  };

  Buf A;
  UBuf ub;
  load_x(A, blockIdx.x, -1);
  load_u(ub, blockIdx.x);
  for (int64_t st = blockIdx.x; st < T; st += step) tile(A, ub, st, st + step);

  // ---- statistics of this workgroup ----
  if (NB == 2 || j < 8) {  // (one column block: lanes j and j + 8 hold the same element)
    const int col = 16 * (j >> 2) + 4 * gq + (j & 3);
    colred[wave * R32 + col] = colacc;
    colyred[wave * R32 + col] = colyacc;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    sa += shfl_xor_d(sa, m);
    sb += shfl_xor_d(sb, m);
    sh += shfl_xor_d(sh, m);
    qq += shfl_xor_d(qq, m);
    yq += shfl_xor_d(yq, m);
  }
  float wbad = (wmx > kWMax || wmx != wmx) ? 1.0f : 0.0f;  // w != w: NaN
  for (int m = 32; m >= 1; m >>= 1) wbad = fmaxf(wbad, shfl_xor_f(wbad, m));
  if (lane == 0) {
    dred[8 * wave + 0] = sa;
    dred[8 * wave + 1] = sb;
    dred[8 * wave + 2] = sh;
    dred[8 * wave + 3] = qq;
    dred[8 * wave + 4] = yq;
    fred[wave] = wbad;
  }
  // ---- partials of Xhat^T W_{t+1} (row splits in order, [f][c] order) and of
  // W^T W (the two halves of each block in order, [k][l] order) ----
  float* comb = reinterpret_cast<float*>(xt);   // RS2 x D32 x R32 (the tiles are no longer read)
  float* gcomb = reinterpret_cast<float*>(wt);  // GS x R32 x R32
  const float unscale = (1.0f / sx) * (1.0f / kWScale);
  {
    const int h = lane >> 5, li = lane & 31;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int f = 32 * fb + 8 * (v >> 2) + 4 * h + (v & 3);
      comb[(rsp * D32 + f) * R32 + 32 * cb2 + li] = acc2[v] * unscale;
      const int k = 32 * ga + 8 * (v >> 2) + 4 * h + (v & 3);
      const int gs = NB == 1 ? wave : gh;  // the Gram split this wave holds
      gcomb[(gs * R32 + (NB == 1 ? k - 32 * ga : k)) * R32 + 32 * cb2 + li] = accg[v] * (1.0f / (kWScale * kWScale));
    }
  }
  __syncthreads();
  double* out = B.b_part + (int64_t)blockIdx.x * (4 + R32);
  double* aout = B.a_part + (int64_t)blockIdx.x * (4 + R32);
  for (int c = tid; c < R32; c += bf8::kThreads8) {
    const double* q = colred + c;
    out[4 + c] = (((q[0] + q[R32]) + (q[2 * R32] + q[3 * R32])) + ((q[4 * R32] + q[5 * R32]) + (q[6 * R32] + q[7 * R32])));
    const double* qy = colyred + c;
    aout[4 + c] =
        (((qy[0] + qy[R32]) + (qy[2 * R32] + qy[3 * R32])) + ((qy[4 * R32] + qy[5 * R32]) + (qy[6 * R32] + qy[7 * R32])));
  }
  if (tid < 5) {
    const double* q = dred + tid;
    const double v = (((q[0] + q[8]) + (q[16] + q[24])) + ((q[32] + q[40]) + (q[48] + q[56])));
    if (tid < 3) out[tid] = v;
    else aout[tid - 3] = v;  // ||q||^2, ytilde^T q
  }
  if (tid == 5) {
    float bad = 0.f;
#pragma unroll
    for (int w = 0; w < 8; ++w) bad = fmaxf(bad, fred[w]);
    out[3] = bad > 0.f ? 1.0 : 0.0;  // W left the range of its split operand
  }
  if (tid == 6) aout[2] = 0.0;
  if (tid == 7) aout[3] = 0.0;
  float* part = B.theta_part + (int64_t)blockIdx.x * g.theta_cols;
  for (int e = tid; e < D32 * R32; e += bf8::kThreads8) {
    float acc = comb[e];
#pragma unroll
    for (int s2 = 1; s2 < P::RS2; ++s2) acc += comb[s2 * D32 * R32 + e];
    part[e] = acc;
  }
  float* gpart = part + D32 * R32;  // W^T W follows Theta in the row
  for (int e = tid; e < R32 * R32; e += bf8::kThreads8) {
    const float* gc = gcomb + e;
    constexpr int RR = R32 * R32;
    if constexpr (NB == 1)
      gpart[e] = ((gc[0] + gc[RR]) + (gc[2 * RR] + gc[3 * RR])) + ((gc[4 * RR] + gc[5 * RR]) + (gc[6 * RR] + gc[7 * RR]));
    else
      gpart[e] = gc[0] + gc[RR];
  }
}

template <int NB, int NCH, bool PAIRS>
static hipError_t pass_bf8_launch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  constexpr int lds = bf8::Shape<NB, NCH>::LDS;
  static_assert(lds <= kMaxFusedLds, "LDS");
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pass_bf8<NB, NCH, PAIRS>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_pass_bf8<NB, NCH, PAIRS>), dim3(g.GB), dim3(bf8::kThreads8), lds, st, g, b, a);
  return hipGetLastError();
}

// shapes of the eight-wave form
// 33..64 columns (r % 4 == 0) with 97..128 features; or at most 16 columns, r even (the
// narrow row pass's order of the row dot), with at most 64 features
bool fused8_shape(int NB, int nch, int r) {
  return (NB == 2 && nch == 4 && r % 4 == 0) || (NB == 1 && nch <= 2 && r <= 16 && r % 2 == 0);
}

static hipError_t pass_bf8_dispatch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  switch (g.NB * 10 + g.nch) {
    case 24: return g.r % 4 == 0 ? pass_bf8_launch<2, 4, false>(g, b, a, st) : hipErrorInvalidValue;
    case 11: return g.r % 4 == 0 ? pass_bf8_launch<1, 1, false>(g, b, a, st) : pass_bf8_launch<1, 1, true>(g, b, a, st);
    case 12: return g.r % 4 == 0 ? pass_bf8_launch<1, 2, false>(g, b, a, st) : pass_bf8_launch<1, 2, true>(g, b, a, st);
    default: return hipErrorInvalidValue;
  }
}

template <int NB, int NCH, bool SPLIT, bool UFLAT, bool X2>
static hipError_t pass_bf_launch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  constexpr int lds = fused_lds_bytes(NB, NCH, SPLIT, UFLAT);
  if (lds > kMaxFusedLds) return hipErrorInvalidValue;
  if (lds > (64 << 10)) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pass_bf<NB, NCH, SPLIT, UFLAT, X2>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((k_pass_bf<NB, NCH, SPLIT, UFLAT, X2>), dim3(g.GB), dim3(kThreads), lds, st, g, b, a);
  return hipGetLastError();
}

template <bool SPLIT, bool UFLAT, bool X2>
static hipError_t pass_bf_dispatch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  switch (g.NB * 10 + g.nch) {
    case 11: return pass_bf_launch<1, 1, SPLIT, UFLAT, X2>(g, b, a, st);
    case 12: return pass_bf_launch<1, 2, SPLIT, UFLAT, X2>(g, b, a, st);
    case 13: return pass_bf_launch<1, 3, SPLIT, UFLAT, X2>(g, b, a, st);
    case 14: return pass_bf_launch<1, 4, SPLIT, UFLAT, X2>(g, b, a, st);
    case 21: return pass_bf_launch<2, 1, SPLIT, UFLAT, X2>(g, b, a, st);
    case 22: return pass_bf_launch<2, 2, SPLIT, UFLAT, X2>(g, b, a, st);
    case 23: return pass_bf_launch<2, 3, SPLIT, UFLAT, X2>(g, b, a, st);
    case 24: return pass_bf_launch<2, 4, SPLIT, UFLAT, X2>(g, b, a, st);
    default: return hipErrorInvalidValue;
  }
}

int fused_lds_need(int NB, int nch, bool split, bool uflat) { return fused_lds_bytes(NB, nch, split, uflat); }

hipError_t launch_pass_bf(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  if (g.fused8) return pass_bf8_dispatch(g, b, a, st);
  if (g.d % 4 != 0) {  // fp32 products only (even d)
    if (g.split_b || g.d % 2 != 0) return hipErrorInvalidValue;
    return g.uflat ? pass_bf_dispatch<false, true, true>(g, b, a, st) : pass_bf_dispatch<false, false, true>(g, b, a, st);
  }
  if (g.uflat) return g.split_b ? pass_bf_dispatch<true, true, false>(g, b, a, st) : pass_bf_dispatch<false, true, false>(g, b, a, st);
  return g.split_b ? pass_bf_dispatch<true, false, false>(g, b, a, st) : pass_bf_dispatch<false, false, false>(g, b, a, st);
}

}  // namespace nlr
