// Device helpers shared by the per-iteration kernels (gfx950).
#pragma once

#include "nlr_internal.hpp"

namespace nlr {

// Forms of the row-resident pass A: with the Theta product, the finish pass
// (materialises U), and the row work alone (fused iteration).
enum PassAMode { kPassIter = 0, kPassFinish = 1, kPassRows = 2 };

__device__ __forceinline__ bool halted(const DevCtl* ctl) {
  return (ctl->stop | ctl->breakdown) != 0;
}

// Whether the stopping rule of the previous iteration (Section 4.3) can still fire
// at this one: its movement is below min(eps_d, eps_c) and t >= T_min; only the
// residual rho of the current factor is then missing, which the row work computes.
// The one-pass iteration writes W over the factor it reads when this is false; when
// true, the row work runs in its own pass first and settles the rule.
__device__ __forceinline__ bool stop_possible(const DevCtl* ctl, const StepArgs& S) {
  const int64_t t = ctl->t_done;
  return S.end_work != 0 && t > 0 && ctl->Delta < S.eps_d * S.eps_d * S.K && ctl->delta < S.eps_c &&
         t >= S.T_min;
}

// Loads W consecutive floats; when !ok the (valid) address is still read and the
// values are replaced by zeros, so no branch is needed.
template <int W>
__device__ __forceinline__ void load_vec(float (&dst)[W], const float* src, bool ok) {
  if constexpr (W == 4) {
    const f32x4 t = *reinterpret_cast<const f32x4*>(src);
    dst[0] = ok ? t.x : 0.f;
    dst[1] = ok ? t.y : 0.f;
    dst[2] = ok ? t.z : 0.f;
    dst[3] = ok ? t.w : 0.f;
  } else if constexpr (W == 2) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    const f32x2 t = *reinterpret_cast<const f32x2*>(src);
    dst[0] = ok ? t.x : 0.f;
    dst[1] = ok ? t.y : 0.f;
  } else {
    const float t = *src;
    dst[0] = ok ? t : 0.f;
  }
}

template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, 0xF, 0xF, false);
  return __hiloint2double(hi, lo);
}
// Sum over the 8 lanes of each DPP half row, bitwise the same in all 8 lanes.
__device__ __forceinline__ double row8_sum_d(double v) {
  v += dpp_d<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_d<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_d<0x141>(v);  // row_half_mirror
  return v;
}

// Sum over the 16 lanes of a DPP row with involution pairings (xor 1, xor 2,
// half-row mirror, row mirror): every step adds two equal partial sums, so all
// lanes end with the same bits.
__device__ __forceinline__ double row16_sum_d(double v) {
  v += dpp_d<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_d<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_d<0x141>(v);  // row_half_mirror
  v += dpp_d<0x140>(v);  // row_mirror
  return v;
}

typedef float f32x4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f32x4v mfma16x16x4(float a, float b, f32x4v c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Reduce-scatter of LEN per-lane values across the lanes that differ in bits
// MASK, MASK/2, ...: afterwards a lane holds LEN >> steps sums, of the upper half
// when its bit is set and of the lower half otherwise.
template <int LEN, int MASK>
__device__ __forceinline__ void reduce_scatter(float* wv, int li) {
  if constexpr (LEN > 1 && MASK > 0) {
    const bool up = (li & MASK) != 0;
#pragma unroll
    for (int k = 0; k < LEN / 2; ++k) {
      const float send = up ? wv[k] : wv[k + LEN / 2];
      const float keep = up ? wv[k + LEN / 2] : wv[k];
      wv[k] = keep + shfl_xor_f(send, MASK);
    }
    reduce_scatter<LEN / 2, MASK / 2>(wv, li);
  }
}

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// D += A * B on the 32x32x16 fp16 matrix core (fp32 accumulate).  Lane l supplies
// A[l%32][8(l/32) + e] and B[8(l/32) + e][l%32] as element e; D has the layout of
// the 32x32x2 fp32 form: lane l, register v holds D[8(v/4)+4(l/32)+v%4][l%32].
__device__ __forceinline__ f32x16 mfma32x32x16h(f16x8 a, f16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Two-term fp16 split of 8 fp32 values after scaling by the power of two s:
// v s = hi + lo + O(2^-22 |v s|), hi = fp16(v s), lo = fp16(v s - hi).  With s chosen
// so that |v s| < 2^15, hi and (for |v s| >= 2^-3) lo are normal fp16 numbers.
__device__ __forceinline__ void split_f16(const float* v, float s, f16x8& hi, f16x8& lo) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float t = v[e] * s;
    const _Float16 h = (_Float16)t;
    hi[e] = h;
    lo[e] = (_Float16)(t - (float)h);
  }
}

// Power of two s with |v| s < 2^15 for every |v| <= vmax (1 when vmax is 0 or not finite).
__device__ __forceinline__ float f16_range_scale(float vmax) {
  if (!(vmax > 0.f) || !(vmax < 3.0e38f)) return 1.0f;
  int e;
  (void)frexpf(vmax, &e);  // vmax < 2^e
  int k = 15 - e;
  if (k > 100) k = 100;
  if (k < -100) k = -100;
  return ldexpf(1.0f, k);
}

// Fixed-order sum over a 512-thread workgroup; result valid in thread 0.
__device__ __forceinline__ double block_sum8_d(double v, double* red) {
  for (int m = 32; m >= 1; m >>= 1) v += shfl_xor_d(v, m);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0) r = (((red[0] + red[1]) + (red[2] + red[3])) + ((red[4] + red[5]) + (red[6] + red[7])));
  __syncthreads();
  return r;
}

}  // namespace nlr
