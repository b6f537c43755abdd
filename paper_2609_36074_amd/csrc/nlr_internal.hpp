// Internal declarations shared by the host controller and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "nlr.h"

namespace nlr {

constexpr int kThreads = 256;     // every kernel uses 256-thread workgroups (4 wave64)
constexpr int kHistCap = 4096;    // per-iteration record ring
constexpr int kTPA = 64;          // rows per pass-A tile
constexpr int kTPB = 128;         // rows per pass-B super-tile (4 waves x 32 rows)
constexpr int kMaxR = 448;        // largest supported rank (fp32 two-pass form above 256)
constexpr int kMaxPanelR = 256;   // largest rank of the split-fp16 panel form
constexpr int kPowerIters = 16;   // refinement power iterations after the squaring phase
constexpr int kSquarings = 20;    // C -> C^(2^20) before the refinement

// DevCtl::breakdown values besides 0: the normalisation breakdown of Algorithm 1,
// and a split-fp16 operand of W out of fp16's range (both stop the iteration, U then
// holds W).
constexpr int32_t kBreakdown = 1;
constexpr int32_t kRangeError = 2;

// Device control block.  Written only by single-workgroup control kernels and
// read uniformly by every kernel at entry.
struct alignas(16) DevCtl {
  int32_t stop;        // stopping rule fired during the current host call
  int32_t breakdown;   // sticky: kBreakdown (normalisation breakdown) or kRangeError
  int32_t gate;        // dual gate of the latest primal step
  int32_t degenerate;  // init: a = ||X_c||_2 is zero or not finite
  int64_t t_done;      // completed primal steps
  int64_t rows_run;    // one-pass iterations whose row work ran in its own pass first
  float c_f;           // lazy scale of the factor buffer (1 when materialised)
  float x_scale;       // power of two keeping |Xhat| x_scale < 2^15 (split-fp16 products)
  float th_scale;      // power of two keeping |Theta| th_scale < 2^15 (panel pass B operand)
  int32_t rows_first;  // one-pass iteration: the row pass runs before the pass -- 1 the stop may
                       // fire (s from the Gram terms), 2 no Gram terms yet (s from the rows)
  double a, b, h;      // fused statistics of the latest primal step
  double Delta;        // squared movement estimate
  double delta;        // movement estimate
  double rho;          // ||q||/sqrt(n) of the current factor
  double objective;    // fhat at the start of the latest iteration
  double theta_fro2;
  double spectral_a;   // ||X_c||_2
  double c_gram;       // scale c of the factor whose Gram terms are stored (one-pass iteration)
};

// Scalars of one iteration, passed by value.
struct StepArgs {
  float alpha_f;       // alpha
  float two_alpha_f;   // 2 alpha
  float gamma_f;       // beta / n (the implementation's penalty on the stored dual)
  float pad;
  double beta;
  double eps_d;
  double eps_c;
  double K;
  double inv_n;
  int64_t T_min;
  int32_t end_work;    // apply the pending end-of-iteration vector work (dual step, rho, stop test)
  int32_t pad32;
};

// Launch geometry; a pure function of (n, d, r) so that reduction orders,
// and therefore results, do not depend on the device.
struct Geometry {
  int64_t n;
  int32_t d, r, K;
  int32_t d32, r32;     // d, r rounded up to multiples of 32
  int32_t MB, NB;       // 32-wide blocks of d and r
  // pass A
  int32_t MBG, NBG;     // m-blocks (1, 2 or 4) / n-blocks (1, 2, 4, 5 or 7) per workgroup group
  int32_t mgroups, ngroups;
  int32_t GA;           // row-chunk workgroups per group
  int64_t tilesA;       // ceil(n / kTPA)
  int32_t xs_stride, us_stride;
  int32_t a_rows;       // 1: register-resident pass A (k_pass_a_rows)
  int32_t a_fv, a_ngf, a_cv;  // its features per lane, feature groups, columns per lane
  // reduce theta
  int32_t RT;
  int32_t SA, SB;       // segments of the two-level partial sums
  // pass B
  int32_t GB;
  int64_t tilesB;       // ceil(n / kTPB)
  int32_t nch;          // 32-feature chunks of d
  int32_t theta_lds;    // 1: Theta staged whole in LDS
  int32_t b_res;        // 1: resident-tile pass B (k_pass_b_res)
  int32_t split_a, split_b;  // 1: split-fp16 products in pass A / pass B
  int32_t fused;        // 1: single-Xhat-pass iteration (row pass + fused pass B)
  int32_t uflat;        // 1: the fused pass B moves U as whole 32-row slabs (r % 4 != 0)
  int32_t fused8;       // 1: the fused pass B in its eight-wave form (k_pass_bf8), one-pass iteration
  int32_t theta_cols;   // floats per row of the Theta partials: d32 r32 (+ r32 r32 of W^T W, one-pass)
  int32_t SAF;          // segments of the fused pass B Theta partials (GB rows)
  int32_t ldsB_bytes;
  // init
  int32_t GI;           // row-chunk workgroups of the init reductions
  int32_t GG;           // row-chunk workgroups of the Gram partials
  int32_t gblk;         // 32-wide blocks of d for the Gram
  int32_t vec_x, vec_u; // 16-byte vector loads allowed on X / U rows
  int32_t GAF;          // workgroups of the finish pass (generic pass A form)
  // split-fp16 panel form (large d x r, two passes)
  int32_t panel;        // 1: k_pass_a_panel / k_pass_b_panel iteration
  int32_t pnbw;         // 32-column blocks per column wave (1, 2 or 4): 64 pnbw columns
  int32_t pfb;          // 256-feature blocks of pass A
  int32_t PS;           // row splits of pass A
  int32_t GPA;          // pass A workgroups (PS pfb: groups of 8 splits on one XCD each, then the rest)
  int64_t tilesP;       // 128-row tiles of pass B
  float su;             // power-of-two scale of U in the split (|u| <= sqrt(K))
};

// Pointers into caller memory and the workspace.
struct Bufs {
  float* X;            // n x d (Xhat after init)
  float* U;            // n x r
  float* y;            // n (stored dual)
  DevCtl* ctl;
  nlr_iter_stats* hist;   // kHistCap records
  float* theta;        // d32*r32, pass-B operand layout
  float* p;            // r32
  float* s;            // r32
  float* theta_part;   // rows of theta_cols floats (GA, GB or PS rows)
  double* a_part;      // GA x (4 + r32): ||q||^2, ytilde^T q, -, -, s partials
  double* seg_theta;   // SA x d32*r32: segment sums of theta_part
  double* seg_a;       // SA x (4 + r32)
  double* seg_b;       // SB x (4 + r32)
  double* th2_part;    // RT
  double* b_part;      // GB x (4 + r32): a, b, h, -, column sums
  float* dump;         // 256 bytes that masked-off lanes store to (never read)
  float* thmax_part;   // RT: per-workgroup max |Theta| of the reduction
  float* ybar;         // n: ybar of the current iteration (panel form: pass A -> pass B)
  void* theta_split;   // panel form: split Theta^T chunks, 64 bytes per (16 features, column)
  // one-pass iteration (eight-wave fused pass B)
  double* gram_vec;    // 3 r32: column sums P of W, W^T ytilde, (W^T W) P (fixed-order sums)
  // init temporaries (alias the pass-A partial region)
  double* i_colsum;    // GI x d
  double* i_xbar;      // d
  double* i_gram;      // GG x d x d
  double* i_C;         // d x d
  double* i_B0;        // d x d
  double* i_B1;        // d x d
  double* i_scal;      // 2*(kSquarings+2)
  double* i_proj;      // GI x (4 + r32)
  // data-informed start (FP64, not aliased)
  double* s_C;         // d x d: Xhat^T Xhat
  double* s_M;         // d x r: Xhat^T Z
  double* s_CM;        // d x r
  double* s_G;         // r x r: M^T C M, then its Cholesky factor L (lower)
  double* s_T;         // d x r: M L^{-T}
};

// Scratch of the spectral label recovery (carved from the Theta-partial region,
// which is free between host calls).
struct LabScratch {
  int32_t GU;          // row chunks of the U^T U partials
  int32_t GA2;         // row chunks of the assignment pass
  double* gpart;       // GU x r x r
  double* A;           // r x r: U^T U, diagonalised in place
  double* V;           // r x r: eigenvectors
  double* P;           // r x K: V_K Lambda_K^(-1/2)
  double* cent;        // K x K centroids
  double* apart;       // GA2 x (K*K + K + 1): cluster sums, counts, changed labels
  int64_t* seeds;      // K seed rows
  int32_t* flag;       // [0] degenerate spectrum, [1] changed labels of the last pass
};
constexpr int kLabMaxK = 128;
size_t lab_scratch_bytes(int64_t n, int32_t r, int32_t K);
LabScratch carve_lab_scratch(int64_t n, int32_t r, int32_t K, char* base);

// aligned16: X and U start on 16-byte boundaries (enables the vector-load kernels)
// split: split-fp16 products requested (NLR_INIT_SPLIT_F16)
Geometry make_geometry(int64_t n, int32_t d, int32_t r, int32_t K, bool aligned16, bool split = false,
                       bool fused = false);
// dynamic LDS of the fused pass B for (NB, nch, split, U moved as whole slabs)
int fused_lds_need(int NB, int nch, bool split, bool uflat);
bool fused8_shape(int NB, int nch, int r);
// generic pass A above 128 columns: a row-work launch (GAF workgroups streaming rows
// of U, storing ybar) and a Theta launch whose workgroups stage only their own columns
__host__ __device__ inline bool pass_a_split(const Geometry& g) { return !g.a_rows && g.r32 > 128; }
constexpr int kMaxFusedLds = 160 << 10;
size_t carve_workspace(const Geometry& g, char* base, Bufs* out);  // base may be null (size only)

// ---- kernel launchers (each returns the launch error) ----
hipError_t launch_ctl_init(const Bufs& b, float gamma_f, hipStream_t st);
hipError_t launch_clear_stop(const Bufs& b, hipStream_t st);
hipError_t launch_colsum(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_gram(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_spectral(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_normalise(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_project(const Geometry& g, const Bufs& b, double K, int in_omega, hipStream_t st);
hipError_t launch_zero_y(const Geometry& g, const Bufs& b, hipStream_t st);

hipError_t launch_pass_a(const Geometry& g, const Bufs& b, const StepArgs& a, bool finish,
                         hipStream_t st);
hipError_t launch_pass_u(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st);
// fused_partials: the partials are Xhat^T W from the fused pass B (GB rows, scaled by c_f)
hipError_t launch_reduce_theta(const Geometry& g, const Bufs& b, bool fused_partials, hipStream_t st);
hipError_t launch_pass_bf(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st);
hipError_t launch_seg_a(const Geometry& g, const Bufs& b, bool finish, hipStream_t st);
hipError_t launch_seg_b(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_ctl_a(const Geometry& g, const Bufs& b, const StepArgs& a, bool finish,
                        hipStream_t st);
hipError_t launch_pass_b(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st);
hipError_t launch_ctl_b(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st);
hipError_t launch_xscale(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_split_x(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_pass_b_split(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st);
hipError_t launch_seg_theta(const Geometry& g, const Bufs& b, int64_t rows, int nseg, hipStream_t st);
hipError_t launch_data_start(const Geometry& g, const Bufs& b, const StepArgs& a0, bool x_normalised,
                             hipStream_t st);
hipError_t launch_lab_embed(const Geometry& g, const Bufs& b, const LabScratch& L, int K, hipStream_t st);
hipError_t launch_lab_pass(const Geometry& g, const Bufs& b, const LabScratch& L, int K, int32_t* labels,
                           int first, hipStream_t st);
hipError_t launch_labels(const Geometry& g, const Bufs& b, int32_t* labels, hipStream_t st);
hipError_t launch_pass_a_panel(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st);
hipError_t launch_theta_split_panel(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_pass_b_panel(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st);
hipError_t launch_split_x8(const Geometry& g, const Bufs& b, hipStream_t st);
// a_part rows written by the latest producer (pass A grid, finish grid or panel splits)
hipError_t launch_seg_a_rows(const Geometry& g, const Bufs& b, int64_t rows, bool finish, hipStream_t st);
hipError_t launch_ctl_one(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st);
hipError_t launch_seg_onepass(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_seg_fused(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_reduce_theta_fused(const Geometry& g, const Bufs& b, hipStream_t st);
hipError_t launch_reduce_theta_onepass(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st);
// start of a host call of the one-pass iteration: s from the stored Gram terms (when
// valid) and whether the first iteration's row pass runs before its pass
hipError_t launch_onepass_begin(const Geometry& g, const Bufs& b, const StepArgs& a, bool gram_valid,
                                hipStream_t st);
hipError_t launch_reduce_theta_rows(const Geometry& g, const Bufs& b, int64_t rows, int nseg, bool scaled,
                                    hipStream_t st);

// ---- device helpers ----
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// D += A * B on the 32x32x2 fp32 matrix core.  Lane l supplies A[l%32][l/32]
// and B[l/32][l%32]; lane l, register v of D holds D[8(v/4)+4(l/32)+v%4][l%32].
__device__ __forceinline__ f32x16 mfma32x32x2(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ double shfl_xor_d(double v, int mask) {
  return __shfl_xor(v, mask, 64);
}
__device__ __forceinline__ float shfl_xor_f(float v, int mask) {
  return __shfl_xor(v, mask, 64);
}

// Fixed-order sum of one double per thread over a 256-thread workgroup.
// Result valid in thread 0.  `red` must hold 4 doubles of shared memory.
__device__ __forceinline__ double block_sum_d(double v, double* red) {
  for (int m = 32; m >= 1; m >>= 1) v += shfl_xor_d(v, m);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0) r = ((red[0] + red[1]) + red[2]) + red[3];
  __syncthreads();
  return r;
}

}  // namespace nlr
