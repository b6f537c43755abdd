// Panel kernels of the split-fp16 two-pass iteration for large d x r (gfx950).
//
// When Theta (d x r) is too large for one workgroup to hold -- the
// single-Xhat-pass form keeps all of Xhat^T W in registers and the resident pass
// B all of Theta in LDS -- the two products of an iteration (Algorithm 1;
// Theta = Xhat^T U, then Xhat Theta with the epilogue of eq. (entrywise-fusion))
// run as LDS-tiled panel products on the 32x32x16 fp16 matrix cores with the
// two-term split of both operands (v s = hi + lo, three products hi*lo, lo*hi,
// hi*hi accumulated in fp32).
//
// Operands reach LDS by direct global-to-LDS loads (global_load_lds_dwordx4:
// each lane moves 16 bytes, a wave instruction fills 1 KiB of LDS), several
// stages ahead of the matrix cores, so no registers are spent on staging.  The
// waits are explicit: before a stage is read, each wave waits until its own
// loads of that stage have landed (vmcnt, loads complete in issue order) and a
// workgroup barrier makes the other waves' loads visible.  The LDS images are
// swizzled at 16-byte granularity so that the operand reads are free of bank
// conflicts; the swizzle is chosen by the global addresses each lane loads from.
//
// Pass A (k_pass_a_panel): workgroup (split s, feature block j) of 8 waves
// accumulates Theta[256 j .. 256 j + 255][all columns] over the rows of split s,
// 16 rows per stage.  Xhat arrives split (stored so since initialisation: every 32
// bytes that held 8 features hold their 8 fp16 hi halves, then their 8 lo
// halves); U arrives as fp32 and is scaled (u = fl(c_f w), the lazy
// normalisation), split and written as fp16 hi/lo slabs; both are read with the
// transposing ds_read_b64_tr_b16.  The workgroups of feature block 0 also do the
// row work that ends the previous iteration and starts this one (q = u.p - 1,
// the gated dual step, ybar, s = U^T ybar, ||q||^2, ytilde^T q) and store ybar
// for pass B.  The feature blocks of one split are launched on the same XCD
// (workgroup ids congruent mod 8) and stream the same U rows at the same time,
// so U is fetched from HBM about once.
//
// Pass B (k_pass_b_panel): workgroups of 2 WR waves over 64 WR-row tiles (one 8-wave
// workgroup per compute unit at 128 columns per column wave, else two of 4 waves),
// 16 features per stage: Theta^T chunks (split and laid out once
// per iteration by k_theta_split_panel) and Xhat row chunks in LDS, then the
// epilogue on the accumulators: w = max(u + 2 alpha G - alpha ybar p - alpha s, 0),
// FP64 a = ||W||^2, b = ||U||^2, h = <W, U>, column sums of W, W stored over U.
#include "k_common.hpp"

namespace nlr {

typedef _Float16 pf16x4 __attribute__((ext_vector_type(4)));
typedef __fp16 ph16x4 __attribute__((__vector_size__(4 * sizeof(__fp16))));
typedef __attribute__((address_space(3))) void lds_void_t;

// 16 bytes per lane from global memory to LDS: lane l writes lds_wave_base + 16 l.
__device__ __forceinline__ void dma16(const void* src, unsigned char* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(src, (lds_void_t*)lds_wave_base, 16, 0, 0);
}
// 4 bytes per lane: lane l writes lds_wave_base + 4 l.
__device__ __forceinline__ void dma4(const void* src, unsigned char* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(src, (lds_void_t*)lds_wave_base, 4, 0, 0);
}

// Wait until at most N vector memory operations of this wave are outstanding and
// its LDS operations are done, then a workgroup barrier.  Written as one asm
// block so that no memory access is moved across it.
template <int N>
__device__ __forceinline__ void wait_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// wait_barrier<n> for a run-time n (values above 31 wait for more than needed: still correct)
__device__ __forceinline__ void wait_barrier_n(int n) {
  switch (n < 31 ? (n < 0 ? 0 : n) : 31) {
#define NLR_WB(k) case k: wait_barrier<k>(); break;
    NLR_WB(0) NLR_WB(1) NLR_WB(2) NLR_WB(3) NLR_WB(4) NLR_WB(5) NLR_WB(6) NLR_WB(7)
    NLR_WB(8) NLR_WB(9) NLR_WB(10) NLR_WB(11) NLR_WB(12) NLR_WB(13) NLR_WB(14) NLR_WB(15)
    NLR_WB(16) NLR_WB(17) NLR_WB(18) NLR_WB(19) NLR_WB(20) NLR_WB(21) NLR_WB(22) NLR_WB(23)
    NLR_WB(24) NLR_WB(25) NLR_WB(26) NLR_WB(27) NLR_WB(28) NLR_WB(29) NLR_WB(30)
#undef NLR_WB
    default: wait_barrier<31>(); break;
  }
}

__device__ __forceinline__ pf16x4 lds_tr16(const _Float16* p) {
  ph16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4f16((__attribute__((address_space(3))) ph16x4*)(p));
  pf16x4 o;
  o[0] = (_Float16)v[0];
  o[1] = (_Float16)v[1];
  o[2] = (_Float16)v[2];
  o[3] = (_Float16)v[3];
  return o;
}

// ===========================================================================
// Pass A
// ===========================================================================
// LDS banks: 64 banks of 4 bytes.  A ds_read_b128 is served 16 lanes at a time
// and a ds_read_b64_tr_b16 32 lanes at a time (256 bytes each); the swizzles
// below give every such group 256 distinct bytes.
constexpr int kPAXStages = 4;   // Xhat ring: loads three stages ahead
constexpr int kPAUStages = 5;   // U ring: a slot also holds its stage's split U until it is read
constexpr int kPAPts = 16;      // rows (points) per stage = one k-step of the 32x32x16 product
constexpr int kPAFeat = 256;    // features per workgroup block
constexpr int kPAThreads = 512;

template <int NBW>
struct PanelA {
  static constexpr int RC = 64 * NBW;                 // columns: two column waves x 32 NBW
  static constexpr int XB = kPAPts * kPAFeat * 4;     // Xhat rows of a stage (split, 1 KiB per row)
  static constexpr int UB = kPAPts * RC * 4;          // U rows of a stage (fp32, then split in place)
  static constexpr int UBP = UB + kPAPts * 4;         // U slot: the U rows, then ytilde of the rows
  static constexpr int XI = XB / 1024;                // 1 KiB load instructions per stage: Xhat
  static constexpr int UI = UB / 1024;                //                                    U
  static constexpr int OPS_X = XI / 8;                // Xhat loads per wave and stage (exact)
  static constexpr int LPP = RC / 8;                  // threads per row in the conversion
  static constexpr int XR = kPAXStages * XB;          // Xhat ring
  static constexpr int UR = kPAUStages * UBP;         // U ring
  static constexpr int LDS = XR + UR + 16 * 8 + RC * 4 + 32;  // rings, reduction, p, dump
  static_assert(XI % 8 == 0, "equal Xhat loads per wave");
  static_assert(UI * 1024 == UB, "U stage in whole KiB");
  static_assert(RC / 4 >= 16, "a U row spans at least 16 pieces (swizzle)");
  static_assert(kPAPts * RC / 8 <= kPAThreads, "one conversion unit per thread");
  static_assert(kPAPts * RC * 8 <= XR + UR, "s combine fits the rings");
};

// 16-byte piece P of row R of a pass-A stage sits in slot P ^ pa_swz(R).  Xhat rows:
// P = 2 unit + (0 hi, 1 lo) of 8 features.  U rows: first P = fp32 columns 4P .. 4P + 3,
// then, split in place, P = 2 unit + (0 hi, 1 lo) of columns 8 unit .. 8 unit + 7 (the
// two pieces of a unit stay in the two slots that held its fp32 values).
__device__ __forceinline__ int pa_swz(int R) { return (R & 1) | ((R & 2) << 2); }

// LDS byte address of this lane's first transposing read of a 32x32x16 operand with
// k = row, from a pass-A stage image at byte offset `base` (rows of `row_bytes`, pieces
// swizzled as above); the second read is 4 rows further.  Together they give lane l
// T[8 (l/32) + e][c0 + l%32] (hi or lo), e = 0..7.
__device__ __forceinline__ uint32_t pa_operand_addr(uint32_t base, int row_bytes, int c0, int hl, int lane) {
  const int gq = lane >> 4, s16 = lane & 15;
  const int R = 8 * (gq >> 1) + (s16 >> 2);  // and R + 4 (same swizzle)
  const int c = c0 + 16 * (gq & 1) + 4 * (s16 & 3);
  const int slot = (2 * (c >> 3) + hl) ^ pa_swz(R);
  return base + (uint32_t)(R * row_bytes + slot * 16 + ((c >> 2) & 1) * 8);
}

__device__ __forceinline__ f16x8 pa_join(pf16x4 a, pf16x4 b) {
  return (f16x8){a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// The transposing reads of one pass-A stage, written as assembly: the compiler treats
// the ds_read_b64_tr_b16 builtin as a possible reader of every global-to-LDS load in
// flight and waits for all of them first, which would empty the load ring every stage.
// One statement issues the reads and waits for their data (lgkmcnt(0)), so its outputs
// are defined only when they hold the data.  X: xa[i][hl] (8 reads, rows 4 apart = XO
// bytes); U: ua[cb][hl] (4 NBW reads, UO bytes).
#define PA_TR(o, a) "ds_read_b64_tr_b16 %" #o ", %" #a "\n\t"
#define PA_TRO(o, a, f) "ds_read_b64_tr_b16 %" #o ", %" #a " offset:%" #f "\n\t"
template <int NBW, int XO, int UO>
__device__ __forceinline__ void pa_stage_reads(const uint32_t (&xa)[2][2], const uint32_t (&ua)[NBW][2],
                                               f16x8 (&ah)[2], f16x8 (&al)[2], f16x8 (&bh)[NBW],
                                               f16x8 (&bl)[NBW]) {
  pf16x4 x0, x1, x2, x3, x4, x5, x6, x7;
  if constexpr (NBW == 1) {
    pf16x4 u0, u1, u2, u3;
    asm volatile(PA_TR(0, 12) PA_TRO(1, 12, 18) PA_TR(2, 13) PA_TRO(3, 13, 18)
                 PA_TR(4, 14) PA_TRO(5, 14, 18) PA_TR(6, 15) PA_TRO(7, 15, 18)
                 PA_TR(8, 16) PA_TRO(9, 16, 19) PA_TR(10, 17) PA_TRO(11, 17, 19)
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(x0), "=&v"(x1), "=&v"(x2), "=&v"(x3), "=&v"(x4), "=&v"(x5), "=&v"(x6), "=&v"(x7),
                   "=&v"(u0), "=&v"(u1), "=&v"(u2), "=&v"(u3)
                 : "v"(xa[0][0]), "v"(xa[0][1]), "v"(xa[1][0]), "v"(xa[1][1]), "v"(ua[0][0]), "v"(ua[0][1]),
                   "n"(XO), "n"(UO)
                 : "memory");
    bh[0] = pa_join(u0, u1);
    bl[0] = pa_join(u2, u3);
  } else {
    // the Xhat reads are issued first and complete with the U reads' wait below
    asm volatile(PA_TR(0, 8) PA_TRO(1, 8, 12) PA_TR(2, 9) PA_TRO(3, 9, 12)
                 PA_TR(4, 10) PA_TRO(5, 10, 12) PA_TR(6, 11) PA_TRO(7, 11, 12)
                 : "=&v"(x0), "=&v"(x1), "=&v"(x2), "=&v"(x3), "=&v"(x4), "=&v"(x5), "=&v"(x6), "=&v"(x7)
                 : "v"(xa[0][0]), "v"(xa[0][1]), "v"(xa[1][0]), "v"(xa[1][1]), "n"(XO)
                 : "memory");
    if constexpr (NBW == 2) {
      pf16x4 u0, u1, u2, u3, u4, u5, u6, u7;
      asm volatile(PA_TR(0, 16) PA_TRO(1, 16, 20) PA_TR(2, 17) PA_TRO(3, 17, 20)
                   PA_TR(4, 18) PA_TRO(5, 18, 20) PA_TR(6, 19) PA_TRO(7, 19, 20)
                   "s_waitcnt lgkmcnt(0)"
                   : "=&v"(u0), "=&v"(u1), "=&v"(u2), "=&v"(u3), "=&v"(u4), "=&v"(u5), "=&v"(u6), "=&v"(u7),
                     "+v"(x0), "+v"(x1), "+v"(x2), "+v"(x3), "+v"(x4), "+v"(x5), "+v"(x6), "+v"(x7)
                   : "v"(ua[0][0]), "v"(ua[0][1]), "v"(ua[1][0]), "v"(ua[1][1]), "n"(UO)
                   : "memory");
      bh[0] = pa_join(u0, u1);
      bl[0] = pa_join(u2, u3);
      bh[1] = pa_join(u4, u5);
      bl[1] = pa_join(u6, u7);
    } else {
      static_assert(NBW == 4, "NBW");
      pf16x4 u[16];
      asm volatile(PA_TR(0, 24) PA_TRO(1, 24, 32) PA_TR(2, 25) PA_TRO(3, 25, 32)
                   PA_TR(4, 26) PA_TRO(5, 26, 32) PA_TR(6, 27) PA_TRO(7, 27, 32)
                   PA_TR(8, 28) PA_TRO(9, 28, 32) PA_TR(10, 29) PA_TRO(11, 29, 32)
                   PA_TR(12, 30) PA_TRO(13, 30, 32) PA_TR(14, 31) PA_TRO(15, 31, 32)
                   "s_waitcnt lgkmcnt(0)"
                   : "=&v"(u[0]), "=&v"(u[1]), "=&v"(u[2]), "=&v"(u[3]), "=&v"(u[4]), "=&v"(u[5]),
                     "=&v"(u[6]), "=&v"(u[7]), "=&v"(u[8]), "=&v"(u[9]), "=&v"(u[10]), "=&v"(u[11]),
                     "=&v"(u[12]), "=&v"(u[13]), "=&v"(u[14]), "=&v"(u[15]),
                     "+v"(x0), "+v"(x1), "+v"(x2), "+v"(x3), "+v"(x4), "+v"(x5), "+v"(x6), "+v"(x7)
                   : "v"(ua[0][0]), "v"(ua[0][1]), "v"(ua[1][0]), "v"(ua[1][1]), "v"(ua[2][0]),
                     "v"(ua[2][1]), "v"(ua[3][0]), "v"(ua[3][1]), "n"(UO)
                   : "memory");
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        bh[cb] = pa_join(u[4 * cb + 0], u[4 * cb + 1]);
        bl[cb] = pa_join(u[4 * cb + 2], u[4 * cb + 3]);
      }
    }
  }
  ah[0] = pa_join(x0, x1);
  al[0] = pa_join(x2, x3);
  ah[1] = pa_join(x4, x5);
  al[1] = pa_join(x6, x7);
}

// Workgroup (split s, feature block j), 8 waves: wave w holds features 64 (w % 4) .. + 63
// of the block and column half w / 4.  Stage t covers rows p0 + 16 t ..; its loads
// (Xhat of stage t, U of stage t + 1) are issued three stages ahead, and the U of
// stage t + 1 is scaled and split (in its ring slot) while the matrix cores work on
// stage t.  The row work of stage t is done by the workgroup with j = t mod (number
// of blocks), so the feature blocks of a split do equal work and stream the same U
// rows at about the same time (they share an XCD: workgroup ids congruent mod 8).
template <int NBW>
__global__ __launch_bounds__(kPAThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_pass_a_panel(
    Geometry g, Bufs B, StepArgs S) {
  using P = PanelA<NBW>;
  if (halted(B.ctl)) return;
  // full groups of eight splits (the blocks of a split congruent mod 8: one XCD), then
  // a partial group of q splits (blocks congruent mod q) on the compute units left over
  const int per = 8 * g.pfb;
  const int full = (g.PS / 8) * per;
  int fb, sp;
  if ((int)blockIdx.x < full) {
    const int grp = blockIdx.x / per;
    const int rem = blockIdx.x - grp * per;
    fb = rem >> 3;
    sp = grp * 8 + (rem & 7);
  } else {
    const int q = g.PS % 8;
    const int rem = blockIdx.x - full;
    fb = rem / q;
    sp = (g.PS / 8) * 8 + rem % q;
  }
  if (sp >= g.PS || fb >= g.pfb) return;

  extern __shared__ __align__(16) unsigned char smem_raw[];
  unsigned char* xring = smem_raw;
  unsigned char* uring = smem_raw + P::XR;
  double* dred = reinterpret_cast<double*>(smem_raw + P::XR + P::UR);
  float* ps = reinterpret_cast<float*>(smem_raw + P::XR + P::UR + 16 * 8);  // p (RC)
  f32x4* ldump = reinterpret_cast<f32x4*>(ps + P::RC);                     // 32 bytes never read
  // LDS byte address of the dynamic area (operand of the assembly reads)
  const uint32_t lds_base =
      (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) unsigned char*)smem_raw);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int fw = wave & 3;
  const int cw = wave >> 2;
  const int64_t n = g.n;
  const int d = g.d, r = g.r;
  const int nfb = g.pfb;
  const float cf = B.ctl->c_f;
  const float su = g.su;
  const bool gate = (S.end_work != 0) && (B.ctl->gate != 0);
  const float gam = S.gamma_f;

  const int64_t p0 = (int64_t)sp * n / g.PS;
  const int64_t p1 = (int64_t)(sp + 1) * n / g.PS;
  const int nst = (int)((p1 - p0 + kPAPts - 1) / kPAPts);

  // conversion unit of this thread: row cr of a stage, columns 8 cu .. 8 cu + 7
  const bool conv = tid < kPAPts * P::LPP;
  const int ct = tid % (kPAPts * P::LPP);  // threads beyond the units repeat one (split only)
  const int cr = ct / P::LPP;
  const int cu = ct - cr * P::LPP;
  const int cc = 8 * cu;
  for (int c = tid; c < P::RC; c += kPAThreads) ps[c] = (c < g.r32) ? B.p[c] : 0.f;  // published by the prologue barrier
  double s_acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) s_acc[e] = 0.0;
  double qq = 0.0, yq = 0.0;

  f32x16 acc[2][NBW];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NBW; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // loads of group t: Xhat of stage t (if t >= 0) and U of stage t + 1 (if it exists)
  auto issue_group = [&](int t) {
    int ln = lane;  // opaque: per-lane offsets are formed here, not kept across the loop
    asm volatile("" : "+v"(ln));
    if (t >= 0) {
      unsigned char* xs = xring + (t % kPAXStages) * P::XB;
      const float* xb = B.X + (p0 + (int64_t)t * kPAPts) * (int64_t)d;
      const int rmax = (int)((p1 - 1) - (p0 + (int64_t)t * kPAPts));
#pragma unroll
      for (int q = 0; q < P::OPS_X; ++q) {
        const int i = wave + 8 * q;  // Xhat row i of the stage
        const int R = i < rmax ? i : rmax;
        const int pc = ln ^ pa_swz(i);
        int unit = fb * (kPAFeat / 8) + (pc >> 1);
        if (8 * unit >= d) unit = 0;  // features >= d: any finite data of the row
        dma16(xb + (R * d + 8 * unit + 4 * (pc & 1)), xs + i * 1024);
      }
    }
    const int tu = t + 1;
    if (tu < nst) {
      unsigned char* us = uring + (tu % kPAUStages) * P::UBP;
      const float* ub = B.U + (p0 + (int64_t)tu * kPAPts) * (int64_t)r;
      const int rmax = (int)((p1 - 1) - (p0 + (int64_t)tu * kPAPts));
#pragma unroll
      for (int q = 0; q < (P::UI + 7) / 8; ++q) {
        const int i = wave + 8 * q;
        if (i < P::UI) {
          const int q4 = 64 * i + ln;               // 16-byte slot of the stage
          const int rr = q4 / (P::RC / 4);
          const int col = 4 * ((q4 - rr * (P::RC / 4)) ^ pa_swz(rr));  // its piece's columns
          const int R = rr < rmax ? rr : rmax;
          dma16(ub + (R * r + (col < r ? col : 0)), us + i * 1024);
        }
      }
      // ytilde of the stage's rows (the row work reads it from LDS: a global load there
      // would have to wait for every ring load issued before it)
      if (wave == 0 && ln < kPAPts) {
        const int R = ln < rmax ? ln : rmax;
        dma4(B.y + (p0 + (int64_t)tu * kPAPts + R), us + P::UB);
      }
    }
  };

  // this thread's 8 values of stage t's U (scaled by c_f, the lazy normalisation)
  auto load_u8 = [&](int t, float (&u)[8], bool& vrow) {
    const float* urow = reinterpret_cast<const float*>(uring + (t % kPAUStages) * P::UBP) + cr * P::RC;
    const f32x4 a0 = reinterpret_cast<const f32x4*>(urow)[(2 * cu) ^ pa_swz(cr)];
    const f32x4 a1 = reinterpret_cast<const f32x4*>(urow)[(2 * cu + 1) ^ pa_swz(cr)];
    const float raw[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
    const int64_t row = p0 + (int64_t)t * kPAPts + cr;
    vrow = row < p1;
#pragma unroll
    for (int e = 0; e < 8; ++e) u[e] = (vrow && cc + e < r) ? raw[e] * cf : 0.f;
  };
  // split stage t's U in place; branch-free, so it can share a block with the products
  // (threads beyond the conversion units repeat one's arithmetic and store to a dump slot:
  // the split is not idempotent, so only the unit's own thread may rewrite it)
  auto split_u = [&](int t) {
    float u[8];
    bool vrow;
    load_u8(t, u, vrow);
    f16x8 hi, lo;
    split_f16(u, su, hi, lo);
    f32x4* urow = reinterpret_cast<f32x4*>(uring + (t % kPAUStages) * P::UBP + cr * P::RC * 4);
    *(conv ? urow + ((2 * cu) ^ pa_swz(cr)) : ldump) = __builtin_bit_cast(f32x4, hi);
    *(conv ? urow + ((2 * cu + 1) ^ pa_swz(cr)) : ldump + 1) = __builtin_bit_cast(f32x4, lo);
  };
  // the row work of stage t (this block's share): reads the fp32 U before it is split
  auto row_work = [&](int t) {
    if (!conv) return;
    float u[8];
    bool vrow;
    load_u8(t, u, vrow);
    const f32x4 p0v = *reinterpret_cast<const f32x4*>(ps + cc);
    const f32x4 p1v = *reinterpret_cast<const f32x4*>(ps + cc + 4);
    const float pr[8] = {p0v.x, p0v.y, p0v.z, p0v.w, p1v.x, p1v.y, p1v.z, p1v.w};
    double dot = 0.0;
#pragma unroll
    for (int e = 0; e < 8; ++e) dot += (double)u[e] * (double)pr[e];
#pragma unroll
    for (int m = 1; m < P::LPP; m <<= 1) dot += shfl_xor_d(dot, m);
    if (vrow) {
      const int64_t row = p0 + (int64_t)t * kPAPts + cr;
      const float q = (float)(dot - 1.0);
      float yt = reinterpret_cast<const float*>(uring + (t % kPAUStages) * P::UBP + P::UB)[cr];
      const bool lead = cu == 0;
      if (gate) {
        yt = fmaf(gam, q, yt);
        if (lead) B.y[row] = yt;
      }
      const float ybar = fmaf(gam, q, yt);
      if (lead) {
        B.ybar[row] = ybar;
        qq += (double)q * (double)q;
        yq += (double)yt * (double)q;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) s_acc[e] = fma((double)ybar, (double)u[e], s_acc[e]);
    }
  };

  // loads this wave issues for group t (t < nst): its Xhat rows, and if stage t + 1
  // exists its U rows and (wave 0) the ytilde of those rows
  const int ops_u = P::UI / 8 + (wave < P::UI % 8 ? 1 : 0) + (wave == 0 ? 1 : 0);
  auto group_ops = [&](int t) { return P::OPS_X + (t + 1 < nst ? ops_u : 0); };

  // prologue: groups -1 (U of stage 0) .. 2; wait for group -1, split U of stage 0
  issue_group(-1);
  for (int t = 0; t < 3 && t < nst; ++t) issue_group(t);
  {
    int newer = 0;  // loads of groups 0 .. 2, issued after group -1
    for (int t = 0; t < 3 && t < nst; ++t) newer += group_ops(t);
    wait_barrier_n(newer);
  }
  if (0 % nfb == fb) row_work(0);
  split_u(0);

  for (int st = 0; st < nst; ++st) {
    // group st (Xhat of stage st, U of stage st + 1) has landed once at most the loads
    // of groups st + 1 and st + 2 (issued after it) are pending; U of stage st is split
    int newer = 0;
    if (st + 1 < nst) newer += group_ops(st + 1);
    if (st + 2 < nst) newer += group_ops(st + 2);
    wait_barrier_n(newer);
    if (st + 3 < nst) issue_group(st + 3);

    // ---- Theta block += Xhat_stage^T U_stage ----
    int x_off = (st % kPAXStages) * P::XB;  // opaque: addresses formed per stage
    asm volatile("" : "+s"(x_off));
    int u_off = (st % kPAUStages) * P::UBP;
    asm volatile("" : "+s"(u_off));
    const uint32_t xbase = lds_base + (uint32_t)x_off;
    const uint32_t ubase = lds_base + (uint32_t)(P::XR + u_off);
    uint32_t xa[2][2], ua[NBW][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int hl = 0; hl < 2; ++hl) xa[i][hl] = pa_operand_addr(xbase, kPAFeat * 4, 64 * fw + 32 * i, hl, lane);
#pragma unroll
    for (int cb = 0; cb < NBW; ++cb)
#pragma unroll
      for (int hl = 0; hl < 2; ++hl) ua[cb][hl] = pa_operand_addr(ubase, P::RC * 4, (P::RC / 2) * cw + 32 * cb, hl, lane);
    f16x8 ah[2], al[2], bh[NBW], bl[NBW];
    pa_stage_reads<NBW, 4 * kPAFeat * 4, 4 * P::RC * 4>(xa, ua, ah, al, bh, bl);
    // the next stage's row work (reads its fp32 U), then its split, which shares this
    // block with the products (on the last stage it rewrites a slot no one reads)
    if (st + 1 < nst && (st + 1) % nfb == fb) row_work(st + 1);
    split_u(st + 1);
#pragma unroll
    for (int cb = 0; cb < NBW; ++cb)
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        acc[i][cb] = mfma32x32x16h(ah[i], bl[cb], acc[i][cb]);
        acc[i][cb] = mfma32x32x16h(al[i], bh[cb], acc[i][cb]);
        acc[i][cb] = mfma32x32x16h(ah[i], bh[cb], acc[i][cb]);
      }
  }
  __syncthreads();

  // ---- Theta partial of this split: rows of this feature block ----
  {
    const float unscale = (1.0f / B.ctl->x_scale) * (1.0f / su);
    float* part = B.theta_part + (int64_t)sp * g.theta_cols;
    const int h = lane >> 5, li = lane & 31;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int cb = 0; cb < NBW; ++cb) {
        const int c = (P::RC / 2) * cw + 32 * cb + li;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int f = kPAFeat * fb + 64 * fw + 32 * i + 8 * (v >> 2) + 4 * h + (v & 3);
          if (f < g.d32 && c < g.r32) part[(int64_t)f * g.r32 + c] = acc[i][cb][v] * unscale;
        }
      }
  }

  // ---- row partials of this workgroup's share: ||q||^2, ytilde^T q, s ----
  {
    double* ap = B.a_part + ((int64_t)sp * nfb + fb) * (4 + g.r32);
    double* sred = reinterpret_cast<double*>(smem_raw);  // kPAPts x RC (the rings are free now)
    if (conv)
#pragma unroll
      for (int e = 0; e < 8; ++e) sred[cr * P::RC + cc + e] = s_acc[e];  // (conv: cr, cc are the thread's own)
    const double tq = block_sum8_d(qq, dred);  // its barriers also publish sred
    const double ty = block_sum8_d(yq, dred);
    if (tid == 0) {
      ap[0] = tq;
      ap[1] = ty;
      ap[2] = ap[3] = 0.0;
    }
    for (int c = tid; c < g.r32; c += kPAThreads) {
      double t = 0.0;
      for (int k = 0; k < kPAPts; ++k) t += sred[k * P::RC + c];
      ap[4 + c] = t;
    }
  }
}

// ===========================================================================
// Theta for pass B: split hi/lo of Theta * s_theta in the pass-B LDS image
// ===========================================================================

template <int NBW, int WR>
struct PanelB {
  static constexpr int ROWS = 64 * WR;            // rows per tile: WR row waves x 64
  static constexpr int NT = 128 * WR;             // threads: WR row waves x 2 column waves
  static constexpr int NW = NT / 64;
  static constexpr int RC = 64 * NBW;             // columns of the two column waves
  static constexpr int TH = RC * 64;              // Theta^T chunk: per column 16 features hi + lo
  static constexpr int XB = ROWS * 64;            // Xhat chunk: per row 16 features split
  static constexpr int STAGE = TH + XB;
  static constexpr int INSTR = STAGE / 1024;
  static constexpr int OPS = INSTR / NW;          // per wave
  static constexpr int STAGES = 3;  // ring of stages: loads two stages ahead
  static constexpr int LDS = STAGES * STAGE + 2 * RC * 4 + (WR * RC + 8) * 8;
  static_assert(INSTR % NW == 0, "equal share of the loads per wave");
};

// Stage k of the Theta image: column c owns 64 bytes = four 16-byte pieces
// P = 2 hl + j (features 16k + 8j .. 16k + 8j + 7, hl = 0 hi / 1 lo), piece P in
// slot P ^ ((c >> 2) & 3).
__global__ __launch_bounds__(kThreads) void k_theta_split_panel(Geometry g, Bufs B, int RC) {
  if (halted(B.ctl)) return;
  __shared__ float red[4];
  float m = 0.f;
  for (int k = threadIdx.x; k < g.RT; k += kThreads) m = fmaxf(m, B.thmax_part[k]);
  for (int k = 32; k >= 1; k >>= 1) m = fmaxf(m, shfl_xor_f(m, k));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  const float sth = f16_range_scale(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])));
  if (blockIdx.x == 0 && threadIdx.x == 0) B.ctl->th_scale = sth;
  const int nk = (g.d + 15) >> 4;
  const int64_t rec = (int64_t)blockIdx.x * kThreads + threadIdx.x;  // (stage, column)
  if (rec >= (int64_t)nk * RC) return;
  const int k = (int)(rec / RC);
  const int c = (int)(rec - (int64_t)k * RC);
  float v[16];
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    const int f = 16 * k + t;
    float x = 0.f;
    if (f < g.d && c < g.r32) {
      const int ch = f >> 5, fin = f & 31;
      const int hh = fin >> 4, j = (fin & 15) >> 2, ee = fin & 3;
      const int mbk = c >> 5, l = hh * 32 + (c & 31);
      x = B.theta[((((int64_t)ch * 4 + j) * g.NB + mbk) * 64 + l) * 4 + ee];
    }
    v[t] = x;
  }
  f16x8 h0, l0, h1, l1;
  split_f16(v, sth, h0, l0);
  split_f16(v + 8, sth, h1, l1);
  f16x8* out = reinterpret_cast<f16x8*>(reinterpret_cast<unsigned char*>(B.theta_split) + rec * 64);
  const int sw = (c >> 2) & 3;
  out[0 ^ sw] = h0;  // P = 0: hi, features 0..7
  out[1 ^ sw] = h1;  // P = 1: hi, features 8..15
  out[2 ^ sw] = l0;  // P = 2: lo, features 0..7
  out[3 ^ sw] = l1;  // P = 3: lo, features 8..15
}

// ===========================================================================
// Pass B
// ===========================================================================
// Row R of a pass-B Xhat chunk: piece P = 2 unit + hl in slot P ^ ((R >> 2) & 3).
// WR row waves of 64 rows (2 WR waves): WR = 2, two 4-wave workgroups per compute unit;
// WR = 4, one 8-wave workgroup per compute unit, so that each staged Theta chunk serves
// twice the rows (half the Theta traffic from L2 per row).
template <int NBW, int WR>
__global__ __launch_bounds__(128 * WR) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_pass_b_panel(
    Geometry g, Bufs B, StepArgs S) {
  using P = PanelB<NBW, WR>;
  constexpr int kPBRows = P::ROWS;
  constexpr int kPBThreads = P::NT;
  constexpr int kPBStages = P::STAGES;
  if (halted(B.ctl)) return;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  unsigned char* ring = smem_raw;
  float* ps = reinterpret_cast<float*>(smem_raw + kPBStages * P::STAGE);
  float* ss = ps + P::RC;
  double* colred = reinterpret_cast<double*>(ss + P::RC);  // WR x RC
  double* dred = colred + WR * P::RC;                      // 8

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int wr = wave >> 1;  // 64-row part of the tile
  const int cw = wave & 1;   // column half
  const int h = lane >> 5;
  const int li = lane & 31;
  const int64_t n = g.n;
  const int d = g.d, r = g.r;
  const int nk = (d + 15) >> 4;
  const float cf = B.ctl->c_f;
  const float two_alpha_s = S.two_alpha_f * (1.0f / B.ctl->x_scale) * (1.0f / B.ctl->th_scale);
  const float neg_alpha = -S.alpha_f;

  for (int c = tid; c < P::RC; c += kPBThreads) {
    ps[c] = (c < g.r32) ? B.p[c] : 0.f;
    ss[c] = (c < g.r32) ? B.s[c] : 0.f;
  }

  const int64_t T = g.tilesP;
  const int G = gridDim.x;
  const int my_tiles = ((int64_t)blockIdx.x < T) ? (int)((T - 1 - blockIdx.x) / G + 1) : 0;
  const int total = my_tiles * nk;  // stages of this workgroup, over all its tiles

  // issue cursor: next stage to load (feature chunk ik of the tile at row ir0) and its ring slot
  int ik = 0, islot = 0, issued = 0;
  int64_t ir0 = (int64_t)blockIdx.x * kPBRows;
  auto issue_next = [&]() {
    unsigned char* slot = ring + islot * P::STAGE;
    // uniform bases plus 32-bit per-lane offsets (no 64-bit per-lane addresses to keep)
    const unsigned char* tb = reinterpret_cast<const unsigned char*>(B.theta_split) + (int64_t)ik * P::TH;
    const float* xb = B.X + ir0 * (int64_t)d;
    const int rmax = (n - 1 - ir0) < (kPBRows - 1) ? (int)(n - 1 - ir0) : (kPBRows - 1);
    int ln = lane;  // opaque: per-lane offsets are formed here, not kept across the loop
    asm volatile("" : "+v"(ln));
#pragma unroll
    for (int q = 0; q < P::OPS; ++q) {
      const int i = wave + P::NW * q;
      const void* src;
      if (i < P::TH / 1024) {
        src = tb + (i * 1024 + ln * 16);
      } else {
        const int R = 16 * (i - P::TH / 1024) + (ln >> 2);
        const int pc = (ln & 3) ^ ((R >> 2) & 3);
        const int Rc = R < rmax ? R : rmax;  // rows >= n: the last row (masked later)
        int unit = 2 * ik + (pc >> 1);
        if (8 * unit >= d) unit = 0;  // features >= d meet zero rows of Theta
        src = xb + (Rc * d + 8 * unit + 4 * (pc & 1));
      }
      dma16(src, slot + i * 1024);
    }
    ++issued;
    if (++ik == nk) {
      ik = 0;
      ir0 += (int64_t)G * kPBRows;
    }
    if (++islot == kPBStages) islot = 0;
  };

  for (int q = 0; q < kPBStages - 1 && q < total; ++q) issue_next();

  double sa = 0.0, sb = 0.0, sh = 0.0;
  double colacc[NBW];
#pragma unroll
  for (int m = 0; m < NBW; ++m) colacc[m] = 0.0;
  int base = 0;
  if (li & 16) base += 8;
  if (li & 8) base += 4;
  if (li & 4) base += 2;
  if (li & 2) base += 1;

  int gs = 0, rslot = 0;  // stage being consumed and its ring slot
  for (int ti = 0; ti < my_tiles; ++ti) {
    const int64_t row0 = ((int64_t)blockIdx.x + (int64_t)ti * G) * kPBRows;
    f32x16 acc[2][NBW];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < NBW; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    for (int k = 0; k < nk; ++k, ++gs) {
      // this wave's loads of stage gs have landed once at most those of stage gs + 1 are pending
      if (issued > gs + 1) wait_barrier<P::OPS>();
      else wait_barrier<0>();
      if (issued < total) issue_next();
      // opaque slot offset: the operand addresses are formed per stage instead of
      // being precomputed for every ring slot (which would not fit in registers)
      int slot_off = rslot * P::STAGE;
      asm volatile("" : "+s"(slot_off));
      if (++rslot == kPBStages) rslot = 0;
      const unsigned char* slot = ring + slot_off;
      f16x8 ah[NBW], al[NBW];
#pragma unroll
      for (int cb = 0; cb < NBW; ++cb) {
        const int c = (P::RC / 2) * cw + 32 * cb + li;
        const int sw = (c >> 2) & 3;
        ah[cb] = *reinterpret_cast<const f16x8*>(slot + c * 64 + ((h ^ sw) << 4));
        al[cb] = *reinterpret_cast<const f16x8*>(slot + c * 64 + (((2 + h) ^ sw) << 4));
      }
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int R = 64 * wr + 32 * i + li;
        const int sw = (R >> 2) & 3;
        const unsigned char* xb = slot + P::TH + R * 64;
        const f16x8 bh = *reinterpret_cast<const f16x8*>(xb + (((2 * h) ^ sw) << 4));
        const f16x8 bl = *reinterpret_cast<const f16x8*>(xb + (((2 * h + 1) ^ sw) << 4));
#pragma unroll
        for (int cb = 0; cb < NBW; ++cb) {
          acc[i][cb] = mfma32x32x16h(ah[cb], bl, acc[i][cb]);
          acc[i][cb] = mfma32x32x16h(al[cb], bh, acc[i][cb]);
          acc[i][cb] = mfma32x32x16h(ah[cb], bh, acc[i][cb]);
        }
      }
    }

    // ---- epilogue (eq. entrywise-fusion) on rows row0 + 64 wr + 32 i + li ----
    // blocks (i, cb) in order; the U loads of the next block are issued before
    // the arithmetic of the current one (scheduling barriers keep it that way)
    f32x4 ubuf[2][4];
    auto load_u = [&](int bi, f32x4 (&dst)[4]) {
      const int i = bi / NBW, cb = bi - (bi / NBW) * NBW;
      const int64_t pt = row0 + 64 * wr + 32 * i + li;
      const float* urow = B.U + (pt < n ? pt : 0) * (int64_t)r;
      const int cbase = (P::RC / 2) * cw + 32 * cb;
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int c = cbase + 8 * qd + 4 * h;
        dst[qd] = *reinterpret_cast<const f32x4*>(urow + (c < r ? c : 0));
      }
    };
    // opaque zero offset: the p and s addresses are formed per tile rather than
    // held in registers across the loop
    int lds_off = 0;
    asm volatile("" : "+v"(lds_off));
    const float* psl = ps + lds_off;
    const float* ssl = ss + lds_off;
    // per-lane column offsets and masks are likewise formed per tile (an opaque lane id)
    int lane_o = lane;
    asm volatile("" : "+v"(lane_o));
    const int h = lane_o >> 5, li = lane_o & 31;
    __builtin_amdgcn_sched_barrier(0);
    load_u(0, ubuf[0]);
    float yb2[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int64_t pt = row0 + 64 * wr + 32 * i + li;
      yb2[i] = pt < n ? B.ybar[pt] : 0.f;
    }
#pragma unroll
    for (int bi = 0; bi < 2 * NBW; ++bi) {
      const int i = bi / NBW, cb = bi - (bi / NBW) * NBW;
      __builtin_amdgcn_sched_barrier(0);
      if (bi + 1 < 2 * NBW) load_u(bi + 1, ubuf[(bi + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
      const int64_t pt = row0 + 64 * wr + 32 * i + li;
      const bool vpt = pt < n;
      float* urow = B.U + (vpt ? pt : 0) * (int64_t)r;
      const float yb = yb2[i];
      const int cbase = (P::RC / 2) * cw + 32 * cb;
      float wv[16];
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int c = cbase + 8 * qd + 4 * h;
        const bool ok = vpt && c < r;  // r % 4 == 0: four columns valid together
        const f32x4 pv = *reinterpret_cast<const f32x4*>(psl + c);
        const f32x4 sv = *reinterpret_cast<const f32x4*>(ssl + c);
        const f32x4 uv = ubuf[bi & 1][qd];
        const float ue[4] = {uv.x, uv.y, uv.z, uv.w};
        const float pe[4] = {pv.x, pv.y, pv.z, pv.w};
        const float se[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float uu = ok ? ue[e] * cf : 0.f;
          float t = fmaf(two_alpha_s, acc[i][cb][4 * qd + e], uu);
          t = fmaf(neg_alpha, yb * pe[e], t);
          t = fmaf(neg_alpha, se[e], t);
          float w = fmaxf(t, 0.f);
          if (!ok) w = 0.f;
          wv[4 * qd + e] = w;
          const double wd = (double)w, ud = (double)uu;
          sa = fma(wd, wd, sa);
          sb = fma(ud, ud, sb);
          sh = fma(wd, ud, sh);
        }
        const f32x4 o = {wv[4 * qd + 0], wv[4 * qd + 1], wv[4 * qd + 2], wv[4 * qd + 3]};
        *reinterpret_cast<f32x4*>(ok ? (urow + c) : B.dump) = o;
      }
      reduce_scatter<16, 16>(wv, li);
      colacc[cb] += (double)wv[0];
    }
    __builtin_amdgcn_sched_barrier(0);
  }

  // ---- statistics of this workgroup ----
  __syncthreads();
  for (int c = tid; c < WR * P::RC; c += kPBThreads) colred[c] = 0.0;
  __syncthreads();
#pragma unroll
  for (int cb = 0; cb < NBW; ++cb) {
    const double v = colacc[cb] + shfl_xor_d(colacc[cb], 1);
    if ((li & 1) == 0) {
      const int col = (P::RC / 2) * cw + 32 * cb + 8 * (base >> 2) + 4 * h + (base & 3);
      colred[wr * P::RC + col] = v;
    }
  }
  __syncthreads();
  double* out = B.b_part + (int64_t)blockIdx.x * (4 + g.r32);
  for (int c = tid; c < g.r32; c += kPBThreads) {
    double t = colred[c] + colred[P::RC + c];
    if (WR == 4) t = t + (colred[2 * P::RC + c] + colred[3 * P::RC + c]);
    out[4 + c] = t;
  }
  const double ta = WR == 4 ? block_sum8_d(sa, dred) : block_sum_d(sa, dred);
  const double tb2 = WR == 4 ? block_sum8_d(sb, dred) : block_sum_d(sb, dred);
  const double th = WR == 4 ? block_sum8_d(sh, dred) : block_sum_d(sh, dred);
  if (tid == 0) {
    out[0] = ta;
    out[1] = tb2;
    out[2] = th;
    out[3] = 0.0;
  }
}

// ===========================================================================
// Split storage of Xhat for the panel kernels: every 32 bytes (8 features) hold
// the 8 fp16 hi halves, then the 8 lo halves, of x * x_scale.
// ===========================================================================
__global__ __launch_bounds__(kThreads) void k_split_x8(Bufs B, int64_t units) {
  const float s = B.ctl->x_scale;
  for (int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x; u < units; u += (int64_t)gridDim.x * kThreads) {
    f32x4* p = reinterpret_cast<f32x4*>(B.X) + 2 * u;
    const f32x4 a = p[0], b = p[1];
    const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    f16x8 hi, lo;
    split_f16(x, s, hi, lo);
    p[0] = __builtin_bit_cast(f32x4, hi);
    p[1] = __builtin_bit_cast(f32x4, lo);
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <int NBW>
static hipError_t pass_a_panel_launch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  constexpr int lds = PanelA<NBW>::LDS;
  static_assert(lds <= (160 << 10), "LDS");
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pass_a_panel<NBW>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_pass_a_panel<NBW>, dim3(g.GPA), dim3(kPAThreads), lds, st, g, b, a);
  return hipGetLastError();
}

template <int NBW, int WR>
static hipError_t pass_b_panel_launch(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  using P = PanelB<NBW, WR>;
  constexpr int lds = P::LDS;
  static_assert(WR == 4 || lds <= (80 << 10), "two workgroups per compute unit");
  static_assert(lds <= (160 << 10), "LDS");
  if (g.tilesP != (g.n + P::ROWS - 1) / P::ROWS) return hipErrorInvalidValue;  // geometry mismatch
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pass_b_panel<NBW, WR>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_pass_b_panel<NBW, WR>), dim3(g.GB), dim3(P::NT), lds, st, g, b, a);
  return hipGetLastError();
}

hipError_t launch_pass_a_panel(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  switch (g.pnbw) {
    case 1: return pass_a_panel_launch<1>(g, b, a, st);
    case 2: return pass_a_panel_launch<2>(g, b, a, st);
    case 4: return pass_a_panel_launch<4>(g, b, a, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_theta_split_panel(const Geometry& g, const Bufs& b, hipStream_t st) {
  const int RC = 64 * g.pnbw;
  const int64_t recs = (int64_t)((g.d + 15) / 16) * RC;
  hipLaunchKernelGGL(k_theta_split_panel, dim3((unsigned)((recs + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                     st, g, b, RC);
  return hipGetLastError();
}

hipError_t launch_pass_b_panel(const Geometry& g, const Bufs& b, const StepArgs& a, hipStream_t st) {
  switch (g.pnbw) {
    case 1: return pass_b_panel_launch<1, 2>(g, b, a, st);
    case 2: return pass_b_panel_launch<2, 2>(g, b, a, st);
    case 4: return pass_b_panel_launch<4, 4>(g, b, a, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_split_x8(const Geometry& g, const Bufs& b, hipStream_t st) {
  const int64_t units = g.n * (int64_t)g.d / 8;  // d % 8 == 0
  hipLaunchKernelGGL(k_split_x8, dim3(4096), dim3(kThreads), 0, st, b, units);
  return hipGetLastError();
}

int panel_lds_a(int nbw) {
  return nbw == 1 ? PanelA<1>::LDS : nbw == 2 ? PanelA<2>::LDS : PanelA<4>::LDS;
}

}  // namespace nlr
