// Host controller behind the C ABI of include/nlr.h: argument validation,
// launch geometry, workspace layout and the iteration state machine.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "nlr.h"
#include "nlr_internal.hpp"

namespace nlr {

static int32_t round_up(int32_t x, int32_t m) { return (x + m - 1) / m * m; }
static int32_t next_pow2(int32_t x) {
  int32_t p = 1;
  while (p < x) p <<= 1;
  return p;
}
static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }


Geometry make_geometry(int64_t n, int32_t d, int32_t r, int32_t K, bool aligned16, bool split, bool fused) {
  Geometry g;
  std::memset(&g, 0, sizeof(g));
  g.n = n;
  g.d = d;
  g.r = r;
  g.K = K;
  g.d32 = round_up(d, 32);
  g.MB = g.d32 / 32;
  // 1, 2, 4 or 8 column blocks; above 256 columns an even number (10, 12, 14), which
  // the two-pass kernels take in groups of two blocks
  g.NB = r <= 256 ? next_pow2((r + 31) / 32) : 2 * ((r + 63) / 64);
  g.r32 = 32 * g.NB;
  // pass A groups: MBG in {1, 2, 4}, NBG in {1, 2, 4, 5, 7} dividing NB; 10 and 14 blocks
  // (above 256 columns, where the product runs in a launch of its own) in two groups
  g.MBG = g.MB >= 3 ? 4 : g.MB;
  g.NBG = g.NB % 4 == 0 ? 4 : (g.NB % 2 == 0 ? 2 : 1);
  if (g.NB == 10 || g.NB == 14) g.NBG = g.NB / 2;
  g.mgroups = (g.MB + g.MBG - 1) / g.MBG;
  g.ngroups = (g.NB + g.NBG - 1) / g.NBG;
  g.tilesA = (n + kTPA - 1) / kTPA;
  {
    const int64_t part_bytes = (int64_t)g.d32 * g.r32 * 4;
    int64_t lim = (int64_t)64 << 20;
    int64_t ga = lim / part_bytes;
    // above 128 columns the product is a launch of its own (two workgroups per compute
    // unit): one full round of them, without a partial second round
    if (g.r32 > 128) ga = 512 / (g.mgroups * g.ngroups);
    if (ga < 16) ga = 16;
    if (ga > 1024) ga = 1024;
    if (ga > g.tilesA) ga = g.tilesA;
    g.GA = (int32_t)ga;
  }
  g.xs_stride = g.MBG * 32;
  g.us_stride = g.r32 + 4;
  // register-resident pass A (16x16x4 blocks): all of Theta in one wave, FV*NGF*CV <= 32
  {
    int fv = 1;
    while (fv < 4 && 16 * fv < d) fv <<= 1;
    if (d % fv != 0) fv = (fv == 4 && d % 2 == 0) ? 2 : 1;  // even d: 8-byte loads
    const int ngf = (d + 16 * fv - 1) / (16 * fv);
    int cv = 1;
    while (cv < 4 && 16 * cv < r) cv <<= 1;
    const bool fits = (16 * cv >= r) && (r % cv == 0);
    const int key = fv * 100 + ngf * 10 + cv;
    const bool known = key == 111 || key == 112 || key == 114 || key == 211 || key == 212 || key == 214 ||
                       key == 221 || key == 222 || key == 224 || key == 241 || key == 242 || key == 244 ||
                       key == 411 || key == 412 || key == 414 ||
                       key == 421 || key == 422 || key == 424;
    g.a_rows = (known && fits && aligned16) ? 1 : 0;
    g.a_fv = fv;
    g.a_ngf = ngf;
    g.a_cv = cv;
    if (g.a_rows) {
      // at least 32 four-row steps per wave, at most 1024 workgroups
      int64_t ga = (((n + 3) / 4) + 4 * 32 - 1) / (4 * 32);
      if (ga > 1024) ga = 1024;
      if (ga < 1) ga = 1;
      g.GA = (int32_t)ga;
    }
  }
  g.SA = (g.GA + 31) / 32;
  if (g.SA > 64) g.SA = 64;
  g.RT = (int32_t)(((int64_t)g.d32 * g.r32 + kThreads - 1) / kThreads);
  g.tilesB = (n + kTPB - 1) / kTPB;
  g.GB = (int32_t)(g.tilesB < 1536 ? g.tilesB : 1536);
  g.nch = g.d32 / 32;
  // Theta resident in pass B's LDS when it fits beside p, s and the reductions in 64 KiB
  g.theta_lds = ((int64_t)g.d32 * g.r32 * 4 + 2 * g.r32 * 4 + (4 * g.r32 + 8) * 8 <= (64 << 10)) ? 1 : 0;
  // the streamed pass B (Theta from L2 through LDS, 16-byte rows): one persistent round of
  // two workgroups per compute unit
  if (!g.theta_lds && aligned16 && d % 4 == 0 && r % 4 == 0 && g.GB > 512) g.GB = 512;
  g.b_res = (g.nch <= 4 && g.NB <= 4 && g.NB * g.nch <= 8 && g.theta_lds && d % 4 == 0 && r % 4 == 0 &&
             aligned16) ? 1 : 0;
  g.ldsB_bytes = (int32_t)((g.theta_lds ? (int64_t)g.d32 * g.r32 * 4 : 0) + 2 * g.r32 * 4 +
                           (4 * g.r32 + 8) * 8);
  g.SB = (g.GB + 31) / 32;
  if (g.SB > 64) g.SB = 64;
  // init reductions
  {
    int64_t gi = (n + 255) / 256;
    if (gi > 512) gi = 512;
    g.GI = (int32_t)gi;
    const int64_t dd8 = (int64_t)d * d * 8;
    int64_t gg = ((int64_t)64 << 20) / (dd8 > 0 ? dd8 : 1);
    // every Gram workgroup resident at once: four per compute unit (their LDS), 256
    // units, shared by the chunks of all nb (nb + 1) / 2 block pairs -- a second,
    // partial wave of workgroups would take as long as the first (2e6 x 768: 14 chunks
    // x 78 pairs, 34.5 ms; 13 chunks, 29.6 ms).  At most 256 chunks: more resident
    // workgroups do not shorten the 128-feature Gram and lengthen its reduction.
    const int64_t nbk = (d + 63) / 64;
    const int64_t resident = 1024 / (nbk * (nbk + 1) / 2);
    if (gg > resident) gg = resident;
    if (gg > 256) gg = 256;
    if (gg < 1) gg = 1;
    const int64_t t64 = (n + 63) / 64;
    if (gg > t64) gg = t64;
    g.GG = (int32_t)gg;
    g.gblk = g.d32 / 32;
  }
  // single-Xhat-pass iteration: the row pass and the fused pass B need the
  // register-resident shapes (d <= 128, r <= 64, 16-byte aligned X and U rows of
  // X; U rows of any length move as whole slabs) and its LDS; one persistent
  // workgroup per compute unit
  // (fp32 products also for even d: X rows then move in 8-byte pieces; the split X stays
  // in 16-byte units of 4 features per row, so split products need d % 4 == 0)
  const bool shape_f = aligned16 && d <= 128 && r <= 64 && (d % 4 == 0 || (!split && d % 2 == 0)) && g.a_rows;
  const bool uflat = r % 4 != 0;
  g.fused = (fused && shape_f && fused_lds_need(g.NB, g.nch, split, uflat) <= kMaxFusedLds) ? 1 : 0;
  g.uflat = (g.fused && uflat) ? 1 : 0;
  g.fused8 = (g.fused && split && fused8_shape(g.NB, g.nch, r)) ? 1 : 0;
  // the one-pass iteration's W^T W partials follow its Theta partials in one row
  g.theta_cols = g.d32 * g.r32 + (g.fused8 ? g.r32 * g.r32 : 0);
  g.SAF = g.SA;
  if (g.fused) {
    // persistent grid: one workgroup per CU; two for the shapes whose kernel holds two
    // workgroups' waves (the four-wave form with one column block and <= 64 features; the
    // one-pass form with one column block and <= 32 features: 73 KiB of LDS, 128 VGPRs)
    const int64_t gmax = (g.NB == 1 && (g.fused8 ? g.nch == 1 : g.nch <= 2)) ? 512 : 256;
    g.GB = (int32_t)(g.tilesB < gmax ? g.tilesB : gmax);
    g.SB = (g.GB + 31) / 32;
    g.SAF = (g.GB + 31) / 32;
    g.split_a = g.split_b = split ? 1 : 0;  // both products live in the fused pass B
  } else {
    // two-pass form: split products in the resident pass B only
    g.split_a = 0;
    g.split_b = (split && g.b_res && aligned16 && d <= 128 && r <= 64 && d % 4 == 0 && r % 4 == 0) ? 1 : 0;
  }
  g.vec_x = (d % 4 == 0 && aligned16) ? 1 : 0;
  g.vec_u = (r % 4 == 0 && aligned16) ? 1 : 0;
  // finish pass of the generic form: no Theta partials, so a grid for the rows alone
  g.GAF = g.a_rows ? g.GA : (int32_t)(g.tilesA < 1024 ? g.tilesA : 1024);
  // split-fp16 panel form: the shapes the single-pass and resident kernels do not take
  g.panel = 0;
  if (split && !g.fused && !g.split_b && aligned16 && d % 8 == 0 && r % 4 == 0 && r <= kMaxPanelR) {
    g.panel = 1;
    g.pnbw = g.NB >= 2 ? g.NB / 2 : 1;
    g.pfb = (d + 255) / 256;
    // one 8-wave workgroup per compute unit; the feature blocks of a split on one XCD,
    // then splits whose blocks are spread over XCDs on the compute units left over
    int64_t ps = 8 * (256 / (8 * g.pfb));
    ps += (256 - ps * g.pfb) / g.pfb;
    const int64_t cap = n / 64 > 1 ? n / 64 : 1;  // at least four 16-row stages per split
    if (ps > cap) ps = cap;
    if (ps < 1) ps = 1;
    g.PS = (int32_t)ps;
    g.GPA = g.PS * g.pfb;
    // pass B: 256-row tiles in one 8-wave workgroup per compute unit at 128 columns per
    // column wave (pnbw = 4), else 128-row tiles in two 4-wave workgroups per compute unit
    const int prow = g.pnbw == 4 ? 256 : 128;
    const int64_t pgrid = g.pnbw == 4 ? 256 : 512;
    g.tilesP = (n + prow - 1) / prow;
    g.GB = (int32_t)(g.tilesP < pgrid ? g.tilesP : pgrid);
    g.SB = (g.GB + 31) / 32;
    // |u| <= sqrt(K) for U in Omega (||U||_F^2 = K); 1% margin for rounding
    int e2;
    (void)std::frexp(1.01 * std::sqrt((double)K), &e2);
    g.su = (float)std::ldexp(1.0, 15 - e2);
  }
  return g;
}

static int32_t lab_gu(int64_t n, int32_t r) {
  int64_t gu = (n + 4095) / 4096;
  const int64_t cap = ((int64_t)16 << 20) / ((int64_t)r * r * 8);  // partials within 16 MiB
  if (gu > cap) gu = cap;
  if (gu > 64) gu = 64;
  return (int32_t)(gu < 1 ? 1 : gu);
}
static int32_t lab_ga2(int64_t n) {
  int64_t ga = (n + 63) / 64;
  return (int32_t)(ga > 256 ? 256 : (ga < 1 ? 1 : ga));
}

size_t lab_scratch_bytes(int64_t n, int32_t r, int32_t K) {
  const size_t rr = (size_t)r * r * 8;
  return align256((size_t)lab_gu(n, r) * rr) + 2 * align256(rr) + align256((size_t)r * K * 8) +
         align256((size_t)K * K * 8) + align256((size_t)lab_ga2(n) * ((size_t)K * K + K + 1) * 8) +
         align256((size_t)K * 8) + align256(64);
}

LabScratch carve_lab_scratch(int64_t n, int32_t r, int32_t K, char* base) {
  LabScratch L;
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    char* p = base + off;
    off += align256(bytes);
    return p;
  };
  const size_t rr = (size_t)r * r * 8;
  L.GU = lab_gu(n, r);
  L.GA2 = lab_ga2(n);
  L.gpart = reinterpret_cast<double*>(take((size_t)L.GU * rr));
  L.A = reinterpret_cast<double*>(take(rr));
  L.V = reinterpret_cast<double*>(take(rr));
  L.P = reinterpret_cast<double*>(take((size_t)r * K * 8));
  L.cent = reinterpret_cast<double*>(take((size_t)K * K * 8));
  L.apart = reinterpret_cast<double*>(take((size_t)L.GA2 * ((size_t)K * K + K + 1) * 8));
  L.seeds = reinterpret_cast<int64_t*>(take((size_t)K * 8));
  L.flag = reinterpret_cast<int32_t*>(take(64));
  return L;
}

size_t carve_workspace(const Geometry& g, char* base, Bufs* out) {
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    char* p = base ? base + off : nullptr;
    off += align256(bytes);
    return p;
  };
  Bufs b;
  std::memset(&b, 0, sizeof(b));
  const size_t d = (size_t)g.d, r32 = (size_t)g.r32;
  b.ctl = reinterpret_cast<DevCtl*>(take(sizeof(DevCtl)));
  b.hist = reinterpret_cast<nlr_iter_stats*>(take(sizeof(nlr_iter_stats) * kHistCap));
  b.theta = reinterpret_cast<float*>(take((size_t)g.d32 * r32 * 4));
  b.p = reinterpret_cast<float*>(take(r32 * 4));
  b.s = reinterpret_cast<float*>(take(r32 * 4));
  b.th2_part = reinterpret_cast<double*>(take((size_t)g.RT * 8));
  b.b_part = reinterpret_cast<double*>(take((size_t)g.GB * (4 + r32) * 8));
  int64_t arows = g.GA > g.GAF ? g.GA : g.GAF;
  if (g.panel && (int64_t)g.PS * g.pfb > arows) arows = (int64_t)g.PS * g.pfb;  // one row per pass-A workgroup
  if (g.fused8 && (int64_t)g.GB > arows) arows = g.GB;  // the one-pass iteration's row statistics
  b.a_part = reinterpret_cast<double*>(take((size_t)arows * (4 + r32) * 8));
  const size_t segs = (size_t)(g.SA > g.SAF ? g.SA : g.SAF);
  b.seg_theta = reinterpret_cast<double*>(take(segs * (size_t)g.theta_cols * 8));
  b.seg_a = reinterpret_cast<double*>(take((size_t)g.SA * (4 + r32) * 8));
  b.seg_b = reinterpret_cast<double*>(take((size_t)g.SB * (4 + r32) * 8));
  b.i_xbar = reinterpret_cast<double*>(take(d * 8));
  b.dump = reinterpret_cast<float*>(take(256));
  b.thmax_part = reinterpret_cast<float*>(take((size_t)g.RT * 4));
  if (g.fused8) b.gram_vec = reinterpret_cast<double*>(take(3 * r32 * 8));
  if (g.panel || pass_a_split(g)) b.ybar = reinterpret_cast<float*>(take((size_t)g.n * 4));
  if (g.panel) {
    b.theta_split = take((size_t)((g.d + 15) / 16) * 64 * g.pnbw * 64);
  }
  b.s_C = reinterpret_cast<double*>(take(d * d * 8));
  b.s_M = reinterpret_cast<double*>(take(d * (size_t)g.r * 8));
  b.s_CM = reinterpret_cast<double*>(take(d * (size_t)g.r * 8));
  b.s_G = reinterpret_cast<double*>(take((size_t)g.r * g.r * 8));
  b.s_T = reinterpret_cast<double*>(take(d * (size_t)g.r * 8));
  // union: pass-A Theta partials | init temporaries
  // rows of Theta partials: pass A's (also the init's pass A of the fused forms), or
  // the fused pass B's (the two-pass forms' pass B writes none)
  size_t prow = (size_t)g.GA;
  if (g.fused && (size_t)g.GB > prow) prow = (size_t)g.GB;
  if (g.panel && (size_t)g.PS > prow) prow = (size_t)g.PS;
  const size_t u_iter = align256(prow * (size_t)g.theta_cols * 4);
  size_t u_init = 0;
  u_init += align256((size_t)g.GI * d * 8);            // colsum
  u_init += align256((size_t)g.GG * d * d * 8);         // gram partials
  u_init += 3 * align256(d * d * 8);                    // C, B0, B1
  u_init += align256(2 * (kSquarings + 2) * 8);         // scal
  u_init += align256((size_t)g.GI * (4 + r32) * 8);     // projection partials
  // the spectral label recovery (between host calls) uses the same region
  const int32_t kmax = g.r < kLabMaxK ? g.r : kLabMaxK;
  const size_t u_lab = lab_scratch_bytes(g.n, g.r, kmax);
  size_t ubytes = u_iter > u_init ? u_iter : u_init;
  if (u_lab > ubytes) ubytes = u_lab;
  char* ub = take(ubytes);
  b.theta_part = reinterpret_cast<float*>(ub);
  if (base) {
    size_t o = 0;
    auto sub = [&](size_t bytes) -> char* {
      char* p = ub + o;
      o += align256(bytes);
      return p;
    };
    b.i_colsum = reinterpret_cast<double*>(sub((size_t)g.GI * d * 8));
    b.i_gram = reinterpret_cast<double*>(sub((size_t)g.GG * d * d * 8));
    b.i_C = reinterpret_cast<double*>(sub(d * d * 8));
    b.i_B0 = reinterpret_cast<double*>(sub(d * d * 8));
    b.i_B1 = reinterpret_cast<double*>(sub(d * d * 8));
    b.i_scal = reinterpret_cast<double*>(sub(2 * (kSquarings + 2) * 8));
    b.i_proj = reinterpret_cast<double*>(sub((size_t)g.GI * (4 + r32) * 8));
  }
  if (out) *out = b;
  return off;
}

}  // namespace nlr

using namespace nlr;

enum KernelKind {
  KK_PASS_A = 0,
  KK_REDUCE_THETA,
  KK_CTL_A,
  KK_PASS_B,
  KK_CTL_B,
  KK_FINISH,
  KK_CTL_FINISH,
  KK_PASS_U,
  KK_PASS_BF,
  KK_COUNT
};
static const char* kKernelNames[KK_COUNT] = {"pass_a", "reduce_theta", "ctl_a",  "pass_b", "ctl_b",
                                             "finish", "ctl_finish",   "pass_u", "pass_bf"};

struct nlr_ctx {
  Geometry g;
  Bufs b;
  hipStream_t stream;
  int device;
  nlr_params prm;
  bool pending;       // end-of-iteration work of the latest pass B not yet applied
  bool gram_valid;    // one-pass iteration: the Gram terms of the latest pass give the next s
  bool failed;        // sticky failure
  bool breakdown;
  bool range_error;   // the breakdown is a split-fp16 range error (NLR_ERANGE)
  int64_t t_host;     // last known iteration counter
  bool t_host_valid;
  DevCtl* host_ctl;   // pinned mirror of the control block
  // profiling
  bool prof;
  int prof_level;     // 1: every launch; 2: the row and pass kernels only
  std::vector<hipEvent_t> ev_pool;
  std::vector<std::pair<int, int>> ev_pairs;  // (kind, index of start event)
  size_t ev_used;
  double prof_ms[KK_COUNT];
  int64_t prof_n[KK_COUNT];
  // nlr_run replays the iterations after a call's first one as captured graphs (one
  // and eight iterations) while profiling is off: one submission instead of a launch
  // per kernel.  Captured on a private stream when first needed, dropped when the
  // step arguments change.
  bool graphs_allowed;  // false for the allocation-free entry point (instantiation allocates)
  hipStream_t cap_stream;
  hipGraphExec_t graph1, graph8;
  hipGraphExec_t lean1, lean8;  // one-pass iterations without the row pass (see enqueue_iteration)
};

static nlr_status hip_fail(nlr_ctx* c) {
  if (c) c->failed = true;
  return NLR_EHIP;
}

static bool params_ok(const nlr_params* p) {
  if (!p) return false;
  if (!(p->alpha > 0.0) || !std::isfinite(p->alpha)) return false;
  if (!(p->beta > 0.0) || !std::isfinite(p->beta)) return false;
  if (!(p->eps_d >= 0.0) || !(p->eps_c >= 0.0)) return false;
  if (std::isnan(p->eps_d) || std::isnan(p->eps_c)) return false;
  if (p->T_min < 0) return false;
  return true;
}

static bool shape_ok(int64_t n, int32_t d, int32_t r) {
  return n >= 1 && d >= 1 && d <= 4096 && r >= 1 && r <= n && n < ((int64_t)1 << 40);
}

static StepArgs make_step_args(const nlr_ctx* c, int end_work) {
  StepArgs a;
  std::memset(&a, 0, sizeof(a));
  a.alpha_f = (float)c->prm.alpha;
  a.two_alpha_f = (float)(2.0 * c->prm.alpha);
  a.gamma_f = (float)(c->prm.beta / (double)c->g.n);
  a.beta = c->prm.beta;
  a.eps_d = c->prm.eps_d;
  a.eps_c = c->prm.eps_c;
  a.K = (double)c->g.K;
  a.inv_n = 1.0 / (double)c->g.n;
  a.T_min = c->prm.T_min;
  a.end_work = end_work;
  return a;
}

// ---- profiling helpers ----
static bool pass_kernel(int kind) {
  return kind == KK_PASS_A || kind == KK_PASS_B || kind == KK_PASS_U || kind == KK_PASS_BF || kind == KK_FINISH;
}
static hipError_t grow_events(nlr_ctx* c, size_t want) {
  while (c->ev_pool.size() < want) {
    hipEvent_t e;
    hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) return err;
    c->ev_pool.push_back(e);
  }
  return hipSuccess;
}
static hipError_t prof_begin(nlr_ctx* c, int kind, int* slot) {
  *slot = -1;
  if (!c->prof) return hipSuccess;
  if (c->prof_level == 2 && !pass_kernel(kind)) return hipSuccess;
  if (c->ev_used + 2 > c->ev_pool.size()) {
    for (int k = 0; k < 64; ++k) {
      hipEvent_t e;
      hipError_t err = hipEventCreate(&e);
      if (err != hipSuccess) return err;
      c->ev_pool.push_back(e);
    }
  }
  *slot = (int)c->ev_used;
  c->ev_used += 2;
  c->ev_pairs.push_back({kind, *slot});
  return hipEventRecord(c->ev_pool[*slot], c->stream);
}
static hipError_t prof_end(nlr_ctx* c, int slot) {
  if (slot < 0) return hipSuccess;
  return hipEventRecord(c->ev_pool[slot + 1], c->stream);
}
static hipError_t prof_collect(nlr_ctx* c) {
  if (!c->prof || c->ev_pairs.empty()) return hipSuccess;
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return e;
  for (auto& pr : c->ev_pairs) {
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, c->ev_pool[pr.second], c->ev_pool[pr.second + 1]);
    if (e != hipSuccess) return e;
    c->prof_ms[pr.first] += ms;
    c->prof_n[pr.first] += 1;
  }
  c->ev_pairs.clear();
  c->ev_used = 0;
  return hipSuccess;
}

#define LAUNCH(kind, expr)                              \
  do {                                                  \
    int slot_;                                          \
    if (prof_begin(c, kind, &slot_) != hipSuccess)      \
      return hip_fail(c);                               \
    if ((expr) != hipSuccess) return hip_fail(c);       \
    if (prof_end(c, slot_) != hipSuccess)               \
      return hip_fail(c);                               \
  } while (0)

// first: the first iteration of a host call (nlr_step, nlr_run), whose step
// arguments may differ from those of the pass before it.  lean (one-pass form, not the
// first iteration): the caller knows that the previous iteration's stopping rule
// cannot fire (t < T_min), so the row pass, its segment sums and k_ctl_a would
// return at entry; they are not launched.
static nlr_status enqueue_iteration(nlr_ctx* c, bool first, bool lean = false) {
  const StepArgs a = make_step_args(c, c->pending ? 1 : 0);
  if (c->g.fused8) {
    // one pass over the rows per iteration, writing W over the factor: the pass does
    // the row work of the iteration (the end of the previous one) as well as the
    // primal step; s comes from the Gram terms of the previous pass (formed after that
    // pass with this call's step arguments, or anew at the start of a call).  When the
    // previous iteration's stopping rule may fire (decided on the device before the
    // pass), or there is no previous pass (after init or a stop), the row pass, its
    // segment sums and k_ctl_a run first (they return at entry otherwise) and settle
    // the rule and s.  Then one launch of segment sums (Theta and W^T W partials, the
    // row statistics), the control, and Theta with (W^T W) P and the next s.
    if (first) LAUNCH(KK_CTL_A, launch_onepass_begin(c->g, c->b, a, c->gram_valid, c->stream));
    if (first || !lean) {
      LAUNCH(KK_PASS_U, launch_pass_u(c->g, c->b, a, c->stream));
      LAUNCH(KK_CTL_A, launch_seg_a(c->g, c->b, false, c->stream));
      LAUNCH(KK_CTL_A, launch_ctl_a(c->g, c->b, a, false, c->stream));
    }
    LAUNCH(KK_PASS_BF, launch_pass_bf(c->g, c->b, a, c->stream));
    LAUNCH(KK_CTL_B, launch_seg_onepass(c->g, c->b, c->stream));
    LAUNCH(KK_CTL_B, launch_ctl_one(c->g, c->b, a, c->stream));
    LAUNCH(KK_REDUCE_THETA, launch_reduce_theta_onepass(c->g, c->b, a, c->stream));
    c->gram_valid = true;
    c->pending = true;
    return NLR_OK;
  }
  if (c->g.fused) {
    // row pass (end of the previous iteration, s, rho, objective terms), control,
    // fused pass B (W and the partials of Xhat^T W), control, Theta of the new factor
    LAUNCH(KK_PASS_U, launch_pass_u(c->g, c->b, a, c->stream));
    LAUNCH(KK_CTL_A, launch_seg_a(c->g, c->b, false, c->stream));
    LAUNCH(KK_CTL_A, launch_ctl_a(c->g, c->b, a, false, c->stream));
    LAUNCH(KK_PASS_BF, launch_pass_bf(c->g, c->b, a, c->stream));
    LAUNCH(KK_CTL_B, launch_seg_fused(c->g, c->b, c->stream));  // statistics and Theta segments
    LAUNCH(KK_CTL_B, launch_ctl_b(c->g, c->b, a, c->stream));
    LAUNCH(KK_REDUCE_THETA, launch_reduce_theta_fused(c->g, c->b, c->stream));
    c->pending = true;
    return NLR_OK;
  }
  if (c->g.panel) {
    // split-fp16 panel products (large d x r): pass A (with the row work, ybar
    // stored), Theta and its split operand, control, pass B, control
    LAUNCH(KK_PASS_A, launch_pass_a_panel(c->g, c->b, a, c->stream));
    LAUNCH(KK_REDUCE_THETA, launch_reduce_theta_rows(c->g, c->b, c->g.PS, c->g.SA, false, c->stream));
    LAUNCH(KK_REDUCE_THETA, launch_theta_split_panel(c->g, c->b, c->stream));
    LAUNCH(KK_CTL_A, launch_seg_a_rows(c->g, c->b, (int64_t)c->g.PS * c->g.pfb, false, c->stream));
    LAUNCH(KK_CTL_A, launch_ctl_a(c->g, c->b, a, false, c->stream));
    LAUNCH(KK_PASS_B, launch_pass_b_panel(c->g, c->b, a, c->stream));
    LAUNCH(KK_CTL_B, launch_seg_b(c->g, c->b, c->stream));
    LAUNCH(KK_CTL_B, launch_ctl_b(c->g, c->b, a, c->stream));
    c->pending = true;
    return NLR_OK;
  }
  LAUNCH(KK_PASS_A, launch_pass_a(c->g, c->b, a, false, c->stream));
  LAUNCH(KK_REDUCE_THETA, launch_reduce_theta(c->g, c->b, false, c->stream));
  LAUNCH(KK_CTL_A, launch_seg_a(c->g, c->b, false, c->stream));
  LAUNCH(KK_CTL_A, launch_ctl_a(c->g, c->b, a, false, c->stream));
  LAUNCH(KK_PASS_B, launch_pass_b(c->g, c->b, a, c->stream));
  LAUNCH(KK_CTL_B, launch_seg_b(c->g, c->b, c->stream));
  LAUNCH(KK_CTL_B, launch_ctl_b(c->g, c->b, a, c->stream));
  c->pending = true;
  return NLR_OK;
}

static void drop_graphs(nlr_ctx* c) {
  for (hipGraphExec_t* gp : {&c->graph1, &c->graph8, &c->lean1, &c->lean8}) {
    if (*gp) (void)hipGraphExecDestroy(*gp);
    *gp = nullptr;
  }
}

// Captures `iters` iterations that follow the first of a host call (their step
// arguments are fixed: the end-of-iteration work of the previous one is pending) as an
// executable graph.  The kernels read the device control block when they run, so a
// replay behaves as the same launches made one by one.  No memset is recorded.
static hipError_t capture_iterations(nlr_ctx* c, int iters, bool lean, hipGraphExec_t* out) {
  *out = nullptr;
  hipError_t e = hipSuccess;
  if (!c->cap_stream) {
    e = hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking);
    if (e != hipSuccess) return e;
  }
  const hipStream_t user = c->stream;
  c->stream = c->cap_stream;
  e = hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeRelaxed);
  if (e != hipSuccess) {
    c->stream = user;
    return e;
  }
  nlr_status s = NLR_OK;
  for (int k = 0; k < iters && s == NLR_OK; ++k) s = enqueue_iteration(c, false, lean);
  hipGraph_t graph = nullptr;
  e = hipStreamEndCapture(c->cap_stream, &graph);
  c->stream = user;
  if (s != NLR_OK && e == hipSuccess) e = hipErrorUnknown;
  if (e == hipSuccess) e = hipGraphInstantiate(out, graph, nullptr, nullptr, 0);
  if (graph) (void)hipGraphDestroy(graph);
  return e;
}

// Enqueues `nb` iterations that follow the first of the call: as graph replays when
// allowed and profiling is off (the events of profiling are per launch), else one by one.
static nlr_status enqueue_steady(nlr_ctx* c, int nb, bool lean) {
  lean = lean && c->g.fused8;
  if (c->graphs_allowed && !c->prof) {
    hipGraphExec_t& g1 = lean ? c->lean1 : c->graph1;
    hipGraphExec_t& g8 = lean ? c->lean8 : c->graph8;
    if (!g1 || !g8) {
      if (capture_iterations(c, 1, lean, &g1) != hipSuccess || capture_iterations(c, 8, lean, &g8) != hipSuccess) {
        drop_graphs(c);
        return hip_fail(c);
      }
    }
    for (; nb >= 8; nb -= 8)
      if (hipGraphLaunch(g8, c->stream) != hipSuccess) return hip_fail(c);
    for (; nb > 0; --nb)
      if (hipGraphLaunch(g1, c->stream) != hipSuccess) return hip_fail(c);
    return NLR_OK;
  }
  for (; nb > 0; --nb) {
    const nlr_status s = enqueue_iteration(c, false, lean);
    if (s != NLR_OK) return s;
  }
  return NLR_OK;
}

static nlr_status enqueue_finish(nlr_ctx* c) {
  const StepArgs a = make_step_args(c, c->pending ? 1 : 0);
  LAUNCH(KK_FINISH, launch_pass_a(c->g, c->b, a, true, c->stream));
  LAUNCH(KK_CTL_FINISH, launch_seg_a(c->g, c->b, true, c->stream));
  LAUNCH(KK_CTL_FINISH, launch_ctl_a(c->g, c->b, a, true, c->stream));
  c->pending = false;
  return NLR_OK;
}

static nlr_status read_ctl(nlr_ctx* c) {
  if (hipMemcpyAsync(c->host_ctl, c->b.ctl, sizeof(DevCtl), hipMemcpyDeviceToHost, c->stream) != hipSuccess)
    return hip_fail(c);
  if (hipStreamSynchronize(c->stream) != hipSuccess) return hip_fail(c);
  c->t_host = c->host_ctl->t_done;
  c->t_host_valid = true;
  return NLR_OK;
}

static nlr_status read_record(nlr_ctx* c, int64_t t, nlr_iter_stats* out) {
  if (hipMemcpyAsync(out, c->b.hist + (t % kHistCap), sizeof(nlr_iter_stats), hipMemcpyDeviceToHost,
                     c->stream) != hipSuccess)
    return hip_fail(c);
  if (hipStreamSynchronize(c->stream) != hipSuccess) return hip_fail(c);
  return NLR_OK;
}

extern "C" {

size_t nlr_workspace_bytes(int64_t n, int32_t d, int32_t r) {
  if (!shape_ok(n, d, r) || r > kMaxR) return 0;
  // the layout differs with the alignment of X and U (vector kernels or not) and
  // with the iteration structure (two passes or fused): cover all of them
  size_t m = 0;
  for (int al = 0; al < 2; ++al)
    for (int fu = 0; fu < 2; ++fu)
      for (int sp = 0; sp < 2; ++sp) {
        const size_t s =
            carve_workspace(make_geometry(n, d, r, 1, al != 0, sp != 0, fu != 0), nullptr, nullptr);
        if (s > m) m = s;
      }
  return m;
}

int32_t nlr_iteration_form(int64_t n, int32_t d, int32_t r, int32_t K, uint32_t flags) {
  if (!shape_ok(n, d, r) || K < 1 || K > r || r > kMaxR) return -1;
  const bool split = (flags & NLR_INIT_SPLIT_F16) != 0;
  const Geometry g = make_geometry(n, d, r, K, true, split, (flags & NLR_INIT_TWO_PASS) == 0);
  if (split && !g.split_b && !g.panel) return -1;
  if (g.fused8) return NLR_FORM_ONE_PASS;
  if (g.fused) return NLR_FORM_SINGLE_PASS;
  if (g.panel) return NLR_FORM_PANEL;
  return NLR_FORM_TWO_PASS;
}

}  // extern "C"

// Argument checks of nlr_init (before any HIP call); on success *g0 is the geometry
// and *need the workspace bytes it takes.
static nlr_status check_init(const float* X, int64_t n, int32_t d, int32_t K, int32_t r, const float* U,
                             const float* y, const nlr_params* params, uint32_t flags, Geometry* g0,
                             size_t* need) {
  if (!X || !U || !y || !params_ok(params)) return NLR_EINVAL;
  if (!shape_ok(n, d, r) || K < 1 || K > r) return NLR_EINVAL;
  if (flags & ~(uint32_t)(NLR_INIT_U_IN_OMEGA | NLR_INIT_KEEP_Y | NLR_INIT_X_NORMALISED | NLR_INIT_SPLIT_F16 |
                          NLR_INIT_TWO_PASS | NLR_INIT_DATA_START))
    return NLR_EINVAL;
  if ((flags & NLR_INIT_DATA_START) && (flags & NLR_INIT_U_IN_OMEGA)) return NLR_EINVAL;
  if (((uintptr_t)X & 3) || ((uintptr_t)U & 3) || ((uintptr_t)y & 3)) return NLR_EINVAL;
  if (r > kMaxR) return NLR_EUNSUPPORTED;
  const bool aligned16 = (((uintptr_t)X & 15) == 0) && (((uintptr_t)U & 15) == 0);
  const bool split = (flags & NLR_INIT_SPLIT_F16) != 0;
  const bool fused = (flags & NLR_INIT_TWO_PASS) == 0;
  *g0 = make_geometry(n, d, r, K, aligned16, split, fused);
  if (split && !g0->split_b && !g0->panel) return NLR_EUNSUPPORTED;
  *need = carve_workspace(*g0, nullptr, nullptr);
  return NLR_OK;
}

// Fills a constructed context (its host_ctl mirror already set) and enqueues the
// initialisation; synchronises once.  Leaves releasing the context to the caller.
static nlr_status init_ctx(nlr_ctx* c, const Geometry& g0, float* X, int32_t K, float* U, float* y,
                           const nlr_params* params, uint32_t flags, void* workspace, void* stream) {
  c->g = g0;
  carve_workspace(c->g, reinterpret_cast<char*>(workspace), &c->b);
  c->b.X = X;
  c->b.U = U;
  c->b.y = y;
  c->stream = reinterpret_cast<hipStream_t>(stream);
  c->prm = *params;
  c->pending = false;
  c->gram_valid = false;
  c->failed = false;
  c->breakdown = false;
  c->range_error = false;
  c->t_host = 0;
  c->t_host_valid = true;
  c->prof = false;
  c->prof_level = 0;
  c->ev_used = 0;
  for (int k = 0; k < KK_COUNT; ++k) {
    c->prof_ms[k] = 0.0;
    c->prof_n[k] = 0;
  }
  c->cap_stream = nullptr;
  c->graph1 = c->graph8 = c->lean1 = c->lean8 = nullptr;
  if (hipGetDevice(&c->device) != hipSuccess) return NLR_EHIP;
  const Geometry& g = c->g;
  const Bufs& b = c->b;
  const int64_t n = g.n;
  const bool split = (flags & NLR_INIT_SPLIT_F16) != 0;
  hipStream_t st = c->stream;
  if (launch_ctl_init(b, (float)(params->beta / (double)n), st) != hipSuccess) return NLR_EHIP;
  if (!(flags & NLR_INIT_X_NORMALISED)) {
    if (launch_colsum(g, b, st) != hipSuccess) return NLR_EHIP;
    if (launch_gram(g, b, st) != hipSuccess) return NLR_EHIP;
    if (launch_spectral(g, b, st) != hipSuccess) return NLR_EHIP;
    if (launch_normalise(g, b, st) != hipSuccess) return NLR_EHIP;
  }
  if (split)
    if (launch_xscale(g, b, st) != hipSuccess) return NLR_EHIP;
  if (flags & NLR_INIT_DATA_START) {
    // U holds Z: replace it by the range finder's orthonormal factor Q (Appendix D)
    const StepArgs a0 = make_step_args(c, 0);
    if (launch_data_start(g, b, a0, (flags & NLR_INIT_X_NORMALISED) != 0, st) != hipSuccess) return NLR_EHIP;
  }
  if (launch_project(g, b, (double)K, (flags & NLR_INIT_U_IN_OMEGA) ? 1 : 0, st) != hipSuccess) return NLR_EHIP;
  if (!(flags & NLR_INIT_KEEP_Y))
    if (launch_zero_y(g, b, st) != hipSuccess) return NLR_EHIP;
  if (g.fused) {
    // Theta_0 = Xhat^T U_0: one pass A (its row partials are recomputed by the first row pass)
    const StepArgs a0 = make_step_args(c, 0);
    if (launch_pass_a(g, b, a0, false, st) != hipSuccess) return NLR_EHIP;
    if (launch_reduce_theta(g, b, false, st) != hipSuccess) return NLR_EHIP;
    // split products: the fused pass B is then the only reader of X; store Xhat split once
    if (g.split_b)
      if (launch_split_x(g, b, st) != hipSuccess) return NLR_EHIP;
  }
  // panel form: both passes read Xhat only as split operands; store it so once
  if (g.panel)
    if (launch_split_x8(g, b, st) != hipSuccess) return NLR_EHIP;
  if (read_ctl(c) != NLR_OK) return NLR_EHIP;
  if (c->host_ctl->degenerate) return NLR_EDEGENERATE;
  if (c->host_ctl->breakdown) return NLR_EBREAKDOWN;
  return NLR_OK;
}

// Up to T iterations and the finish pass (the body of nlr_run).
static nlr_status run_iterations(nlr_ctx* c, int32_t T, int32_t* iters_done, nlr_iter_stats* last) {
  if (!c->t_host_valid)
    if (read_ctl(c) != NLR_OK) return NLR_EHIP;
  const int64_t t0 = c->t_host;
  if (launch_clear_stop(c->b, c->stream) != hipSuccess) return hip_fail(c);
  // no iteration of this call can stop while t < T_min: its row pass would not run
  // (one-pass form), so it is not launched
  const bool lean = t0 + T - 1 < (int64_t)c->prm.T_min;
  // the stop flag is polled every 32 iterations; kernels after a stop return at entry
  for (int32_t k = 0; k < T;) {
    if (k > 0 && (k % 32) == 0) {
      if (read_ctl(c) != NLR_OK) return NLR_EHIP;
      if (c->host_ctl->stop || c->host_ctl->breakdown) break;
    }
    if (k == 0) {
      nlr_status s = enqueue_iteration(c, true);
      if (s != NLR_OK) return s;
      ++k;
      continue;
    }
    const int32_t to_poll = 32 - (k % 32);
    const int32_t nb = (T - k) < to_poll ? (T - k) : to_poll;
    nlr_status s = enqueue_steady(c, nb, lean);
    if (s != NLR_OK) return s;
    k += nb;
  }
  nlr_status s = enqueue_finish(c);
  if (s != NLR_OK) return s;
  if (read_ctl(c) != NLR_OK) return NLR_EHIP;
  if (prof_collect(c) != hipSuccess) return hip_fail(c);
  const int64_t t1 = c->host_ctl->t_done;
  if (iters_done) *iters_done = (int32_t)(t1 - t0);
  // (one-pass iteration: a stop fires after the row pass, before the pass; the Gram
  // terms of the latest pass stay those of the current factor, with the dual step of
  // its end counted by the stored gate, so they still give the next call's s)
  if (c->host_ctl->breakdown) {
    c->failed = true;
    c->breakdown = true;
    c->range_error = c->host_ctl->breakdown == kRangeError;
  }
  if (last) {
    if (t1 > t0 || c->host_ctl->breakdown) {
      const int64_t t = c->host_ctl->breakdown ? t1 : t1 - 1;
      if (read_record(c, t, last) != NLR_OK) return NLR_EHIP;
    } else {
      std::memset(last, 0, sizeof(*last));
      last->t = -1;
    }
  }
  return c->breakdown ? (c->range_error ? NLR_ERANGE : NLR_EBREAKDOWN) : NLR_OK;
}

// ---- the allocation-free entry point ----
// Device scratch that nlr_solve_static uses in place of a caller's workspace: one
// copy per GPU the library runs on, held until the process ends, shared by every
// such call on that GPU (calls that overlap on one GPU race on it).  In host code
// the array's name is not a device address: the address of the current device's
// copy comes from hipGetSymbolAddress, taken once per device by the first call
// there and kept in g_scratch_ptr.
static __device__ __align__(256) unsigned char scratch[NLR_STATIC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};

static nlr_status static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return NLR_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return NLR_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return NLR_OK;
}

extern "C" {

nlr_status nlr_init(nlr_ctx** ctx, float* X, int64_t n, int32_t d, int32_t K, int32_t r, float* U, float* y,
                    const nlr_params* params, uint32_t flags, void* workspace, size_t workspace_bytes,
                    void* stream) {
  if (!ctx) return NLR_EINVAL;
  *ctx = nullptr;
  Geometry g0;
  size_t need = 0;
  const nlr_status chk = check_init(X, n, d, K, r, U, y, params, flags, &g0, &need);
  if (chk != NLR_OK) return chk;
  if (!workspace || ((uintptr_t)workspace & 255) || workspace_bytes < need) return NLR_EWORKSPACE;
  nlr_ctx* c = new (std::nothrow) nlr_ctx();
  if (!c) return NLR_EHIP;
  c->graphs_allowed = true;
  if (hipHostMalloc(reinterpret_cast<void**>(&c->host_ctl), sizeof(DevCtl), hipHostMallocDefault) != hipSuccess) {
    delete c;
    return NLR_EHIP;
  }
  const nlr_status s = init_ctx(c, g0, X, K, U, y, params, flags, workspace, stream);
  if (s != NLR_OK) {
    nlr_destroy(c);
    return s;
  }
  *ctx = c;
  return NLR_OK;
}

nlr_status nlr_solve_static(float* X, int64_t n, int32_t d, int32_t K, int32_t r, float* U, float* y,
                            const nlr_params* params, uint32_t flags, int32_t T, int32_t* iters_done,
                            nlr_iter_stats* last, void* stream) {
  if (T < 0) return NLR_EINVAL;
  Geometry g0;
  size_t need = 0;
  const nlr_status chk = check_init(X, n, d, K, r, U, y, params, flags, &g0, &need);
  if (chk != NLR_OK) return chk;
  if (need > NLR_STATIC_SCRATCH_BYTES) return NLR_EWORKSPACE;
  void* ws = nullptr;
  if (static_scratch(&ws) != NLR_OK) return NLR_EHIP;
  // the context lives on this stack frame; the control-block mirror is ordinary host
  // memory (no pinned allocation); profiling stays off, so no events are created
  nlr_ctx c;
  c.graphs_allowed = false;  // graph instantiation allocates
  DevCtl mirror;
  std::memset(&mirror, 0, sizeof(mirror));
  c.host_ctl = &mirror;
  nlr_status s = init_ctx(&c, g0, X, K, U, y, params, flags, ws, stream);
  if (s != NLR_OK) return s;
  return run_iterations(&c, T, iters_done, last);
}

nlr_status nlr_set_params(nlr_ctx* c, const nlr_params* params) {
  if (!c || !params_ok(params)) return NLR_EINVAL;
  if (c->failed) return NLR_ESTATE;
  c->prm = *params;
  drop_graphs(c);  // their kernels carry the old step arguments
  return NLR_OK;
}

nlr_status nlr_step(nlr_ctx* c, nlr_iter_stats* stats) {
  if (!c) return NLR_EINVAL;
  if (c->failed) return NLR_ESTATE;
  if (launch_clear_stop(c->b, c->stream) != hipSuccess) return hip_fail(c);
  nlr_status s = enqueue_iteration(c, true);
  if (s != NLR_OK) return s;
  s = enqueue_finish(c);
  if (s != NLR_OK) return s;
  c->t_host_valid = false;
  if (stats) {
    if (read_ctl(c) != NLR_OK) return NLR_EHIP;
    if (c->host_ctl->breakdown) {
      c->failed = true;
      c->breakdown = true;
      c->range_error = c->host_ctl->breakdown == kRangeError;
    }
    const int64_t t = c->host_ctl->t_done - (c->host_ctl->breakdown ? 0 : 1);
    if (read_record(c, t < 0 ? 0 : t, stats) != NLR_OK) return NLR_EHIP;
    if (prof_collect(c) != hipSuccess) return hip_fail(c);
    if (c->breakdown) return c->range_error ? NLR_ERANGE : NLR_EBREAKDOWN;
  }
  return NLR_OK;
}

nlr_status nlr_run(nlr_ctx* c, int32_t T, int32_t* iters_done, nlr_iter_stats* last) {
  if (!c || T < 0) return NLR_EINVAL;
  if (c->failed) return NLR_ESTATE;
  return run_iterations(c, T, iters_done, last);
}

nlr_status nlr_labels(nlr_ctx* c, int32_t* labels) {
  if (!c || !labels || ((uintptr_t)labels & 3)) return NLR_EINVAL;
  if (c->failed) return NLR_ESTATE;
  if (launch_labels(c->g, c->b, labels, c->stream) != hipSuccess) return hip_fail(c);
  return NLR_OK;
}

nlr_status nlr_labels_spectral(nlr_ctx* c, int32_t K, const int64_t* seed_rows, int32_t max_iter,
                               int32_t* labels, int32_t* passes_done) {
  if (!c || !labels || !seed_rows || ((uintptr_t)labels & 3) || max_iter < 1) return NLR_EINVAL;
  if (K < 1 || K > c->g.r) return NLR_EINVAL;
  if (K > kLabMaxK) return NLR_EUNSUPPORTED;
  for (int32_t k = 0; k < K; ++k)
    if (seed_rows[k] < 0 || seed_rows[k] >= c->g.n) return NLR_EINVAL;
  if (c->failed) return NLR_ESTATE;
  const Geometry& g = c->g;
  LabScratch L = carve_lab_scratch(g.n, g.r, K, reinterpret_cast<char*>(c->b.theta_part));
  int32_t flags[2] = {0, 0};
  if (hipMemcpyAsync(L.seeds, seed_rows, (size_t)K * sizeof(int64_t), hipMemcpyHostToDevice, c->stream) !=
      hipSuccess)
    return hip_fail(c);
  if (launch_lab_embed(g, c->b, L, K, c->stream) != hipSuccess) return hip_fail(c);
  if (hipMemcpyAsync(flags, L.flag, sizeof(flags), hipMemcpyDeviceToHost, c->stream) != hipSuccess)
    return hip_fail(c);
  if (hipStreamSynchronize(c->stream) != hipSuccess) return hip_fail(c);
  if (flags[0]) return NLR_EDEGENERATE;
  int32_t pass = 0;
  while (pass < max_iter) {
    ++pass;
    if (launch_lab_pass(g, c->b, L, K, labels, pass == 1 ? 1 : 0, c->stream) != hipSuccess) return hip_fail(c);
    if (hipMemcpyAsync(flags, L.flag, sizeof(flags), hipMemcpyDeviceToHost, c->stream) != hipSuccess)
      return hip_fail(c);
    if (hipStreamSynchronize(c->stream) != hipSuccess) return hip_fail(c);
    if (pass > 1 && flags[1] == 0) break;
  }
  if (passes_done) *passes_done = pass;
  return NLR_OK;
}

nlr_status nlr_history(nlr_ctx* c, nlr_iter_stats* out, int32_t max_records, int32_t* count) {
  if (!c || !out || max_records < 0 || !count) return NLR_EINVAL;
  if (read_ctl(c) != NLR_OK) return NLR_EHIP;
  const int64_t t1 = c->host_ctl->t_done + (c->host_ctl->breakdown ? 1 : 0);
  int64_t avail = t1 < kHistCap ? t1 : kHistCap;
  if (avail > max_records) avail = max_records;
  const int64_t first = t1 - avail;
  std::vector<nlr_iter_stats> all(kHistCap);
  if (hipMemcpyAsync(all.data(), c->b.hist, sizeof(nlr_iter_stats) * kHistCap, hipMemcpyDeviceToHost,
                     c->stream) != hipSuccess)
    return hip_fail(c);
  if (hipStreamSynchronize(c->stream) != hipSuccess) return hip_fail(c);
  for (int64_t k = 0; k < avail; ++k) out[k] = all[(first + k) % kHistCap];
  *count = (int32_t)avail;
  return NLR_OK;
}

nlr_status nlr_normaliser(nlr_ctx* c, double* a, double* xbar_host) {
  if (!c || !a) return NLR_EINVAL;
  if (read_ctl(c) != NLR_OK) return NLR_EHIP;
  *a = c->host_ctl->spectral_a;
  if (xbar_host) {
    if (hipMemcpyAsync(xbar_host, c->b.i_xbar, sizeof(double) * c->g.d, hipMemcpyDeviceToHost, c->stream) !=
        hipSuccess)
      return hip_fail(c);
    if (hipStreamSynchronize(c->stream) != hipSuccess) return hip_fail(c);
  }
  return NLR_OK;
}

nlr_status nlr_inspect(nlr_ctx* c, int32_t what, void* host_dst, size_t bytes) {
  if (!c || !host_dst) return NLR_EINVAL;
  const Geometry& g = c->g;
  if (what == 0) {
    if (bytes < (size_t)g.d * g.r * 4) return NLR_EINVAL;
    std::vector<float> lay((size_t)g.d32 * g.r32);
    if (hipMemcpyAsync(lay.data(), c->b.theta, lay.size() * 4, hipMemcpyDeviceToHost, c->stream) != hipSuccess)
      return hip_fail(c);
    if (hipStreamSynchronize(c->stream) != hipSuccess) return hip_fail(c);
    float* out = reinterpret_cast<float*>(host_dst);
    for (int f = 0; f < g.d; ++f)
      for (int col = 0; col < g.r; ++col) {
        const int ch = f >> 5, fin = f & 31, hh = fin >> 4, j = (fin & 15) >> 2, ee = fin & 3;
        const int mbk = col >> 5, l = hh * 32 + (col & 31);
        const size_t idx = ((((size_t)ch * 4 + j) * g.NB + mbk) * 64 + l) * 4 + ee;
        out[(size_t)f * g.r + col] = lay[idx];
      }
    return NLR_OK;
  }
  if (what == 3) {
    if (bytes < sizeof(int64_t)) return NLR_EINVAL;
    if (read_ctl(c) != NLR_OK) return NLR_EHIP;
    const int64_t v = c->host_ctl->rows_run;
    std::memcpy(host_dst, &v, sizeof v);
    return NLR_OK;
  }
  if (what == 1 || what == 2) {
    if (bytes < (size_t)g.r * 4) return NLR_EINVAL;
    if (hipMemcpyAsync(host_dst, what == 1 ? c->b.p : c->b.s, (size_t)g.r * 4, hipMemcpyDeviceToHost,
                       c->stream) != hipSuccess)
      return hip_fail(c);
    if (hipStreamSynchronize(c->stream) != hipSuccess) return hip_fail(c);
    return NLR_OK;
  }
  return NLR_EINVAL;
}

nlr_status nlr_set_profiling(nlr_ctx* c, int32_t enable) {
  if (!c || enable < 0 || enable > 2) return NLR_EINVAL;
  if (c->prof && !enable) {
    if (prof_collect(c) != hipSuccess) return hip_fail(c);
  }
  c->prof = enable != 0;
  c->prof_level = enable;
  // events for a few hundred launches exist before timing starts
  if (c->prof && grow_events(c, 1024) != hipSuccess) return hip_fail(c);
  for (int k = 0; k < KK_COUNT; ++k) {
    c->prof_ms[k] = 0.0;
    c->prof_n[k] = 0;
  }
  c->ev_pairs.clear();
  c->ev_used = 0;
  return NLR_OK;
}

nlr_status nlr_kernel_times(nlr_ctx* c, const char** names, double* total_ms, int64_t* launches,
                            int32_t* n_kernels) {
  if (!c || !names || !total_ms || !launches || !n_kernels) return NLR_EINVAL;
  if (prof_collect(c) != hipSuccess) return hip_fail(c);
  for (int k = 0; k < KK_COUNT; ++k) {
    names[k] = kKernelNames[k];
    total_ms[k] = c->prof_ms[k];
    launches[k] = c->prof_n[k];
  }
  *n_kernels = KK_COUNT;
  return NLR_OK;
}

void nlr_destroy(nlr_ctx* c) {
  if (!c) return;
  drop_graphs(c);
  if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
  for (auto e : c->ev_pool) (void)hipEventDestroy(e);
  if (c->host_ctl) (void)hipHostFree(c->host_ctl);
  delete c;
}

const char* nlr_status_string(nlr_status s) {
  // a C caller may pass any int; reading it through the enum type would be
  // undefined in C++ for values outside the enumerators' range
  int v;
  std::memcpy(&v, &s, sizeof v);
  switch (v) {
    case NLR_OK: return "ok";
    case NLR_EINVAL: return "invalid argument";
    case NLR_EWORKSPACE: return "workspace missing, misaligned or too small";
    case NLR_EBREAKDOWN: return "normalisation breakdown (||W_+||_F <= 1e-20)";
    case NLR_EDEGENERATE: return "degenerate input (zero centred data, or a rank-deficient sample or spectrum)";
    case NLR_EHIP: return "HIP runtime error";
    case NLR_ESTATE: return "context failed earlier or used out of order";
    case NLR_EUNSUPPORTED: return "shape outside the compiled kernel family";
    case NLR_ERANGE: return "split-fp16 products: W left the range of its fp16 operand (use fp32 products or a smaller step)";
  }
  return "unknown status";
}

const char* nlr_version(void) { return "nlr-gfx950 0.1"; }

}  // extern "C"
