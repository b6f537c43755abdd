/*
 * nlr.h — C ABI of the MI355X (gfx950) NLR K-means iteration library (libnlr.so).
 *
 * The library runs the spectrally normalised nonnegative low-rank (NLR)
 * projected-gradient iteration for the K-means SDP relaxation (GEM-KMeans):
 *
 *   minimise  fhat_y(U) = <Ahat, U U^T> + y^T h(U) + beta/2 ||h(U)||^2
 *   over      Omega = { U in R^{n x r} : U >= 0, ||U||_F^2 = K },
 *   with      Ahat = -Xhat Xhat^T,  h(U) = (U U^T 1 - 1) / sqrt(n)
 *
 * (paper Section 2, eq. Kmeans_NLR; Section 3, eq. normalized).  One
 * iteration is Algorithm 1 (Section 4.3): Theta = Xhat^T U; the gradient step
 * and positive part of eq. (gpu-positive-update) fused with the statistics of
 * eq. (fused-statistics); the normalising multiplier, movement estimate
 * (eq. movement-estimate), gated dual ascent and stopping rule.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All matrices are row-major and contiguous.  X is n x d, U is n x r.
 * - Pointers named X, U, y, labels, workspace are DEVICE pointers owned by
 *   the caller; the library never allocates, frees or retains device memory
 *   beyond the lifetime the caller gives it.  Pointers must be 4-byte aligned
 *   (16-byte alignment enables vector loads), the workspace 256-byte aligned.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   Every kernel is enqueued on it; host-visible results are synchronised on
 *   it only where a function says so.
 * - Functions return nlr_status.  Argument errors are detected before any
 *   HIP call and leave device memory untouched.  A HIP failure or a
 *   normalisation breakdown makes the context sticky-failed: later calls on
 *   it return NLR_ESTATE (nlr_destroy still works).
 * - A context is not thread-safe; two contexts may share a device and stream.
 * - The dual buffer y holds the STORED dual ytilde = y_math / sqrt(n), and the
 *   penalty is applied as beta / n (Section 3, Appendix C "Storage and
 *   parameter conventions").
 */
#ifndef NLR_H
#define NLR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct nlr_ctx nlr_ctx; /* opaque host-side handle: scalars + borrowed pointers */

typedef enum {
  NLR_OK = 0,
  NLR_EINVAL = 1,       /* invalid argument (nothing enqueued) */
  NLR_EWORKSPACE = 2,   /* workspace NULL, misaligned or smaller than nlr_workspace_bytes */
  NLR_EBREAKDOWN = 3,   /* normalisation breakdown: ||W_+||_F <= 1e-20 (Algorithm 1) */
  NLR_EDEGENERATE = 4,  /* centred data is zero, so a = ||X_c||_2 = 0 (Section 3 needs a > 0) */
  NLR_EHIP = 5,         /* a HIP runtime call failed */
  NLR_ESTATE = 6,       /* context failed earlier, or was used out of order */
  NLR_EUNSUPPORTED = 7, /* shape outside the compiled kernel family (see nlr_init) */
  NLR_ERANGE = 8        /* split-fp16 products: W left the range of its fp16 operand (see
                           NLR_INIT_SPLIT_F16); sticky like NLR_EBREAKDOWN, U then holds W */
} nlr_status;

/* Algorithm parameters (Algorithm 1 "Require" line).  The paper fixes no
 * values; alpha must be > 0 and finite, beta > 0, eps_d >= 0, eps_c >= 0,
 * T_min >= 0. */
typedef struct {
  double alpha;   /* primal step size */
  double beta;    /* augmentation (penalty) parameter; the kernels use beta/n */
  double eps_d;   /* dual-ascent tolerance: dual step iff Delta < eps_d^2 K */
  double eps_c;   /* convergence tolerance on movement and feasibility */
  int32_t T_min;  /* stop only once at least T_min iterations are done */
  int32_t reserved;
} nlr_params;

/* Per-iteration record.  For iteration t (0-based; it maps U_t to U_{t+1}):
 *   objective, theta_fro2 : fhat_{y_t}(U_t) and ||Xhat^T U_t||_F^2 (eq. normalized)
 *   a, b, h               : ||W||_F^2, ||U_t||_F^2, <W, U_t>_F, FP64 (eq. fused-statistics)
 *   c                     : FP32(sqrt(K)/sqrt(a)) computed from an FP64 ratio (Appendix B, Alg. 2)
 *   delta                 : sqrt(max(c^2 a + b - 2 c h, 0) / K) with the rounded c (eq. movement-estimate)
 *   dual_step             : Delta < eps_d^2 K, the dual step taken at the end of iteration t
 *   rho                   : ||q_{t+1}||_2 / sqrt(n), q = U p - 1 of U_{t+1}
 *   stop                  : the stopping rule of Section 4.3 fired at iteration t
 *   breakdown             : 1 normalisation breakdown at iteration t (U then holds W);
 *                           2 W out of the split-fp16 range at iteration t (NLR_ERANGE) */
typedef struct {
  int64_t t;
  double objective;
  double theta_fro2;
  double a, b, h;
  double delta;
  double rho;
  float c;
  int32_t dual_step;
  int32_t stop;
  int32_t breakdown;
} nlr_iter_stats;

/* nlr_init flags */
enum {
  NLR_INIT_U_IN_OMEGA = 1, /* U already lies in Omega: skip the projection (resume) */
  NLR_INIT_KEEP_Y = 2,     /* keep the caller's y instead of zeroing it (resume) */
  NLR_INIT_X_NORMALISED = 4, /* X already holds Xhat: skip centring and spectral normalisation */
  /* Run the products of the iteration on the fp16 matrix cores (both products in
   * the single-Xhat-pass form; Xhat Theta only with NLR_INIT_TWO_PASS) with a
   * two-term split of every fp32 operand:
   * v = s (hi + lo), hi = fp16(v / s), lo = fp16(v / s - hi), with s a power of
   * two chosen from a bound on |v| so that hi and lo stay in fp16's normal
   * range, and v w ~ s_v s_w (hi_v hi_w + hi_v lo_w + lo_v hi_w) accumulated in
   * fp32.  The representation error is about 2^-22 relative per operand, below
   * the TF32 products of the paper's CUTLASS kernel (Appendix C), at about a fifth of the fp32 matrix
   * work.  X and U must be 16-byte aligned.  Supported shapes: d <= 128, r <= 64,
   * d % 4 == 0 (and r % 4 == 0 with NLR_INIT_TWO_PASS), run in the
   * single-Xhat-pass form; and, for every other shape with d % 8 == 0,
   * r % 4 == 0 and r <= 256, the two-pass panel form (LDS-tiled products, both
   * split; ybar is kept in the workspace between the passes).  Other shapes
   * return NLR_EUNSUPPORTED.  X is left holding Xhat in split form after
   * nlr_init, so it no longer reads as fp32 (do not pass it to nlr_init again
   * with NLR_INIT_X_NORMALISED): in the single-Xhat-pass and one-pass forms each 16 bytes that
   * held 4 consecutive features hold their 4 fp16 hi halves then their 4 fp16 lo
   * halves of x * s (s a power of two); in the panel form each 32 bytes that held
   * 8 features hold their 8 hi halves then their 8 lo halves.  U_0 must lie in
   * Omega (|u| <= sqrt(K)); nlr_init projects it unless NLR_INIT_U_IN_OMEGA.
   * Range precondition of the single-Xhat-pass and one-pass forms: the fresh
   * update W (before its normalisation) is split at the fixed scale 2^10, so
   * every entry must stay at or below 65504 / 2^10 (about 64).  A factor in
   * Omega has |u| <= sqrt(K) <= 8, and every gradient entry is at most
   * sqrt(K) (2 + 2 ||y|| + 2 beta (K + 1)) in size, so a step size within the
   * Prop. 1 bound at the current dual (alpha <= 1/L(y), eq. L) keeps
   * |w| <= 2 sqrt(K) <= 16; a step several times larger may not (the dual grows
   * with dual steps while alpha stays fixed).  An iteration whose W
   * leaves the range stops with NLR_ERANGE before any operand that left fp16's
   * range reaches Theta or s; fp32 products (without this flag) have no such
   * limit. */
  NLR_INIT_SPLIT_F16 = 8,
  /* Use the two-pass iteration (pass A: Theta = Xhat^T U with the row work; pass
   * B: Xhat Theta with the fused epilogue) even where the single-Xhat-pass form
   * is available.  By default, for d <= 128 and r <= 64 (d % 4 == 0, 16-byte
   * aligned X and U), each iteration reads Xhat once: pass B also forms
   * the partials of Xhat^T W_{t+1}, and Theta_{t+1} = c_{t+1} Xhat^T W_{t+1}
   * (U_{t+1} = c_{t+1} W_{t+1}, Algorithm 1), while a row pass over U and ytilde
   * does the rest of pass A's work.  With NLR_INIT_SPLIT_F16 and 97..128
   * features with 33..64 columns (d % 4 == 0, r % 4 == 0), or at most 64
   * features with at most 16 columns (d % 4 == 0, r even) the default is the
   * one-pass form: the same kernel also does the row work (q, the gated dual
   * step, ybar), s = U^T ybar is formed from W^T W, W^T ytilde and the column sums
   * of the previous pass's W, and W is written over U in place.  At iterations
   * where the previous iteration's stopping rule can fire (its movement is below
   * min(eps_d, eps_c) and t >= T_min; the residual rho is then still needed) the
   * row work runs in a pass of its own first and settles the rule.  All forms
   * compute the same iteration; they differ by floating-point rounding only. */
  NLR_INIT_TWO_PASS = 16,
  /* Data-informed start (Appendix D, "Initialization"): U holds Z on input (e.g.
   * i.i.d. N(0,1) entries) and is replaced by U_0 = Pi_Omega(Q), where Q is the
   * orthonormal factor of V = Xhat Xhat^T Z computed by Cholesky QR in feature
   * space: M = Xhat^T Z, C = Xhat^T Xhat, M^T C M = R^T R, Q = Xhat (M R^{-1})
   * (FP64 for the d x r and r x r algebra).  Needs V of full column rank
   * (r <= rank Xhat); otherwise nlr_init returns NLR_EDEGENERATE.  Not combinable
   * with NLR_INIT_U_IN_OMEGA. */
  NLR_INIT_DATA_START = 32
};

/* Cluster labels by spectral embedding and K-means (Appendix D, "Recover
 * cluster labels from U"): the rows of the leading K left singular vectors of
 * the current U embed the n points (computed as U V_K Lambda_K^(-1/2) from the
 * FP64 eigendecomposition of U^T U); Lloyd's iteration starts from the embedded
 * rows seed_rows[0..K-1] (host array of row indices, e.g. drawn at random by the
 * caller), assigns every row to its nearest centroid (squared Euclidean distance
 * in FP64, lowest centroid index on ties), stops after the first pass that
 * changes no label or after max_iter passes, and moves each centroid to the
 * mean of its rows in between (a centroid without rows stays in place).
 * labels: device int32[n] (written every pass).  passes_done: host, nullable.
 * Needs 1 <= K <= r (K <= 128, else NLR_EUNSUPPORTED), seed rows in [0, n);
 * NLR_EDEGENERATE if the K-th eigenvalue of U^T U is not above 1e-14 of the
 * largest.  Call between iterations (it uses the context's workspace) on the
 * context's stream; synchronises once per pass. */
nlr_status nlr_labels_spectral(nlr_ctx* ctx, int32_t K, const int64_t* seed_rows, int32_t max_iter,
                               int32_t* labels, int32_t* passes_done);

/* Bytes of device workspace nlr_init needs for an (n, d, r) problem (the
 * storage model of Section 4.4, eq. gpu-storage: besides Xhat, the one n x r
 * factor and the stored dual, only per-workgroup partial sums -- fp32 Theta
 * partials, FP64 statistics -- and a few d x r / r-vectors; the panel form and
 * the two-pass form above 128 columns add ybar, n floats).  Depends only on (n, d, r).  Returns 0 when the shape is
 * invalid or unsupported. */
size_t nlr_workspace_bytes(int64_t n, int32_t d, int32_t r);

/* The iteration form nlr_init chooses for a shape and flags, assuming 16-byte
 * aligned X and U (as any allocator's base address is); host-only, no HIP call.
 * Every form computes Algorithm 1; they differ in how the passes over the rows
 * are fused (Section 4.2) and by floating-point rounding only.  Returns an
 * nlr_form value, or -1 for invalid arguments or an unsupported shape. */
enum {
  NLR_FORM_TWO_PASS = 0,     /* pass A (Theta = Xhat^T U, row work), pass B (Xhat Theta, epilogue) */
  NLR_FORM_PANEL = 1,        /* two passes with LDS-tiled split-fp16 products (large d x r) */
  NLR_FORM_SINGLE_PASS = 2,  /* row pass over U, then pass B that also forms Xhat^T W: Xhat read once */
  NLR_FORM_ONE_PASS = 3      /* one kernel per iteration: row work, primal step, next Theta and s terms */
};
int32_t nlr_iteration_form(int64_t n, int32_t d, int32_t r, int32_t K, uint32_t flags);

/* Prepares a problem and enqueues the initialisation on `stream`:
 *   1. centring and spectral normalisation of X in place (Section 3):
 *      xbar (FP64 column means), C = X_c^T X_c (FP64), a = sqrt(lambda_max(C))
 *      by power iteration, X <- (X - 1 xbar^T) / a   [skipped with X_NORMALISED]
 *   2. U <- Pi_Omega(U) = sqrt(K) U_+ / ||U_+||_F (eq. projected-primal-step)
 *      [skipped with U_IN_OMEGA]; p = U^T 1
 *   3. y <- 0 [skipped with KEEP_Y]
 * X: device n*d floats (in: data, out: Xhat).  U: device n*r floats (in: U_0,
 * e.g. the paper's random start Z with N(0,1) entries; out: Pi_Omega(U_0)).
 * y: device n floats (stored dual).  Requires 1 <= K <= r <= 448, r <= n,
 * 1 <= d <= 4096, n < 2^40 (r > 448 returns NLR_EUNSUPPORTED; above 256 columns
 * only the fp32 two-pass form runs).  Synchronises `stream` once at the end to report
 * NLR_EDEGENERATE / NLR_EBREAKDOWN (U_0 with no positive entry).  On success
 * *ctx receives a new context. */
nlr_status nlr_init(nlr_ctx** ctx, float* X, int64_t n, int32_t d, int32_t K, int32_t r,
                    float* U, float* y, const nlr_params* params, uint32_t flags,
                    void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): nlr_init followed by
 * nlr_run(T) in one call that allocates nothing -- no workspace argument, no
 * context left behind, no pinned host memory.  Arguments, in-place outputs (X
 * becomes Xhat, U the iterate after the run, y the stored dual) and statuses are
 * those of nlr_init and nlr_run; *iters_done and *last (both nullable) as in
 * nlr_run.  Its scratch is a device array inside the library of
 * NLR_STATIC_SCRATCH_BYTES (64 MiB), one per GPU the library runs on, held until
 * the process ends: a shape whose nlr_workspace_bytes exceeds it returns
 * NLR_EWORKSPACE before any HIP call (every benchmark shape up to 1e7 x 128 x 64
 * fits; 2e6 x 768 x 256 does not).  Every call on a GPU uses that GPU's one
 * array, and everything a call reads from it is written by the same call first;
 * calls that overlap on one GPU (other threads, other streams) race on it and
 * must be serialised by the caller.  Synchronises `stream` as nlr_init and
 * nlr_run do. */
#define NLR_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
nlr_status nlr_solve_static(float* X, int64_t n, int32_t d, int32_t K, int32_t r, float* U, float* y,
                            const nlr_params* params, uint32_t flags, int32_t T, int32_t* iters_done,
                            nlr_iter_stats* last, void* stream);

/* Replaces the algorithm parameters of a context (takes effect at the next step). */
nlr_status nlr_set_params(nlr_ctx* ctx, const nlr_params* params);

/* One iteration of Algorithm 1, enqueued asynchronously.  On return U holds
 * U_{t+1} and y the stored dual after the (gated) dual step.  When `stats` is
 * non-NULL the stream is synchronised and the iteration's record written.
 * Returns NLR_EBREAKDOWN if the iteration broke down (only known when stats
 * is non-NULL; otherwise reported by the next synchronising call). */
nlr_status nlr_step(nlr_ctx* ctx, nlr_iter_stats* stats);

/* Up to T iterations of Algorithm 1, stopping early by the rule of Section
 * 4.3 (movement < min(eps_d, eps_c), rho < eps_c, t+1 >= T_min).  The device
 * decides; the host polls a flag every 32 iterations and synchronises once
 * at the end.  *iters_done (nullable) receives the iterations done by this
 * call; *last (nullable) the record of the last one.  nlr_run(T) and T calls
 * of nlr_step give bitwise-identical U and y.  While profiling is off, the
 * iterations after the call's first are replayed from HIP graphs the context
 * captures on first use (on a private stream; held until nlr_destroy, dropped
 * by nlr_set_params); when every iteration of the call has t < T_min, the
 * one-pass form leaves out the row pass that only the stopping rule needs. */
nlr_status nlr_run(nlr_ctx* ctx, int32_t T, int32_t* iters_done, nlr_iter_stats* last);

/* Row-argmax labels of the current U: labels[i] = argmax_j U_ij, lowest j on
 * ties (int32, device pointer, n entries).  Appendix D ("Recover cluster labels
 * from U"): under exact recovery with r = K the solution is U = H, one positive
 * entry 1/sqrt(n_k) per row in the column of the row's cluster, so the argmax
 * of a row is its cluster; for r > K use nlr_labels_spectral.  Argmax of W
 * equals argmax of U = c W (c > 0).  Returns NLR_EINVAL for a NULL or
 * misaligned labels pointer, NLR_ESTATE on a failed context.  Asynchronous. */
nlr_status nlr_labels(nlr_ctx* ctx, int32_t* labels);

/* Copies the records of the most recent iterations (oldest first, at most the
 * last 4096) into host memory `out` (capacity `max_records`); *count receives
 * the number written.  Synchronises the stream. */
nlr_status nlr_history(nlr_ctx* ctx, nlr_iter_stats* out, int32_t max_records, int32_t* count);

/* Synchronises and returns the spectral normaliser a = ||X_c||_2 and, when
 * xbar_host is non-NULL, the d column means (FP64) found by nlr_init. */
nlr_status nlr_normaliser(nlr_ctx* ctx, double* a, double* xbar_host);

/* Diagnostic read-back (synchronises): what = 0 copies Theta = Xhat^T U of the
 * latest iteration as d*r row-major floats; 1 copies p = U^T 1 (r floats) of
 * the current U; 2 copies s = U^T ybar (r floats) of the latest iteration's
 * starting factor -- in the one-pass form (split products at the shapes listed
 * under NLR_INIT_TWO_PASS) of the current U instead, formed after each pass for the next
 * one with the step arguments of that call; 3 copies an int64: the number of
 * one-pass iterations since nlr_init whose row work ran in a pass of its own
 * before the primal step (the first iteration after nlr_init, and those at which
 * the previous iteration's stopping rule could fire).  Other values, or `bytes`
 * too small, return NLR_EINVAL. */
nlr_status nlr_inspect(nlr_ctx* ctx, int32_t what, void* host_dst, size_t bytes);

/* Per-kernel timing with HIP events recorded on the context's stream around
 * the launches made by nlr_step / nlr_run (off by default): enable = 1 around
 * every launch, 2 around the row and pass kernels only (pass_a, pass_b, pass_u,
 * pass_bf, finish: fewer events in the stream); 0 turns it off and clears the
 * totals; other values return NLR_EINVAL. */
nlr_status nlr_set_profiling(nlr_ctx* ctx, int32_t enable);

/* Kernel timing totals since profiling was enabled (synchronises).  For kernel
 * k < *n_kernels: names[k] (static string), total_ms[k], launches[k].
 * Arrays must hold NLR_MAX_KERNEL_KINDS entries. */
#define NLR_MAX_KERNEL_KINDS 16
nlr_status nlr_kernel_times(nlr_ctx* ctx, const char** names, double* total_ms,
                            int64_t* launches, int32_t* n_kernels);

/* Releases the host-side handle (device memory stays the caller's). */
void nlr_destroy(nlr_ctx* ctx);

const char* nlr_status_string(nlr_status s);

/* Library build identification (static string). */
const char* nlr_version(void);

#ifdef __cplusplus
}
#endif
#endif /* NLR_H */
