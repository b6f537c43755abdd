/* Host-side checks of the C ABI under AddressSanitizer and UndefinedBehaviorSanitizer
 * (built with the library's host code instrumented; no GPU is touched): every path
 * that returns before a HIP call, with extreme and invalid sizes.  Exit status 0 when
 * every check holds; a sanitizer finding aborts. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "nlr.h"

static int fails = 0;
#define CHECK(cond)                                                      \
  do {                                                                   \
    if (!(cond)) {                                                       \
      fprintf(stderr, "FAIL %s:%d: %s\n", __FILE__, __LINE__, #cond);    \
      ++fails;                                                           \
    }                                                                    \
  } while (0)

/* 256-byte aligned addresses that are never dereferenced: every call below
 * fails validation first */
#define FAKE ((void*)(uintptr_t)(1u << 20))

static nlr_status init(float* X, int64_t n, int32_t d, int32_t K, int32_t r, float* U, float* y,
                       const nlr_params* p, uint32_t flags, void* ws, size_t wsb, nlr_ctx** out) {
  nlr_ctx* c = (nlr_ctx*)(uintptr_t)123;
  const nlr_status s = nlr_init(&c, X, n, d, K, r, U, y, p, flags, ws, wsb, NULL);
  if (out) *out = c;
  return s;
}

int main(void) {
  CHECK(strncmp(nlr_version(), "nlr-gfx950", 10) == 0);
  for (int s = 0; s < 9; ++s) CHECK(strcmp(nlr_status_string((nlr_status)s), "unknown status") != 0);
  CHECK(strcmp(nlr_status_string((nlr_status)99), "unknown status") == 0);
  CHECK(strcmp(nlr_status_string((nlr_status)-1), "unknown status") == 0);

  /* workspace sizes over valid, extreme and invalid shapes */
  const int64_t ns[] = {1, 2, 3, 255, 256, 257, 1000, 10000000, (int64_t)1 << 31, ((int64_t)1 << 40) - 1,
                        (int64_t)1 << 40, INT64_MAX / 2, INT64_MAX, 0, -1, INT64_MIN};
  const int32_t ds[] = {1, 3, 4, 13, 16, 64, 65, 100, 128, 129, 256, 768, 4096, 4097, 0, -1, INT32_MAX, INT32_MIN};
  const int32_t rs[] = {1, 2, 4, 10, 16, 33, 64, 65, 128, 256, 257, 300, 448, 449, 0, -1, INT32_MAX, INT32_MIN};
  for (size_t a = 0; a < sizeof(ns) / sizeof(ns[0]); ++a)
    for (size_t b = 0; b < sizeof(ds) / sizeof(ds[0]); ++b)
      for (size_t c = 0; c < sizeof(rs) / sizeof(rs[0]); ++c) {
        const int64_t n = ns[a];
        const int32_t d = ds[b], r = rs[c];
        const size_t w = nlr_workspace_bytes(n, d, r);
        CHECK(w == nlr_workspace_bytes(n, d, r));
        const int valid = n >= 1 && n < ((int64_t)1 << 40) && d >= 1 && d <= 4096 && r >= 1 && r <= 448 && r <= n;
        if (!valid) CHECK(w == 0);
        else CHECK(w > 0 && w < ((size_t)1 << 60));
      }

  /* nlr_init: argument errors are reported before any HIP call */
  const nlr_params ok = {0.01, 1.0, 1e-4, 1e-4, 0, 0};
  const size_t wsb = nlr_workspace_bytes(1000, 16, 4);
  float* X = (float*)FAKE;
  float* U = (float*)FAKE;
  float* y = (float*)FAKE;
  CHECK(nlr_init(NULL, X, 1000, 16, 4, 4, U, y, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  nlr_ctx* c = NULL;
  CHECK(init(NULL, 1000, 16, 4, 4, U, y, &ok, 0, FAKE, wsb, &c) == NLR_EINVAL && c == NULL);
  CHECK(init(X, 1000, 16, 4, 4, NULL, y, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, 16, 4, 4, U, NULL, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, 16, 4, 4, U, y, NULL, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, 16, 0, 4, U, y, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, 16, 5, 4, U, y, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 3, 16, 2, 4, U, y, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, INT64_MAX, 16, 4, 4, U, y, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, INT64_MIN, 16, 4, 4, U, y, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, INT32_MAX, 4, 4, U, y, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, 16, INT32_MAX, INT32_MAX, U, y, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, 16, 4, 449, U, y, &ok, 0, FAKE, wsb, NULL) == NLR_EUNSUPPORTED);
  const nlr_params bad[] = {{0.0, 1.0, 1e-4, 1e-4, 0, 0}, {INFINITY, 1.0, 1e-4, 1e-4, 0, 0},
                            {NAN, 1.0, 1e-4, 1e-4, 0, 0},  {0.1, -1.0, 1e-4, 1e-4, 0, 0},
                            {0.1, 1.0, -1.0, 1e-4, 0, 0},  {0.1, 1.0, 1e-4, NAN, 0, 0},
                            {0.1, 1.0, 1e-4, 1e-4, -1, 0}, {0.1, 1.0, 1e-4, 1e-4, INT32_MIN, 0}};
  for (size_t i = 0; i < sizeof(bad) / sizeof(bad[0]); ++i)
    CHECK(init(X, 1000, 16, 4, 4, U, y, &bad[i], 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, 16, 4, 4, U, y, &ok, 1u << 7, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, 16, 4, 4, U, y, &ok, 0xffffffffu, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, 16, 4, 4, U, y, &ok, NLR_INIT_DATA_START | NLR_INIT_U_IN_OMEGA, FAKE, wsb, NULL) ==
        NLR_EINVAL);
  CHECK(init((float*)((char*)FAKE + 2), 1000, 16, 4, 4, U, y, &ok, 0, FAKE, wsb, NULL) == NLR_EINVAL);
  CHECK(init(X, 1000, 16, 4, 4, U, y, &ok, 0, NULL, wsb, NULL) == NLR_EWORKSPACE);
  CHECK(init(X, 1000, 16, 4, 4, U, y, &ok, 0, (char*)FAKE + 64, wsb, NULL) == NLR_EWORKSPACE);
  CHECK(init(X, 1000, 16, 4, 4, U, y, &ok, 0, FAKE, 1024, &c) == NLR_EWORKSPACE && c == NULL);
  CHECK(init(X, 1000, 16, 4, 4, U, y, &ok, 0, FAKE, 0, NULL) == NLR_EWORKSPACE);
  /* split-fp16 products: shapes and alignments outside the supported set */
  CHECK(init(X, 1000, 13, 4, 4, U, y, &ok, NLR_INIT_SPLIT_F16, FAKE, wsb, NULL) == NLR_EUNSUPPORTED);
  CHECK(init(X, 1000, 132, 4, 4, U, y, &ok, NLR_INIT_SPLIT_F16, FAKE, (size_t)1 << 40, NULL) == NLR_EUNSUPPORTED);
  CHECK(init((float*)((char*)FAKE + 4), 1000, 16, 4, 4, U, y, &ok, NLR_INIT_SPLIT_F16, FAKE, wsb, NULL) ==
        NLR_EUNSUPPORTED);

  /* calls without a context */
  nlr_iter_stats st;
  int32_t cnt = 0, done = 0;
  double a = 0.0;
  const char* names[NLR_MAX_KERNEL_KINDS];
  double ms[NLR_MAX_KERNEL_KINDS];
  int64_t launches[NLR_MAX_KERNEL_KINDS];
  CHECK(nlr_step(NULL, NULL) == NLR_EINVAL);
  CHECK(nlr_step(NULL, &st) == NLR_EINVAL);
  CHECK(nlr_run(NULL, 5, &done, &st) == NLR_EINVAL);
  CHECK(nlr_labels(NULL, (int32_t*)FAKE) == NLR_EINVAL);
  CHECK(nlr_labels_spectral(NULL, 2, NULL, 10, (int32_t*)FAKE, NULL) == NLR_EINVAL);
  CHECK(nlr_set_params(NULL, &ok) == NLR_EINVAL);
  CHECK(nlr_set_profiling(NULL, 1) == NLR_EINVAL);
  CHECK(nlr_history(NULL, &st, 1, &cnt) == NLR_EINVAL);
  CHECK(nlr_normaliser(NULL, &a, NULL) == NLR_EINVAL);
  CHECK(nlr_inspect(NULL, 0, &a, sizeof(a)) == NLR_EINVAL);
  CHECK(nlr_kernel_times(NULL, names, ms, launches, &cnt) == NLR_EINVAL);
  nlr_destroy(NULL);

  /* nlr_solve_static: the same argument checks, and shapes beyond its scratch, before any HIP call */
  done = -7;
  CHECK(nlr_solve_static(X, 1000, 16, 4, 4, U, y, &ok, 0, -1, &done, &st, NULL) == NLR_EINVAL && done == -7);
  CHECK(nlr_solve_static(NULL, 1000, 16, 4, 4, U, y, &ok, 0, 5, &done, &st, NULL) == NLR_EINVAL);
  CHECK(nlr_solve_static(X, 1000, 16, 4, 4, U, y, NULL, 0, 5, &done, &st, NULL) == NLR_EINVAL);
  CHECK(nlr_solve_static(X, 1000, 16, 5, 4, U, y, &ok, 0, 5, NULL, NULL, NULL) == NLR_EINVAL);
  CHECK(nlr_solve_static(X, INT64_MAX, 16, 4, 4, U, y, &ok, 0, 5, NULL, NULL, NULL) == NLR_EINVAL);
  CHECK(nlr_solve_static(X, 1000, 16, 4, 449, U, y, &ok, 0, 5, NULL, NULL, NULL) == NLR_EUNSUPPORTED);
  CHECK(nlr_solve_static(X, 1000, 16, 4, 4, U, y, &ok, 1u << 7, 5, NULL, NULL, NULL) == NLR_EINVAL);
  CHECK(nlr_workspace_bytes(2000000, 768, 256) > NLR_STATIC_SCRATCH_BYTES);
  CHECK(nlr_solve_static(X, 2000000, 768, 256, 256, U, y, &ok, 0, 5, NULL, NULL, NULL) == NLR_EWORKSPACE);
  CHECK(nlr_solve_static(X, ((int64_t)1 << 40) - 1, 4096, 256, 256, U, y, &ok, 0, 5, NULL, NULL, NULL) ==
        NLR_EWORKSPACE);

  if (fails) fprintf(stderr, "%d checks failed\n", fails);
  else printf("all checks passed\n");
  return fails ? 1 : 0;
}
