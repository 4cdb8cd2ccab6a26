/* A plain C consumer of the library's C ABI (no Python, no torch): host-only
 * calls that need no GPU.  Prints one line per check; exits non-zero on the
 * first failure.  Built and run by tests/test_abi_c.py. */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "allegro_layer.h"
#include "allegro_tp.h"

#define CHECK(cond, ...)                  \
  do {                                    \
    if (!(cond)) {                        \
      printf("FAIL: " __VA_ARGS__);       \
      printf(" (%s)\n", allegro_last_error()); \
      return 1;                           \
    }                                     \
  } while (0)

int main(void) {
  /* (lmax, full parity) -> (d1, d2, paths, nnz), as the oracle counts them */
  const int expect[6][6] = {{1, 0, 4, 4, 4, 10},     {1, 1, 8, 4, 10, 32},   {2, 0, 9, 9, 11, 83},
                            {2, 1, 18, 9, 30, 274}, {3, 0, 16, 16, 23, 353}, {3, 1, 32, 16, 68, 1222}};
  for (int c = 0; c < 6; ++c) {
    const int lmax = expect[c][0], full = expect[c][1];
    allegro_tp_plan *plan = NULL;
    int rc = allegro_tp_plan_create(&plan, lmax, 64, full ? ALLEGRO_FULL_PARITY : 0);
    CHECK(rc == ALLEGRO_OK && plan, "plan_create lmax=%d full=%d", lmax, full);
    int d1 = 0, d2 = 0, np = 0, nnz = 0;
    CHECK(allegro_tp_plan_query(plan, &d1, &d2, &np, NULL, &nnz) == ALLEGRO_OK, "query");
    CHECK(d1 == expect[c][2] && d2 == expect[c][3] && np == expect[c][4] && nnz == expect[c][5],
          "sizes lmax=%d full=%d: %d %d %d %d", lmax, full, d1, d2, np, nnz);
    int *desc = (int *)malloc(sizeof(int) * 6 * (size_t)np);
    int *idx = (int *)malloc(sizeof(int) * 4 * (size_t)nnz);
    double *val = (double *)malloc(sizeof(double) * (size_t)nnz);
    CHECK(desc && idx && val, "malloc");
    CHECK(allegro_tp_plan_query(plan, NULL, NULL, NULL, desc, NULL) == ALLEGRO_OK, "path_desc");
    /* every path obeys the triangle and parity selection rules */
    for (int p = 0; p < np; ++p) {
      const int l1 = desc[6 * p], p1 = desc[6 * p + 1], l2 = desc[6 * p + 2], p2 = desc[6 * p + 3];
      const int l3 = desc[6 * p + 4], p3 = desc[6 * p + 5];
      CHECK(abs(l1 - l2) <= l3 && l3 <= l1 + l2 && p3 == p1 * p2, "selection rule, path %d", p);
    }
    CHECK(allegro_tp_plan_cg(plan, idx, val) == ALLEGRO_OK, "cg");
    /* per path and output component m3, the coefficients are orthonormal: sum C^2 = 1 */
    double *norm = (double *)calloc((size_t)np * (size_t)d1, sizeof(double));
    CHECK(norm != NULL, "calloc");
    for (int t = 0; t < nnz; ++t) norm[idx[4 * t] * d1 + idx[4 * t + 3]] += val[t] * val[t];
    for (int p = 0; p < np; ++p)
      for (int k = 0; k < d1; ++k)
        CHECK(norm[p * d1 + k] == 0.0 || (norm[p * d1 + k] > 1 - 1e-12 && norm[p * d1 + k] < 1 + 1e-12),
              "normalisation path %d component %d: %.17g", p, k, norm[p * d1 + k]);
    size_t bytes = 0;
    /* per-center rows and 128 range sums, or at lmax 3 at most one per-wave row
     * round per center (at most 1024 rounds) */
    const size_t rows = lmax >= 3 ? 1000 : 1000 + 128;
    CHECK(allegro_tp_backward_workspace(plan, 1000, &bytes) == ALLEGRO_OK &&
              bytes == rows * (size_t)np * 64 * sizeof(float),
          "workspace size %zu", bytes);
    CHECK(lmax < 3 || (allegro_tp_backward_workspace(plan, 5000, &bytes) == ALLEGRO_OK &&
                       bytes == (size_t)1024 * (size_t)np * 64 * sizeof(float)),
          "workspace size %zu at N=5000", bytes);
    /* rejected before any GPU call */
    CHECK(allegro_tp_forward(plan, -1, 0, NULL, NULL, NULL, NULL, NULL, NULL) == ALLEGRO_E_INVALID, "N<0");
    CHECK(strstr(allegro_last_error(), "negative") != NULL, "message");
    CHECK(allegro_tp_forward(plan, 0, 0, NULL, NULL, NULL, NULL, NULL, NULL) == ALLEGRO_OK, "empty no-op");
    CHECK(allegro_sh_forward(plan, 0, NULL, NULL, NULL) == ALLEGRO_OK, "empty harmonics");
    free(norm);
    free(desc);
    free(idx);
    free(val);
    CHECK(allegro_tp_plan_destroy(plan) == ALLEGRO_OK, "destroy");
    printf("ok lmax=%d full=%d d1=%d d2=%d paths=%d nnz=%d\n", lmax, full, d1, d2, np, nnz);
  }
  /* the layer's buffer sizes are host arithmetic; its shape checks run before any GPU call */
  {
    allegro_tp_plan *plan = NULL;
    CHECK(allegro_tp_plan_create(&plan, 3, 64, ALLEGRO_FULL_PARITY) == ALLEGRO_OK, "layer plan");
    size_t saved = 0, work = 0;
    CHECK(allegro_layer_buffers(plan, 64, 128, 100, 5000, &saved, &work) == ALLEGRO_OK, "layer buffers");
    /* saved holds at least w [E][U], env [N][U][d2], T [E][U][d1], s [E][U] and a [E][H] */
    const size_t floats = (size_t)5000 * 64 + (size_t)100 * 64 * 16 + (size_t)5000 * 64 * 32 + (size_t)5000 * 64 +
                          (size_t)5000 * 128;
    CHECK(saved >= floats * sizeof(float) && saved < floats * sizeof(float) + 5 * 256, "saved bytes %zu", saved);
    CHECK(work > (size_t)5000 * 64 * 32 * sizeof(float), "workspace bytes %zu", work);
    CHECK(allegro_layer_buffers(plan, 48, 128, 100, 5000, &saved, &work) == ALLEGRO_E_UNSUPPORTED, "L=48");
    CHECK(allegro_layer_forward(plan, 64, 128, 0, 5, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL,
                                NULL, NULL, 0, NULL) == ALLEGRO_E_INVALID,
          "layer E>0 with N=0");
    CHECK(allegro_layer_forward(plan, 64, 128, 0, 0, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL,
                                NULL, NULL, 0, NULL) == ALLEGRO_OK,
          "layer empty no-op");
    CHECK(allegro_tp_plan_destroy(plan) == ALLEGRO_OK, "destroy");
    allegro_tp_plan *narrow = NULL;
    CHECK(allegro_tp_plan_create(&narrow, 2, 32, ALLEGRO_FULL_PARITY) == ALLEGRO_OK, "U=32 plan");
    CHECK(allegro_layer_buffers(narrow, 64, 64, 10, 10, &saved, &work) == ALLEGRO_E_UNSUPPORTED, "layer U=32");
    CHECK(allegro_tp_plan_destroy(narrow) == ALLEGRO_OK, "destroy");
    printf("ok layer\n");
  }
  allegro_tp_plan *bad = (allegro_tp_plan *)1;
  CHECK(allegro_tp_plan_create(&bad, 4, 64, 0) == ALLEGRO_E_UNSUPPORTED && bad == NULL, "lmax 4 rejected");
  printf("ok errors\n");
  return 0;
}
