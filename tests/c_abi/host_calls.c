/* A C99 client of libwino: the header compiles as plain C, and the host-side
 * calls (no device work) behave as include/wino.h states.  Prints one line
 * per check and exits non-zero on the first failure. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

#include "wino.h"

#define CHECK(cond, what)                                   \
  do {                                                      \
    if (!(cond)) {                                          \
      fprintf(stderr, "FAIL: %s (line %d)\n", what, __LINE__); \
      return 1;                                             \
    }                                                       \
    printf("ok: %s\n", what);                               \
  } while (0)

int main(void) {
  const int64_t dims[4] = {8, 16, 56, 56};
  wino_opts o = {{1, 1, 1}, NULL, 0, WINO_RELU, 0.0f, {0, 0, 0}};
  wino_plan_t* p = NULL;
  CHECK(wino_plan(3, 2, 3, 64, 128, dims, &o, &p) == WINO_OK && p != NULL, "plan F(2^3,3^3)");

  wino_plan_desc d;
  CHECK(wino_plan_describe(p, &d) == WINO_OK, "describe");
  CHECK(d.alpha == 4 && d.n_xi == 64 && d.T == 8 * 8 * 28 * 28, "alpha, elements, tiles");
  CHECK(d.Y[0] == 16 && d.Y[1] == 56 && d.Y[2] == 56, "output extents");
  CHECK(wino_filter_bytes(p) == (size_t)4 * 64 * d.C_pad * d.K_pad, "filter bytes");
  CHECK(wino_workspace_bytes(p) >= (size_t)4 * 64 * d.C_pad * d.T_pad, "workspace holds V");
  CHECK(wino_weight_gradient_workspace_bytes(p) > wino_workspace_bytes(p), "weight-gradient workspace");
  CHECK(wino_forward_workspace_bytes(p) == wino_workspace_bytes(p), "two-stage forward workspace");

  /* per-axis tiles: 2 on the first axis, 4 on the others (eq. 4) */
  wino_opts ot = {{1, 1, 1}, NULL, 0, 0u, 0.0f, {2, 4, 4}};
  wino_plan_t* pa = NULL;
  const int64_t dims_a[4] = {2, 7, 13, 11};
  CHECK(wino_plan(3, 4, 3, 20, 24, dims_a, &ot, &pa) == WINO_OK && pa != NULL, "plan with per-axis tiles");
  wino_plan_desc dd;
  CHECK(wino_plan_describe(pa, &dd) == WINO_OK && dd.n_xi == 4 * 6 * 6 && dd.tile[0] == 2 && dd.alpha_axis[1] == 6,
        "per-axis tiles described");
  wino_destroy(pa);

  int64_t out[5];
  CHECK(wino_output_dims(p, out) == WINO_OK && out[0] == 8 && out[1] == 128 && out[4] == 56, "output dims");

  double AT[2 * 4], BT[4 * 4], G[4 * 3];
  CHECK(wino_get_matrices(p, AT, BT, G) == WINO_OK, "matrices");
  /* F(2,3) on {0, 1, -1, inf}: A^T = [[1,1,1,0],[0,1,-1,-1]], G rows 1 and 2 carry 1/2 */
  CHECK(AT[0] == 1 && AT[3] == 0 && AT[5] == 1 && AT[6] == -1 && fabs(G[3]) == 0.5, "F(2,3) entries");

  wino_plan_t* a = NULL;
  CHECK(wino_plan_adjoint(p, &a) == WINO_OK && a != NULL, "adjoint plan");
  wino_plan_desc da;
  CHECK(wino_plan_describe(a, &da) == WINO_OK && da.C == 128 && da.K == 64 && da.X[2] == 56 && da.Y[2] == 56,
        "adjoint: C and K swapped, extents kept at pad 1");

  double pts[5], growth = 0.0, g_def = 0.0;
  CHECK(wino_search_points(3, 4, 3, pts, &growth) == WINO_OK && growth > 0.0, "point search");
  CHECK(wino_points_error_growth(3, 4, 3, NULL, 0, &g_def) == WINO_OK && growth <= g_def, "searched <= default");

  wino_plan_t* bad = NULL;
  CHECK(wino_plan(3, 3, 3, 4, 4, dims, NULL, &bad) == WINO_EUNSUPPORTED && bad == NULL, "unsupported size");
  CHECK(wino_plan(3, 2, 3, 0, 4, dims, NULL, &bad) == WINO_EINVAL && bad == NULL, "zero channels");
  CHECK(wino_forward(p, NULL, NULL, NULL, NULL, 0, NULL) == WINO_EINVAL, "forward rejects NULL");
  CHECK(wino_status_string(WINO_EWORKSPACE) != NULL, "status string");

  wino_destroy(a);
  wino_destroy(p);
  printf("all host calls ok\n");
  return 0;
}
