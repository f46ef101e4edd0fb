/* A plain C99 consumer of the libzo C ABI (include/zo.h), compiled with gcc: checks that the
 * header is valid C and exercises the host-only paths (coefficients, validation, strings),
 * which need no GPU. Prints one line per check; exit status 0 when all pass. */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "zo.h"

static int failures = 0;

static void check(int ok, const char* what) {
  printf("%s %s\n", ok ? "ok" : "FAIL", what);
  if (!ok) ++failures;
}

int main(void) {
  /* coefficients of one probe by hand (fp64, same operation order as the header states):
   * d2 = (Lp - 2 L0) + Lm, chat = d2 / eps^2, w = 1 / max(lambda, |chat|^alpha),
   * c = ((Lp - Lm) w) / (2 K eps) */
  const double lp[2] = {2.5, 1.0}, lm[2] = {1.5, 1.0};
  const double l0 = 1.0, eps = 0.5;
  float c[2] = {0.0f, 0.0f};
  double c64[2], curv[2], w[2];
  check(zo_probe_coeffs_ex(lp, lm, 2, l0, eps, 1.0, 1.0, c, c64, curv, w) == ZO_OK, "zo_probe_coeffs_ex status");
  /* probe 0: d2 = 2.0, chat = 8.0, w = 1/8, c = (1.0 / 8) / (4 * 0.5) = 0.0625 */
  check(curv[0] == 8.0 && w[0] == 0.125 && c64[0] == 0.0625 && c[0] == 0.0625f, "probe 0 by hand");
  /* probe 1: equal losses: chat = 0, w = 1 (lambda), c = 0 */
  check(curv[1] == 0.0 && w[1] == 1.0 && c64[1] == 0.0 && c[1] == 0.0f, "probe 1 by hand");
  /* alpha = 0.1 default: w = 1 / max(1, 8^0.1) */
  check(zo_probe_coeffs(lp, lm, 2, l0, eps, c) == ZO_OK && c[0] == (float)((1.0 / pow(8.0, 0.1)) / 2.0),
        "zo_probe_coeffs default alpha");

  /* validation returns before any HIP call */
  check(zo_probe_coeffs(lp, lm, 2, l0, 0.0, c) == ZO_ERR_ARG, "eps = 0 refused");
  check(zo_probe_coeffs(NULL, lm, 2, l0, eps, c) == ZO_ERR_NULL, "null losses refused");
  check(zo_perturb(NULL, ZO_BF16, 0, 10, 1, 1, 0, 1e-3f, NULL) == ZO_ERR_NULL, "perturb null params");
  check(zo_perturb((void*)0x1001, ZO_BF16, 0, 10, 1, 1, 0, 1e-3f, NULL) == ZO_ERR_ARG, "perturb misaligned");
  check(zo_perturb((void*)0x1000, (zo_dtype)7, 0, 10, 1, 1, 0, 1e-3f, NULL) == ZO_ERR_ARG, "perturb bad dtype");
  check(zo_perturb((void*)0x1000, ZO_F32, 0, 10, 1, 1, 0, INFINITY, NULL) == ZO_ERR_NONFINITE, "perturb inf eps");
  check(zo_perturb(NULL, ZO_F32, 0, 0, 1, 1, 0, 1e-3f, NULL) == ZO_OK, "perturb n = 0 no-op");
  check(zo_update((void*)0x1000, ZO_F32, 10, 1, 1, ZO_K_MAX + 1, c, 1e-3f, NULL) == ZO_ERR_ARG, "update K > K_MAX");
  check(zo_update((void*)0x1000, ZO_F32, 10, 1, 1, 2, NULL, 1e-3f, NULL) == ZO_ERR_NULL, "update null c");
  {
    const zo_segment segs[2] = {{(void*)0x10000, 0, 100}, {(void*)0x10020, 100, 100}};
    check(zo_perturb_segments(segs, 2, ZO_F32, 1, 1, 0, 1e-3f, 0, 0.0f, NULL) == ZO_ERR_ARG,
          "overlapping segments refused");
  }
  check(strlen(zo_strerror(ZO_ERR_NONFINITE)) > 0 && strlen(zo_version()) > 0, "strings");
  return failures ? 1 : 0;
}
