/* Plain C client of the LinSimp C ABI: includes the three headers, links
 * liblinsimp.so and calls the entry points that need no GPU (sizes, version,
 * argument errors).  Exit status 0 when every check holds. */
#include <stdio.h>
#include <string.h>

#include "linsimp.h"
#include "linsimp_bank.h"
#include "linsimp_head.h"

static int fails = 0;
#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) { fprintf(stderr, "check failed: %s\n", #c); ++fails; } \
  } while (0)

int main(void) {
  linsimp_dims d;
  memset(&d, 0, sizeof d);
  d.B = 2; d.H = 16; d.n = 16384; d.D = 128; d.Dv = 128; d.m = 128; d.w = 64;
  d.dtype = LINSIMP_BF16; d.eps = 1e-30f;
  const size_t fw = linsimp_workspace_size(&d, 0), bw = linsimp_workspace_size(&d, 1);
  CHECK(fw > 0 && bw > fw);
  CHECK(linsimp_head_saved_size(&d) > 0);
  CHECK(linsimp_head_workspace_size(&d, 1) >= bw);
  CHECK(linsimp_version() > 0);

  linsimp_dims bad = d;
  bad.w = 65;                                   /* beyond the supported window */
  CHECK(linsimp_workspace_size(&bad, 0) == 0);
  CHECK(strlen(linsimp_last_error()) > 0);

  /* a NULL input is reported, never dereferenced */
  CHECK(linsimp_fwd(&d, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL) ==
        LINSIMP_E_INVALID_ARG);
  CHECK(linsimp_feature_bank(16, 128, 48, NULL, NULL, NULL, 1, NULL) != LINSIMP_OK);

  printf("linsimp C ABI: version %d, workspace %zu / %zu bytes, %d failure(s)\n", linsimp_version(),
         fw, bw, fails);
  return fails == 0 ? 0 : 1;
}
