/*
 * A plain C99 caller of libpace.so, built against include/pace.h alone: the host-only
 * helpers and the argument checks that return before any launch (no GPU needed).
 * Prints "c abi ok" and exits 0 when every check holds.
 */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "pace.h"

static int failures = 0;

#define CHECK(cond)                                                           \
  do {                                                                        \
    if (!(cond)) {                                                            \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond);     \
      ++failures;                                                             \
    }                                                                         \
  } while (0)

int main(void) {
  /* keep counts: ceil(ratio * n - 1e-9), clamped to [0, n] (Section 3.3's top-K) */
  CHECK(pace_keep_count(0.10, 10549) == 1055);
  CHECK(pace_keep_count(0.1, 30) == 3);
  CHECK(pace_keep_count(0.0, 100) == 0);
  CHECK(pace_keep_count(1.0, 100) == 100);
  CHECK(pace_keep_count(2.0, 100) == 100);
  CHECK(pace_keep_count(0.5, -1) == -1);
  CHECK(pace_keep_count(NAN, 10) == -1);

  /* resize target: no budget in force keeps sqrt(rho) per side, snapped to 28 */
  int oh = 0, ow = 0;
  CHECK(pace_apc_target_size(0.25, 2156, 3836, 1.0, 1e12, 28, &oh, &ow) == PACE_OK);
  CHECK(oh == 1092 && ow == 1932);   /* 1078 -> 38.5 -> 39 * 28; 1918 -> 68.5 -> 69 * 28 */
  CHECK(pace_apc_target_size(0.25, 0, 3836, 1.0, 1e12, 28, &oh, &ow) == PACE_ERR_INVALID_ARG);
  CHECK(strlen(pace_last_error()) > 0);
  CHECK(pace_apc_target_size(0.25, 100, 100, 1.0, 1e12, 28, NULL, &ow) == PACE_ERR_INVALID_ARG);

  /* workspace sizes grow with the problem */
  CHECK(pace_apc_density_workspace_size(2156, 3836, 14) > pace_apc_density_workspace_size(448, 448, 14));
  CHECK(pace_ddae_select_workspace_size(10549, 1) >= 3u * 10549u * 4u);
  CHECK(pace_prefill_attention_workspace_size(10677, 28) >= 28u * 10677u * 4u);

  /* refusals before any launch */
  static char fake[256] __attribute__((aligned(16)));   /* a host address, never dereferenced here */
  CHECK(pace_apc_downsample(NULL, 10, 10, (uint8_t*)fake, 5, 5, NULL) == PACE_ERR_INVALID_ARG);
  CHECK(pace_apc_downsample((const uint8_t*)fake, 10, 10, (uint8_t*)fake, 11, 10, NULL) == PACE_ERR_INVALID_ARG);
  CHECK(pace_apc_density((const uint8_t*)fake, 100, 98, 14, 0.1f, 0.6f, 1.5f, NULL, (float*)fake,
                         fake, (size_t)1 << 30, NULL) == PACE_ERR_INVALID_ARG);
  CHECK(pace_apc_density((const uint8_t*)fake, 448, 448, 14, 0.1f, 0.6f, 1.5f, NULL, (float*)fake,
                         fake, 16, NULL) == PACE_ERR_WORKSPACE);
  {
    /* head dim outside {80, 128}: valid arguments otherwise, refused as unsupported */
    const int32_t* cu = (const int32_t*)fake;
    const pace_status_t st = pace_vit_attention((const uint16_t*)fake, (const uint16_t*)fake,
                                                (const uint16_t*)fake, 64, 2, 64, cu, 1, 64, 0.125f,
                                                (uint16_t*)fake, NULL, NULL, NULL, 0, NULL);
    CHECK(st == PACE_ERR_UNSUPPORTED);
    CHECK(strstr(pace_last_error(), "head dim") != NULL);
  }
  CHECK(pace_topk_gather((const float*)fake, 10, 11, NULL, 0, (int32_t*)fake, NULL, NULL, 0, NULL) ==
        PACE_ERR_INVALID_ARG);

  if (failures == 0) printf("c abi ok\n");
  return failures == 0 ? 0 : 1;
}
