/* Plain C99 client of include/headcast.h: compiles with a C compiler, links
 * against libheadcast.so and exercises the host-only entry points (no GPU).
 * Exit status 0 when every check holds; the failing check is printed. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "headcast.h"

static int fails = 0;
#define CHECK(cond)                                             \
  do {                                                          \
    if (!(cond)) {                                              \
      fprintf(stderr, "check failed: %s (line %d)\n", #cond, __LINE__); \
      ++fails;                                                  \
    }                                                           \
  } while (0)

int main(void) {
  hc_config cfg;
  hc_ctx *ctx = NULL;
  int32_t w;
  int64_t b;

  memset(&cfg, 0xff, sizeof cfg);
  hc_config_default(&cfg);
  CHECK(cfg.n_layers == 30 && cfg.n_heads == 12 && cfg.head_dim == 128);
  CHECK(cfg.frames_per_block == 3 && cfg.window_blocks == 7);
  CHECK(cfg.spatial_radius == 4 && cfg.proxy_radius == 2);
  CHECK(cfg.theta_score > 0.75f && cfg.theta_score < 0.76f && cfg.gamma == 5.0f);
  CHECK(hc_validate_config(&cfg) == HC_OK);
  CHECK(hc_validate_config(NULL) == HC_E_INVAL);

  cfg.head_dim = 96;                       /* only 64 and 128 */
  CHECK(hc_validate_config(&cfg) == HC_E_INVAL);
  CHECK(hc_create(&cfg, 0, &ctx) == HC_E_INVAL && ctx == NULL);
  hc_config_default(&cfg);
  cfg.window_blocks = 1;
  CHECK(hc_validate_config(&cfg) == HC_E_INVAL);

  /* ring: block 0 -> slot 0; block b >= 1 -> 1 + (b - 1) mod (W - 1) */
  for (w = 2; w <= 9; ++w) {
    CHECK(hc_ring_slot(0, w) == 0);
    for (b = 1; b < 40; ++b) CHECK(hc_ring_slot(b, w) == 1 + (int32_t)((b - 1) % (w - 1)));
  }
  CHECK(hc_ring_slot(-1, 7) < 0);

  CHECK(strcmp(hc_status_string(HC_OK), "") != 0);
  CHECK(strcmp(hc_status_string(HC_E_ORDER), hc_status_string(HC_E_STATE)) != 0);
  CHECK(hc_last_error(NULL) != NULL);
  CHECK(hc_classify_outputs(NULL, HC_CLS_O_REF, NULL, NULL) == HC_E_INVAL);
  hc_destroy(NULL);

  if (fails) return 1;
  printf("abi_check: ok\n");
  return 0;
}
