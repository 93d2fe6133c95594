/* Compiles include/cheb.h as C99 and links libcheb.so from plain C.  Runs
 * host-only calls (weights, layout, ring bookkeeping, error codes); it never
 * launches GPU work, so it runs without a GPU. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "cheb.h"

#define CHECK(cond)                                                        \
  do {                                                                     \
    if (!(cond)) {                                                         \
      fprintf(stderr, "check failed at line %d: %s (%s)\n", __LINE__,      \
              #cond, cheb_last_error());                                   \
      return 1;                                                            \
    }                                                                      \
  } while (0)

int main(void) {
  CHECK(cheb_version() == CHEB_VERSION);
  /* Newton one-step-ahead weights for four equispaced nodes: -1 4 -6 4. */
  const double hist[4] = {999.0, 979.0, 959.0, 939.0};
  const double target[1] = {919.0};
  double w[4];
  CHECK(cheb_precompute_weights(hist, 4, target, 1, w) == CHEB_OK);
  const double expect[4] = {-1.0, 4.0, -6.0, 4.0};
  for (int k = 0; k < 4; ++k) CHECK(fabs(w[k] - expect[k]) < 1e-12);
  const double dup[3] = {1.0, 2.0, 1.0};
  CHECK(cheb_precompute_weights(dup, 3, target, 1, w) == CHEB_E_DUPNODE);
  CHECK(strlen(cheb_last_error()) > 0);

  const int64_t seg[3] = {13, 8, 4096};
  int64_t off[3], slot_numel = 0;
  size_t stride = 0, arena = 0;
  CHECK(cheb_cache_layout(4, CHEB_BF16, seg, 3, off, &slot_numel, &stride, &arena) == CHEB_OK);
  CHECK(off[0] == 0 && off[1] == 16 && off[2] == 24 && slot_numel == 24 + 4096);
  CHECK(stride % 256 == 0 && arena == 4 * stride);

  /* A handle over an address that is never dereferenced: metadata only. */
  void *fake = (void *)(uintptr_t)((uint64_t)1 << 40);
  cheb_cache *c = NULL;
  CHECK(cheb_cache_create(&c, 4, CHEB_BF16, seg, 3, fake, arena) == CHEB_OK);
  void *slot = NULL;
  for (int i = 0; i < 6; ++i) {
    CHECK(cheb_cache_begin_push(c, &slot) == CHEB_OK);
    CHECK(cheb_cache_commit(c, 100.0 - i) == CHEB_OK);
  }
  double held[CHEB_MAX_SLOTS];
  int32_t count = 0;
  CHECK(cheb_cache_history(c, held, &count) == CHEB_OK && count == 4);
  CHECK(held[0] == 98.0 && held[3] == 95.0);
  CHECK(cheb_cache_begin_push(c, &slot) == CHEB_OK);
  CHECK(cheb_extrapolate(c, w, fake, NULL) == CHEB_E_NOTREADY);
  CHECK(cheb_cache_destroy(c) == CHEB_OK);

  uint8_t full[20];
  CHECK(cheb_schedule(20, 2, 1, 4, full) == CHEB_OK);
  const int want[20] = {1, 1, 1, 0, 0, 0, 1, 0, 0, 0, 1, 0, 0, 0, 1, 0, 0, 0, 1, 1};
  for (int s = 0; s < 20; ++s) CHECK(full[s] == want[s]);

  cheb_launch_config cfg;
  CHECK(cheb_get_launch_config(&cfg) == CHEB_OK && cfg.block == 1024);
  printf("c abi ok\n");
  return 0;
}
