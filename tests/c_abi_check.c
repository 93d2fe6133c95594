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

int main(int argc, char **argv) {
  const char *table_path = argc > 1 ? argv[1] : NULL;
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
  size_t arena2 = 0, stride2 = 0;
  CHECK(cheb_cache_arena_bytes(4, CHEB_BF16, seg, 3, &arena2, &stride2) == CHEB_OK);
  CHECK(arena2 == arena && stride2 == stride);
  CHECK(cheb_cache_arena_bytes(4, CHEB_BF16, seg, 3, &arena2, NULL) == CHEB_OK && arena2 == arena);
  CHECK(cheb_cache_arena_bytes(0, CHEB_BF16, seg, 3, &arena2, &stride2) == CHEB_E_INVAL);
  CHECK(cheb_cache_arena_bytes(4, 7, seg, 3, &arena2, &stride2) == CHEB_E_DTYPE);
  CHECK(cheb_cache_arena_bytes(4, CHEB_BF16, seg, 3, NULL, &stride2) == CHEB_E_INVAL);

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

  /* Offline table: build, query, save, load, compare bit for bit. */
  double tsteps[50];
  for (int s = 0; s < 50; ++s) tsteps[s] = 1.0 - s / 50.0;
  cheb_table *t = NULL, *u = NULL;
  CHECK(cheb_table_build(&t, 50, 1, 1, 6, 6, tsteps, CHEB_SHORT_LOWER) == CHEB_OK);
  int32_t T = 0, nh = 0, pol = 0, nfull = 0;
  CHECK(cheb_table_info(t, &T, &nh, &pol, &nfull) == CHEB_OK && T == 50 && nfull == 10);
  if (table_path) {
    CHECK(cheb_table_save(t, table_path) == CHEB_OK);
    CHECK(cheb_table_load(&u, table_path) == CHEB_OK);
    for (int s = 0; s < 50; ++s) {
      int32_t p1, p2, n1, n2, s1[CHEB_MAX_SLOTS], s2[CHEB_MAX_SLOTS];
      double w1[CHEB_MAX_SLOTS], w2[CHEB_MAX_SLOTS];
      CHECK(cheb_table_step(t, s, &p1, &n1, s1, w1) == CHEB_OK);
      CHECK(cheb_table_step(u, s, &p2, &n2, s2, w2) == CHEB_OK);
      CHECK(p1 == p2 && n1 == n2);
      CHECK(memcmp(s1, s2, sizeof(int32_t) * (size_t)n1) == 0);
      CHECK(memcmp(w1, w2, sizeof(double) * (size_t)n1) == 0);
    }
    CHECK(cheb_table_destroy(u) == CHEB_OK);
  }
  CHECK(cheb_table_load(&u, "/nonexistent/dir/table") == CHEB_E_IO);
  uint8_t mask[50] = {0};
  mask[0] = mask[7] = mask[19] = mask[33] = 1;
  CHECK(cheb_table_build_mask(&u, 50, mask, 3, tsteps, CHEB_SHORT_FULL) == CHEB_OK);
  CHECK(cheb_table_destroy(u) == CHEB_OK);
  CHECK(cheb_table_destroy(t) == CHEB_OK);

  /* Refused before any launch: residual and stateless-combination checks. */
  {
    const void *src[2] = {fake, (char *)fake + (1 << 20)};
    double w2[2] = {0.5, 0.5};
    CHECK(cheb_combine(src, 2, w2, (char *)fake + 8, 100, CHEB_BF16, NULL) == CHEB_E_ALIGN);
    CHECK(cheb_combine(src, 9, w2, (char *)fake + (2 << 20), 100, CHEB_BF16, NULL) == CHEB_E_INVAL);
    int64_t segn[2] = {64, 64}, roff[2] = {0, 4};
    float *xo = (float *)((char *)fake + (4 << 20));
    CHECK(cheb_residual_reduce(src, segn, roff, 2, CHEB_BF16, NULL, xo, 64, NULL) == CHEB_E_ALIGN);
    roff[1] = 8;
    CHECK(cheb_residual_reduce(src, segn, roff, 2, CHEB_BF16, NULL, xo, 64, NULL) == CHEB_E_INVAL);
    CHECK(cheb_residual_reduce(src, segn, roff, 2, 5, NULL, xo, 64, NULL) == CHEB_E_DTYPE);
  }
  double nodes_out[8];
  CHECK(cheb_chebyshev_nodes(8, 1, 0.0, 49.0, nodes_out) == CHEB_OK && nodes_out[0] > nodes_out[7]);
  double wv[4];
  CHECK(cheb_precompute_weights_variant(hist, 4, target, 1, CHEB_RHO_ALTERNATING, wv) == CHEB_OK);

  cheb_launch_config cfg;
  CHECK(cheb_get_launch_config(&cfg) == CHEB_OK && cfg.block == 64 && cfg.waves_per_cu == 0);
  printf("c abi ok\n");
  return 0;
}
