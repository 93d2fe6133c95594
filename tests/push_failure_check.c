/* A copy push whose launches fail part-way (Algorithm 1, full computation:
 * store (s, f_s) in H; Section 3.3, FIFO eviction), on the CPU: the
 * library's host sources are linked against tests/host_stubs.cpp, whose
 * segment-copy launcher succeeds for a set number of 64-segment batches and
 * then fails.  The FLUX.1-dev 1024 layout has 76 cached tensors, so every
 * push takes two launches.  The arena address is never dereferenced.
 *
 * Checks: a push into a full ring that fails on its second launch leaves
 * the history without the entry whose slot it was overwriting (so no
 * prediction can read that slot), records nothing, and the next push reuses
 * the slot; a push that fails into a ring with a free slot leaves the
 * history as it was. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "cheb.h"

void stub_gather_batches_ok(int n);

#define CHECK(cond)                                                        \
  do {                                                                     \
    if (!(cond)) {                                                         \
      fprintf(stderr, "check failed at line %d: %s (%s)\n", __LINE__,      \
              #cond, cheb_last_error());                                   \
      return 1;                                                            \
    }                                                                      \
  } while (0)

int main(void) {
  int64_t seg[76];
  for (int b = 0; b < 19; ++b) {
    seg[2 * b] = 4096LL * 3072;     /* double-stream block b, image tokens */
    seg[2 * b + 1] = 512LL * 3072;  /* double-stream block b, text tokens */
  }
  for (int b = 0; b < 38; ++b) seg[38 + b] = 4608LL * 3072; /* single-stream */
  size_t arena = 0, stride = 0;
  CHECK(cheb_cache_arena_bytes(6, CHEB_BF16, seg, 76, &arena, &stride) == CHEB_OK);
  CHECK(stride == 806879232ULL * 2 && arena == 6 * stride);

  void *base = (void *)(uintptr_t)((uint64_t)1 << 44);
  const void *src[76];
  for (int s = 0; s < 76; ++s) src[s] = (const void *)(uintptr_t)(((uint64_t)1 << 45) + 4096u * (uint64_t)s);
  cheb_cache *c = NULL;
  CHECK(cheb_cache_create(&c, 6, CHEB_BF16, seg, 76, base, arena) == CHEB_OK);

  /* Six pushes, two launches each, fill the ring. */
  stub_gather_batches_ok(12);
  for (int i = 0; i < 6; ++i) CHECK(cheb_cache_push(c, 10.0 * i, src, NULL) == CHEB_OK);
  double held[CHEB_MAX_SLOTS];
  int32_t count = 0;
  CHECK(cheb_cache_history(c, held, &count) == CHEB_OK && count == 6);
  void *oldest = NULL;
  CHECK(cheb_cache_entry(c, 0, &oldest) == CHEB_OK && oldest == base);

  /* The seventh push goes into the oldest entry's slot; its second launch
   * fails after the first has written 64 of the 76 segments. */
  stub_gather_batches_ok(1);
  CHECK(cheb_cache_push(c, 60.0, src, NULL) == CHEB_E_HIP);
  CHECK(strstr(cheb_last_error(), "launch 1") != NULL);
  CHECK(cheb_cache_history(c, held, &count) == CHEB_OK && count == 5);
  for (int a = 0; a < 5; ++a) CHECK(held[a] == 10.0 * (a + 1)); /* 0 dropped, 60 not held */
  for (int a = 0; a < 5; ++a) {
    void *p = NULL;
    CHECK(cheb_cache_entry(c, a, &p) == CHEB_OK && p != base);
  }
  double w[6] = {0, 0, 0, 0, 0, 1};
  void *out = (void *)(uintptr_t)((uint64_t)1 << 46);
  CHECK(cheb_extrapolate(c, w, out, NULL) == CHEB_E_NOTREADY);
  CHECK(cheb_extrapolate_at(c, 65.0, out, NULL, NULL) == CHEB_E_NOTREADY);

  /* The next push reuses that slot and fills the ring again. */
  stub_gather_batches_ok(2);
  CHECK(cheb_cache_push(c, 60.0, src, NULL) == CHEB_OK);
  CHECK(cheb_cache_history(c, held, &count) == CHEB_OK && count == 6);
  CHECK(held[0] == 10.0 && held[5] == 60.0);
  void *newest = NULL;
  CHECK(cheb_cache_entry(c, 5, &newest) == CHEB_OK && newest == base);

  /* A failed push into a ring with a free slot changes nothing. */
  CHECK(cheb_cache_reset(c) == CHEB_OK);
  stub_gather_batches_ok(4);
  CHECK(cheb_cache_push(c, 1.0, src, NULL) == CHEB_OK);
  CHECK(cheb_cache_push(c, 2.0, src, NULL) == CHEB_OK);
  stub_gather_batches_ok(0);
  CHECK(cheb_cache_push(c, 3.0, src, NULL) == CHEB_E_HIP);
  CHECK(cheb_cache_history(c, held, &count) == CHEB_OK && count == 2);
  CHECK(held[0] == 1.0 && held[1] == 2.0);
  stub_gather_batches_ok(2);
  CHECK(cheb_cache_push(c, 3.0, src, NULL) == CHEB_OK);
  CHECK(cheb_cache_history(c, held, &count) == CHEB_OK && count == 3 && held[2] == 3.0);

  CHECK(cheb_cache_destroy(c) == CHEB_OK);

  /* The same ring in the interleaved layout over an arena that is 256-byte
   * but not 64 KiB aligned: the lanes start at the next 64 KiB boundary,
   * 32 KiB apart, entry j of the ring in lane j mod 6; a failed push drops
   * the oldest entry as above. */
  CHECK(cheb_cache_arena_bytes_ex(6, CHEB_BF16, seg, 76, CHEB_LAYOUT_INTERLEAVED, &arena) ==
        CHEB_OK);
  const uint64_t chunks = (806879232ULL / 8 + 2047) / 2048;
  CHECK(arena == chunks * 6 * 32768 + 65536);
  char *ibase = (char *)(uintptr_t)(((uint64_t)1 << 44) + 256);
  char *region = (char *)(uintptr_t)(((uint64_t)1 << 44) + 65536);
  CHECK(cheb_cache_create_ex(&c, 6, CHEB_BF16, seg, 76, CHEB_LAYOUT_INTERLEAVED, ibase,
                             arena - 1) == CHEB_E_MISMATCH);
  CHECK(cheb_cache_create_ex(&c, 6, CHEB_BF16, seg, 76, CHEB_LAYOUT_INTERLEAVED, ibase, arena) ==
        CHEB_OK);
  int32_t lay = -1;
  int64_t chunk_elems = 0, lane_stride = 0;
  CHECK(cheb_cache_geometry(c, &lay, &chunk_elems, &lane_stride) == CHEB_OK);
  CHECK(lay == CHEB_LAYOUT_INTERLEAVED && chunk_elems == 16384 && lane_stride == 6 * 16384);
  void *slot_base = NULL;
  CHECK(cheb_cache_begin_push(c, &slot_base) == CHEB_E_INVAL);
  stub_gather_batches_ok(2 * 8);
  for (int i = 0; i < 8; ++i) CHECK(cheb_cache_push(c, 5.0 * i, src, NULL) == CHEB_OK);
  CHECK(cheb_cache_history(c, held, &count) == CHEB_OK && count == 6 && held[0] == 10.0);
  for (int a = 0; a < 6; ++a) {
    void *p = NULL;
    CHECK(cheb_cache_entry(c, a, &p) == CHEB_OK);
    CHECK(p == region + 32768 * ((a + 2) % 6));
  }
  stub_gather_batches_ok(1);
  CHECK(cheb_cache_push(c, 40.0, src, NULL) == CHEB_E_HIP);
  CHECK(cheb_cache_history(c, held, &count) == CHEB_OK && count == 5 && held[0] == 15.0);
  CHECK(cheb_extrapolate(c, w, out, NULL) == CHEB_E_NOTREADY);
  CHECK(cheb_cache_destroy(c) == CHEB_OK);
  printf("push failure ok\n");
  return 0;
}
