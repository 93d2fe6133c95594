/*
 * A plain C99 program that uses libcheb on the GPU with no Python and no
 * torch: device memory from the HIP runtime's C API, six full steps pushed
 * into a five-entry ring (ragged segment sizes), single- and multi-target
 * predictions, each checked against the fp64 oracle on the host copies of
 * the pushed values.  Prints "c gpu ok" and exits 0 when every check holds.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "cheb.h"
#include "oracle.h"

#define N_SEGS 3
#define N_SLOTS 5
#define N_PUSH 6
#define N_TARGETS 3

static int failures = 0;

#define CHECK_CHEB(call)                                                       \
  do {                                                                         \
    int rc_ = (call);                                                          \
    if (rc_ != CHEB_OK) {                                                      \
      fprintf(stderr, "%s failed: %d %s\n", #call, rc_, cheb_last_error());    \
      return 1;                                                                \
    }                                                                          \
  } while (0)

#define CHECK_HIP(call)                                                        \
  do {                                                                         \
    hipError_t e_ = (call);                                                    \
    if (e_ != hipSuccess) {                                                    \
      fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));        \
      return 1;                                                                \
    }                                                                          \
  } while (0)

static uint32_t lcg(uint32_t *s) {
  *s = *s * 1664525u + 1013904223u;
  return *s;
}

/* A finite bf16 pattern: sign, exponent near 1.0, random mantissa. */
static uint16_t random_bf16(uint32_t *s) {
  uint32_t r = lcg(s);
  uint16_t sign = (uint16_t)((r >> 31) << 15);
  uint16_t expo = (uint16_t)((0x7e + ((r >> 8) & 1u)) << 7);
  return (uint16_t)(sign | expo | (r & 0x7fu));
}

/* Floored relative error of one segment's prediction against the oracle. */
static double segment_error(const uint16_t *got, const uint16_t *const *hist, const double *w,
                            int64_t count) {
  double *expect = malloc(sizeof(double) * (size_t)count);
  double *mag = malloc(sizeof(double) * (size_t)count);
  double worst = 0.0;
  oracle_extrapolate_bf16(hist, N_SLOTS, w, count, expect, mag);
  for (int64_t i = 0; i < count; ++i) {
    double g = oracle_bf16_to_f64(got[i]);
    double floor_ = fmax(fabs(expect[i]), 1e-3 * mag[i]);
    double e = floor_ > 0.0 ? fabs(g - expect[i]) / floor_ : fabs(g - expect[i]);
    if (e > worst) worst = e;
  }
  free(expect);
  free(mag);
  return worst;
}

int main(void) {
  const int64_t seg_numel[N_SEGS] = {100003, 4096, 17};
  const double t[N_PUSH] = {0.96, 0.9, 0.8, 0.72, 0.6, 0.5};
  const double targets[N_TARGETS] = {0.48, 0.46, 0.42};
  int64_t seg_offset[N_SEGS], slot_numel = 0;
  size_t stride = 0, arena_bytes = 0;
  CHECK_CHEB(cheb_cache_layout(N_SLOTS, CHEB_BF16, seg_numel, N_SEGS, seg_offset, &slot_numel,
                               &stride, &arena_bytes));
  size_t arena_bytes2 = 0;
  CHECK_CHEB(cheb_cache_arena_bytes(N_SLOTS, CHEB_BF16, seg_numel, N_SEGS, &arena_bytes2, NULL));
  if (arena_bytes2 != arena_bytes) {
    fprintf(stderr, "arena bytes disagree: %zu vs %zu\n", arena_bytes2, arena_bytes);
    return 1;
  }
  void *arena = NULL;
  CHECK_HIP(hipMalloc(&arena, arena_bytes));
  cheb_cache *cache = NULL;
  CHECK_CHEB(cheb_cache_create(&cache, N_SLOTS, CHEB_BF16, seg_numel, N_SEGS, arena,
                               arena_bytes));

  /* Host values of every pushed segment, and device copies to push from. */
  uint16_t *host[N_PUSH][N_SEGS];
  void *dev[N_PUSH][N_SEGS];
  uint32_t seed = 2025u;
  for (int p = 0; p < N_PUSH; ++p) {
    for (int s = 0; s < N_SEGS; ++s) {
      const size_t bytes = sizeof(uint16_t) * (size_t)seg_numel[s];
      host[p][s] = malloc(bytes);
      for (int64_t i = 0; i < seg_numel[s]; ++i) host[p][s][i] = random_bf16(&seed);
      CHECK_HIP(hipMalloc(&dev[p][s], bytes));
      CHECK_HIP(hipMemcpy(dev[p][s], host[p][s], bytes, hipMemcpyHostToDevice));
    }
    const void *src[N_SEGS] = {dev[p][0], dev[p][1], dev[p][2]};
    CHECK_CHEB(cheb_cache_push(cache, t[p], src, NULL));
  }
  double held[N_SLOTS];
  int32_t count = 0;
  CHECK_CHEB(cheb_cache_history(cache, held, &count));
  if (count != N_SLOTS) failures++;
  for (int k = 0; k < N_SLOTS; ++k)
    if (held[k] != t[k + 1]) failures++;

  /* One target, then every target from one pass. */
  const size_t out_bytes = sizeof(uint16_t) * (size_t)slot_numel;
  void *out[N_TARGETS];
  for (int m = 0; m < N_TARGETS; ++m) CHECK_HIP(hipMalloc(&out[m], out_bytes));
  double w_single[N_SLOTS];
  CHECK_CHEB(cheb_extrapolate_at(cache, targets[0], out[0], NULL, w_single));
  CHECK_HIP(hipDeviceSynchronize());
  uint16_t *got = malloc(out_bytes);
  double worst = 0.0;
  {
    double w[N_SLOTS];
    if (oracle_weights_row(held, N_SLOTS, targets[0], w) != 0) failures++;
    CHECK_HIP(hipMemcpy(got, out[0], out_bytes, hipMemcpyDeviceToHost));
    for (int s = 0; s < N_SEGS; ++s) {
      const uint16_t *hist[N_SLOTS];
      for (int k = 0; k < N_SLOTS; ++k) hist[k] = host[k + 1][s];
      double e = segment_error(got + seg_offset[s], hist, w, seg_numel[s]);
      if (e > worst) worst = e;
    }
  }
  double w_multi[N_TARGETS * N_SLOTS];
  CHECK_CHEB(cheb_extrapolate_at_multi(cache, targets, N_TARGETS, out, NULL, w_multi));
  CHECK_HIP(hipDeviceSynchronize());
  for (int m = 0; m < N_TARGETS; ++m) {
    double w[N_SLOTS];
    if (oracle_weights_row(held, N_SLOTS, targets[m], w) != 0) failures++;
    CHECK_HIP(hipMemcpy(got, out[m], out_bytes, hipMemcpyDeviceToHost));
    for (int s = 0; s < N_SEGS; ++s) {
      const uint16_t *hist[N_SLOTS];
      for (int k = 0; k < N_SLOTS; ++k) hist[k] = host[k + 1][s];
      double e = segment_error(got + seg_offset[s], hist, w, seg_numel[s]);
      if (e > worst) worst = e;
    }
  }
  printf("floored error %.3e over %d predictions\n", worst, 1 + N_TARGETS);
  if (!(worst <= 1e-2)) failures++;

  for (int m = 0; m < N_TARGETS; ++m) CHECK_HIP(hipFree(out[m]));
  for (int p = 0; p < N_PUSH; ++p)
    for (int s = 0; s < N_SEGS; ++s) {
      CHECK_HIP(hipFree(dev[p][s]));
      free(host[p][s]);
    }
  free(got);
  CHECK_CHEB(cheb_cache_destroy(cache));
  CHECK_HIP(hipFree(arena));
  if (failures) {
    fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  printf("c gpu ok\n");
  return 0;
}
