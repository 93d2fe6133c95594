// Several threads drive the library's host code at once (weights, tables,
// launch shape, error messages, one ring handle per thread), for a build
// under ThreadSanitizer with the device launchers stubbed out.  Prints
// "threads ok" and exits 0 when every check holds.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <string>
#include <thread>
#include <vector>

#include "cheb.h"

namespace {

std::atomic<int> g_failures{0};

void check(bool ok, const char *what) {
  if (!ok) {
    fprintf(stderr, "check failed: %s\n", what);
    g_failures.fetch_add(1);
  }
}

void worker(int id, const std::vector<double> &ref_w) {
  const double x[6] = {0.96, 0.9, 0.8, 0.72, 0.6, 0.5};
  const double targets[4] = {0.48, 0.46, 0.44, 0.42};
  std::vector<double> abscissa(50);
  for (int s = 0; s < 50; ++s) abscissa[size_t(s)] = 1.0 - s / 50.0;
  const int64_t seg[3] = {4096, 1000, 24};
  for (int it = 0; it < 200; ++it) {
    // weights, compared bit for bit with the single-threaded result
    double w[24];
    check(cheb_precompute_weights(x, 6, targets, 4, w) == CHEB_OK, "weights");
    check(memcmp(w, ref_w.data(), sizeof w) == 0, "weights equal the reference");
    check(strcmp(cheb_last_error(), "") == 0, "no error after success");
    // an error whose message names a value only this thread uses
    const double dup = 100.0 + id;
    const double bad[3] = {dup, 1.0, dup};
    check(cheb_precompute_weights(bad, 3, targets, 1, w) == CHEB_E_DUPNODE, "duplicate");
    char want[64];
    snprintf(want, sizeof want, "(%.17g)", dup);
    check(strstr(cheb_last_error(), want) != nullptr, "error message is this thread's");
    // launch shape: set and read back a whole setting
    cheb_launch_config c = {id % 2 ? 256 : 64, id % 2 ? 4 : 1, 1, 0, id % 2 ? 12 : 8};
    check(cheb_set_launch_config(&c) == CHEB_OK, "set launch shape");
    cheb_launch_config g;
    check(cheb_get_launch_config(&g) == CHEB_OK, "get launch shape");
    check((g.block == 256 && g.unroll == 4 && g.waves_per_cu == 12) ||
              (g.block == 64 && g.unroll == 1 && g.waves_per_cu == 8),
          "launch shape is one whole setting");
    // a table per thread
    cheb_table *t = nullptr;
    check(cheb_table_build(&t, 50, 1, 1, 6, 6, abscissa.data(), CHEB_SHORT_LOWER) == CHEB_OK,
          "table build");
    int32_t pred = 0, used = 0, nodes[8];
    double row[8];
    check(cheb_table_step(t, 27, &pred, &used, nodes, row) == CHEB_OK && pred == 1 && used == 6,
          "table step");
    cheb_table_destroy(t);
    // a ring handle per thread over a fake, never dereferenced arena
    size_t arena_bytes = 0;
    check(cheb_cache_layout(4, CHEB_BF16, seg, 3, nullptr, nullptr, nullptr, &arena_bytes) ==
              CHEB_OK,
          "layout");
    void *arena = reinterpret_cast<void *>(uintptr_t(1) << 40);
    cheb_cache *c4 = nullptr;
    check(cheb_cache_create(&c4, 4, CHEB_BF16, seg, 3, arena, arena_bytes) == CHEB_OK, "create");
    for (int k = 0; k < 6; ++k) {
      void *slot = nullptr;
      check(cheb_cache_begin_push(c4, &slot) == CHEB_OK, "begin push");
      check(cheb_cache_commit(c4, double(k) + 0.25 * id) == CHEB_OK, "commit");
    }
    double held[4];
    int32_t count = 0;
    check(cheb_cache_history(c4, held, &count) == CHEB_OK && count == 4, "history");
    check(held[0] == 2.0 + 0.25 * id && held[3] == 5.0 + 0.25 * id, "FIFO order");
    cheb_cache_destroy(c4);
  }
}

}  // namespace

int main() {
  const double x[6] = {0.96, 0.9, 0.8, 0.72, 0.6, 0.5};
  const double targets[4] = {0.48, 0.46, 0.44, 0.42};
  std::vector<double> ref_w(24);
  if (cheb_precompute_weights(x, 6, targets, 4, ref_w.data()) != CHEB_OK) return 1;
  std::vector<std::thread> ts;
  for (int i = 0; i < 8; ++i) ts.emplace_back(worker, i, std::cref(ref_w));
  for (auto &t : ts) t.join();
  if (g_failures.load() != 0) return 1;
  printf("threads ok\n");
  return 0;
}
