// Stand-ins for the device launchers of libcheb, for a host-only build of
// the library's C++ sources under AddressSanitizer / UBSan / ThreadSanitizer.
// Prediction and residual launches always report an error (the host test
// programs never reach one with valid arguments).  The segment-copy launcher
// models the real one's batches of 64 segments: a budget set by
// stub_gather_batches_ok() says how many batches succeed before one fails,
// so a push that fails part-way through its launches can be tested on the
// CPU.  The budget starts at 0 (every copy fails).
#include <atomic>

#include "internal.h"

namespace {
std::atomic<int> g_gather_batches_ok{0};
}

extern "C" void stub_gather_batches_ok(int n) { g_gather_batches_ok.store(n); }

namespace cheb {

int launch_combine(int, const void *const *, int, const double *, int, void *const *, int64_t,
                   int64_t, hipStream_t) {
  return fail(CHEB_E_HIP, "host-only build: no device launch");
}

int launch_gather(int, void *, const GatherSeg *, int n_segs, int64_t, hipStream_t) {
  for (int first = 0; first < n_segs; first += 64) {
    if (g_gather_batches_ok.fetch_sub(1) <= 0) {
      g_gather_batches_ok.store(0);
      return fail(CHEB_E_HIP, "host-only build: copy launch %d refused", first / 64);
    }
  }
  return ok();
}

int residual_max_cover() { return 128; }

int launch_residual(int, int, const uint64_t *, const double *, const int64_t *, int,
                    const float *, float *, int64_t, int64_t, int64_t, hipStream_t) {
  return fail(CHEB_E_HIP, "host-only build: no device launch");
}

}  // namespace cheb
