// Stand-ins for the device launchers of libcheb, for a host-only build of
// the library's C++ sources under AddressSanitizer / UBSan.  The host test
// program never reaches a launch (every call it makes is refused during
// argument checking, or is metadata only), so each stub reports an error.
#include "internal.h"

namespace cheb {

int launch_combine(int, const void *const *, int, const double *, int, void *const *, int64_t,
                   hipStream_t) {
  return fail(CHEB_E_HIP, "host-only build: no device launch");
}

int launch_gather(int, void *, const GatherSeg *, int, hipStream_t) {
  return fail(CHEB_E_HIP, "host-only build: no device launch");
}

int residual_max_cover() { return 128; }

int launch_residual(int, int, const uint64_t *, const double *, const int64_t *, int,
                    const float *, float *, int64_t, int64_t, hipStream_t) {
  return fail(CHEB_E_HIP, "host-only build: no device launch");
}

}  // namespace cheb
