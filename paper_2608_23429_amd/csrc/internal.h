// Internal declarations shared by the host sources and the kernel launchers
// of libcheb.  Not installed; the public interface is include/cheb.h.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "cheb.h"

namespace cheb {

// Records a message for cheb_last_error() and returns `code`.
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
// Clears the thread's message and returns CHEB_OK.
int ok();

// Storage type traits.
inline int elem_bytes(int dtype) { return dtype == CHEB_F32 ? 4 : 2; }
inline int elems_per_vec(int dtype) { return 16 / elem_bytes(dtype); }
inline bool valid_dtype(int dtype) {
  return dtype == CHEB_BF16 || dtype == CHEB_F32 || dtype == CHEB_F16;
}

// Largest number of 16-byte vectors one streaming launch covers (keeps every
// in-kernel index below 2^31 so 32-bit index arithmetic cannot wrap).
constexpr int64_t kMaxVecs = int64_t(1) << 31;

// History entries in the interleaved layout: the arena is cut into chunks of
// kChunkVecs 16-byte vectors (32 KiB); chunk c of entry ("lane") j sits at
// lane_base_j + c * super_vecs vectors, with lane_base_j = region + j chunks
// and super_vecs = n_slots * kChunkVecs.  The region starts on a kLaneAlign
// boundary.  Vector v of an entry is therefore at
//     lane_base + (v / kChunkVecs) * super_vecs + v % kChunkVecs,
// which is v itself for super_vecs == kChunkVecs: the slot layout (every
// entry contiguous) is the same formula with that stride.
constexpr int kChunkShift = 11;
constexpr int64_t kChunkVecs = int64_t(1) << kChunkShift;
constexpr size_t kChunkBytes = size_t(kChunkVecs) * 16;
constexpr size_t kLaneAlign = size_t(64) << 10;

// Current process-wide launch shape.
cheb_launch_config launch_shape();

// Compute units and LDS bytes per compute unit of the current device
// (cached per device).
int device_info(int *cus, int *lds_per_cu);

// One row of barycentric interpolation coefficients (host, fp64).  Returns
// CHEB_OK or an error code with the message set.
int weights_row(const double *x, int n, double target, double *w);

// out[m][i] = sum_k w[m * n + k] * src[k][i], i < numel, m < n_out, in one
// launch.  Arguments already validated: 1 <= n <= CHEB_MAX_SLOTS,
// 1 <= n_out <= CHEB_MAX_OUTPUTS, pointers 16-byte aligned, numel below the
// limit.  src[k] is an entry base; super_vecs is kChunkVecs for contiguous
// sources, else the interleaved chunk stride (then numel is a whole number
// of vectors).  Outputs are always contiguous.
int launch_combine(int dtype, const void *const *src, int n, const double *w, int n_out,
                   void *const *out, int64_t numel, int64_t super_vecs, hipStream_t stream);

// Validation of cheb_combine_multi's arguments followed by launch_combine.
int combine_checked(const void *const *src, int32_t n_src, const double *w, int32_t n_out,
                    void *const *out, int64_t numel, int32_t dtype, int64_t super_vecs,
                    void *stream);

// Prediction from the newest `used` entries of the ring (oldest of them
// first): out[m] = sum_j w[m * used + j] * entry_j, with the cache's checks.
int extrapolate_newest(cheb_cache *c, int32_t used, const double *w, int32_t n_out,
                       void *const *out, void *stream);

// Segment copy into one slot; zero-fills each segment's padding up to the
// next 16-byte boundary.
struct GatherSeg {
  const void *src;     // device, 16-byte aligned
  int64_t dst_offset;  // elements from the slot base (16-byte multiple)
  int64_t numel;       // elements to copy
};
int launch_gather(int dtype, void *slot_base, const GatherSeg *segs, int n_segs,
                  int64_t super_vecs, hipStream_t stream);

// Read-only view of a cache's layout and ring state (cache.cpp).
struct CacheView {
  int32_t n_slots, dtype, count, n_segs, layout;
  bool push_open;
  const int64_t *seg_numel, *seg_offset;
  int64_t slot_numel;
  int64_t super_vecs;  // kChunkVecs for the slot layout
  const char *arena;
  size_t arena_bytes;
};
int cache_view(const cheb_cache *c, CacheView *v);

// Residual kernel (kernels.hip): x_out[j] = x_in[j] + sum over the ncover
// offsets delta[c] and entries k < n of w[k] * (the 16-byte vector at
//   contiguous (super_vecs == kChunkVecs): base[k] + delta[c] + 16 * j bytes;
//   interleaved: vector v = delta[c] + j of the entry at base[k], placed by
//   the chunk formula above),
// for residual vectors j in [vec_begin, vec_begin + n_vec).
// ncover <= residual_max_cover(); vector indices below 2^31.
int residual_max_cover();
int launch_residual(int dtype, int n, const uint64_t *base, const double *w,
                    const int64_t *delta, int ncover, const float *x_in, float *x_out,
                    int64_t vec_begin, int64_t n_vec, int64_t super_vecs, hipStream_t stream);

}  // namespace cheb
