// Stream ceilings of the benchmark (gfx950): trivial-body kernels with the
// access pattern of the skipped-step prediction, timed in the same run as
// the prediction so that its bandwidth can be read against what the chip
// sustains for the same mix of reads and writes.
//
// Every kernel moves 16-byte vectors with non-temporal loads and stores, one
// vector per lane, one block per block-sized run of vectors, in one of the
// prediction's two launch shapes: 1024-lane blocks at full occupancy, or
// 64-lane blocks with the waves per compute unit capped by a reservation of
// LDS that the kernel never touches.  The body is an XOR of the loaded
// vectors, so arithmetic costs nothing.
//   kind 0  read n_src contiguous streams, no store (a store that the data
//           never triggers keeps the loads alive)
//   kind 1  read n_src contiguous streams, write one stream
//   kind 2  read n_src chunk-interleaved lanes of one region (32 KiB chunks,
//           lane k of chunk c at (c * n_src + k) chunks from src[0]), write
//           one contiguous stream
//   kind 3  write one stream
//   kind 4  read as kind 2, no store (interleaved read-only)
//   kind 5  read as kind 2, store with plain (cached) stores into a window of
//           window_vecs vectors at dst, wrapping: sized to stay in the
//           XCDs' L2 or in the last-level cache, it shows what the stores
//           cost when they leave the L2 but not the chip, or not the XCD
// Built by __graft_entry__.build() into bench_ceiling.so beside this file;
// only bench.py loads it.
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kChunkShift = 11;  // 2048 vectors = 32 KiB
constexpr uint32_t kChunkVecs = 1u << kChunkShift;

struct Srcs {
  const u32x4 *p[8];
};

template <int NS, int KIND, int BLK>
__global__ __launch_bounds__(BLK) void stream_kernel(Srcs s, u32x4 *__restrict__ dst,
                                                     uint32_t n_vec, uint32_t window_mask) {
  const uint32_t i = blockIdx.x * uint32_t(BLK) + threadIdx.x;
  if (i >= n_vec) return;
  u32x4 x = {i, 0u, 0u, 0u};
  if constexpr (KIND != 3) {
    u32x4 v[NS];
    if constexpr (KIND == 2 || KIND == 4 || KIND == 5) {
      const uint64_t base = uint64_t(i >> kChunkShift) * uint64_t(NS) * kChunkVecs +
                            (i & (kChunkVecs - 1));
#pragma unroll
      for (int k = 0; k < NS; ++k)
        v[k] = __builtin_nontemporal_load(s.p[0] + base + uint64_t(k) * kChunkVecs);
    } else {
#pragma unroll
      for (int k = 0; k < NS; ++k) v[k] = __builtin_nontemporal_load(s.p[k] + i);
    }
    x = v[0];
#pragma unroll
    for (int k = 1; k < NS; ++k) x ^= v[k];
  }
  if constexpr (KIND == 0 || KIND == 4) {
    // Taken only if four words match a fixed pattern; dst[i] is in bounds.
    if (x[0] == 0x9e3779b9u && x[1] == 0x7f4a7c15u && x[2] == 0xf39cc060u && x[3] == 0x5ced7e1bu)
      dst[i] = x;
  } else if constexpr (KIND == 5) {
    dst[i & window_mask] = x;
  } else {
    __builtin_nontemporal_store(x, dst + i);
  }
}

template <int KIND, int BLK>
hipError_t launch_kind(int n_src, const Srcs &s, u32x4 *dst, uint32_t n_vec, uint32_t mask,
                       size_t lds, hipStream_t st) {
  const dim3 grid((n_vec + BLK - 1) / BLK);
  switch (n_src) {
#define CEIL_CASE(N) \
  case N: hipLaunchKernelGGL((stream_kernel<N, KIND, BLK>), grid, dim3(BLK), lds, st, s, dst, n_vec, mask); break;
    CEIL_CASE(1) CEIL_CASE(2) CEIL_CASE(3) CEIL_CASE(4) CEIL_CASE(5) CEIL_CASE(6) CEIL_CASE(7)
    CEIL_CASE(8)
#undef CEIL_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int BLK>
hipError_t launch(int kind, int n_src, const Srcs &s, u32x4 *d, uint32_t n, uint32_t mask,
                  size_t lds, hipStream_t st) {
  switch (kind) {
    case 0: return launch_kind<0, BLK>(n_src, s, d, n, mask, lds, st);
    case 1: return launch_kind<1, BLK>(n_src, s, d, n, mask, lds, st);
    case 2: return launch_kind<2, BLK>(n_src, s, d, n, mask, lds, st);
    case 4: return launch_kind<4, BLK>(n_src, s, d, n, mask, lds, st);
    case 5: return launch_kind<5, BLK>(n_src, s, d, n, mask, lds, st);
    default: return launch_kind<3, BLK>(1, s, d, n, mask, lds, st);
  }
}

}  // namespace

// Launches one ceiling kernel over n_vec 16-byte vectors on `stream`.
//   kind   0..5 as above; n_src 1..8 (ignored for kind 3).
//   src    [n_src] device pointers, 16-byte aligned, n_vec vectors each
//          (kinds 2, 4, 5: src[0] is the interleaved region, n_src * n_vec
//          vectors rounded up to whole chunks per lane).
//   dst    device pointer to n_vec vectors (kinds 0 and 4: written only in
//          the never-taken case; kind 5: window_vecs vectors).
//   window_vecs  kind 5 only: a power of two, 1 .. n_vec.
//   waves_per_cu  0: 1024-lane blocks at full occupancy; 3..32: 64-lane
//          blocks, each reserving 1/waves_per_cu of the compute unit's LDS
//          (rounded down to 512 bytes, at most 64 KiB), so that about that
//          many waves share a compute unit.
// Returns 0, or -1 for arguments out of range, or the HIP error code of the
// launch or of the device query.
extern "C" __attribute__((visibility("default"))) int ceiling_stream(int kind, const void *const *src,
                                                                     int n_src, void *dst,
                                                                     int64_t n_vec,
                                                                     int64_t window_vecs,
                                                                     int waves_per_cu,
                                                                     void *stream) {
  if (kind < 0 || kind > 5 || n_vec < 0 || n_vec >= (int64_t(1) << 31) || !dst) return -1;
  if (waves_per_cu != 0 && (waves_per_cu < 3 || waves_per_cu > 32)) return -1;
  if (kind == 5 && (window_vecs < 1 || window_vecs > n_vec || (window_vecs & (window_vecs - 1))))
    return -1;
  if (kind != 3 && (n_src < 1 || n_src > 8 || !src)) return -1;
  if (n_vec == 0) return 0;
  Srcs s = {};
  if (kind != 3)
    for (int k = 0; k < (kind == 2 || kind == 4 || kind == 5 ? 1 : n_src); ++k) {
      if (!src[k]) return -1;
      s.p[k] = static_cast<const u32x4 *>(src[k]);
    }
  u32x4 *d = static_cast<u32x4 *>(dst);
  const uint32_t n = uint32_t(n_vec);
  const uint32_t mask = kind == 5 ? uint32_t(window_vecs - 1) : 0u;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (waves_per_cu == 0) {
    e = launch<1024>(kind, n_src, s, d, n, mask, 0, st);
  } else {
    int dev = 0, lds_per_cu = 0;
    e = hipGetDevice(&dev);
    if (e == hipSuccess)
      e = hipDeviceGetAttribute(&lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev);
    if (e != hipSuccess) return int(e);
    const size_t lds = size_t(lds_per_cu / waves_per_cu) / 512 * 512;
    if (lds > (size_t(64) << 10)) return -1;
    e = launch<64>(kind, n_src, s, d, n, mask, lds, st);
  }
  return e == hipSuccess ? 0 : int(e);
}

// LDS bytes per compute unit of the current device, as the runtime reports
// it (what the occupancy cap divides), or -1 if the query fails.
extern "C" __attribute__((visibility("default"))) int ceiling_lds_per_cu(void) {
  int dev = 0, lds = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) !=
      hipSuccess)
    return -1;
  return lds;
}
