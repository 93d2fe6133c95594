// Device kernels of libcheb for gfx950 (CDNA4, wave64).
//
// 1. The skipped-step prediction (paper, Section 3.3, forward application
//    equation; Algorithm 1, extrapolation branch): out = sum_k w_k H_k over
//    the flattened feature cache, for one target or for several targets at
//    once (all of them depend on the same history).  Pure streaming work:
//    (n+1) x 16 bytes of HBM traffic per 16-byte output vector and 2n flops
//    per element, far below the fp32 ridge point, so the kernel is laid out
//    for bandwidth: 128-bit coalesced loads (a wave covers 1 KiB contiguous
//    per load instruction), all n x unroll loads of a thread issued before
//    any arithmetic, weights as kernel arguments (they live in SGPRs), fp32
//    accumulation for bf16 and fp16 storage and fp64 for fp32 storage, and
//    one hardware round-to-nearest-even pack per element pair
//    (v_cvt_pk_bf16_f32, v_cvt_pk_f16_f32).  No LDS: nothing is reused
//    across lanes.
// 2. The full-step push (Algorithm 1, full computation: store (s, f_s) in
//    the history): one launch copies up to 64 segments into a slot.
// 3. Residual application on a skipped step (Section 3.1, block equation):
//    the block stack's sum of predicted module outputs added to the
//    residual stream in one pass.
// History entries are either contiguous slots or chunk-interleaved lanes
// (internal.h): vector v of an entry is at (v / 2048) * super + v % 2048
// from the entry's base, which is v itself when super is 2048.  Every
// kernel tests that one uniform value and takes the plain 32-bit indexing
// for contiguous entries.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include <algorithm>

#include "internal.h"

namespace cheb {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

template <bool NT>
__device__ __forceinline__ u32x4 load16(const u32x4 *p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}

template <bool NT>
__device__ __forceinline__ void store16(u32x4 *p, u32x4 v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

// History pointers (oldest to newest), output pointers and one weight row
// per output, passed by value as kernel arguments (they land in SGPRs).
// `super` is the entries' chunk stride in vectors (kChunkVecs: contiguous).
template <int NS, int NO, typename W>
struct Hist {
  const u32x4 *p[NS];
  u32x4 *o[NO];
  W w[NO][NS];
  uint64_t super;
};

// Vector v of an interleaved entry, relative to the entry's base.
__device__ __forceinline__ uint64_t lane_vec(uint64_t v, uint64_t super) {
  return (v >> kChunkShift) * super + (v & uint64_t(kChunkVecs - 1));
}

// Ragged end of a stateless combination: `count` (< elements per vector)
// trailing elements starting at element `first`, done by block 0.
struct Tail {
  uint32_t count;
  uint64_t first;
};

// ---- bfloat16 storage, fp32 accumulation ---------------------------------

struct Bf16Op {
  using W = float;
  using E = uint16_t;

  __device__ __forceinline__ static float lo(uint32_t word) {
    return __uint_as_float(word << 16);  // element 2q (low half)
  }
  __device__ __forceinline__ static float hi(uint32_t word) {
    return __uint_as_float(word & 0xffff0000u);  // element 2q+1
  }

  template <int NS>
  __device__ __forceinline__ static u32x4 vec(const u32x4 (&v)[NS], const W (&w)[NS]) {
    float a[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      a[2 * q] = w[0] * lo(v[0][q]);
      a[2 * q + 1] = w[0] * hi(v[0][q]);
    }
#pragma unroll
    for (int k = 1; k < NS; ++k) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        a[2 * q] = fmaf(w[k], lo(v[k][q]), a[2 * q]);
        a[2 * q + 1] = fmaf(w[k], hi(v[k][q]), a[2 * q + 1]);
      }
    }
    u32x4 r;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f32x2 pair = {a[2 * q], a[2 * q + 1]};
      r[q] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pair, bf16x2));
    }
    return r;
  }

  template <int NS>
  __device__ __forceinline__ static E scalar(const E *const (&p)[NS], const W (&w)[NS],
                                             uint64_t i) {
    float a = w[0] * __uint_as_float(uint32_t(p[0][i]) << 16);
#pragma unroll
    for (int k = 1; k < NS; ++k) a = fmaf(w[k], __uint_as_float(uint32_t(p[k][i]) << 16), a);
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(a));
  }
};

// ---- binary16 storage, fp32 accumulation ---------------------------------

struct F16Op {
  using W = float;
  using E = uint16_t;

  __device__ __forceinline__ static f32x2 pair(uint32_t word) {  // elements 2q, 2q+1
    return __builtin_convertvector(__builtin_bit_cast(f16x2, word), f32x2);
  }

  template <int NS>
  __device__ __forceinline__ static u32x4 vec(const u32x4 (&v)[NS], const W (&w)[NS]) {
    float a[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x2 p = pair(v[0][q]);
      a[2 * q] = w[0] * p.x;
      a[2 * q + 1] = w[0] * p.y;
    }
#pragma unroll
    for (int k = 1; k < NS; ++k) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x2 p = pair(v[k][q]);
        a[2 * q] = fmaf(w[k], p.x, a[2 * q]);
        a[2 * q + 1] = fmaf(w[k], p.y, a[2 * q + 1]);
      }
    }
    u32x4 r;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f32x2 pr = {a[2 * q], a[2 * q + 1]};
      r[q] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pr, f16x2));
    }
    return r;
  }

  template <int NS>
  __device__ __forceinline__ static E scalar(const E *const (&p)[NS], const W (&w)[NS],
                                             uint64_t i) {
    float a = w[0] * float(__builtin_bit_cast(_Float16, p[0][i]));
#pragma unroll
    for (int k = 1; k < NS; ++k) a = fmaf(w[k], float(__builtin_bit_cast(_Float16, p[k][i])), a);
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(a));
  }
};

// ---- binary32 storage, fp64 accumulation ---------------------------------

struct F32Op {
  using W = double;
  using E = float;

  template <int NS>
  __device__ __forceinline__ static u32x4 vec(const u32x4 (&v)[NS], const W (&w)[NS]) {
    double a[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) a[q] = w[0] * double(__uint_as_float(v[0][q]));
#pragma unroll
    for (int k = 1; k < NS; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) a[q] = fma(w[k], double(__uint_as_float(v[k][q])), a[q]);
    u32x4 r;
#pragma unroll
    for (int q = 0; q < 4; ++q) r[q] = __float_as_uint(float(a[q]));
    return r;
  }

  template <int NS>
  __device__ __forceinline__ static E scalar(const E *const (&p)[NS], const W (&w)[NS],
                                             uint64_t i) {
    double a = w[0] * double(p[0][i]);
#pragma unroll
    for (int k = 1; k < NS; ++k) a = fma(w[k], double(p[k][i]), a);
    return float(a);
  }
};

// ---- the streaming kernel -------------------------------------------------
//
// The vector range [0, n_vec) is cut into tiles of BLK * U vectors.  A block
// takes tiles blockIdx.x, blockIdx.x + gridDim.x, ... (one tile per block
// when the grid covers the range, a persistent loop otherwise).  In a tile,
// lane t handles vectors t, t + BLK, ..., so every load instruction of a
// wave reads 64 consecutive 16-byte vectors (1 KiB).  A scheduling barrier
// keeps all NS x U loads of a thread ahead of its arithmetic, so each wave
// has its whole working set in flight before it waits.  With NO > 1 the same
// loaded history feeds NO weight rows and NO outputs: every skipped step
// between two full steps is predicted in one pass over the history.
template <class Op, int NS, int NO, int BLK, int U, bool NT>
__global__ __launch_bounds__(BLK) void combine_kernel(Hist<NS, NO, typename Op::W> h,
                                                      uint32_t n_vec, uint32_t n_tiles,
                                                      Tail tail) {
  const bool flat = h.super == uint64_t(kChunkVecs);
  for (uint32_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    const uint32_t base = tile * uint32_t(BLK * U) + threadIdx.x;
    if (base + uint32_t((U - 1) * BLK) < n_vec) {
      u32x4 v[U][NS];
      if (flat) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int k = 0; k < NS; ++k) v[u][k] = load16<NT>(h.p[k] + base + u * BLK);
      } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const uint64_t off = lane_vec(base + u * BLK, h.super);
#pragma unroll
          for (int k = 0; k < NS; ++k) v[u][k] = load16<NT>(h.p[k] + off);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int m = 0; m < NO; ++m)
          store16<NT>(h.o[m] + base + u * BLK, Op::template vec<NS>(v[u], h.w[m]));
    } else {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t i = base + u * BLK;
        if (i < n_vec) {
          const uint64_t off = flat ? uint64_t(i) : lane_vec(i, h.super);
          u32x4 v[NS];
#pragma unroll
          for (int k = 0; k < NS; ++k) v[k] = load16<NT>(h.p[k] + off);
#pragma unroll
          for (int m = 0; m < NO; ++m) store16<NT>(h.o[m] + i, Op::template vec<NS>(v, h.w[m]));
        }
      }
    }
  }
  // A ragged tail only exists for contiguous sources (the host ensures it).
  if (tail.count != 0 && blockIdx.x == 0 && threadIdx.x < tail.count) {
    using E = typename Op::E;
    const E *p[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) p[k] = reinterpret_cast<const E *>(h.p[k]);
    const uint64_t i = tail.first + threadIdx.x;
#pragma unroll
    for (int m = 0; m < NO; ++m)
      reinterpret_cast<E *>(h.o[m])[i] = Op::template scalar<NS>(p, h.w[m], i);
  }
}

// The device the launch goes to.
struct Gpu {
  int cus;         // compute units
  int lds_per_cu;  // LDS bytes per compute unit
  int waves;       // occupancy cap in waves per compute unit, 0: none
};

// Waves per compute unit the prediction streams best with, from the history
// size NS and the number of outputs NO.  Measured on MI355X (FLUX- and
// DiT-sized bf16 streams): the mix of NS reads and the output's writes runs
// fastest with about 44 KiB of loads in flight per compute unit for one
// output (NS x 1 KiB per 64-lane wave: 7 waves for NS = 6, 9 for NS = 5)
// and about 36 KiB for several (6 and 7); more waves flood the memory queues
// and slow the writes.  Below 6 waves the latency is no longer covered and
// the rate falls steeply, hence the floor.  Two entries or fewer stream as
// well at full occupancy: no cap.
int auto_waves(int ns, int no) {
  if (ns <= 2) return 0;
  const int kib = no == 1 ? 44 : 36;
  return std::max(6, (kib + ns / 2) / ns);
}

// Dynamic LDS a block reserves, and never touches, so that about `waves`
// waves of the kernel share a compute unit (the LDS is what runs out): an
// equal share of the compute unit's LDS, rounded down to 512 bytes.  Zero
// when there is no cap, when the cap is at the hardware's own limit, or when
// one block would need more than the default 64 KiB of dynamic LDS.
template <int BLK>
size_t occupancy_lds(const Gpu &g) {
  constexpr int kWavesPerBlock = BLK / 64;
  if (g.waves <= 0 || g.lds_per_cu <= 0) return 0;
  const int blocks = std::max(1, g.waves / kWavesPerBlock);
  if (blocks * kWavesPerBlock >= 32) return 0;
  const size_t per = size_t(g.lds_per_cu / blocks) / 512 * 512;
  return per <= size_t(64) << 10 ? per : 0;
}

template <class Op, int NS, int NO, int BLK, int U, bool NT>
hipError_t launch_shape(const Hist<NS, NO, typename Op::W> &h, uint32_t n_vec, Tail tail,
                        int blocks_per_cu, const Gpu &g, hipStream_t s) {
  const uint32_t per_tile = uint32_t(BLK * U);
  const uint32_t n_tiles = (n_vec + per_tile - 1) / per_tile;
  uint32_t grid = std::max<uint32_t>(n_tiles, 1u);
  if (blocks_per_cu > 0) grid = std::min<uint32_t>(grid, uint32_t(blocks_per_cu) * uint32_t(g.cus));
  hipLaunchKernelGGL((combine_kernel<Op, NS, NO, BLK, U, NT>), dim3(grid), dim3(BLK),
                     occupancy_lds<BLK>(g), s, h, n_vec, n_tiles, tail);
  return hipGetLastError();
}

// Single output: every launch shape of the tuning interface.
template <class Op, int NS, bool NT>
hipError_t launch_one(const Hist<NS, 1, typename Op::W> &h, uint32_t n_vec, Tail tail,
                      const cheb_launch_config &cfg, const Gpu &dev, hipStream_t s) {
  const int b = cfg.block, u = cfg.unroll, g = cfg.blocks_per_cu;
  // A problem too small to give every compute unit a few 1024-thread blocks
  // runs with 256-thread blocks instead (four times as many blocks).
  const bool small = uint64_t(n_vec) < uint64_t(4 * 1024) * uint64_t(dev.cus);
  if (b == 64) return launch_shape<Op, NS, 1, 64, 1, NT>(h, n_vec, tail, g, dev, s);
  if (b == 1024 && small) return launch_shape<Op, NS, 1, 256, 1, NT>(h, n_vec, tail, g, dev, s);
  if (b == 1024) return launch_shape<Op, NS, 1, 1024, 1, NT>(h, n_vec, tail, g, dev, s);
  if (b == 512) {
    if (u == 1) return launch_shape<Op, NS, 1, 512, 1, NT>(h, n_vec, tail, g, dev, s);
    return launch_shape<Op, NS, 1, 512, 2, NT>(h, n_vec, tail, g, dev, s);
  }
  if (u == 1) return launch_shape<Op, NS, 1, 256, 1, NT>(h, n_vec, tail, g, dev, s);
  if (u == 2) return launch_shape<Op, NS, 1, 256, 2, NT>(h, n_vec, tail, g, dev, s);
  return launch_shape<Op, NS, 1, 256, 4, NT>(h, n_vec, tail, g, dev, s);
}

// Several outputs: one vector per lane, a grid covering the range, 64-lane
// blocks (under the occupancy cap) or 1024-lane blocks for any other
// configured block, and the non-temporal hint as configured; this keeps the
// number of kernel instances bounded.
template <class Op, int NS, int NO>
hipError_t launch_many(const Hist<NS, NO, typename Op::W> &h, uint32_t n_vec, Tail tail,
                       const cheb_launch_config &cfg, const Gpu &dev, hipStream_t s) {
  if (cfg.block == 64)
    return cfg.nontemporal ? launch_shape<Op, NS, NO, 64, 1, true>(h, n_vec, tail, 0, dev, s)
                           : launch_shape<Op, NS, NO, 64, 1, false>(h, n_vec, tail, 0, dev, s);
  return cfg.nontemporal ? launch_shape<Op, NS, NO, 1024, 1, true>(h, n_vec, tail, 0, dev, s)
                         : launch_shape<Op, NS, NO, 1024, 1, false>(h, n_vec, tail, 0, dev, s);
}

template <class Op, int NS, int NO>
hipError_t launch_ns_no(const void *const *src, const double *w, void *const *out,
                        int64_t numel, int64_t super_vecs, const cheb_launch_config &cfg,
                        const Gpu &dev0, hipStream_t s) {
  constexpr int kVec = 16 / int(sizeof(typename Op::E));
  Gpu dev = dev0;
  dev.waves = cfg.waves_per_cu == 0 ? auto_waves(NS, NO) : std::max(0, cfg.waves_per_cu);
  Hist<NS, NO, typename Op::W> h;
  h.super = uint64_t(super_vecs);
  for (int k = 0; k < NS; ++k) h.p[k] = static_cast<const u32x4 *>(src[k]);
  for (int m = 0; m < NO; ++m) {
    h.o[m] = static_cast<u32x4 *>(out[m]);
    for (int k = 0; k < NS; ++k) h.w[m][k] = static_cast<typename Op::W>(w[m * NS + k]);
  }
  const uint32_t n_vec = uint32_t(numel / kVec);
  Tail tail{uint32_t(numel % kVec), uint64_t(numel / kVec) * kVec};
  if constexpr (NO == 1) {
    return cfg.nontemporal ? launch_one<Op, NS, true>(h, n_vec, tail, cfg, dev, s)
                           : launch_one<Op, NS, false>(h, n_vec, tail, cfg, dev, s);
  } else {
    return launch_many<Op, NS, NO>(h, n_vec, tail, cfg, dev, s);
  }
}

template <class Op, int NS>
hipError_t launch_ns(const void *const *src, const double *w, int n_out, void *const *out,
                     int64_t numel, int64_t sv, const cheb_launch_config &cfg, const Gpu &cus,
                     hipStream_t s) {
  switch (n_out) {
    case 1: return launch_ns_no<Op, NS, 1>(src, w, out, numel, sv, cfg, cus, s);
    case 2: return launch_ns_no<Op, NS, 2>(src, w, out, numel, sv, cfg, cus, s);
    case 3: return launch_ns_no<Op, NS, 3>(src, w, out, numel, sv, cfg, cus, s);
    case 4: return launch_ns_no<Op, NS, 4>(src, w, out, numel, sv, cfg, cus, s);
    case 5: return launch_ns_no<Op, NS, 5>(src, w, out, numel, sv, cfg, cus, s);
    case 6: return launch_ns_no<Op, NS, 6>(src, w, out, numel, sv, cfg, cus, s);
    case 7: return launch_ns_no<Op, NS, 7>(src, w, out, numel, sv, cfg, cus, s);
    default: return launch_ns_no<Op, NS, 8>(src, w, out, numel, sv, cfg, cus, s);
  }
}

template <class Op>
hipError_t launch_op(const void *const *src, int n, const double *w, int n_out,
                     void *const *out, int64_t numel, int64_t sv,
                     const cheb_launch_config &cfg, const Gpu &cus, hipStream_t s) {
  switch (n) {
    case 1: return launch_ns<Op, 1>(src, w, n_out, out, numel, sv, cfg, cus, s);
    case 2: return launch_ns<Op, 2>(src, w, n_out, out, numel, sv, cfg, cus, s);
    case 3: return launch_ns<Op, 3>(src, w, n_out, out, numel, sv, cfg, cus, s);
    case 4: return launch_ns<Op, 4>(src, w, n_out, out, numel, sv, cfg, cus, s);
    case 5: return launch_ns<Op, 5>(src, w, n_out, out, numel, sv, cfg, cus, s);
    case 6: return launch_ns<Op, 6>(src, w, n_out, out, numel, sv, cfg, cus, s);
    case 7: return launch_ns<Op, 7>(src, w, n_out, out, numel, sv, cfg, cus, s);
    default: return launch_ns<Op, 8>(src, w, n_out, out, numel, sv, cfg, cus, s);
  }
}

// ---- full-step push: segment gather into one slot --------------------------

constexpr int kGatherMax = 64;
// One 16-byte vector per lane.  256-lane blocks copy into an interleaved
// lane 4-5% faster than 1024-lane ones on MI355X (and as fast into a
// contiguous slot); 64-lane blocks lose on the blocks that find no work.
constexpr int kGatherBlock = 256;
constexpr uint32_t kGatherChunk = kGatherBlock;  // vectors per block

struct GatherArgs {
  const void *src[kGatherMax];
  uint64_t dst_offset[kGatherMax];  // elements
  uint64_t numel[kGatherMax];
  int32_t n;
};

// Grid: x = 256-vector chunk within a segment, y = segment.  Blocks past
// their segment's end return at once, so no block searches for its
// segment.  Source reads and slot writes are streaming (each byte is touched
// once per push), so both carry the non-temporal hint.  Vector v of the
// entry goes v vectors past `slot` (contiguous entry) or to its chunk
// position in an interleaved lane.
template <typename E>
__global__ __launch_bounds__(kGatherBlock) void gather_kernel(GatherArgs a, char *__restrict__ slot,
                                                              uint64_t super) {
  constexpr int kVec = 16 / int(sizeof(E));
  const int s = int(blockIdx.y);
  const uint64_t numel = a.numel[s];
  const uint64_t n_full = numel / kVec;
  const uint32_t rem = uint32_t(numel % kVec);
  const uint64_t i = uint64_t(blockIdx.x) * kGatherChunk + threadIdx.x;
  if (i > n_full || (i == n_full && rem == 0)) return;
  const u32x4 *src = static_cast<const u32x4 *>(a.src[s]);
  const uint64_t v = a.dst_offset[s] / kVec + i;  // segment offsets are whole vectors
  u32x4 *dst = reinterpret_cast<u32x4 *>(slot) +
               (super == uint64_t(kChunkVecs) ? v : lane_vec(v, super));
  if (i < n_full) {
    store16<true>(dst, load16<true>(src + i));
  } else {
    // Last, partial vector: copy the remaining elements one by one and zero
    // the padding up to the 16-byte boundary.
    const E *src_e = static_cast<const E *>(a.src[s]);
    E tmp[kVec];
#pragma unroll
    for (int e = 0; e < kVec; ++e) tmp[e] = (uint32_t(e) < rem) ? src_e[n_full * kVec + e] : E(0);
    u32x4 packed;
    memcpy(&packed, tmp, 16);
    *dst = packed;
  }
}

// ---- residual application on a skipped step ---------------------------------
//
// A DiT block adds its module outputs to the residual stream (Section 3.1,
// block equation).  When every module output of a step is predicted, the
// block stack adds sum_k w_k H_k[segment] for every cached segment, so
//     x_out[j] = x_in[j] + sum_{segments s covering j} sum_k w_k H_k[s, j]
// can be formed in one pass that reads the history once and never writes
// the per-module predictions.  One launch covers one interval of the
// residual on which the set of covering segments is constant (all of it for
// DiT; the text and image parts for FLUX).  The covering segments travel as
// byte offsets in the kernel arguments: entry k's element j of segment s is
// at base[k] + delta[s] + 16 * (vector index of j).  Accumulation is fp64
// (hundreds of terms per element), output fp32.

struct Bf16Dec {
  static constexpr int kVec = 8;
  __device__ __forceinline__ static void add(double (&a)[8], u32x4 v, double w) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      a[2 * q] = fma(w, double(__uint_as_float(v[q] << 16)), a[2 * q]);
      a[2 * q + 1] = fma(w, double(__uint_as_float(v[q] & 0xffff0000u)), a[2 * q + 1]);
    }
  }
};

struct F16Dec {
  static constexpr int kVec = 8;
  __device__ __forceinline__ static void add(double (&a)[8], u32x4 v, double w) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x2 p = F16Op::pair(v[q]);
      a[2 * q] = fma(w, double(p.x), a[2 * q]);
      a[2 * q + 1] = fma(w, double(p.y), a[2 * q + 1]);
    }
  }
};

struct F32Dec {
  static constexpr int kVec = 4;
  __device__ __forceinline__ static void add(double (&a)[4], u32x4 v, double w) {
#pragma unroll
    for (int q = 0; q < 4; ++q) a[q] = fma(w, double(__uint_as_float(v[q])), a[q]);
  }
};

constexpr int kResCover = 128;
constexpr int kResBlock = 1024;

template <int NS>
struct ResArgs {
  uint64_t base[NS];
  double w[NS];
  int64_t delta[kResCover];  // bytes (contiguous entries) or vectors (interleaved)
  const float *x_in;  // may be null: zero
  float *x_out;
  uint64_t super;
  uint32_t vec_begin;
  uint32_t n_vec;
  int32_t ncover;
};

// Source vector of residual vector j in covering segment s of the entry at
// `base`.
template <int NS>
__device__ __forceinline__ const u32x4 *res_src(const ResArgs<NS> &a, bool flat, uint64_t base,
                                                int32_t s, uint64_t j) {
  if (flat) return reinterpret_cast<const u32x4 *>(base + uint64_t(a.delta[s]) + j * 16u);
  return reinterpret_cast<const u32x4 *>(base) + lane_vec(uint64_t(a.delta[s]) + j, a.super);
}

// Each block starts its walk over the covering segments at a different
// segment (its index times two, modulo the count), so at any moment the
// chip's reads spread over many segments instead of all blocks reading the
// same one: measured 5-10% faster on the FLUX image interval.  Each
// element's sum is still over every covering segment exactly once.
template <class Dec, int NS>
__global__ __launch_bounds__(kResBlock) void residual_kernel(ResArgs<NS> a) {
  constexpr int V = Dec::kVec;
  const uint32_t i = blockIdx.x * uint32_t(kResBlock) + threadIdx.x;
  if (i >= a.n_vec) return;
  const uint64_t j = uint64_t(a.vec_begin) + i;  // residual vector index
  double acc[V];
  if (a.x_in) {
    const u32x4 *xi = reinterpret_cast<const u32x4 *>(a.x_in + j * V);
#pragma unroll
    for (int h = 0; h < V / 4; ++h) {
      const u32x4 x = xi[h];
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[4 * h + q] = double(__uint_as_float(x[q]));
    }
  } else {
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] = 0.0;
  }
  const bool flat = a.super == uint64_t(kChunkVecs);
  const int32_t nc = a.ncover;
  const int32_t start = nc > 0 ? int32_t((uint64_t(blockIdx.x) * 2u) % uint32_t(nc)) : 0;
  int32_t c = 0;
  for (; c + 1 < nc; c += 2) {  // two segments' loads in flight
    int32_t s0 = start + c, s1 = start + c + 1;
    if (s0 >= nc) s0 -= nc;
    if (s1 >= nc) s1 -= nc;
    u32x4 v0[NS], v1[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      v0[k] = __builtin_nontemporal_load(res_src(a, flat, a.base[k], s0, j));
      v1[k] = __builtin_nontemporal_load(res_src(a, flat, a.base[k], s1, j));
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      Dec::add(acc, v0[k], a.w[k]);
      Dec::add(acc, v1[k], a.w[k]);
    }
  }
  if (c < nc) {
    int32_t s0 = start + c;
    if (s0 >= nc) s0 -= nc;
    u32x4 v0[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) v0[k] = __builtin_nontemporal_load(res_src(a, flat, a.base[k], s0, j));
#pragma unroll
    for (int k = 0; k < NS; ++k) Dec::add(acc, v0[k], a.w[k]);
  }
  u32x4 *xo = reinterpret_cast<u32x4 *>(a.x_out + j * V);
#pragma unroll
  for (int h = 0; h < V / 4; ++h) {
    u32x4 r;
#pragma unroll
    for (int q = 0; q < 4; ++q) r[q] = __float_as_uint(float(acc[4 * h + q]));
    xo[h] = r;
  }
}

template <class Dec, int NS>
hipError_t launch_residual_ns(const uint64_t *base, const double *w, const int64_t *delta,
                              int ncover, const float *x_in, float *x_out, uint32_t vec_begin,
                              uint32_t n_vec, uint64_t super, hipStream_t s) {
  ResArgs<NS> a;
  memset(&a, 0, sizeof a);
  a.super = super;
  for (int k = 0; k < NS; ++k) {
    a.base[k] = base[k];
    a.w[k] = w[k];
  }
  for (int c = 0; c < ncover; ++c) a.delta[c] = delta[c];
  a.x_in = x_in;
  a.x_out = x_out;
  a.vec_begin = vec_begin;
  a.n_vec = n_vec;
  a.ncover = ncover;
  const uint32_t grid = (n_vec + kResBlock - 1) / kResBlock;
  hipLaunchKernelGGL((residual_kernel<Dec, NS>), dim3(grid), dim3(kResBlock), 0, s, a);
  return hipGetLastError();
}

template <class Dec>
hipError_t launch_residual_dec(int n, const uint64_t *base, const double *w, const int64_t *delta,
                               int ncover, const float *x_in, float *x_out, uint32_t vec_begin,
                               uint32_t n_vec, uint64_t sv, hipStream_t s) {
  switch (n) {
#define CHEB_RES_CASE(N) \
  case N: return launch_residual_ns<Dec, N>(base, w, delta, ncover, x_in, x_out, vec_begin, n_vec, sv, s);
    CHEB_RES_CASE(1) CHEB_RES_CASE(2) CHEB_RES_CASE(3) CHEB_RES_CASE(4)
    CHEB_RES_CASE(5) CHEB_RES_CASE(6) CHEB_RES_CASE(7)
#undef CHEB_RES_CASE
    default: return launch_residual_ns<Dec, 8>(base, w, delta, ncover, x_in, x_out, vec_begin, n_vec, sv, s);
  }
}

}  // namespace

int launch_combine(int dtype, const void *const *src, int n, const double *w, int n_out,
                   void *const *out, int64_t numel, int64_t super_vecs, hipStream_t stream) {
  if (numel == 0) return ok();
  Gpu cus{0, 0, 0};
  int rc = device_info(&cus.cus, &cus.lds_per_cu);
  if (rc != CHEB_OK) return rc;
  const cheb_launch_config cfg = launch_shape();
  hipError_t e;
  switch (dtype) {
    case CHEB_BF16:
      e = launch_op<Bf16Op>(src, n, w, n_out, out, numel, super_vecs, cfg, cus, stream);
      break;
    case CHEB_F16:
      e = launch_op<F16Op>(src, n, w, n_out, out, numel, super_vecs, cfg, cus, stream);
      break;
    default:
      e = launch_op<F32Op>(src, n, w, n_out, out, numel, super_vecs, cfg, cus, stream);
      break;
  }
  if (e != hipSuccess) return fail(CHEB_E_HIP, "combine launch failed: %s", hipGetErrorString(e));
  return ok();
}

int launch_gather(int dtype, void *slot_base, const GatherSeg *segs, int n_segs,
                  int64_t super_vecs, hipStream_t stream) {
  const int vec = elems_per_vec(dtype);
  for (int first = 0; first < n_segs; first += kGatherMax) {
    const int count = std::min(kGatherMax, n_segs - first);
    GatherArgs a;
    memset(&a, 0, sizeof a);
    uint64_t max_chunks = 0;
    int used = 0;
    for (int j = 0; j < count; ++j) {
      const GatherSeg &g = segs[first + j];
      const uint64_t vecs = (uint64_t(g.numel) + vec - 1) / vec;
      const uint64_t chunks = (vecs + kGatherChunk - 1) / kGatherChunk;
      if (chunks == 0) continue;  // empty segment: nothing to copy
      a.src[used] = g.src;
      a.dst_offset[used] = uint64_t(g.dst_offset);
      a.numel[used] = uint64_t(g.numel);
      max_chunks = std::max(max_chunks, chunks);
      ++used;
    }
    if (used == 0) continue;
    a.n = used;
    char *slot = static_cast<char *>(slot_base);
    const dim3 grid{static_cast<uint32_t>(max_chunks), static_cast<uint32_t>(used), 1u};
    const uint64_t sv = uint64_t(super_vecs);
    if (elem_bytes(dtype) == 2)
      hipLaunchKernelGGL(gather_kernel<uint16_t>, grid, dim3(kGatherBlock), 0, stream, a, slot, sv);
    else
      hipLaunchKernelGGL(gather_kernel<float>, grid, dim3(kGatherBlock), 0, stream, a, slot, sv);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(CHEB_E_HIP, "push launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

}  // namespace cheb

namespace cheb {

int residual_max_cover() { return kResCover; }

int launch_residual(int dtype, int n, const uint64_t *base, const double *w, const int64_t *delta,
                    int ncover, const float *x_in, float *x_out, int64_t vec_begin,
                    int64_t n_vec, int64_t super_vecs, hipStream_t stream) {
  if (n_vec == 0) return ok();
  const uint32_t vb = uint32_t(vec_begin), nv = uint32_t(n_vec);
  const uint64_t sv = uint64_t(super_vecs);
  hipError_t e;
  switch (dtype) {
    case CHEB_BF16:
      e = launch_residual_dec<Bf16Dec>(n, base, w, delta, ncover, x_in, x_out, vb, nv, sv, stream);
      break;
    case CHEB_F16:
      e = launch_residual_dec<F16Dec>(n, base, w, delta, ncover, x_in, x_out, vb, nv, sv, stream);
      break;
    default:
      e = launch_residual_dec<F32Dec>(n, base, w, delta, ncover, x_in, x_out, vb, nv, sv, stream);
      break;
  }
  if (e != hipSuccess) return fail(CHEB_E_HIP, "residual launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace cheb
