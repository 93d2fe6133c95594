// Residual application on a skipped step (paper, Section 3.1, block
// equation: a block adds its module outputs to the residual stream;
// Section 3.3 and Algorithm 1: on a skipped step every module output is the
// prediction sum_k w_k f_{s_k}).  The block stack's whole contribution,
// x_out = x_in + sum over cached segments of their predictions, is formed in
// one pass over the history, and the same kernel folds a full step's module
// outputs into one residual-sized entry for a collapsed history.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "internal.h"

using namespace cheb;

namespace {

struct Interval {
  int64_t begin, end;          // residual elements
  std::vector<int32_t> segs;   // segments adding into all of [begin, end)
};

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Cuts the residual into intervals on which the covering segments do not
// change.  Segments with a negative residual offset (or no elements) are
// not added.
int plan(const int64_t *seg_numel, const int64_t *res_offset, int32_t n_segs,
         int64_t res_numel, int vec, std::vector<Interval> *out) {
  if (res_numel <= 0 || res_numel % vec != 0)
    return fail(CHEB_E_INVAL, "residual size %lld must be a positive multiple of %d",
                (long long)res_numel, vec);
  if (res_numel / vec >= kMaxVecs) return fail(CHEB_E_INVAL, "residual too large");
  std::vector<int64_t> bounds = {0, res_numel};
  for (int32_t s = 0; s < n_segs; ++s) {
    if (res_offset[s] < 0 || seg_numel[s] == 0) continue;
    if (res_offset[s] % vec != 0 || seg_numel[s] % vec != 0)
      return fail(CHEB_E_ALIGN, "segment %d: residual offset and size must be multiples of %d",
                  s, vec);
    if (res_offset[s] + seg_numel[s] > res_numel)
      return fail(CHEB_E_INVAL, "segment %d ends past the residual", s);
    bounds.push_back(res_offset[s]);
    bounds.push_back(res_offset[s] + seg_numel[s]);
  }
  std::sort(bounds.begin(), bounds.end());
  bounds.erase(std::unique(bounds.begin(), bounds.end()), bounds.end());
  out->clear();
  for (size_t b = 0; b + 1 < bounds.size(); ++b) {
    Interval iv{bounds[b], bounds[b + 1], {}};
    for (int32_t s = 0; s < n_segs; ++s) {
      if (res_offset[s] < 0 || seg_numel[s] == 0) continue;
      if (res_offset[s] <= iv.begin && res_offset[s] + seg_numel[s] >= iv.end)
        iv.segs.push_back(s);
    }
    out->push_back(std::move(iv));
  }
  return CHEB_OK;
}

int check_residual_buffers(const float *x_in, float *x_out, int64_t res_numel) {
  if (!x_out) return fail(CHEB_E_INVAL, "x_out is NULL");
  if (!aligned16(x_out) || (x_in && !aligned16(x_in)))
    return fail(CHEB_E_ALIGN, "x_in and x_out must be 16-byte aligned");
  if (x_in && x_in != x_out) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(x_in), b = reinterpret_cast<uintptr_t>(x_out);
    const uintptr_t bytes = uintptr_t(res_numel) * 4u;
    if (a < b + bytes && b < a + bytes) return fail(CHEB_E_INVAL, "x_in partly overlaps x_out");
  }
  return CHEB_OK;
}

// Runs the plan: per interval, the covering segments in chunks of the
// kernel's table size; the first chunk reads x_in, later ones x_out.
template <class DeltaFn>
int run(int dtype, int n, const uint64_t *base, const double *w,
        const std::vector<Interval> &plan_iv, DeltaFn delta_of, const float *x_in, float *x_out,
        int64_t super_vecs, hipStream_t stream) {
  const int vec = elems_per_vec(dtype);
  const int max_cover = residual_max_cover();
  std::vector<int64_t> delta;
  for (const Interval &iv : plan_iv) {
    const int64_t vb = iv.begin / vec, nv = (iv.end - iv.begin) / vec;
    size_t first = 0;
    do {
      const size_t count = std::min(iv.segs.size() - first, size_t(max_cover));
      delta.assign(count, 0);
      for (size_t c = 0; c < count; ++c) delta[c] = delta_of(iv.segs[first + c]);
      const float *in = first == 0 ? x_in : x_out;
      int rc = launch_residual(dtype, n, base, w, delta.data(), int(count), in, x_out, vb, nv,
                               super_vecs, stream);
      if (rc != CHEB_OK) return rc;
      first += count;
    } while (first < iv.segs.size());
  }
  return ok();
}

}  // namespace

extern "C" {

int cheb_residual_apply(cheb_cache *c, const double *w, const int64_t *res_offset,
                        int64_t res_numel, const float *x_in, float *x_out, void *stream) {
  CacheView v;
  int rc = cache_view(c, &v);
  if (rc != CHEB_OK) return rc;
  if (!w || !res_offset) return fail(CHEB_E_INVAL, "w or res_offset is NULL");
  if (v.push_open) return fail(CHEB_E_NOTREADY, "a fused push is open");
  if (v.count < v.n_slots)
    return fail(CHEB_E_NOTREADY, "history holds %d of %d entries", v.count, v.n_slots);
  for (int32_t k = 0; k < v.n_slots; ++k)
    if (!isfinite(w[k])) return fail(CHEB_E_NONFINITE, "w[%d] is not finite", k);
  rc = check_residual_buffers(x_in, x_out, res_numel);
  if (rc != CHEB_OK) return rc;
  const uintptr_t o = reinterpret_cast<uintptr_t>(x_out), a = reinterpret_cast<uintptr_t>(v.arena);
  if (o < a + v.arena_bytes && a < o + uintptr_t(res_numel) * 4u)
    return fail(CHEB_E_INVAL, "x_out overlaps the cache arena");
  std::vector<Interval> iv;
  rc = plan(v.seg_numel, res_offset, v.n_segs, res_numel, elems_per_vec(v.dtype), &iv);
  if (rc != CHEB_OK) return rc;
  uint64_t base[CHEB_MAX_SLOTS];
  for (int32_t k = 0; k < v.n_slots; ++k) {
    void *p = nullptr;
    rc = cheb_cache_entry(c, k, &p);
    if (rc != CHEB_OK) return rc;
    base[k] = reinterpret_cast<uint64_t>(p);
  }
  // Contiguous entries: byte offset from the entry base to the segment's
  // element of residual element 0; interleaved: the same in vectors (the
  // kernel places each vector by its chunk).
  const int64_t esize = elem_bytes(v.dtype), vec = elems_per_vec(v.dtype);
  const bool contiguous = v.super_vecs == kChunkVecs;
  auto delta_of = [&](int32_t s) {
    const int64_t d = v.seg_offset[s] - res_offset[s];
    return contiguous ? d * esize : d / vec;
  };
  return run(v.dtype, v.n_slots, base, w, iv, delta_of, x_in, x_out, v.super_vecs,
             static_cast<hipStream_t>(stream));
}

int cheb_residual_reduce(const void *const *seg_src, const int64_t *seg_numel,
                         const int64_t *res_offset, int32_t n_segs, int32_t dtype,
                         const float *x_in, float *x_out, int64_t res_numel, void *stream) {
  if (!valid_dtype(dtype)) return fail(CHEB_E_DTYPE, "unknown dtype %d", dtype);
  if (!seg_src || !seg_numel || !res_offset) return fail(CHEB_E_INVAL, "segment arrays NULL");
  if (n_segs < 1) return fail(CHEB_E_INVAL, "n_segs must be at least 1");
  for (int32_t s = 0; s < n_segs; ++s) {
    if (seg_numel[s] < 0) return fail(CHEB_E_INVAL, "seg_numel[%d] is negative", s);
    if (res_offset[s] < 0 || seg_numel[s] == 0) continue;
    if (!seg_src[s]) return fail(CHEB_E_INVAL, "seg_src[%d] is NULL", s);
    if (!aligned16(seg_src[s])) return fail(CHEB_E_ALIGN, "seg_src[%d] is not 16-byte aligned", s);
  }
  int rc = check_residual_buffers(x_in, x_out, res_numel);
  if (rc != CHEB_OK) return rc;
  std::vector<Interval> iv;
  rc = plan(seg_numel, res_offset, n_segs, res_numel, elems_per_vec(dtype), &iv);
  if (rc != CHEB_OK) return rc;
  const int64_t esize = elem_bytes(dtype);
  const uint64_t base[1] = {0};
  const double one[1] = {1.0};
  auto delta_of = [&](int32_t s) {
    return int64_t(reinterpret_cast<uintptr_t>(seg_src[s])) - res_offset[s] * esize;
  };
  return run(dtype, 1, base, one, iv, delta_of, x_in, x_out, kChunkVecs,
             static_cast<hipStream_t>(stream));
}

}  // extern "C"
