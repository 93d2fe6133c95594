// History cache: the fixed-size FIFO of full-step features (paper,
// Section 3.3, forward application; Algorithm 1, online stage) kept as a
// ring of entries in one caller-owned device arena, either as contiguous
// slots or as chunk-interleaved lanes (internal.h).
#include <math.h>
#include <string.h>

#include <new>
#include <vector>

#include "internal.h"

using namespace cheb;

struct cheb_cache {
  int32_t n_slots = 0;
  int32_t dtype = CHEB_BF16;
  std::vector<int64_t> seg_numel;
  std::vector<int64_t> seg_offset;
  int64_t slot_numel = 0;
  size_t slot_stride = 0;
  char *arena = nullptr;
  size_t arena_bytes = 0;
  int32_t layout = CHEB_LAYOUT_SLOTS;
  char *region = nullptr;          // interleaved: first lane, on a kLaneAlign boundary
  int64_t super_vecs = kChunkVecs; // chunk stride of an entry (vectors)
  // Ring state: `head` is the slot the next entry goes to; the `count` held
  // entries, oldest first, are in slots head - count, ..., head - 1 (mod n).
  double slot_t[CHEB_MAX_SLOTS] = {0};
  int32_t head = 0;
  int32_t count = 0;
  bool push_open = false;

  int32_t slot_of_age(int32_t age) const {
    return ((head - count + age) % n_slots + n_slots) % n_slots;
  }
  // Base of the entry stored in `slot` (its first vector).
  char *slot_ptr(int32_t slot) const {
    return layout == CHEB_LAYOUT_SLOTS ? arena + size_t(slot) * slot_stride
                                       : region + size_t(slot) * kChunkBytes;
  }
};

namespace {

constexpr size_t kSlotAlign = 256;

int layout(int32_t n_slots, int32_t dtype, const int64_t *seg_numel, int32_t n_segs,
           std::vector<int64_t> *offsets, int64_t *slot_numel, size_t *stride,
           size_t *arena_bytes) {
  if (!valid_dtype(dtype)) return fail(CHEB_E_DTYPE, "unknown dtype %d", dtype);
  if (n_slots < 1 || n_slots > CHEB_MAX_SLOTS)
    return fail(CHEB_E_INVAL, "n_slots %d outside 1..%d", n_slots, CHEB_MAX_SLOTS);
  if (n_segs < 1) return fail(CHEB_E_INVAL, "n_segs must be at least 1");
  if (!seg_numel) return fail(CHEB_E_INVAL, "seg_numel is NULL");
  const int64_t vec = elems_per_vec(dtype);
  offsets->assign(size_t(n_segs), 0);
  int64_t pos = 0;
  for (int32_t s = 0; s < n_segs; ++s) {
    if (seg_numel[s] < 0) return fail(CHEB_E_INVAL, "seg_numel[%d] is negative", s);
    (*offsets)[size_t(s)] = pos;
    pos += (seg_numel[s] + vec - 1) / vec * vec;
    if (pos / vec >= kMaxVecs) return fail(CHEB_E_INVAL, "cache slot too large");
  }
  const size_t bytes = size_t(pos) * size_t(elem_bytes(dtype));
  const size_t str = (bytes + kSlotAlign - 1) / kSlotAlign * kSlotAlign;
  *slot_numel = pos;
  *stride = str;
  *arena_bytes = str * size_t(n_slots);
  return CHEB_OK;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Arena bytes of the interleaved layout: every lane padded to whole chunks,
// plus room to start the region on a kLaneAlign boundary.
size_t interleaved_bytes(int32_t n_slots, int64_t slot_numel, int dtype) {
  const int64_t vecs = slot_numel / elems_per_vec(dtype);
  const int64_t chunks = (vecs + kChunkVecs - 1) / kChunkVecs;
  return size_t(chunks) * size_t(n_slots) * kChunkBytes + kLaneAlign;
}

bool valid_layout(int32_t layout) {
  return layout == CHEB_LAYOUT_SLOTS || layout == CHEB_LAYOUT_INTERLEAVED;
}

// CHEB_E_DUPNODE when t equals an abscissa that stays held after the next
// entry goes in (a full ring drops its oldest first).
int check_new_abscissa(const cheb_cache *c, double t) {
  if (!isfinite(t)) return fail(CHEB_E_NONFINITE, "abscissa is not finite");
  const int32_t first = (c->count == c->n_slots) ? 1 : 0;
  for (int32_t a = first; a < c->count; ++a)
    if (c->slot_t[c->slot_of_age(a)] == t)
      return fail(CHEB_E_DUPNODE, "abscissa %.17g is already held", t);
  return CHEB_OK;
}

// Claims the slot for the next entry, dropping the oldest entry if full.
int32_t claim_slot(cheb_cache *c) {
  if (c->count == c->n_slots) c->count -= 1;  // the oldest lives in slot `head`
  return c->head;
}

void record(cheb_cache *c, double t) {
  c->slot_t[c->head] = t;
  c->head = (c->head + 1) % c->n_slots;
  c->count += 1;
}

}  // namespace

namespace cheb {

// Prediction from the newest `used` held entries (oldest of them first).
int extrapolate_newest(cheb_cache *c, int32_t used, const double *w, int32_t n_out,
                       void *const *out, void *stream) {
  if (!c || !w || !out) return fail(CHEB_E_INVAL, "cache, w or out is NULL");
  if (c->push_open) return fail(CHEB_E_NOTREADY, "a fused push is open");
  if (used < 1 || used > c->count)
    return fail(CHEB_E_NOTREADY, "history holds %d entries, %d needed", c->count, used);
  if (n_out < 1 || n_out > CHEB_MAX_OUTPUTS)
    return fail(CHEB_E_INVAL, "n_out %d outside 1..%d", n_out, CHEB_MAX_OUTPUTS);
  const void *src[CHEB_MAX_SLOTS];
  for (int32_t j = 0; j < used; ++j) src[j] = c->slot_ptr(c->slot_of_age(c->count - used + j));
  // Outputs may not touch the arena (for interleaved entries the sources
  // spread over all of it).
  if (c->slot_numel > 0) {
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(c->arena);
    const uintptr_t ob = uintptr_t(c->slot_numel) * uintptr_t(elem_bytes(c->dtype));
    for (int32_t m = 0; m < n_out; ++m) {
      if (!out[m]) return fail(CHEB_E_INVAL, "out[%d] is NULL", m);
      const uintptr_t o0 = reinterpret_cast<uintptr_t>(out[m]);
      if (o0 < a0 + c->arena_bytes && a0 < o0 + ob)
        return fail(CHEB_E_INVAL, "out[%d] overlaps the cache arena", m);
    }
  }
  return combine_checked(src, used, w, n_out, out, c->slot_numel, c->dtype, c->super_vecs,
                         stream);
}

int cache_view(const cheb_cache *c, CacheView *v) {
  if (!c || !v) return fail(CHEB_E_INVAL, "cache is NULL");
  v->n_slots = c->n_slots;
  v->dtype = c->dtype;
  v->count = c->count;
  v->n_segs = int32_t(c->seg_numel.size());
  v->push_open = c->push_open;
  v->seg_numel = c->seg_numel.data();
  v->seg_offset = c->seg_offset.data();
  v->slot_numel = c->slot_numel;
  v->layout = c->layout;
  v->super_vecs = c->super_vecs;
  v->arena = c->arena;
  v->arena_bytes = c->arena_bytes;
  return CHEB_OK;
}

}  // namespace cheb

extern "C" {

int cheb_cache_arena_bytes(int32_t n_slots, int32_t dtype, const int64_t *seg_numel,
                           int32_t n_segs, size_t *arena_bytes, size_t *slot_stride_bytes) {
  if (!arena_bytes) return fail(CHEB_E_INVAL, "arena_bytes is NULL");
  std::vector<int64_t> off;
  int64_t sn = 0;
  size_t st = 0, ab = 0;
  int rc = layout(n_slots, dtype, seg_numel, n_segs, &off, &sn, &st, &ab);
  if (rc != CHEB_OK) return rc;
  *arena_bytes = ab;
  if (slot_stride_bytes) *slot_stride_bytes = st;
  return ok();
}

int cheb_cache_layout(int32_t n_slots, int32_t dtype, const int64_t *seg_numel, int32_t n_segs,
                      int64_t *seg_offset, int64_t *slot_numel, size_t *slot_stride_bytes,
                      size_t *arena_bytes) {
  std::vector<int64_t> off;
  int64_t sn = 0;
  size_t st = 0, ab = 0;
  int rc = layout(n_slots, dtype, seg_numel, n_segs, &off, &sn, &st, &ab);
  if (rc != CHEB_OK) return rc;
  if (seg_offset) memcpy(seg_offset, off.data(), sizeof(int64_t) * off.size());
  if (slot_numel) *slot_numel = sn;
  if (slot_stride_bytes) *slot_stride_bytes = st;
  if (arena_bytes) *arena_bytes = ab;
  return ok();
}

int cheb_cache_arena_bytes_ex(int32_t n_slots, int32_t dtype, const int64_t *seg_numel,
                              int32_t n_segs, int32_t layout_kind, size_t *arena_bytes) {
  if (!arena_bytes) return fail(CHEB_E_INVAL, "arena_bytes is NULL");
  if (!valid_layout(layout_kind)) return fail(CHEB_E_INVAL, "unknown layout %d", layout_kind);
  std::vector<int64_t> off;
  int64_t sn = 0;
  size_t st = 0, ab = 0;
  int rc = layout(n_slots, dtype, seg_numel, n_segs, &off, &sn, &st, &ab);
  if (rc != CHEB_OK) return rc;
  *arena_bytes = layout_kind == CHEB_LAYOUT_SLOTS ? ab : interleaved_bytes(n_slots, sn, dtype);
  return ok();
}

int cheb_cache_create_ex(cheb_cache **out, int32_t n_slots, int32_t dtype,
                         const int64_t *seg_numel, int32_t n_segs, int32_t layout_kind,
                         void *arena, size_t arena_bytes) {
  if (!out) return fail(CHEB_E_INVAL, "out is NULL");
  *out = nullptr;
  if (!valid_layout(layout_kind)) return fail(CHEB_E_INVAL, "unknown layout %d", layout_kind);
  std::vector<int64_t> off;
  int64_t sn = 0;
  size_t st = 0, need = 0;
  int rc = layout(n_slots, dtype, seg_numel, n_segs, &off, &sn, &st, &need);
  if (rc != CHEB_OK) return rc;
  if (layout_kind == CHEB_LAYOUT_INTERLEAVED) need = interleaved_bytes(n_slots, sn, dtype);
  if (!arena) return fail(CHEB_E_INVAL, "arena is NULL");
  if (!aligned(arena, kSlotAlign)) return fail(CHEB_E_ALIGN, "arena is not 256-byte aligned");
  if (arena_bytes < need)
    return fail(CHEB_E_MISMATCH, "arena holds %zu bytes, the layout needs %zu", arena_bytes, need);
  cheb_cache *c = new (std::nothrow) cheb_cache();
  if (!c) return fail(CHEB_E_INVAL, "out of host memory");
  c->n_slots = n_slots;
  c->dtype = dtype;
  c->seg_numel.assign(seg_numel, seg_numel + n_segs);
  c->seg_offset = std::move(off);
  c->slot_numel = sn;
  c->slot_stride = st;
  c->arena = static_cast<char *>(arena);
  c->arena_bytes = arena_bytes;
  c->layout = layout_kind;
  if (layout_kind == CHEB_LAYOUT_INTERLEAVED) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(arena);
    c->region = reinterpret_cast<char *>((a + kLaneAlign - 1) / kLaneAlign * kLaneAlign);
    c->super_vecs = int64_t(n_slots) * kChunkVecs;
  }
  *out = c;
  return ok();
}

int cheb_cache_create(cheb_cache **out, int32_t n_slots, int32_t dtype, const int64_t *seg_numel,
                      int32_t n_segs, void *arena, size_t arena_bytes) {
  return cheb_cache_create_ex(out, n_slots, dtype, seg_numel, n_segs, CHEB_LAYOUT_SLOTS, arena,
                              arena_bytes);
}

int cheb_cache_geometry(const cheb_cache *c, int32_t *layout_kind, int64_t *chunk_elems,
                        int64_t *entry_stride_elems) {
  if (!c) return fail(CHEB_E_INVAL, "cache is NULL");
  const int64_t vec = elems_per_vec(c->dtype);
  if (layout_kind) *layout_kind = c->layout;
  if (chunk_elems) *chunk_elems = kChunkVecs * vec;
  if (entry_stride_elems) *entry_stride_elems = c->super_vecs * vec;
  return ok();
}

int cheb_cache_destroy(cheb_cache *c) {
  delete c;
  return ok();
}

int cheb_cache_reset(cheb_cache *c) {
  if (!c) return fail(CHEB_E_INVAL, "cache is NULL");
  c->head = 0;
  c->count = 0;
  c->push_open = false;
  return ok();
}

int cheb_cache_push(cheb_cache *c, double t, const void *const *seg_src, void *stream) {
  if (!c) return fail(CHEB_E_INVAL, "cache is NULL");
  if (c->push_open) return fail(CHEB_E_NOTREADY, "a fused push is open");
  if (!seg_src) return fail(CHEB_E_INVAL, "seg_src is NULL");
  int rc = check_new_abscissa(c, t);
  if (rc != CHEB_OK) return rc;
  const size_t n_segs = c->seg_numel.size();
  std::vector<GatherSeg> segs(n_segs);
  for (size_t s = 0; s < n_segs; ++s) {
    if (c->seg_numel[s] > 0) {
      if (!seg_src[s]) return fail(CHEB_E_INVAL, "seg_src[%zu] is NULL", s);
      if (!aligned(seg_src[s], 16))
        return fail(CHEB_E_ALIGN, "seg_src[%zu] is not 16-byte aligned", s);
    }
    segs[s] = GatherSeg{seg_src[s], c->seg_offset[s], c->seg_numel[s]};
  }
  // The entry goes to slot `head`: the next free slot, or the oldest entry's
  // slot when the ring is full.  That entry leaves the history before the
  // first launch, so a launch that fails after an earlier one has written
  // part of the slot cannot leave a half-overwritten entry in the history.
  const int32_t slot = claim_slot(c);
  rc = launch_gather(c->dtype, c->slot_ptr(slot), segs.data(), int(n_segs), c->super_vecs,
                     static_cast<hipStream_t>(stream));
  if (rc != CHEB_OK) return rc;
  record(c, t);
  return ok();
}

int cheb_cache_begin_push(cheb_cache *c, void **slot_base) {
  if (!c || !slot_base) return fail(CHEB_E_INVAL, "cache or slot_base is NULL");
  if (c->layout != CHEB_LAYOUT_SLOTS)
    return fail(CHEB_E_INVAL, "a fused push needs contiguous slots (CHEB_LAYOUT_SLOTS)");
  if (c->push_open) return fail(CHEB_E_NOTREADY, "a fused push is already open");
  const int32_t slot = claim_slot(c);
  c->push_open = true;
  *slot_base = c->slot_ptr(slot);
  return ok();
}

int cheb_cache_commit(cheb_cache *c, double t) {
  if (!c) return fail(CHEB_E_INVAL, "cache is NULL");
  if (!c->push_open) return fail(CHEB_E_NOTREADY, "no fused push is open");
  if (!isfinite(t)) return fail(CHEB_E_NONFINITE, "abscissa is not finite");
  for (int32_t a = 0; a < c->count; ++a)
    if (c->slot_t[c->slot_of_age(a)] == t)
      return fail(CHEB_E_DUPNODE, "abscissa %.17g is already held", t);
  record(c, t);
  c->push_open = false;
  return ok();
}

int cheb_cache_abort_push(cheb_cache *c) {
  if (!c) return fail(CHEB_E_INVAL, "cache is NULL");
  if (!c->push_open) return fail(CHEB_E_NOTREADY, "no fused push is open");
  c->push_open = false;  // claim_slot already dropped the slot's old entry
  return ok();
}

int cheb_cache_history(const cheb_cache *c, double *t_out, int32_t *count) {
  if (!c || !count) return fail(CHEB_E_INVAL, "cache or count is NULL");
  *count = c->count;
  if (t_out)
    for (int32_t a = 0; a < c->count; ++a) t_out[a] = c->slot_t[c->slot_of_age(a)];
  return ok();
}

int cheb_cache_entry(const cheb_cache *c, int32_t idx, void **slot_base) {
  if (!c || !slot_base) return fail(CHEB_E_INVAL, "cache or slot_base is NULL");
  if (idx < 0 || idx >= c->count)
    return fail(CHEB_E_INVAL, "entry %d outside 0..%d", idx, c->count - 1);
  *slot_base = c->slot_ptr(c->slot_of_age(idx));
  return ok();
}

int cheb_cache_segment_offset(const cheb_cache *c, int32_t seg, int64_t *elem_offset) {
  if (!c || !elem_offset) return fail(CHEB_E_INVAL, "cache or elem_offset is NULL");
  if (seg < 0 || size_t(seg) >= c->seg_offset.size())
    return fail(CHEB_E_INVAL, "segment %d out of range", seg);
  *elem_offset = c->seg_offset[size_t(seg)];
  return ok();
}

int cheb_cache_dtype(const cheb_cache *c, int32_t *dtype) {
  if (!c || !dtype) return fail(CHEB_E_INVAL, "cache or dtype is NULL");
  *dtype = c->dtype;
  return ok();
}

int cheb_cache_slot_numel(const cheb_cache *c, int64_t *numel) {
  if (!c || !numel) return fail(CHEB_E_INVAL, "cache or numel is NULL");
  *numel = c->slot_numel;
  return ok();
}

int cheb_extrapolate_multi(cheb_cache *c, const double *w, int32_t n_out, void *const *out,
                           void *stream) {
  if (!c) return fail(CHEB_E_INVAL, "cache is NULL");
  if (!c->push_open && c->count < c->n_slots)
    return fail(CHEB_E_NOTREADY, "history holds %d of %d entries", c->count, c->n_slots);
  return cheb::extrapolate_newest(c, c->n_slots, w, n_out, out, stream);
}

int cheb_extrapolate(cheb_cache *c, const double *w, void *out, void *stream) {
  void *outs[1] = {out};
  if (!out && c && c->slot_numel > 0) return fail(CHEB_E_INVAL, "out is NULL");
  return cheb_extrapolate_multi(c, w, 1, outs, stream);
}

int cheb_extrapolate_at_multi(cheb_cache *c, const double *target_t, int32_t n_out,
                              void *const *out, void *stream, double *w_used) {
  if (!c || !target_t) return fail(CHEB_E_INVAL, "cache or target_t is NULL");
  if (c->push_open) return fail(CHEB_E_NOTREADY, "a fused push is open");
  if (c->count < c->n_slots)
    return fail(CHEB_E_NOTREADY, "history holds %d of %d entries", c->count, c->n_slots);
  if (n_out < 1 || n_out > CHEB_MAX_OUTPUTS)
    return fail(CHEB_E_INVAL, "n_out %d outside 1..%d", n_out, CHEB_MAX_OUTPUTS);
  double t[CHEB_MAX_SLOTS], w[CHEB_MAX_OUTPUTS * CHEB_MAX_SLOTS];
  for (int32_t a = 0; a < c->n_slots; ++a) t[a] = c->slot_t[c->slot_of_age(a)];
  for (int32_t m = 0; m < n_out; ++m) {
    int rc = weights_row(t, c->n_slots, target_t[m], w + m * c->n_slots);
    if (rc != CHEB_OK) return rc;
  }
  int rc = cheb_extrapolate_multi(c, w, n_out, out, stream);
  if (rc == CHEB_OK && w_used)
    memcpy(w_used, w, sizeof(double) * size_t(n_out) * size_t(c->n_slots));
  return rc;
}

int cheb_extrapolate_at(cheb_cache *c, double target_t, void *out, void *stream,
                        double *w_used) {
  void *outs[1] = {out};
  if (!out && c && c->slot_numel > 0) return fail(CHEB_E_INVAL, "out is NULL");
  return cheb_extrapolate_at_multi(c, &target_t, 1, outs, stream, w_used);
}

}  // extern "C"
