/*
 * cheb.h: C ABI of libcheb, the ChebBooster online stage on AMD MI355X
 * (gfx950).
 *
 * ChebBooster skips a diffusion-transformer forward pass at some steps.  On
 * such a step it predicts every cached module output as a fixed linear
 * combination of the last n = K+1 fully computed ones:
 *
 *     f_t = sum_j w_t^j f_{s_j}   (paper, Section 3.3, forward application;
 *                                   Algorithm 1, online stage)
 *
 * The weights w_t^j are Lagrange interpolation coefficients in barycentric
 * form (Section 3.2, coefficient equation; Appendix A, general weights and
 * second form).  They depend only on the history abscissae and the target,
 * so they are computed once on the host in fp64 (Section 3.3, weight
 * precomputation).  The per-step work is a streaming weighted sum over every
 * cached tensor, run here as one HIP launch.
 *
 * Conventions for every call
 *   - Return value: CHEB_OK (0) or a negative cheb_status.  On failure,
 *     cheb_last_error() returns a message for the calling thread.  Every
 *     argument is checked on the host before anything is enqueued, so a
 *     call refused for its arguments has enqueued no GPU work.  A call that
 *     launches more than once can fail with CHEB_E_HIP after an earlier
 *     launch went in; cheb_cache_push documents what it leaves behind.
 *   - Device memory (history arena, sources, outputs) belongs to the caller.
 *     The library never allocates or frees device memory.  It owns only the
 *     host-side handle returned by cheb_cache_create.
 *   - `stream` is a hipStream_t passed as void*.  NULL means the default
 *     stream.  GPU work is asynchronous on that stream.  Calls enqueue work in
 *     program order; the caller orders work across streams.
 *   - History order is always oldest to newest.
 *   - Storage types: CHEB_BF16 (bfloat16) and CHEB_F16 (binary16) storage
 *     with fp32 weights and accumulation and round-to-nearest-even output;
 *     CHEB_F32 (binary32) storage with fp64 weights and accumulation and
 *     round-to-nearest-even output.
 *   - Distinct cache handles may be used from different threads at once.  One
 *     handle must not be used by two threads at the same time.
 */
#ifndef CHEB_H
#define CHEB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CHEB_VERSION 4

#if defined(__GNUC__) || defined(__clang__)
#define CHEB_API __attribute__((visibility("default")))
#else
#define CHEB_API
#endif

/* Largest history (K+1) the device kernels take. */
#define CHEB_MAX_SLOTS 8
/* Largest number of outputs (targets) one multi-target call produces. */
#define CHEB_MAX_OUTPUTS 8
/* Largest node count cheb_precompute_weights takes. */
#define CHEB_MAX_NODES 64

typedef enum cheb_status {
  CHEB_OK = 0,
  CHEB_E_INVAL = -1,     /* null pointer, count or enum out of range */
  CHEB_E_DUPNODE = -2,   /* two equal history abscissae (also once mapped onto [-1, 1]) */
  CHEB_E_NOTREADY = -3,  /* history holds fewer than n entries, or a push is open */
  CHEB_E_DTYPE = -4,     /* unknown storage type */
  CHEB_E_ALIGN = -5,     /* device pointer not aligned as documented */
  CHEB_E_HIP = -6,       /* the HIP runtime reported an error */
  CHEB_E_MISMATCH = -7,  /* sizes disagree (arena too small, ...) */
  CHEB_E_NONFINITE = -8, /* NaN or infinite abscissa or weight, or a weight row
                            past fp64's resolution (see cheb_precompute_weights) */
  CHEB_E_IO = -9         /* table file cannot be read or written, or is malformed */
} cheb_status;

/* Storage types of history entries and outputs.  bf16 and fp16 are
 * accumulated in fp32 with fp32 weights and rounded to nearest-even once;
 * fp32 is accumulated in fp64 with fp64 weights. */
typedef enum cheb_dtype { CHEB_BF16 = 0, CHEB_F32 = 1, CHEB_F16 = 2 } cheb_dtype;

/* Message for the last failed call on this thread ("" if none).  The
 * pointer stays valid until the next failing call on the same thread. */
CHEB_API const char *cheb_last_error(void);

/* CHEB_VERSION of the built library. */
CHEB_API int cheb_version(void);

/* ------------------------------------------------------------------------ */
/* Weight precomputation (host, fp64).                                       */
/* ------------------------------------------------------------------------ */

/* Interpolation coefficients of the degree-(n_hist-1) polynomial through the
 * history abscissae, evaluated at each target (Section 3.2, coefficient
 * equation; Appendix A, rho_j = 1/omega'(x_j) and second barycentric form;
 * Section 3.3, nodes and target mapped affinely onto [-1, 1]).
 *
 *   hist_t   [n_hist] host fp64: history abscissae (timesteps or sigma),
 *            oldest to newest, finite and pairwise distinct.
 *   target_t [n_target] host fp64: finite targets.  A target equal to a
 *            history abscissa gets the unit row of that entry.
 *   w_out    [n_target][n_hist] host fp64, row-major, caller-owned.  Row m
 *            sums to 1 up to rounding.
 *
 * The products of the second form are carried with a separate power-of-two
 * exponent, so closely clustered abscissae do not underflow them.  A row is
 * refused (CHEB_E_NONFINITE) when a weight is not finite or when
 * n_hist * 2^-53 * sum_j |w_j|, the second form's bound on each weight's
 * relative rounding error, exceeds 2^-24: fp64 then no longer gives the
 * coefficients to the fp32 precision the bf16 kernel uses them at.  Distinct
 * abscissae that the map onto [-1, 1] rounds together are CHEB_E_DUPNODE.
 *
 * 1 <= n_hist <= CHEB_MAX_NODES, n_target >= 0.  Errors: CHEB_E_INVAL,
 * CHEB_E_NONFINITE, CHEB_E_DUPNODE.  w_out is not written on error. */
CHEB_API int cheb_precompute_weights(const double *hist_t, int32_t n_hist,
                            const double *target_t, int32_t n_target,
                            double *w_out);

/* Weight variants for cheb_precompute_weights_variant. */
enum {
  CHEB_RHO_GENERAL = 0,     /* rho_j = 1/omega'(x_j) (Appendix A): the
                               Lagrange interpolant, as cheb_precompute_weights */
  CHEB_RHO_ALTERNATING = 1, /* rho_j = (-1)^j (1/2 at both ends, else 1), the
                               weights printed in Section 3.2: exact for
                               Chebyshev extrema, a rational interpolant that
                               reproduces degree <= 1 at equispaced nodes */
  CHEB_TAYLOR = 2           /* not a barycentric form: the Taylor expansion
                               about the newest abscissa, the i-th derivative
                               over i! estimated by the divided difference over
                               the newest i+1 abscissae (the Taylor comparison
                               of Section 3.2's Runge study); reproduces
                               degree <= 1, and the unit row at the newest
                               abscissa only */
};

/* cheb_precompute_weights with a choice of coefficient generator: the
 * barycentric weights rho_j of the coefficient equation of Section 3.2, or
 * the Taylor expansion above.  Arguments and errors as
 * cheb_precompute_weights, plus CHEB_E_INVAL for an unknown variant. */
CHEB_API int cheb_precompute_weights_variant(const double *hist_t, int32_t n_hist,
                                             const double *target_t, int32_t n_target,
                                             int32_t variant, double *w_out);

/* Chebyshev points on [a, b], largest first, for schedules that place full
 * steps at them: kind 1 the roots cos((2j-1) pi / 2n), j = 1..n (Section
 * 3.2, node equation); kind 2 the extrema cos((j-1) pi / (n-1)) (n >= 2).
 *   x_out [n] host fp64.  1 <= n <= CHEB_MAX_NODES.
 * Errors: CHEB_E_INVAL, CHEB_E_NONFINITE. */
CHEB_API int cheb_chebyshev_nodes(int32_t n, int32_t kind, double a, double b, double *x_out);

/* ------------------------------------------------------------------------ */
/* Stateless combination.                                                    */
/* ------------------------------------------------------------------------ */

/* out[i] = sum_{k=0}^{n_src-1} w[k] * src[k][i] for 0 <= i < numel
 * (Section 3.3, forward application), in one launch.
 *
 *   src     [n_src] host array of device pointers, each to numel elements of
 *           `dtype`, 16-byte aligned.
 *   w       [n_src] host fp64 weights, finite (converted to fp32 on the bf16
 *           path, where a magnitude above FLT_MAX is CHEB_E_NONFINITE).
 *   out     device pointer to numel elements of `dtype`, 16-byte aligned.
 *           It may not overlap any source.
 *   numel   >= 0, below 2^34.  Any value; a ragged tail is handled.
 *
 * 1 <= n_src <= CHEB_MAX_SLOTS.  Errors: CHEB_E_INVAL, CHEB_E_DTYPE,
 * CHEB_E_ALIGN, CHEB_E_NONFINITE, CHEB_E_HIP. */
CHEB_API int cheb_combine(const void *const *src, int32_t n_src, const double *w,
                 void *out, int64_t numel, int32_t dtype, void *stream);

/* Several targets from one pass over the sources:
 *     out[m][i] = sum_k w[m * n_src + k] * src[k][i],  m < n_out.
 * Every prediction between two full steps depends only on the same history
 * (Section 3.3, forward application; Algorithm 1, the history changes only
 * at full steps), so all of them can be formed while the history is read
 * once: (n_src + n_out) x numel elements of traffic instead of
 * n_out x (n_src + 1) x numel.
 *   w    [n_out][n_src] host fp64, row-major.
 *   out  [n_out] host array of device pointers, each 16-byte aligned, to
 *        numel elements; outputs overlap neither each other nor a source.
 * 1 <= n_out <= CHEB_MAX_OUTPUTS; other arguments as cheb_combine.
 * Errors: as cheb_combine. */
CHEB_API int cheb_combine_multi(const void *const *src, int32_t n_src, const double *w,
                                int32_t n_out, void *const *out, int64_t numel,
                                int32_t dtype, void *stream);

/* ------------------------------------------------------------------------ */
/* History cache: a ring of n entries in one caller-owned device arena.      */
/* ------------------------------------------------------------------------ */

/* The fixed-size history buffer H of (abscissa, features) pairs holding the
 * n most recent full steps; a push into a full buffer evicts the oldest
 * (Section 3.3, forward application; Algorithm 1, online stage).
 *
 * Layout.  One entry ("slot") holds every cached tensor ("segment") of one
 * full step, back to back.  Segment s starts at element seg_offset[s], with
 * offsets rounded up to 16 bytes (8 bf16 or 4 fp32 elements).  Elements
 * between segments are padding.  slot_numel is the end of the last segment,
 * rounded up the same way.  Slots are slot_stride_bytes apart (a multiple of
 * 256) from the start of the arena.  Outputs of cheb_extrapolate use the same
 * flat layout: segment s of the prediction is at out + seg_offset[s]. */
typedef struct cheb_cache cheb_cache;

/* Device bytes the history buffer H of n_slots entries needs (Section 3.3,
 * forward application: a fixed-size buffer of the n most recent full
 * steps; Algorithm 1: each full step stores (s, f_s) in H), so that the
 * caller can allocate the arena before cheb_cache_create.
 *   seg_numel         [n_segs] host, element counts of the cached tensors of
 *                     one full step (each >= 0).
 *   arena_bytes       out: bytes of the whole arena (n_slots slots).
 *   slot_stride_bytes out: bytes from one slot to the next (a multiple of
 *                     256); may be NULL.
 * 1 <= n_slots <= CHEB_MAX_SLOTS, n_segs >= 1.  Errors: CHEB_E_INVAL,
 * CHEB_E_DTYPE.  Nothing is written on error. */
CHEB_API int cheb_cache_arena_bytes(int32_t n_slots, int32_t dtype, const int64_t *seg_numel,
                                    int32_t n_segs, size_t *arena_bytes,
                                    size_t *slot_stride_bytes);

/* The whole layout of that buffer (Section 3.3; Algorithm 1, as
 * cheb_cache_arena_bytes), also giving where each cached tensor lives in a
 * slot and in an output.
 *   seg_numel  [n_segs] element counts (each >= 0).
 *   seg_offset [n_segs] out, may be NULL.
 *   slot_numel, slot_stride_bytes, arena_bytes: out, each may be NULL.
 * 1 <= n_slots <= CHEB_MAX_SLOTS, n_segs >= 1.  Errors: CHEB_E_INVAL,
 * CHEB_E_DTYPE. */
CHEB_API int cheb_cache_layout(int32_t n_slots, int32_t dtype, const int64_t *seg_numel,
                      int32_t n_segs, int64_t *seg_offset, int64_t *slot_numel,
                      size_t *slot_stride_bytes, size_t *arena_bytes);

/* How the entries of H are laid out in the arena.
 *   CHEB_LAYOUT_SLOTS        each entry contiguous ("slot"), slots
 *                            slot_stride_bytes apart: the layout of
 *                            cheb_cache_create, the only one a fused push
 *                            (cheb_cache_begin_push) can write into.
 *   CHEB_LAYOUT_INTERLEAVED  the arena is cut into 32 KiB chunks taken by the
 *                            entries in turn: chunk c of the entry in lane j
 *                            sits (c * n_slots + j) chunks past the first
 *                            64 KiB boundary of the arena.  One prediction
 *                            then reads a single region of the arena instead
 *                            of n separate ones, which streams faster on
 *                            MI355X; entries are filled by cheb_cache_push.
 * Outputs of the predictions are contiguous in both layouts. */
enum { CHEB_LAYOUT_SLOTS = 0, CHEB_LAYOUT_INTERLEAVED = 1 };

/* cheb_cache_arena_bytes for either layout (Section 3.3; Algorithm 1, as
 * cheb_cache_arena_bytes): arena bytes for n_slots entries laid out as
 * `layout` (the interleaved layout includes room to start on a 64 KiB
 * boundary).  Errors: CHEB_E_INVAL, CHEB_E_DTYPE. */
CHEB_API int cheb_cache_arena_bytes_ex(int32_t n_slots, int32_t dtype, const int64_t *seg_numel,
                                       int32_t n_segs, int32_t layout, size_t *arena_bytes);

/* Creates the history buffer H of Section 3.3 (n = n_slots entries, empty
 * at the start of sampling; Algorithm 1, online stage) over `arena`
 * (device, 256-byte aligned, at least the bytes cheb_cache_arena_bytes
 * gives).  The arena stays caller-owned and must outlive the handle.
 * Errors: CHEB_E_INVAL, CHEB_E_DTYPE, CHEB_E_ALIGN, CHEB_E_MISMATCH. */
CHEB_API int cheb_cache_create(cheb_cache **out, int32_t n_slots, int32_t dtype,
                      const int64_t *seg_numel, int32_t n_segs, void *arena,
                      size_t arena_bytes);

/* cheb_cache_create with a choice of layout (CHEB_LAYOUT_SLOTS, as
 * cheb_cache_create, or CHEB_LAYOUT_INTERLEAVED); arena_bytes at least
 * cheb_cache_arena_bytes_ex for that layout.  Errors: as
 * cheb_cache_create. */
CHEB_API int cheb_cache_create_ex(cheb_cache **out, int32_t n_slots, int32_t dtype,
                                  const int64_t *seg_numel, int32_t n_segs, int32_t layout,
                                  void *arena, size_t arena_bytes);

/* Where the elements of an entry lie: element e of the entry whose base
 * cheb_cache_entry gives is at
 *     base + (e / chunk_elems) * entry_stride_elems + e % chunk_elems
 * elements.  For CHEB_LAYOUT_SLOTS entry_stride_elems == chunk_elems, so
 * the entry is contiguous.  Every output may be NULL.  Errors:
 * CHEB_E_INVAL. */
CHEB_API int cheb_cache_geometry(const cheb_cache *c, int32_t *layout, int64_t *chunk_elems,
                                 int64_t *entry_stride_elems);

/* Ends the history buffer H of Section 3.3 (Algorithm 1, end of the
 * sampling loop): frees the handle, not the arena.  NULL is accepted. */
CHEB_API int cheb_cache_destroy(cheb_cache *c);

/* Empties H for a new sampling run (Algorithm 1 starts the online stage
 * with an empty history): metadata only; arena contents are left as they
 * are. */
CHEB_API int cheb_cache_reset(cheb_cache *c);

/* Stores the full step at abscissa t: copies segment s from seg_src[s]
 * (device, 16-byte aligned, seg_numel[s] elements) into the slot of the
 * oldest entry (or the next free one), zero-fills the padding after each
 * segment, records t and advances the ring (Algorithm 1, full computation:
 * store (s, f_s) in H; Section 3.3, the oldest entry is evicted).  One
 * launch per 64 segments, asynchronous on `stream`.
 * A launch failure (CHEB_E_HIP) after the arguments were accepted leaves
 * the history without the entry whose slot the copy was writing: a full
 * ring has dropped its oldest entry (the launches before the failing one
 * may have overwritten part of its slot), a ring with a free slot is as
 * before, and t is not recorded.  Every other held entry is untouched, so
 * a later prediction never reads a half-written slot.
 * Errors: CHEB_E_INVAL, CHEB_E_NONFINITE, CHEB_E_DUPNODE (t already held),
 * CHEB_E_ALIGN, CHEB_E_NOTREADY (a fused push is open), CHEB_E_HIP. */
CHEB_API int cheb_cache_push(cheb_cache *c, double t, const void *const *seg_src,
                    void *stream);

/* Fused push, part 1 (Algorithm 1, full computation: store (s, f_s) in H;
 * Section 3.3, the oldest entry is evicted): returns in *slot_base the
 * device address of the slot the next entry will occupy, so the full step
 * can write its outputs there directly (segment s at slot_base +
 * seg_offset[s] elements).  The entry that slot held is dropped from the
 * history at once.  The library writes nothing into the slot: the padding
 * after each segment keeps whatever the slot held, so the padding elements
 * of later predictions are unspecified (they may be NaN); every segment's
 * own elements are exact.  Until cheb_cache_commit, pushes and
 * extrapolations fail with CHEB_E_NOTREADY.  Only for CHEB_LAYOUT_SLOTS.
 * Errors: CHEB_E_INVAL (also for an interleaved cache), CHEB_E_NOTREADY
 * (already open). */
CHEB_API int cheb_cache_begin_push(cheb_cache *c, void **slot_base);

/* Fused push, part 2 (Algorithm 1, full computation: store (s, f_s) in H):
 * records abscissa t for the open slot (metadata only; no GPU work).  The caller orders the writes into the slot before any later
 * use of the cache on its streams.  Errors: CHEB_E_INVAL, CHEB_E_NONFINITE,
 * CHEB_E_DUPNODE, CHEB_E_NOTREADY (no push open). */
CHEB_API int cheb_cache_commit(cheb_cache *c, double t);

/* Fused push, abandoned (Algorithm 1 stores only completed full steps in
 * H): closes the open push without recording an entry
 * (for a full step that failed before its outputs were complete).  The
 * entry that slot held stays dropped, so a full ring holds one entry fewer
 * afterwards; the others are untouched.  Errors: CHEB_E_INVAL,
 * CHEB_E_NOTREADY (no push open). */
CHEB_API int cheb_cache_abort_push(cheb_cache *c);

/* The abscissae s_j held in H (Section 3.3; Algorithm 1), oldest to newest,
 * the order the weight rows of cheb_precompute_weights and
 * cheb_extrapolate use: t_out[0 .. *count-1] (t_out has room for n_slots
 * values; it may be NULL).  Errors: CHEB_E_INVAL. */
CHEB_API int cheb_cache_history(const cheb_cache *c, double *t_out, int32_t *count);

/* Device address of the features f_{s_j} of held entry j (Section 3.3;
 * Algorithm 1), j = `idx` counted from the oldest (0): the entry's first
 * element; the others follow cheb_cache_geometry.  Errors: CHEB_E_INVAL
 * (idx outside 0 .. count-1). */
CHEB_API int cheb_cache_entry(const cheb_cache *c, int32_t idx, void **slot_base);

/* Element offset of cached tensor `seg` (one module output of the block
 * equation of Section 3.1) in a slot of H and in a prediction output
 * (Section 3.3, forward application: the prediction has the layout of the
 * features it combines).  Errors: CHEB_E_INVAL. */
CHEB_API int cheb_cache_segment_offset(const cheb_cache *c, int32_t seg,
                              int64_t *elem_offset);

/* Storage type (cheb_dtype) of the entries of H and of its predictions
 * (Section 3.3).  Errors: CHEB_E_INVAL. */
CHEB_API int cheb_cache_dtype(const cheb_cache *c, int32_t *dtype);

/* Elements of one entry of H, which is also the element count of one
 * prediction output (Section 3.3, forward application).  Errors:
 * CHEB_E_INVAL. */
CHEB_API int cheb_cache_slot_numel(const cheb_cache *c, int64_t *numel);

/* The skipped-step prediction (Section 3.3, forward application equation;
 * Algorithm 1, extrapolation branch):
 *     out[i] = sum_{k=0}^{n-1} w[k] * H_k[i],  H_0 oldest .. H_{n-1} newest,
 * over every element of every segment, in one launch.
 *   w    [n_slots] host fp64, aligned with cheb_cache_history's order (for
 *        example a row of cheb_precompute_weights over those abscissae).
 *   out  device, 16-byte aligned, cheb_cache_slot_numel elements, not
 *        overlapping the arena.  Padding elements of out are unspecified.
 * Requires a full history (|H| = n; Section 3.3).  Errors: CHEB_E_INVAL,
 * CHEB_E_NOTREADY, CHEB_E_ALIGN, CHEB_E_NONFINITE, CHEB_E_HIP. */
CHEB_API int cheb_extrapolate(cheb_cache *c, const double *w, void *out, void *stream);

/* The predictions for n_out targets from one pass over the history (see
 * cheb_combine_multi): out[m] = sum_k w[m * n_slots + k] * H_k.
 *   w    [n_out][n_slots] host fp64, rows aligned with cheb_cache_history.
 *   out  [n_out] host array of device pointers, as cheb_extrapolate's out.
 * Errors: as cheb_extrapolate, and CHEB_E_INVAL for n_out outside
 * 1..CHEB_MAX_OUTPUTS. */
CHEB_API int cheb_extrapolate_multi(cheb_cache *c, const double *w, int32_t n_out,
                                    void *const *out, void *stream);

/* Readiness check, weight row and prediction in one call: computes the fp64
 * coefficients of the held abscissae at `target_t` (as
 * cheb_precompute_weights) and runs cheb_extrapolate with them.  The weights
 * used can be read back through w_used ([n_slots] host fp64, may be NULL).
 * Errors: those of cheb_precompute_weights and cheb_extrapolate. */
CHEB_API int cheb_extrapolate_at(cheb_cache *c, double target_t, void *out,
                        void *stream, double *w_used);

/* cheb_extrapolate_at for n_out targets in one pass over the history.
 *   target_t  [n_out] host fp64.
 *   out       [n_out] host array of device pointers.
 *   w_used    [n_out][n_slots] host fp64 out, may be NULL.
 * Errors: as cheb_extrapolate_at and cheb_extrapolate_multi. */
CHEB_API int cheb_extrapolate_at_multi(cheb_cache *c, const double *target_t, int32_t n_out,
                                       void *const *out, void *stream, double *w_used);

/* ------------------------------------------------------------------------ */
/* Offline stage: schedule and weight table.                                 */
/* ------------------------------------------------------------------------ */

/* The full-computation schedule F of Section 3.3 (weight precomputation):
 * step s of 0..T-1 runs the full network when s < s0, or s > T-1-s1, or r
 * divides s - s0.  is_full [T] host out: 1 for s in F, else 0.
 * 1 <= T <= 2^20, s0 >= 0, s1 >= 0, r >= 1.  Errors: CHEB_E_INVAL. */
CHEB_API int cheb_schedule(int32_t T, int32_t s0, int32_t s1, int32_t r, uint8_t *is_full);

/* What a skipped step does when fewer than n_hist full steps precede it
 * (the paper requires |H| = n and leaves this case open). */
enum { CHEB_SHORT_FULL = 0,   /* run the full network instead (it joins H) */
       CHEB_SHORT_LOWER = 1 }; /* predict from the entries held (lower degree) */

/* The weight table of the offline stage (Algorithm 1, offline stage;
 * Section 3.3): for every step outside F (and the policy's extra full
 * steps), the steps of the history it predicts from (the n_hist most recent
 * steps that ran the network, or fewer under CHEB_SHORT_LOWER) and its fp64
 * coefficients over their abscissae at the step's own abscissa
 * (cheb_precompute_weights).  Host-only object, library-owned. */
typedef struct cheb_table cheb_table;

/* Builds the table.  abscissa [T] host fp64: the value each step is
 * interpolated in (timestep t or sigma), finite; steps that share a
 * history must have distinct abscissae.  1 <= n_hist <= CHEB_MAX_SLOTS.
 * Errors: CHEB_E_INVAL, CHEB_E_NONFINITE, CHEB_E_DUPNODE. */
CHEB_API int cheb_table_build(cheb_table **out, int32_t T, int32_t s0, int32_t s1, int32_t r,
                              int32_t n_hist, const double *abscissa, int32_t policy);

/* The same for an arbitrary set of full steps (for example steps placed at
 * rounded Chebyshev points, cheb_chebyshev_nodes, instead of on the grid
 * F): is_full [T] host, nonzero where the step runs the network.  The
 * table records r = 0 (no grid).  Errors: as cheb_table_build. */
CHEB_API int cheb_table_build_mask(cheb_table **out, int32_t T, const uint8_t *is_full,
                                   int32_t n_hist, const double *abscissa, int32_t policy);

/* Frees the table.  NULL is accepted. */
CHEB_API int cheb_table_destroy(cheb_table *t);

/* Sizes of a table; every output may be NULL.  n_full counts the steps that
 * run the network (the schedule's plus the policy's). */
CHEB_API int cheb_table_info(const cheb_table *t, int32_t *T, int32_t *n_hist,
                             int32_t *policy, int32_t *n_full);

/* Row of one step: *predicted (1 predicted, 0 full), *n_used (entries the
 * prediction uses), node_steps [n_hist] (their steps, oldest to newest) and
 * w [n_hist] (their coefficients); node_steps and w may be NULL.
 * Errors: CHEB_E_INVAL. */
CHEB_API int cheb_table_step(const cheb_table *t, int32_t step, int32_t *predicted,
                             int32_t *n_used, int32_t *node_steps, double *w);

/* Writes the table as text (hexadecimal floats, so it reads back bit for
 * bit) to `path`: the "prepackaged" tables of Section 3.3.  Errors:
 * CHEB_E_INVAL, CHEB_E_IO. */
CHEB_API int cheb_table_save(const cheb_table *t, const char *path);

/* Reads a table written by cheb_table_save.  Rows are taken as stored,
 * after structural checks (step order, node steps before the step and
 * increasing, finite values).  Errors: CHEB_E_INVAL, CHEB_E_IO. */
CHEB_API int cheb_table_load(cheb_table **out, const char *path);

/* The online stage driven by a table (Algorithm 1, extrapolation branch;
 * Section 3.3, forward application): predicts steps first_step ..
 * first_step + n_steps - 1, which must all be predicted steps sharing one
 * history, from one pass over that history.  The newest n_used entries of
 * the cache must hold exactly the abscissae of the row's nodes (the row
 * matches the ring), else CHEB_E_MISMATCH.  out [n_steps] device pointers as
 * in cheb_extrapolate_multi.  Errors: CHEB_E_INVAL, CHEB_E_MISMATCH,
 * CHEB_E_NOTREADY, and those of cheb_extrapolate_multi. */
CHEB_API int cheb_extrapolate_steps(cheb_cache *c, const cheb_table *t, int32_t first_step,
                                    int32_t n_steps, void *const *out, void *stream);

/* ------------------------------------------------------------------------ */
/* Residual application on a skipped step.                                   */
/* ------------------------------------------------------------------------ */

/* A DiT block adds its module outputs to the residual stream,
 * x_{l+1} = x_l + S^l + C^l + M^l (Section 3.1, block equation).  On a skipped
 * step every module output is the prediction sum_k w_k H_k[segment]
 * (Section 3.3; Algorithm 1), so the whole block stack adds
 *     x_out[j] = x_in[j] + sum over segments s with res_offset[s] >= 0 and
 *                j in [res_offset[s], res_offset[s] + seg_numel[s]) of
 *                sum_k w_k H_k[seg_offset[s] + j - res_offset[s]].
 * This call forms it in one pass over the history: the per-module
 * predictions are never written.  fp64 accumulation, fp32 residual.
 *   w          [n_slots] host fp64, aligned with cheb_cache_history.
 *   res_offset [n_segs] host: element of the residual where segment s adds;
 *              negative: segment s is not added.  Offsets and segment sizes
 *              of added segments are multiples of 16 bytes' worth of the
 *              storage type (8 bf16 / 4 fp32 elements).
 *   res_numel  elements of the residual (same multiple).
 *   x_in       device fp32 [res_numel], 16-byte aligned, or NULL (zero);
 *              it may be x_out itself (in place), not a partial overlap.
 *   x_out      device fp32 [res_numel], 16-byte aligned, outside the arena.
 * Requires a full history.  Errors: CHEB_E_INVAL, CHEB_E_NOTREADY,
 * CHEB_E_ALIGN, CHEB_E_NONFINITE, CHEB_E_HIP. */
CHEB_API int cheb_residual_apply(cheb_cache *c, const double *w, const int64_t *res_offset,
                                 int64_t res_numel, const float *x_in, float *x_out,
                                 void *stream);

/* The same mapping applied to one full step's module outputs:
 *     x_out[j] = x_in[j] + sum over added segments s covering j of
 *                seg_src[s][j - res_offset[s]].
 * Written into a slot of an fp32 cache with one segment of res_numel
 * elements (cheb_cache_begin_push / cheb_cache_commit), it keeps a collapsed
 * history: the block stack's total contribution per full step, from which
 * cheb_residual_apply (res_offset = {0}) predicts a skipped step's residual
 * at a cost of res_numel instead of the whole cache per entry.  Equal to
 * the full form by linearity of the prediction.
 *   seg_src [n_segs] device pointers, 16-byte aligned (NULL allowed for
 *           segments not added), seg_numel[s] elements of `dtype` each.
 * Other arguments as cheb_residual_apply.  Errors: CHEB_E_INVAL,
 * CHEB_E_DTYPE, CHEB_E_ALIGN, CHEB_E_HIP. */
CHEB_API int cheb_residual_reduce(const void *const *seg_src, const int64_t *seg_numel,
                                  const int64_t *res_offset, int32_t n_segs, int32_t dtype,
                                  const float *x_in, float *x_out, int64_t res_numel,
                                  void *stream);

/* ------------------------------------------------------------------------ */
/* Launch shape (tuning).                                                    */
/* ------------------------------------------------------------------------ */

/* Launch shape of the streaming kernels, process-wide.
 *   block        threads per block: 64, 256, 512 or 1024.
 *   unroll       16-byte vectors per thread per history entry in flight;
 *                block * unroll must not exceed 1024 (64: 1; 256: 1, 2
 *                or 4; 512: 1 or 2; 1024: 1).
 *   nontemporal  1: history loads and output stores carry the non-temporal
 *                hint; 0: ordinary loads and stores.
 *   blocks_per_cu  0: one block per tile of block x unroll vectors (the grid
 *                covers the whole problem); 1..64: a persistent grid of that
 *                many blocks per compute unit, each looping over tiles.
 *   waves_per_cu  cap on the prediction kernel's 64-lane waves resident on
 *                one compute unit.  0: chosen from the history size n and
 *                the number of outputs: for one output max(6, 44/n rounded)
 *                (7 for 6 entries, 9 for 5), for several max(6, 36/n
 *                rounded), no cap for n <= 2; -1: no cap; 1..32: that cap.
 *                Each block reserves an equal share of the compute unit's
 *                LDS, rounded down to 512 bytes, which the kernel never
 *                touches, so that no more blocks fit; the cap applies only
 *                where that share is at most 64 KiB (64- and 256-thread
 *                blocks) and is ignored otherwise.  While a prediction
 *                runs, kernels on other streams find that LDS taken; -1
 *                leaves it free.
 * Default {64, 1, 1, 0, 0}.  On MI355X a bf16 history of 5-6 entries
 * streams at about 0.85 of the HBM peak under the chosen cap, against 0.75
 * with 1024-thread blocks at full occupancy: fewer waves keep enough loads
 * in flight without crowding out the output's stores.  With
 * block 1024, a problem under 4096 vectors per compute unit runs with
 * 256-thread blocks.  The history ring's push (a copy) always runs at full
 * occupancy.  Errors: CHEB_E_INVAL. */
typedef struct cheb_launch_config {
  int32_t block;
  int32_t unroll;
  int32_t nontemporal;
  int32_t blocks_per_cu;
  int32_t waves_per_cu;
} cheb_launch_config;

CHEB_API int cheb_get_launch_config(cheb_launch_config *cfg);
CHEB_API int cheb_set_launch_config(const cheb_launch_config *cfg);

#ifdef __cplusplus
}
#endif

#endif /* CHEB_H */
