"""ctypes binding of libcheb.so: the C entry points under their own names.

Argument marshalling only.  Every step of the path runs in the library; there
is no fallback: when libcheb.so is missing or does not load, importing the
package fails.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcheb.so")

# The library version this binding's structures match (CHEB_VERSION).
CHEB_VERSION = 4

CHEB_OK = 0
CHEB_E_INVAL = -1
CHEB_E_DUPNODE = -2
CHEB_E_NOTREADY = -3
CHEB_E_DTYPE = -4
CHEB_E_ALIGN = -5
CHEB_E_HIP = -6
CHEB_E_MISMATCH = -7
CHEB_E_NONFINITE = -8
CHEB_E_IO = -9

CHEB_SHORT_FULL = 0
CHEB_SHORT_LOWER = 1

CHEB_RHO_GENERAL = 0
CHEB_RHO_ALTERNATING = 1
CHEB_TAYLOR = 2

CHEB_LAYOUT_SLOTS = 0
CHEB_LAYOUT_INTERLEAVED = 1

CHEB_BF16 = 0
CHEB_F32 = 1
CHEB_F16 = 2
CHEB_MAX_SLOTS = 8
CHEB_MAX_OUTPUTS = 8
CHEB_MAX_NODES = 64

STATUS_NAMES = {
    CHEB_E_INVAL: "CHEB_E_INVAL", CHEB_E_DUPNODE: "CHEB_E_DUPNODE",
    CHEB_E_NOTREADY: "CHEB_E_NOTREADY", CHEB_E_DTYPE: "CHEB_E_DTYPE",
    CHEB_E_ALIGN: "CHEB_E_ALIGN", CHEB_E_HIP: "CHEB_E_HIP",
    CHEB_E_MISMATCH: "CHEB_E_MISMATCH", CHEB_E_NONFINITE: "CHEB_E_NONFINITE",
    CHEB_E_IO: "CHEB_E_IO",
}


class ChebError(RuntimeError):
    def __init__(self, code, message):
        self.code = code
        self.name = STATUS_NAMES.get(code, str(code))
        super().__init__(f"{self.name}: {message}")


class cheb_launch_config(ctypes.Structure):
    _fields_ = [("block", ctypes.c_int32), ("unroll", ctypes.c_int32),
                ("nontemporal", ctypes.c_int32), ("blocks_per_cu", ctypes.c_int32),
                ("waves_per_cu", ctypes.c_int32)]


# The library's launch shape at load time (64-lane blocks, occupancy capped by
# history size).
DEFAULT_LAUNCH_CONFIG = {"block": 64, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 0,
                         "waves_per_cu": 0}


_dp = ctypes.POINTER(ctypes.c_double)
_i64p = ctypes.POINTER(ctypes.c_int64)
_i32p = ctypes.POINTER(ctypes.c_int32)
_szp = ctypes.POINTER(ctypes.c_size_t)
_vp = ctypes.c_void_p
_vpp = ctypes.POINTER(ctypes.c_void_p)

# name -> (argtypes)
SIGNATURES = {
    "cheb_last_error": [],
    "cheb_version": [],
    "cheb_precompute_weights": [_dp, ctypes.c_int32, _dp, ctypes.c_int32, _dp],
    "cheb_precompute_weights_variant": [_dp, ctypes.c_int32, _dp, ctypes.c_int32,
                                        ctypes.c_int32, _dp],
    "cheb_chebyshev_nodes": [ctypes.c_int32, ctypes.c_int32, ctypes.c_double, ctypes.c_double,
                             _dp],
    "cheb_combine": [_vpp, ctypes.c_int32, _dp, _vp, ctypes.c_int64, ctypes.c_int32, _vp],
    "cheb_combine_multi": [_vpp, ctypes.c_int32, _dp, ctypes.c_int32, _vpp, ctypes.c_int64,
                           ctypes.c_int32, _vp],
    "cheb_cache_arena_bytes": [ctypes.c_int32, ctypes.c_int32, _i64p, ctypes.c_int32, _szp, _szp],
    "cheb_cache_arena_bytes_ex": [ctypes.c_int32, ctypes.c_int32, _i64p, ctypes.c_int32,
                                  ctypes.c_int32, _szp],
    "cheb_cache_create_ex": [ctypes.POINTER(_vp), ctypes.c_int32, ctypes.c_int32, _i64p,
                             ctypes.c_int32, ctypes.c_int32, _vp, ctypes.c_size_t],
    "cheb_cache_geometry": [_vp, _i32p, _i64p, _i64p],
    "cheb_cache_layout": [ctypes.c_int32, ctypes.c_int32, _i64p, ctypes.c_int32, _i64p,
                          _i64p, _szp, _szp],
    "cheb_cache_create": [ctypes.POINTER(_vp), ctypes.c_int32, ctypes.c_int32, _i64p,
                          ctypes.c_int32, _vp, ctypes.c_size_t],
    "cheb_cache_destroy": [_vp],
    "cheb_cache_reset": [_vp],
    "cheb_cache_push": [_vp, ctypes.c_double, _vpp, _vp],
    "cheb_cache_begin_push": [_vp, _vpp],
    "cheb_cache_commit": [_vp, ctypes.c_double],
    "cheb_cache_abort_push": [_vp],
    "cheb_cache_history": [_vp, _dp, _i32p],
    "cheb_cache_entry": [_vp, ctypes.c_int32, _vpp],
    "cheb_cache_segment_offset": [_vp, ctypes.c_int32, _i64p],
    "cheb_cache_slot_numel": [_vp, _i64p],
    "cheb_cache_dtype": [_vp, _i32p],
    "cheb_schedule": [ctypes.c_int32] * 4 + [ctypes.POINTER(ctypes.c_uint8)],
    "cheb_table_build": [ctypes.POINTER(_vp)] + [ctypes.c_int32] * 5 + [_dp, ctypes.c_int32],
    "cheb_table_build_mask": [ctypes.POINTER(_vp), ctypes.c_int32, ctypes.POINTER(ctypes.c_uint8),
                              ctypes.c_int32, _dp, ctypes.c_int32],
    "cheb_table_destroy": [_vp],
    "cheb_table_info": [_vp, _i32p, _i32p, _i32p, _i32p],
    "cheb_table_step": [_vp, ctypes.c_int32, _i32p, _i32p, _i32p, _dp],
    "cheb_table_save": [_vp, ctypes.c_char_p],
    "cheb_table_load": [ctypes.POINTER(_vp), ctypes.c_char_p],
    "cheb_extrapolate_steps": [_vp, _vp, ctypes.c_int32, ctypes.c_int32, _vpp, _vp],
    "cheb_extrapolate": [_vp, _dp, _vp, _vp],
    "cheb_extrapolate_at": [_vp, ctypes.c_double, _vp, _vp, _dp],
    "cheb_extrapolate_multi": [_vp, _dp, ctypes.c_int32, _vpp, _vp],
    "cheb_extrapolate_at_multi": [_vp, _dp, ctypes.c_int32, _vpp, _vp, _dp],
    "cheb_residual_apply": [_vp, _dp, _i64p, ctypes.c_int64, _vp, _vp, _vp],
    "cheb_residual_reduce": [_vpp, _i64p, _i64p, ctypes.c_int32, ctypes.c_int32, _vp, _vp,
                             ctypes.c_int64, _vp],
    "cheb_get_launch_config": [ctypes.POINTER(cheb_launch_config)],
    "cheb_set_launch_config": [ctypes.POINTER(cheb_launch_config)],
}


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run __graft_entry__.build() (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, argtypes in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = argtypes
        fn.restype = ctypes.c_char_p if name == "cheb_last_error" else ctypes.c_int
    if lib.cheb_version() != CHEB_VERSION:
        raise ImportError(f"{LIB_PATH} is version {lib.cheb_version()}, the binding expects "
                          f"{CHEB_VERSION}; rebuild with __graft_entry__.build()")
    return lib


LIB = _load()


def _check(rc):
    if rc != CHEB_OK:
        raise ChebError(rc, LIB.cheb_last_error().decode(errors="replace"))
    return rc


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _dptr(a):
    return a.ctypes.data_as(_dp)


def _voidp_array(ptrs):
    return (ctypes.c_void_p * max(1, len(ptrs)))(*[ctypes.c_void_p(int(p)) for p in ptrs])


def cheb_version() -> int:
    return LIB.cheb_version()


def cheb_last_error() -> str:
    return LIB.cheb_last_error().decode(errors="replace")


def cheb_precompute_weights(hist_t, target_t) -> np.ndarray:
    """[n_target, n_hist] fp64 coefficient table (host)."""
    h = _f64(hist_t).reshape(-1)
    t = _f64(target_t).reshape(-1)
    w = np.empty((t.size, h.size), dtype=np.float64)
    _check(LIB.cheb_precompute_weights(_dptr(h), h.size, _dptr(t) if t.size else None,
                                       t.size, _dptr(w) if w.size else None))
    return w


def cheb_precompute_weights_variant(hist_t, target_t, variant=CHEB_RHO_GENERAL) -> np.ndarray:
    h = _f64(hist_t).reshape(-1)
    t = _f64(target_t).reshape(-1)
    w = np.empty((t.size, h.size), dtype=np.float64)
    _check(LIB.cheb_precompute_weights_variant(_dptr(h), h.size, _dptr(t) if t.size else None,
                                               t.size, int(variant), _dptr(w) if w.size else None))
    return w


def cheb_chebyshev_nodes(n, kind=1, a=-1.0, b=1.0) -> np.ndarray:
    x = np.empty(int(n), dtype=np.float64)
    _check(LIB.cheb_chebyshev_nodes(int(n), int(kind), float(a), float(b), _dptr(x)))
    return x


def cheb_combine(src_ptrs, w, out_ptr, numel, dtype, stream=0):
    w = _f64(w).reshape(-1)
    arr = _voidp_array(src_ptrs)
    _check(LIB.cheb_combine(arr, len(src_ptrs), _dptr(w), ctypes.c_void_p(int(out_ptr)),
                            int(numel), int(dtype), ctypes.c_void_p(int(stream))))


def cheb_combine_multi(src_ptrs, w, out_ptrs, numel, dtype, stream=0):
    """w: [n_out, n_src] fp64."""
    w = _f64(w)
    n_out = len(out_ptrs)
    w = w.reshape(n_out, len(src_ptrs))
    _check(LIB.cheb_combine_multi(_voidp_array(src_ptrs), len(src_ptrs), _dptr(w), n_out,
                                  _voidp_array(out_ptrs), int(numel), int(dtype),
                                  ctypes.c_void_p(int(stream))))


def cheb_cache_arena_bytes(n_slots, dtype, seg_numel):
    """(arena_bytes, slot_stride_bytes) of a history of n_slots entries."""
    seg = np.ascontiguousarray(seg_numel, dtype=np.int64).reshape(-1)
    arena = ctypes.c_size_t()
    stride = ctypes.c_size_t()
    _check(LIB.cheb_cache_arena_bytes(int(n_slots), int(dtype), seg.ctypes.data_as(_i64p),
                                      seg.size, ctypes.byref(arena), ctypes.byref(stride)))
    return arena.value, stride.value


def cheb_cache_arena_bytes_ex(n_slots, dtype, seg_numel, layout):
    seg = np.ascontiguousarray(seg_numel, dtype=np.int64).reshape(-1)
    arena = ctypes.c_size_t()
    _check(LIB.cheb_cache_arena_bytes_ex(int(n_slots), int(dtype), seg.ctypes.data_as(_i64p),
                                         seg.size, int(layout), ctypes.byref(arena)))
    return arena.value


def cheb_cache_create_ex(n_slots, dtype, seg_numel, layout, arena_ptr, arena_bytes):
    seg = np.ascontiguousarray(seg_numel, dtype=np.int64).reshape(-1)
    h = ctypes.c_void_p()
    _check(LIB.cheb_cache_create_ex(ctypes.byref(h), int(n_slots), int(dtype),
                                    seg.ctypes.data_as(_i64p), seg.size, int(layout),
                                    ctypes.c_void_p(int(arena_ptr)), int(arena_bytes)))
    return h


def cheb_cache_geometry(handle):
    """(layout, chunk_elems, entry_stride_elems) of a cache."""
    lay = ctypes.c_int32()
    chunk = ctypes.c_int64()
    stride = ctypes.c_int64()
    _check(LIB.cheb_cache_geometry(handle, ctypes.byref(lay), ctypes.byref(chunk),
                                   ctypes.byref(stride)))
    return lay.value, chunk.value, stride.value


def cheb_cache_layout(n_slots, dtype, seg_numel):
    seg = np.ascontiguousarray(seg_numel, dtype=np.int64).reshape(-1)
    off = np.empty_like(seg)
    slot_numel = ctypes.c_int64()
    stride = ctypes.c_size_t()
    arena = ctypes.c_size_t()
    _check(LIB.cheb_cache_layout(int(n_slots), int(dtype), seg.ctypes.data_as(_i64p), seg.size,
                                 off.ctypes.data_as(_i64p), ctypes.byref(slot_numel),
                                 ctypes.byref(stride), ctypes.byref(arena)))
    return {"seg_offset": off, "slot_numel": slot_numel.value,
            "slot_stride_bytes": stride.value, "arena_bytes": arena.value}


def cheb_cache_create(n_slots, dtype, seg_numel, arena_ptr, arena_bytes):
    seg = np.ascontiguousarray(seg_numel, dtype=np.int64).reshape(-1)
    h = ctypes.c_void_p()
    _check(LIB.cheb_cache_create(ctypes.byref(h), int(n_slots), int(dtype),
                                 seg.ctypes.data_as(_i64p), seg.size,
                                 ctypes.c_void_p(int(arena_ptr)), int(arena_bytes)))
    return h


def cheb_cache_destroy(handle):
    _check(LIB.cheb_cache_destroy(handle))


def cheb_cache_reset(handle):
    _check(LIB.cheb_cache_reset(handle))


def cheb_cache_push(handle, t, seg_ptrs, stream=0):
    arr = _voidp_array(seg_ptrs)
    _check(LIB.cheb_cache_push(handle, float(t), arr, ctypes.c_void_p(int(stream))))


def cheb_cache_begin_push(handle) -> int:
    p = ctypes.c_void_p()
    _check(LIB.cheb_cache_begin_push(handle, ctypes.byref(p)))
    return int(p.value or 0)


def cheb_cache_commit(handle, t):
    _check(LIB.cheb_cache_commit(handle, float(t)))


def cheb_cache_abort_push(h):
    _check(LIB.cheb_cache_abort_push(h))


def cheb_cache_history(handle, n_slots=CHEB_MAX_SLOTS):
    t = np.empty(CHEB_MAX_SLOTS, dtype=np.float64)
    n = ctypes.c_int32()
    _check(LIB.cheb_cache_history(handle, _dptr(t), ctypes.byref(n)))
    return t[:n.value].copy()


def cheb_cache_entry(handle, idx) -> int:
    p = ctypes.c_void_p()
    _check(LIB.cheb_cache_entry(handle, int(idx), ctypes.byref(p)))
    return int(p.value or 0)


def cheb_cache_segment_offset(handle, seg) -> int:
    o = ctypes.c_int64()
    _check(LIB.cheb_cache_segment_offset(handle, int(seg), ctypes.byref(o)))
    return o.value


def cheb_cache_slot_numel(handle) -> int:
    n = ctypes.c_int64()
    _check(LIB.cheb_cache_slot_numel(handle, ctypes.byref(n)))
    return n.value


def cheb_cache_dtype(handle) -> int:
    d = ctypes.c_int32()
    _check(LIB.cheb_cache_dtype(handle, ctypes.byref(d)))
    return d.value


def cheb_schedule(T, s0, s1, r) -> np.ndarray:
    """Boolean mask over steps 0..T-1 of the full-computation schedule."""
    mask = np.zeros(int(T), dtype=np.uint8)
    _check(LIB.cheb_schedule(int(T), int(s0), int(s1), int(r),
                             mask.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))))
    return mask.astype(bool)


def cheb_table_build(T, s0, s1, r, n_hist, abscissa, policy=CHEB_SHORT_FULL):
    x = _f64(abscissa).reshape(-1)
    h = ctypes.c_void_p()
    _check(LIB.cheb_table_build(ctypes.byref(h), int(T), int(s0), int(s1), int(r), int(n_hist),
                                _dptr(x), int(policy)))
    return h


def cheb_table_build_mask(is_full, n_hist, abscissa, policy=CHEB_SHORT_FULL):
    mask = np.ascontiguousarray(is_full, dtype=np.uint8).reshape(-1)
    x = _f64(abscissa).reshape(-1)
    h = ctypes.c_void_p()
    _check(LIB.cheb_table_build_mask(ctypes.byref(h), mask.size,
                                     mask.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
                                     int(n_hist), _dptr(x), int(policy)))
    return h


def cheb_table_destroy(table):
    _check(LIB.cheb_table_destroy(table))


def cheb_table_info(table):
    T, n, p, f = (ctypes.c_int32() for _ in range(4))
    _check(LIB.cheb_table_info(table, ctypes.byref(T), ctypes.byref(n), ctypes.byref(p),
                               ctypes.byref(f)))
    return {"T": T.value, "n_hist": n.value, "policy": p.value, "n_full": f.value}


def cheb_table_step(table, step):
    """(predicted, node steps, weights) of one step."""
    pred, used = ctypes.c_int32(), ctypes.c_int32()
    nodes = (ctypes.c_int32 * CHEB_MAX_SLOTS)()
    w = np.zeros(CHEB_MAX_SLOTS, dtype=np.float64)
    _check(LIB.cheb_table_step(table, int(step), ctypes.byref(pred), ctypes.byref(used), nodes,
                               _dptr(w)))
    return bool(pred.value), [nodes[j] for j in range(used.value)], w[:used.value].copy()


def cheb_table_save(table, path):
    _check(LIB.cheb_table_save(table, os.fsencode(path)))


def cheb_table_load(path):
    h = ctypes.c_void_p()
    _check(LIB.cheb_table_load(ctypes.byref(h), os.fsencode(path)))
    return h


def cheb_extrapolate_steps(handle, table, first_step, out_ptrs, stream=0):
    _check(LIB.cheb_extrapolate_steps(handle, table, int(first_step), len(out_ptrs),
                                      _voidp_array(out_ptrs), ctypes.c_void_p(int(stream))))


def cheb_extrapolate(handle, w, out_ptr, stream=0):
    w = _f64(w).reshape(-1)
    _check(LIB.cheb_extrapolate(handle, _dptr(w), ctypes.c_void_p(int(out_ptr)),
                                ctypes.c_void_p(int(stream))))


def cheb_extrapolate_at(handle, target_t, out_ptr, stream=0, n_slots=CHEB_MAX_SLOTS):
    w = np.zeros(CHEB_MAX_SLOTS, dtype=np.float64)
    _check(LIB.cheb_extrapolate_at(handle, float(target_t), ctypes.c_void_p(int(out_ptr)),
                                   ctypes.c_void_p(int(stream)), _dptr(w)))
    return w[:n_slots].copy()


def cheb_extrapolate_multi(handle, w, out_ptrs, stream=0):
    """w: [n_out, n_slots] fp64, rows aligned with cheb_cache_history."""
    w = _f64(w).reshape(len(out_ptrs), -1)
    _check(LIB.cheb_extrapolate_multi(handle, _dptr(w), len(out_ptrs), _voidp_array(out_ptrs),
                                      ctypes.c_void_p(int(stream))))


def cheb_extrapolate_at_multi(handle, targets, out_ptrs, stream=0, n_slots=CHEB_MAX_SLOTS):
    t = _f64(targets).reshape(-1)
    if t.size != len(out_ptrs):
        raise ChebError(CHEB_E_INVAL, "one output per target")
    w = np.zeros((CHEB_MAX_OUTPUTS, CHEB_MAX_SLOTS), dtype=np.float64)
    _check(LIB.cheb_extrapolate_at_multi(handle, _dptr(t), t.size, _voidp_array(out_ptrs),
                                         ctypes.c_void_p(int(stream)), _dptr(w)))
    return w.reshape(-1)[:t.size * n_slots].reshape(t.size, n_slots).copy()


def cheb_residual_apply(handle, w, res_offset, res_numel, x_in_ptr, x_out_ptr, stream=0):
    w = _f64(w).reshape(-1)
    ro = np.ascontiguousarray(res_offset, dtype=np.int64).reshape(-1)
    _check(LIB.cheb_residual_apply(handle, _dptr(w), ro.ctypes.data_as(_i64p), int(res_numel),
                                   ctypes.c_void_p(int(x_in_ptr or 0)),
                                   ctypes.c_void_p(int(x_out_ptr)), ctypes.c_void_p(int(stream))))


def cheb_residual_reduce(seg_ptrs, seg_numel, res_offset, dtype, x_in_ptr, x_out_ptr, res_numel,
                         stream=0):
    sn = np.ascontiguousarray(seg_numel, dtype=np.int64).reshape(-1)
    ro = np.ascontiguousarray(res_offset, dtype=np.int64).reshape(-1)
    _check(LIB.cheb_residual_reduce(_voidp_array(seg_ptrs), sn.ctypes.data_as(_i64p),
                                    ro.ctypes.data_as(_i64p), sn.size, int(dtype),
                                    ctypes.c_void_p(int(x_in_ptr or 0)),
                                    ctypes.c_void_p(int(x_out_ptr)), int(res_numel),
                                    ctypes.c_void_p(int(stream))))


def cheb_get_launch_config():
    c = cheb_launch_config()
    _check(LIB.cheb_get_launch_config(ctypes.byref(c)))
    return {"block": c.block, "unroll": c.unroll, "nontemporal": c.nontemporal,
            "blocks_per_cu": c.blocks_per_cu, "waves_per_cu": c.waves_per_cu}


def cheb_set_launch_config(block=64, unroll=1, nontemporal=1, blocks_per_cu=0, waves_per_cu=0):
    c = cheb_launch_config(int(block), int(unroll), int(nontemporal), int(blocks_per_cu),
                           int(waves_per_cu))
    _check(LIB.cheb_set_launch_config(ctypes.byref(c)))
