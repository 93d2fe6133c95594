"""fp64 CPU oracle for the ChebBooster online stage.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg load it; the product package never does.  It is a ctypes view
of ``oracle.c`` (plain C, fp64), which shares no code with the HIP library.
Every function's paper citation is in ``oracle.c``.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None

_c_double_p = ctypes.POINTER(ctypes.c_double)
_c_u16_p = ctypes.POINTER(ctypes.c_uint16)
_c_f32_p = ctypes.POINTER(ctypes.c_float)


class OracleError(ValueError):
    pass


_NODE_ERRORS = {-1: "bad node count", -2: "non-finite node or target",
                -3: "repeated node"}


def lib():
    """Load liboracle.so, building it first only when it is not there."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _LIB = bind(_build.LIB)
    return _LIB


def bind(path):
    """ctypes handle of an oracle library at ``path`` with its signatures."""
    L = ctypes.CDLL(path)
    L.oracle_set_threads.argtypes = [ctypes.c_int]
    L.oracle_set_threads.restype = ctypes.c_int
    L.oracle_max_threads.restype = ctypes.c_int
    L.oracle_check_nodes.argtypes = [_c_double_p, ctypes.c_int]
    L.oracle_normalise.argtypes = [_c_double_p, ctypes.c_int, ctypes.c_double,
                                   _c_double_p, _c_double_p]
    L.oracle_normalise.restype = None
    L.oracle_barycentric_rho.argtypes = [_c_double_p, ctypes.c_int, _c_double_p]
    L.oracle_barycentric_rho.restype = None
    for name in ("oracle_weights_row", "oracle_lagrange_row"):
        getattr(L, name).argtypes = [_c_double_p, ctypes.c_int, ctypes.c_double,
                                     _c_double_p]
    L.oracle_weights.argtypes = [_c_double_p, ctypes.c_int, _c_double_p,
                                 ctypes.c_int, _c_double_p]
    L.oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
    L.oracle_bf16_to_f64.restype = ctypes.c_double
    L.oracle_round_bf16.argtypes = [ctypes.c_double]
    L.oracle_round_bf16.restype = ctypes.c_uint16
    L.oracle_round_f32.argtypes = [ctypes.c_double]
    L.oracle_round_f32.restype = ctypes.c_float
    L.oracle_decode_bf16.argtypes = [_c_u16_p, ctypes.c_int64, _c_double_p]
    L.oracle_decode_bf16.restype = None
    L.oracle_encode_bf16.argtypes = [_c_double_p, ctypes.c_int64, _c_u16_p]
    L.oracle_encode_bf16.restype = None
    L.oracle_extrapolate_bf16.argtypes = [ctypes.POINTER(_c_u16_p), ctypes.c_int,
                                          _c_double_p, ctypes.c_int64,
                                          _c_double_p, _c_double_p]
    L.oracle_extrapolate_bf16.restype = None
    L.oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
    L.oracle_f16_to_f64.restype = ctypes.c_double
    L.oracle_round_f16.argtypes = [ctypes.c_double]
    L.oracle_round_f16.restype = ctypes.c_uint16
    L.oracle_decode_f16.argtypes = [_c_u16_p, ctypes.c_int64, _c_double_p]
    L.oracle_decode_f16.restype = None
    L.oracle_encode_f16.argtypes = [_c_double_p, ctypes.c_int64, _c_u16_p]
    L.oracle_encode_f16.restype = None
    L.oracle_extrapolate_f16.argtypes = [ctypes.POINTER(_c_u16_p), ctypes.c_int,
                                         _c_double_p, ctypes.c_int64,
                                         _c_double_p, _c_double_p]
    L.oracle_extrapolate_f16.restype = None
    L.oracle_extrapolate_f32.argtypes = [ctypes.POINTER(_c_f32_p), ctypes.c_int,
                                         _c_double_p, ctypes.c_int64,
                                         _c_double_p, _c_double_p]
    L.oracle_extrapolate_f32.restype = None
    L.oracle_extrapolate_f64.argtypes = [ctypes.POINTER(_c_double_p), ctypes.c_int,
                                         _c_double_p, ctypes.c_int64, _c_double_p]
    L.oracle_extrapolate_f64.restype = None
    L.oracle_full_schedule.argtypes = [ctypes.c_int] * 4 + [
        ctypes.POINTER(ctypes.c_uint8)]
    L.oracle_chebyshev_nodes.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                         ctypes.c_double, _c_double_p]
    L.oracle_weights_row_alternating.argtypes = [_c_double_p, ctypes.c_int, ctypes.c_double,
                                                 _c_double_p]
    L.oracle_weights_row_taylor.argtypes = [_c_double_p, ctypes.c_int, ctypes.c_double,
                                            _c_double_p]
    _i64 = ctypes.POINTER(ctypes.c_int64)
    L.oracle_residual_bf16.argtypes = [ctypes.POINTER(_c_u16_p), ctypes.c_int, _c_double_p,
                                       _i64, _i64, _i64, ctypes.c_int, _c_double_p,
                                       ctypes.c_int64, _c_double_p, _c_double_p]
    L.oracle_residual_f32.argtypes = [ctypes.POINTER(_c_f32_p), ctypes.c_int, _c_double_p,
                                      _i64, _i64, _i64, ctypes.c_int, _c_double_p,
                                      ctypes.c_int64, _c_double_p, _c_double_p]
    L.oracle_residual_f16.argtypes = L.oracle_residual_bf16.argtypes
    _ip = ctypes.POINTER(ctypes.c_int)
    L.oracle_table_row_mask.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_uint8), ctypes.c_int,
                                        _c_double_p, ctypes.c_int, ctypes.c_int, _ip, _ip, _ip,
                                        _c_double_p]
    L.oracle_table_row.argtypes = [ctypes.c_int] * 5 + [_c_double_p, ctypes.c_int, ctypes.c_int,
                                                        _ip, _ip, _ip, _c_double_p]
    return L


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _check(rc):
    if rc != 0:
        raise OracleError(_NODE_ERRORS.get(rc, f"oracle error {rc}"))


def set_threads(n: int) -> int:
    return lib().oracle_set_threads(int(n))


def max_threads() -> int:
    return lib().oracle_max_threads()


def check_nodes(x) -> int:
    x = _f64(x)
    return lib().oracle_check_nodes(_ptr(x, ctypes.c_double), len(x))


def normalise(x, xstar):
    x = _f64(x)
    y = np.empty_like(x)
    ys = ctypes.c_double()
    lib().oracle_normalise(_ptr(x, ctypes.c_double), len(x), float(xstar),
                           _ptr(y, ctypes.c_double), ctypes.byref(ys))
    return y, ys.value


def barycentric_rho(y):
    y = _f64(y)
    rho = np.empty_like(y)
    lib().oracle_barycentric_rho(_ptr(y, ctypes.c_double), len(y),
                                 _ptr(rho, ctypes.c_double))
    return rho


def weights_row(x, xstar):
    x = _f64(x)
    w = np.empty_like(x)
    _check(lib().oracle_weights_row(_ptr(x, ctypes.c_double), len(x), float(xstar),
                                    _ptr(w, ctypes.c_double)))
    return w


def weights(x, targets):
    """Table w[m, j] for targets m and nodes j (oldest to newest)."""
    x = _f64(x)
    t = _f64(np.atleast_1d(targets))
    w = np.empty((len(t), len(x)), dtype=np.float64)
    _check(lib().oracle_weights(_ptr(x, ctypes.c_double), len(x),
                                _ptr(t, ctypes.c_double), len(t),
                                _ptr(w, ctypes.c_double)))
    return w


def lagrange_row(x, xstar):
    x = _f64(x)
    w = np.empty_like(x)
    _check(lib().oracle_lagrange_row(_ptr(x, ctypes.c_double), len(x), float(xstar),
                                     _ptr(w, ctypes.c_double)))
    return w


def bf16_to_f64(h):
    h = np.ascontiguousarray(h, dtype=np.uint16).reshape(-1)
    out = np.empty(h.shape, dtype=np.float64)
    lib().oracle_decode_bf16(_ptr(h, ctypes.c_uint16), h.size, _ptr(out, ctypes.c_double))
    return out


def round_bf16(v):
    """Correctly rounded (ties-to-even) bfloat16 bit patterns of fp64 values."""
    v = _f64(v).reshape(-1)
    out = np.empty(v.shape, dtype=np.uint16)
    lib().oracle_encode_bf16(_ptr(v, ctypes.c_double), v.size, _ptr(out, ctypes.c_uint16))
    return out


def f16_to_f64(h):
    """Exact values of binary16 bit patterns (uint16 arrays)."""
    h = np.ascontiguousarray(h, dtype=np.uint16).reshape(-1)
    out = np.empty(h.shape, dtype=np.float64)
    lib().oracle_decode_f16(_ptr(h, ctypes.c_uint16), h.size, _ptr(out, ctypes.c_double))
    return out


def round_f16(v):
    """Correctly rounded (ties-to-even) binary16 bit patterns of fp64 values."""
    v = _f64(v).reshape(-1)
    out = np.empty(v.shape, dtype=np.uint16)
    lib().oracle_encode_f16(_ptr(v, ctypes.c_double), v.size, _ptr(out, ctypes.c_uint16))
    return out


def _slots(slots, dtype):
    arrs = [np.ascontiguousarray(s, dtype=dtype).reshape(-1) for s in slots]
    if not arrs:
        raise OracleError("no history entries")
    count = arrs[0].size
    if any(a.size != count for a in arrs):
        raise OracleError("history entries differ in length")
    return arrs, count


def extrapolate_bf16(slots, w, want_absmag=True):
    """fp64 sum_k w[k] * F_k over bfloat16 bit patterns (uint16 arrays)."""
    arrs, count = _slots(slots, np.uint16)
    w = _f64(w)
    if len(w) != len(arrs):
        raise OracleError("weight count differs from history size")
    ptrs = (_c_u16_p * len(arrs))(*[_ptr(a, ctypes.c_uint16) for a in arrs])
    out = np.empty(count, dtype=np.float64)
    mag = np.empty(count, dtype=np.float64) if want_absmag else None
    lib().oracle_extrapolate_bf16(ptrs, len(arrs), _ptr(w, ctypes.c_double), count,
                                  _ptr(out, ctypes.c_double),
                                  _ptr(mag, ctypes.c_double) if want_absmag else None)
    return (out, mag) if want_absmag else out


def extrapolate_f16(slots, w, want_absmag=True):
    """fp64 sum_k w[k] * F_k over binary16 bit patterns (uint16 arrays)."""
    arrs, count = _slots(slots, np.uint16)
    w = _f64(w)
    if len(w) != len(arrs):
        raise OracleError("weight count differs from history size")
    ptrs = (_c_u16_p * len(arrs))(*[_ptr(a, ctypes.c_uint16) for a in arrs])
    out = np.empty(count, dtype=np.float64)
    mag = np.empty(count, dtype=np.float64) if want_absmag else None
    lib().oracle_extrapolate_f16(ptrs, len(arrs), _ptr(w, ctypes.c_double), count,
                                 _ptr(out, ctypes.c_double),
                                 _ptr(mag, ctypes.c_double) if want_absmag else None)
    return (out, mag) if want_absmag else out


def extrapolate_f32(slots, w, want_absmag=True):
    arrs, count = _slots(slots, np.float32)
    w = _f64(w)
    if len(w) != len(arrs):
        raise OracleError("weight count differs from history size")
    ptrs = (_c_f32_p * len(arrs))(*[_ptr(a, ctypes.c_float) for a in arrs])
    out = np.empty(count, dtype=np.float64)
    mag = np.empty(count, dtype=np.float64) if want_absmag else None
    lib().oracle_extrapolate_f32(ptrs, len(arrs), _ptr(w, ctypes.c_double), count,
                                 _ptr(out, ctypes.c_double),
                                 _ptr(mag, ctypes.c_double) if want_absmag else None)
    return (out, mag) if want_absmag else out


def extrapolate_f64(slots, w):
    arrs, count = _slots(slots, np.float64)
    w = _f64(w)
    if len(w) != len(arrs):
        raise OracleError("weight count differs from history size")
    ptrs = (_c_double_p * len(arrs))(*[_ptr(a, ctypes.c_double) for a in arrs])
    out = np.empty(count, dtype=np.float64)
    lib().oracle_extrapolate_f64(ptrs, len(arrs), _ptr(w, ctypes.c_double), count,
                                 _ptr(out, ctypes.c_double))
    return out


def full_schedule(T, s0, s1, r):
    """Boolean mask over steps 0..T-1: True where the full network runs."""
    mask = np.zeros(int(T), dtype=np.uint8)
    rc = lib().oracle_full_schedule(int(T), int(s0), int(s1), int(r),
                                    _ptr(mask, ctypes.c_uint8))
    if rc < 0:
        raise OracleError("bad schedule parameters")
    return mask.astype(bool)


def parity_error(got, expect, absmag, floor=1e-3):
    """Floored relative error max_i |g - o| / max(|o|, floor * absmag).

    ``absmag`` is sum_k |w_k| |F_k[i]|, the size of the terms that cancel in
    element i; the floor keeps the ratio meaningful where they cancel to
    (almost) zero.  Returns (floored max, unfloored max over elements where
    the floor is inactive, normwise error, fraction of floored elements).
    """
    got = np.asarray(got, dtype=np.float64)
    expect = np.asarray(expect, dtype=np.float64)
    absmag = np.asarray(absmag, dtype=np.float64)
    if got.size == 0:
        return 0.0, 0.0, 0.0, 0.0
    diff = np.abs(got - expect)
    scale = np.maximum(np.abs(expect), floor * absmag)
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = np.where(scale > 0, diff / scale, np.where(diff > 0, np.inf, 0.0))
    floored = np.abs(expect) < floor * absmag
    unfl = diff[~floored] / np.abs(expect[~floored]) if (~floored).any() else np.zeros(1)
    unfl = unfl[np.isfinite(unfl)] if unfl.size else unfl
    denom = np.max(np.abs(expect))
    normwise = float(np.max(diff) / denom) if denom > 0 else float(np.max(diff))
    return (float(np.max(rel)), float(np.max(unfl)) if unfl.size else 0.0,
            normwise, float(np.mean(floored)))


def table_row_mask(full_mask, n, abscissa, policy, step):
    """table_row for an arbitrary full-step mask."""
    mask = np.ascontiguousarray(full_mask, dtype=np.uint8)
    x = _f64(abscissa)
    T = mask.size
    if x.size != T:
        raise OracleError("one abscissa per step")
    kind, n_used = ctypes.c_int(), ctypes.c_int()
    nodes = (ctypes.c_int * 64)()
    w = np.zeros(64, dtype=np.float64)
    rc = lib().oracle_table_row_mask(T, mask.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), int(n),
                                     _ptr(x, ctypes.c_double), int(policy), int(step),
                                     ctypes.byref(kind), ctypes.byref(n_used), nodes,
                                     _ptr(w, ctypes.c_double))
    if rc != 0:
        raise OracleError(_NODE_ERRORS.get(rc, f"oracle error {rc}"))
    return kind.value, [nodes[j] for j in range(n_used.value)], w[:n_used.value].copy()


def table_row(T, s0, s1, r, n, abscissa, policy, step):
    """(kind, node steps, weights) of `step` by simulating Algorithm 1:
    kind 0 = full step, 1 = predicted from the listed entries."""
    x = _f64(abscissa)
    if x.size != T:
        raise OracleError("one abscissa per step")
    kind, n_used = ctypes.c_int(), ctypes.c_int()
    nodes = (ctypes.c_int * 64)()
    w = np.zeros(64, dtype=np.float64)
    rc = lib().oracle_table_row(int(T), int(s0), int(s1), int(r), int(n),
                                _ptr(x, ctypes.c_double), int(policy), int(step),
                                ctypes.byref(kind), ctypes.byref(n_used), nodes,
                                _ptr(w, ctypes.c_double))
    if rc != 0:
        raise OracleError(_NODE_ERRORS.get(rc, f"oracle error {rc}"))
    return kind.value, [nodes[j] for j in range(n_used.value)], w[:n_used.value].copy()


def residual(slots, w, slot_offset, seg_numel, res_offset, res_numel, x_in=None,
             dtype="bf16"):
    """x_in + sum over mapped segments of the predicted module outputs (fp64),
    and the magnitude of its terms.  slots: history entries (uint16 patterns
    for bf16 and f16, float32 for f32); res_offset[s] < 0 leaves segment s
    out."""
    half = dtype in ("bf16", "f16")
    ctype = ctypes.c_uint16 if half else ctypes.c_float
    np_t = np.uint16 if half else np.float32
    arrs = [np.ascontiguousarray(a, dtype=np_t).reshape(-1) for a in slots]
    w = _f64(w)
    if len(w) != len(arrs):
        raise OracleError("weight count differs from history size")
    so = np.ascontiguousarray(slot_offset, dtype=np.int64)
    sn = np.ascontiguousarray(seg_numel, dtype=np.int64)
    ro = np.ascontiguousarray(res_offset, dtype=np.int64)
    for a in arrs:
        if np.any((so + sn > a.size) & (ro >= 0)):
            raise OracleError("segment outside a history entry")
    xi = None if x_in is None else _f64(x_in).reshape(-1)
    out = np.empty(int(res_numel), dtype=np.float64)
    mag = np.empty(int(res_numel), dtype=np.float64)
    P = ctypes.POINTER(ctype)
    ptrs = (P * len(arrs))(*[_ptr(a, ctype) for a in arrs])
    fn = {"bf16": lib().oracle_residual_bf16, "f16": lib().oracle_residual_f16,
          "f32": lib().oracle_residual_f32}[dtype]
    rc = fn(ptrs, len(arrs), _ptr(w, ctypes.c_double), _ptr(so, ctypes.c_int64),
            _ptr(sn, ctypes.c_int64), _ptr(ro, ctypes.c_int64), len(sn),
            None if xi is None else _ptr(xi, ctypes.c_double), int(res_numel),
            _ptr(out, ctypes.c_double), _ptr(mag, ctypes.c_double))
    if rc != 0:
        raise OracleError("segment outside the residual")
    return out, mag


def chebyshev_nodes(n, kind=1, a=-1.0, b=1.0):
    """Chebyshev roots (kind 1) or extrema (kind 2) on [a, b], largest first."""
    x = np.empty(int(n), dtype=np.float64)
    if lib().oracle_chebyshev_nodes(int(n), int(kind), float(a), float(b),
                                    _ptr(x, ctypes.c_double)) != 0:
        raise OracleError("bad Chebyshev node request")
    return x


def weights_row_alternating(x, xstar):
    """Coefficients from the alternating weights printed in Section 3.2."""
    x = _f64(x)
    w = np.empty_like(x)
    _check(lib().oracle_weights_row_alternating(_ptr(x, ctypes.c_double), len(x), float(xstar),
                                                _ptr(w, ctypes.c_double)))
    return w


def weights_row_taylor(x, xstar):
    """Coefficients of the Taylor expansion about the newest node with
    divided-difference derivative estimates (the Taylor comparison of
    Section 3.2's Runge study)."""
    x = _f64(x)
    w = np.empty_like(x)
    _check(lib().oracle_weights_row_taylor(_ptr(x, ctypes.c_double), len(x), float(xstar),
                                           _ptr(w, ctypes.c_double)))
    return w
