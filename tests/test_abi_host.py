"""Host-side checks of libcheb through its C ABI (no GPU needed).

The library validates every argument before it touches the HIP runtime, so
everything here (exports, weights, layout, ring bookkeeping, error codes)
runs on the CPU.  Calls that would enqueue GPU work are not made.
"""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
import paper_2608_23429_amd as cheb
from paper_2608_23429_amd import _binding as B
from synth import CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cheb.h")
FAKE_ARENA = 1 << 40      # 256-byte aligned address; never dereferenced here


def _declared():
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"CHEB_API\s+[^;(]*?\b(cheb_\w+)\s*\(", text)))


def test_header_declares_expected_entry_points():
    names = _declared()
    for must in ("cheb_precompute_weights", "cheb_cache_arena_bytes", "cheb_cache_create",
                 "cheb_cache_push", "cheb_cache_begin_push", "cheb_cache_commit",
                 "cheb_cache_history", "cheb_cache_segment_offset", "cheb_extrapolate",
                 "cheb_cache_destroy", "cheb_last_error"):
        assert must in names
    assert len(names) == len(B.SIGNATURES)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(B.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), name
        assert name in B.SIGNATURES, name
        assert hasattr(cheb, name), name       # same name in the binding


def test_version():
    assert cheb.cheb_version() == 4


def _wtol(w, factor=8.0):
    s = float(np.abs(w).sum())
    return factor * len(w) * 2.0 ** -53 * s * max(s, 1.0)


@pytest.mark.parametrize("cfg", CONFIGS, ids=lambda c: c.name)
def test_weights_match_oracle_on_workloads(cfg):
    cases = [(cfg.nodes, cfg.targets)]
    if cfg.alt_nodes is not None:
        cases.append((cfg.alt_nodes, cfg.alt_targets))
    for nodes, targets in cases:
        w = cheb.cheb_precompute_weights(nodes, targets)
        ref = oracle.weights(nodes, targets)
        for m in range(len(targets)):
            assert np.max(np.abs(w[m] - ref[m])) <= _wtol(ref[m]), (cfg.name, targets[m])


def test_weights_match_oracle_random():
    rng = np.random.default_rng(101)
    for n in range(1, 9):
        for _ in range(40):
            x = rng.uniform(-50, 50, n)
            if n > 1 and np.min(np.diff(np.sort(x))) < 1.0:
                continue
            t = rng.uniform(-80, 80, 3)
            w = cheb.cheb_precompute_weights(x, t)
            ref = oracle.weights(x, t)
            for m in range(3):
                assert np.max(np.abs(w[m] - ref[m])) <= _wtol(ref[m], 32.0)


def test_weights_node_hit_and_single_node():
    x = [0.96, 0.9, 0.8, 0.72, 0.6, 0.5]
    w = cheb.cheb_precompute_weights(x, x)
    assert np.array_equal(w, np.eye(6))
    assert cheb.cheb_precompute_weights([3.0], [1.0, 7.0]).tolist() == [[1.0], [1.0]]


def test_weights_errors_leave_output_untouched():
    h = np.array([1.0, 2.0, 1.0])
    t = np.array([4.0])
    w = np.full((1, 3), 7.0)
    rc = B.LIB.cheb_precompute_weights(B._dptr(h), 3, B._dptr(t), 1, B._dptr(w))
    assert rc == B.CHEB_E_DUPNODE
    assert np.all(w == 7.0)
    assert "equal" in cheb.cheb_last_error()
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_precompute_weights([1.0, np.nan], [3.0])
    assert e.value.code == B.CHEB_E_NONFINITE
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_precompute_weights([1.0, 2.0], [np.inf])
    assert e.value.code == B.CHEB_E_NONFINITE
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_precompute_weights([], [1.0])
    assert e.value.code == B.CHEB_E_INVAL
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_precompute_weights(np.arange(65.0), [100.0])
    assert e.value.code == B.CHEB_E_INVAL
    assert cheb.cheb_precompute_weights(np.arange(64.0), []).shape == (0, 64)


def _clustered(count=30, step=2.0 ** -40):
    """Two end nodes at -1 and 1 (the map onto [-1, 1] is then the identity)
    and `count` nodes `step` apart at 0: omega'(x_j) of a clustered node is
    about step^(count-1), below the smallest double for these defaults."""
    return [-1.0] + [k * step for k in range(count)] + [1.0]


def test_weights_of_clustered_nodes_match_exact():
    """The products of the second form leave the double range here; the
    weights still match the exact rational Lagrange coefficients (Appendix
    A, Lagrange basis) at targets inside the cluster, each to within the
    second form's rounding bound n 2^-53 sum|w| relative to itself."""
    from tests.lagrange_exact import lagrange_weights
    x = _clustered()
    assert abs(math.prod(x[1] - v for v in x[2:])) < 1e-300
    for target in [14.5 * 2.0 ** -40, 3.25 * 2.0 ** -40, 27.75 * 2.0 ** -40]:
        w = cheb.cheb_precompute_weights(x, [target])[0]
        exact = np.array([float(v) for v in lagrange_weights(x, target)])
        mass = float(np.abs(exact).sum())
        bound = 4 * len(x) * 2.0 ** -53 * mass
        assert np.all(np.abs(w - exact) <= bound * np.abs(exact) + 1e-300), (target, mass)


def test_weights_beyond_fp64_resolution_are_an_error():
    """Where the second form's rounding bound n 2^-53 sum|w| passes 2^-24
    (the fp32 resolution the bf16 kernel uses the row at), or the exact
    coefficients exceed the double range, the call fails with
    CHEB_E_NONFINITE and leaves w_out alone."""
    from tests.lagrange_exact import lagrange_weights
    x = _clustered()
    t_ill = 29.5 * 2.0 ** -40
    mass = float(sum(abs(v) for v in lagrange_weights(x, t_ill)))
    assert len(x) * 2.0 ** -53 * mass > 2.0 ** -24
    assert max(abs(v) for v in lagrange_weights(x, 0.5)) > 2 ** 1024
    h = np.array(x)
    for target in (t_ill, 0.5):
        t = np.array([target])
        w = np.full((1, len(x)), 7.0)
        rc = B.LIB.cheb_precompute_weights(B._dptr(h), len(x), B._dptr(t), 1, B._dptr(w))
        assert rc == B.CHEB_E_NONFINITE, target
        assert np.all(w == 7.0)
        assert "not finite" in cheb.cheb_last_error() or "ill-conditioned" in cheb.cheb_last_error()


def test_nodes_that_the_map_merges_are_duplicates():
    """Distinct abscissae that round to one value once mapped onto [-1, 1]
    are reported as duplicates instead of giving non-finite weights."""
    x = [-7.002881094626153, -6.668508865894732, -6.668508865894731, 4.804184990778926]
    mid, inv_half = 0.5 * (x[0] + x[3]), 2.0 / (x[3] - x[0])
    assert x[1] != x[2] and (x[1] - mid) * inv_half == (x[2] - mid) * inv_half
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_precompute_weights(x, [5.0])
    assert e.value.code == B.CHEB_E_DUPNODE
    assert "coincide" in str(e.value) or "coincide" in cheb.cheb_last_error()


# --------------------------------------------------------------------------
# Layout
# --------------------------------------------------------------------------

def _expected_layout(n_slots, esize, seg):
    vec = 16 // esize
    off, pos = [], 0
    for n in seg:
        off.append(pos)
        pos += -(-n // vec) * vec
    stride = -(-(pos * esize) // 256) * 256
    return off, pos, stride, stride * n_slots


@pytest.mark.parametrize("dtype,esize", [(B.CHEB_BF16, 2), (B.CHEB_F16, 2), (B.CHEB_F32, 4)])
def test_layout_rounding(dtype, esize):
    seg = [1, 8, 13, 0, 1000003, 3, 4096 * 3072]
    lay = cheb.cheb_cache_layout(5, dtype, seg)
    off, pos, stride, arena = _expected_layout(5, esize, seg)
    assert lay["seg_offset"].tolist() == off
    assert lay["slot_numel"] == pos
    assert lay["slot_stride_bytes"] == stride and stride % 256 == 0
    assert lay["arena_bytes"] == arena
    assert cheb.cheb_cache_arena_bytes(5, dtype, seg) == (arena, stride)


def test_layout_of_workloads_has_no_padding():
    for c in CONFIGS:
        lay = cheb.cheb_cache_layout(c.n_hist, B.CHEB_BF16 if c.dtype == "bf16" else B.CHEB_F32,
                                     c.seg_numel)
        assert lay["slot_numel"] == c.numel
        assert lay["seg_offset"].tolist() == list(np.cumsum([0] + c.seg_numel[:-1]))


def test_layout_errors():
    for args, code in [((0, 0, [4]), B.CHEB_E_INVAL), ((9, 0, [4]), B.CHEB_E_INVAL),
                       ((2, 5, [4]), B.CHEB_E_DTYPE), ((2, 0, [-1]), B.CHEB_E_INVAL),
                       ((2, 0, [1 << 40]), B.CHEB_E_INVAL)]:
        with pytest.raises(cheb.ChebError) as e:
            cheb.cheb_cache_layout(*args)
        assert e.value.code == code
        with pytest.raises(cheb.ChebError) as e:
            cheb.cheb_cache_arena_bytes(*args)
        assert e.value.code == code


# --------------------------------------------------------------------------
# Ring bookkeeping (metadata paths only; no GPU work is enqueued)
# --------------------------------------------------------------------------

def _fake_cache(n_slots=4, seg=(1000, 24), dtype=B.CHEB_BF16):
    lay = cheb.cheb_cache_layout(n_slots, dtype, list(seg))
    h = cheb.cheb_cache_create(n_slots, dtype, list(seg), FAKE_ARENA, lay["arena_bytes"])
    return h, lay


def test_create_errors():
    lay = cheb.cheb_cache_layout(4, B.CHEB_BF16, [1000])
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_create(4, B.CHEB_BF16, [1000], FAKE_ARENA + 16, lay["arena_bytes"])
    assert e.value.code == B.CHEB_E_ALIGN
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_create(4, B.CHEB_BF16, [1000], FAKE_ARENA, lay["arena_bytes"] - 1)
    assert e.value.code == B.CHEB_E_MISMATCH
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_create(4, B.CHEB_BF16, [1000], 0, lay["arena_bytes"])
    assert e.value.code == B.CHEB_E_INVAL


def test_fifo_order_and_eviction():
    """Algorithm 1: H holds the n most recent (s, f_s); the oldest is dropped."""
    h, lay = _fake_cache(n_slots=4)
    stride = lay["slot_stride_bytes"]
    seen = []
    for i, t in enumerate([999.0, 979.0, 959.0, 939.0, 919.0, 899.0, 879.0]):
        base = cheb.cheb_cache_begin_push(h)
        assert base == FAKE_ARENA + (i % 4) * stride      # slots reused round robin
        cheb.cheb_cache_commit(h, t)
        seen.append(t)
        hist = cheb.cheb_cache_history(h)
        assert hist.tolist() == seen[-4:]
        for age in range(len(hist)):
            j = len(seen) - len(hist) + age            # push index of this entry
            assert cheb.cheb_cache_entry(h, age) == FAKE_ARENA + (j % 4) * stride
    cheb.cheb_cache_reset(h)
    assert cheb.cheb_cache_history(h).size == 0
    cheb.cheb_cache_destroy(h)


def test_not_ready_until_full_and_while_push_open():
    h, lay = _fake_cache(n_slots=3)
    out = FAKE_ARENA + 4 * lay["arena_bytes"]
    for t in [1.0, 2.0]:
        with pytest.raises(cheb.ChebError) as e:
            cheb.cheb_extrapolate(h, [0.2, 0.3, 0.5], out)
        assert e.value.code == B.CHEB_E_NOTREADY
        with pytest.raises(cheb.ChebError) as e:
            cheb.cheb_extrapolate_at(h, 9.0, out)
        assert e.value.code == B.CHEB_E_NOTREADY
        cheb.cheb_cache_begin_push(h)
        cheb.cheb_cache_commit(h, t)
    cheb.cheb_cache_begin_push(h)
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_extrapolate(h, [0.2, 0.3, 0.5], out)
    assert e.value.code == B.CHEB_E_NOTREADY
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_begin_push(h)
    assert e.value.code == B.CHEB_E_NOTREADY
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_push(h, 5.0, [FAKE_ARENA * 2, FAKE_ARENA * 3])
    assert e.value.code == B.CHEB_E_NOTREADY
    cheb.cheb_cache_commit(h, 3.0)
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_commit(h, 4.0)
    assert e.value.code == B.CHEB_E_NOTREADY
    cheb.cheb_cache_destroy(h)


def test_abort_push_keeps_the_other_entries():
    """An abandoned fused push records nothing; on a full ring the entry its
    slot held stays dropped, every other entry stays, and the ring goes on."""
    h, _ = _fake_cache(n_slots=3)
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_abort_push(h)
    assert e.value.code == B.CHEB_E_NOTREADY
    first = cheb.cheb_cache_begin_push(h)
    cheb.cheb_cache_abort_push(h)                     # not full: nothing changes
    assert cheb.cheb_cache_history(h).tolist() == []
    assert cheb.cheb_cache_begin_push(h) == first     # the same slot again
    cheb.cheb_cache_commit(h, 1.0)
    for t in (2.0, 3.0):
        cheb.cheb_cache_begin_push(h)
        cheb.cheb_cache_commit(h, t)
    slots = [cheb.cheb_cache_entry(h, k) for k in range(3)]
    oldest_slot = cheb.cheb_cache_begin_push(h)
    assert oldest_slot == slots[0]
    cheb.cheb_cache_abort_push(h)
    assert cheb.cheb_cache_history(h).tolist() == [2.0, 3.0]
    assert [cheb.cheb_cache_entry(h, k) for k in range(2)] == slots[1:]
    assert cheb.cheb_cache_begin_push(h) == oldest_slot
    cheb.cheb_cache_commit(h, 1.5)                    # 1.0 is gone, so any value but 2, 3
    assert cheb.cheb_cache_history(h).tolist() == [2.0, 3.0, 1.5]
    cheb.cheb_cache_destroy(h)


def test_duplicate_abscissa_rules():
    h, _ = _fake_cache(n_slots=3)
    for t in [10.0, 20.0, 30.0]:
        cheb.cheb_cache_begin_push(h)
        cheb.cheb_cache_commit(h, t)
    # Full: the next push drops 10, so 10 may come back but 20 may not.
    cheb.cheb_cache_begin_push(h)
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_commit(h, 20.0)
    assert e.value.code == B.CHEB_E_DUPNODE
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_commit(h, float("nan"))
    assert e.value.code == B.CHEB_E_NONFINITE
    cheb.cheb_cache_commit(h, 10.0)
    assert cheb.cheb_cache_history(h).tolist() == [20.0, 30.0, 10.0]
    cheb.cheb_cache_destroy(h)


def test_push_validation_before_launch():
    h, _ = _fake_cache(n_slots=2, seg=(1000, 24))
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_push(h, 1.0, [FAKE_ARENA * 2 + 8, FAKE_ARENA * 3])
    assert e.value.code == B.CHEB_E_ALIGN
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_push(h, 1.0, [0, FAKE_ARENA * 3])
    assert e.value.code == B.CHEB_E_INVAL
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_push(h, float("inf"), [FAKE_ARENA * 2, FAKE_ARENA * 3])
    assert e.value.code == B.CHEB_E_NONFINITE
    assert cheb.cheb_cache_history(h).size == 0     # nothing recorded
    cheb.cheb_cache_destroy(h)


def test_segment_offsets_and_slot_numel():
    h, lay = _fake_cache(n_slots=2, seg=(5, 17, 8))
    assert [cheb.cheb_cache_segment_offset(h, s) for s in range(3)] == lay["seg_offset"].tolist()
    assert cheb.cheb_cache_slot_numel(h) == lay["slot_numel"] == 8 + 24 + 8
    with pytest.raises(cheb.ChebError):
        cheb.cheb_cache_segment_offset(h, 3)
    with pytest.raises(cheb.ChebError):
        cheb.cheb_cache_entry(h, 0)
    cheb.cheb_cache_destroy(h)


def test_combine_validation_before_launch():
    a, b, o = FAKE_ARENA, FAKE_ARENA + (1 << 30), FAKE_ARENA + (2 << 30)
    cases = [
        (([a, b], [0.5, 0.5], o, 100, 7), B.CHEB_E_DTYPE),
        (([], [], o, 100, 0), B.CHEB_E_INVAL),
        (([a] * 9, [0.1] * 9, o, 100, 0), B.CHEB_E_INVAL),
        (([a + 2, b], [0.5, 0.5], o, 100, 0), B.CHEB_E_ALIGN),
        (([a, b], [0.5, 0.5], o + 4, 100, 0), B.CHEB_E_ALIGN),
        (([a, b], [0.5, float("nan")], o, 100, 0), B.CHEB_E_NONFINITE),
        (([a, b], [0.5, 1e39], o, 100, 0), B.CHEB_E_NONFINITE),     # past fp32 (bf16 path)
        (([a, b], [0.5, 0.5], a + 64, 100, 0), B.CHEB_E_INVAL),      # overlap
        (([a, b], [0.5, 0.5], o, -1, 0), B.CHEB_E_INVAL),
        (([a, b], [0.5, 0.5], o, 1 << 34, 0), B.CHEB_E_INVAL),
        (([a, 0], [0.5, 0.5], o, 100, 0), B.CHEB_E_INVAL),
    ]
    for args, code in cases:
        with pytest.raises(cheb.ChebError) as e:
            cheb.cheb_combine(*args)
        assert e.value.code == code, (args, e.value)
    cheb.cheb_combine([a, b], [0.5, 0.5], o, 0, 0)          # empty: no work, OK


def test_launch_config_roundtrip_and_validation():
    old = cheb.cheb_get_launch_config()
    assert old == {"block": 64, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 0,
                   "waves_per_cu": 0}
    assert old == cheb.DEFAULT_LAUNCH_CONFIG
    try:
        cheb.cheb_set_launch_config(256, 2, 0, 8, 12)
        assert cheb.cheb_get_launch_config() == {"block": 256, "unroll": 2, "nontemporal": 0,
                                                 "blocks_per_cu": 8, "waves_per_cu": 12}
        for w in (-1, 1, 32):
            cheb.cheb_set_launch_config(64, 1, 1, 0, w)
            assert cheb.cheb_get_launch_config()["waves_per_cu"] == w
        cheb.cheb_set_launch_config(256, 2, 0, 8, 12)
        for bad in [(256, 3, 1, 0), (256, 4, 2, 0), (256, 4, 1, -1), (256, 4, 1, 65),
                    (128, 1, 1, 0), (512, 4, 1, 0), (1024, 2, 1, 0), (64, 2, 1, 0),
                    (64, 1, 1, 0, -2), (64, 1, 1, 0, 33)]:
            with pytest.raises(cheb.ChebError):
                cheb.cheb_set_launch_config(*bad)
        assert cheb.cheb_get_launch_config()["block"] == 256     # unchanged by failures
    finally:
        cheb.cheb_set_launch_config(**old)


def test_combine_multi_validation_before_launch():
    a, b = FAKE_ARENA, FAKE_ARENA + (1 << 30)
    o1, o2 = FAKE_ARENA + (2 << 30), FAKE_ARENA + (3 << 30)
    w2 = [[0.5, 0.5], [-1.0, 2.0]]
    cases = [
        (([a, b], [[0.5, 0.5]] * 9, [o1 + (k << 28) for k in range(9)], 100, 0), B.CHEB_E_INVAL),
        (([a, b], w2, [o1, o1 + 64], 100, 0), B.CHEB_E_INVAL),         # outputs overlap
        (([a, b], w2, [o1, b + 32], 100, 0), B.CHEB_E_INVAL),          # output overlaps a source
        (([a, b], w2, [o1, o2 + 8], 100, 0), B.CHEB_E_ALIGN),
        (([a, b], [[0.5, 0.5], [np.inf, 0.0]], [o1, o2], 100, 0), B.CHEB_E_NONFINITE),
        (([a, b], w2, [o1, 0], 100, 0), B.CHEB_E_INVAL),
        (([a, b], w2, [o1, o2], 100, 9), B.CHEB_E_DTYPE),
    ]
    for args, code in cases:
        with pytest.raises(cheb.ChebError) as e:
            cheb.cheb_combine_multi(*args)
        assert e.value.code == code, (args, e.value)
    cheb.cheb_combine_multi([a, b], w2, [o1, o2], 0, 0)       # empty: no work


def test_extrapolate_multi_not_ready_and_limits():
    h, lay = _fake_cache(n_slots=2)
    outs = [FAKE_ARENA + (4 + k) * lay["arena_bytes"] for k in range(3)]
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_extrapolate_at_multi(h, [5.0, 6.0, 7.0], outs)
    assert e.value.code == B.CHEB_E_NOTREADY
    for t in [1.0, 2.0]:
        cheb.cheb_cache_begin_push(h)
        cheb.cheb_cache_commit(h, t)
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_extrapolate_multi(h, np.zeros((9, 2)), [outs[0]] * 9)
    assert e.value.code == B.CHEB_E_INVAL
    with pytest.raises(cheb.ChebError) as e:         # output inside the arena
        cheb.cheb_extrapolate_multi(h, np.ones((1, 2)), [FAKE_ARENA + 256])
    assert e.value.code == B.CHEB_E_INVAL
    with pytest.raises(cheb.ChebError) as e:         # duplicate of a held node is fine, NaN is not
        cheb.cheb_extrapolate_at_multi(h, [float("nan")], outs[:1])
    assert e.value.code == B.CHEB_E_NONFINITE
    cheb.cheb_cache_destroy(h)


# --------------------------------------------------------------------------
# Interleaved layout (host side: sizes, geometry, what it refuses)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,esize", [(B.CHEB_BF16, 2), (B.CHEB_F16, 2), (B.CHEB_F32, 4)])
def test_interleaved_arena_bytes(dtype, esize):
    seg = [1, 8, 13, 0, 1000003, 3, 4096 * 3072]
    _, pos, stride, arena = _expected_layout(5, esize, seg)
    assert cheb.cheb_cache_arena_bytes_ex(5, dtype, seg, B.CHEB_LAYOUT_SLOTS) == arena
    vecs = pos * esize // 16
    chunks = -(-vecs // 2048)
    assert cheb.cheb_cache_arena_bytes_ex(5, dtype, seg, B.CHEB_LAYOUT_INTERLEAVED) == \
        chunks * 5 * 32768 + 65536
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_arena_bytes_ex(5, dtype, seg, 2)
    assert e.value.code == B.CHEB_E_INVAL


def test_interleaved_create_geometry_and_refusals():
    seg = [40000, 24, 1 << 20]
    need = cheb.cheb_cache_arena_bytes_ex(6, B.CHEB_BF16, seg, B.CHEB_LAYOUT_INTERLEAVED)
    arena = FAKE_ARENA + 256          # 256-byte aligned, not on a 64 KiB boundary
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_create_ex(6, B.CHEB_BF16, seg, B.CHEB_LAYOUT_INTERLEAVED, arena, need - 1)
    assert e.value.code == B.CHEB_E_MISMATCH
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_create_ex(6, B.CHEB_BF16, seg, 7, arena, need)
    assert e.value.code == B.CHEB_E_INVAL
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_cache_create_ex(6, B.CHEB_BF16, seg, B.CHEB_LAYOUT_INTERLEAVED, arena + 16, need)
    assert e.value.code == B.CHEB_E_ALIGN
    h = cheb.cheb_cache_create_ex(6, B.CHEB_BF16, seg, B.CHEB_LAYOUT_INTERLEAVED, arena, need)
    try:
        assert cheb.cheb_cache_geometry(h) == (B.CHEB_LAYOUT_INTERLEAVED, 16384, 6 * 16384)
        with pytest.raises(cheb.ChebError) as e:
            cheb.cheb_cache_begin_push(h)       # a fused push needs contiguous slots
        assert e.value.code == B.CHEB_E_INVAL
        with pytest.raises(cheb.ChebError) as e:
            cheb.cheb_extrapolate(h, [1.0 / 6] * 6, FAKE_ARENA + (1 << 36), 0)
        assert e.value.code == B.CHEB_E_NOTREADY
    finally:
        cheb.cheb_cache_destroy(h)
    h = cheb.cheb_cache_create(6, B.CHEB_F32, seg, FAKE_ARENA,
                               cheb.cheb_cache_arena_bytes_ex(6, B.CHEB_F32, seg,
                                                              B.CHEB_LAYOUT_SLOTS))
    try:
        assert cheb.cheb_cache_geometry(h) == (B.CHEB_LAYOUT_SLOTS, 8192, 8192)
    finally:
        cheb.cheb_cache_destroy(h)
