"""Property-based checks (hypothesis) of the host weights: the library
against the oracle on arbitrary distinct abscissae, partition of unity, and
exact reproduction of every polynomial of degree <= K; and the offline table
against the oracle's Algorithm-1 simulation on arbitrary schedules."""
import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import paper_2608_23429_amd as cheb
from paper_2608_23429_amd import _binding as B

SETTINGS = settings(max_examples=150, deadline=None,
                    suppress_health_check=[HealthCheck.too_slow])


def _spread(xs):
    xs = sorted(xs)
    return min(b - a for a, b in zip(xs, xs[1:])) if len(xs) > 1 else 1.0


nodes_st = st.lists(st.floats(-1e3, 1e3, allow_nan=False, allow_infinity=False),
                    min_size=1, max_size=8, unique=True).filter(
    lambda xs: _spread(xs) > 1e-2 * (max(xs) - min(xs) + 1e-9) and _spread(xs) > 1e-6)


def _cond(w):
    s = float(np.abs(w).sum())
    return s * max(s, 1.0)


# The library refuses a row once n 2^-53 sum|w| exceeds 2^-24.
LIMIT = 2.0 ** -24


def _weights_or_refusal(nodes, t):
    """The library's row, or None where it refused one; a refusal must come
    from a row the oracle also finds past the limit (up to a factor 2 for
    the two sides' own rounding)."""
    mass = float(np.abs(oracle.weights_row(nodes, t)).sum())
    load = len(nodes) * 2.0 ** -53 * mass
    try:
        w = cheb.cheb_precompute_weights(nodes, [t])[0]
    except cheb.ChebError as e:
        assert e.code == B.CHEB_E_NONFINITE
        assert not np.isfinite(mass) or load > LIMIT / 2, (nodes, t, mass)
        return None
    assert load <= 2 * LIMIT, (nodes, t, mass)
    return w


@SETTINGS
@given(nodes=nodes_st, t=st.floats(-3e3, 3e3, allow_nan=False, allow_infinity=False))
def test_library_weights_agree_with_oracle(nodes, t):
    w = _weights_or_refusal(nodes, t)
    if w is None:
        return
    ref = oracle.weights_row(nodes, t)
    assert np.max(np.abs(w - ref)) <= 64 * len(nodes) * 2.0 ** -53 * _cond(ref) + 1e-300
    assert abs(w.sum() - 1.0) <= 64 * len(nodes) * 2.0 ** -53 * _cond(w)


@SETTINGS
@given(nodes=nodes_st, t=st.floats(-3e3, 3e3, allow_nan=False, allow_infinity=False),
       seed=st.integers(0, 2 ** 31))
def test_polynomials_of_degree_at_most_K_reproduced(nodes, t, seed):
    rng = np.random.default_rng(seed)
    x = np.array(nodes)
    c = rng.standard_normal(len(nodes))             # degree len(nodes) - 1
    # evaluate in a centred, scaled frame so the values stay well conditioned
    mid, half = (x.max() + x.min()) / 2, max((x.max() - x.min()) / 2, 1.0)
    f = lambda z: np.polynomial.polynomial.polyval((z - mid) / half, c)
    w = _weights_or_refusal(nodes, t)
    if w is None:
        return
    got, want = w @ f(x), f(t)
    scale = np.abs(w) @ np.abs(f(x)) + abs(want)
    assert abs(got - want) <= 1e3 * len(nodes) * 2.0 ** -53 * max(_cond(w), 1.0) * max(scale, 1.0)


@settings(max_examples=60, deadline=None)
@given(T=st.integers(1, 40), s0=st.integers(0, 5), s1=st.integers(0, 5), r=st.integers(1, 7),
       n=st.integers(1, 8), policy=st.integers(0, 1))
def test_table_agrees_with_algorithm_one(T, s0, s1, r, n, policy):
    x = 999.0 - 23.0 * np.arange(T)
    t = cheb.ChebTable(T, s0, s1, r, n, x, policy)
    for s in range(T):
        pred, nodes, w = t.step(s)
        kind, onodes, ow = oracle.table_row(T, s0, s1, r, n, x, policy, s)
        assert pred == bool(kind) and nodes == onodes
        if pred:
            assert np.max(np.abs(w - ow)) <= 64 * n * 2.0 ** -53 * _cond(ow)


@SETTINGS
@given(nodes=nodes_st, t=st.floats(-3e3, 3e3, allow_nan=False, allow_infinity=False))
def test_taylor_weights_agree_with_oracle(nodes, t):
    """The Taylor-style row (explicit divided-difference products in the
    library, the recursive divided-difference table in the oracle)."""
    ref = oracle.weights_row_taylor(nodes, t)
    mass = float(np.abs(ref).sum())
    try:
        w = cheb.cheb_precompute_weights_variant(nodes, [t], cheb.CHEB_TAYLOR)[0]
    except cheb.ChebError as e:
        assert e.code == B.CHEB_E_NONFINITE
        assert not np.isfinite(mass) or len(nodes) * 2.0 ** -53 * mass > LIMIT / 2
        return
    assert np.max(np.abs(w - ref)) <= 64 * len(nodes) * 2.0 ** -53 * _cond(ref) + 1e-300
