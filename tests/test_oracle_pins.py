"""Pins of the fp64 CPU oracle against what the paper and mathematics fix.

Nothing here compares the oracle with itself: each check goes through an
independent route (exact rational Lagrange coefficients, closed forms from
Appendix A, the interpolation error theorem, a textbook finite-difference
identity, format definitions checked by brute force, a library decoder).
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from synth import CONFIGS, make_history_f64, by_name
from tests.lagrange_exact import lagrange_weights

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _all_config_cases():
    for c in CONFIGS:
        yield c.name, c.nodes, c.targets
        if c.alt_nodes is not None:
            yield c.name + "_alt", c.alt_nodes, c.alt_targets


def _rand_nodes(rng, n, lo=-3.0, hi=5.0):
    while True:
        x = rng.uniform(lo, hi, size=n)
        if n == 1 or np.min(np.diff(np.sort(x))) > 1e-3 * (hi - lo):
            return x


def _wtol(w, factor=4.0):
    """Rounding bound for a weight row from the second barycentric form: the
    denominator cancels down to 1/omega(x), so each weight carries a relative
    error of order n u sum|w|, i.e. an absolute one of n u (sum|w|)^2."""
    s = float(np.abs(w).sum())
    return factor * len(w) * 2.0 ** -53 * s * max(s, 1.0)


# --------------------------------------------------------------------------
# Weights
# --------------------------------------------------------------------------

@pytest.mark.parametrize("case", list(_all_config_cases()), ids=lambda c: c[0])
def test_config_weights_equal_exact_lagrange(case):
    """Second barycentric form on normalised nodes == exact Lagrange basis."""
    _, nodes, targets = case
    w = oracle.weights(nodes, targets)
    for m, t in enumerate(targets):
        exact = lagrange_weights(nodes, t)
        scale = float(sum(abs(e) for e in exact))
        err = max(abs(w[m, j] - float(e)) for j, e in enumerate(exact))
        assert err <= 1e-13 * scale, (t, w[m], [float(e) for e in exact])
        assert sum(exact) == 1


def test_tiny_weights_exact_fractions():
    """Tiny workload, target 938: exact coefficients worked by hand from the
    Lagrange basis on nodes 999, 979, 959, 939 (spacing -20, target at
    offset 61/20 spacings): l_j = prod (3.05 - k) / (j - k)."""
    w = oracle.weights([999, 979, 959, 939], [938])[0]
    expect = [Fraction(-287, 16000), Fraction(1281, 16000), Fraction(-2501, 16000),
              Fraction(17507, 16000)]
    np.testing.assert_allclose(w, [float(e) for e in expect], rtol=0, atol=1e-15)


def test_random_weights_equal_exact_lagrange():
    rng = np.random.default_rng(7)
    for n in range(1, 9):
        for _ in range(20):
            x = _rand_nodes(rng, n)
            t = float(rng.uniform(-6, 8))
            w = oracle.weights_row(x, t)
            exact = lagrange_weights(x, t)
            scale = float(sum(abs(e) for e in exact))
            err = max(abs(w[j] - float(e)) for j, e in enumerate(exact))
            # The second form's denominator sum_j rho_j/(x - x_j) cancels down
            # to 1/omega(x); its relative rounding error, and so each weight's,
            # grows like u * sum|w|.
            assert err <= 4 * n * 2.0 ** -53 * scale * max(scale, 1.0), (n, x, t)


def test_partition_of_unity():
    """Appendix A: 1 = omega(x) sum_j rho_j / (x - x_j), i.e. sum_j w_j = 1."""
    rng = np.random.default_rng(11)
    for n in range(1, 9):
        for _ in range(50):
            x = _rand_nodes(rng, n)
            w = oracle.weights_row(x, float(rng.uniform(-10, 10)))
            assert abs(w.sum() - 1.0) <= _wtol(w)


def test_target_at_node_is_unit_vector():
    x = [0.96, 0.9, 0.8, 0.72, 0.6, 0.5]
    for j, xj in enumerate(x):
        w = oracle.weights_row(x, xj)
        assert w.tolist() == [1.0 if k == j else 0.0 for k in range(len(x))]


def test_single_node_is_reuse():
    """K = 0: the interpolant is the constant through the one cached value."""
    assert oracle.weights_row([500.0], 480.0).tolist() == [1.0]


def test_equispaced_rho_matches_appendix():
    """Appendix A: at equispaced nodes x_j = -1 + (j-1)h, h = 2/(N-1),
    omega'(x_j) = h^(N-1) (j-1)! (-1)^(N-j) (N-j)!, and after dropping the
    common factor rho_j = (-1)^(j-1) C(N-1, j-1) (golden table)."""
    rows = {}
    with open(os.path.join(GOLDEN, "equispaced_rho.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            vals = [int(v) for v in line.split()]
            rows[vals[0]] = vals[1:]
    assert sorted(rows) == list(range(1, 9))
    for N, golden in rows.items():
        if N == 1:
            continue
        h = 2.0 / (N - 1)
        y = np.array([-1.0 + (j - 1) * h for j in range(1, N + 1)])
        rho = oracle.barycentric_rho(y)
        closed = np.array([1.0 / (h ** (N - 1) * math.factorial(j - 1) * (-1) ** (N - j)
                                  * math.factorial(N - j)) for j in range(1, N + 1)])
        np.testing.assert_allclose(rho, closed, rtol=1e-13)
        ratio = rho / np.array(golden, dtype=np.float64)
        np.testing.assert_allclose(ratio, ratio[0], rtol=1e-13)


def test_normalisation_maps_span_to_unit_interval():
    y, ys = oracle.normalise([999, 979, 959, 939], 919)
    np.testing.assert_allclose(y, [1.0, 1 / 3, -1 / 3, -1.0], rtol=0, atol=1e-15)
    assert abs(ys - (-5 / 3)) < 1e-15
    y, ys = oracle.normalise([0.96, 0.9, 0.8, 0.72, 0.6, 0.5], 0.48)
    assert y.min() == -1.0 and y.max() == 1.0 and ys < -1.0


def test_one_step_ahead_equispaced_is_newton_difference():
    """Textbook: for K+1 equispaced nodes the degree-K extrapolant one spacing
    past the newest node has w_j = (-1)^(K-j) C(K+1, j) (the (K+1)-th forward
    difference of a degree-K polynomial vanishes)."""
    for K in range(0, 8):
        x = [999.0 - 20.0 * j for j in range(K + 1)]
        w = oracle.weights_row(x, 999.0 - 20.0 * (K + 1))
        expect = [(-1) ** (K - j) * math.comb(K + 1, j) for j in range(K + 1)]
        np.testing.assert_allclose(w, expect, rtol=0, atol=1e-12 * sum(map(abs, expect)))


def test_affine_invariance():
    """Lagrange coefficients do not depend on the affine frame of the nodes."""
    rng = np.random.default_rng(3)
    for n in range(2, 8):
        x = _rand_nodes(rng, n)
        t = float(rng.uniform(-6, 8))
        w = oracle.weights_row(x, t)
        for a, b in [(1000.0, 3.0), (-0.02, 1.0), (7.5, -250.0)]:
            w2 = oracle.weights_row(a * x + b, a * t + b)
            np.testing.assert_allclose(w2, w, rtol=0, atol=_wtol(w, 64.0))


def test_permutation_equivariance():
    rng = np.random.default_rng(5)
    for n in range(2, 8):
        x = _rand_nodes(rng, n)
        t = float(rng.uniform(-6, 8))
        w = oracle.weights_row(x, t)
        p = rng.permutation(n)
        np.testing.assert_allclose(oracle.weights_row(x[p], t), w[p], rtol=0,
                                   atol=_wtol(w, 16.0))


def test_lagrange_product_route_agrees():
    rng = np.random.default_rng(9)
    for n in range(1, 8):
        x = _rand_nodes(rng, n)
        t = float(rng.uniform(-6, 8))
        w = oracle.lagrange_row(x, t)
        np.testing.assert_allclose(oracle.weights_row(x, t), w, rtol=0, atol=_wtol(w, 16.0))


def test_bad_nodes_rejected():
    with pytest.raises(oracle.OracleError):
        oracle.weights_row([1.0, 2.0, 1.0], 3.0)
    with pytest.raises(oracle.OracleError):
        oracle.weights_row([1.0, float("nan")], 3.0)
    with pytest.raises(oracle.OracleError):
        oracle.weights_row([1.0, 2.0], float("inf"))
    with pytest.raises(oracle.OracleError):
        oracle.weights_row([], 3.0)


# --------------------------------------------------------------------------
# The combination
# --------------------------------------------------------------------------

def test_polynomials_up_to_degree_K_reproduced():
    """Appendix A error term f^(N)(xi)/N! omega(x) vanishes for degree <= N-1:
    every element's own random polynomial of degree <= K comes back exactly."""
    rng = np.random.default_rng(13)
    E = 4096
    for c in CONFIGS:
        x = np.array(c.nodes)
        for deg in range(0, c.K + 1):
            coef = rng.standard_normal((deg + 1, E))
            vals = np.stack([np.polynomial.polynomial.polyval(xk, coef) for xk in x])
            for t in c.targets:
                w = oracle.weights_row(x, t)
                got = oracle.extrapolate_f64(list(vals), w)
                want = np.polynomial.polynomial.polyval(t, coef)
                mag = np.abs(w) @ np.abs(vals)
                assert np.all(np.abs(got - want) <= 1e-12 * (mag + np.abs(want))), (c.name, deg, t)


def test_error_theorem_for_monomial_of_degree_N():
    """For f(x) = x^N with N nodes, f^(N)/N! = 1, so f(x) - P(x) = omega(x)."""
    rng = np.random.default_rng(17)
    for N in range(1, 8):
        x = _rand_nodes(rng, N, -1.0, 1.0)
        for t in rng.uniform(-2.5, 2.5, size=6):
            w = oracle.weights_row(x, t)
            P = oracle.extrapolate_f64([np.array([xk ** N]) for xk in x], w)[0]
            omega = float(np.prod(t - x))
            scale = np.abs(w) @ np.abs(x ** N) + abs(t) ** N + abs(omega)
            tol = _wtol(w, 16.0) * np.max(np.abs(x ** N)) + 16 * N * 2.0 ** -53 * scale
            assert abs((t ** N - P) - omega) <= tol, (N, t)


def test_tiny_generator_linearity():
    """Tiny workload: F_k = A + B tau_k + C tau_k^2 + 1e-3 eta_k (fp64, unrounded).
    The K=3 combination returns the quadratic at the target exactly plus the
    combined noise 1e-3 sum_k w_k eta_k."""
    c = by_name("tiny")
    E = 20000
    entries, coeffs, eta, taus = make_history_f64(c, E)
    for t in list(c.targets) + list(c.alt_targets):
        w = oracle.weights_row(c.nodes, t)
        got = oracle.extrapolate_f64(list(entries), w)
        tau = t / c.time_scale
        want = coeffs[0] + coeffs[1] * tau + coeffs[2] * tau * tau + c.noise_std * (w @ eta)
        mag = np.abs(w) @ np.abs(entries)
        assert np.all(np.abs(got - want) <= 1e-13 * (mag + 1.0))


def test_extrapolate_bf16_decodes_and_reports_magnitude():
    rng = np.random.default_rng(19)
    n, E = 6, 3001
    vals = rng.standard_normal((n, E)).astype(np.float32)
    bits = [torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
            for v in vals]
    dec = np.stack([torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).double().numpy()
                    for b in bits])
    w = oracle.weights_row([2, 5, 10, 14, 20, 25], 27)
    out, mag = oracle.extrapolate_bf16(bits, w)
    ref = np.zeros(E)
    for k in range(n):            # written out: oldest to newest, fp64
        ref = ref + w[k] * dec[k]
    np.testing.assert_array_equal(out, ref)
    np.testing.assert_allclose(mag, np.abs(w) @ np.abs(dec), rtol=1e-15)


def test_extrapolate_f32_exact_decode():
    rng = np.random.default_rng(23)
    vals = rng.standard_normal((4, 1000)).astype(np.float32)
    w = np.array([-1.0, 4.0, -6.0, 4.0])
    out, _ = oracle.extrapolate_f32(list(vals), w)
    ref = (((w[0] * vals[0].astype(np.float64)) + w[1] * vals[1].astype(np.float64))
           + w[2] * vals[2].astype(np.float64)) + w[3] * vals[3].astype(np.float64)
    np.testing.assert_array_equal(out, ref)


# --------------------------------------------------------------------------
# Storage formats
# --------------------------------------------------------------------------

def test_bf16_decode_all_patterns_matches_torch():
    bits = np.arange(65536, dtype=np.uint16)
    mine = oracle.bf16_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(mine), nan)
    assert np.array_equal(mine[~nan], ref[~nan])
    assert np.array_equal(np.signbit(mine[~nan]), np.signbit(ref[~nan]))


def _decode(b):
    return oracle.bf16_to_f64(np.array([b], dtype=np.uint16))[0]


def test_round_bf16_is_nearest_ties_to_even():
    """Brute force over neighbours: the chosen pattern is the nearest finite
    bfloat16, and on an exact tie it has an even last significand bit."""
    rng = np.random.default_rng(29)
    exps = rng.integers(-140, 128, size=3000)
    v = rng.uniform(1.0, 2.0, size=3000) * np.ldexp(1.0, exps) * rng.choice([-1, 1], 3000)
    ties = np.array([_decode(b) for b in range(0x3F80, 0x3F90)])
    mids = (ties[:-1] + ties[1:]) / 2            # exact midpoints
    v = np.concatenate([v, mids, -mids, [0.0, -0.0, 1e-50, 3.0e38, 3.4e38]])
    got = oracle.round_bf16(v)
    for x, b in zip(v, got):
        b = int(b)
        d = _decode(b)
        if math.isinf(d):
            assert abs(x) >= 3.3895313892515355e38  # past the largest finite + half ulp
            continue
        cand = [c for c in ((b - 1) & 0xFFFF, (b + 1) & 0xFFFF) if (c & 0x7F80) != 0x7F80]
        for c in cand:
            dc = _decode(c)
            assert abs(x - d) <= abs(x - dc), (x, hex(b), hex(c))
            if abs(x - d) == abs(x - dc) and dc != d:
                assert b % 2 == 0, (x, hex(b))
    # the midpoints between consecutive patterns go to the even one
    for m, lo in zip(mids, range(0x3F80, 0x3F8F)):
        assert int(oracle.round_bf16([m])[0]) == (lo if lo % 2 == 0 else lo + 1)


def test_round_bf16_agrees_with_torch_on_f32_inputs():
    """torch's float32 -> bfloat16 is round-to-nearest-even; for inputs that
    are already binary32 the single rounding must agree."""
    rng = np.random.default_rng(31)
    v32 = (rng.standard_normal(200000) * np.exp(rng.uniform(-30, 30, 200000))).astype(np.float32)
    mine = oracle.round_bf16(v32.astype(np.float64))
    ref = torch.from_numpy(v32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mine, ref)


def test_f16_decode_all_patterns_matches_numpy():
    bits = np.arange(65536, dtype=np.uint16)
    mine = oracle.f16_to_f64(bits)
    ref = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(mine), nan)
    assert np.array_equal(mine[~nan], ref[~nan])
    assert np.array_equal(np.signbit(mine[~nan]), np.signbit(ref[~nan]))
    # spot values from the format's definition
    assert oracle.f16_to_f64([0x3C00, 0x7BFF, 0x0001, 0x0400, 0xC000]).tolist() == \
        [1.0, 65504.0, 2.0 ** -24, 2.0 ** -14, -2.0]


def _decode16(b):
    return oracle.f16_to_f64(np.array([b], dtype=np.uint16))[0]


def test_round_f16_is_nearest_ties_to_even():
    """Brute force over neighbours: the chosen pattern is the nearest finite
    binary16 value, and on an exact tie it has an even last significand bit;
    values from 65520 up (the largest finite plus half its spacing) become
    infinity."""
    rng = np.random.default_rng(37)
    exps = rng.integers(-27, 17, size=3000)
    v = rng.uniform(1.0, 2.0, size=3000) * np.ldexp(1.0, exps) * rng.choice([-1, 1], 3000)
    ties = np.array([_decode16(b) for b in list(range(0x3C00, 0x3C10)) + list(range(0x0001, 0x0011))])
    mids = np.concatenate([(ties[:15] + ties[1:16]) / 2, (ties[16:-1] + ties[17:]) / 2])
    v = np.concatenate([v, mids, -mids, [0.0, -0.0, 1e-12, 65504.0, 65519.99, 65520.0, 7e4]])
    got = oracle.round_f16(v)
    for x, b in zip(v, got):
        b = int(b)
        d = _decode16(b)
        if math.isinf(d):
            assert abs(x) >= 65520.0
            continue
        cand = [c for c in ((b - 1) & 0xFFFF, (b + 1) & 0xFFFF) if (c & 0x7C00) != 0x7C00]
        for c in cand:
            dc = _decode16(c)
            assert abs(x - d) <= abs(x - dc), (x, hex(b), hex(c))
            if abs(x - d) == abs(x - dc) and dc != d:
                assert b % 2 == 0, (x, hex(b))
    for lo in list(range(0x3C00, 0x3C0F)) + list(range(0x0001, 0x0010)):
        m = (_decode16(lo) + _decode16(lo + 1)) / 2
        assert int(oracle.round_f16([m])[0]) == (lo if lo % 2 == 0 else lo + 1), hex(lo)


def test_round_f16_agrees_with_numpy():
    """numpy's float64 -> float16 conversion rounds to nearest even."""
    rng = np.random.default_rng(41)
    v = rng.standard_normal(200000) * np.exp(rng.uniform(-20, 12, 200000))
    with np.errstate(over="ignore"):
        ref = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(oracle.round_f16(v), ref)


# Storage encodings of small integers, made by torch and numpy (not by the
# oracle), with the round trip checked: the polynomial pins below need the
# stored values to be the integers themselves.
_INT_LIMIT = {"bf16": 256, "f16": 2048, "f32": 1 << 24}


def _encode_ints(vals, dtype):
    v = np.asarray(vals, dtype=np.int64)
    if dtype == "bf16":
        t = torch.from_numpy(v.astype(np.float32)).to(torch.bfloat16)
        assert torch.equal(t.double(), torch.from_numpy(v.astype(np.float64)))
        return t.view(torch.int16).numpy().view(np.uint16)
    if dtype == "f16":
        h = v.astype(np.float16)
        assert np.array_equal(h.astype(np.int64), v)
        return h.view(np.uint16)
    f = v.astype(np.float32)
    assert np.array_equal(f.astype(np.int64), v)
    return f


def _extrapolate(dtype, entries, w):
    fn = {"bf16": oracle.extrapolate_bf16, "f16": oracle.extrapolate_f16,
          "f32": oracle.extrapolate_f32}[dtype]
    return fn(entries, w)


def _integer_polynomials(rng, nodes, deg, count, limit):
    """Integer coefficient rows (count x (deg+1)) whose values at every node
    are integers of magnitude <= limit (rejection sampling), and those values
    (exact integer arithmetic)."""
    X = np.array([[int(x) ** d for d in range(deg + 1)] for x in nodes], dtype=np.int64)
    rows, vals = [], []
    while sum(len(r) for r in rows) < count:
        c = rng.integers(-4, 5, size=(4 * count, deg + 1))
        v = c @ X.T
        ok = np.all(np.abs(v) <= limit, axis=1)
        rows.append(c[ok])
        vals.append(v[ok])
    return np.concatenate(rows)[:count], np.concatenate(vals)[:count]


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_stored_polynomials_reproduced_by_each_storage_sum(dtype):
    """Appendix A error term: a polynomial of degree <= K is its own
    interpolant, so the prediction from K+1 stored node values is the
    polynomial's value at the target.  Integer polynomials whose node values
    are exact in the storage format; the expected value p(t) is Horner's rule
    on the integer coefficients, in exact rationals.  Through each storage
    type's own sum, equispaced and uneven integer nodes, degree up to K."""
    from fractions import Fraction
    rng = np.random.default_rng({"bf16": 101, "f16": 103, "f32": 107}[dtype])
    node_sets = [[0, 1], [-1, 0, 1], [-1, 0, 1, 2], [-2, -1, 0, 1, 2], [-3, -1, 0, 2],
                 [-2, -1, 0, 1, 2, 3], [-3, -2, 0, 1, 3]]
    for nodes in node_sets:
        K = len(nodes) - 1
        for deg in sorted({0, K // 2, K}):
            coef, vals = _integer_polynomials(rng, nodes, deg, 512, _INT_LIMIT[dtype])
            entries = [_encode_ints(vals[:, k], dtype) for k in range(K + 1)]
            for t in (max(nodes) + 1, max(nodes) + 2, max(nodes) + 0.5, min(nodes) - 1.5):
                w = oracle.weights_row(nodes, t)
                got, mag = _extrapolate(dtype, entries, w)
                ft = Fraction(t)
                want = np.array([float(sum(int(c) * ft ** d for d, c in enumerate(row)))
                                 for row in coef])
                tol = 64 * len(w) * 2.0 ** -53 * np.abs(w).sum() * (mag + np.abs(want)) + 1e-300
                assert np.all(np.abs(got - want) <= tol), (dtype, nodes, deg, t)


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_newton_weights_on_stored_cubics_exact(dtype):
    """Closed form with no weight computation: w = (-1, 4, -6, 4), the
    fourth forward difference of a cubic being zero, predicts p(4) from
    p(0..3) exactly for every integer cubic (all terms exact in fp64); the
    magnitude is sum_k |w_k| |p(k)|."""
    rng = np.random.default_rng(109)
    coef, vals = _integer_polynomials(rng, [0, 1, 2, 3], 3, 400, _INT_LIMIT[dtype])
    entries = [_encode_ints(vals[:, k], dtype) for k in range(4)]
    w = np.array([-1.0, 4.0, -6.0, 4.0])
    got, mag = _extrapolate(dtype, entries, w)
    want = coef @ np.array([1, 4, 16, 64])
    assert np.array_equal(got, want.astype(np.float64))
    assert np.array_equal(mag, (np.abs(vals) @ np.abs(w)).astype(np.float64))


def test_extrapolate_f16_decodes_exactly():
    rng = np.random.default_rng(43)
    vals = (rng.standard_normal((5, 2001)) * 3).astype(np.float16)
    bits = [v.view(np.uint16) for v in vals]
    w = oracle.weights_row([4, 8, 12, 16, 20], 21)
    out, mag = oracle.extrapolate_f16(bits, w)
    dec = vals.astype(np.float64)
    ref = np.zeros(vals.shape[1])
    for k in range(5):            # written out: oldest to newest, fp64
        ref = ref + w[k] * dec[k]
    np.testing.assert_array_equal(out, ref)
    np.testing.assert_allclose(mag, np.abs(w) @ np.abs(dec), rtol=1e-15)


# --------------------------------------------------------------------------
# Schedule
# --------------------------------------------------------------------------

def test_full_schedule_golden():
    with open(os.path.join(GOLDEN, "full_schedule.txt")) as f:
        lines = [l.split("#")[0].strip() for l in f]
    n = 0
    for line in lines:
        if not line:
            continue
        head, tail = line.split(":")
        kind, T, s0, s1, r = head.split()
        mask = oracle.full_schedule(int(T), int(s0), int(s1), int(r))
        if kind == "set":
            assert np.flatnonzero(mask).tolist() == [int(v) for v in tail.split()], line
        else:
            assert int(mask.sum()) == int(tail), line
        n += 1
    assert n == 9


def test_table_rows_golden():
    """The oracle's Algorithm-1 simulation against hand-worked rows; the
    coefficients of a predicted step are the (pinned) weights of its nodes."""
    with open(os.path.join(GOLDEN, "table_rows.txt")) as f:
        lines = [l.split("#")[0].strip() for l in f]
    n_cases = 0
    for line in lines:
        if not line:
            continue
        head, tail = line.split(":")
        T, s0, s1, r, n, policy = (int(v) for v in head.split())
        items = tail.split()
        assert len(items) == T
        x = 999.0 - 37.0 * np.arange(T)             # any distinct abscissae
        for s, item in enumerate(items):
            kind, nodes, w = oracle.table_row(T, s0, s1, r, n, x, policy, s)
            if item == "F":
                assert kind == 0 and nodes == [], (line, s)
            else:
                want = [int(v) for v in item.split("+")]
                assert kind == 1 and nodes == want, (line, s, nodes)
                exact = lagrange_weights(x[want], x[s])
                assert np.allclose(w, [float(e) for e in exact], rtol=0, atol=1e-12 * max(1, np.abs(w).sum()))
        n_cases += 1
    assert n_cases == 5


# --------------------------------------------------------------------------
# Residual application
# --------------------------------------------------------------------------

def _bf16_bits(vals):
    return torch.tensor(vals, dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_residual_hand_worked():
    """Two entries (w = [-1, 2]), a 4-element residual, three segments: the
    first adds everywhere, the second into elements 2..3, the third is not
    added.  Worked by hand from x_{l+1} = x_l + (module outputs)."""
    F0 = _bf16_bits([1, 2, 3, 4, 5, 6, 7, 8])
    F1 = _bf16_bits([1, 1, 1, 1, 2, 2, 2, 2])
    out, mag = oracle.residual([F0, F1], [-1.0, 2.0], slot_offset=[0, 4, 6],
                               seg_numel=[4, 2, 2], res_offset=[0, 2, -1], res_numel=4,
                               x_in=[10.0, 20.0, 30.0, 40.0])
    assert out.tolist() == [11.0, 20.0, 28.0, 36.0]
    assert mag.tolist() == [13.0, 24.0, 44.0, 56.0]


def test_residual_hand_worked_f32():
    """binary32 entries (values that need all 24 significand bits),
    w = [-1, 2], a 4-element residual: segment 0 (slot 0..3) adds at 0..3,
    segment 1 (slot 4..5) at 1..2, overlapping it, segment 2 (slot 6..9) is
    not added.  Per slot element p = -F0 + 2 F1:
        p0..p5 = 0, 0.5 + 2^-19, 4, 2 - 2^-22, 2, -6
    so x = [0, 2.5 + 2^-19, -2, 2 - 2^-22] without x_in; the magnitudes
    |F0| + 2|F1| are 1, 3.5 + 2^-19, 4, 8 + 2^-22, 22, 34."""
    u = 2.0 ** -22
    F0 = np.array([0.5, 1.5, -2.0, 3.0 + u, 10.0, 20.0, 99.0, 99.0, 99.0, 99.0], np.float32)
    F1 = np.array([0.25, 1.0 + 2.0 ** -20, 1.0, 2.5, 6.0, 7.0, 99.0, 99.0, 99.0, 99.0],
                  np.float32)
    assert float(F0[3]) == 3.0 + u and float(F1[1]) == 1.0 + 2.0 ** -20
    kw = dict(slot_offset=[0, 4, 6], seg_numel=[4, 2, 4], res_offset=[0, 1, -1], res_numel=4,
              dtype="f32")
    out, mag = oracle.residual([F0, F1], [-1.0, 2.0], **kw)
    assert out.tolist() == [0.0, 2.5 + 2.0 ** -19, -2.0, 2.0 - u]
    assert mag.tolist() == [1.0, 25.5 + 2.0 ** -19, 38.0, 8.0 + u]
    out, mag = oracle.residual([F0, F1], [-1.0, 2.0], x_in=[1.0, -1.0, 0.25, 100.0], **kw)
    assert out.tolist() == [1.0, 1.5 + 2.0 ** -19, -1.75, 102.0 - u]
    assert mag.tolist() == [2.0, 26.5 + 2.0 ** -19, 38.25, 108.0 + u]


def test_residual_hand_worked_f16():
    """binary16 entries with subnormals (2^-24, 3 * 2^-24), the smallest
    normal 2^-14, an 11-bit significand (1 + 2^-10) and the largest finite
    value 65504; three entries, w = [0.5, -1.5, 2]; segment 0 (slot 0..1)
    adds at residual 2..3, segment 1 (slot 2..5) at 0..3, residual element
    4 is covered by none.  Per slot element p = 0.5 F0 - 1.5 F1 + 2 F2:
        p0 = 2^-13 - 2^-22, p1 = 3 + 2^-11, p2 = 1, p3 = 1, p4 = 1.875,
        p5 = 31218,
    so x = [1, 1, 1.875 + 2^-13 - 2^-22, 31221 + 2^-11, 0]; the magnitudes
    0.5|F0| + 1.5|F1| + 2|F2| are 5 * 2^-24 + 2^-13, 6 + 2^-11, 7, 9, 2.625,
    34290."""
    bits = lambda v: np.array(v, dtype=np.uint16)
    F0 = bits([0x0001, 0x3C01, 0x4400, 0xC800, 0x3800, 0x7BFF])   # 2^-24, 1+2^-10, 4, -8, .5, 65504
    F1 = bits([0x0003, 0x3C00, 0x4000, 0xC000, 0x3400, 0x6400])   # 3*2^-24, 1, 2, -2, .25, 1024
    F2 = bits([0x0400, 0x4000, 0x3C00, 0x3C00, 0x3C00, 0x3C00])   # 2^-14, 2, 1, 1, 1, 1
    dec = [np.array(f).view(np.float16).astype(np.float64).tolist() for f in (F0, F1, F2)]
    assert dec[0] == [2.0 ** -24, 1 + 2.0 ** -10, 4.0, -8.0, 0.5, 65504.0]
    assert dec[1] == [3 * 2.0 ** -24, 1.0, 2.0, -2.0, 0.25, 1024.0]
    assert dec[2] == [2.0 ** -14, 2.0, 1.0, 1.0, 1.0, 1.0]
    kw = dict(slot_offset=[0, 2], seg_numel=[2, 4], res_offset=[2, 0], res_numel=5, dtype="f16")
    w = [0.5, -1.5, 2.0]
    out, mag = oracle.residual([F0, F1, F2], w, **kw)
    assert out.tolist() == [1.0, 1.0, 1.875 + 2.0 ** -13 - 2.0 ** -22, 31221.0 + 2.0 ** -11, 0.0]
    assert mag.tolist() == [7.0, 9.0, 2.625 + 5 * 2.0 ** -24 + 2.0 ** -13,
                            34296.0 + 2.0 ** -11, 0.0]
    x_in = [0.5, -0.5, 0.0, 2.0, 7.0]
    out, mag = oracle.residual([F0, F1, F2], w, x_in=x_in, **kw)
    assert out.tolist() == [1.5, 0.5, 1.875 + 2.0 ** -13 - 2.0 ** -22, 31223.0 + 2.0 ** -11, 7.0]
    assert mag.tolist() == [7.5, 9.5, 2.625 + 5 * 2.0 ** -24 + 2.0 ** -13,
                            34298.0 + 2.0 ** -11, 7.0]


def test_residual_single_segment_is_the_prediction():
    rng = np.random.default_rng(37)
    E = 5000
    F = [_bf16_bits(rng.standard_normal(E)) for _ in range(5)]
    w = oracle.weights_row([900, 820, 740, 660, 580], 560)
    out, mag = oracle.residual(F, w, [0], [E], [0], E)
    ref, rmag = oracle.extrapolate_bf16(F, w)
    np.testing.assert_array_equal(out, ref)
    np.testing.assert_array_equal(mag, rmag)


def test_residual_blocks_sum_and_order():
    """DiT-like mapping (every segment adds into the whole residual): the
    result is x_in plus the sum of the per-segment predictions, whatever the
    segment order; x_in enters linearly."""
    rng = np.random.default_rng(41)
    L, nseg, n = 777, 6, 4
    F = [_bf16_bits(rng.standard_normal(L * nseg)) for _ in range(n)]
    w = oracle.weights_row([999, 979, 959, 939], 919)
    so = np.arange(nseg) * L
    x_in = rng.standard_normal(L)
    out, _ = oracle.residual(F, w, so, [L] * nseg, [0] * nseg, L, x_in=x_in)
    parts = [oracle.extrapolate_bf16([f[o:o + L] for f in F], w, want_absmag=False) for o in so]
    ref = x_in + np.sum(parts, axis=0)
    assert np.max(np.abs(out - ref)) <= 1e-12 * (1 + np.max(np.abs(ref)))
    p = rng.permutation(nseg)
    out2, _ = oracle.residual(F, w, so[p], [L] * nseg, [0] * nseg, L, x_in=x_in)
    assert np.max(np.abs(out2 - out)) <= 1e-12 * (1 + np.max(np.abs(ref)))
    out0, _ = oracle.residual(F, w, so, [L] * nseg, [0] * nseg, L)
    assert np.max(np.abs((out - out0) - x_in)) <= 1e-12 * (1 + np.max(np.abs(ref)))


def test_residual_rejects_segment_outside():
    F = [_bf16_bits([1.0] * 8)]
    with pytest.raises(oracle.OracleError):
        oracle.residual(F, [1.0], [0], [8], [1], 8)


# --------------------------------------------------------------------------
# Node and weight variants (Section 3.2)
# --------------------------------------------------------------------------

def test_chebyshev_nodes_are_roots_and_extrema():
    """Kind 1 are the zeros of T_N, kind 2 the points where |T_{N-1}| = 1
    (checked with numpy's Chebyshev series evaluation)."""
    for N in range(2, 10):
        r = oracle.chebyshev_nodes(N, 1)
        assert np.max(np.abs(np.polynomial.chebyshev.chebval(r, [0] * N + [1]))) < 1e-14
        e = oracle.chebyshev_nodes(N, 2)
        assert np.allclose(np.abs(np.polynomial.chebyshev.chebval(e, [0] * (N - 1) + [1])), 1.0,
                           atol=1e-14)
        assert np.all(np.diff(r) < 0) and np.all(np.diff(e) < 0)
    x = oracle.chebyshev_nodes(5, 1, 200.0, 1000.0)
    assert np.allclose((x - 600.0) / 400.0, oracle.chebyshev_nodes(5, 1))


def test_general_weights_at_chebyshev_points_closed_forms():
    """Textbook closed forms of rho_j = 1/omega'(x_j): at the roots of T_N,
    proportional to (-1)^j sin((2j-1) pi / 2N); at the extrema, proportional
    to the alternating weights printed in Section 3.2."""
    for N in range(2, 10):
        x = oracle.chebyshev_nodes(N, 1)
        rho = oracle.barycentric_rho(x)
        cf = np.array([(-1) ** j * np.sin((2 * j - 1) * np.pi / (2 * N)) for j in range(1, N + 1)])
        ratio = rho / cf
        assert np.allclose(ratio, ratio[0], rtol=1e-12)
        e = oracle.chebyshev_nodes(N, 2)
        alt = np.array([(-1) ** j * (0.5 if j in (0, N - 1) else 1.0) for j in range(N)])
        ratio = oracle.barycentric_rho(e) / alt
        assert np.allclose(ratio, ratio[0], rtol=1e-12)
        for t in (1.3, -1.7, 0.123):
            np.testing.assert_allclose(oracle.weights_row_alternating(e, t),
                                       oracle.weights_row(e, t), rtol=0, atol=_wtol(oracle.weights_row(e, t), 64))


def test_alternating_weights_at_equispaced_nodes_reproduce_degree_one_only():
    """Reading of Section 3.2 against Appendix A: the printed alternating
    weights at equispaced nodes form a rational interpolant that reproduces
    constants and straight lines but not quadratics; Appendix A's general
    weights reproduce every degree up to N-1."""
    x = np.linspace(-1.0, 1.0, 6)
    rng = np.random.default_rng(43)
    for deg, exact in [(0, True), (1, True), (2, False), (3, False)]:
        c = rng.standard_normal(deg + 1)
        f = np.polynomial.polynomial.polyval(x, c)
        for t in (1.2, 1.5):
            err = abs(oracle.weights_row_alternating(x, t) @ f - np.polynomial.polynomial.polyval(t, c))
            assert (err < 1e-12) == exact, (deg, t, err)
            assert abs(oracle.weights_row(x, t) @ f - np.polynomial.polynomial.polyval(t, c)) < 1e-11
    assert oracle.weights_row_alternating(x, x[2]).tolist() == [0, 0, 1, 0, 0, 0]


def _taylor_by_backward_differences(x, t):
    """Textbook finite-difference Taylor polynomial about the newest of
    equispaced nodes, sum_i (nabla^i f)_newest / (i! h^i) (t - x_newest)^i,
    with the backward differences taken by numpy on each unit vector."""
    n = len(x)
    h = x[1] - x[0] if n > 1 else 1.0
    d = t - x[-1]
    w = np.zeros(n)
    for j in range(n):
        e = np.zeros(n)
        e[j] = 1.0
        w[j] = sum((np.diff(e, i)[-1] if i else e[-1]) / (math.factorial(i) * h ** i) * d ** i
                   for i in range(n))
    return w


def test_taylor_weights_equal_finite_difference_taylor_on_equispaced_nodes():
    for n in range(1, 9):
        for x0, h in [(0.0, 1.0), (999.0, -20.0), (0.96, -0.02), (-1.0, 2.0 / 7.0)]:
            x = x0 + h * np.arange(n)
            for t in (x[-1] + h, x[-1] + 2.5 * h, x[-1] - 0.5 * h, x[0]):
                got = oracle.weights_row_taylor(x, t)
                want = _taylor_by_backward_differences(x, t)
                assert np.max(np.abs(got - want)) <= 1e-12 * max(1.0, np.abs(want).sum()), (n, h, t)


def test_taylor_weights_closed_forms():
    """Any distinct nodes: constants and lines are reproduced; for f = x^2
    the expansion misses by exactly (t - x_K)(x_{K-1} - x_K) once three or
    more nodes are held; the newest node gets the unit row; two nodes give
    the Lagrange (linear) row; an affine map of nodes and target changes
    nothing."""
    rng = np.random.default_rng(47)
    for _ in range(200):
        n = int(rng.integers(1, 9))
        x = np.sort(rng.uniform(-3.0, 3.0, n))[::-1] if rng.random() < 0.5 else rng.uniform(-3.0, 3.0, n)
        if len(set(x.tolist())) < n or (n > 1 and np.min(np.abs(np.subtract.outer(x, x)) + np.eye(n)) < 0.05):
            continue
        t = float(rng.uniform(-5.0, 5.0))
        w = oracle.weights_row_taylor(x, t)
        scale = max(1.0, np.abs(w).sum())
        assert abs(w.sum() - 1.0) <= 1e-11 * scale
        if n >= 2:
            assert abs(w @ x - t) <= 1e-11 * scale * max(1.0, np.abs(x).max(), abs(t))
        if n >= 3:
            miss = w @ (x * x) - t * t
            want = (t - x[-1]) * (x[-2] - x[-1])
            assert abs(miss - want) <= 1e-10 * scale * max(1.0, np.abs(x).max(), abs(t)) ** 2, (n, miss, want)
        assert oracle.weights_row_taylor(x, x[-1]).tolist() == [0.0] * (n - 1) + [1.0]
        if n == 2:
            np.testing.assert_allclose(w, oracle.weights_row(x, t), rtol=0, atol=1e-12 * scale)
        a, b = 3.5, -1.25
        np.testing.assert_allclose(oracle.weights_row_taylor(a * x + b, a * t + b), w,
                                   rtol=0, atol=1e-10 * scale)


def test_table_mask_of_schedule_equals_schedule_rows():
    x = 999.0 - 37.0 * np.arange(20)
    mask = oracle.full_schedule(20, 2, 1, 4)
    for policy in (0, 1):
        for s in range(20):
            a = oracle.table_row(20, 2, 1, 4, 3, x, policy, s)
            b = oracle.table_row_mask(mask, 3, x, policy, s)
            assert a[0] == b[0] and a[1] == b[1] and np.array_equal(a[2], b[2])
