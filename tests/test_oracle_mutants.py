"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's C source (a wrong
sign, a dropped term, a transposed or shifted index, a wrong rounding rule),
builds it with gcc into a temporary library, points the oracle's Python
binding at it and runs the pin battery of ``test_oracle_pins``; at least one
pin must fail.  All on the CPU; the real oracle is restored afterwards.
Planted mistakes keep every access in bounds, so a mutant fails a pin
rather than the process.
"""
import functools
import os
import tempfile

import pytest

import oracle
from oracle import build as oracle_build
from tests import test_oracle_pins as pins

# (name, text in oracle.c, replacement, which occurrence (0-based))
MUTANTS = [
    ("rho sign", "if (k != j) d *= (y[j] - y[k]);", "if (k != j) d *= (y[j] + y[k]);", 0),
    ("rho drops factors", "if (k != j) d *= (y[j] - y[k]);",
     "if (k > j) d *= (y[j] - y[k]);", 0),
    ("denominator drops a term", "denom += q[j];", "if (j > 0) denom += q[j];", 0),
    ("q multiplies", "q[j] = rho[j] / diff;", "q[j] = rho[j] * diff;", 0),
    ("target mirrored", "*ystar = (2.0 * xstar - (a + b)) / (b - a);",
     "*ystar = (2.0 * xstar - (a + b)) / (a - b);", 0),
    ("target shifted", "*ystar = (2.0 * xstar - (a + b)) / (b - a);",
     "*ystar = (2.0 * xstar - (a + a)) / (b - a);", 0),
    ("node hit picks wrong slot", "w[k] = (k == j) ? 1.0 : 0.0;",
     "w[k] = (k == 0) ? 1.0 : 0.0;", 0),
    ("history order reversed (bf16)", "double f = oracle_bf16_to_f64(F[k][i]);",
     "double f = oracle_bf16_to_f64(F[n - 1 - k][i]);", 0),
    ("newest entry dropped (bf16)", "for (int k = 0; k < n; ++k) {\n      double f = oracle_bf16",
     "for (int k = 0; k < n - 1; ++k) {\n      double f = oracle_bf16", 0),
    ("magnitude keeps sign", "m += fabs(w[k]) * fabs(f);", "m += w[k] * fabs(f);", 0),
    ("f32 decode drops oldest", "double f = (double)F[k][i];", "double f = (double)F[k ? k : 1][i];", 0),
    ("f64 sum uses wrong index", "for (int k = 0; k < n; ++k) s += w[k] * F[k][i];",
     "for (int k = 0; k < n; ++k) s += w[k] * F[k][i > 0 ? i - 1 : 0];", 0),
    ("bf16 decode shift", "uint32_t u = (uint32_t)h << 16;", "uint32_t u = (uint32_t)h << 15;", 0),
    ("ties to odd", "fmod(r, 2.0) != 0.0", "fmod(r, 2.0) == 0.0", 0),
    ("nine significand bits", "int qexp = (e < -126) ? -133 : e - 7;",
     "int qexp = (e < -126) ? -133 : e - 8;", 0),
    ("rounding truncates", "if (frac > 0.5 ||", "if (frac > 1.5 ||", 0),
    ("schedule end off by one", "(s > T - 1 - s1)", "(s > T - s1)", 0),
    ("schedule grid offset", "((s - s0) % r) == 0", "((s - s0 + 1) % r) == 0", 0),
    ("table keeps oldest", "for (int j = 1; j < n; ++j) hist[j - 1] = hist[j];",
     "for (int j = 1; j < n - 1; ++j) hist[j] = hist[j + 1];", 0),
    ("table ignores short-history policy", "(count < n && policy == 0)", "(count < n && policy == 1)", 0),
    ("residual drops x_in", "x_out[j] = x_in ? x_in[j] : 0.0;\n    if (absmag) absmag[j] = x_in ? fabs",
     "x_out[j] = 0.0;\n    if (absmag) absmag[j] = x_in ? fabs", 0),
    ("residual shifted target", "x_out[res_offset[s] + e] += acc;", "x_out[res_offset[s] + (e > 0 ? e - 1 : e)] += acc;", 0),
    ("residual magnitude drops x_in", "if (absmag) absmag[j] = x_in ? fabs(x_in[j]) : 0.0;\n  }\n  for (int s = 0; s < n_segs; ++s) {\n    if (res_offset[s] < 0) continue;\n#pragma omp parallel for schedule(static)\n    for (int64_t e = 0; e < seg_numel[s]; ++e) {\n      double acc = 0.0, mag = 0.0;\n      for (int k = 0; k < n; ++k) {\n        double f = oracle_bf16",
     "if (absmag) absmag[j] = 0.0;\n  }\n  for (int s = 0; s < n_segs; ++s) {\n    if (res_offset[s] < 0) continue;\n#pragma omp parallel for schedule(static)\n    for (int64_t e = 0; e < seg_numel[s]; ++e) {\n      double acc = 0.0, mag = 0.0;\n      for (int k = 0; k < n; ++k) {\n        double f = oracle_bf16", 0),
    ("alternating weights keep end halves off", "((j == 0 || j == n - 1) ? 0.5 : 1.0)",
     "((j == 0) ? 0.5 : 1.0)", 0),
    ("alternating weights without sign", "double rho = ((j % 2) ? -1.0 : 1.0)", "double rho = ((j % 2) ? 1.0 : 1.0)", 0),
    ("Chebyshev roots shifted", "cos((2.0 * j - 1.0) * pi / (2.0 * n))", "cos((2.0 * j) * pi / (2.0 * n))", 0),
    ("f16 exponent bias", "v = ldexp((double)(1024 + frac), expo - 25);",
     "v = ldexp((double)(1024 + frac), expo - 24);", 0),
    ("f16 subnormal scale", "v = ldexp((double)frac, -24);", "v = ldexp((double)frac, -25);", 0),
    ("f16 ties away from zero", "if (frac > 0.5 || (frac == 0.5 && fmod(r, 2.0) != 0.0)) r += 1.0;\n  const double rounded",
     "if (frac >= 0.5) r += 1.0;\n  const double rounded", 0),
    ("f16 overflow loses the sign", "if (rounded >= 65536.0) return (uint16_t)(sign | 0x7C00);",
     "if (rounded >= 65536.0) return (uint16_t)0x7C00;", 0),
    ("Taylor about the oldest node", "const double d = xstar - x[n - 1];", "const double d = xstar - x[0];", 0),
    ("Taylor divided difference over adjacent nodes only",
     "(table[k] - table[k - 1]) / (x[k] - x[k - i])", "(table[k] - table[k - 1]) / (x[k] - x[k - 1])", 0),
    ("Taylor drops the top order", "for (int i = 1; i < n; ++i) {\n      for (int k = n - 1; k >= i; --k)",
     "for (int i = 1; i < n - 1; ++i) {\n      for (int k = n - 1; k >= i; --k)", 0),
    ("table uses step not abscissa", "return oracle_weights_row(x, count, abscissa[s], w);",
     "return oracle_weights_row(x, count, abscissa[s] + 1.0, w);", 0),
    # one planted mistake in each storage type's own sum (the occurrences of
    # the sum line are the bf16, binary32 and binary16 versions, in that order)
    ("bf16 sum pairs weight k-1 with entry k", "s += w[k] * f;", "s += w[k > 0 ? k - 1 : 0] * f;", 0),
    ("f32 sum pairs weight k-1 with entry k", "s += w[k] * f;", "s += w[k > 0 ? k - 1 : 0] * f;", 1),
    ("f16 sum pairs weight k-1 with entry k", "s += w[k] * f;", "s += w[k > 0 ? k - 1 : 0] * f;", 2),
    ("f16 sum history reversed", "double f = oracle_f16_to_f64(F[k][i]);",
     "double f = oracle_f16_to_f64(F[n - 1 - k][i]);", 0),
    # the binary32 and binary16 residual checkers
    ("residual f32 drops x_in", "x_out[j] = x_in ? x_in[j] : 0.0;", "x_out[j] = 0.0;", 1),
    ("residual f32 reads the previous segment's slot", "double f = (double)F[k][slot_offset[s] + e];",
     "double f = (double)F[k][slot_offset[s > 0 ? s - 1 : s] + e];", 0),
    ("residual f16 decodes as bfloat16", "double f = oracle_f16_to_f64(F[k][slot_offset[s] + e]);",
     "double f = oracle_bf16_to_f64(F[k][slot_offset[s] + e]);", 0),
    ("residual f16 magnitude keeps the weight's sign", "mag += fabs(w[k]) * fabs(f);",
     "mag += w[k] * fabs(f);", 2),
    ("residual f16 skips the last covering segment", "for (int s = 0; s < n_segs; ++s) {\n    if (res_offset[s] < 0) continue;",
     "for (int s = 0; s < n_segs - 1; ++s) {\n    if (res_offset[s] < 0) continue;", 2),
]


def _battery():
    tests = []
    for name in sorted(dir(pins)):
        if not name.startswith("test_"):
            continue
        fn = getattr(pins, name)
        marks = [m for m in getattr(fn, "pytestmark", []) if m.name == "parametrize"]
        if marks:                       # one parameter: expand its values
            argname, values = marks[0].args[0], marks[0].args[1]
            for v in values:
                tests.append((f"{name}[{v!r}]", functools.partial(fn, **{argname: v})))
        else:
            tests.append((name, fn))
    return tests


def _replace_nth(text, old, new, n):
    start = -1
    for _ in range(n + 1):
        start = text.index(old, start + 1)
    return text[:start] + new + text[start + len(old):]


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda m: m[0])
def test_pins_catch_mutant(mutant, tmp_path):
    name, old, new, nth = mutant
    with open(oracle_build.SRC) as f:
        src = f.read()
    assert old in src, f"mutation site for {name!r} not found"
    mutated = _replace_nth(src, old, new, nth)
    path = os.path.join(tmp_path, "oracle_mutant.c")
    with open(path, "w") as f:
        f.write(mutated)
    lib = oracle_build.build(src=path, out=os.path.join(tmp_path, "liboracle_mutant.so"))
    saved = oracle.lib()
    oracle._LIB = oracle.bind(lib)
    caught = []
    try:
        for tname, fn in _battery():
            try:
                fn()
            except (AssertionError, oracle.OracleError, ValueError, ZeroDivisionError,
                    OverflowError):
                caught.append(tname)
                break
    finally:
        oracle._LIB = saved
    assert caught, f"no pin failed for planted mistake {name!r}"


def test_unmutated_oracle_passes_battery():
    for tname, fn in _battery():
        fn()
