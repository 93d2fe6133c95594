"""Exact rational Lagrange coefficients, from the plain definition.

l_j(x) = prod_{k != j} (x - x_k) / (x_j - x_k)  (paper, Appendix A, Lagrange
basis), evaluated in Python ``fractions`` on the exact binary values of the
given floats.  Pure-Python loops, for the small node counts of the method.
"""
from fractions import Fraction
from typing import List, Sequence


def lagrange_weights(nodes: Sequence[float], target: float) -> List[Fraction]:
    xs = [Fraction(v) for v in nodes]
    t = Fraction(target)
    out = []
    for j, xj in enumerate(xs):
        num = Fraction(1)
        den = Fraction(1)
        for k, xk in enumerate(xs):
            if k == j:
                continue
            num *= (t - xk)
            den *= (xj - xk)
        out.append(num / den)
    return out
