"""Writes scalar_map.txt: the singular-value map of the quintic NS step.

By the SVD argument (X X^T = U S^2 U^T, so (aI + bA + cA^2) X = U p(S) V^T),
each NS step sends every singular value x to p(x) = a x + b x^3 + c x^5
(Eq. 2).  This script composes p exactly with rational arithmetic starting
from x = 1 (the value every singular value of a rank-1 matrix takes after
Frobenius normalisation) and also writes the positive fixed points of p,
the roots of c y^2 + b y + (a - 1) = 0 with y = x^2.  It uses no code from
the oracle or the HIP library.
"""
from fractions import Fraction
import math
import os

A, B, C = Fraction("3.4445"), Fraction("-4.7750"), Fraction("2.0315")


def p(x):
    return A * x + B * x ** 3 + C * x ** 5


def main():
    lines = ["# quintic NS singular-value map, (a,b,c) = (3.4445, -4.7750, 2.0315)",
             "# k  p^{ok}(1)  (exact rational composition, printed to 17 significant digits)"]
    x = Fraction(1)
    for k in range(1, 6):
        x = p(x)
        lines.append(f"compose {k} {float(x):.17g}")
    disc = float(B * B - 4 * C * (A - 1))
    for sgn in (+1, -1):
        y = (-float(B) + sgn * math.sqrt(disc)) / (2 * float(C))
        lines.append(f"fixed_point {math.sqrt(y):.17g}")
    lines.append(f"derivative_at_0 {float(A):.17g}")
    lines.append(f"derivative_at_1 {float(A + 3 * B + 5 * C):.17g}")
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "scalar_map.txt")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
