"""Writes tests/golden/wigner_d_exact.txt: Wigner d^l_{mn}(beta) at the angle
with cos(beta/2) = 3/5, sin(beta/2) = 4/5, from the textbook sum evaluated in
exact rational arithmetic (only the final square root is rounded).  Calls
only oracle/.  Run from the repository root:
    python tests/golden/make_wigner_golden.py
"""

import os
import sys
from fractions import Fraction

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
import oracle as O  # noqa: E402

CASES = []
for l in (0, 1, 2, 3, 7, 12, 20, 33, 47):
    for m in sorted({-l, -l // 2, -1, 0, 1, l // 3, l}):
        for n in sorted({-l, -2, -1, 0, 1, 2, l}):
            if abs(m) <= l and abs(n) <= l:
                CASES.append((l, m, n))

out = os.path.join(os.path.dirname(os.path.abspath(__file__)), "wigner_d_exact.txt")
with open(out, "w") as f:
    f.write("# Wigner d^l_{mn}(beta), cos(beta/2)=3/5, sin(beta/2)=4/5, convention\n")
    f.write("# d^1_{10}(beta) = -sin(beta)/sqrt(2).  Textbook sum (Wigner 1931;\n")
    f.write("# Sakurai, Modern Quantum Mechanics, eq. 3.8.33) in exact rationals.\n")
    f.write("# columns: l m n value\n")
    for l, m, n in CASES:
        v = O.wigner_d_sum_exact(l, m, n, Fraction(3, 5), Fraction(4, 5))
        f.write(f"{l} {m} {n} {v:.17e}\n")
print(out, len(CASES))
