"""Writes abar_linear.txt: abar_t = prod_{i<=t} (1 - beta_i) for the linear schedule
beta_i = 0.00085 + (0.012 - 0.00085) * i / 999, i = 0..999, evaluated exactly with
rational arithmetic (fractions.Fraction) and rounded to 12 significant digits.

Independent of the oracle's NumPy schedule (no numpy, exact arithmetic)."""
from fractions import Fraction
import pathlib

T = 1000
b0, b1 = Fraction(85, 100000), Fraction(12, 1000)
want = [0, 1, 2, 100, 500, 901, 981, 999]
prod = Fraction(1)
vals = {}
for i in range(T):
    beta = b0 + (b1 - b0) * i / (T - 1)
    prod *= (1 - beta)
    if i in want:
        vals[i] = prod
lines = ["# t abar_t  (linear beta 0.00085..0.012, T=1000, exact rationals rounded to 12 sig. digits)"]
for t in want:
    lines.append(f"{t} {float(vals[t]):.12e}")
pathlib.Path(__file__).with_name("abar_linear.txt").write_text("\n".join(lines) + "\n")
