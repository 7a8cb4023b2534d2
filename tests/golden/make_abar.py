"""Writes the cumulative noise-schedule products abar_t = prod_{i<=t} (1 - beta_i) at
selected t, over T = 1000 training steps with beta_start = 0.00085, beta_end = 0.012:

* abar_linear.txt:        beta_i = b0 + (b1 - b0) * i / (T - 1), evaluated exactly with
                          rational arithmetic (fractions.Fraction);
* abar_scaled_linear.txt: beta_i = (sqrt(b0) + (sqrt(b1) - sqrt(b0)) * i / (T - 1))^2,
                          evaluated with decimal arithmetic at 60 significant digits
                          (the square roots are irrational; 1000 products lose far
                          fewer than the 48 digits kept beyond the 12 printed).

Both are rounded to 12 significant digits. Independent of the oracle's NumPy schedule
(no numpy, no oracle import)."""
from decimal import Decimal, getcontext
from fractions import Fraction
import pathlib

T = 1000
WANT = [0, 1, 2, 100, 500, 901, 981, 999]
HERE = pathlib.Path(__file__).parent


def write(name, header, vals):
    lines = [header] + [f"{t} {vals[t]:.12e}" for t in WANT]
    (HERE / name).write_text("\n".join(lines) + "\n")


def linear():
    b0, b1 = Fraction(85, 100000), Fraction(12, 1000)
    prod, vals = Fraction(1), {}
    for i in range(T):
        prod *= 1 - (b0 + (b1 - b0) * i / (T - 1))
        if i in WANT:
            vals[i] = float(prod)
    write("abar_linear.txt",
          "# t abar_t  (linear beta 0.00085..0.012, T=1000, exact rationals rounded to 12 sig. digits)", vals)


def scaled_linear():
    getcontext().prec = 60
    s0, s1 = Decimal("0.00085").sqrt(), Decimal("0.012").sqrt()
    prod, vals = Decimal(1), {}
    for i in range(T):
        r = s0 + (s1 - s0) * Decimal(i) / Decimal(T - 1)
        prod *= 1 - r * r
        if i in WANT:
            vals[i] = float(prod)
    write("abar_scaled_linear.txt",
          "# t abar_t  (scaled-linear beta (sqrt lerp)^2 0.00085..0.012, T=1000, 60-digit decimals rounded to 12 sig. digits)",
          vals)


if __name__ == "__main__":
    linear()
    scaled_linear()
