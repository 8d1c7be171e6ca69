"""Coefficients of the GELU epilogue's complementary error function.

For a >= 0, erfc(a) = k * P(k) * exp(-a^2) with k = 1 / (1 + a / 2) and P a
degree-8 polynomial: P(k) approximates erfcx(a) / k, where erfcx(a) =
exp(a^2) erfc(a) is smooth and slowly varying on [0, inf) (it falls like
1 / (a sqrt(pi))), so a low-degree polynomial in k, which maps [0, inf) onto
(0, 1], fits it closely.  The fit is least squares in relative error on a
dense grid of [0, 10] (erfc(10) is far below the float32 range).

Run with no arguments to print the coefficients (constant term first) as
the kernel source holds them, and the largest relative error of erfc when
the formula is evaluated in float32 (Horner's rule, the square of a with its
exact residual as the kernel forms it) against SciPy's erfc on [0, 9.2].
"""
import numpy as np
from scipy.special import erfc, erfcx

P_SHIFT = 0.5
DEGREE = 8


def coefficients():
    a = np.concatenate([np.linspace(0.0, 1.0, 4000), np.linspace(1.0, 10.0, 20000)])
    k = 1.0 / (1.0 + P_SHIFT * a)
    target = erfcx(a) / k
    v = np.vander(k, DEGREE + 1, increasing=True)
    w = 1.0 / target
    c, *_ = np.linalg.lstsq(v * w[:, None], target * w, rcond=None)
    return c.astype(np.float32)


def erfc_f32(a32, c):
    f32 = np.float32
    k = (f32(1) / (f32(1) + f32(P_SHIFT) * a32)).astype(f32)
    p = np.full_like(a32, c[-1])
    for ci in c[-2::-1]:
        p = (p * k + ci).astype(f32)
    s = (a32 * a32).astype(f32)
    r = (a32.astype(np.float64) ** 2 - s.astype(np.float64)).astype(f32)  # fma(a, a, -s): exact
    e = np.exp(-s).astype(f32)
    e = (e - e * r).astype(f32)
    return (k * p * e).astype(f32)


if __name__ == "__main__":
    c = coefficients()
    print("constexpr float kErfcP[%d] = {%s};" % (len(c), ", ".join("%.9ef" % x for x in c)))
    a = np.linspace(0.0, 9.2, 400001).astype(np.float32)
    ref = erfc(a.astype(np.float64))
    print("max relative error of erfc in float32: %.2e" % float(np.max(np.abs(erfc_f32(a, c) - ref) / ref)))
