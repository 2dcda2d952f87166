"""The W1 CDF kernel evaluates Phi from a cubic Hermite table (step 1/64 on
[-8, 8], coefficients from erfc and the normal density) and recomputes with
erfc in double every grid point whose 16-bit quantised mixture value lies
within 1e-4 of a step (in units of 2^-16). That is exact only if the table's
error stays far inside the band: checked here against scipy's ndtr on a
dense sample of every interval, and at the ends, where Phi is replaced by 0
and 1."""
import math

import numpy as np
from scipy.special import ndtr

STEPS, Z = 64, 8.0
N = int(2 * Z * STEPS)
BAND = 1e-4


def table():
    h = 1.0 / STEPS
    z0 = -Z + np.arange(N) * h
    z1 = -Z + (np.arange(N) + 1) * h
    phi = np.vectorize(lambda z: 0.5 * math.erfc(-z / math.sqrt(2.0)))
    dphi = lambda z: h / math.sqrt(2.0 * math.pi) * np.exp(-0.5 * z * z)
    y0, y1, m0, m1 = phi(z0), phi(z1), dphi(z0), dphi(z1)
    return np.stack([y0, m0, 3 * (y1 - y0) - 2 * m0 - m1, 2 * (y0 - y1) + m0 + m1], axis=1)


def test_interpolation_error_is_far_inside_the_band():
    c = table()
    t = np.linspace(0.0, 1.0, 65)
    p = c[:, 0:1] + t * (c[:, 1:2] + t * (c[:, 2:3] + t * c[:, 3:4]))
    z = -Z + (np.arange(N)[:, None] + t[None, :]) / STEPS
    err = np.abs(p - ndtr(z)).max()
    assert err < 2e-10
    # a mixture has weights summing to 1: its error in units of 2^-16
    assert 65536 * err < BAND / 5


def test_tails_replaced_by_zero_and_one():
    assert 65536 * ndtr(-Z) < BAND / 1000
    assert 65536 * (1.0 - ndtr(Z)) < BAND / 1000
