"""The MatMul regression fit of the calibration tool (host-side: no GPU)."""
import numpy as np

from paper_2111_05426_amd import calibrate


def test_fit_recovers_exact_coefficients():
    """Samples generated from known non-negative coefficients are fitted
    back to within rounding."""
    rng = np.random.default_rng(3)
    m, n, k = (rng.integers(16, 20000, 60) for _ in range(3))
    fl, by = 2.0 * m * n * k, 2.0 * (m * k + k * n + m * n)
    c = (4.2e-6, 4.0e-16, 2.0e-13)
    t = c[0] + c[1] * fl + c[2] * by
    got, worst = calibrate.fit(fl, by, t)
    assert np.allclose(got, c, rtol=1e-6, atol=0) and worst < 1e-9


def test_fit_keeps_coefficients_non_negative():
    """A regression whose unconstrained optimum has a negative term is
    clipped to the best non-negative one (the device model needs c >= 0)."""
    fl = np.array([1e9, 2e9, 4e9, 8e9, 16e9])
    by = np.array([1e6, 1e6, 1e6, 1e6, 1e6])
    t = 1e-5 + 1e-13 * fl - 1e-12 * by   # a negative bytes term
    c, _ = calibrate.fit(fl, by, t)
    assert all(v >= 0 for v in c)
    pred = calibrate.design(fl, by) @ np.array(c)
    assert np.max(np.abs(pred - t) / t) < 0.05


def test_shapes_cover_the_models():
    s = calibrate.SHAPES
    assert len(s) == len(set(s)) >= 40
    assert min(m * n * k for m, n, k in s) < 1e7 < 1e12 < max(m * n * k for m, n, k in s)
