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


def _stored_fp16_samples():
    """The 48 fp16 products measured on MI355X (profiles/), as rows of
    (m, n, k, flops, bytes, seconds)."""
    import os
    import re
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "profiles",
                        "calibration__matmul_mi355x.md")
    rows = []
    with open(path) as f:
        for line in f:
            m = re.match(r"\|\s*(\d+)\s*\|\s*(\d+)\s*\|\s*(\d+)\s*\|\s*([\d.e+-]+)\s*\|", line)
            if m:
                M, N, K = (int(m.group(i)) for i in (1, 2, 3))
                rows.append((M, N, K, 2 * M * N * K, 2 * (M * K + K * N + M * N), float(m.group(4))))
    return rows


def test_max_form_recovers_exact_coefficients():
    """Samples generated from a known max(floor, linear + c3 k) form, the
    floor binding on some of them, are fitted back with no error."""
    rng = np.random.default_rng(5)
    m, n, k = (rng.integers(16, 20000, 80) for _ in range(3))
    fl, by = 2.0 * m * n * k, 2.0 * (m * k + k * n + m * n)
    c = (3.0e-6, 5.0e-16, 2.0e-13, 2.5e-9, 4.0e-5)
    t = calibrate.predict(c, fl, by, k)
    assert np.any(t == c[4]) and np.any(t > c[4])
    got, worst = calibrate.fit_max(fl, by, k, t, tol=1e-9)
    assert worst < 1e-6
    assert all(v >= 0 for v in got)


def test_max_form_is_the_minimax_fit():
    """No coefficients found by a derivative-free search from many starts
    beat the bisection's worst relative error on the measured samples."""
    from scipy.optimize import minimize
    rows = _stored_fp16_samples()
    fl, by, k, t = (np.array([r[i] for r in rows], np.float64) for i in (3, 4, 2, 5))
    coef, worst = calibrate.fit_max(fl, by, k, t)
    scale = np.array([1e-5, 1e-15, 1e-13, 1e-9, 1e-5])

    def err(p):
        return np.max(np.abs(calibrate.predict(np.abs(p) * scale, fl, by, k) - t) / t)
    rng = np.random.default_rng(0)
    best = min(minimize(err, rng.uniform(0.1, 3.0, 5), method="Nelder-Mead",
                        options=dict(maxiter=6000, xatol=1e-9, fatol=1e-12)).fun for _ in range(12))
    assert worst <= best + 1e-4


def test_measured_fp16_products_within_a_quarter():
    """On the 48 products measured on MI355X the paper's linear form is off
    by up to 0.67; with the reduction length and the floor every product is
    within 0.25, in every shape class."""
    rows = _stored_fp16_samples()
    assert len(rows) == 48
    fl, by, k, t = ([r[i] for r in rows] for i in (3, 4, 2, 5))
    lin, worst_lin = calibrate.fit(fl, by, t)
    coef, worst = calibrate.fit_max(fl, by, k, t)
    assert worst_lin > 0.6 and worst <= 0.25
    assert max(calibrate.error_by_class(rows, coef).values()) <= 0.25
