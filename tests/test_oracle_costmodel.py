"""Pins of the oracle's Eq. 9 cost model (Sec. 3.3, "Estimating t_fwd").

The fit is least squares of the context overhead t(i, j) - t(i, 0) on the
four terms 1, i, j, i j.  Pins that do not re-run the oracle's own solver:
exact recovery of coefficients from samples that lie on the model (the
minimum of a sum of squares is zero there), recovery from samples with
symmetric +/- perturbations (the perturbations cancel in the normal
equations), the orthogonality of the residual to every term (the defining
property of a least-squares minimiser), linearity in the measurements, and
the table layout rules (j = 0 entries are the measured t(i, 0); entries past
the sequence are -1).
"""
import itertools

import numpy as np
import pytest

from oracle import cost_table_from_model, fit_ctx_model

UNIT = 16
U = 32
COEF = (1500.0, 3.0, 7.0, 1.0 / 256)  # ns, ns/token, ns/token, ns/token^2 (exact on the grid)


def _t0(seed=0):
    rng = np.random.default_rng(seed)
    return [int(v) for v in 20000 + 900 * np.arange(1, U + 1) + rng.integers(0, 500, U)]


def _grid():
    pts = []
    for k in (1, 2, 4, 8, 12, 16, 24):
        for j in (1, 3, 6, 8, 12, 20):
            if k + j <= U:
                pts.append((k * UNIT, j * UNIT))
    return pts


def _model(i, j, c=COEF):
    return c[0] + c[1] * i + c[2] * j + c[3] * i * j


def test_exact_recovery_on_model_samples():
    t0 = _t0()
    # integer-valued overheads: choose points where the model is an integer
    samples = [(i, j, t0[i // UNIT - 1] + int(round(_model(i, j)))) for i, j in _grid()]
    for i, j, t in samples:
        assert t - t0[i // UNIT - 1] == _model(i, j)  # the grid keeps them exact
    coef = fit_ctx_model(t0, UNIT, samples)
    np.testing.assert_allclose(coef, COEF, rtol=1e-9, atol=1e-7)


def test_symmetric_perturbations_cancel():
    t0 = _t0(1)
    samples = []
    for n, (i, j) in enumerate(_grid()):
        d = 37 * (n % 5 + 1)
        base = t0[i // UNIT - 1] + _model(i, j)
        samples += [(i, j, base + d), (i, j, base - d)]
    coef = fit_ctx_model(t0, UNIT, samples)
    np.testing.assert_allclose(coef, COEF, rtol=1e-9, atol=1e-7)


def test_residual_orthogonal_to_every_term():
    t0 = _t0(2)
    rng = np.random.default_rng(3)
    samples = [(i, j, t0[i // UNIT - 1] + int(_model(i, j) + rng.normal(0, 300)))
               for i, j in _grid()]
    a = fit_ctx_model(t0, UNIT, samples)
    r = np.array([t - t0[i // UNIT - 1] - _model(i, j, a) for i, j, t in samples])
    for f in (lambda i, j: 1.0, lambda i, j: i, lambda i, j: j, lambda i, j: i * j):
        col = np.array([f(i, j) for i, j, _ in samples], float)
        assert abs(col @ r) <= 1e-7 * np.linalg.norm(col) * max(1.0, np.linalg.norm(r))
    # and it beats every nearby coefficient vector (a minimiser, not just a stationary point)
    def sse(c):
        return sum((t - t0[i // UNIT - 1] - _model(i, j, c)) ** 2 for i, j, t in samples)
    base = sse(a)
    for d in itertools.product((-1, 1), repeat=4):
        step = [1.0, 0.01, 0.01, 1e-5]
        assert sse([a[q] + d[q] * step[q] for q in range(4)]) > base


def test_linear_in_measurements():
    t0 = _t0(4)
    rng = np.random.default_rng(5)
    samples = [(i, j, t0[i // UNIT - 1] + int(_model(i, j) + rng.normal(0, 200)))
               for i, j in _grid()]
    a = fit_ctx_model(t0, UNIT, samples)
    shifted = [(i, j, t + 250 + 2 * j) for i, j, t in samples]  # overhead + 250 + 2 j
    b = fit_ctx_model(t0, UNIT, shifted)
    np.testing.assert_allclose(b, (a[0] + 250, a[1], a[2] + 2, a[3]), rtol=1e-9, atol=1e-6)


def test_degenerate_samples_rejected():
    t0 = _t0()
    samples = [(4 * UNIT, j * UNIT, t0[3] + 1000 * j) for j in range(1, 9)]  # one length only
    with pytest.raises(ValueError):
        fit_ctx_model(t0, UNIT, samples)


def test_table_layout():
    t0 = _t0(6)
    cost = cost_table_from_model(t0, UNIT, COEF)
    assert cost.shape == (U, U) and cost.dtype == np.int64
    for k in range(1, U + 1):
        assert cost[k - 1, 0] == t0[k - 1]
        for j in range(U):
            if k + j > U:
                assert cost[k - 1, j] == -1
            elif j > 0:
                assert cost[k - 1, j] == t0[k - 1] + round(_model(k * UNIT, j * UNIT))


def test_table_rounds_half_away_and_clamps():
    t0 = [100, 100, 100, 100]
    # overhead exactly 2.5 at (16, 16): a0 = 2.5, others 0 -> 103; -2.5 -> 97
    assert cost_table_from_model(t0, UNIT, (2.5, 0, 0, 0))[0, 1] == 103
    assert cost_table_from_model(t0, UNIT, (-2.5, 0, 0, 0))[0, 1] == 97
    # a negative total is clamped to 0
    assert cost_table_from_model(t0, UNIT, (-1e6, 0, 0, 0))[0, 1] == 0
