"""Pins of the field-coupling oracle (oracle/field.py, Section 3.4's dynamics
variant): hand-worked rows, closed forms of degenerate coordinates, Section
7's saturated-kernel observation (tests/golden/field_section7.json), causality
and normalisation, the invariances of a distance kernel, and the backward
against central differences."""
import json
import os

import numpy as np
import pytest

from oracle import field
from paper_2609_18145_amd.inputs import make_field

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def rand_case(batch=2, n=9, c=3, width=5, seed=0, spread=1.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((batch, n, c)) * spread, rng.standard_normal((batch, n, width)),
            rng.standard_normal((batch, n, width)))


@pytest.mark.parametrize("tau", [1.0, 0.3, 2.5])
def test_two_points_scaled_is_independent_of_distance(tau):
    # Row 1 sees D = [d^2, 0]; its causal mean is d^2 / 2, so the logits are
    # [-2 / tau, 0] whatever d is.
    for d in (0.01, 1.0, 37.0):
        p = np.array([[[0.0, 0.0], [d * 0.6, d * 0.8]]])
        _, C, eff = field.forward(p, np.zeros((1, 2, 1)), tau, scaled=True)
        w = np.exp(-2.0 / tau)
        assert np.allclose(C[0, 1], [w / (1 + w), 1 / (1 + w)], rtol=1e-14)
        assert np.allclose(C[0, 0], [1.0, 0.0])
        assert eff[0, 0] == pytest.approx(1.0)


def test_two_points_unscaled():
    p = np.array([[[0.0], [1.5]]])
    _, C, _ = field.forward(p, np.zeros((1, 2, 1)), 0.5, scaled=False)
    w = np.exp(-2.25 / 0.5)
    assert np.allclose(C[0, 1], [w / (1 + w), 1 / (1 + w)], rtol=1e-14)


def test_three_points_by_hand():
    # Coordinates 0, 1, 3 on a line: row 2 has D = [9, 4, 0] and mean 13/3,
    # so its scaled logits are [-27/13, -12/13, 0] / tau.
    p = np.array([[[0.0], [1.0], [3.0]]])
    x = np.array([[[1.0, 0.0], [0.0, 1.0], [2.0, -1.0]]])
    tau = 0.8
    y, C, _ = field.forward(p, x, tau, scaled=True)
    e = np.exp(np.array([-27 / 13, -12 / 13, 0.0]) / tau)
    assert np.allclose(C[0, 2], e / e.sum(), rtol=1e-14)
    assert np.allclose(y[0, 2], (e[0] * x[0, 0] + e[1] * x[0, 1] + e[2] * x[0, 2]) / e.sum())
    # row 1: D = [1, 0], mean 1/2
    e1 = np.exp(np.array([-2.0, 0.0]) / tau)
    assert np.allclose(C[0, 1, :2], e1 / e1.sum(), rtol=1e-14)


@pytest.mark.parametrize("scaled", [True, False])
def test_equal_coordinates_give_causal_prefix_means(scaled):
    n, width = 7, 4
    p = np.full((1, n, 3), 2.5)
    x = np.random.default_rng(1).standard_normal((1, n, width))
    y, C, eff = field.forward(p, x, 1.0, scaled=scaled)
    for i in range(n):
        assert np.allclose(C[0, i, :i + 1], 1.0 / (i + 1))
        assert np.allclose(C[0, i, i + 1:], 0.0)
        assert np.allclose(y[0, i], x[0, :i + 1].mean(axis=0))
        assert eff[0, i] == pytest.approx(i + 1)


def test_unscaled_equally_spaced_line_is_a_discrete_gaussian():
    n, h, tau = 12, 0.7, 1.3
    p = (np.arange(n) * h).reshape(1, n, 1)
    _, C, _ = field.forward(p, np.zeros((1, n, 1)), tau, scaled=False)
    for i in range(n):
        k = np.arange(i, -1, -1)            # i - j for j = 0..i
        g = np.exp(-(k * h) ** 2 / tau)
        assert np.allclose(C[0, i, :i + 1], g / g.sum(), rtol=1e-13)


def test_section7_saturation_and_its_fix():
    with open(os.path.join(ROOT, "tests", "golden", "field_section7.json")) as f:
        g = json.load(f)
    u = g["unscaled_at_init"]
    inp = make_field(2, u["n"], 8, coord_dim=32, mean_sq_dist=u["mean_sq_dist"], seed=3)
    _, C, eff = field.forward(inp.p, inp.x, u["tau"], scaled=False)
    assert round(float(eff.mean()), 2) == u["effective_partners"]
    assert np.allclose(np.diagonal(C, axis1=1, axis2=2), 1.0, atol=1e-12)   # one-hot on self
    _, _, eff_s = field.forward(inp.p, inp.x, u["tau"], scaled=True)
    assert eff_s.mean() > 10 * u["effective_partners"]
    # the scaled form's partners grow with the causal row length
    assert eff_s[:, -1].mean() > 0.5 * u["n"]


@pytest.mark.parametrize("scaled", [True, False])
def test_rows_are_causal_distributions(scaled):
    p, x, _ = rand_case(n=11, seed=4)
    y, C, eff = field.forward(p, x, 0.9, scaled=scaled)
    assert np.all(C >= 0)
    assert np.allclose(C.sum(axis=2), 1.0)
    assert np.all(np.triu(C[0], 1) == 0) and np.all(np.triu(C[1], 1) == 0)
    idx = np.arange(11)
    assert np.all(eff >= 1 - 1e-12) and np.all(eff <= idx + 1 + 1e-9)
    # a later position's coordinates or values never reach an earlier row
    p2, x2 = p.copy(), x.copy()
    p2[:, 6:] += 5.0
    x2[:, 6:] *= -3.0
    y2, _, _ = field.forward(p2, x2, 0.9, scaled=scaled)
    assert np.allclose(y2[:, :6], y[:, :6], rtol=0, atol=0)
    assert not np.allclose(y2[:, 6:], y[:, 6:])


def test_distance_kernel_invariances():
    p, x, _ = rand_case(batch=1, n=10, c=4, seed=5)
    q, _ = np.linalg.qr(np.random.default_rng(6).standard_normal((4, 4)))
    t = np.array([3.0, -1.0, 0.5, 2.0])
    for scaled in (True, False):
        y, C, _ = field.forward(p, x, 0.7, scaled)
        _, C2, _ = field.forward(p @ q + t, x, 0.7, scaled)
        assert np.allclose(C2, C, rtol=1e-10, atol=1e-14)
    # the scaled form ignores the coordinates' scale; the unscaled one trades it for tau
    _, C, _ = field.forward(p, x, 0.7, True)
    _, C3, _ = field.forward(4.0 * p, x, 0.7, True)
    assert np.allclose(C3, C, rtol=1e-10, atol=1e-14)
    _, C, _ = field.forward(p, x, 0.7, False)
    _, C4, _ = field.forward(2.0 * p, x, 0.7 * 4.0, False)
    assert np.allclose(C4, C, rtol=1e-10, atol=1e-14)


def loss(p, x, dy, tau, scaled):
    y, _, _ = field.forward(p, x, tau, scaled)
    return float((y * dy).sum())


@pytest.mark.parametrize("scaled", [True, False])
def test_backward_matches_central_differences(scaled):
    p, x, dy = rand_case(batch=2, n=9, c=3, width=5, seed=7)
    tau = 0.7 if scaled else 3.0
    dp, dx = field.backward(p, x, dy, tau, scaled)
    h = 1e-6
    num_dp = np.zeros_like(p)
    for idx in np.ndindex(p.shape):
        a, b = p.copy(), p.copy()
        a[idx] += h
        b[idx] -= h
        num_dp[idx] = (loss(a, x, dy, tau, scaled) - loss(b, x, dy, tau, scaled)) / (2 * h)
    assert np.allclose(dp, num_dp, rtol=1e-6, atol=1e-7 * np.abs(num_dp).max())
    # y is linear in x: one-sided differences with a unit step are exact
    num_dx = np.zeros_like(x)
    base = loss(p, x, dy, tau, scaled)
    for idx in np.ndindex(x.shape):
        a = x.copy()
        a[idx] += 1.0
        num_dx[idx] = loss(p, a, dy, tau, scaled) - base
    assert np.allclose(dx, num_dx, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("scaled", [True, False])
def test_backward_invariants(scaled):
    p, x, dy = rand_case(batch=2, n=13, c=4, width=6, seed=8)
    dp, _ = field.backward(p, x, dy, 1.1, scaled)
    scale = np.abs(dp).max()
    # translation invariance: the coordinate gradient sums to zero
    assert np.allclose(dp.sum(axis=1), 0.0, atol=1e-12 * scale * 13)
    # rotation invariance: P^T dP is symmetric
    for t in range(2):
        m = p[t].T @ dp[t]
        assert np.allclose(m, m.T, atol=1e-10 * np.abs(m).max())
    if scaled:
        # scale invariance (Euler): sum_i p_i . dp_i = 0
        assert abs((p * dp).sum()) < 1e-10 * np.abs(p * dp).sum()


def test_degenerate_rows_have_zero_coordinate_gradient():
    # All coordinates equal: every scaled row is uniform with m = 0, and the
    # coupling does not depend on the coordinates there.
    p = np.zeros((1, 5, 2))
    x = np.random.default_rng(9).standard_normal((1, 5, 3))
    dy = np.random.default_rng(10).standard_normal((1, 5, 3))
    dp, dx = field.backward(p, x, dy, 1.0, True)
    assert np.all(dp == 0)
    C = np.tril(np.ones((5, 5))) / np.arange(1, 6)[:, None]
    assert np.allclose(dx[0], C.T @ dy[0])


def test_row_stats_closed_forms():
    # two points at distance d: m_1 = d^2 / 2 and ln Z_1 = ln(1 + exp(-2 / tau)) (scaled),
    # ln(1 + exp(-d^2 / tau)) (unscaled); row 0 always has m = 0 and ln Z = 0
    p = np.array([[[0.0, 0.0], [3.0, 4.0]]])
    m, lse = field.row_stats(p, 0.5, True)
    assert np.allclose(m[0], [0.0, 12.5]) and np.allclose(lse[0], [0.0, np.log1p(np.exp(-4.0))])
    m, lse = field.row_stats(p, 20.0, False)
    assert np.allclose(lse[0], [0.0, np.log1p(np.exp(-25.0 / 20.0))])
    # equal coordinates: m = 0, ln Z = ln(i + 1)
    m, lse = field.row_stats(np.ones((1, 6, 3)), 1.0, True)
    assert np.all(m == 0) and np.allclose(lse[0], np.log(np.arange(1, 7)))
