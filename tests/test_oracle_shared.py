"""Pins of the channel-shared mixing oracle (oracle/shared_mix.py): the
paper's parameter totals (n^2 mixing parameters per layer), a dense masked
matrix product over positions built from a brute-force partner rule, the
reduction to Eq. (1) with scalar maps, closed forms of all-ones tables, and
the backward against torch autograd and central differences."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import shared_mix

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def totals():
    with open(os.path.join(ROOT, "tests", "golden", "paper_parameter_totals.json")) as f:
        return json.load(f)


def model_params(V, n, w, L, A, mixing_per_layer):
    """Token and position embeddings, a final normalisation, a head with bias,
    and per layer an MLP of hidden 2w with biases, two normalisations and the
    mixing parameters; 4 w^2 more per attention layer."""
    per_layer = 4 * w * w + 3 * w + 4 * w + mixing_per_layer
    return 2 * V * w + V + n * w + 2 * w + L * per_layer + A * 4 * w * w


def test_parameter_totals_fix_an_n_by_n_table_per_layer(totals):
    V = totals["vocab"]
    for key in ("window256_enwik8", "window64_repository"):
        g = totals[key]
        n, w, L = g["n"], g["width"], g["layers"]
        for form, rec in g["totals"].items():
            got = model_params(V[g["corpus"]], n, w, L, rec["attention_layers"], n * n)
            assert got == rec["weights"], (key, form, got)
            # the literal two width x width maps instead of the table do not fit
            alt = model_params(V[g["corpus"]], n, w, L, rec["attention_layers"], 2 * w * w)
            assert alt != rec["weights"]
    g = totals["window256_repository"]
    for form, rec in g["totals_millions"].items():
        got = model_params(V[g["corpus"]], g["n"], g["width"], g["layers"],
                           rec["attention_layers"], g["n"] ** 2)
        assert round(got / 1e6, 1) == rec["weights"], (form, got)


def brute_mask(n, layer, causal):
    """Link mask of one layer from a brute-force partner rule: add 2^d when bit
    d is clear, subtract it when set; the local layer links i to i - 1."""
    m = np.zeros((n, n))
    for i in range(n):
        m[i, i] = 1.0
        if layer == oracle.NEAR:
            if i >= 1:
                m[i, i - 1] = 1.0
            continue
        d = layer % int(np.log2(n))
        s = 1 << d
        up = (i // s) % 2 == 1
        j = i - s if up else i + s
        if not causal or up:
            m[i, j] = 1.0
    return m


CASES = [(16, 3, True), (16, 0, False), (64, 5, True), (64, oracle.NEAR, True), (8, 7, True),
         (32, 2, False)]


@pytest.mark.parametrize("n,layer,causal", CASES)
def test_forward_is_the_masked_table_along_positions(n, layer, causal):
    rng = np.random.default_rng(n + layer)
    x = rng.standard_normal((3, n, 5))
    t = rng.standard_normal((n, n))
    y = shared_mix.forward(x, t, layer, causal)
    dense = brute_mask(n, layer, causal) * t
    want = np.stack([dense @ x[b] for b in range(3)])     # library matmul over positions
    assert np.allclose(y, want, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("n,layer,causal", CASES)
def test_scalar_table_is_eq1_with_scaled_identities(n, layer, causal):
    """T[i][i] = a and T[i][p(i)] = c for every i (anything elsewhere) is Eq. (1)
    with W_self = a I and W_off = c I: the main oracle, pinned on its own."""
    rng = np.random.default_rng(7)
    w = 6
    x = rng.standard_normal((2, n, w))
    a, c = 0.75, -1.25
    mask = brute_mask(n, layer, causal)
    t = rng.standard_normal((n, n)) * 100.0            # entries off the links: never read
    t[mask > 0] = c
    t[np.arange(n), np.arange(n)] = a
    y = shared_mix.forward(x, t, layer, causal)
    want = oracle.forward(x, a * np.eye(w), c * np.eye(w), layer, causal)
    assert np.allclose(y, want, rtol=1e-13, atol=1e-12)


def test_all_ones_tables_give_the_subset_sums_and_the_window_sum():
    """Causal: one round of b rotated layers with an all-ones table sums, at
    position i, the inputs at the positions whose bits are a subset of i's
    (the causal XOR rule); bidirectional: every position gets the window sum."""
    n, b = 16, 4
    x = np.random.default_rng(3).integers(-5, 6, (2, n, 3)).astype(np.float64)
    ones = [np.ones((n, n))] * b
    y = shared_mix.stack_forward(x, ones, list(range(b)), True)[-1]
    for i in range(n):
        want = sum(x[:, j] for j in range(n) if j & i == j)
        assert np.array_equal(y[:, i], want)
    y = shared_mix.stack_forward(x, ones, list(range(b)), False)[-1]
    assert np.array_equal(y, np.broadcast_to(x.sum(axis=1, keepdims=True), x.shape))


@pytest.mark.parametrize("n,layer,causal", CASES)
def test_backward_matches_torch_autograd_of_the_dense_form(n, layer, causal):
    rng = np.random.default_rng(11 + n)
    x = rng.standard_normal((2, n, 4))
    t = rng.standard_normal((n, n))
    g = rng.standard_normal((2, n, 4))
    dx, dt = shared_mix.backward(x, t, g, layer, causal)
    tx = torch.tensor(x, requires_grad=True)
    tt = torch.tensor(t, requires_grad=True)
    m = torch.tensor(brute_mask(n, layer, causal))
    y = torch.einsum("ij,bjc->bic", m * tt, tx)
    (y * torch.tensor(g)).sum().backward()
    assert np.allclose(dx, tx.grad.numpy(), rtol=1e-12, atol=1e-12)
    assert np.allclose(dt, tt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_stack_backward_central_differences():
    n, L = 16, 5
    layers = [0, oracle.NEAR, 3, 1, 2]
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, n, 3))
    ts = [rng.standard_normal((n, n)) * 0.5 for _ in range(L)]
    g = rng.standard_normal((2, n, 3))

    def loss(x_, ts_):
        return float(np.sum(shared_mix.stack_forward(x_, ts_, layers, True)[-1] * g))

    xs = shared_mix.stack_forward(x, ts, layers, True)
    dx, dts = shared_mix.stack_backward(xs, ts, layers, g, True)
    h = 1e-6
    for (b, i, c) in [(0, 0, 0), (1, 7, 2), (0, 15, 1)]:
        xp, xm = x.copy(), x.copy()
        xp[b, i, c] += h
        xm[b, i, c] -= h
        assert abs((loss(xp, ts) - loss(xm, ts)) / (2 * h) - dx[b, i, c]) < 1e-6
    for l, (i, j) in [(0, (1, 0)), (1, (5, 4)), (2, (9, 1)), (4, (6, 6)), (3, (3, 2))]:
        tp = [t.copy() for t in ts]
        tm = [t.copy() for t in ts]
        tp[l][i, j] += h
        tm[l][i, j] -= h
        fd = (loss(x, tp) - loss(x, tm)) / (2 * h)
        assert abs(fd - dts[l][i, j]) < 1e-6, (l, i, j)
    # off the links the gradient is exactly zero
    for l in range(L):
        assert np.all(dts[l][brute_mask(n, layers[l], True) == 0] == 0)
