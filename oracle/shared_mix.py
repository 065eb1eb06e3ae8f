"""Channel-shared mixing layer -- TEST INFRASTRUCTURE ONLY (CPU oracle,
float64, plain definitions).

Reading taken (the paper gives no separate equation for it): the sparse
layer of Eq. (1) with both linear maps reduced to per-position scalars shared
by every channel, y_i = a_i x_i + b_i x_partner(i), the scalars being two
entries of an n x n table T_l per layer:

    y[t][i][c] = T[i][i] x[t][i][c] + m(i) T[i][p(i)] x[t][p(i)][c]

with the partner p and the mask m of Section 3.1 (hypercube layer: p = i XOR
2^d, causal m = bit d of i; local layer: p = i - 1, m = (i >= 1)).  So the
layer is the n x n table masked to the layer's links, applied along the
position axis, identically for every channel: y[t] = (M_l * T_l) x[t].  The
parameter totals of Section 5 (Table B2ecost, Table B1cost) are fitted exactly
by n^2 mixing parameters per layer, and the dense schedule there has the same
total as the sparse ones, i.e. it uses the whole table; that is what this
reading rests on.  Entries of T off the layer's links are never read, and
their gradient is zero.

Backward (chain rule; scatter form, each receiver pushing to its sender):
    dx[t][j][c]  = T[j][j] dy[t][j][c] + sum over receivers i of j of T[i][j] dy[t][i][c]
    dT[i][i]     = sum over (t, c) of dy[t][i][c] x[t][i][c]
    dT[i][p(i)]  = m(i) sum over (t, c) of dy[t][i][c] x[t][p(i)][c]
Only the tests and ``bench.py``'s CPU-baseline leg may use this module.
"""
from __future__ import annotations

import numpy as np

import oracle


def _links(n: int, layer: int, causal: bool):
    """(i, p(i), m(i)) of every position of one layer, from the main oracle's
    partner rule (Section 3.1)."""
    out = []
    for i in range(n):
        take = oracle.receives(i, layer, n, causal)
        assert take >= 0, (i, layer, n, causal)
        out.append((i, oracle.partner(i, layer, n), take))
    return out


def forward(x, table, layer: int, causal: bool) -> np.ndarray:
    """One channel-shared layer on x [batch, n, width]; table [n, n]."""
    x = np.asarray(x, dtype=np.float64)
    t = np.asarray(table, dtype=np.float64)
    n = x.shape[1]
    assert t.shape == (n, n)
    y = np.empty_like(x)
    for i, p, take in _links(n, layer, causal):
        y[:, i, :] = t[i, i] * x[:, i, :]
        if take:
            y[:, i, :] += t[i, p] * x[:, p, :]
    return y


def backward(x, table, dy, layer: int, causal: bool):
    """Adjoint of ``forward``: returns (dx, dT) with dT [n, n], zero off the
    layer's links."""
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    t = np.asarray(table, dtype=np.float64)
    n = x.shape[1]
    dx = np.zeros_like(x)
    dt = np.zeros((n, n))
    for i, p, take in _links(n, layer, causal):
        dx[:, i, :] += t[i, i] * dy[:, i, :]
        dt[i, i] = np.sum(dy[:, i, :] * x[:, i, :])
        if take:
            dx[:, p, :] += t[i, p] * dy[:, i, :]
            dt[i, p] = np.sum(dy[:, i, :] * x[:, p, :])
    return dx, dt


def stack_forward(x, tables, layers, causal: bool):
    """[x_0, x_1, ..., x_L] through the layers in order."""
    xs = [np.asarray(x, dtype=np.float64)]
    for t, layer in zip(tables, layers):
        xs.append(forward(xs[-1], t, layer, causal))
    return xs


def stack_backward(xs, tables, layers, dy, causal: bool):
    """Backward through the stack from the saved inputs xs[l]: (dx_0, [dT_l])."""
    g = np.asarray(dy, dtype=np.float64)
    dts = [None] * len(layers)
    for l in reversed(range(len(layers))):
        g, dts[l] = backward(xs[l], tables[l], g, layers[l], causal)
    return g, dts
