"""Field coupling of the dynamics variant -- TEST INFRASTRUCTURE ONLY (CPU
oracle, float64, plain definitions).

Section 3.4 describes a variant in which every position i carries a
coordinate p_i, positions are coupled by a Gaussian of their squared
distance, exp(-||p_i - p_j||^2 / tau), and the scaled form ("field") divides
each squared distance by its causal row mean before the exponential.
Section 7 measures such couplings by their effective number of partners, the
exponential of each row's entropy.  Reading taken (the paper gives no
formula beyond these words):

    D[i][j] = ||p_i - p_j||^2                        for j <= i (causal)
    m[i]    = (1 / (i + 1)) * sum over j <= i of D[i][j]   (the causal row mean)
    a[i][j] = -D[i][j] / (tau * m[i])   (scaled; 0 for every j when m[i] = 0)
            = -D[i][j] / tau            (unscaled)
    C[i][j] = exp(a[i][j]) / sum over k <= i of exp(a[i][k]),  C[i][j] = 0 for j > i
    y_i     = sum over j <= i of C[i][j] x_j
    e_i     = exp(-sum over j of C[i][j] ln C[i][j])        (effective partners)

Rows are normalised: the paper's entropy of a row, and its observation that
an underflowing kernel collapses to a one-hot pointer, both need a
distribution per row.  The force that moves the coordinates, and the number
of repetitions T, belong to the model and are not specified: the
coordinates are an input, and T steps are T applications.

Backward (chain rule): dx_j = sum over i >= j of C[i][j] dy_i; through the
softmax, da[i][j] = C[i][j] (dy_i . x_j - dy_i . y_i); through the scaled
logits, dD[i][j] = -da[i][j] / (tau m[i]) + dm[i] / (i + 1) with
dm[i] = sum over j of da[i][j] D[i][j] / (tau m[i]^2); and dp_i collects
2 dD[i][j] (p_i - p_j) from its row and 2 dD[k][i] (p_i - p_k) from its
column.  Only the tests and bench.py's CPU-baseline leg may use this module.
"""
from __future__ import annotations

import numpy as np


def _window(p, x, tau, scaled):
    """One window: returns (y, C, D, m)."""
    n = p.shape[0]
    diff = p[:, None, :] - p[None, :, :]
    D = (diff * diff).sum(axis=2)
    mask = np.tril(np.ones((n, n), dtype=bool))
    counts = np.arange(1, n + 1, dtype=np.float64)
    m = np.where(mask, D, 0.0).sum(axis=1) / counts
    if scaled:
        with np.errstate(divide="ignore", invalid="ignore"):
            a = np.where(m[:, None] > 0, -D / (tau * m[:, None]), 0.0)
    else:
        a = -D / tau
    a = np.where(mask, a, -np.inf)
    a = a - a.max(axis=1, keepdims=True)
    e = np.exp(a)
    C = e / e.sum(axis=1, keepdims=True)
    y = C @ x
    return y, C, D, m


def forward(p, x, tau: float, scaled: bool = True):
    """p [batch, n, c], x [batch, n, width] -> (y [batch, n, width], C [batch, n, n],
    effective partners [batch, n])."""
    p = np.asarray(p, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    ys, Cs, effs = [], [], []
    for t in range(p.shape[0]):
        y, C, _, _ = _window(p[t], x[t], tau, scaled)
        with np.errstate(divide="ignore", invalid="ignore"):
            ent = -np.where(C > 0, C * np.log(C), 0.0).sum(axis=1)
        ys.append(y)
        Cs.append(C)
        effs.append(np.exp(ent))
    return np.stack(ys), np.stack(Cs), np.stack(effs)


def row_stats(p, tau: float, scaled: bool = True):
    """(m [batch, n], ln Z [batch, n]): each row's causal mean squared
    distance and the log of its softmax denominator sum over j <= i of
    exp(a[i][j]) (the row maximum is the diagonal's logit, 0)."""
    p = np.asarray(p, dtype=np.float64)
    ms, ls = [], []
    for t in range(p.shape[0]):
        n = p.shape[1]
        _, _, D, m = _window(p[t], np.zeros((n, 1)), tau, scaled)
        if scaled:
            with np.errstate(divide="ignore", invalid="ignore"):
                a = np.where(m[:, None] > 0, -D / (tau * m[:, None]), 0.0)
        else:
            a = -D / tau
        a = np.where(np.tril(np.ones((n, n), dtype=bool)), a, -np.inf)
        ms.append(m)
        ls.append(np.log(np.exp(a).sum(axis=1)))
    return np.stack(ms), np.stack(ls)


def backward(p, x, dy, tau: float, scaled: bool = True):
    """Returns (dp [batch, n, c], dx [batch, n, width])."""
    p = np.asarray(p, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    dps, dxs = [], []
    for t in range(p.shape[0]):
        pt, xt, gt = p[t], x[t], dy[t]
        n = pt.shape[0]
        y, C, D, m = _window(pt, xt, tau, scaled)
        dxs.append(C.T @ gt)
        dC = gt @ xt.T                                   # dy_i . x_j
        rowdot = (gt * y).sum(axis=1, keepdims=True)     # dy_i . y_i
        da = C * (dC - rowdot)
        if scaled:
            dD = np.zeros((n, n))
            for i in range(n):
                if m[i] > 0:
                    dm = (da[i, :i + 1] * D[i, :i + 1]).sum() / (tau * m[i] ** 2)
                    dD[i, :i + 1] = -da[i, :i + 1] / (tau * m[i]) + dm / (i + 1)
        else:
            dD = np.tril(-da / tau)
        diff = pt[:, None, :] - pt[None, :, :]          # p_i - p_j
        dp = 2.0 * (dD[:, :, None] * diff).sum(axis=1) - 2.0 * (dD[:, :, None] * diff).sum(axis=0)
        dps.append(dp)
    return np.stack(dps), np.stack(dxs)
