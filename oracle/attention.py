"""Causal multi-head softmax attention -- TEST INFRASTRUCTURE ONLY (CPU oracle).

The attention layers of the paper's hybrid schedules (Section 3.3: "standard
multi-head attention" replacing two layers of the local/jump backbone; the
window-256 hybrid of Appendix A keeps two among sixteen), written out from the
definition in float64 with numpy matrix products as the only library step.
Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use it; it shares nothing with the GPU library.

Layouts (those of the GPU entry points):
  qkv  [batch, n, 3, heads, head_dim]  -- Q, K, V of every position
  out  [batch, n, heads, head_dim]
  lse  [batch, heads, n]               -- log of each query row's softmax denominator
For one batch entry and head, with s = 1/sqrt(head_dim):
  S = s Q K^T with S[i, j] = -inf for j > i (a position sees itself and the past)
  P = row softmax of S,  O = P V,  lse[i] = log sum_j exp(S[i, j])
Backward (the chain rule through those three steps):
  dV = P^T dO,  dP = dO V^T,  dS = P * (dP - rowsum(dO * O)),
  dQ = s dS K,  dK = s dS^T Q.
"""
from __future__ import annotations

import numpy as np


def _split(qkv):
    qkv = np.asarray(qkv, dtype=np.float64)
    assert qkv.ndim == 5 and qkv.shape[2] == 3, "qkv must be [batch, n, 3, heads, head_dim]"
    return qkv[:, :, 0], qkv[:, :, 1], qkv[:, :, 2]


def _probs(q, k):
    """Scaled, masked scores of one (batch, head) and their row softmax."""
    n, hd = q.shape
    s = (q @ k.T) / np.sqrt(hd)
    s[np.triu_indices(n, 1)] = -np.inf
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    z = e.sum(axis=1, keepdims=True)
    return e / z, (m + np.log(z))[:, 0]


def forward(qkv):
    """Returns (out [batch, n, heads, head_dim], lse [batch, heads, n]) in float64."""
    q, k, v = _split(qkv)
    batch, n, heads, hd = q.shape
    out = np.empty((batch, n, heads, hd))
    lse = np.empty((batch, heads, n))
    for b in range(batch):
        for h in range(heads):
            p, lse[b, h] = _probs(q[b, :, h], k[b, :, h])
            out[b, :, h] = p @ v[b, :, h]
    return out, lse


def backward(qkv, dout):
    """Gradient of the loss with respect to qkv, given dout = dL/dout."""
    q, k, v = _split(qkv)
    dout = np.asarray(dout, dtype=np.float64)
    batch, n, heads, hd = q.shape
    dqkv = np.empty((batch, n, 3, heads, hd))
    s = 1.0 / np.sqrt(hd)
    for b in range(batch):
        for h in range(heads):
            qb, kb, vb, do = q[b, :, h], k[b, :, h], v[b, :, h], dout[b, :, h]
            p, _ = _probs(qb, kb)
            o = p @ vb
            dv = p.T @ do
            dp = do @ vb.T
            ds = p * (dp - (do * o).sum(axis=1, keepdims=True))
            dqkv[b, :, 0, h] = s * (ds @ kb)
            dqkv[b, :, 1, h] = s * (ds.T @ qb)
            dqkv[b, :, 2, h] = dv
    return dqkv
