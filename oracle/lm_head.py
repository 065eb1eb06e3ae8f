"""Token embedding, output head and cross-entropy of the language-model
workloads -- TEST INFRASTRUCTURE ONLY (CPU oracle, float64, plain definitions).

Section 5 trains character-level language models and reports held-out bits
per character, i.e. the mean cross-entropy of next-symbol prediction; the
model's symbols enter through an embedding table and leave through a linear
output head with a bias (the parameter counts of Section 5 include V w for the
table, V w + V for the head).  Written from those definitions:
  x[r]            = table[tokens[r]]
  dtable[v]       = sum of dx[r] over the rows r with tokens[r] == v
  logits[r]       = W x[r] + bias                 (W: [V][width])
  loss[r]         = log sum_v exp(logits[r][v]) - logits[r][targets[r]]
  dlogits[r][v]   = scale (softmax(logits[r])[v] - [v == targets[r]])
(scale = 1 / rows for the mean loss).  Only the tests, ``__graft_entry__``
and ``bench.py``'s CPU-baseline leg may use this module.
"""
from __future__ import annotations

import numpy as np


def embedding_forward(table, tokens):
    table = np.asarray(table, dtype=np.float64)
    return table[np.asarray(tokens)]


def embedding_backward(tokens, dx, vocab):
    tokens = np.asarray(tokens).reshape(-1)
    dx = np.asarray(dx, dtype=np.float64).reshape(tokens.size, -1)
    out = np.zeros((vocab, dx.shape[1]))
    for v in range(vocab):
        rows = tokens == v
        if rows.any():
            out[v] = dx[rows].sum(axis=0)
    return out


def head_cross_entropy(x, w, bias, targets, scale):
    """Returns (loss per row, dlogits) for rows of x ([rows][width])."""
    x = np.asarray(x, dtype=np.float64).reshape(-1, np.shape(w)[1])
    w = np.asarray(w, dtype=np.float64)
    targets = np.asarray(targets).reshape(-1)
    logits = x @ w.T + np.asarray(bias, dtype=np.float64)[None, :]
    m = logits.max(axis=1, keepdims=True)
    z = np.exp(logits - m).sum(axis=1, keepdims=True)
    lse = (m + np.log(z))[:, 0]
    rows = np.arange(x.shape[0])
    loss = lse - logits[rows, targets]
    d = np.exp(logits - lse[:, None])
    d[rows, targets] -= 1.0
    return loss, scale * d


def head_backward(x, w, dlogits):
    """The head's input and weight gradients for logits = W x + bias, given
    dlogits = d(loss)/d(logits): (dlogits W, dlogits^T x) (the chain rule
    through the linear map; Section 5's language models end in this head)."""
    x = np.asarray(x, dtype=np.float64).reshape(-1, np.shape(w)[1])
    w = np.asarray(w, dtype=np.float64)
    d = np.asarray(dlogits, dtype=np.float64).reshape(x.shape[0], -1)
    return d @ w, d.T @ x
