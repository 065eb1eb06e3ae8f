"""A hybrid stack's step -- TEST INFRASTRUCTURE ONLY (CPU oracle, float64).

Section 3.3's hybrid schedules keep a backbone of sparse layers and replace a
few of them with standard multi-head attention.  An attention layer here is
the attention core (oracle/attention.py) between two linear maps, the query /
key / value projection and the output projection:
    qkv = x W_qkv^T   (W_qkv [3 heads head_dim][width], the rows Q, K, V in turn)
    o   = attention(qkv)
    y   = o W_out^T   (W_out [width][heads head_dim])
with no residual, normalisation or bias, like the sparse layers (Eq. (1)).
The schedule is a list whose entries are sparse layer codes (run by the main
oracle, several in a row forming one stack) or the string "attn".  Backward:
the chain rule through the same steps, the linear maps' gradients being the
plain products dx = dy W and dW = dy^T x (numpy matrix products as the only
library step).  Only the tests may use this module.
"""
from __future__ import annotations

import numpy as np

import oracle
from oracle import attention


def linear_forward(x, w):
    """y = x W^T: x [rows, in], W [out, in]."""
    return np.asarray(x, dtype=np.float64) @ np.asarray(w, dtype=np.float64).T


def linear_backward(x, w, dy):
    """(dx, dW) of y = x W^T: dx = dy W, dW = dy^T x."""
    dy = np.asarray(dy, dtype=np.float64)
    return dy @ np.asarray(w, dtype=np.float64), dy.T @ np.asarray(x, dtype=np.float64)


def _segments(schedule):
    """Runs of sparse layers (lists of (sparse index, code)) and attention layers
    (their index), in order."""
    segs, cur, ns, na = [], [], 0, 0
    for e in schedule:
        if e == "attn":
            if cur:
                segs.append(("sparse", cur))
            segs.append(("attn", na))
            cur, na = [], na + 1
        else:
            cur.append((ns, e))
            ns += 1
    if cur:
        segs.append(("sparse", cur))
    return segs


def forward(x, schedule, w_self, w_off, attn_w, heads, causal=True):
    """Forward of the whole schedule; returns (y, saved) with saved the inputs
    each segment needs for the backward."""
    x = np.asarray(x, dtype=np.float64)
    batch, n, width = x.shape
    saved = []
    for kind, arg in _segments(schedule):
        if kind == "sparse":
            idx = [j for j, _ in arg]
            xs = oracle.stack_forward(x, [w_self[j] for j in idx], [w_off[j] for j in idx],
                                      [c for _, c in arg], causal)
            saved.append(xs)
            x = xs[-1]
        else:
            wqkv, wout = (np.asarray(t, dtype=np.float64) for t in attn_w[arg])
            hd = wqkv.shape[0] // (3 * heads)
            qkv = linear_forward(x.reshape(-1, width), wqkv).reshape(batch, n, 3, heads, hd)
            o, _ = attention.forward(qkv)
            o2 = o.reshape(-1, heads * hd)
            saved.append((x, qkv, o2))
            x = linear_forward(o2, wout).reshape(batch, n, -1)
    return x, saved


def backward(saved, dy, schedule, w_self, w_off, attn_w, heads, causal=True):
    """Returns (dx, dW_self per sparse layer, dW_off per sparse layer,
    [(dW_qkv, dW_out)] per attention layer)."""
    g = np.asarray(dy, dtype=np.float64)
    batch, n, width = g.shape
    segs = _segments(schedule)
    ns = sum(len(arg) for kind, arg in segs if kind == "sparse")
    dws, dwo = [None] * ns, [None] * ns
    dattn = [None] * len(attn_w)
    for (kind, arg), sv in zip(reversed(segs), reversed(saved)):
        if kind == "sparse":
            idx = [j for j, _ in arg]
            g, a, b = oracle.stack_backward(sv, [w_self[j] for j in idx], [w_off[j] for j in idx],
                                            [c for _, c in arg], g, causal)
            for k, j in enumerate(idx):
                dws[j], dwo[j] = a[k], b[k]
        else:
            x, qkv, o2 = sv
            wqkv, wout = (np.asarray(t, dtype=np.float64) for t in attn_w[arg])
            hd = wqkv.shape[0] // (3 * heads)
            d_o, d_wout = linear_backward(o2, wout, g.reshape(-1, width))
            dqkv = attention.backward(qkv, d_o.reshape(batch, n, heads, hd)).reshape(-1, 3 * heads * hd)
            g, d_wqkv = linear_backward(x.reshape(-1, width), wqkv, dqkv)
            g = g.reshape(batch, n, width)
            dattn[arg] = (d_wqkv, d_wout)
    return g, dws, dwo, dattn
