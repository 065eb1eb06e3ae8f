"""Pins of the hybrid-step oracle (oracle/hybrid.py): the chain rule through
sparse stacks, attention cores and linear maps, checked by central
differences of a scalar loss in float64 and by torch autograd of the same
composition written densely (every sparse layer as its n x n masked matrix)."""
import numpy as np
import torch

import oracle
from oracle import hybrid


def setup(seed=0, n=8, width=8, heads=2, hd=4):
    rng = np.random.default_rng(seed)
    schedule = [0, "attn", oracle.NEAR, 2, "attn", 1]
    ns = sum(1 for e in schedule if e != "attn")
    ws = [rng.standard_normal((width, width)) / np.sqrt(width) for _ in range(ns)]
    wo = [rng.standard_normal((width, width)) / np.sqrt(width) for _ in range(ns)]
    attn = [(rng.standard_normal((3 * heads * hd, width)) / np.sqrt(width),
             rng.standard_normal((width, heads * hd)) / np.sqrt(heads * hd)) for _ in range(2)]
    x = rng.standard_normal((2, n, width))
    g = rng.standard_normal((2, n, width))
    return schedule, ws, wo, attn, x, g, heads


def loss(x, schedule, ws, wo, attn, g, heads):
    y, _ = hybrid.forward(x, schedule, ws, wo, attn, heads)
    return float(np.sum(y * g))


def test_hybrid_backward_central_differences():
    schedule, ws, wo, attn, x, g, heads = setup()
    y, saved = hybrid.forward(x, schedule, ws, wo, attn, heads)
    dx, dws, dwo, dattn = hybrid.backward(saved, g, schedule, ws, wo, attn, heads)
    h = 1e-6

    def fd(mutate):
        plus, minus = mutate(h), mutate(-h)
        return (loss(*plus, heads) - loss(*minus, heads)) / (2 * h)

    def bump_x(idx):
        def m(e):
            xx = x.copy()
            xx[idx] += e
            return xx, schedule, ws, wo, attn, g
        return m
    for idx in [(0, 0, 0), (1, 5, 3), (0, 7, 7)]:
        assert abs(fd(bump_x(idx)) - dx[idx]) < 1e-6

    def bump_attn(a, t, idx):
        def m(e):
            at = [list(p) for p in attn]
            at[a][t] = at[a][t].copy()
            at[a][t][idx] += e
            return x, schedule, ws, wo, [tuple(p) for p in at], g
        return m
    for a, t, idx in [(0, 0, (3, 2)), (0, 1, (1, 6)), (1, 0, (20, 7)), (1, 1, (7, 0))]:
        assert abs(fd(bump_attn(a, t, idx)) - dattn[a][t][idx]) < 1e-6

    def bump_sparse(which, l, idx):
        def m(e):
            a = [w.copy() for w in (ws if which == 0 else wo)]
            a[l][idx] += e
            return (x, schedule, a, wo, attn, g) if which == 0 else (x, schedule, ws, a, attn, g)
        return m
    for which, l, idx in [(0, 0, (1, 2)), (1, 1, (4, 4)), (1, 3, (0, 7)), (0, 2, (6, 1))]:
        want = (dws if which == 0 else dwo)[l][idx]
        assert abs(fd(bump_sparse(which, l, idx)) - want) < 1e-6


def dense_mask(n, layer):
    m = np.zeros((n, n))
    for i in range(n):
        m[i, i] = 1.0
        if oracle.receives(i, layer, n, True):
            m[i, oracle.partner(i, layer, n)] = 1.0
    return m


def test_hybrid_matches_torch_autograd_of_a_dense_composition():
    """Each sparse layer as y[t] = X Ws^T + (Moff) X Wo^T with Moff the 0/1
    partner matrix of positions, attention through torch's own softmax; torch
    autograd in float64 gives every gradient."""
    schedule, ws, wo, attn, x, g, heads = setup(seed=3)
    n, width = x.shape[1], x.shape[2]
    y, saved = hybrid.forward(x, schedule, ws, wo, attn, heads)
    dx, dws, dwo, dattn = hybrid.backward(saved, g, schedule, ws, wo, attn, heads)
    T = lambda a: torch.tensor(a, dtype=torch.float64, requires_grad=True)   # noqa: E731
    tx, tws, two = T(x), [T(a) for a in ws], [T(a) for a in wo]
    tat = [(T(a), T(b)) for a, b in attn]
    h = tx
    sp = at = 0
    for e in schedule:
        if e == "attn":
            wq, wout = tat[at]
            hd = wq.shape[0] // (3 * heads)
            qkv = (h @ wq.T).reshape(2, n, 3, heads, hd)
            q, k, v = (qkv[:, :, j].transpose(1, 2) for j in range(3))
            s = q @ k.transpose(-1, -2) / hd ** 0.5
            s = s.masked_fill(torch.ones(n, n, dtype=torch.bool).triu(1), float("-inf"))
            o = (s.softmax(-1) @ v).transpose(1, 2).reshape(2, n, heads * hd)
            h = o @ wout.T
            at += 1
        else:
            moff = torch.tensor(dense_mask(n, e) - np.eye(n))
            h = h @ tws[sp].T + moff @ (h @ two[sp].T)
            sp += 1
    assert np.allclose(h.detach().numpy(), y, rtol=1e-12, atol=1e-12)
    (h * torch.tensor(g)).sum().backward()
    assert np.allclose(tx.grad.numpy(), dx, rtol=1e-10, atol=1e-12)
    for t, r in zip(tws + two, dws + dwo):
        assert np.allclose(t.grad.numpy(), r, rtol=1e-10, atol=1e-12)
    for (a, b), (ra, rb) in zip(tat, dattn):
        assert np.allclose(a.grad.numpy(), ra, rtol=1e-10, atol=1e-12)
        assert np.allclose(b.grad.numpy(), rb, rtol=1e-10, atol=1e-12)
