"""Pins of the attention oracle against what the definition fixes (closed
forms, invariances, causality) and against independent routines (torch
autograd in float64, central differences)."""
import numpy as np
import pytest
import torch

from oracle import attention


def rnd(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def test_zero_queries_give_the_prefix_mean():
    """Q = 0: every visible score is equal, so O[i] = mean(V[0..i]) and lse[i] = log(i + 1)."""
    B, n, H, hd = 2, 37, 3, 8
    qkv = rnd((B, n, 3, H, hd), 0)
    qkv[:, :, 0] = 0.0
    out, lse = attention.forward(qkv)
    v = qkv[:, :, 2]
    prefix = np.cumsum(v, axis=1) / np.arange(1, n + 1)[None, :, None, None]
    assert np.allclose(out, prefix, rtol=1e-12, atol=1e-12)
    assert np.allclose(lse, np.log(np.arange(1, n + 1))[None, None, :], rtol=0, atol=1e-12)


def test_one_distinguished_key_has_the_closed_form_weight():
    """Q[i] = a e_0 and K[j] = e_0 for one j* <= i, K[j] = 0 otherwise: the
    visible scores are a / sqrt(hd) at j* and 0 elsewhere, so
    O[i] = (e^t V[j*] + sum_{j != j*, j <= i} V[j]) / (e^t + i),  t = a / sqrt(hd)."""
    n, hd, a = 16, 4, 3.0
    for i, js in [(15, 4), (7, 7), (3, 0)]:
        qkv = np.zeros((1, n, 3, 1, hd))
        qkv[0, :, 2, 0] = rnd((n, hd), i)
        qkv[0, i, 0, 0, 0] = a
        qkv[0, js, 1, 0, 0] = 1.0
        out, _ = attention.forward(qkv)
        t = np.exp(a / np.sqrt(hd))
        v = qkv[0, :, 2, 0]
        want = (t * v[js] + v[:i + 1].sum(axis=0) - v[js]) / (t + i)
        assert np.allclose(out[0, i, 0], want, rtol=1e-12, atol=1e-12)


def test_softmax_rows_sum_to_one_and_keys_shift_invariance():
    B, n, H, hd = 1, 24, 2, 8
    qkv = rnd((B, n, 3, H, hd), 1)
    out, lse = attention.forward(qkv)
    q, k = qkv[:, :, 0], qkv[:, :, 1]
    for h in range(H):
        s = q[0, :, h] @ k[0, :, h].T / np.sqrt(hd)
        s[np.triu_indices(n, 1)] = -np.inf
        assert np.allclose(np.exp(s - lse[0, h][:, None]).sum(axis=1), 1.0, atol=1e-12)
    # adding one vector to every key shifts each query's scores by a constant
    shifted = qkv.copy()
    shifted[:, :, 1] += rnd((1, 1, H, hd), 2)
    out2, _ = attention.forward(shifted)
    assert np.allclose(out, out2, rtol=1e-10, atol=1e-10)


def test_causal_outputs_ignore_later_positions():
    B, n, H, hd = 1, 20, 2, 8
    qkv = rnd((B, n, 3, H, hd), 3)
    out, _ = attention.forward(qkv)
    for i in (0, 5, 13):
        pert = qkv.copy()
        pert[:, i + 1:] += rnd(pert[:, i + 1:].shape, 4)
        out2, _ = attention.forward(pert)
        assert np.array_equal(out[:, :i + 1], out2[:, :i + 1])


def torch_reference(qkv, dout):
    t = torch.tensor(qkv, dtype=torch.float64, requires_grad=True)
    q, k, v = (t[:, :, j].transpose(1, 2) for j in range(3))   # [B, H, n, hd]
    n, hd = q.shape[2], q.shape[3]
    s = torch.matmul(q, k.transpose(-1, -2)) / hd ** 0.5
    s = s.masked_fill(torch.ones(n, n, dtype=torch.bool).triu(1), float("-inf"))
    o = torch.matmul(torch.softmax(s, dim=-1), v).transpose(1, 2)
    o.backward(torch.tensor(dout, dtype=torch.float64))
    return o.detach().numpy(), t.grad.numpy()


@pytest.mark.parametrize("n,H,hd", [(17, 2, 8), (64, 3, 16)])
def test_forward_and_backward_match_torch_autograd(n, H, hd):
    B = 2
    qkv = rnd((B, n, 3, H, hd), 5)
    dout = rnd((B, n, H, hd), 6)
    o_ref, g_ref = torch_reference(qkv, dout)
    out, _ = attention.forward(qkv)
    assert np.allclose(out, o_ref, rtol=1e-12, atol=1e-12)
    assert np.allclose(attention.backward(qkv, dout), g_ref, rtol=1e-10, atol=1e-12)


def test_backward_matches_central_differences():
    B, n, H, hd = 1, 6, 1, 4
    qkv = rnd((B, n, 3, H, hd), 7)
    dout = rnd((B, n, H, hd), 8)
    g = attention.backward(qkv, dout)
    eps = 1e-6
    rng = np.random.default_rng(9)
    for _ in range(12):
        idx = tuple(rng.integers(0, s) for s in qkv.shape)
        a, b = qkv.copy(), qkv.copy()
        a[idx] += eps
        b[idx] -= eps
        fd = ((attention.forward(a)[0] - attention.forward(b)[0]) * dout).sum() / (2 * eps)
        assert abs(fd - g[idx]) <= 1e-7 * max(1.0, abs(fd))
