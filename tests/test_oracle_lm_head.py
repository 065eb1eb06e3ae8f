"""Pins of the embedding / output-head / cross-entropy oracle: closed forms and
torch's own routines (embedding, linear, cross_entropy, autograd) in float64."""
import numpy as np
import torch
import torch.nn.functional as F

from oracle import lm_head


def test_uniform_logits_give_log_vocab():
    """w = 0, bias = 0: every logit is 0, so the loss is log V and the
    gradient is scale (1/V - onehot)."""
    rows, width, V = 7, 16, 256
    x = np.random.default_rng(0).standard_normal((rows, width))
    t = np.arange(rows) * 31 % V
    loss, d = lm_head.head_cross_entropy(x, np.zeros((V, width)), np.zeros(V), t, 0.5)
    assert np.allclose(loss, np.log(V), atol=1e-14)
    want = np.full((rows, V), 0.5 / V)
    want[np.arange(rows), t] -= 0.5
    assert np.allclose(d, want, atol=1e-15)


def test_bias_only_logits_are_a_fixed_distribution():
    """w = 0: the prediction is softmax(bias) for every row, loss = -log p[target]."""
    rows, width, V = 5, 8, 32
    bias = np.random.default_rng(1).standard_normal(V)
    t = np.array([0, 3, 31, 3, 17])
    loss, _ = lm_head.head_cross_entropy(np.ones((rows, width)), np.zeros((V, width)), bias, t, 1.0)
    p = np.exp(bias) / np.exp(bias).sum()
    assert np.allclose(loss, -np.log(p[t]), rtol=1e-13)


def test_embedding_backward_sums_rows_per_token():
    tokens = np.array([[3, 1, 3], [0, 3, 1]])
    dx = np.arange(6 * 4, dtype=np.float64).reshape(2, 3, 4)
    g = lm_head.embedding_backward(tokens, dx, 5)
    flat = dx.reshape(6, 4)
    assert np.array_equal(g[3], flat[0] + flat[2] + flat[4])
    assert np.array_equal(g[1], flat[1] + flat[5])
    assert np.array_equal(g[0], flat[3])
    assert not g[2].any() and not g[4].any()


def test_against_torch_autograd():
    rng = np.random.default_rng(2)
    rows, width, V = 40, 24, 256
    table = rng.standard_normal((V, width))
    tokens = rng.integers(0, V, rows)
    targets = rng.integers(0, V, rows)
    w = rng.standard_normal((V, width)) / np.sqrt(width)
    bias = rng.standard_normal(V) * 0.1
    tt = torch.tensor(table, requires_grad=True)
    tw = torch.tensor(w)
    x = F.embedding(torch.tensor(tokens), tt)
    xr = x.detach().requires_grad_(True)
    logits = F.linear(xr, tw, torch.tensor(bias)).requires_grad_(True)
    logits.retain_grad()
    loss = F.cross_entropy(logits, torch.tensor(targets), reduction="mean")
    loss.backward()
    x.backward(xr.grad)
    l_rows, d = lm_head.head_cross_entropy(lm_head.embedding_forward(table, tokens), w, bias,
                                           targets, 1.0 / rows)
    assert np.allclose(l_rows.mean(), loss.item(), rtol=1e-13)
    assert np.allclose(d, logits.grad.numpy(), rtol=1e-12, atol=1e-16)
    dx = d @ w
    assert np.allclose(lm_head.embedding_backward(tokens, dx, V), tt.grad.numpy(), rtol=1e-12,
                       atol=1e-14)


def test_head_backward_is_the_loss_gradient():
    """The head's input and weight gradients equal central differences of the
    mean cross-entropy (the loss itself, not the products), on a tiny head."""
    rng = np.random.default_rng(9)
    rows, width, vocab = 5, 6, 4
    x = rng.standard_normal((rows, width))
    w = rng.standard_normal((vocab, width)) * 0.5
    bias = rng.standard_normal(vocab) * 0.1
    targets = rng.integers(0, vocab, rows)
    scale = 1.0 / rows

    def mean_loss(xx, ww):
        return scale * lm_head.head_cross_entropy(xx, ww, bias, targets, scale)[0].sum()

    _, dlog = lm_head.head_cross_entropy(x, w, bias, targets, scale)
    gx, dw = lm_head.head_backward(x, w, dlog)
    h = 1e-6
    for arr, grad in ((x, gx), (w, dw)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + h
            up = mean_loss(x, w)
            arr[idx] = old - h
            down = mean_loss(x, w)
            arr[idx] = old
            num[idx] = (up - down) / (2 * h)
        assert np.abs(num - grad).max() <= 1e-8 * max(1.0, np.abs(num).max())
