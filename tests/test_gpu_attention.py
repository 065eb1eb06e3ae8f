"""The HIP attention core against the attention oracle, through the C ABI.

Inputs are exact bf16 values; the kernel rounds P and dS to bf16 for its
second products (fp32 accumulation), so results are compared by relative
error: per row (one position and head, 64 values) for the output, and per
(window, head) Frobenius ratio for each of dQ, dK and dV, against the bf16
bound of the stack (2e-2)."""
import numpy as np
import pytest
import torch

from oracle import attention
from paper_2609_18145_amd import hcmix, inputs
from tests.util import to_dev, to_host

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def draw(batch, n, heads, seed, qk_scale=1.0):
    rng = np.random.default_rng(seed)
    qkv = rng.standard_normal((batch, n, 3, heads, 64))
    qkv[:, :, :2] *= qk_scale
    dout = rng.standard_normal((batch, n, heads, 64))
    return inputs.round_bf16(qkv.astype(np.float32)), inputs.round_bf16(dout.astype(np.float32))


def row_err(got, ref):
    g, r = got.reshape(-1, 64), ref.reshape(-1, 64)
    return float((np.linalg.norm(g - r, axis=1) / np.maximum(np.linalg.norm(r, axis=1), 1e-30)).max())


def grad_err(got, ref):
    """max over (window, head) and over Q, K, V of the Frobenius ratio."""
    worst = 0.0
    for b in range(ref.shape[0]):
        for h in range(ref.shape[3]):
            for t in range(3):
                g, r = got[b, :, t, h], ref[b, :, t, h]
                worst = max(worst, np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30))
    return worst


# (batch, n, heads, qk_scale): every tile count the kernels are built for, and
# sharper softmax rows (scores scaled up by 3)
CASES = [(2, 32, 3, 1.0), (2, 96, 2, 1.0), (2, 160, 2, 3.0), (1, 224, 1, 1.0), (2, 256, 3, 1.0),
         (2, 256, 2, 3.0), (3, 64, 4, 1.0), (1, 128, 2, 1.0), (1, 192, 1, 1.0)]


@pytest.mark.parametrize("batch,n,heads,qs", CASES)
def test_attention_matches_oracle(batch, n, heads, qs):
    print(f"case: attention B={batch} n={n} heads={heads} qk_scale={qs}", flush=True)
    qkv, dout = draw(batch, n, heads, seed=n + heads, qk_scale=qs)
    dq = to_dev(qkv, "bf16")
    out, lse = hcmix.attention_forward(dq)
    dqkv = hcmix.attention_backward(dq, out, lse, to_dev(dout, "bf16"))
    torch.cuda.synchronize()
    r_out, r_lse = attention.forward(qkv)
    r_g = attention.backward(qkv, dout)
    e_o = row_err(to_host(out), r_out)
    e_l = float(np.abs(to_host(lse) - r_lse).max())
    e_g = grad_err(to_host(dqkv), r_g)
    print(f"  out row err {e_o:.2e}  lse abs err {e_l:.2e}  grad fro err {e_g:.2e}", flush=True)
    assert e_o <= TOL
    assert e_l <= 1e-4 * max(1.0, float(np.abs(r_lse).max()))
    assert e_g <= TOL


def test_attention_full_hybrid_shape_sampled():
    """64 windows of 256 positions, 8 heads (the hybrid workload's attention
    layer) in one launch; four (window, head) pairs recomputed by the oracle."""
    batch, n, heads = 64, 256, 8
    qkv, dout = draw(batch, n, heads, seed=3)
    dq = to_dev(qkv, "bf16")
    out, lse = hcmix.attention_forward(dq)
    dqkv = hcmix.attention_backward(dq, out, lse, to_dev(dout, "bf16"))
    torch.cuda.synchronize()
    out, lse, dqkv = to_host(out), to_host(lse), to_host(dqkv)
    for b, h in [(0, 0), (17, 5), (40, 2), (63, 7)]:
        sl = qkv[b:b + 1, :, :, h:h + 1]
        r_out, r_lse = attention.forward(sl)
        r_g = attention.backward(sl, dout[b:b + 1, :, h:h + 1])
        assert row_err(out[b:b + 1, :, h:h + 1], r_out) <= TOL
        assert np.abs(lse[b:b + 1, h:h + 1] - r_lse).max() <= 1e-3
        assert grad_err(dqkv[b:b + 1, :, :, h:h + 1], r_g) <= TOL


def test_attention_never_looks_ahead():
    """Changing positions after i leaves every output at and before i bitwise equal."""
    qkv, _ = draw(2, 256, 2, seed=4)
    a = to_dev(qkv, "bf16")
    out_a, lse_a = hcmix.attention_forward(a)
    for i in (0, 31, 100, 254):
        pert = qkv.copy()
        pert[:, i + 1:] = inputs.round_bf16(
            np.random.default_rng(i).standard_normal(pert[:, i + 1:].shape).astype(np.float32))
        out_b, lse_b = hcmix.attention_forward(to_dev(pert, "bf16"))
        torch.cuda.synchronize()
        assert torch.equal(out_a[:, :i + 1], out_b[:, :i + 1])
        assert torch.equal(lse_a[:, :, :i + 1], lse_b[:, :, :i + 1])


def test_attention_autograd_function():
    qkv, dout = draw(2, 128, 2, seed=5)
    x = to_dev(qkv, "bf16").requires_grad_(True)
    y = hcmix.Attention.apply(x)
    y.backward(to_dev(dout, "bf16"))
    torch.cuda.synchronize()
    assert row_err(to_host(y), attention.forward(qkv)[0]) <= TOL
    assert grad_err(to_host(x.grad), attention.backward(qkv, dout)) <= TOL
