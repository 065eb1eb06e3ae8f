"""hcmix_stack_weight_gradients against the oracle: every layer's dW_self and
dW_off from independent seeded inputs and output gradients (the weight
gradients do not depend on the weights), through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_18145_amd import hcmix, inputs
from tests.util import fro_rel_err, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def draw(batch, n, width, num_layers, dtype, seed):
    rng = np.random.default_rng(seed)
    fin = (lambda a: inputs.round_bf16(a.astype(np.float32))) if dtype == "bf16" else \
        (lambda a: a.astype(np.float32))
    xs = [fin(rng.standard_normal((batch, n, width))) for _ in range(num_layers)]
    gs = [fin(rng.standard_normal((batch, n, width))) for _ in range(num_layers)]
    return xs, gs


def reference(xs, gs, layers, causal, width):
    zero = np.zeros((width, width), dtype=np.float32)
    dws, dwo = [], []
    for x, g, layer in zip(xs, gs, layers):
        _, a, b = oracle.backward(x, zero, zero, g, layer, causal)
        dws.append(a)
        dwo.append(b)
    return dws, dwo


# (batch, n, width, layers, causal, dtype): the full-tile launch (16 x 16
# tiles), the row-range launch with its fixed-order sum (5 layers of one
# tile), local layers, bidirectional, the per-layer kernels (width 192, fp32)
CASES = [
    (4, 256, 512, list(range(16)), True, "bf16"),
    (4, 256, 128, [0, 1, 2, 3, 4], True, "bf16"),
    (3, 64, 256, [oracle.NEAR, 5, oracle.NEAR, 2, 0, oracle.NEAR], True, "bf16"),
    (4, 128, 128, [6, 0, 3], False, "bf16"),
    (2, 64, 192, [0, 5, 3], True, "bf16"),
    (2, 16, 32, [0, 1, 2, 3], False, "f32"),
]


@pytest.mark.parametrize("batch,n,width,layers,causal,dtype", CASES)
def test_weight_gradients_match_oracle(batch, n, width, layers, causal, dtype):
    print(f"case: weight gradients B={batch} n={n} w={width} layers={layers} causal={causal} "
          f"{dtype}", flush=True)
    xs, gs = draw(batch, n, width, len(layers), dtype, seed=21)
    dws, dwo = hcmix.stack_weight_gradients([to_dev(a, dtype) for a in xs],
                                            [to_dev(a, dtype) for a in gs], layers, causal)
    torch.cuda.synchronize()
    rws, rwo = reference(xs, gs, layers, causal, width)
    tol = 1e-5 if dtype == "f32" else 1e-4     # exact inputs, fp32 accumulation
    err = max(max(fro_rel_err(to_host(a), b) for a, b in zip(dws, rws)),
              max(fro_rel_err(to_host(a), b) for a, b in zip(dwo, rwo)))
    print(f"  dW fro err {err:.3e}", flush=True)
    assert err <= tol


def test_weight_gradients_accumulate_and_repeat_bitwise():
    """accumulate adds to what the outputs hold; repeated calls are bitwise equal."""
    layers = [0, 1, 2, 3, 4]
    xs, gs = draw(4, 256, 128, len(layers), "bf16", seed=22)
    dxs = [to_dev(a, "bf16") for a in xs]
    dgs = [to_dev(a, "bf16") for a in gs]
    a_s, a_o = hcmix.stack_weight_gradients(dxs, dgs, layers, True)
    b_s, b_o = hcmix.stack_weight_gradients(dxs, dgs, layers, True)
    torch.cuda.synchronize()
    for p, q in zip(a_s + a_o, b_s + b_o):
        assert torch.equal(p, q)
    base = [t.clone() for t in a_s + a_o]
    hcmix.stack_weight_gradients(dxs, dgs, layers, True, dws=a_s, dwo=a_o, accumulate=True)
    torch.cuda.synchronize()
    for got, b in zip(a_s + a_o, base):
        assert torch.equal(got, 2 * b)      # x + x is exact
