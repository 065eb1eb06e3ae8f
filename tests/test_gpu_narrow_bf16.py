"""bf16 widths that are a multiple of 8 but not of 64 (the boundary accepts
any multiple of 8; the MFMA tiles need 64, so these run on the fp32 FMA
kernels with bf16 storage): the local layer, whole stacks (rotated and mixa
schedules, causal and bidirectional), the backward's data chain and weight
gradients on their own, the decode step and the no-allocation backward,
against the oracle or bitwise against the entry point they must equal.  The
single-layer probe and parity cases at these widths are in test_gpu_layer."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_18145_amd import hcmix, inputs
from tests.util import TOL, fro_rel_err, row_rel_err, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def log(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("width", [24, 136])
def test_local_layer(width):
    batch, n = 3, 32
    log(f"case: local layer bf16 B={batch} n={n} w={width}")
    x, ws, wo, dy = inputs.make_layer(batch, n, width, "bf16", seed=width)
    tx, tws, two, tdy = (to_dev(a, "bf16") for a in (x, ws, wo, dy))
    y = hcmix.forward(tx, tws, two, hcmix.LAYER_NEAR, True)
    dx, dws, dwo = hcmix.backward(tx, tws, two, tdy, hcmix.LAYER_NEAR, True)
    torch.cuda.synchronize()
    ry = oracle.forward(x, ws, wo, oracle.NEAR, True)
    rdx, rws, rwo = oracle.backward(x, ws, wo, dy, oracle.NEAR, True)
    assert row_rel_err(to_host(y), ry) <= TOL["bf16"]
    assert row_rel_err(to_host(dx), rdx) <= TOL["bf16"]
    assert fro_rel_err(to_host(dws), rws) <= 1e-4 and fro_rel_err(to_host(dwo), rwo) <= 1e-4


@pytest.mark.parametrize("batch,n,width,schedule,causal,rounds", [
    (3, 64, 72, "rot", True, 2), (2, 16, 40, "rot", False, 2), (2, 64, 72, "mixa", True, 0),
    # width 8: one round only.  With 8 values per row, bf16 rounding of each
    # layer's output compounds without averaging: an exact bf16 chain (fp64
    # sums, every layer rounded) is already 2.4% from the fp64 oracle after 7
    # layers of 16 at window 256, beyond the tolerance, and ~1% after 4.
    (4, 16, 8, "rot", True, 1),
])
def test_stack_against_oracle(batch, n, width, schedule, causal, rounds):
    layers = (oracle.schedule_rot(rounds * oracle.log2n(n)) if schedule == "rot"
              else oracle.schedule_mixa(n))
    log(f"case: stack bf16 B={batch} n={n} w={width} {schedule} L={len(layers)} causal={causal}")
    s = inputs.make_stack(batch, n, width, len(layers), causal, "bf16", seed=width + n,
                          layers=layers)
    x = to_dev(s.x, "bf16")
    ws = [to_dev(w, "bf16") for w in s.w_self]
    wo = [to_dev(w, "bf16") for w in s.w_off]
    xs = hcmix.stack_forward(x, ws, wo, s.layers, s.causal)
    dx, dws, dwo = hcmix.stack_backward(xs, ws, wo, s.layers, to_dev(s.dy, "bf16"), s.causal)
    torch.cuda.synchronize()
    ref = oracle.stack_forward(s.x, s.w_self, s.w_off, s.layers, s.causal)
    rdx, rws, rwo = oracle.stack_backward(ref, s.w_self, s.w_off, s.layers, s.dy, s.causal)
    for l in range(1, len(layers) + 1):
        assert row_rel_err(to_host(xs[l]), ref[l]) <= TOL["bf16"], f"x_{l}"
    assert row_rel_err(to_host(dx), rdx) <= TOL["bf16"]
    for l in range(len(layers)):
        assert fro_rel_err(to_host(dws[l]), rws[l]) <= TOL["bf16"], f"dW_self {l}"
        assert fro_rel_err(to_host(dwo[l]), rwo[l]) <= TOL["bf16"], f"dW_off {l}"


def test_data_chain_and_weight_gradients_equal_the_stack_backward():
    """hcmix_stack_backward_data then hcmix_stack_weight_gradients, bitwise
    against hcmix_stack_backward (the same kernels in the same order)."""
    layers = oracle.schedule_rot(6)
    s = inputs.make_stack(2, 64, 40, len(layers), True, "bf16", seed=5, layers=layers)
    log("case: bf16 w=40 data chain + weight gradients vs stack backward")
    x = to_dev(s.x, "bf16")
    ws = [to_dev(w, "bf16") for w in s.w_self]
    wo = [to_dev(w, "bf16") for w in s.w_off]
    dy = to_dev(s.dy, "bf16")
    xs = hcmix.stack_forward(x, ws, wo, layers, True)
    dx, dws, dwo = hcmix.stack_backward(xs, ws, wo, layers, dy, True)
    dx2, grads = hcmix.stack_backward_data(ws, wo, layers, dy, True)
    gws, gwo = hcmix.stack_weight_gradients(xs[:len(layers)], [*grads, dy], layers, True)
    torch.cuda.synchronize()
    assert torch.equal(dx, dx2)
    for a, b in zip(dws + dwo, gws + gwo):
        assert torch.equal(a, b)


@pytest.mark.parametrize("width,schedule", [(24, "rot"), (72, "mixa")])
def test_decode_every_position(width, schedule):
    batch, n = 5, 16
    layers = oracle.schedule_rot(2 * oracle.log2n(n)) if schedule == "rot" else oracle.schedule_mixa(n)
    log(f"case: decode bf16 B={batch} n={n} w={width} {schedule}")
    s = inputs.make_stack(batch, n, width, len(layers), True, "bf16", seed=width, layers=layers,
                          with_dy=False)
    want = oracle.stack_forward(s.x, s.w_self, s.w_off, layers, True)[-1]
    x = to_dev(s.x, "bf16")
    ws = [to_dev(w, "bf16") for w in s.w_self]
    wo = [to_dev(w, "bf16") for w in s.w_off]
    cache = hcmix.alloc_decode_cache(batch, n, width, layers, x.dtype, x.device)
    cache.fill_(0xFF)          # never-written contents must never be read
    got = np.zeros_like(want)
    for pos in range(n):
        y = hcmix.decode_step(x[:, pos].contiguous(), ws, wo, layers, n, pos, cache)
        got[:, pos] = to_host(y)
    torch.cuda.synchronize()
    assert row_rel_err(got, want) <= TOL["bf16"]


def test_no_alloc_backward_equals_backward():
    batch, n, width = 4, 64, 72
    log(f"case: no-alloc backward bf16 w={width}")
    x, ws, wo, dy = inputs.make_layer(batch, n, width, "bf16", seed=9)
    tx, tws, two, tdy = (to_dev(a, "bf16") for a in (x, ws, wo, dy))
    dx, dws, dwo = hcmix.backward(tx, tws, two, tdy, 3, True)
    dx2 = torch.empty_like(dx)
    dws2, dwo2 = torch.empty_like(dws), torch.empty_like(dwo)
    hcmix.backward_no_alloc(tx, tws, two, tdy, 3, True, dx2, dws2, dwo2)
    torch.cuda.synchronize()
    assert torch.equal(dx, dx2) and torch.equal(dws, dws2) and torch.equal(dwo, dwo2)
