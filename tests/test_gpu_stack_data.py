"""hcmix_stack_backward_data (the dX chain alone, intermediate gradients kept)
followed by hcmix_stack_weight_gradients: every intermediate gradient against
the oracle's adjoint of its layer, and the pair against hcmix_stack_backward,
bitwise where both run the same kernels (layer-by-layer and deferred paths)."""
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


# (batch, n, width, layers, causal, dtype, (dx, dW) from the same kernels as
# hcmix_stack_backward)
CASES = [
    (4, 256, 512, list(range(16)), True, "bf16", (True, True)),   # deferred path
    (3, 64, 256, [oracle.NEAR, 5, oracle.NEAR, 2, 0, oracle.NEAR], True, "bf16", (True, True)),
    (2, 64, 192, [0, 5, 3], True, "bf16", (True, True)),          # layer by layer
    (3, 32, 128, [2], True, "bf16", (True, False)),               # one layer: split-K dW there
    (4, 128, 64, list(range(7)), False, "bf16", (False, False)),  # stack backward is fused here
    (2, 16, 32, [0, 1, 2, 3], False, "f32", (True, True)),
    (1, 512, 1024, [0, 8, 3], True, "bf16", (True, True)),       # 256-column mix tiles
    (3, 32, 1280, [4, 1], False, "bf16", (True, True)),          # ragged, bidirectional
]


@pytest.mark.parametrize("batch,n,width,layers,causal,dtype,same", CASES)
def test_data_chain_then_weight_gradients(batch, n, width, layers, causal, dtype, same):
    L = len(layers)
    print(f"case: stack backward data B={batch} n={n} w={width} layers={layers} causal={causal} "
          f"{dtype}", flush=True)
    s = inputs.make_stack(batch=batch, n=n, width=width, num_layers=L, causal=causal, dtype=dtype,
                          seed=61, layers=layers)
    x = to_dev(s.x, dtype)
    ws = [to_dev(w, dtype) for w in s.w_self]
    wo = [to_dev(w, dtype) for w in s.w_off]
    dy = to_dev(s.dy, dtype)
    xs = hcmix.stack_forward(x, ws, wo, layers, causal)
    dx, grads = hcmix.stack_backward_data(ws, wo, layers, dy, causal)
    assert len(grads) == L - 1
    outs = [*grads, dy]                       # gradient of each layer's output
    dws, dwo = hcmix.stack_weight_gradients(xs[:L], outs, layers, causal)
    torch.cuda.synchronize()

    # every layer's dX against the oracle's adjoint of that layer, fed the
    # library's own output gradient (no compounding)
    ins = [dx, *grads]
    for l in range(L):
        want, _, _ = oracle.backward(to_host(xs[l]), s.w_self[l], s.w_off[l], to_host(outs[l]),
                                     layers[l], causal)
        err = row_rel_err(to_host(ins[l]), want)
        assert err <= TOL[dtype], (l, err)

    ref_dx, ref_dws, ref_dwo = hcmix.stack_backward(xs, ws, wo, layers, dy, causal)
    torch.cuda.synchronize()
    if same[0]:
        assert torch.equal(dx, ref_dx)
    else:
        assert row_rel_err(to_host(dx), to_host(ref_dx)) <= TOL[dtype]
    for a, b in zip(dws + dwo, ref_dws + ref_dwo):
        if same[1]:
            assert torch.equal(a, b)
        else:
            # the same output gradients (bitwise dx chain): only the summation
            # order differs; otherwise the intermediate gradients may differ
            # in their bf16 rounding too
            assert fro_rel_err(to_host(a), to_host(b)) <= (1e-4 if same[0] else TOL[dtype])


def test_segments_then_one_weight_gradient_launch():
    """Two sparse segments with an elementwise layer between them (a stand-in
    for an attention layer): both segments' data chains, then the weight
    gradients of all their layers in one call, equal the two segments'
    stack backward calls."""
    batch, n, width = 4, 256, 256
    la, lb = [0, 1, 2], [3, 4, 5, 6, 7]
    L = len(la) + len(lb)
    s = inputs.make_stack(batch=batch, n=n, width=width, num_layers=L, causal=True, dtype="bf16",
                          seed=62, layers=la + lb)
    ws = [to_dev(w, "bf16") for w in s.w_self]
    wo = [to_dev(w, "bf16") for w in s.w_off]
    x = to_dev(s.x, "bf16")
    dy = to_dev(s.dy, "bf16")
    xa = hcmix.stack_forward(x, ws[:3], wo[:3], la, True)
    mid = (xa[-1].float() * 0.5).to(torch.bfloat16)
    xb = hcmix.stack_forward(mid, ws[3:], wo[3:], lb, True)
    gb_dx, gb = hcmix.stack_backward_data(ws[3:], wo[3:], lb, dy, True)
    ga_in = (gb_dx.float() * 0.5).to(torch.bfloat16)
    ga_dx, ga = hcmix.stack_backward_data(ws[:3], wo[:3], la, ga_in, True)
    dws, dwo = hcmix.stack_weight_gradients(xa[:3] + xb[:5], [*ga, ga_in, *gb, dy], la + lb, True)
    ra_dx, ra_ws, ra_wo = hcmix.stack_backward(xa, ws[:3], wo[:3], la, ga_in, True)
    rb_dx, rb_ws, rb_wo = hcmix.stack_backward(xb, ws[3:], wo[3:], lb, dy, True)
    torch.cuda.synchronize()
    assert torch.equal(gb_dx, rb_dx) and torch.equal(ga_dx, ra_dx)
    # the row-range split of the weight-gradient launch depends on the layer
    # count, so compare to tolerance, and each against the oracle
    for a, b in zip(dws + dwo, ra_ws + rb_ws + ra_wo + rb_wo):
        assert fro_rel_err(to_host(a), to_host(b)) <= 1e-4
    zero = np.zeros((width, width), dtype=np.float32)
    for l, (xl, gl) in enumerate(zip(xa[:3] + xb[:5], [*ga, ga_in, *gb, dy])):
        _, want_s, want_o = oracle.backward(to_host(xl), zero, zero, to_host(gl), (la + lb)[l], True)
        assert fro_rel_err(to_host(dws[l]), want_s) <= 1e-4
        assert fro_rel_err(to_host(dwo[l]), want_o) <= 1e-4
