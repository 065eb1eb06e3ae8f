"""Maximum sizes: activations of more than 2^31 elements (16386 windows of 256
positions at width 512, 4.3 GB per bf16 tensor), so that every element offset
past 2^31 goes through the kernels' 64-bit address arithmetic.

Forward and dX are compared with the oracle on whole windows (the first, a
middle one, the two on either side of element 2^31 and the last), each run
through the oracle on its own.  The weight gradients, sums over all 4.2
million rows, are checked by a property that holds at any size: they are
additive over windows, so the library's gradient of the whole batch must
equal the sum of its gradients of two halves whose offsets all fit in 31
bits (and the halves' path is the one the oracle tests check at smaller
sizes).  Inputs are seeded normal draws made on the device."""
import pytest
import torch

import oracle
from paper_2609_18145_amd import hcmix
from tests.util import TOL, fro_rel_err, row_rel_err, to_host

pytestmark = pytest.mark.gpu

B, N, W = 16386, 256, 512          # B * N * W = 2^31 + 2^18 elements
HALF = 8193                        # each half below 2^31 elements
WINDOWS = (0, 8191, 16383, 16384, 16385)   # window 16384 starts at element 2^31


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def log(msg):
    print(msg, flush=True)


def draw(shape, seed, scale=1.0):
    g = torch.Generator(device="cuda").manual_seed(seed)
    t = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    step = 1 << 28
    flat = t.view(-1)
    for i in range(0, flat.numel(), step):
        m = min(step, flat.numel() - i)
        flat[i:i + m] = (torch.randn(m, generator=g, device="cuda") * scale).to(torch.bfloat16)
    return t


def host_window(t, w):
    return to_host(t[w:w + 1])


def test_single_layer_beyond_2_31_elements():
    assert B * N * W > 2 ** 31 and HALF * N * W < 2 ** 31
    layer, causal = 7, True          # stride 128: partners across the tile halves
    log(f"case: single layer B={B} n={N} w={W} layer={layer} causal ({B * N * W} elements)")
    x = draw((B, N, W), 1)
    dy = draw((B, N, W), 2)
    ws = draw((W, W), 3, W ** -0.5)
    wo = draw((W, W), 4, W ** -0.5)
    y = hcmix.forward(x, ws, wo, layer, causal)
    dx, dws, dwo = hcmix.backward(x, ws, wo, dy, layer, causal)
    torch.cuda.synchronize()
    hws, hwo = to_host(ws), to_host(wo)
    for w in WINDOWS:
        xw, dyw = host_window(x, w), host_window(dy, w)
        ref = oracle.stack_forward(xw, [hws], [hwo], [layer], causal)
        rdx, _, _ = oracle.stack_backward(ref, [hws], [hwo], [layer], dyw, causal)
        e_y = row_rel_err(host_window(y, w), ref[-1])
        e_dx = row_rel_err(host_window(dx, w), rdx)
        log(f"  window {w}: y {e_y:.2e} dx {e_dx:.2e}")
        assert e_y <= TOL["bf16"] and e_dx <= TOL["bf16"]
    del y, dx
    # additivity of the weight gradients over windows
    _, s1, o1 = hcmix.backward(x[:HALF], ws, wo, dy[:HALF], layer, causal)
    _, s2, o2 = hcmix.backward(x[HALF:], ws, wo, dy[HALF:], layer, causal)
    torch.cuda.synchronize()
    e_s = fro_rel_err(to_host(dws), to_host(s1) + to_host(s2))
    e_o = fro_rel_err(to_host(dwo), to_host(o1) + to_host(o2))
    log(f"  dW additivity: self {e_s:.2e} off {e_o:.2e}")
    assert e_s <= 1e-5 and e_o <= 1e-5


def test_stack_beyond_2_31_elements():
    """Two causal layers through hcmix_stack_forward / _backward (the deferred
    path: dX chain, then one weight-gradient launch for both layers)."""
    layers, causal = [7, 0], True
    log(f"case: stack B={B} n={N} w={W} layers={layers} causal")
    x = draw((B, N, W), 11)
    dy = draw((B, N, W), 12)
    ws = [draw((W, W), 13 + i, W ** -0.5) for i in range(2)]
    wo = [draw((W, W), 15 + i, W ** -0.5) for i in range(2)]
    xs = hcmix.stack_forward(x, ws, wo, layers, causal)
    dx, dws, dwo = hcmix.stack_backward(xs, ws, wo, layers, dy, causal)
    torch.cuda.synchronize()
    hws, hwo = [to_host(w) for w in ws], [to_host(w) for w in wo]
    for w in WINDOWS:
        xw, dyw = host_window(x, w), host_window(dy, w)
        ref = oracle.stack_forward(xw, hws, hwo, layers, causal)
        rdx, _, _ = oracle.stack_backward(ref, hws, hwo, layers, dyw, causal)
        e_y = row_rel_err(host_window(xs[-1], w), ref[-1])
        e_dx = row_rel_err(host_window(dx, w), rdx)
        log(f"  window {w}: y {e_y:.2e} dx {e_dx:.2e}")
        assert e_y <= TOL["bf16"] and e_dx <= TOL["bf16"]
    del dx
    parts = []
    for sl in (slice(0, HALF), slice(HALF, B)):
        xh = [t[sl] for t in xs]
        _, a, b = hcmix.stack_backward(xh, ws, wo, layers, dy[sl], causal)
        parts.append((a, b))
    torch.cuda.synchronize()
    for l in range(2):
        e_s = fro_rel_err(to_host(dws[l]), to_host(parts[0][0][l]) + to_host(parts[1][0][l]))
        e_o = fro_rel_err(to_host(dwo[l]), to_host(parts[0][1][l]) + to_host(parts[1][1][l]))
        log(f"  layer {l} dW additivity: self {e_s:.2e} off {e_o:.2e}")
        assert e_s <= 1e-5 and e_o <= 1e-5
