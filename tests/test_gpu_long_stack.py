"""The long-window stack (n=4096, width 1024, 24 rotated causal layers: every
dimension twice, partner strides 1 .. 2048 rows) end to end through
hcmix_stack_forward / hcmix_stack_backward, in the launch configuration the
long-window workload uses: the 256-column mix tiles for the forward and for
the dX chain on transposed weight copies, then one weight-gradient launch
over 24 layers x 64 tiles with no row splits.

Batch 1 keeps every one of those kernel instances (only the number of row
tiles changes) while the oracle can still form every output, including all
48 weight gradients, in fp64."""
import time

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


@pytest.mark.timeout(600)
def test_long4096_whole_stack_against_oracle():
    s = inputs.make_preset("long4096", batch=1)
    L, dt = len(s.layers), s.dtype
    assert L == 24 and s.causal and s.x.shape == (1, 4096, 1024)
    log("case: long4096 whole stack, B=1 n=4096 w=1024 L=24 causal bf16, seed 0")
    x = to_dev(s.x, dt)
    ws = [to_dev(w, dt) for w in s.w_self]
    wo = [to_dev(w, dt) for w in s.w_off]
    dy = to_dev(s.dy, dt)
    xs = hcmix.stack_forward(x, ws, wo, s.layers, s.causal)
    dx, dws, dwo = hcmix.stack_backward(xs, ws, wo, s.layers, dy, s.causal)
    torch.cuda.synchronize()
    got_y, got_dx = to_host(xs[-1]), to_host(dx)
    got_dws = [to_host(t) for t in dws]
    got_dwo = [to_host(t) for t in dwo]
    log("  GPU done; oracle forward (fp64, no intermediate rounding)")

    t0 = time.perf_counter()
    ref = [s.x.astype(np.float64)]
    for l in range(L):
        ref.append(oracle.forward(ref[-1], s.w_self[l], s.w_off[l], s.layers[l], True))
        if l % 6 == 5:
            log(f"  oracle forward layer {l} done, {time.perf_counter() - t0:.0f} s")
    e_y = row_rel_err(got_y, ref[-1])
    log(f"  y row err {e_y:.3e}")
    assert e_y <= TOL["bf16"]

    g = s.dy.astype(np.float64)
    e_w = 0.0
    for l in reversed(range(L)):
        g, rws, rwo = oracle.backward(ref[l], s.w_self[l], s.w_off[l], g, s.layers[l], True)
        e_w = max(e_w, fro_rel_err(got_dws[l], rws), fro_rel_err(got_dwo[l], rwo))
        if l % 6 == 0:
            log(f"  oracle backward layer {l} done, {time.perf_counter() - t0:.0f} s, "
                f"dW fro err so far {e_w:.3e}")
    e_dx = row_rel_err(got_dx, g)
    log(f"  dx row err {e_dx:.3e}, dW fro err {e_w:.3e}")
    assert e_dx <= TOL["bf16"]
    assert e_w <= TOL["bf16"]


def probe_codes(rows, width):
    """x[r, c] = bit c of r for c < 15 (exact in bf16)."""
    x = np.zeros((rows, width), dtype=np.float32)
    for c in range(min(width, 15)):
        x[:, c] = (np.arange(rows) >> c) & 1
    return x


def brute_gather(v, n, d, take_when_bit):
    """Row r takes row (r's partner along d, found by adding or subtracting
    2^d) where bit d of its position equals take_when_bit, else zero."""
    rows = v.shape[0]
    out = np.zeros_like(v)
    s = 1 << d
    for r in range(rows):
        i = r % n
        bit = (i >> d) & 1
        if bit == take_when_bit:
            out[r] = v[r - s] if bit else v[r + s]
    return out


def test_long4096_index_probe_through_the_stack_paths():
    """W_self = 0, W_off = I on layers of dimension 9, 10 and 11 (strides 512
    to 2048 rows, across the 256-row tiles): the forward chain through
    hcmix_stack_forward and the dX chain through hcmix_stack_backward_data (the
    256-column mix tiles on transposed weight copies) are pure partner
    permutations of a code that is exact in bf16, compared bit for bit with a
    brute-force partner after every layer."""
    B, n, w = 2, 4096, 1024
    layers = [9, 10, 11]
    rows = B * n
    log(f"case: long4096 index probe B={B} n={n} w={w} layers={layers} causal")
    codes = probe_codes(rows, w)
    x = to_dev(codes.reshape(B, n, w), "bf16")
    zero = torch.zeros((w, w), dtype=torch.bfloat16, device="cuda")
    eye = torch.eye(w, dtype=torch.bfloat16, device="cuda")
    L = len(layers)
    xs = hcmix.stack_forward(x, [zero] * L, [eye] * L, layers, True)
    dx, grads = hcmix.stack_backward_data([zero] * L, [eye] * L, layers, x, True)
    torch.cuda.synchronize()
    # forward: receivers (bit d set) take the partner below them
    want = codes
    for l, d in enumerate(layers):
        want = brute_gather(want, n, d, 1)
        assert np.array_equal(to_host(xs[l + 1]).reshape(rows, w), want), f"forward layer {l}"
    # dX: senders (bit d clear) take the gradient of the partner above them
    outs = [dx, *grads]          # outs[l] = gradient of layer l's input
    want = codes
    for l in reversed(range(L)):
        want = brute_gather(want, n, layers[l], 0)
        assert np.array_equal(to_host(outs[l]).reshape(rows, w), want), f"dX layer {l}"
