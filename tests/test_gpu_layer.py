"""Single-layer parity of the HIP path against the CPU oracle (through the C ABI).

Index work is compared bit-exactly; floating point within the stated
tolerances (util.TOL): 1e-5 for fp32, 2e-2 for bf16 with fp32 accumulation.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_18145_amd import hcmix, inputs
from tests.util import TOL, fro_rel_err, row_rel_err, to_dev, to_host, torch_dtype

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def log(msg):
    print(msg, flush=True)


# (batch, n, width, dtype): several tiles, ragged tails, n = 2, strides up to n/2 = 2048
SHAPES = [
    (2, 16, 32, "f32"), (3, 8, 40, "f32"), (1, 2, 8, "f32"), (1, 4096, 32, "f32"),
    (2, 16, 64, "bf16"), (3, 8, 64, "bf16"), (1, 2, 64, "bf16"), (5, 64, 192, "bf16"),
    (4, 256, 128, "bf16"), (1, 4096, 64, "bf16"), (2, 512, 256, "bf16"),
    (1, 64, 1024, "bf16"), (3, 32, 1280, "bf16"),      # 256-column tiles, ragged row tiles
    # bf16 widths that are a multiple of 8 but not of 64: the FMA kernels
    (2, 16, 8, "bf16"), (3, 8, 24, "bf16"), (2, 64, 72, "bf16"), (1, 512, 200, "bf16"),
    (2, 32, 96, "bf16"),
]


def probe_codes(rows, width):
    """x[r, c] = bit c of r for c < 15 (exact in bf16 and fp32)."""
    x = np.zeros((rows, width), dtype=np.float32)
    for c in range(min(width, 15)):
        x[:, c] = (np.arange(rows) >> c) & 1
    return x


def brute_partner(i, d):
    s = 2 ** d
    return i + s if (i // s) % 2 == 0 else i - s


@pytest.mark.parametrize("batch,n,width,dtype", SHAPES)
@pytest.mark.parametrize("causal", [False, True])
def test_index_probe_bit_exact(batch, n, width, dtype, causal):
    """W_self = 0, W_off = I: the output row is the partner's code (or zero
    where the link is masked), compared bit for bit with a brute-force partner."""
    log(f"probe {batch}x{n}x{width} {dtype} causal={causal}")
    rows = batch * n
    codes = probe_codes(rows, width)
    x = to_dev(codes.reshape(batch, n, width), dtype)
    zero = torch.zeros((width, width), dtype=torch_dtype(dtype), device="cuda")
    eye = torch.eye(width, dtype=torch_dtype(dtype), device="cuda")
    b = oracle.log2n(n)
    for layer in range(b):
        want = np.zeros_like(codes)
        want_dx = np.zeros_like(codes)
        for r in range(rows):
            t, i = divmod(r, n)
            p = t * n + brute_partner(i, layer)
            bit = (i >> layer) & 1
            if not causal or bit:
                want[r] = codes[p]
            if not causal or not bit:
                want_dx[r] = codes[p]
        y = hcmix.forward(x, zero, eye, layer, causal)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(y).reshape(rows, width), want), f"layer {layer}"
        # identity through the self map
        y2 = hcmix.forward(x, eye, zero, layer, causal)
        assert np.array_equal(to_host(y2).reshape(rows, width), codes)
        # backward: dx = W_off^T dy of the partner on the sending side
        dx, _, _ = hcmix.backward(x, zero, eye, x, layer, causal)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(dx).reshape(rows, width), want_dx), f"layer {layer} dx"


def layers_for(n):
    b = oracle.log2n(n)
    return list(range(b)) if b <= 4 else sorted({0, 1, b // 2, b - 1})


@pytest.mark.parametrize("batch,n,width,dtype", SHAPES)
@pytest.mark.parametrize("causal", [False, True])
def test_layer_forward_backward_parity(batch, n, width, dtype, causal):
    tol = TOL[dtype]
    for layer in layers_for(n):
        log(f"layer parity {batch}x{n}x{width} {dtype} causal={causal} layer={layer}")
        x, ws, wo, dy = inputs.make_layer(batch, n, width, dtype, seed=100 + layer)
        tx, tws, two, tdy = (to_dev(a, dtype) for a in (x, ws, wo, dy))
        y = hcmix.forward(tx, tws, two, layer, causal)
        dx, dws, dwo = hcmix.backward(tx, tws, two, tdy, layer, causal)
        torch.cuda.synchronize()
        ry = oracle.forward(x, ws, wo, layer, causal)
        rdx, rdws, rdwo = oracle.backward(x, ws, wo, dy, layer, causal)
        assert row_rel_err(to_host(y), ry) <= tol
        assert row_rel_err(to_host(dx), rdx) <= tol
        assert fro_rel_err(to_host(dws), rdws) <= tol
        assert fro_rel_err(to_host(dwo), rdwo) <= tol
        if dtype == "bf16":
            # weight gradients see no bf16 rounding: only fp32 summation order
            assert fro_rel_err(to_host(dws), rdws) <= 1e-4
            assert fro_rel_err(to_host(dwo), rdwo) <= 1e-4


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_weight_gradient_accumulate(dtype):
    batch, n, width = 2, 64, 64
    x, ws, wo, dy = inputs.make_layer(batch, n, width, dtype, seed=7)
    tx, tws, two, tdy = (to_dev(a, dtype) for a in (x, ws, wo, dy))
    _, g1, h1 = hcmix.backward(tx, tws, two, tdy, 3, True)
    base_s = torch.full_like(g1, 0.25)
    base_o = torch.full_like(h1, -0.5)
    _, g2, h2 = hcmix.backward(tx, tws, two, tdy, 3, True, dw_self=base_s.clone(),
                               dw_off=base_o.clone(), accumulate=True)
    torch.cuda.synchronize()
    np.testing.assert_allclose(to_host(g2), to_host(g1) + 0.25, rtol=0, atol=1e-5)
    np.testing.assert_allclose(to_host(h2), to_host(h1) - 0.5, rtol=0, atol=1e-5)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_repeated_calls_are_bitwise_identical(dtype):
    batch, n, width = 8, 256, 128
    x, ws, wo, dy = inputs.make_layer(batch, n, width, dtype, seed=11)
    tx, tws, two, tdy = (to_dev(a, dtype) for a in (x, ws, wo, dy))
    outs = []
    for _ in range(2):
        y = hcmix.forward(tx, tws, two, 5, True)
        dx, dws, dwo = hcmix.backward(tx, tws, two, tdy, 5, True)
        outs.append([t.clone() for t in (y, dx, dws, dwo)])
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [False, True])
def test_outputs_stay_inside_their_buffers(dtype, causal):
    """Outputs are views in the middle of NaN-filled buffers; the guard bands
    must come back untouched (compared as raw bits)."""
    batch, n, width = 3, 32, 64
    x, ws, wo, dy = inputs.make_layer(batch, n, width, dtype, seed=13)
    tx, tws, two, tdy = (to_dev(a, dtype) for a in (x, ws, wo, dy))
    td = torch_dtype(dtype)
    G = 4096
    numel = batch * n * width

    def guarded(count, dt):
        buf = torch.full((count + 2 * G,), float("nan"), dtype=dt, device="cuda")
        return buf, buf[G:G + count]

    ybuf, yv = guarded(numel, td)
    dxbuf, dxv = guarded(numel, td)
    sbuf, sv = guarded(width * width, torch.float32)
    obuf, ov = guarded(width * width, torch.float32)
    hcmix.forward(tx, tws, two, 2, causal, out=yv.view(batch, n, width))
    hcmix.backward(tx, tws, two, tdy, 2, causal, dx=dxv.view(batch, n, width),
                   dw_self=sv.view(width, width), dw_off=ov.view(width, width))
    torch.cuda.synchronize()
    for buf, count in ((ybuf, numel), (dxbuf, numel), (sbuf, width * width), (obuf, width * width)):
        guard = torch.cat([buf[:G], buf[G + count:]])
        assert torch.isnan(guard).all()
        assert not torch.isnan(buf[G:G + count]).any()


def test_device_side_validation():
    x = torch.zeros((2, 16, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((64, 64), dtype=torch.bfloat16, device="cuda")
    flat = torch.zeros(2 * 16 * 64 + 8, dtype=torch.bfloat16, device="cuda")
    misaligned = flat[1:1 + 2 * 16 * 64].view(2, 16, 64)
    with pytest.raises(hcmix.HcmixError) as e:
        hcmix.forward(misaligned, w, w, 0, False)
    assert e.value.status == hcmix.HCMIX_ERR_UNSUPPORTED
    with pytest.raises(hcmix.HcmixError) as e:
        hcmix.forward(x, w, w, 0, False, out=x)
    assert e.value.status == hcmix.HCMIX_ERR_INVALID_VALUE
