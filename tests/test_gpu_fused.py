"""The whole-stack entry points, in particular the fused small-width path
(bf16, width 64, n in {64, 128, 256}: every window resident in LDS across
layers), against the CPU oracle and against the layer-by-layer path."""
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


def gpu_stack(s, accumulate_into=None):
    x = to_dev(s.x, "bf16")
    ws = [to_dev(w, "bf16") for w in s.w_self]
    wo = [to_dev(w, "bf16") for w in s.w_off]
    xs = hcmix.stack_forward(x, ws, wo, s.layers, s.causal)
    kw = {}
    if accumulate_into is not None:
        kw = dict(dws=[t.clone() for t in accumulate_into[0]],
                  dwo=[t.clone() for t in accumulate_into[1]], accumulate=True)
    dx, dws, dwo = hcmix.stack_backward(xs, ws, wo, s.layers, to_dev(s.dy, "bf16"), s.causal, **kw)
    torch.cuda.synchronize()
    return xs, dx, dws, dwo


def schedule(kind, L, n):
    if kind == "rot":
        return oracle.schedule_rot(L)
    if kind == "fixed":
        return oracle.schedule_fixed(L)
    return oracle.schedule_gray(L)


@pytest.mark.parametrize("n", [64, 128, 256])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("kind", ["rot", "fixed", "gray"])
def test_fused_stack_matches_oracle(n, causal, kind):
    L = 2 * oracle.log2n(n) if kind != "gray" else 7
    batch = 3 if n == 64 else 5
    s = inputs.make_stack(batch=batch, n=n, width=64, num_layers=L, causal=causal, dtype="bf16",
                          seed=20 + n, layers=schedule(kind, L, n))
    log(f"fused n={n} causal={causal} {kind} L={L}")
    xs, dx, dws, dwo = gpu_stack(s)
    rxs = oracle.stack_forward(s.x, s.w_self, s.w_off, s.layers, causal)
    rdx, rws, rwo = oracle.stack_backward(rxs, s.w_self, s.w_off, s.layers, s.dy, causal)
    for l in range(1, L + 1):
        assert row_rel_err(to_host(xs[l]), rxs[l]) <= TOL["bf16"], f"x_{l}"
    assert row_rel_err(to_host(dx), rdx) <= TOL["bf16"]
    for l in range(L):
        assert fro_rel_err(to_host(dws[l]), rws[l]) <= TOL["bf16"], f"dW_self {l}"
        assert fro_rel_err(to_host(dwo[l]), rwo[l]) <= TOL["bf16"], f"dW_off {l}"


def test_fused_single_layer_weight_gradients_are_tight():
    """With one layer there is no bf16 chain: weight gradients only differ
    from the oracle by fp32 summation order."""
    for causal in (False, True):
        for layer in (0, 3, 7):
            s = inputs.make_stack(batch=4, n=256, width=64, num_layers=1, causal=causal,
                                  dtype="bf16", seed=30 + layer, layers=[layer])
            xs, dx, dws, dwo = gpu_stack(s)
            rx = oracle.forward(s.x, s.w_self[0], s.w_off[0], layer, causal)
            rdx, rws, rwo = oracle.backward(s.x, s.w_self[0], s.w_off[0], s.dy, layer, causal)
            assert row_rel_err(to_host(xs[1]), rx) <= TOL["bf16"]
            assert row_rel_err(to_host(dx), rdx) <= TOL["bf16"]
            assert fro_rel_err(to_host(dws[0]), rws) <= 1e-4
            assert fro_rel_err(to_host(dwo[0]), rwo) <= 1e-4


def test_fused_equals_layer_by_layer_forward_bitwise():
    """Each fused layer rounds once to bf16 exactly like hcmix_forward, and the
    fp32 sums run over the same k order, so the saved activations agree."""
    s = inputs.make_preset("reach", batch=8)
    x = to_dev(s.x, "bf16")
    ws = [to_dev(w, "bf16") for w in s.w_self]
    wo = [to_dev(w, "bf16") for w in s.w_off]
    xs = hcmix.stack_forward(x, ws, wo, s.layers, s.causal)
    cur = x
    for l, layer in enumerate(s.layers):
        cur = hcmix.forward(cur, ws[l], wo[l], layer, s.causal)
        torch.cuda.synchronize()
        diff = (cur.float() - xs[l + 1].float()).abs().max().item()
        scale = cur.float().abs().max().item()
        assert diff <= 1e-2 * scale, f"layer {l}: {diff} vs {scale}"
        cur = xs[l + 1]   # continue from the fused value so differences do not compound


def test_fused_accumulate_and_determinism():
    s = inputs.make_preset("reach", batch=16)
    _, dx1, dws1, dwo1 = gpu_stack(s)
    _, dx2, dws2, dwo2 = gpu_stack(s)
    assert torch.equal(dx1, dx2)
    for a, b in zip(dws1 + dwo1, dws2 + dwo2):
        assert torch.equal(a, b)
    base = ([torch.full_like(t, 0.5) for t in dws1], [torch.full_like(t, -1.0) for t in dwo1])
    _, _, dws3, dwo3 = gpu_stack(s, accumulate_into=base)
    for a, b in zip(dws3, dws1):
        np.testing.assert_allclose(to_host(a), to_host(b) + 0.5, rtol=0, atol=1e-4)
    for a, b in zip(dwo3, dwo1):
        np.testing.assert_allclose(to_host(a), to_host(b) - 1.0, rtol=0, atol=1e-4)


@pytest.mark.parametrize("causal", [False, True])
def test_fused_backward_split_invariance_and_unsplit_path(causal):
    """Small batches share each window's backward among up to four blocks
    (every block replays the dX chain and forms the weight gradients of its
    own layers); large batches run one block per window.  The same windows
    inside batches of 256, 128 and 64 (one, two and four blocks per window
    on 256 compute units) give bitwise the same dx, since the windows are
    independent; at batch 256, dx and the weight gradients against the
    oracle (the unsplit path)."""
    s = inputs.make_preset("reach", batch=256)
    if causal:
        s = inputs.make_stack(batch=256, n=256, width=64, num_layers=8, causal=True,
                              dtype="bf16", seed=11)
    log(f"case: fused backward split invariance B=256/128/64 n=256 w=64 L=8 causal={causal}")
    x = to_dev(s.x, "bf16")
    ws = [to_dev(w, "bf16") for w in s.w_self]
    wo = [to_dev(w, "bf16") for w in s.w_off]
    dy = to_dev(s.dy, "bf16")
    dxs = {}
    for b in (256, 128, 64):
        xs = hcmix.stack_forward(x[:b].contiguous(), ws, wo, s.layers, s.causal)
        dx, dws, dwo = hcmix.stack_backward(xs, ws, wo, s.layers, dy[:b].contiguous(), s.causal)
        torch.cuda.synchronize()
        dxs[b] = dx
        if b == 256:
            ref = oracle.stack_forward(s.x, s.w_self, s.w_off, s.layers, s.causal)
            rdx, rws, rwo = oracle.stack_backward(ref, s.w_self, s.w_off, s.layers, s.dy, s.causal)
            assert row_rel_err(to_host(dx), rdx) <= TOL["bf16"]
            e_w = max(fro_rel_err(to_host(g), r) for g, r in zip(dws + dwo, rws + rwo))
            log(f"  B=256 dW err {e_w:.2e}")
            assert e_w <= TOL["bf16"]
    assert torch.equal(dxs[128], dxs[256][:128])
    assert torch.equal(dxs[64], dxs[256][:64])


def test_layer_by_layer_stack_path_fp32_and_wide_bf16():
    """Shapes outside the fused path go layer by layer inside the library."""
    for (batch, n, width, dtype, causal) in [(2, 16, 32, "f32", False), (2, 64, 128, "bf16", True)]:
        s = inputs.make_stack(batch=batch, n=n, width=width, num_layers=5, causal=causal,
                              dtype=dtype, seed=40)
        x = to_dev(s.x, dtype)
        ws = [to_dev(w, dtype) for w in s.w_self]
        wo = [to_dev(w, dtype) for w in s.w_off]
        xs = hcmix.stack_forward(x, ws, wo, s.layers, causal)
        dx, dws, dwo = hcmix.stack_backward(xs, ws, wo, s.layers, to_dev(s.dy, dtype), causal)
        torch.cuda.synchronize()
        rxs = oracle.stack_forward(s.x, s.w_self, s.w_off, s.layers, causal)
        rdx, rws, rwo = oracle.stack_backward(rxs, s.w_self, s.w_off, s.layers, s.dy, causal)
        tol = TOL[dtype]
        assert row_rel_err(to_host(xs[-1]), rxs[-1]) <= tol
        assert row_rel_err(to_host(dx), rdx) <= tol
        for l in range(5):
            assert fro_rel_err(to_host(dws[l]), rws[l]) <= tol
            assert fro_rel_err(to_host(dwo[l]), rwo[l]) <= tol


def test_stack_rejects_aliasing_on_device():
    s = inputs.make_preset("reach", batch=2, num_layers=2)
    x = to_dev(s.x, "bf16")
    ws = [to_dev(w, "bf16") for w in s.w_self]
    wo = [to_dev(w, "bf16") for w in s.w_off]
    out = torch.empty_like(x)
    with pytest.raises(hcmix.HcmixError) as e:
        hcmix.stack_forward(x, ws, wo, s.layers, False, outs=[out, out])
    assert e.value.status == hcmix.HCMIX_ERR_INVALID_VALUE
    with pytest.raises(hcmix.HcmixError) as e:
        hcmix.stack_forward(x, ws, wo, s.layers, False, outs=[x, out])
    assert e.value.status == hcmix.HCMIX_ERR_INVALID_VALUE
